"""MI355X-native multi-stage KV-cache live migration (Llumnix, arXiv 2406.03243).

The migration path is the HIP library ``libllmig.so`` (C ABI declared in
``include/llmig.h``), built in-tree for gfx950 and bound to Python by
:mod:`paper_2406_03243_amd.llmig`.  :mod:`paper_2406_03243_amd.workloads`
draws the seeded synthetic inputs.
"""
