"""MI355X (gfx950) sparse-decode attention for Sparrow's sparse rollout (arXiv 2606.08446).

Modules: ``sparrow`` (binding of the C ABI in include/sparrow.h; the kernels are in
``csrc/``), ``workloads`` (seeded synthetic inputs), ``cost_model`` (the paper's rollout
cost model), ``build`` (compiles libsparrow.so for gfx950).
"""
