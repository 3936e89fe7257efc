"""PHub exchange step on MI355X: a fused, chunk-scheduled N-way gradient sum
plus momentum/Nesterov SGD with weight decay, as a HIP library with a C
interface (``include/phub.h``) and a thin Python binding (``phub``).

Importing the package loads nothing; ``paper_1805_07891_amd.phub.load()``
loads the built library, and ``paper_1805_07891_amd.job`` wraps one job
around torch-allocated device memory.
"""
