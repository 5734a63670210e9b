"""tfk: MI355X (gfx950) kernels for one synchronous SGD step of a convnet replica.

``ops`` binds the C ABI of libtfk.so (include/tfk.h) over torch device
tensors; ``step.Replica`` drives a whole step of a workload from
``workloads``.  The HIP library must be built first
(``python -m paper_1605_08695_amd.build``); nothing here falls back to the CPU.
"""
__all__ = ["ops", "step", "workloads", "build"]
