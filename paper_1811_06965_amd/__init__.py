"""MI355X-native hot path of GPipe's micro-batch pipelining: one partition.

The work (forward over M micro-batches keeping only boundary inputs,
re-materialising backward in reverse micro-batch order, in-place fp32
gradient accumulation, one synchronous update) runs in the HIP kernels of
``_lib/libgp.so`` behind the C ABI declared in ``include/gp.h``.  ``gp`` is
its ctypes binding; ``runtime`` adds torch-tensor convenience on top.
"""
from . import gp  # noqa: F401
