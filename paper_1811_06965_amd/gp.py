"""ctypes binding of the partition's C ABI (include/gp.h).

Argument marshalling only: every step of the partition's work runs in the HIP
kernels of libgp.so.  Device buffers are passed as integer device addresses
(e.g. ``tensor.data_ptr()``) and streams as raw HIP stream handles (e.g.
``torch.cuda.current_stream().cuda_stream``).  If the library has not been
built the import-time loader raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libgp.so")

GP_OK, GP_ERR_INVALID_ARG, GP_ERR_STATE, GP_ERR_OOM, GP_ERR_HIP, GP_ERR_NONFINITE, GP_ERR_UNSUPPORTED = range(7)
STATUS_NAMES = {0: "GP_OK", 1: "GP_ERR_INVALID_ARG", 2: "GP_ERR_STATE", 3: "GP_ERR_OOM", 4: "GP_ERR_HIP",
                5: "GP_ERR_NONFINITE", 6: "GP_ERR_UNSUPPORTED"}
GP_F32, GP_BF16 = 0, 1
GP_ENCODER, GP_DECODER_CROSS = 0, 1
GP_LOSS_NONE, GP_LOSS_MSE, GP_LOSS_XENT_LS = 0, 1, 2
GP_OPT_SGD, GP_OPT_RMSPROP = 0, 1

PARAM_IDS = ["ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "ln2_g", "ln2_b",
             "w1", "b1", "w2", "b2", "xwq", "xbq", "xwk", "xbk", "xwv", "xbv", "xwo", "xbo",
             "ln3_g", "ln3_b", "lnf_g", "lnf_b", "wout", "bout"]
PARAM_ID = {name: i for i, name in enumerate(PARAM_IDS)}

# gp_kernel_role: launch roles of the timers
KERNEL_ROLES = ["none", "qkv.fwd", "qkv.dx", "qkv.dw", "o.fwd", "o.dx", "o.dw", "ffn1.fwd", "ffn1.dx", "ffn1.dw",
                "ffn2.fwd", "ffn2.dx", "ffn2.dw", "xq.fwd", "xq.dx", "xq.dw", "xkv.fwd", "xkv.dx", "xkv.dw",
                "xo.fwd", "xo.dx", "xo.dw", "head.fwd", "head.dx", "head.dw", "attn.fwd", "attn.bwd",
                "xattn.fwd", "xattn.bwd", "ln.fwd", "ln.bwd"]
KERNEL_ROLE = {name: i for i, name in enumerate(KERNEL_ROLES)}
GP_K_NONE, GP_K_COUNT = 0, len(KERNEL_ROLES)

EXPORTS = ["gp_partition_create", "gp_partition_configure", "gp_partition_destroy", "gp_set_param",
           "gp_get_param", "gp_get_grad", "gp_partition_memory", "gp_param_count", "gp_forward_microbatch",
           "gp_backward_microbatch_remat", "gp_accumulate_and_step", "gp_timer_select", "gp_timer_read",
           "gp_timer_reset", "gp_timer_sample", "gp_mfma_peak", "gp_recomputed_output", "gp_memory_plan",
           "gp_forward_microbatch_noalloc", "gp_plan_cells", "gp_stream_create", "gp_stream_destroy", "gp_last_error"]


class gp_config(ctypes.Structure):
    _fields_ = [("seq_len", ctypes.c_int), ("seqs_per_microbatch", ctypes.c_int),
                ("num_microbatches", ctypes.c_int), ("dtype", ctypes.c_int), ("kind", ctypes.c_int),
                ("mem_seq_len", ctypes.c_int), ("loss", ctypes.c_int), ("vocab", ctypes.c_int),
                ("label_smoothing", ctypes.c_float), ("ln_eps", ctypes.c_float),
                ("check_finite", ctypes.c_int), ("keep_activations", ctypes.c_int), ("optimizer", ctypes.c_int),
                ("rms_decay", ctypes.c_float), ("rms_eps", ctypes.c_float), ("logit_clip", ctypes.c_float)]


class GpError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libgp.so (once).  Raises if it is missing: build it first."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build the HIP library first (python -m paper_1811_06965_amd.build)")
    lib = ctypes.CDLL(path)
    P, VP, I, SZ = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    FP = ctypes.POINTER(ctypes.c_float)
    lib.gp_partition_create.argtypes = [I, I, I, I, ctypes.POINTER(P)]
    lib.gp_partition_configure.argtypes = [P, ctypes.POINTER(gp_config)]
    lib.gp_partition_destroy.argtypes = [P]
    for f in (lib.gp_set_param, lib.gp_get_param, lib.gp_get_grad):
        f.argtypes = [P, I, I, FP, SZ]
    lib.gp_partition_memory.argtypes = [P] + [ctypes.POINTER(SZ)] * 4
    lib.gp_param_count.argtypes = [P, ctypes.POINTER(SZ)]
    lib.gp_forward_microbatch.argtypes = [P, I, VP, VP, VP, VP]
    lib.gp_forward_microbatch_noalloc.argtypes = [P, I, VP, VP, VP, VP]
    lib.gp_plan_cells.argtypes = [ctypes.POINTER(ctypes.c_double), I, I, ctypes.POINTER(ctypes.c_int),
                                  ctypes.POINTER(ctypes.c_double)]
    lib.gp_backward_microbatch_remat.argtypes = [P, I, VP, VP, VP, VP]
    lib.gp_accumulate_and_step.argtypes = [P, ctypes.c_float, ctypes.POINTER(ctypes.c_double), VP]
    D = ctypes.POINTER(ctypes.c_double)
    lib.gp_timer_select.argtypes = [P, I]
    lib.gp_timer_read.argtypes = [P, I, D, ctypes.POINTER(ctypes.c_long), D, D]
    lib.gp_timer_reset.argtypes = [P]
    lib.gp_timer_sample.argtypes = [P, I]
    lib.gp_mfma_peak.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]
    lib.gp_recomputed_output.argtypes = [P, VP, VP]
    lib.gp_stream_create.argtypes = [ctypes.POINTER(VP)]
    lib.gp_stream_destroy.argtypes = [VP]
    lib.gp_memory_plan.argtypes = [I, I, I, I, ctypes.POINTER(gp_config)] + [ctypes.POINTER(SZ)] * 4
    lib.gp_last_error.argtypes = []
    lib.gp_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name != "gp_last_error":
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def gp_last_error() -> str:
    return load().gp_last_error().decode()


def _check(status):
    if status != GP_OK:
        raise GpError(status, gp_last_error())


def _fptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


# --- one function per C entry point, same names -------------------------------
def gp_partition_create(layers, d_model, d_ff, heads):
    h = ctypes.c_void_p()
    _check(load().gp_partition_create(layers, d_model, d_ff, heads, ctypes.byref(h)))
    return h


def gp_partition_configure(h, cfg: gp_config):
    _check(load().gp_partition_configure(h, ctypes.byref(cfg)))


def gp_partition_destroy(h):
    _check(load().gp_partition_destroy(h))


def gp_set_param(h, layer, pid, host):
    """host: C-contiguous float32 numpy array."""
    _check(load().gp_set_param(h, layer, pid, _fptr(host), host.size))


def gp_get_param(h, layer, pid, host):
    _check(load().gp_get_param(h, layer, pid, _fptr(host), host.size))


def gp_get_grad(h, layer, pid, host):
    _check(load().gp_get_grad(h, layer, pid, _fptr(host), host.size))


def gp_partition_memory(h):
    v = [ctypes.c_size_t() for _ in range(4)]
    _check(load().gp_partition_memory(h, *[ctypes.byref(x) for x in v]))
    return dict(params=v[0].value, grads=v[1].value, stash=v[2].value, workspace=v[3].value)


def gp_memory_plan(layers, d_model, d_ff, heads, cfg: gp_config):
    """Byte counts of a partition configured with cfg, computed on the host."""
    v = [ctypes.c_size_t() for _ in range(4)]
    _check(load().gp_memory_plan(layers, d_model, d_ff, heads, ctypes.byref(cfg), *[ctypes.byref(x) for x in v]))
    return dict(params=v[0].value, grads=v[1].value, stash=v[2].value, workspace=v[3].value)


def gp_plan_cells(costs, cells):
    """Least-variance split of the layers (costs: 1-D float array) into
    `cells` cells; returns (first layer of each cell, variance)."""
    import numpy as np
    c = np.ascontiguousarray(costs, dtype=np.float64)
    first = (ctypes.c_int * max(cells, 1))()
    var = ctypes.c_double()
    _check(load().gp_plan_cells(c.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), c.size, cells, first,
                                ctypes.byref(var)))
    return [int(v) for v in first[:cells]], var.value


def gp_param_count(h):
    v = ctypes.c_size_t()
    _check(load().gp_param_count(h, ctypes.byref(v)))
    return v.value


def gp_forward_microbatch(h, mb, x, mem, y, stream):
    _check(load().gp_forward_microbatch(h, mb, x, mem, y, stream))


def gp_forward_microbatch_noalloc(h, mb, x, mem, y, stream):
    _check(load().gp_forward_microbatch_noalloc(h, mb, x, mem, y, stream))


def gp_backward_microbatch_remat(h, mb, dy_or_target, dx, dmem, stream):
    _check(load().gp_backward_microbatch_remat(h, mb, dy_or_target, dx, dmem, stream))


def gp_accumulate_and_step(h, lr, want_loss, stream):
    if want_loss:
        v = ctypes.c_double()
        _check(load().gp_accumulate_and_step(h, lr, ctypes.byref(v), stream))
        return v.value
    _check(load().gp_accumulate_and_step(h, lr, None, stream))
    return None


def gp_timer_select(h, role):
    _check(load().gp_timer_select(h, role))


def gp_timer_read(h, role):
    """(milliseconds, launches, FLOPs, bytes) of one launch role."""
    ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    n = ctypes.c_long()
    _check(load().gp_timer_read(h, role, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl), ctypes.byref(by)))
    return ms.value, n.value, fl.value, by.value


def gp_timer_reset(h):
    _check(load().gp_timer_reset(h))


def gp_timer_sample(h, every):
    _check(load().gp_timer_sample(h, every))


def gp_stream_create():
    """A non-blocking stream of default priority (its raw handle)."""
    s = ctypes.c_void_p()
    _check(load().gp_stream_create(ctypes.byref(s)))
    return s.value


def gp_stream_destroy(stream):
    _check(load().gp_stream_destroy(stream))


def gp_recomputed_output(h, y, stream):
    """y: device address of an [n, S, D] buffer in the partition dtype."""
    _check(load().gp_recomputed_output(h, y, stream))


def gp_mfma_peak(stream=None):
    """Sustained bf16 MFMA-loop rate of the current device, TFLOP/s."""
    t = ctypes.c_double()
    _check(load().gp_mfma_peak(stream, ctypes.byref(t)))
    return t.value
