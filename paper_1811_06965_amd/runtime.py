"""Torch-facing driver of one partition (marshalling only).

Torch provides device memory and the stream; every step of the partition's
work runs in libgp.so.  ``Partition.step`` issues GPipe's schedule for one
mini-batch (Section 2.2): M forwards in order, M re-materialising backwards in
reverse order, then the one synchronous update.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import gp

# One second stream per device for the odd micro-batches, created by the
# library once per process (a stream from torch's pool may share a hardware
# queue with one of the library's streams).
_SECOND_STREAM: Dict[int, "torch.cuda.ExternalStream"] = {}


def second_stream():
    dev = torch.cuda.current_device()
    if dev not in _SECOND_STREAM:
        _SECOND_STREAM[dev] = torch.cuda.ExternalStream(gp.gp_stream_create(), device=dev)
    return _SECOND_STREAM[dev]


DTYPES = {"f32": (gp.GP_F32, torch.float32), "bf16": (gp.GP_BF16, torch.bfloat16)}
KINDS = {"encoder": gp.GP_ENCODER, "decoder": gp.GP_DECODER_CROSS}
LOSSES = {"none": gp.GP_LOSS_NONE, "mse": gp.GP_LOSS_MSE, "xent_ls": gp.GP_LOSS_XENT_LS}
OPTIMIZERS = {"sgd": gp.GP_OPT_SGD, "rmsprop": gp.GP_OPT_RMSPROP}


def make_config(cfg, micro: Optional[int] = None, check_finite: bool = False,
                keep_activations: bool = False) -> gp.gp_config:
    M = cfg.micro if micro is None else micro
    if cfg.batch % M:
        raise ValueError("mini-batch must split into M equal micro-batches")
    c = gp.gp_config()
    c.seq_len = cfg.seq
    c.seqs_per_microbatch = cfg.batch // M
    c.num_microbatches = M
    c.dtype = DTYPES[cfg.dtype][0]
    c.kind = KINDS[cfg.kind]
    c.mem_seq_len = cfg.mem_seq
    c.loss = LOSSES[cfg.loss]
    c.vocab = cfg.vocab
    c.label_smoothing = cfg.label_smoothing
    c.ln_eps = cfg.ln_eps
    c.check_finite = 1 if check_finite else 0
    c.keep_activations = 1 if keep_activations else 0
    c.optimizer = OPTIMIZERS[cfg.optimizer]
    if cfg.optimizer == "rmsprop":
        c.rms_decay = cfg.rms_decay
        c.rms_eps = cfg.rms_eps
    c.logit_clip = cfg.logit_clip
    return c


class Partition:
    """One configured partition on the current HIP device."""

    def __init__(self, cfg, micro: Optional[int] = None, check_finite: bool = False,
                 keep_activations: bool = False):
        self.cfg = cfg
        self.M = cfg.micro if micro is None else micro
        self.tdtype = DTYPES[cfg.dtype][1]
        self._lane = None  # second stream for the odd micro-batches
        self.h = gp.gp_partition_create(cfg.layers, cfg.d_model, cfg.d_ff, cfg.heads)
        try:
            gp.gp_partition_configure(self.h, make_config(cfg, self.M, check_finite, keep_activations))
        except Exception:
            gp.gp_partition_destroy(self.h)
            raise

    def close(self):
        if self.h is not None:
            gp.gp_partition_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # -------------------------------------------------------------- params
    def load_params(self, layers: List[Dict[str, np.ndarray]], head: Dict[str, np.ndarray]):
        for l, p in enumerate(layers):
            for name, arr in p.items():
                gp.gp_set_param(self.h, l, gp.PARAM_ID[name], np.ascontiguousarray(arr, dtype=np.float32))
        for name, arr in head.items():
            gp.gp_set_param(self.h, -1, gp.PARAM_ID[name], np.ascontiguousarray(arr, dtype=np.float32))

    def _read(self, fn, shapes_layers, shapes_head):
        layers = []
        for l in range(self.cfg.layers):
            d = {}
            for name, shp in shapes_layers.items():
                a = np.empty(shp, dtype=np.float32)
                fn(self.h, l, gp.PARAM_ID[name], a)
                d[name] = a
            layers.append(d)
        head = {}
        for name, shp in shapes_head.items():
            a = np.empty(shp, dtype=np.float32)
            fn(self.h, -1, gp.PARAM_ID[name], a)
            head[name] = a
        return layers, head

    def grads(self):
        return self._read(gp.gp_get_grad, self.cfg.param_shapes(), self.cfg.head_shapes())

    def params(self):
        return self._read(gp.gp_get_param, self.cfg.param_shapes(), self.cfg.head_shapes())

    def memory(self):
        return gp.gp_partition_memory(self.h)

    def param_count(self):
        return gp.gp_param_count(self.h)

    # ------------------------------------------------------------ schedule
    def device_inputs(self, case, device="cuda"):
        """Move a synthetic case's boundary tensors to the device."""
        t = lambda a: torch.tensor(a, dtype=torch.float32).to(device=device, dtype=self.tdtype).contiguous()
        out = {"x": t(case["x"]), "mem": None if case.get("mem") is None else t(case["mem"])}
        if self.cfg.loss == "mse":
            out["dy"] = t(case["target"])
        elif self.cfg.loss == "none":
            out["dy"] = t(case["dy"])
        else:
            out["dy"] = torch.tensor(case["labels"], dtype=torch.int32, device=device).contiguous()
        return out

    def step(self, x, mem, dy, lr=0.0, want_y=True, want_dx=True, want_dmem=True, want_loss=True,
             stream=None, y=None, dx=None, dmem=None, want_recomputed=False, noalloc=False, fwd_streams=2,
             bwd_streams=2):
        """One mini-batch through GPipe's schedule.  x/mem/dy: device tensors
        of the whole mini-batch (dim 0 = sequences).  Returns dict(y, dx, dmem,
        loss); with want_recomputed also "y_remat", the partition output as
        each backward call re-materialised it (gp_recomputed_output), in
        mini-batch order.  noalloc: the forwards go through
        gp_forward_microbatch_noalloc.  fwd_streams=2: the odd micro-batches'
        forwards are issued on a second stream, so that consecutive forwards
        run side by side (the library keeps one first-pass slot per parity);
        the launch stream waits for it before the backwards.  bwd_streams=2:
        likewise the odd micro-batches' backwards (the library runs the two
        members of a recompute pair side by side where it has two backward
        lanes, and orders them itself otherwise); the launch stream waits for
        the second stream before the update."""
        M = self.M
        main = torch.cuda.current_stream() if stream is None else torch.cuda.ExternalStream(stream)
        st = main.cuda_stream
        lanes = [st]
        if (fwd_streams > 1 or bwd_streams > 1) and M > 1 and self._lane is None:
            self._lane = second_stream()
        if fwd_streams > 1 and M > 1:
            self._lane.wait_stream(main)
            lanes.append(self._lane.cuda_stream)
        if want_y and y is None:
            y = torch.empty_like(x)
        if want_dx and dx is None:
            dx = torch.empty_like(x)
        if mem is not None and want_dmem and dmem is None:
            dmem = torch.empty_like(mem)
        xs = x.chunk(M)
        ms = mem.chunk(M) if mem is not None else [None] * M
        ys = y.chunk(M) if y is not None else [None] * M
        dys = dy.chunk(M)
        dxs = dx.chunk(M) if dx is not None else [None] * M
        dms = dmem.chunk(M) if dmem is not None else [None] * M
        ptr = lambda t: None if t is None else t.data_ptr()
        fwd = gp.gp_forward_microbatch_noalloc if noalloc else gp.gp_forward_microbatch
        for m in range(M):
            fwd(self.h, m, ptr(xs[m]), ptr(ms[m]), ptr(ys[m]), lanes[m % len(lanes)])
        if len(lanes) > 1:
            main.wait_stream(self._lane)
        y_remat = torch.empty_like(x) if want_recomputed else None
        yr = y_remat.chunk(M) if want_recomputed else None
        blanes = [st]
        if bwd_streams > 1 and M > 1:
            self._lane.wait_stream(main)
            blanes.append(self._lane.cuda_stream)
        for m in range(M - 1, -1, -1):
            bs = blanes[m % len(blanes)]
            gp.gp_backward_microbatch_remat(self.h, m, ptr(dys[m]), ptr(dxs[m]), ptr(dms[m]), bs)
            if want_recomputed:
                gp.gp_recomputed_output(self.h, ptr(yr[m]), bs)
        if len(blanes) > 1:
            main.wait_stream(self._lane)
        loss = gp.gp_accumulate_and_step(self.h, lr, want_loss, st)
        out = {"y": y, "dx": dx, "dmem": dmem, "loss": loss}
        if want_recomputed:
            out["y_remat"] = y_remat
        return out

    def capture_step(self, x, mem, dy, lr=0.0, dx=None, dmem=None, want_y=False, y=None):
        """Capture one whole mini-batch step (M forwards, M backwards, the
        update) into a HIP graph on a capture stream and return it; replay()
        runs the step again on the same buffers.  The capture itself runs no
        work.  The loss is not read (that would synchronise), and the
        partition must not check gradients for finiteness (same reason).
        The step is captured on the capture stream alone (one stream for the
        forwards and the backwards): a capture of the step issued over two
        streams ended in a segmentation fault inside the HIP runtime's end of
        capture, cause not found."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(x, mem, dy, lr=lr, want_y=want_y, want_dx=dx is not None, want_dmem=dmem is not None,
                      want_loss=False, y=y, dx=dx, dmem=dmem, fwd_streams=1, bwd_streams=1)
        return g

    # ------------------------------------------------------------ timers
    def timer_select(self, role):
        """role: a name from gp.KERNEL_ROLES, "all", or None to stop."""
        r = gp.GP_K_NONE if role is None else gp.GP_K_COUNT if role == "all" else gp.KERNEL_ROLE[role]
        gp.gp_timer_select(self.h, r)

    def timer_read(self, role):
        ms, n, flops, nbytes = gp.gp_timer_read(self.h, gp.KERNEL_ROLE[role])
        return {"ms": ms, "launches": n, "flops": flops, "bytes": nbytes}

    def timer_reset(self):
        gp.gp_timer_reset(self.h)

    def timer_sample(self, every):
        """Time one launch in `every` of the selected role (1: all)."""
        gp.gp_timer_sample(self.h, every)
