"""Seeded synthetic workloads shared by the oracle, the tests and the benchmark.

This module holds the workload *shapes* and the random draws only; none of the
method's arithmetic lives here.  Both the fp64 CPU oracle and the HIP path
receive exactly the arrays produced below (after the optional storage-precision
rounding), so parity measures compute error and not input quantisation.

Generation order (fixed, so a seed names one case): for each layer in turn the
parameters in parameter-id order, then the loss head's parameters, then the
boundary input X [N, S, D], then the decoder memory [N, S_mem, D], then the
loss-specific tensor (MSE targets, boundary gradients, or token labels).

Distributions (the workload recipe of the partition configurations):
  * weight matrices: Xavier-uniform, U(-a, a) with a = sqrt(6 / (fan_in + fan_out))
    per logical [in, out] matrix; with ``fixup_layers`` = L > 0 the feed-forward
    matrices w1 and w2 are drawn the same way and divided by L (the scaled-down
    feed-forward initialisation of the paper's Section 5);
  * biases 0, LayerNorm gain 1 and shift 0 -- unless ``perturb`` is set, in
    which case they are drawn as N(0, 0.1^2) (biases, shifts) and
    1 + N(0, 0.1^2) (gains) so that every parameter path carries signal;
  * X, memory, MSE targets and boundary gradients: N(0, 1);
  * labels: uniform integers in [0, vocab).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# Parameter ids, in the order the C ABI enumerates them.  Per-layer ids apply
# to layers 0..L-1; head ids apply to the loss head (layer index -1).
ENCODER_PARAMS = ["ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv",
                  "wo", "bo", "ln2_g", "ln2_b", "w1", "b1", "w2", "b2"]
DECODER_EXTRA = ["xwq", "xbq", "xwk", "xbk", "xwv", "xbv", "xwo", "xbo",
                 "ln3_g", "ln3_b"]
HEAD_PARAMS = ["lnf_g", "lnf_b", "wout", "bout"]
PARAM_IDS = ENCODER_PARAMS + DECODER_EXTRA + HEAD_PARAMS


@dataclasses.dataclass(frozen=True)
class PartitionConfig:
    """One pipeline partition workload.

    layers, d_model, d_ff, heads: the partition's Transformer stack.
    seq: sequence length S; batch: mini-batch N in sequences; micro: M.
    kind: "encoder" (pre-LN self-attention + FFN) or "decoder" (causal
    self-attention, cross-attention to a memory, FFN).
    loss: "none" (gradients arrive at the boundary), "mse" or "xent_ls".
    """
    name: str
    layers: int
    d_model: int
    d_ff: int
    heads: int
    seq: int
    batch: int
    micro: int
    dtype: str = "bf16"          # "f32" or "bf16" (bf16 operands, fp32 accumulation)
    kind: str = "encoder"
    loss: str = "none"
    vocab: int = 0
    label_smoothing: float = 0.0
    mem_seq: int = 0
    ln_eps: float = 1e-5
    # the one synchronous update: "sgd" or "rmsprop" (decay rho, eps inside the square root)
    optimizer: str = "sgd"
    rms_decay: float = 0.9
    rms_eps: float = 1e-10
    # cross-entropy head: clip the logits to [-logit_clip, logit_clip] (0 = off)
    logit_clip: float = 0.0
    # initialisation: > 0 divides the Xavier-uniform draws of the feed-forward
    # matrices (w1, w2) by this number of layers of the whole model
    fixup_layers: int = 0

    @property
    def d_head(self) -> int:
        return self.d_model // self.heads

    @property
    def micro_batch(self) -> int:
        return self.batch // self.micro

    def with_(self, **kw) -> "PartitionConfig":
        return dataclasses.replace(self, **kw)

    def param_shapes(self) -> Dict[str, tuple]:
        """Logical shapes of one layer's parameters (W stored as [in, out])."""
        D, F = self.d_model, self.d_ff
        shp = {"ln1_g": (D,), "ln1_b": (D,),
               "wq": (D, D), "bq": (D,), "wk": (D, D), "bk": (D,),
               "wv": (D, D), "bv": (D,), "wo": (D, D), "bo": (D,),
               "ln2_g": (D,), "ln2_b": (D,),
               "w1": (D, F), "b1": (F,), "w2": (F, D), "b2": (D,)}
        if self.kind == "decoder":
            shp.update({"xwq": (D, D), "xbq": (D,), "xwk": (D, D), "xbk": (D,),
                        "xwv": (D, D), "xbv": (D,), "xwo": (D, D), "xbo": (D,),
                        "ln3_g": (D,), "ln3_b": (D,)})
        return shp

    def head_shapes(self) -> Dict[str, tuple]:
        if self.loss != "xent_ls":
            return {}
        D, V = self.d_model, self.vocab
        return {"lnf_g": (D,), "lnf_b": (D,), "wout": (D, V), "bout": (V,)}


# The five partition workloads (tiny parity case, encoder partitions of
# growing width, and the final decoder partition with its vocabulary head).
CONFIGS: Dict[str, PartitionConfig] = {
    "tiny": PartitionConfig("tiny", layers=2, d_model=64, d_ff=256, heads=4, seq=32,
                            batch=8, micro=4, dtype="f32", loss="mse"),
    "enc512": PartitionConfig("enc512", layers=8, d_model=512, d_ff=2048, heads=8, seq=128,
                              batch=32, micro=8, dtype="bf16", loss="mse"),
    "enc1024": PartitionConfig("enc1024", layers=16, d_model=1024, d_ff=8192, heads=16,
                               seq=256, batch=64, micro=8, dtype="bf16", loss="none"),
    "enc2048": PartitionConfig("enc2048", layers=8, d_model=2048, d_ff=16384, heads=32,
                               seq=256, batch=128, micro=32, dtype="bf16", loss="none"),
    "dec1024": PartitionConfig("dec1024", layers=8, d_model=1024, d_ff=8192, heads=16,
                               seq=256, batch=64, micro=16, dtype="bf16", kind="decoder",
                               loss="xent_ls", vocab=32000, label_smoothing=0.1, mem_seq=256),
}


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned as float64.

    Storage-precision rounding of the generated inputs: the value first goes to
    float32, whose top 16 bits are then kept with round-to-nearest-even.
    """
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32)
    # u + 0x7FFF + lsb stays below 2^32 for every non-NaN input (the largest
    # finite pattern is 0xFF7FFFFF), so the sum needs no wider type
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r &= np.uint32(0xFFFF0000)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = np.uint32(0x7FC00000)
    return r.view(np.float32).astype(np.float64)


def round_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the partition's storage precision, returned as float64."""
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def _xavier(rng: np.random.Generator, shape) -> np.ndarray:
    fan_in, fan_out = shape
    a = np.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-a, a, size=shape)


FFN_MATRICES = ("w1", "w2")


def _draw_param(rng, name, shape, perturb, fixup_layers=0):
    if len(shape) == 2:
        w = _xavier(rng, shape)
        # Section 5: the initialisation of every feed-forward layer is scaled
        # down by the number of layers of the model
        return w / fixup_layers if fixup_layers > 0 and name in FFN_MATRICES else w
    if name.endswith("_g"):
        return 1.0 + 0.1 * rng.standard_normal(shape) if perturb else np.ones(shape)
    return 0.1 * rng.standard_normal(shape) if perturb else np.zeros(shape)


def make_params(cfg: PartitionConfig, seed: int, perturb: bool = False):
    """Draw the partition's parameters; returns (layers, head) of float64 arrays
    already rounded to the storage precision.  ``layers`` is a list of dicts
    keyed by parameter id; ``head`` is a dict (empty without a vocabulary head).
    """
    rng = np.random.default_rng(seed)
    return _make_params(rng, cfg, perturb)


def _make_params(rng, cfg, perturb):
    shapes = cfg.param_shapes()
    order = [p for p in PARAM_IDS if p in shapes]
    layers = []
    for _ in range(cfg.layers):
        layers.append({p: round_storage(_draw_param(rng, p, shapes[p], perturb, cfg.fixup_layers), cfg.dtype)
                       for p in order})
    hshapes = cfg.head_shapes()
    head = {p: round_storage(_draw_param(rng, p, hshapes[p], perturb), cfg.dtype)
            for p in HEAD_PARAMS if p in hshapes}
    return layers, head


def make_case(cfg: PartitionConfig, seed: int, perturb: bool = False,
              batch: Optional[int] = None) -> dict:
    """Draw one full case: parameters, boundary input, memory, loss tensor.

    Returns a dict with keys layers, head, x [N,S,D], mem [N,S_mem,D] or None,
    and one of target [N,S,D] (mse), dy [N,S,D] (boundary gradient) or
    labels int32 [N,S] (xent_ls).  Floating arrays are float64 holding values
    exactly representable in the partition's storage precision.
    """
    rng = np.random.default_rng(seed)
    layers, head = _make_params(rng, cfg, perturb)
    N = cfg.batch if batch is None else batch
    S, D = cfg.seq, cfg.d_model
    case = {"layers": layers, "head": head}
    case["x"] = round_storage(rng.standard_normal((N, S, D)), cfg.dtype)
    case["mem"] = (round_storage(rng.standard_normal((N, cfg.mem_seq, D)), cfg.dtype)
                   if cfg.kind == "decoder" else None)
    if cfg.loss == "mse":
        case["target"] = round_storage(rng.standard_normal((N, S, D)), cfg.dtype)
    elif cfg.loss == "none":
        case["dy"] = round_storage(rng.standard_normal((N, S, D)), cfg.dtype)
    elif cfg.loss == "xent_ls":
        case["labels"] = rng.integers(0, cfg.vocab, size=(N, S)).astype(np.int32)
    else:
        raise ValueError(cfg.loss)
    return case
