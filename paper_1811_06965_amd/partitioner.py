"""Cost-balanced partitioning of a Transformer into K pipeline cells.

GPipe lets every layer carry a cost estimate c_i (Section 2.1) and splits
the L layers into K cells of consecutive layers whose summed costs C_k have
the least variance (Section 2.2).  Here the costs are measured from this
library's own kernels: the time of one training step (M forwards, M
re-materialising backwards, the update) of a partition of one layer kind at
the workload's micro-batch shape, differenced over the layer count so that
the fixed per-step costs cancel:

  c_encoder = t(2 encoder layers) - t(1 encoder layer)
  c_decoder = t(2 decoder layers) - t(1 decoder layer)     (boundary loss)
  c_head    = t(1 decoder layer + cross-entropy head) - t(1 decoder layer)

The split itself is gp_plan_cells (an exact dynamic program in the library).
Usage:  python -m paper_1811_06965_amd.partitioner --encoder 16 --decoder 8
        --cells 4 [--config dec1024] prints the measured costs and the cells.
"""
from __future__ import annotations

import argparse
import json
from typing import Dict, List, Sequence

import numpy as np

from . import gp


def _step_ms(cfg, steps: int, warmup: int) -> float:
    import torch

    import synth
    from .runtime import Partition
    case = synth.make_case(cfg, 0)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = {"dx": torch.empty_like(inp["x"])}
        for _ in range(warmup):
            part.step(inp["x"], inp["mem"], inp["dy"], want_y=False, want_loss=False, dx=out["dx"])
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for _ in range(steps):
            part.step(inp["x"], inp["mem"], inp["dy"], want_y=False, want_loss=False, dx=out["dx"])
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / steps


def measure_layer_costs(cfg, steps: int = 5, warmup: int = 2) -> Dict[str, float]:
    """Milliseconds per training step that one encoder layer, one decoder
    layer and the vocabulary head add, at cfg's widths and micro-batch shape
    (cfg.vocab for the head; mem_seq defaults to seq)."""
    mem = cfg.mem_seq or cfg.seq
    enc = cfg.with_(kind="encoder", loss="none", vocab=0, label_smoothing=0.0, mem_seq=0, logit_clip=0.0)
    dec = cfg.with_(kind="decoder", loss="none", vocab=0, label_smoothing=0.0, mem_seq=mem, logit_clip=0.0)
    t = {}
    t["enc1"] = _step_ms(enc.with_(layers=1), steps, warmup)
    t["enc2"] = _step_ms(enc.with_(layers=2), steps, warmup)
    t["dec1"] = _step_ms(dec.with_(layers=1), steps, warmup)
    t["dec2"] = _step_ms(dec.with_(layers=2), steps, warmup)
    costs = {"encoder": t["enc2"] - t["enc1"], "decoder": t["dec2"] - t["dec1"]}
    if cfg.vocab:
        head = dec.with_(layers=1, loss="xent_ls", vocab=cfg.vocab, label_smoothing=cfg.label_smoothing or 0.1)
        costs["head"] = _step_ms(head, steps, warmup) - t["dec1"]
    return costs


def plan(layer_kinds: Sequence[str], costs: Dict[str, float], cells: int):
    """Cells of least cost variance for a model given as its sequence of layer
    kinds; returns (first layer of each cell, cell costs, variance)."""
    c = np.array([costs[k] for k in layer_kinds], dtype=np.float64)
    first, var = gp.gp_plan_cells(c, cells)
    bounds = list(first) + [len(c)]
    cell_costs = [float(c[bounds[k]:bounds[k + 1]].sum()) for k in range(cells)]
    return first, cell_costs, var


def main(argv: List[str] = None) -> None:
    import synth
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="dec1024", help="widths and micro-batch shape of the layers")
    ap.add_argument("--encoder", type=int, default=0, help="encoder layers, first in the model")
    ap.add_argument("--decoder", type=int, default=8, help="decoder layers after them")
    ap.add_argument("--cells", type=int, default=2)
    ap.add_argument("--steps", type=int, default=5)
    a = ap.parse_args(argv)
    cfg = synth.CONFIGS[a.config]
    costs = measure_layer_costs(cfg, a.steps)
    kinds = ["encoder"] * a.encoder + ["decoder"] * a.decoder + (["head"] if "head" in costs else [])
    first, cell_costs, var = plan(kinds, costs, a.cells)
    print(json.dumps({"config": cfg.name, "micro_batches": cfg.micro, "layer_costs_ms": costs,
                      "layers": kinds, "cells": a.cells, "first_layer_of_cell": first,
                      "cell_costs_ms": cell_costs, "variance_ms2": var}))


if __name__ == "__main__":
    main()
