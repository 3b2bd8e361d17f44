"""Throughput of one GPipe partition step on one MI355X.

Workload: one-eighth of a 128-layer Transformer -- a partition of 16 pre-LN
encoder layers, d_model 1024, 16 heads, d_ff 8192, ReLU, sequence 256, a
mini-batch of 64 sequences split into M micro-batches (default 8), bf16
operands with fp32 accumulation, random N(0,1) boundary inputs and boundary
gradients, Xavier-uniform weights (synthetic data).

One step = M x gp_forward_microbatch + M x gp_backward_microbatch_remat +
gp_accumulate_and_step (GPipe, Sections 2.2-2.3), all enqueued on one stream.
W untimed warm-up steps, then K steps timed between two synchronisations.
Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "train tokens/s, one partition fwd+remat-bwd over M micro-batches; MFMA %"
PEAK_BF16 = 2.5e15  # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12   # MI355X HBM3E, B/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--micro", type=int, default=8, help="micro-batches M of the timed workload")
    ap.add_argument("--config", default="enc1024")
    ap.add_argument("--sweep", action="store_true", help="also time M in {4, 8, 16, 32}")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=2, help="layers in the oracle's timed sample")
    return ap.parse_args()


def time_steps(part, inp, steps, warmup):
    import torch
    st = torch.cuda.current_stream()
    for _ in range(warmup):
        part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_y=False, want_dx=True, want_loss=False)
    torch.cuda.synchronize()
    y = None
    dx = torch.empty_like(inp["x"])
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(st)
    for _ in range(steps):
        part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_y=False, want_dx=True, want_loss=False, dx=dx)
    t1.record(st)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def cpu_baseline(cfg, layers):
    """The fp64 oracle on a bounded sample of the workload: `layers` of the 16
    layers, one micro-batch of the timed M (all three passes: forward,
    re-materialised forward, backward), scaled to whole-partition tokens/s."""
    import numpy as np
    import synth
    from oracle import gpipe
    n = cfg.batch // cfg.micro
    sample = cfg.with_(layers=layers, batch=n, micro=1)
    case = synth.make_case(sample, 0)
    t = time.perf_counter()
    gpipe.gpipe_step(sample, case, 1)
    dt = time.perf_counter() - t
    tok_s = n * cfg.seq / (dt * cfg.layers / layers)
    return {"value": tok_s, "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
            "sample": f"{layers} of {cfg.layers} layers, one micro-batch of {n} sequences x {cfg.seq} tokens, "
                      f"forward + re-materialised forward + backward in fp64 numpy ({dt:.1f} s), "
                      f"scaled by {cfg.layers}/{layers} layers"}


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one partition on one GPU; --gpus {a.gpus} is not supported "
              "(multi-GPU pipelines are outside this build)", file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    from paper_1811_06965_amd import accounting
    from paper_1811_06965_amd.runtime import Partition

    torch.cuda.set_device(0)
    base = synth.CONFIGS[a.config]
    cfg = base.with_(micro=a.micro)
    case = synth.make_case(cfg, 0)
    results = {}
    Ms = [a.micro] + ([m for m in (4, 8, 16, 32) if m != a.micro] if a.sweep else [])
    for M in Ms:
        c = base.with_(micro=M)
        with Partition(c) as part:
            part.load_params(case["layers"], case["head"])
            inp = part.device_inputs(case)
            ms = time_steps(part, inp, a.steps if M == a.micro else max(3, a.steps // 2), a.warmup)
            mem = part.memory()
            del inp
        model, hw = accounting.step_flops(c)
        results[M] = {"M": M, "ms_per_step": ms, "tokens_per_s": c.batch * c.seq / (ms * 1e-3),
                      "hfu": hw / (ms * 1e-3) / PEAK_BF16, "mfu": model / (ms * 1e-3) / PEAK_BF16,
                      "memory_bytes": mem}
        print(f"[bench] M={M}: {ms:.2f} ms/step, {results[M]['tokens_per_s']:.0f} tokens/s, "
              f"HFU {100 * results[M]['hfu']:.1f}%", file=sys.stderr, flush=True)
    r = results[a.micro]
    out = {
        "metric": METRIC, "value": r["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.layers}-layer pre-LN encoder partition, d_model {cfg.d_model}, "
                               f"{cfg.heads} heads, d_ff {cfg.d_ff}, ReLU, seq {cfg.seq}, mini-batch {cfg.batch} "
                               f"in M={cfg.micro} micro-batches, boundary gradients",
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "micro_batches": cfg.micro,
                   "parallelism": "one pipeline partition on one GPU"},
        "hfu": r["hfu"], "mfu": r["mfu"],
    }
    if a.sweep:
        out["sweep"] = [{k: v for k, v in results[M].items() if k != "memory_bytes"} for M in sorted(results)]
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, a.cpu_layers)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
