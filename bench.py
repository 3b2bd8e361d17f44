"""Throughput of one GPipe partition step on one MI355X.

Workload: one-eighth of a 128-layer Transformer -- a partition of 16 pre-LN
encoder layers, d_model 1024, 16 heads, d_ff 8192, ReLU, sequence 256, a
mini-batch of 64 sequences split into M micro-batches (8 for the headline
value; every M in {4, 8, 16, 32} is timed too, each beside the
stored-activation baseline that keeps every intermediate instead of
recomputing it), bf16 operands with fp32 accumulation, random N(0,1)
boundary inputs and boundary gradients, Xavier-uniform weights (synthetic
data).

One step = M x gp_forward_microbatch + M x gp_backward_microbatch_remat +
gp_accumulate_and_step (GPipe, Sections 2.2-2.3), enqueued by
runtime.Partition.step: even micro-batches on the launch stream, odd ones on
a second stream from gp_stream_create (consecutive forwards, and the two
backwards of a recompute pair, run side by side), joined before the update;
the library runs the weight gradients and the recompute-ahead on streams of
its own.  W untimed warm-up steps, one untimed census
step that times every launch role to find the dominant one, then K eager
steps timed between two events on the launch stream, with one launch in
TIMER_EVERY of the dominant role bracketed by dispatch events inside the timed
region.  --graph captures the step once into a HIP graph and times K replays
instead (the role is then timed over a few eager steps right after).  Prints
one JSON line.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "train tokens/s, one partition fwd+remat-bwd over M micro-batches"
PEAK_BF16 = 2.5e15  # MI355X dense bf16 MFMA, FLOP/s
PEAK_FP32 = 157.3e12  # MI355X fp32 vector, FLOP/s
PEAK_HBM = 8.0e12   # MI355X HBM3E, B/s
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--micro", type=int, default=8, help="micro-batches M of the timed workload")
    ap.add_argument("--config", default="enc1024")
    ap.add_argument("--no-sweep", action="store_true",
                    help="time only --micro (by default M in {4, 8, 16, 32} are all timed, and the stored-"
                         "activation baseline beside each)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=16, help="layers in the oracle's timed sample")
    ap.add_argument("--role", default=None, help="time this launch role instead of the dominant one")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured once into a HIP graph instead of eager steps "
                         "(the dominant role is then timed over eager steps right after)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (calibrates the PMC byte counters)")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="summarise rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of `--role R` (with "
                         "GP_TIMER_MARKERS=1) and of --copy-calibration into the stored traffic figures")
    ap.add_argument("--counter-summary", metavar="DIR",
                    help="print, as JSON, the median per launch of `--role R` of every counter in a rocprofv3 "
                         "--pmc run of that role (GP_TIMER_MARKERS=1), summed over the counter's instances")
    ap.add_argument("--kernel-summary", metavar="DIR",
                    help="print a markdown summary of a rocprofv3 --kernel-trace database under DIR "
                         "(per-kernel totals, and per-role launch durations when GP_TIMER_MARKERS=1 was set)")
    ap.add_argument("--command", default="", help="the profiled command, quoted in --kernel-summary output")
    ap.add_argument("--roles-json", default=None,
                    help="with --kernel-summary: also store the per-role launch durations of the trace here "
                         "(read back by the benchmark's roofline figure)")
    return ap.parse_args()


def _short(name):
    import re
    import shutil
    import subprocess
    if name.startswith("_Z") and shutil.which("c++filt"):
        # GNU c++filt does not know the bf16 builtin type code; spell it as a vendor type
        out = subprocess.run(["c++filt", name.replace("DF16b", "u6__bf16")], capture_output=True, text=True)
        name = out.stdout.strip() or name
    name = re.sub(r"\(anonymous namespace\)::|gp::|void ", "", name)
    return re.sub(r"\(gp::(GemmArgs|AttnArgs)\)|\(gp::GemmArgs, int\)", "", name)[:110]


def kernel_summary(d, command, top=25, roles_json=None):
    """Markdown summary of a rocprofv3 kernel-trace database."""
    import glob
    import sqlite3
    from paper_1811_06965_amd import gp
    db = sqlite3.connect(glob.glob(os.path.join(d, "**", "*results.db"), recursive=True)[0])
    rows = db.execute("select name, grid_x, grid_y, workgroup_x, start, end from kernels order by start").fetchall()
    total = sum(r[5] - r[4] for r in rows if "role_marker" not in r[0])
    print("# Kernel summary\n")
    print(f"Command: `{command}`\n")
    print(f"{len(rows)} dispatches, {total / 1e6:.2f} ms of kernel time (markers excluded).\n")
    agg = {}
    for name, gx, gy, wx, t0, t1 in rows:
        if "role_marker" in name:
            continue
        k = (_short(name), gx // max(wx, 1), gy)
        c, s = agg.get(k, (0, 0))
        agg[k] = (c + 1, s + t1 - t0)
    print("| kernel | grid | calls | mean us | % of kernel time |\n|---|---|---|---|---|")
    for (n, gx, gy), (c, s) in sorted(agg.items(), key=lambda kv: -kv[1][1])[:top]:
        print(f"| `{n}` | ({gx},{gy}) | {c} | {s / c / 1e3:.1f} | {100 * s / total:.1f} |")
    # launches between role markers, on the marker's stream, in enqueue order
    spans, cur = {}, {}
    for name, gx, gy, wx, t0, t1, sid in db.execute(
            "select name, grid_x, grid_y, workgroup_x, start, end, stream_id from kernels order by dispatch_id"):
        if "role_marker" in name:
            role, edge = gx // max(wx, 1), gy - 1
            if edge == 0:
                cur[sid] = (role, [])
            elif sid in cur:
                spans.setdefault(cur[sid][0], []).append(cur.pop(sid)[1])
        elif sid in cur:
            cur[sid][1].append((_short(name), t0, t1))
    if spans and roles_json:
        rec = {"source_sha256": source_digest(), "command": command, "roles": {}}
        for role, ls in spans.items():
            ls = [l for l in ls if l]
            if ls:
                rec["roles"][gp.KERNEL_ROLES[role]] = {
                    "launches": len(ls),
                    "mean_kernel_us": sum(t1 - t0 for l in ls for _, t0, t1 in l) / len(ls) / 1e3,
                    "mean_span_us": sum(l[-1][2] - l[0][1] for l in ls) / len(ls) / 1e3,
                    "kernels": sorted({n for l in ls for n, _, _ in l})}
        with open(roles_json, "w") as f:
            json.dump(rec, f, indent=1)
    if spans:
        print("\n## Launch roles (kernels between role markers)\n")
        print("| role | launches | mean kernel us per launch | mean first-start to last-end us | kernels |\n|---|---|---|---|---|")
        for role, ls in sorted(spans.items(), key=lambda kv: -sum(t1 - t0 for l in kv[1] for _, t0, t1 in l)):
            ls = [l for l in ls if l]
            if not ls:
                continue
            busy = sum(t1 - t0 for l in ls for _, t0, t1 in l) / len(ls) / 1e3
            span = sum(l[-1][2] - l[0][1] for l in ls) / len(ls) / 1e3
            names = sorted({n for l in ls for n, _, _ in l})
            print(f"| {gp.KERNEL_ROLES[role]} | {len(ls)} | {busy:.1f} | {span:.1f} | " +
                  "<br>".join(f"`{n}`" for n in names) + " |")


COPY_BYTES = 1 << 30


def copy_calibration():
    """A plain copy of known size: reads and writes COPY_BYTES each, three times."""
    import torch
    a = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    print(f"[bench] copy calibration: 3 x neg over {COPY_BYTES} bytes", file=sys.stderr)


def _pmc_rows(d):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def _per_dispatch(rows, counter):
    """[(queue id, kernel name, counter value)] in dispatch order for one
    counter (summed over its instances)."""
    acc = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        k = int(r["Dispatch_Id"])
        q, name, v = acc.get(k, (r["Queue_Id"], r["Kernel_Name"], 0.0))
        acc[k] = (q, name, v + float(r["Counter_Value"]))
    return [(q, n, v) for k, (q, n, v) in sorted(acc.items())]


def _between_markers(disp):
    """Counter sums of the launches between role_marker pairs, on the
    marker's hardware queue (each library stream has its own)."""
    out, cur = [], {}
    for q, name, v in disp:
        if "role_marker" in name:
            if q not in cur:
                cur[q] = [0.0, []]
            else:
                out.append(cur.pop(q))
        elif q in cur:
            cur[q][0] += v
            cur[q][1].append(name)
    return out


def counter_summary(d, role):
    """Median per launch of the role (the kernels between its markers) of
    every counter collected under d."""
    rows = _pmc_rows(d)
    out = {"role": role, "counters": {}}
    for c in sorted({r["Counter_Name"] for r in rows}):
        launches = _between_markers(_per_dispatch(rows, c))
        vals = sorted(l[0] for l in launches)
        if vals:
            out["counters"][c] = vals[len(vals) // 2]
            out["launches"] = len(vals)
            out["kernels"] = sorted({k for l in launches for k in l[1]})
    print(json.dumps(out, indent=1))


def traffic_summary(fetch_dir, write_dir, cal_fetch_dir, cal_write_dir, role, workload):
    """FETCH_SIZE and WRITE_SIZE are in KiB per dispatch; each is scaled by
    the known bytes of the copy kernel over what the counter read for it."""
    cal = {}
    for ctr, d in (("FETCH_SIZE", cal_fetch_dir), ("WRITE_SIZE", cal_write_dir)):
        vals = [v for _, n, v in _per_dispatch(_pmc_rows(d), ctr) if "neg" in n or "elementwise" in n]
        big = [v for v in vals if v * 1024 > COPY_BYTES / 2]
        cal[ctr] = COPY_BYTES / (sorted(big)[len(big) // 2] * 1024)
    res = {}
    for ctr, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        launches = _between_markers(_per_dispatch(_pmc_rows(d), ctr))
        kib = sorted(l[0] for l in launches)
        res[ctr] = {"launches": len(kib), "median_kib": kib[len(kib) // 2], "kernels": sorted({k for l in launches for k in l[1]})}
    fetch = res["FETCH_SIZE"]["median_kib"] * 1024 * cal["FETCH_SIZE"]
    write = res["WRITE_SIZE"]["median_kib"] * 1024 * cal["WRITE_SIZE"]
    entry = {"bytes_per_launch": fetch + write, "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
             "fetch_scale": cal["FETCH_SIZE"], "write_scale": cal["WRITE_SIZE"],
             "launches": res["FETCH_SIZE"]["launches"], "kernels": res["FETCH_SIZE"]["kernels"]}
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        t = {}
    if t.get("source_sha256") != source_digest() or t.get("workload") != workload:
        t = {"source_sha256": source_digest(), "workload": workload, "roles": {}}
    t["roles"][role] = entry
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(t, f, indent=1)
    print(json.dumps({role: entry}, indent=1))


def run_steps(part, inp, n, out):
    """n whole steps with every boundary output the pipeline passes on: y to
    the next partition (forward), dX to the previous one (backward)."""
    for _ in range(n):
        part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_loss=False, y=out["y"], dx=out["dx"])


def census(part, inp, out):
    """One untimed step with every launch role timed; roles by total time."""
    import torch
    from paper_1811_06965_amd import gp
    part.timer_reset()
    part.timer_select("all")
    run_steps(part, inp, 1, out)
    torch.cuda.synchronize()
    part.timer_select(None)
    roles = {}
    for name in gp.KERNEL_ROLES[1:]:
        r = part.timer_read(name)
        if r["launches"]:
            roles[name] = r
    part.timer_reset()
    return dict(sorted(roles.items(), key=lambda kv: -kv[1]["ms"]))


def dominant_role(roles):
    """The role with the most launch time in the census step; roles within
    10% of it count as tied (the split of a step between concurrent streams
    moves by that much from run to run), and a tie goes to the role doing the
    most algorithmic work per step, then to the one with more time."""
    top = next(iter(roles.values()))["ms"]
    tied = [(r["flops"], r["ms"], name) for name, r in roles.items() if r["ms"] >= 0.9 * top]
    return max(tied)[2]


# One launch in this many of the timed role is bracketed by dispatch events
# inside the timed region (each bracket holds the next launch back by a few
# microseconds; bracketing all 256 ffn2.fwd launches of an M = 8 step cost
# 0.6-0.7 ms of it).
TIMER_EVERY = 8


def timed_eager(part, inp, steps, out, role):
    """K eager steps between two events on the launch stream, with every
    TIMER_EVERY-th launch of the role bracketed by dispatch events."""
    import torch
    st = torch.cuda.current_stream()
    part.timer_reset()
    part.timer_sample(TIMER_EVERY)
    part.timer_select(role)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(st)
    run_steps(part, inp, steps, out)
    t1.record(st)
    torch.cuda.synchronize()
    part.timer_select(None)
    timed = part.timer_read(role)
    part.timer_reset()
    part.timer_sample(1)
    return t0.elapsed_time(t1) / steps, timed


def device_free():
    import torch
    torch.cuda.synchronize()
    return torch.cuda.mem_get_info()[0]


def time_plain(part, inp, steps, warmup):
    """Milliseconds per step over `steps` eager steps after `warmup`, between
    two events on the launch stream, no launch timed."""
    import torch
    out = {"y": torch.empty_like(inp["x"]), "dx": torch.empty_like(inp["x"])}
    run_steps(part, inp, warmup, out)
    st = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(st)
    run_steps(part, inp, steps, out)
    t1.record(st)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def timed_graph(part, inp, steps, out):
    """The step captured once into a HIP graph, then K replays between two
    events on the replay stream."""
    import torch
    g = part.capture_step(inp["x"], inp["mem"], inp["dy"], lr=0.0, dx=out["dx"], want_y=True, y=out["y"])
    g.replay()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(st)
    for _ in range(steps):
        g.replay()
    t1.record(st)
    torch.cuda.synchronize()
    del g
    return t0.elapsed_time(t1) / steps


def time_steps(part, inp, steps, warmup, role=None, graph=False):
    """Returns (ms per step, role, role timings, census, how the role was timed)."""
    import torch
    out = {"y": torch.empty_like(inp["x"]), "dx": torch.empty_like(inp["x"])}
    run_steps(part, inp, warmup, out)
    torch.cuda.synchronize()
    roles = census(part, inp, out) if role is None else None
    if role is None:
        role = dominant_role(roles)
    if not graph:
        ms, timed = timed_eager(part, inp, steps, out, role)
        return ms, role, timed, roles, (f"HIP events attached to the dispatches of every {TIMER_EVERY}th launch of "
                                        "the role inside the timed eager steps (the kernels share the GPU with the "
                                        "weight-gradient and recompute streams)")
    ms = timed_graph(part, inp, steps, out)
    _, timed = timed_eager(part, inp, max(1, min(steps, 3)), out, role)
    return ms, role, timed, roles, (f"dispatch events on every {TIMER_EVERY}th launch over eager steps run after "
                                    "the graph-replay timed region")


def source_digest():
    """SHA-256 over the HIP sources and the compiler flags they are built
    with: a stored traffic figure is only valid for the kernels it was
    measured on."""
    from paper_1811_06965_amd import build
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1811_06965_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".hpp")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + b"\0" + fh.read())
    h.update(repr((build.FLAGS, sorted(build.EXTRA_FLAGS.items()))).encode())
    return h.hexdigest()


def stored_traffic(role, workload):
    """HBM bytes per launch of `role` from the PMC runs stored with the
    profiles (FETCH_SIZE + WRITE_SIZE, calibrated), if they were taken on the
    current kernels and workload; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    e = t.get("roles", {}).get(role)
    if not e or t.get("source_sha256") != source_digest() or t.get("workload") != workload:
        return None
    return e["bytes_per_launch"]


ROLES_FILE = os.path.join(ROOT, "profiles", "kernel_roles_enc1024_m8.json")


def profiled_launch(role):
    """The role's mean kernel time per launch in the committed rocprofv3
    kernel trace of the benchmark (kernels between the role's markers), if
    that trace was taken on the current kernels; else None."""
    try:
        with open(ROLES_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    e = rec.get("roles", {}).get(role)
    if not e or rec.get("source_sha256") != source_digest():
        return None
    return dict(e, command=rec.get("command", ""))


def roofline(role, timed, workload):
    """Roofline figure of the dominant launch role: algorithmic work per launch
    over the mean event-to-event launch duration measured in this run; beside
    it the same figure from the committed kernel trace's mean kernel time."""
    n = max(timed["launches"], 1)
    dur = timed["ms"] * 1e-3 / n
    per = timed["flops"] / n if timed["flops"] > 0 else timed["bytes"] / n
    if timed["flops"] > 0:
        scale, peak, unit, bound = 1e12, PEAK_BF16 / 1e12, "TFLOP/s", "mfma"
    else:
        scale, peak, unit, bound = 1e9, PEAK_HBM / 1e9, "GB/s", "hbm"
    achieved = per / dur / scale
    out = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
           "traffic": stored_traffic(role, workload), "role": role, "launches_timed": timed["launches"],
           "mean_launch_us": dur * 1e6, "algorithmic_flops_per_launch": timed["flops"] / n,
           "algorithmic_bytes_per_launch": timed["bytes"] / n}
    prof = profiled_launch(role)
    if prof:
        out["rocprof"] = {"file": os.path.relpath(ROLES_FILE, ROOT), "command": prof["command"],
                          "mean_kernel_us": prof["mean_kernel_us"], "launches": prof["launches"],
                          "achieved": per / (prof["mean_kernel_us"] * 1e-6) / scale,
                          "frac": per / (prof["mean_kernel_us"] * 1e-6) / scale / peak}
    else:
        out["rocprof"] = None
    return out


def blas_info():
    """(threads, description) of the BLAS numpy runs on."""
    try:
        from threadpoolctl import threadpool_info
        libs = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    except Exception:
        libs = []
    if not libs:
        return len(os.sched_getaffinity(0)), "unknown BLAS"
    lib = max(libs, key=lambda i: i["num_threads"])
    desc = f"{lib.get('internal_api', 'blas')} {lib.get('version', '')} ({lib.get('architecture', '')} kernels, " \
           f"{lib['num_threads']} threads)"
    return lib["num_threads"], desc


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(cfg, layers):
    """The fp64 oracle on a bounded sample of the workload: `layers` of the 16
    layers, one micro-batch of the timed M (all three passes: forward,
    re-materialised forward, backward), scaled to whole-partition tokens/s."""
    import synth
    from oracle import gpipe
    n = cfg.batch // cfg.micro
    sample = cfg.with_(layers=layers, batch=n, micro=1)
    case = synth.make_case(sample, 0)
    t = time.perf_counter()
    gpipe.gpipe_step(sample, case, 1)
    dt = time.perf_counter() - t
    tok_s = n * cfg.seq / (dt * cfg.layers / layers)
    threads, blas = blas_info()
    return {"value": tok_s, "unit": "tokens/s", "cores": threads, "kind": "oracle", "cpu": cpu_model(),
            "blas": blas, "host_cpus_available": len(os.sched_getaffinity(0)),
            "sample": f"{layers} of {cfg.layers} layers, one micro-batch of {n} sequences x {cfg.seq} tokens, "
                      f"forward + re-materialised forward + backward in fp64 numpy ({dt:.1f} s), "
                      f"scaled by {cfg.layers}/{layers} layers"}


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one partition on one GPU; --gpus {a.gpus} is not supported "
              "(the library implements one GPU's partition; a K-stage pipeline over several GPUs is not "
              "implemented)", file=sys.stderr)
        sys.exit(2)
    import synth
    base = synth.CONFIGS[a.config]
    cfg = base.with_(micro=a.micro)
    workload = (f"{cfg.name}: {cfg.layers}-layer pre-LN {cfg.kind} partition, d_model {cfg.d_model}, "
                f"{cfg.heads} heads, d_ff {cfg.d_ff}, ReLU, seq {cfg.seq}, mini-batch {cfg.batch} "
                f"in M={cfg.micro} micro-batches, " +
                ("boundary gradients" if cfg.loss == "none" else f"{cfg.loss} loss"))
    if a.kernel_summary:
        kernel_summary(a.kernel_summary, a.command, roles_json=a.roles_json)
        return
    if a.counter_summary:
        if not a.role:
            sys.exit("--counter-summary needs --role")
        counter_summary(a.counter_summary, a.role)
        return
    if a.traffic_summary:
        if not a.role:
            sys.exit("--traffic-summary needs --role")
        traffic_summary(*a.traffic_summary, a.role, workload)
        return
    import torch
    from paper_1811_06965_amd import accounting
    from paper_1811_06965_amd.runtime import Partition

    torch.cuda.set_device(0)
    if a.copy_calibration:
        copy_calibration()
        return
    case = synth.make_case(cfg, 0)
    results = {}
    Ms = [a.micro] + ([] if a.no_sweep else [m for m in (4, 8, 16, 32) if m != a.micro])
    for M in Ms:
        c = base.with_(micro=M)
        steps = a.steps if M == a.micro else max(3, a.steps // 2)
        f0 = device_free()
        with Partition(c) as part:
            allocated = f0 - device_free()
            part.load_params(case["layers"], case["head"])
            inp = part.device_inputs(case)
            ms, role, timed, roles, how = time_steps(part, inp, steps, a.warmup, a.role, graph=a.graph)
            mem = part.memory()
            del inp
        model, hw = accounting.step_flops(c)
        results[M] = {"M": M, "ms_per_step": ms, "tokens_per_s": c.batch * c.seq / (ms * 1e-3),
                      "hfu": hw / (ms * 1e-3) / PEAK_BF16, "mfu": model / (ms * 1e-3) / PEAK_BF16,
                      "memory_bytes": mem, "device_bytes_measured": allocated,
                      "role": role, "timed": timed, "roles": roles, "how": how}
        print(f"[bench] M={M}: {ms:.2f} ms/step, {results[M]['tokens_per_s']:.0f} tokens/s, "
              f"HFU {100 * results[M]['hfu']:.1f}%, dominant role {role}, device memory "
              f"{allocated / 2**30:.2f} GiB", file=sys.stderr, flush=True)
        if not a.no_sweep:
            # the stored-activation baseline: every micro-batch keeps its
            # intermediates, no recompute (3 forward passes of work instead of 4)
            f0 = device_free()
            with Partition(c, keep_activations=True) as part:
                allocated = f0 - device_free()
                part.load_params(case["layers"], case["head"])
                inp = part.device_inputs(case)
                kms = time_plain(part, inp, max(3, a.steps // 2), a.warmup)
                kmem = part.memory()
                del inp
            results[M]["stored_activations"] = {
                "ms_per_step": kms, "tokens_per_s": c.batch * c.seq / (kms * 1e-3),
                "hfu": model / (kms * 1e-3) / PEAK_BF16, "memory_bytes": kmem, "device_bytes_measured": allocated}
            print(f"[bench] M={M} stored activations: {kms:.2f} ms/step, device memory "
                  f"{allocated / 2**30:.2f} GiB", file=sys.stderr, flush=True)
    # the sustained MFMA-loop rate of this device, measured after the timed runs
    from paper_1811_06965_amd import gp
    peak_meas = gp.gp_mfma_peak(torch.cuda.current_stream().cuda_stream) * 1e12
    for res in results.values():
        res["hfu_measured_peak"] = res["hfu"] * PEAK_BF16 / peak_meas
    r = results[a.micro]
    out = {
        "metric": METRIC, "value": r["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": workload, "global_batch": cfg.batch, "seq_len": cfg.seq, "micro_batches": cfg.micro,
                   "parallelism": "one pipeline partition on one GPU"},
        "hfu": r["hfu"], "mfu": r["mfu"], "memory_bytes": r["memory_bytes"],
        "mfma_peak_measured_tflops": peak_meas * 1e-12, "hfu_measured_peak": r["hfu_measured_peak"],
        "roofline": roofline(r["role"], r["timed"], workload),
        "launch": "HIP graph: the whole step captured once, replayed" if a.graph else "eager (host-enqueued launches)",
    }
    out["roofline"]["timing"] = r["how"]
    if out["roofline"]["bound"] == "mfma":
        out["roofline"]["frac_of_measured_peak"] = out["roofline"]["achieved"] * 1e12 / peak_meas
    if r["roles"]:
        step_ms = r["ms_per_step"]
        out["roles_ms_per_step"] = {k: round(v["ms"], 3) for k, v in r["roles"].items()}
        out["roles_note"] = f"census step with every launch bracketed; step time {step_ms:.2f} ms unbracketed"
    if not a.no_sweep:
        keys = ("M", "ms_per_step", "tokens_per_s", "hfu", "mfu", "hfu_measured_peak", "memory_bytes",
                "device_bytes_measured", "stored_activations")
        out["sweep"] = [dict({k: v for k, v in results[M].items() if k in keys},
                             roles_ms_per_step={k: round(v["ms"], 3) for k, v in (results[M]["roles"] or {}).items()})
                        for M in sorted(results)]
        out["sweep_note"] = ("re-materialised steps (4 forward passes of work: hfu) beside the stored-activation "
                             "baseline (no recompute, 3 forward passes: its hfu counts those); memory_bytes is the "
                             "library's plan, device_bytes_measured the drop in free device memory at configure")
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, a.cpu_layers)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
