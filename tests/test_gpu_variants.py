"""GPU checks of the partition's variants, through the C ABI:

* the stored-activation baseline (keep_activations: no recompute) against
  re-materialisation, bit for bit (Section 2.3: the recompute is the same F_k);
* device memory measured around configure and across steps, against the
  library's plan, with and without re-materialisation (Section 2.3, Table 1);
* GP_POISON=1 (every workspace region filled with NaN before the phase that
  rewrites it) leaves every result bit-identical, with all three streams on;
* forwards issued on two streams (two first-pass slots) against one, the two
  members of a recompute pair back-propagated side by side (two backward
  lanes) against one lane, and the per-layer update against the whole update
  after the last backward, bit for bit;
* RMSProp (Table 1's optimizer), logit clipping and the scaled-down
  feed-forward initialisation (Section 5) against the fp64 oracle.

Tolerances as in test_gpu_parity: fp32 max-abs relative error <= 1e-4;
bf16 outputs and loss <= 2e-2, gradients cosine >= 0.999.
"""
import numpy as np
import pytest

import synth
from parity import compare_grads, cosine, rel_err, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TINY = synth.CONFIGS["tiny"]
ENC512_SMALL = synth.CONFIGS["enc512"].with_(name="enc512_small", layers=2, batch=8, micro=4)
RAGGED_BF16 = synth.PartitionConfig("ragged_bf16", layers=2, d_model=512, d_ff=2048, heads=8, seq=96,
                                    batch=6, micro=2, dtype="bf16", loss="none")
DEC_SMALL_BF16 = synth.PartitionConfig("dec_small_bf16", layers=2, d_model=256, d_ff=512, heads=4, seq=64, batch=4,
                                       micro=2, kind="decoder", mem_seq=64, loss="xent_ls", vocab=512,
                                       label_smoothing=0.1)
DEC_F32 = synth.PartitionConfig("dec_f32", layers=2, d_model=32, d_ff=64, heads=2, seq=8, batch=4, micro=2,
                                dtype="f32", kind="decoder", loss="xent_ls", vocab=40, label_smoothing=0.1,
                                mem_seq=6)
DEC_BF16 = synth.PartitionConfig("dec_bf16", layers=2, d_model=128, d_ff=256, heads=2, seq=64, batch=4, micro=2,
                                 dtype="bf16", kind="decoder", loss="xent_ls", vocab=1000,
                                 label_smoothing=0.1, mem_seq=32)


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _flat(part):
    gl, gh = part.grads()
    return np.concatenate([v.ravel() for p in gl for v in p.values()] + [v.ravel() for v in gh.values()])


def _steps(cfg, seed, n=2, keep=False, lr=0.0, fwd_streams=2, bwd_streams=2):
    """n steps of one partition; per step the outputs, the loss and every
    gradient (fp32 arrays / tensors)."""
    from paper_1811_06965_amd.runtime import Partition
    case = synth.make_case(cfg, seed, perturb=True)
    out = []
    with Partition(cfg, keep_activations=keep) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        for _ in range(n):
            o = part.step(inp["x"], inp["mem"], inp["dy"], lr=lr, want_recomputed=True, fwd_streams=fwd_streams,
                          bwd_streams=bwd_streams)
            torch.cuda.synchronize()
            out.append(dict(y=_bits(o["y"]), y_remat=_bits(o["y_remat"]), dx=_bits(o["dx"]),
                            dmem=None if o["dmem"] is None else _bits(o["dmem"]), loss=o["loss"], g=_flat(part)))
    return out


def _same(a, b):
    for ra, rb in zip(a, b):
        for k in ("y", "y_remat", "dx", "dmem"):
            if ra[k] is None:
                assert rb[k] is None
                continue
            assert torch.equal(ra[k], rb[k]), k
        assert (ra["loss"] or 0.0) == (rb["loss"] or 0.0)
        assert np.array_equal(ra["g"], rb["g"])


# ------------------------------------------------ stored activations (f2)
@pytest.mark.parametrize("cfg", [TINY, ENC512_SMALL, RAGGED_BF16, DEC_SMALL_BF16], ids=lambda c: c.name)
def test_kept_activations_equal_rematerialisation_bitwise(cfg):
    """Keeping every micro-batch's intermediates (no recompute) and
    re-materialising them give the same outputs, loss and gradients bit for
    bit: the recompute is the same F_k, run by the same kernels."""
    remat = _steps(cfg, 21, lr=1e-3 if cfg.loss != "none" else 0.0)
    keep = _steps(cfg, 21, keep=True, lr=1e-3 if cfg.loss != "none" else 0.0)
    _same(remat, keep)
    for r in keep:
        assert torch.equal(r["y"], r["y_remat"])


def _free():
    torch.cuda.synchronize()
    return torch.cuda.mem_get_info()[0]


@pytest.mark.parametrize("keep", [False, True], ids=["remat", "kept"])
def test_device_memory_matches_the_plan_and_steps_allocate_nothing(keep):
    """Free device memory before and after configure differs by the planned
    bytes (params, grads, stash, workspace; the allocator rounds each of the
    few buffers up to its page size), and after a first step, two full steps
    -- every micro-batch's forward and backward and the update -- change it by
    nothing."""
    from paper_1811_06965_amd import gp
    from paper_1811_06965_amd.runtime import Partition, make_config
    cfg = ENC512_SMALL.with_(layers=4)
    case = synth.make_case(cfg, 22, perturb=True)
    x = torch.tensor(case["x"], dtype=torch.float32).to("cuda", torch.bfloat16)
    t = torch.tensor(case["target"], dtype=torch.float32).to("cuda", torch.bfloat16)
    y, dx = torch.empty_like(x), torch.empty_like(x)
    plan = gp.gp_memory_plan(cfg.layers, cfg.d_model, cfg.d_ff, cfg.heads, make_config(cfg, cfg.micro,
                                                                                         keep_activations=keep))
    planned = sum(plan.values())
    f0 = _free()
    with Partition(cfg, keep_activations=keep) as part:
        f1 = _free()
        assert part.memory() == plan
        used = f0 - f1
        assert planned <= used <= planned + 64 * 2 ** 20, (used, planned)
        part.load_params(case["layers"], case["head"])
        part.step(x, None, t, lr=1e-3, y=y, dx=dx)  # first launches load the kernels' code
        f2 = _free()
        for _ in range(2):
            part.step(x, None, t, lr=1e-3, y=y, dx=dx)
        f3 = _free()
        assert f3 == f2, (f2, f3)
    print(f"{'kept' if keep else 'remat'}: planned {planned / 2**20:.1f} MiB, measured {used / 2**20:.1f} MiB")


# ---------------------------------------------------------------- poison
@pytest.mark.parametrize("cfg,keep,env", [(TINY, False, {}), (ENC512_SMALL, False, {}),
                                          (RAGGED_BF16, False, {"GP_GEMM_TILE": "18", "GP_GEMM_SPLITS": "2"}),
                                          (DEC_SMALL_BF16, False, {}), (ENC512_SMALL, True, {}), (DEC_F32, False, {}),
                                          (ENC512_SMALL.with_(batch=12, micro=6), False, {"GP_DW_GROUP": "4"})],
                         ids=["tiny", "enc512_small", "ragged_split2", "dec_small", "enc512_kept", "dec_f32",
                              "enc512_m6_groups_of_4"])
def test_poisoned_workspace_changes_no_bit(cfg, keep, env, monkeypatch):
    """GP_POISON=1 fills every workspace set with NaN before the pass that
    rewrites it, the backward scratch, the split-K partials of all three
    streams and the loss partials before each backward, and the gradient
    accumulators and LayerNorm partial sums before the first backward of each
    mini-batch.  A read of anything stale would turn results into NaN: two
    steps are bit-identical to the unpoisoned ones."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    lr = 1e-3 if cfg.loss != "none" else 0.0
    clean = _steps(cfg, 23, keep=keep, lr=lr)
    monkeypatch.setenv("GP_POISON", "1")
    poisoned = _steps(cfg, 23, keep=keep, lr=lr)
    for r in poisoned:
        assert np.isfinite(r["g"]).all()
    _same(clean, poisoned)


# ---------------------------------------------- forwards on two streams
@pytest.mark.parametrize("cfg,keep", [(TINY, False), (ENC512_SMALL, False), (RAGGED_BF16, False),
                                      (DEC_SMALL_BF16, False), (ENC512_SMALL, True),
                                      (ENC512_SMALL.with_(batch=12, micro=6), False)],
                         ids=["tiny", "enc512_small", "ragged_pairs", "dec_small", "enc512_kept", "enc512_m6"])
def test_forwards_on_two_streams_change_no_bit(cfg, keep, monkeypatch):
    """The odd micro-batches' forwards issued on a second stream (the library's
    second first-pass slot; with recompute pairs, the early recompute of the
    last pair reads the stash the other stream wrote) against every forward on
    the launch stream in one slot (GP_FWD_LANES=1), with the workspace
    poisoned: three steps with an update between them (which the second
    stream's forwards must wait for) are bit-identical."""
    lr = 1e-3 if cfg.loss != "none" else 0.0
    monkeypatch.setenv("GP_POISON", "1")
    monkeypatch.setenv("GP_FWD_LANES", "1")
    one = _steps(cfg, 31, n=3, keep=keep, lr=lr, fwd_streams=1)
    monkeypatch.delenv("GP_FWD_LANES")
    two = _steps(cfg, 31, n=3, keep=keep, lr=lr, fwd_streams=2)
    for r in two:
        assert np.isfinite(r["g"]).all()
    _same(one, two)


LANES_F32 = synth.PartitionConfig("lanes_f32", layers=2, d_model=64, d_ff=128, heads=2, seq=16, batch=8, micro=4,
                                  dtype="f32", loss="none")
LANES_DEC = synth.PartitionConfig("lanes_dec", layers=2, d_model=256, d_ff=512, heads=4, seq=64, batch=4, micro=2,
                                  kind="decoder", mem_seq=64, loss="none")


@pytest.mark.parametrize("cfg", [RAGGED_BF16, RAGGED_BF16.with_(name="ragged_m3", batch=9, micro=3),
                                 RAGGED_BF16.with_(name="ragged_m6", batch=18, micro=6), LANES_F32, LANES_DEC,
                                 ENC512_SMALL, DEC_SMALL_BF16, DEC_SMALL_BF16.with_(name="dec_xent_m3", batch=6,
                                                                                   micro=3)],
                         ids=lambda c: c.name)
def test_backward_lanes_change_no_bit(cfg, monkeypatch):
    """The two members of a recompute pair back-propagated side by side (the
    odd micro-batch on a second stream, in the library's second backward
    lane; M odd leaves the top micro-batch alone) against one lane on one
    stream, with the workspace poisoned: three steps with updates between
    them are bit-identical, the loss included (the LayerNorm partial sums,
    the loss sum and the head's gradient keep their micro-batch order)."""
    from paper_1811_06965_amd.runtime import Partition
    monkeypatch.setenv("GP_POISON", "1")
    monkeypatch.setenv("GP_BWD_LANES", "1")
    with Partition(cfg) as part:
        ws_one = part.memory()["workspace"]
    one = _steps(cfg, 37, n=3, lr=1e-3, fwd_streams=1, bwd_streams=1)
    monkeypatch.delenv("GP_BWD_LANES")
    with Partition(cfg) as part:
        assert part.memory()["workspace"] > ws_one  # the second lane's scratch: the lanes are on
    two = _steps(cfg, 37, n=3, lr=1e-3)
    for r in two:
        assert np.isfinite(r["g"]).all()
    _same(one, two)


@pytest.mark.parametrize("cfg", [RAGGED_BF16.with_(name="ragged_m6", batch=18, micro=6), DEC_SMALL_BF16],
                         ids=lambda c: c.name)
def test_backward_lanes_without_early_recompute_change_no_bit(cfg, monkeypatch):
    """As above with the early recompute off (GP_REMAT_EARLY=0, the default
    at 2048 rows per micro-batch): the top pair is then re-materialised by
    the odd member's call on its own stream, in the second lane's scratch."""
    monkeypatch.setenv("GP_REMAT_EARLY", "0")
    test_backward_lanes_change_no_bit(cfg, monkeypatch)


@pytest.mark.parametrize("cfg", [RAGGED_BF16, ENC512_SMALL, DEC_SMALL_BF16, LANES_DEC], ids=lambda c: c.name)
def test_per_layer_update_changes_no_bit(cfg, monkeypatch):
    """Each layer's weights updated as soon as the last backward is past that
    layer (on the recompute stream, beside the backward of the layers below)
    against the whole update after the last backward (GP_LAYER_UPDATE=0):
    three steps with lr > 0 and the workspace poisoned are bit-identical, so
    no backward read of a layer's weights sees them updated."""
    monkeypatch.setenv("GP_POISON", "1")
    monkeypatch.setenv("GP_LAYER_UPDATE", "0")
    whole = _steps(cfg, 41, n=3, lr=1e-3)
    monkeypatch.delenv("GP_LAYER_UPDATE")
    per_layer = _steps(cfg, 41, n=3, lr=1e-3)
    _same(whole, per_layer)


# --------------------------------------------------------------- RMSProp
def test_rmsprop_two_steps_match_oracle():
    """Two mini-batches with RMSProp (fp32): parameters after each update
    against the oracle's, relative to the size of the update."""
    from oracle import gpipe
    from paper_1811_06965_amd.runtime import Partition
    cfg = TINY.with_(optimizer="rmsprop", rms_decay=0.9, rms_eps=1e-8)
    case = synth.make_case(cfg, 24, perturb=True)
    lr = 1e-3
    ref_case, state = case, None
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        for step in range(2):
            ref = gpipe.gpipe_step(cfg, ref_case, cfg.micro, lr=lr, opt_state=state)
            part.step(inp["x"], inp["mem"], inp["dy"], lr=lr)
            pl, _ = part.params()
            for l in range(cfg.layers):
                for k, v in ref["layers"][l].items():
                    delta = np.abs(v - case["layers"][l][k]).max()
                    err = np.abs(pl[l][k] - v).max()
                    if k == "bk":  # analytically zero gradient: round-off / sqrt(eps) only
                        assert err <= 1e-6, (step, l, k, err)
                        continue
                    assert err <= 1e-4 * delta + 1e-7 * np.abs(v).max(), (step, l, k, err, delta)
            ref_case, state = dict(case, layers=ref["layers"], head=ref["head"]), ref["opt_state"]


def test_rmsprop_bf16_runs_and_holds_twelve_bytes_per_parameter():
    from paper_1811_06965_amd.runtime import Partition
    cfg = ENC512_SMALL.with_(optimizer="rmsprop", rms_decay=0.9, rms_eps=1e-8)
    case = synth.make_case(cfg, 25, perturb=True)
    with Partition(cfg) as part, Partition(cfg.with_(optimizer="sgd")) as sgd:
        # masters, gradient accumulators and running mean squares: 12 bytes per parameter
        assert part.memory()["params"] - sgd.memory()["params"] == part.memory()["grads"]
        part.load_params(case["layers"], case["head"])
        before, _ = part.params()
        inp = part.device_inputs(case)
        loss = part.step(inp["x"], inp["mem"], inp["dy"], lr=1e-4)["loss"]
        after, _ = part.params()
        assert np.isfinite(loss)
        moved = np.abs(after[0]["w1"] - before[0]["w1"])
        assert np.isfinite(after[0]["w1"]).all() and 0 < moved.max() < 1e-3


@pytest.mark.parametrize("opt", ["sgd", "rmsprop"])
@pytest.mark.parametrize("cfg", [ENC512_SMALL, DEC_BF16], ids=lambda c: c.name)
def test_bf16_update_applies_the_accumulated_gradient(cfg, opt):
    """The bf16 partitions' step: every parameter tensor, head included,
    moves by exactly the SGD or RMSProp step of its accumulated gradient (fp32
    on the host, within two roundings of the parameter and a few of the
    step), two steps in a row.  The encoder's linears are whole 64 x 64 tiles, so its weights
    are updated in the pass that rewrites their working copies (biases and
    LayerNorm parameters from a range table); the decoder's 1000-way head is
    not, so it takes the separate update and refresh kernels."""
    from paper_1811_06965_amd.runtime import Partition
    cfg = cfg.with_(optimizer=opt, rms_decay=0.9, rms_eps=1e-8)
    case = synth.make_case(cfg, 26, perturb=True)
    lr, rho, eps = np.float32(1e-3), np.float32(0.9), np.float32(1e-8)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        ms = None
        for _ in range(2):
            w0 = part.params()
            out = part.step(inp["x"], inp["mem"], inp["dy"], lr=float(lr), want_y=False)
            torch.cuda.synchronize()
            g = part.grads()
            w1 = part.params()
            if ms is None:
                ms = ([{k: np.zeros_like(v) for k, v in d.items()} for d in g[0]], {k: np.zeros_like(v) for k, v in g[1].items()})
            for side in (0, 1):
                groups = zip(w0[0], g[0], w1[0], ms[0]) if side == 0 else [(w0[1], g[1], w1[1], ms[1])]
                for a, gg, b, m in groups:
                    for k in a:
                        gk = gg[k].astype(np.float32)
                        if opt == "sgd":
                            step = lr * gk
                        else:
                            m[k] = rho * m[k] + (np.float32(1) - rho) * (gk * gk)
                            step = lr * gk / np.sqrt(m[k] + eps)
                        want = a[k] - step
                        # one rounding of the parameter, plus a few of the step's
                        # own (a fused multiply-add, the square root and the
                        # division may round differently from the host's)
                        tol = (np.spacing(np.maximum(np.abs(want), np.abs(a[k]))) * 2
                               + np.spacing(np.abs(step)) * 8).astype(np.float32)
                        assert (np.abs(b[k] - want) <= tol).all(), (k, np.abs(b[k] - want).max())


# ------------------------------------------------------- logit clipping
def _clip_at(cfg, case, q):
    """A clip bound at the q-quantile of the oracle's |logits|."""
    from oracle import gpipe, transformer as tf
    y, _ = gpipe.partition_forward(cfg, case["layers"], case["x"], case["mem"])
    h, _ = tf.layer_norm(y, case["head"]["lnf_g"], case["head"]["lnf_b"], cfg.ln_eps)
    return float(np.quantile(np.abs(tf.linear(h, case["head"]["wout"], case["head"]["bout"])), q))


@pytest.mark.parametrize("cfg", [DEC_F32, DEC_BF16], ids=lambda c: c.name)
def test_logit_clipping_matches_oracle(cfg):
    """Section 5: logits clipped to [-c, c] with c at the 70th percentile of
    their magnitude (most rows have clipped entries), loss and every gradient
    against the oracle."""
    from oracle import gpipe
    from paper_1811_06965_amd.runtime import Partition
    case = synth.make_case(cfg, 26, perturb=True)
    wout = synth.round_storage(4.0 * case["head"]["wout"], cfg.dtype)
    case["head"] = dict(case["head"], wout=wout)
    cfg = cfg.with_(logit_clip=_clip_at(cfg, case, 0.7))
    ref = gpipe.gpipe_step(cfg, case, cfg.micro)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0)
        torch.cuda.synchronize()
        gl, gh = part.grads()
    mode, tol, out_tol = ("rel", 1e-4, 1e-4) if cfg.dtype == "f32" else ("cos", 0.999, 2e-2)
    assert abs(out["loss"] - ref["loss"]) <= out_tol * abs(ref["loss"]), (out["loss"], ref["loss"])
    dx = to_np(out["dx"])
    if mode == "rel":
        assert rel_err(dx, ref["dx"]) <= tol
    else:
        assert cosine(dx, ref["dx"]) >= tol
    compare_grads(gl, gh, ref["grads"], ref["head_grads"], mode, tol)


# ------------------------------------------- scaled-down FFN initialisation
def test_fixup_initialised_stack_matches_oracle():
    """The 8-layer enc512 workload with its feed-forward matrices initialised
    at 1/8 of Xavier-uniform (Section 5): a feed-forward branch about 64 times
    smaller than the residual stream, through the bf16 path."""
    from oracle import gpipe
    from paper_1811_06965_amd.runtime import Partition
    cfg = synth.CONFIGS["enc512"].with_(name="enc512_fixup", batch=8, micro=4, fixup_layers=8)
    case = synth.make_case(cfg, 27, perturb=True)
    ref = gpipe.gpipe_step(cfg, case, cfg.micro)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0)
        torch.cuda.synchronize()
        gl, gh = part.grads()
    assert rel_err(to_np(out["y"]), ref["y"]) <= 2e-2
    assert abs(out["loss"] - ref["loss"]) <= 2e-2 * abs(ref["loss"])
    assert cosine(to_np(out["dx"]), ref["dx"]) >= 0.999
    compare_grads(gl, gh, ref["grads"], ref["head_grads"], "cos", 0.999)


# ----------------------------------------------- grouped weight gradients
RAGGED_F32_M3 = synth.PartitionConfig("ragged_f32_m3", layers=2, d_model=96, d_ff=160, heads=3, seq=40,
                                      batch=6, micro=3, dtype="f32", loss="none")
RAGGED_F32_M5 = RAGGED_F32_M3.with_(name="ragged_f32_m5", batch=10, micro=5)
DEC_SMALL_BF16_M6 = DEC_SMALL_BF16.with_(name="dec_small_bf16_m6", batch=6, micro=6)


@pytest.mark.parametrize("group", ["2", "4"])
@pytest.mark.parametrize("cfg", [TINY, RAGGED_F32_M3, RAGGED_F32_M5, DEC_SMALL_BF16, DEC_SMALL_BF16_M6],
                         ids=lambda c: c.name)
def test_grouped_weight_gradients_match_ungrouped(cfg, group, monkeypatch):
    """The weight gradients of a group of micro-batches (two, or four; the
    last group cut short when M is not a multiple) as one GEMM over the
    members' rows (GP_PAIR_DW with GP_DW_GROUP) against one GEMM per
    micro-batch: outputs and input gradients are bit-identical (they do not
    depend on the weight gradients), the accumulated gradients agree to the
    rounding of the accumulation order (fp32: 1e-5; bf16 parts: 1e-3)."""
    res = {}
    for pair in ("0", "1"):
        monkeypatch.setenv("GP_PAIR_DW", pair)
        monkeypatch.setenv("GP_DW_GROUP", group)
        res[pair] = _steps(cfg, 28, n=2, lr=1e-3 if cfg.loss != "none" else 0.0)
    tol = 1e-5 if cfg.dtype == "f32" else 1e-3
    for step, (a, b) in enumerate(zip(res["0"], res["1"])):
        # with lr > 0 the second step starts from slightly different parameters
        if step == 0 or cfg.loss == "none":
            for k in ("y", "y_remat", "dx", "dmem"):
                if a[k] is not None:
                    assert torch.equal(a[k], b[k]), (step, k)
        assert np.abs(a["g"] - b["g"]).max() <= tol * np.abs(a["g"]).max(), step


# ------------------------------------------------------------------ resume
@pytest.mark.parametrize("cfg", [TINY, ENC512_SMALL], ids=lambda c: c.name)
def test_resume_from_parameters_reproduces_the_next_step_bitwise(cfg):
    """Checkpoint and resume: one step, gp_get_param of every tensor, a new
    partition loaded with gp_set_param, one more step -- the same parameters,
    gradients and boundary outputs, bit for bit, as two steps in one partition
    (the working copies are rebuilt from the fp32 masters by the same rounding)."""
    from paper_1811_06965_amd.runtime import Partition
    case = synth.make_case(cfg, 29, perturb=True)
    lr = 1e-3
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        part.step(inp["x"], inp["mem"], inp["dy"], lr=lr)
        mid_layers, mid_head = part.params()
        o = part.step(inp["x"], inp["mem"], inp["dy"], lr=lr)
        torch.cuda.synchronize()
        ref = (_bits(o["y"]), _bits(o["dx"]), o["loss"], _flat(part), part.params())
    with Partition(cfg) as part:
        part.load_params(mid_layers, mid_head)
        inp = part.device_inputs(case)
        o = part.step(inp["x"], inp["mem"], inp["dy"], lr=lr)
        torch.cuda.synchronize()
        got = (_bits(o["y"]), _bits(o["dx"]), o["loss"], _flat(part), part.params())
    assert torch.equal(ref[0], got[0]) and torch.equal(ref[1], got[1])
    assert ref[2] == got[2]
    assert np.array_equal(ref[3], got[3])
    for a, b in zip(ref[4][0], got[4][0]):
        for k in a:
            assert np.array_equal(a[k], b[k]), k
