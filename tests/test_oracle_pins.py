"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each check is chosen so that a plausible mistake in the oracle (a dropped
term, a wrong sign or index, a transposed operand) fails at least one of them:

* central finite differences of the forward pin every hand-derived gradient;
* an independent library implementation (torch's fp64 CPU layer_norm,
  scaled_dot_product_attention, cross_entropy with label smoothing and
  autograd) pins the forward definitions and again the gradients;
* the GPipe invariants (Sections 2.2-2.3): the sum of the micro-batch
  gradients equals the mini-batch gradient, and the re-materialised backward
  equals the stored-activation backward bit for bit;
* closed forms and special cases (identity residual, uniform attention,
  LayerNorm moments, ln V for a zero vocabulary projection, zero MSE);
* Table 1's Transformer-L parameter counts (Section 3).
"""
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle import gpipe, transformer as tf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TINY = synth.CONFIGS["tiny"]
TINY_BOUNDARY = TINY.with_(name="tiny_boundary", loss="none")
TINY_DEC = synth.PartitionConfig("tiny_dec", layers=2, d_model=32, d_ff=64, heads=2, seq=8,
                                 batch=4, micro=2, dtype="f32", kind="decoder",
                                 loss="xent_ls", vocab=40, label_smoothing=0.1, mem_seq=6)


def _loss_of(cfg, case):
    return gpipe.minibatch_step(cfg, case)["loss"]


def _with_param(case, where, name, value):
    c = dict(case)
    if where == "head":
        c["head"] = dict(case["head"])
        c["head"][name] = value
    else:
        c["layers"] = [dict(p) for p in case["layers"]]
        c["layers"][where][name] = value
    return c


def _relu_masks(cfg, case):
    out = []
    _, caches = gpipe.partition_forward(cfg, case["layers"], case["x"], case["mem"])
    for c in caches:
        out.append(c["z"] > 0)
    return out


def _central(f, h):
    """Fourth-order central difference of t -> f(t) at 0:
    (-f(2h) + 8 f(h) - 8 f(-h) + f(-2h)) / (12 h); error O(h^4)."""
    return (-f(2 * h) + 8 * f(h) - 8 * f(-h) + f(-2 * h)) / (12 * h)


def _fd_directional(cfg, case, where, name, direction, h):
    base = case["head"][name] if where == "head" else case["layers"][where][name]
    at = lambda t: _with_param(case, where, name, base + t * direction)
    # guard against crossing a ReLU kink inside the stencil
    m0 = _relu_masks(cfg, at(-2 * h))
    same = all((a == b).all() for a, b in zip(m0, _relu_masks(cfg, at(2 * h))))
    return _central(lambda t: _loss_of(cfg, at(t)), h), same


def _fd_check(cfg, seed, n_dirs=4, n_coords=6, h=1e-4, tol=1e-6):
    """Compare analytic gradients with central finite differences (fp64).

    Directional derivatives along random unit directions per parameter tensor
    and along single coordinates, with the fourth-order central stencil.
    Pass when |fd - an| <= tol * max(|fd|, |an|, 1e-3 ||g||_2) + atol, where
    atol = 20 eps max(|L|, 1) / h bounds the stencil's fp64 round-off, so a
    gradient that is analytically zero is compared at that level.  A stencil whose points lie on different sides
    of a ReLU kink is redrawn (up to 5 times) and otherwise skipped; at most a
    quarter of the checks may be skipped."""
    rng = np.random.default_rng(1000 + seed)
    case = synth.make_case(cfg, seed, perturb=True)
    ref = gpipe.minibatch_step(cfg, case)
    atol = 20 * np.finfo(np.float64).eps * max(abs(ref["loss"]), 1.0) / h
    targets = [(l, k) for l in range(cfg.layers) for k in case["layers"][l]]
    targets += [("head", k) for k in case["head"]]
    worst, done, skipped = 0.0, 0, 0
    for where, name in targets:
        g = ref["head_grads"][name] if where == "head" else ref["grads"][where][name]
        scale = 1e-3 * np.linalg.norm(g)
        checks = []
        for _ in range(n_dirs):
            d = rng.standard_normal(g.shape)
            checks.append(("dir", d / np.linalg.norm(d)))
        for _ in range(n_coords):
            checks.append(("coord", None))
        for kind, d in checks:
            for _attempt in range(5):
                if kind == "coord":
                    e = np.zeros(g.size)
                    e[rng.integers(g.size)] = 1.0
                    d = e.reshape(g.shape)
                fd, same = _fd_directional(cfg, case, where, name, d, h)
                if same:
                    break
                if kind == "dir":
                    d = rng.standard_normal(g.shape)
                    d /= np.linalg.norm(d)
            if not same:
                skipped += 1
                continue
            an = float((g * d).sum())
            err, bound = abs(fd - an), tol * max(abs(fd), abs(an), scale) + atol
            worst = max(worst, err / bound)
            done += 1
            assert err <= bound, (where, name, fd, an, err, bound)
    assert skipped <= (done + skipped) // 4, (skipped, done)
    # input gradient (and memory gradient for the decoder), same kink guard
    for key, gkey in (("x", "dx"), ("mem", "dmem")):
        if case.get(key) is None:
            continue
        g = ref[gkey]
        done_x = 0
        for _ in range(4 * n_dirs):
            d = rng.standard_normal(g.shape)
            d /= np.linalg.norm(d)

            def at(t):
                c = dict(case)
                c[key] = case[key] + t * d
                return c
            m0 = _relu_masks(cfg, at(-2 * h))
            if not all((a == b).all() for a, b in zip(m0, _relu_masks(cfg, at(2 * h)))):
                continue
            fd = _central(lambda t: _loss_of(cfg, at(t)), h)
            an = float((g * d).sum())
            err = abs(fd - an)
            assert err <= tol * max(abs(fd), abs(an), 1e-3 * np.linalg.norm(g)) + atol, (key, fd, an)
            done_x += 1
            if done_x == n_dirs:
                break
        assert done_x >= 1, key
    return worst


def test_finite_differences_tiny_mse():
    _fd_check(TINY, seed=0)


def test_finite_differences_tiny_boundary():
    _fd_check(TINY_BOUNDARY, seed=1, n_dirs=3, n_coords=3)


def test_finite_differences_tiny_decoder_xent():
    _fd_check(TINY_DEC, seed=2, n_dirs=3, n_coords=3)


# -------------------------------------------------------- GPipe invariants
def _rel(a, b):
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def _grad_rel(a, b, gref):
    """Max-abs relative error of one gradient tensor; tensors whose gradient is
    analytically zero (the key biases) are measured against 1e-6 of the
    largest gradient of the case instead of their own round-off noise."""
    top = max(np.abs(v).max() for v in gref.values())
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-6 * top))


def _all_grads(res):
    out = {}
    for l, g in enumerate(res["grads"]):
        for k, v in g.items():
            out[(l, k)] = v
    for k, v in res["head_grads"].items():
        out[("head", k)] = v
    return out


@pytest.mark.parametrize("cfg", [TINY, TINY_BOUNDARY, TINY_DEC], ids=lambda c: c.name)
def test_microbatch_sum_equals_minibatch_gradient(cfg):
    """Sections 2.2 and 1: accumulated micro-batch gradients equal the
    mini-batch gradient, whatever M (1e-10 relative in fp64)."""
    case = synth.make_case(cfg, 3, perturb=True)
    ref = gpipe.minibatch_step(cfg, case, lr=0.1)
    gref = _all_grads(ref)
    for M in (1, 2, 4):
        if cfg.batch % M:
            continue
        out = gpipe.gpipe_step(cfg, case, M, lr=0.1)
        for k, v in _all_grads(out).items():
            assert _grad_rel(v, gref[k], gref) < 1e-10, (M, k)
        assert _rel(out["y"], ref["y"]) < 1e-12
        assert _rel(out["dx"], ref["dx"]) < 1e-10
        if cfg.kind == "decoder":
            assert _rel(out["dmem"], ref["dmem"]) < 1e-10
        assert abs(out["loss"] - ref["loss"]) <= 1e-10 * abs(ref["loss"])
        for lnew, lref in zip(out["layers"], ref["layers"]):
            for k in lnew:
                assert _rel(lnew[k], lref[k]) < 1e-12


def test_microbatch_sum_eight_microbatches():
    case = synth.make_case(TINY, 4, perturb=True)
    ref = _all_grads(gpipe.minibatch_step(TINY, case))
    out = _all_grads(gpipe.gpipe_step(TINY, case, 8))
    for k in ref:
        assert _grad_rel(out[k], ref[k], ref) < 1e-10, k


@pytest.mark.parametrize("cfg", [TINY, TINY_DEC], ids=lambda c: c.name)
def test_remat_equals_stored_activations_bitwise(cfg):
    """Section 2.3: recomputing F_k in the backward pass yields exactly the
    gradients of the stored-activation backward."""
    case = synth.make_case(cfg, 5, perturb=True)
    a = gpipe.gpipe_step(cfg, case, 2, remat=True)
    b = gpipe.gpipe_step(cfg, case, 2, remat=False)
    ga, gb = _all_grads(a), _all_grads(b)
    for k in ga:
        assert np.array_equal(ga[k], gb[k]), k
    assert np.array_equal(a["dx"], b["dx"])
    assert a["loss"] == b["loss"]


def test_schedule_order():
    trace = []
    case = synth.make_case(TINY, 0)
    gpipe.gpipe_step(TINY, case, 4, trace=trace)
    assert trace == [("fwd", 0), ("fwd", 1), ("fwd", 2), ("fwd", 3),
                     ("remat", 3), ("bwd", 3), ("remat", 2), ("bwd", 2),
                     ("remat", 1), ("bwd", 1), ("remat", 0), ("bwd", 0)]


def test_unequal_split_rejected():
    case = synth.make_case(TINY, 0)
    with pytest.raises(ValueError):
        gpipe.gpipe_step(TINY, case, 3)


def test_boundary_linearity():
    """Boundary partitions: gradients are linear in the arriving gradient G."""
    cfg = TINY_BOUNDARY
    c1 = synth.make_case(cfg, 6, perturb=True)
    c2 = dict(c1)
    c2["dy"] = np.random.default_rng(7).standard_normal(c1["dy"].shape)
    c3 = dict(c1)
    c3["dy"] = 0.5 * c1["dy"] - 2.0 * c2["dy"]
    r1, r2, r3 = (gpipe.minibatch_step(cfg, c) for c in (c1, c2, c3))
    g1, g2, g3 = _all_grads(r1), _all_grads(r2), _all_grads(r3)
    for k in g1:
        comb = 0.5 * g1[k] - 2.0 * g2[k]
        top = max(np.abs(v).max() for v in g3.values())
        assert np.abs(g3[k] - comb).max() <= 1e-12 * max(np.abs(comb).max(), 1e-3 * top), k
    assert np.abs(r3["dx"] - (0.5 * r1["dx"] - 2.0 * r2["dx"])).max() < 1e-12


def test_step_is_sgd():
    case = synth.make_case(TINY, 8, perturb=True)
    lr = 0.37
    out = gpipe.gpipe_step(TINY, case, 2, lr=lr)
    for p, g, pn in zip(case["layers"], out["grads"], out["layers"]):
        for k in p:
            assert np.array_equal(pn[k], p[k] - lr * g[k])


# ------------------------------------------------------------ closed forms
def test_residual_identity():
    """Wo = W2 = 0 and zero biases make every layer the identity; the
    gradients of everything upstream of the zeroed projections vanish."""
    cfg = TINY_BOUNDARY
    case = synth.make_case(cfg, 9)
    for p in case["layers"]:
        for k in p:
            if k in ("wo", "w2") or k.startswith("b") and k != "b1":
                p[k] = np.zeros_like(p[k])
    res = gpipe.minibatch_step(cfg, case)
    assert np.array_equal(res["y"], case["x"])
    assert np.array_equal(res["dx"], case["dy"])
    for g in res["grads"]:
        for k in ("wq", "wk", "wv", "bq", "bk", "bv", "w1", "b1", "ln1_g", "ln1_b",
                  "ln2_g", "ln2_b"):
            assert not g[k].any(), k
        assert g["wo"].any() and g["w2"].any()


def test_attention_special_cases():
    rng = np.random.default_rng(10)
    n, S, D, H = 2, 5, 12, 3
    q, k, v = (rng.standard_normal((n, S, D)) for _ in range(3))
    # single key: attention returns the value row
    out, _ = tf.attention(q[:, :1], k[:, :1], v[:, :1], H, causal=False)
    assert np.abs(out - v[:, :1]).max() < 1e-14
    # zero queries: uniform weights, output = mean of values over keys
    out, _ = tf.attention(np.zeros_like(q), k, v, H, causal=False)
    assert np.abs(out - v.mean(axis=1, keepdims=True)).max() < 1e-14
    # causal: query 0 sees key 0 only; query i averages keys <= i when q = 0
    out, _ = tf.attention(q, k, v, H, causal=True)
    assert np.abs(out[:, 0] - v[:, 0]).max() < 1e-14
    out, _ = tf.attention(np.zeros_like(q), k, v, H, causal=True)
    cum = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None]
    assert np.abs(out - cum).max() < 1e-14


def test_key_bias_gradient_vanishes():
    """Adding b_k to every key shifts each score row by the constant q.b_k,
    which the row softmax ignores: the key-bias gradient is exactly zero in
    exact arithmetic, while the query and value biases carry signal."""
    for cfg in (TINY, TINY_DEC):
        res = gpipe.minibatch_step(cfg, synth.make_case(cfg, 15, perturb=True))
        for g in res["grads"]:
            assert np.abs(g["bk"]).max() <= 1e-12 * np.abs(g["bv"]).max()
            assert np.abs(g["bq"]).max() > 1e-6 * np.abs(g["bv"]).max()
            if cfg.kind == "decoder":
                assert np.abs(g["xbk"]).max() <= 1e-12 * np.abs(g["xbv"]).max()


def test_layer_norm_moments():
    rng = np.random.default_rng(11)
    x = 3.0 + 2.0 * rng.standard_normal((7, 33))
    eps = 1e-5
    y, _ = tf.layer_norm(x, np.ones(33), np.zeros(33), eps)
    var = x.var(axis=-1)
    assert np.abs(y.mean(axis=-1)).max() < 1e-14
    assert np.abs(y.var(axis=-1) - var / (var + eps)).max() < 1e-14


def test_xent_zero_projection_is_log_vocab():
    V = 32000
    rng = np.random.default_rng(12)
    y = rng.standard_normal((2, 3, 16))
    hp = {"lnf_g": np.ones(16), "lnf_b": np.zeros(16), "wout": np.zeros((16, V)),
          "bout": np.zeros(V)}
    labels = rng.integers(0, V, size=(2, 3))
    for ls in (0.0, 0.1, 0.5):
        loss, dy, g = tf.xent_ls_head(y, labels, hp, ls, 1e-5, 6.0)
        assert abs(loss - 10.373491181781864) < 1e-12
        assert abs(math.log(V) - 10.373491181781864) < 1e-15
    # every row of dZ sums to zero, so the bias gradient sums to zero
    assert abs(g["bout"].sum()) < 1e-14


def test_xent_without_smoothing_is_textbook():
    rng = np.random.default_rng(13)
    y = rng.standard_normal((1, 4, 8))
    hp = {"lnf_g": np.ones(8), "lnf_b": np.zeros(8), "wout": rng.standard_normal((8, 11)),
          "bout": rng.standard_normal(11)}
    labels = rng.integers(0, 11, size=(1, 4))
    loss, _, _ = tf.xent_ls_head(y, labels, hp, 0.0, 1e-5, 4.0)
    h, _ = tf.layer_norm(y, hp["lnf_g"], hp["lnf_b"], 1e-5)
    Z = (h @ hp["wout"] + hp["bout"])[0]
    ref = 0.0
    for t in range(4):
        ref += -Z[t, labels[0, t]] + math.log(sum(math.exp(z) for z in Z[t]))
    assert abs(loss - ref / 4) < 1e-13


def test_mse_zero_when_target_is_output():
    case = synth.make_case(TINY, 14, perturb=True)
    case["target"] = gpipe.minibatch_step(TINY, case)["y"]
    res = gpipe.minibatch_step(TINY, case)
    assert res["loss"] == 0.0
    for g in res["grads"]:
        for k, v in g.items():
            assert not v.any(), k
    assert not res["dx"].any()


# ------------------------------------------------ Table 1 parameter counts
def test_table1_transformer_parameter_counts():
    """Per-layer count (4 D^2 + 2 D F weights, 4 D + F + D biases, 4 D LayerNorm)
    times L, plus untied input and output 32k x D matrices, reproduces the
    Transformer-L parameter counts of Table 1 to the printed digits."""
    with open(os.path.join(GOLDEN, "table1_transformer_params.json")) as f:
        t1 = json.load(f)
    D, F, V = t1["d_model"], t1["d_ff"], t1["vocab"]
    for L, pub, digits in zip(t1["layers"], t1["params_published"], t1["params_published_digits"]):
        cfg = synth.PartitionConfig("t1", layers=L, d_model=D, d_ff=F, heads=t1["heads"],
                                    seq=1024, batch=32, micro=1)
        total = gpipe.param_count(cfg) + 2 * V * D
        mag = 10 ** (math.floor(math.log10(pub)) - digits + 1)
        assert abs(total - pub) <= mag, (L, total, pub)


def test_param_count_matches_arrays():
    for cfg in (TINY, TINY_DEC, synth.CONFIGS["enc512"]):
        layers, head = synth.make_params(cfg, 0)
        n = sum(v.size for p in layers for v in p.values()) + sum(v.size for v in head.values())
        assert n == gpipe.param_count(cfg)
