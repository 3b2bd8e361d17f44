"""GPU parity at the workloads' full sizes.

Two kinds of check, both against the fp64 oracle on the same seeded inputs:

* The launch configuration the benchmark times (enc1024 at every M of its
  sweep, enc2048 at M = 32, dec1024 at M = 16), checked on sampled
  sequences.  Sequences of a mini-batch are independent in a partition:
  attention mixes positions of one sequence only and LayerNorm works per
  token.  So the output y and the input gradient dX of a sequence depend only
  on that sequence, and the oracle can compute them for a few sampled
  sequences.  For the parameter gradients, the boundary loss sum <Y, G> is
  linear in G: a GPU step with the boundary gradient zeroed outside the sample
  gives exactly the gradient the oracle computes over the sample alone.  One
  oracle run per seed serves every M (the accumulated gradient does not depend
  on M, Section 2.2).
* The real per-micro-batch shape (n = 4 sequences, T = 1024 token rows: the
  same kernels, tiles and launch shapes as the full workload) over a
  mini-batch of 8 sequences in M = 2 micro-batches, small enough for the
  oracle to run the whole mini-batch: every parameter gradient (the
  32000-way head's included), the loss, dX and dMem.

Tolerances as for the small bf16 cases: outputs and the loss max-abs relative
error <= 2e-2, gradients cosine >= 0.999.  The max-abs relative error of dX
and dMem is printed as well.
"""
import numpy as np
import pytest

import synth
from parity import compare_grads, cosine, rel_err, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _sub(case, sample):
    sub = {k: case[k][sample] for k in ("x", "mem", "dy", "target", "labels") if case.get(k) is not None}
    sub.setdefault("mem", None)
    return sub


def _oracle_on(cfg, case, sample):
    """The oracle's mini-batch forward, loss and backward over the sampled
    sequences alone (no update: the tests compare gradients at lr = 0)."""
    from oracle import gpipe
    sub = _sub(case, sample)
    cfg1 = cfg.with_(batch=len(sample), micro=1)
    y, caches = gpipe.partition_forward(cfg1, case["layers"], sub["x"], sub["mem"])
    loss, dy, g_head = gpipe.loss_and_grad(cfg1, case["head"], y, sub, gpipe.loss_norm(cfg1, len(sample)))
    dx, dmem, g_layers = gpipe.partition_backward(cfg1, case["layers"], caches, dy)
    return dict(y=y, dx=dx, dmem=dmem, loss=loss, grads=g_layers, head_grads=g_head)


def _sampled_step(cfg, case, sample, M):
    """One GPU step at M micro-batches with the boundary gradient zeroed
    outside the sample: y (every sequence), dX of the sample, and the
    parameter gradients over the sample."""
    from paper_1811_06965_amd.runtime import Partition
    with Partition(cfg, micro=M) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        keep = torch.zeros(cfg.batch, 1, 1, dtype=inp["dy"].dtype, device=inp["dy"].device)
        keep[sample] = 1
        out = part.step(inp["x"], None, (inp["dy"] * keep).contiguous(), lr=0.0, want_loss=False)
        torch.cuda.synchronize()
        gl, gh = part.grads()
        return to_np(out["y"]), to_np(out["dx"]), gl, gh


@pytest.fixture(scope="module")
def enc1024():
    cfg = synth.CONFIGS["enc1024"]
    case = synth.make_case(cfg, 5)
    sample = [3, 42]
    return cfg, case, sample, _oracle_on(cfg, case, sample)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("M", [4, 8, 16, 32, 64])
def test_enc1024_full_size_every_micro_batch_count(enc1024, M):
    """enc1024 (16 layers, d_model 1024, d_ff 8192, 16 heads, S 256, N 64) at
    each M of the benchmark sweep, and at M = 64 (one sequence per
    micro-batch, 256-row GEMMs); M = 4 runs the 4-wave attention kernels
    (4096 query blocks per launch), M = 32 the 512-row GEMM tiles."""
    cfg, case, sample, ref = enc1024
    y, dx, gl, gh = _sampled_step(cfg, case, sample, M)
    e_y, e_dx, c_dx = rel_err(y[sample], ref["y"]), rel_err(dx[sample], ref["dx"]), cosine(dx[sample], ref["dx"])
    print(f"enc1024 M={M}: y rel {e_y:.2e}, dx rel {e_dx:.2e} cos {c_dx:.6f}")
    assert e_y <= 2e-2, e_y
    assert c_dx >= 0.999, c_dx
    worst = compare_grads(gl, gh, ref["grads"], ref["head_grads"], "cos", 0.999)
    print(f"enc1024 M={M}: worst gradient cosine {worst:.6f}")


@pytest.fixture(scope="module")
def enc2048_case():
    cfg = synth.CONFIGS["enc2048"]
    return cfg, synth.make_case(cfg, 5)


@pytest.mark.timeout(600)
def test_enc2048_full_size_sampled(enc2048_case):
    """enc2048 (8 layers, d_model 2048, d_ff 16384, 32 heads) in its
    benchmark launch configuration, N = 128 in M = 32: y and dX of a sampled
    sequence and every parameter gradient over it."""
    cfg, case = enc2048_case
    sample = [77]
    y, dx, gl, gh = _sampled_step(cfg, case, sample, cfg.micro)
    ref = _oracle_on(cfg, case, sample)
    e_y, e_dx, c_dx = rel_err(y[sample], ref["y"]), rel_err(dx[sample], ref["dx"]), cosine(dx[sample], ref["dx"])
    print(f"enc2048 M=32 sampled: y rel {e_y:.2e}, dx rel {e_dx:.2e} cos {c_dx:.6f}")
    assert e_y <= 2e-2, e_y
    assert c_dx >= 0.999, c_dx
    compare_grads(gl, gh, ref["grads"], ref["head_grads"], "cos", 0.999)


def _whole_minibatch(cfg, case, M):
    """GPU step over the whole (small) mini-batch at M, and the oracle's plain
    mini-batch definition over the same inputs."""
    from oracle import gpipe
    from paper_1811_06965_amd.runtime import Partition
    with Partition(cfg, micro=M) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_loss=True)
        torch.cuda.synchronize()
        gl, gh = part.grads()
        res = dict(y=to_np(out["y"]), dx=to_np(out["dx"]), loss=out["loss"],
                   dmem=None if out["dmem"] is None else to_np(out["dmem"]))
    ref = gpipe.minibatch_step(cfg, case)
    return res, (gl, gh), ref


@pytest.mark.timeout(900)
def test_enc2048_real_micro_batch_shape_whole_minibatch(enc2048_case):
    """enc2048 at its real micro-batch shape (n = 4, T = 1024), all 8 layers,
    over the first 8 sequences of the seeded mini-batch in M = 2: y, dX and
    every parameter gradient against the oracle's whole mini-batch."""
    big_cfg, big = enc2048_case
    cfg = big_cfg.with_(batch=8, micro=2)
    case = dict(big, x=big["x"][:8], dy=big["dy"][:8])
    res, (gl, gh), ref = _whole_minibatch(cfg, case, 2)
    e_y, e_dx, c_dx = rel_err(res["y"], ref["y"]), rel_err(res["dx"], ref["dx"]), cosine(res["dx"], ref["dx"])
    print(f"enc2048 N=8 M=2: y rel {e_y:.2e}, dx rel {e_dx:.2e} cos {c_dx:.6f}")
    assert e_y <= 2e-2, e_y
    assert c_dx >= 0.999, c_dx
    worst = compare_grads(gl, gh, ref["grads"], ref["head_grads"], "cos", 0.999)
    print(f"enc2048 N=8 M=2: worst gradient cosine {worst:.6f}")


@pytest.fixture(scope="module")
def dec1024_case():
    cfg = synth.CONFIGS["dec1024"]
    return cfg, synth.make_case(cfg, 6)


@pytest.mark.timeout(600)
def test_decoder_head_full_size_sampled(dec1024_case):
    """dec1024: 8 decoder layers + 32000-way label-smoothed cross-entropy in
    the benchmark launch configuration, M = 16.  The loss is normalised by the
    whole mini-batch (N S tokens), so the sampled sequences' dX and dMem are
    the oracle's over the sample scaled by (sample size) / N."""
    from paper_1811_06965_amd.runtime import Partition
    cfg, case = dec1024_case
    sample = [9, 50]
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_loss=True)
        dx, dmem, loss = to_np(out["dx"]), to_np(out["dmem"]), out["loss"]
    ref = _oracle_on(cfg, case, sample)
    scale = len(sample) / cfg.batch
    c_dx, c_dm = cosine(dx[sample], ref["dx"] * scale), cosine(dmem[sample], ref["dmem"] * scale)
    print(f"dec1024 M=16 sampled: dx rel {rel_err(dx[sample], ref['dx'] * scale):.2e} cos {c_dx:.6f}, "
          f"dmem rel {rel_err(dmem[sample], ref['dmem'] * scale):.2e} cos {c_dm:.6f}")
    assert c_dx >= 0.999, c_dx
    assert c_dm >= 0.999, c_dm
    # per-token loss of random labels under Xavier weights stays near ln V
    assert np.isfinite(loss) and abs(loss - np.log(cfg.vocab)) < 1.0, loss


@pytest.mark.timeout(900)
def test_decoder_head_real_micro_batch_shape_whole_minibatch(dec1024_case):
    """dec1024 at its real micro-batch shape (n = 4, T = 1024), all 8 decoder
    layers and the 32000-way head, over the first 8 sequences of the seeded
    mini-batch in M = 2: the loss, dX, dMem and every parameter gradient --
    W_out, b_out and the final LayerNorm included -- against the oracle."""
    big_cfg, big = dec1024_case
    cfg = big_cfg.with_(batch=8, micro=2)
    case = dict(big, x=big["x"][:8], mem=big["mem"][:8], labels=big["labels"][:8])
    res, (gl, gh), ref = _whole_minibatch(cfg, case, 2)
    e_l = abs(res["loss"] - ref["loss"]) / abs(ref["loss"])
    e_dx, c_dx = rel_err(res["dx"], ref["dx"]), cosine(res["dx"], ref["dx"])
    e_dm, c_dm = rel_err(res["dmem"], ref["dmem"]), cosine(res["dmem"], ref["dmem"])
    print(f"dec1024 N=8 M=2: loss rel {e_l:.2e}, dx rel {e_dx:.2e} cos {c_dx:.6f}, dmem rel {e_dm:.2e} "
          f"cos {c_dm:.6f}")
    assert e_l <= 2e-2, (res["loss"], ref["loss"])
    assert c_dx >= 0.999, c_dx
    assert c_dm >= 0.999, c_dm
    worst = compare_grads(gl, gh, ref["grads"], ref["head_grads"], "cos", 0.999)
    print(f"dec1024 N=8 M=2: worst gradient cosine {worst:.6f}")
