"""gp_forward_microbatch_noalloc against gp_forward_microbatch, through the
C ABI: the same mini-batch with every forward through the no-allocation
entry point (its split-K partials in the library's static scratch array)
gives bit for bit the outputs y, the re-materialised outputs, dX and every
gradient of the regular entry point -- on two partitions in a row, the
second with a smaller input, so the second call reuses the array the first
one left behind.  A partition whose forward needs more scratch than the
array holds is rejected with GP_ERR_UNSUPPORTED and left usable."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# T = 2048 token rows: the chooser splits the K = 8192 feed-forward output GEMM in two
BIG = synth.PartitionConfig("noalloc_big", layers=1, d_model=1024, d_ff=8192, heads=16, seq=256, batch=16,
                            micro=2, dtype="bf16", loss="none")
# T = 288 ragged rows, every GEMM forced to split 2
SMALL = synth.PartitionConfig("noalloc_small", layers=2, d_model=512, d_ff=2048, heads=8, seq=96, batch=6,
                              micro=2, dtype="bf16", loss="none")


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _run(cfg, seed, noalloc):
    from paper_1811_06965_amd.runtime import Partition
    case = synth.make_case(cfg, seed, perturb=True)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        o = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0, want_recomputed=True, noalloc=noalloc)
        torch.cuda.synchronize()
        gl, gh = part.grads()
        g = np.concatenate([v.ravel() for p in gl for v in p.values()])
        return [_bits(o["y"]), _bits(o["y_remat"]), _bits(o["dx"])], g


def test_noalloc_forward_matches_the_regular_entry_point(monkeypatch):
    for cfg, seed, forced in ((BIG, 31, None), (SMALL, 32, ("18", "2"))):
        if forced:
            monkeypatch.setenv("GP_GEMM_TILE", forced[0])
            monkeypatch.setenv("GP_GEMM_SPLITS", forced[1])
        ref_t, ref_g = _run(cfg, seed, noalloc=False)
        got_t, got_g = _run(cfg, seed, noalloc=True)
        for a, b in zip(ref_t, got_t):
            assert torch.equal(a, b), cfg.name
        assert np.isfinite(got_g).all()
        assert np.array_equal(ref_g, got_g), cfg.name


def test_noalloc_forward_rejects_a_forward_beyond_the_scratch(monkeypatch):
    from paper_1811_06965_amd import gp
    from paper_1811_06965_amd.runtime import Partition
    # T = 4096 rows, the feed-forward output GEMM forced to 4 splits: 64 MiB of partials
    cfg = BIG.with_(name="noalloc_too_big", batch=32)
    monkeypatch.setenv("GP_GEMM_TILE", "18")
    monkeypatch.setenv("GP_GEMM_SPLITS", "4")
    case = synth.make_case(cfg, 33, perturb=True)
    with Partition(cfg) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        st = torch.cuda.current_stream().cuda_stream
        x0 = inp["x"].chunk(cfg.micro)[0]
        with pytest.raises(gp.GpError) as e:
            gp.gp_forward_microbatch_noalloc(part.h, 0, x0.data_ptr(), None, None, st)
        assert e.value.status == gp.GP_ERR_UNSUPPORTED
        assert "MiB" in str(e.value)
        # nothing was enqueued and the partition takes the regular entry point
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0)
        torch.cuda.synchronize()
        assert torch.isfinite(out["dx"].float()).all()
