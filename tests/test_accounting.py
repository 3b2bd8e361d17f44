"""The benchmark's FLOP counts (HFU = 4 forwards, MFU = 3) against an
independent count: torch's FLOP counter over a plain float32 forward of a
small pre-LN partition (every matrix product of the layers and the head,
attention per head), with the causal self-attention products taken at half
because the kernels skip the blocks above the diagonal.  CPU only."""
import pytest
import torch
from torch.utils.flop_counter import FlopCounterMode

import synth
from paper_1811_06965_amd import accounting


def _attention(q, k, v, heads):
    """q [T_q, D], k/v [T_k, D] of one sequence: per-head softmax(q k^T) v."""
    dh = q.shape[1] // heads
    out = []
    for h in range(heads):
        s = q[:, h * dh:(h + 1) * dh] @ k[:, h * dh:(h + 1) * dh].T.contiguous()
        out.append(torch.softmax(s, dim=-1) @ v[:, h * dh:(h + 1) * dh])
    return torch.cat(out, dim=1)


def _count(cfg):
    """(all matmul FLOPs, self-attention matmul FLOPs) of one forward."""
    g = torch.Generator().manual_seed(0)
    D, F, S, H = cfg.d_model, cfg.d_ff, cfg.seq, cfg.heads
    r = lambda *s: torch.randn(*s, generator=g)
    dec = cfg.kind == "decoder"
    total, self_attn = 0, 0
    for _ in range(cfg.batch):
        x = r(S, D)
        mem = r(cfg.mem_seq, D) if dec else None
        for _ in range(cfg.layers):
            u = torch.nn.functional.layer_norm(x, (D,))
            with FlopCounterMode(display=False) as fc:
                qkv = u @ r(D, 3 * D)
            total += fc.get_total_flops()
            with FlopCounterMode(display=False) as fc:
                c = _attention(qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], H)
            total += fc.get_total_flops()
            self_attn += fc.get_total_flops()
            with FlopCounterMode(display=False) as fc:
                x = x + c @ r(D, D)
                if dec:
                    uc = torch.nn.functional.layer_norm(x, (D,))
                    kv = mem @ r(D, 2 * D)
                    x = x + _attention(uc @ r(D, D), kv[:, :D], kv[:, D:], H) @ r(D, D)
                v = torch.nn.functional.layer_norm(x, (D,))
                x = x + torch.relu(v @ r(D, F)) @ r(F, D)
            total += fc.get_total_flops()
        if cfg.loss == "xent_ls":
            with FlopCounterMode(display=False) as fc:
                _ = torch.nn.functional.layer_norm(x, (D,)) @ r(D, cfg.vocab)
            total += fc.get_total_flops()
    return total, self_attn


ENC = synth.PartitionConfig("acct_enc", layers=2, d_model=64, d_ff=96, heads=4, seq=24, batch=3, micro=1)
DEC = synth.PartitionConfig("acct_dec", layers=2, d_model=64, d_ff=96, heads=2, seq=16, batch=2, micro=1,
                            kind="decoder", mem_seq=40, loss="xent_ls", vocab=72, label_smoothing=0.1)


@pytest.mark.parametrize("cfg", [ENC, DEC], ids=lambda c: c.name)
def test_forward_flops_match_an_independent_count(cfg):
    total, self_attn = _count(cfg)
    expected = total - (self_attn // 2 if cfg.kind == "decoder" else 0)
    assert accounting.forward_flops(cfg) == pytest.approx(expected, rel=1e-12)
    model, hw = accounting.step_flops(cfg)
    assert (model, hw) == (3 * accounting.forward_flops(cfg), 4 * accounting.forward_flops(cfg))


def test_gemm_flops_is_one_linear_product():
    with FlopCounterMode(display=False) as fc:
        torch.zeros(37, 64) @ torch.zeros(64, 48)
    assert accounting.gemm_flops(37, 64, 48) == fc.get_total_flops()
