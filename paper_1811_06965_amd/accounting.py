"""Algorithmic work of one partition step (FLOPs and bytes), for reporting.

FLOPs count matrix products only (the GEMMs, Q K^T and P V).  Per token and
layer the encoder forward is 8 D^2 + 4 D F + 4 S D (QKV and output
projections, FFN, two attention products); the decoder adds the cross block
(4 D^2 for the query and output projections, 4 D^2 S_mem / S for the memory
keys/values, 4 S_mem D for its attention) and counts the causal self-attention
at half (2 S D).  The vocabulary head adds 2 D V per token.
Model FLOPs = 3 x forward (forward + backward); hardware FLOPs = 4 x forward,
because re-materialisation runs every forward twice (GPipe, Section 2.3).  Both
count bf16 matrix work only: the fp4 correction term of the bf16 feed-forward
input projection (2 D F per token and layer, in the forward and the recompute,
at four times the bf16 rate) is not included.
"""


def forward_flops_per_token_layer(cfg) -> float:
    D, F, S = cfg.d_model, cfg.d_ff, cfg.seq
    if cfg.kind == "decoder":
        Sm = cfg.mem_seq
        return 8 * D * D + 4 * D * F + 2 * S * D + 4 * D * D + 4 * D * D * Sm / S + 4 * Sm * D
    return 8 * D * D + 4 * D * F + 4 * S * D


def forward_flops(cfg, batch=None) -> float:
    N = cfg.batch if batch is None else batch
    tokens = N * cfg.seq
    f = tokens * cfg.layers * forward_flops_per_token_layer(cfg)
    if cfg.loss == "xent_ls":
        f += tokens * 2 * cfg.d_model * cfg.vocab
    return float(f)


def step_flops(cfg, batch=None):
    """(model FLOPs, hardware FLOPs) of one mini-batch step."""
    f = forward_flops(cfg, batch)
    return 3 * f, 4 * f


# Linear layers of an encoder layer: name -> (in, out)
def encoder_linears(cfg):
    D, F = cfg.d_model, cfg.d_ff
    return {"qkv": (D, 3 * D), "o": (D, D), "ffn1": (D, F), "ffn2": (F, D)}


def gemm_flops(rows, lin_in, lin_out) -> float:
    """One linear layer's forward (or dX, or dW) GEMM over `rows` token rows."""
    return 2.0 * rows * lin_in * lin_out
