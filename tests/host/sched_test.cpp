// Host-only checks of the partition's validation, parameter plan and
// micro-batch state machine (no HIP).  Prints "ok <name>" per check and exits
// non-zero on the first failure.
#include <cstdio>
#include <cstdlib>
#include <set>
#include <string>
#include <utility>
#include <vector>

#include "../../paper_1811_06965_amd/csrc/sched.hpp"

using namespace gp;

static int fails = 0;
#define CHECK(cond, name)                                                  \
    do {                                                                   \
        if (cond) std::printf("ok %s\n", name);                            \
        else { std::printf("FAIL %s (line %d)\n", name, __LINE__); ++fails; } \
    } while (0)

static gp_config base_cfg() {
    gp_config c{};
    c.seq_len = 256; c.seqs_per_microbatch = 8; c.num_microbatches = 8;
    c.dtype = GP_BF16; c.kind = GP_ENCODER; c.mem_seq_len = 0; c.loss = GP_LOSS_NONE;
    c.vocab = 0; c.label_smoothing = 0.f; c.ln_eps = 1e-5f; c.check_finite = 0;
    return c;
}

int main() {
    std::string msg;
    // ---- dimensions
    CHECK(check_dims(16, 1024, 8192, 16, msg) == GP_OK, "dims_ok");
    CHECK(check_dims(0, 1024, 8192, 16, msg) == GP_ERR_INVALID_ARG, "dims_zero_layers");
    CHECK(check_dims(2, 1000, 8192, 16, msg) == GP_ERR_INVALID_ARG, "dims_heads_divide");
    // ---- configuration
    Dims d{16, 1024, 8192, 16};
    gp_config c = base_cfg();
    CHECK(check_config(d, c, msg) == GP_OK, "cfg_ok");
    c.seq_len = 0; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_zero_seq"); c = base_cfg();
    c.seq_len = 96 + 8; CHECK(check_config(d, c, msg) == GP_ERR_UNSUPPORTED, "cfg_bf16_seq_not_32"); c = base_cfg();
    c.seq_len = 288; CHECK(check_config(d, c, msg) == GP_ERR_UNSUPPORTED, "cfg_bf16_seq_over_256"); c = base_cfg();
    c.mem_seq_len = 64; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_encoder_memory"); c = base_cfg();
    c.kind = GP_DECODER_CROSS; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_decoder_no_memory");
    c.mem_seq_len = 128; CHECK(check_config(d, c, msg) == GP_OK, "cfg_decoder_ok"); c = base_cfg();
    c.loss = GP_LOSS_XENT_LS; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_xent_needs_vocab");
    c.vocab = 32000; CHECK(check_config(d, c, msg) == GP_OK, "cfg_xent_ok");
    c.vocab = 32001; CHECK(check_config(d, c, msg) == GP_ERR_UNSUPPORTED, "cfg_vocab_multiple_of_8"); c = base_cfg();
    c.vocab = 8; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_vocab_without_head"); c = base_cfg();
    c.label_smoothing = 1.f; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_ls_range"); c = base_cfg();
    c.ln_eps = 0.f; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_eps_positive"); c = base_cfg();
    c.dtype = 7; CHECK(check_config(d, c, msg) == GP_ERR_INVALID_ARG, "cfg_dtype"); c = base_cfg();
    Dims d2{2, 1024, 8192, 8};  // head dim 128
    CHECK(check_config(d2, c, msg) == GP_ERR_UNSUPPORTED, "cfg_bf16_head_dim");
    c.dtype = GP_F32; CHECK(check_config(d2, c, msg) == GP_ERR_UNSUPPORTED, "cfg_f32_head_dim");
    Dims d3{2, 96, 160, 3};
    c.seq_len = 40; CHECK(check_config(d3, c, msg) == GP_OK, "cfg_f32_ragged_ok");
    c.seq_len = 2048; CHECK(check_config(d3, c, msg) == GP_ERR_UNSUPPORTED, "cfg_f32_seq_limit"); c = base_cfg();

    // ---- parameter plan: Table 1 count and non-overlapping 256-byte-aligned blocks
    Geometry g; g.S = 256; g.n = 8; g.M = 8;
    ParamPlan p = plan_params(d, g);
    const size_t per_layer = 4 * 1024 * 1024 + 4 * 1024 + 2 * 1024 * 8192 + 8192 + 1024 + 4 * 1024;
    CHECK(p.count == 16 * per_layer, "plan_count_encoder");
    std::set<std::pair<size_t, size_t>> spans;
    bool aligned = true, disjoint = true;
    for (const Linear* x : p.linears()) {
        aligned = aligned && x->w % 64 == 0 && x->kn % 128 == 0;
        spans.insert({x->w, x->b + x->out});
    }
    size_t end = 0;
    for (auto& s : spans) { disjoint = disjoint && s.first >= end; end = s.second; }
    CHECK(aligned, "plan_aligned");
    CHECK(disjoint, "plan_disjoint");
    // roles: forward role of each linear; +1 dX, +2 dW stay inside the role range
    bool roles = true;
    for (const Linear* x : p.linears()) roles = roles && x->role > GP_K_NONE && x->role + 2 < GP_K_ATTN_FWD;
    CHECK(roles, "plan_roles");
    // decoder + head adds cross-attention and the vocabulary projection
    Geometry gd = g; gd.kind = GP_DECODER_CROSS; gd.Smem = 128; gd.loss = GP_LOSS_XENT_LS; gd.V = 32000;
    ParamPlan pd = plan_params(d, gd);
    const size_t cross = 4 * 1024 * 1024 + 4 * 1024 + 2 * 1024;
    CHECK(pd.count == 16 * (per_layer + cross) + 2 * 1024 + 1024 * 32000 + 32000, "plan_count_decoder_head");

    // ---- the bf16 update's range table: weights in tiles, every other parameter in a range
    std::vector<long> ranges;
    CHECK(plan_update_ranges(p, ranges) && ranges.size() == 2 * (4 * 16 + 2 * 16), "update_ranges_encoder");
    bool biases = true;
    for (size_t i = 0; i < ranges.size(); i += 2) biases = biases && ranges[i] % 64 == 0 && ranges[i + 1] > 0;
    CHECK(biases && ranges[0] == (long)p.layers[0].qkv.b && ranges[1] == 3 * 1024, "update_ranges_first_bias");
    CHECK(plan_update_ranges(pd, ranges) && ranges.size() == 2 * (7 * 16 + 3 * 16 + 2), "update_ranges_decoder_head");
    Geometry gv = gd; gv.V = 1000;  // a head that is not a whole number of 64-wide tiles
    CHECK(!plan_update_ranges(plan_params(d, gv), ranges) && ranges.empty(), "update_ranges_ragged_head");
    CHECK(!plan_update_ranges(plan_params(d3, g), ranges) && ranges.empty(), "update_ranges_ragged_widths");

    // ---- parameter resolution: q/k/v are column slices of the packed projection
    ParamRef r;
    CHECK(resolve_param(p, d, 3, GP_P_WK, r, msg) == GP_OK && r.off == p.layers[3].qkv.w + 1024 &&
              r.rows == 1024 && r.cols == 1024 && r.ld == 3072 && r.lin == &p.layers[3].qkv, "resolve_wk");
    CHECK(resolve_param(p, d, 0, GP_P_BV, r, msg) == GP_OK && r.off == p.layers[0].qkv.b + 2048 && r.rows == 1,
          "resolve_bv");
    CHECK(resolve_param(p, d, 0, GP_P_XWQ, r, msg) == GP_ERR_INVALID_ARG, "resolve_absent_cross");
    CHECK(resolve_param(p, d, 16, GP_P_WQ, r, msg) == GP_ERR_INVALID_ARG, "resolve_layer_range");
    CHECK(resolve_param(p, d, -1, GP_P_WOUT, r, msg) == GP_ERR_INVALID_ARG, "resolve_absent_head");
    CHECK(resolve_param(pd, d, -1, GP_P_WOUT, r, msg) == GP_OK && r.cols == 32000, "resolve_head");

    // ---- state machine: forwards 0..M-1, backwards M-1..0, one step
    Sched s;
    CHECK(s.can_forward(0, msg) == GP_ERR_STATE, "sched_unconfigured");
    CHECK(s.configure(3, msg) == GP_OK, "sched_configure");
    CHECK(s.configure(3, msg) == GP_ERR_STATE, "sched_configure_twice");
    CHECK(s.can_backward(2, msg) == GP_ERR_STATE, "sched_backward_before_forward");
    CHECK(s.can_forward(1, msg) == GP_ERR_STATE, "sched_forward_out_of_order");
    CHECK(s.can_forward(3, msg) == GP_ERR_INVALID_ARG, "sched_forward_range");
    bool fwd_ok = true;
    for (int m = 0; m < 3; ++m) { fwd_ok = fwd_ok && s.can_forward(m, msg) == GP_OK; s.did_forward(); }
    CHECK(fwd_ok, "sched_forward_in_order");
    CHECK(s.can_forward(0, msg) == GP_ERR_STATE, "sched_no_forward_after_all");
    CHECK(s.can_set_param(msg) == GP_ERR_STATE, "sched_no_param_change_mid_batch");
    CHECK(s.can_step(msg) == GP_ERR_STATE, "sched_step_needs_backward");
    CHECK(s.can_backward(0, msg) == GP_ERR_STATE, "sched_backward_reverse_order");
    CHECK(s.first_backward(), "sched_first_backward");
    bool bwd_ok = true;
    for (int m = 2; m >= 0; --m) { bwd_ok = bwd_ok && s.can_backward(m, msg) == GP_OK; s.did_backward(); }
    CHECK(bwd_ok, "sched_backward_in_reverse");
    CHECK(s.can_step(msg) == GP_OK, "sched_step_ready");
    s.did_step();
    CHECK(s.can_set_param(msg) == GP_OK && s.can_forward(0, msg) == GP_OK, "sched_next_minibatch");
    std::printf("%d failures\n", fails);
    return fails ? 1 : 0;
}
