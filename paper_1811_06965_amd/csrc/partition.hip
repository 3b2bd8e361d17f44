// partition.hip -- the C ABI of one GPipe partition and its layer drivers.
//
// GPipe, Sections 2.2-2.3: the mini-batch is split into M equal
// micro-batches; the forward pass of each keeps only the partition's boundary
// input (the stash); the backward pass recomputes the partition's forward from
// the stash (re-materialisation) keeping that one micro-batch's intermediates,
// then back-propagates layer by layer, adding each parameter gradient into an
// fp32 accumulator; one synchronous update ends the mini-batch.
//
// Device memory (one partition):
//   master, grads   fp32, identical layout: per linear W [in, out] then b [out];
//                   per LayerNorm gamma [D] then beta [D]
//   welt            working copies in the partition dtype: W [in, out] and W^T [out, in]
//   stash           M boundary inputs [n, S, D] (and decoder memories [n, S_mem, D])
//   workspace       per set: residual stream xs[0..L] fp32 [T, D] (T = n S) and
//                   per-layer intermediates of one micro-batch; backward scratch
// The first forward pass writes its intermediates into a layer slot of its
// own (one of two, by micro-batch parity, so that forwards issued on two
// streams run side by side) and ping-pongs that slot's two residual buffers;
// the re-materialising pass of micro-batch m uses its set (set_of: sets rotate
// so that the one being rebuilt ahead is never one still read), slot l and
// xs[l] for layer l.  Sets come in groups of two or four micro-batches whose
// buffers hold them back to back, so that the weight gradients of a group run
// as one GEMM and a pair can be recomputed in one pass.  All passes run the
// same kernels with the same tile splits, so the recomputed activations equal
// the first pass bit for bit.
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <utility>
#include <vector>

#include "common.hpp"
#include "kernels.hpp"
#include "sched.hpp"

namespace gp {

static thread_local std::string g_err;
static thread_local LaunchEvents g_launch_events;

LaunchEvents& launch_events() { return g_launch_events; }
static thread_local hipError_t g_launch_status = hipSuccess;
hipError_t& launch_status() { return g_launch_status; }

gp_status set_error(gp_status s, const char* msg) {
    g_err = msg;
    return s;
}
gp_status hip_fail(hipError_t e, const char* file, int line) {
    g_err = std::string("HIP error: ") + hipGetErrorString(e) + " at " + file + ":" + std::to_string(line);
    return GP_ERR_HIP;
}

struct Arena {
    char* base = nullptr;
    size_t off = 0;
    size_t mark() {  // aligned offset of the next buffer
        off = align_up(off, 256);
        return off;
    }
    template <typename X> X* take(size_t count) {
        off = align_up(off, 256);
        X* p = reinterpret_cast<X*>(base + off);
        off += count * sizeof(X);
        return p;
    }
    void* take_elt(size_t count, size_t esz) {
        off = align_up(off, 256);
        void* p = base + off;
        off += count * esz;
        return p;
    }
};

struct LayerWs {
    float *st1 = nullptr, *lse = nullptr, *x1 = nullptr;
    void *u = nullptr, *qkv = nullptr, *c = nullptr;
    float *stc = nullptr, *xlse = nullptr, *x2 = nullptr;
    void *uc = nullptr, *xq = nullptr, *xkv = nullptr, *xc = nullptr;
    float* stf = nullptr;
    void *v = nullptr, *a = nullptr;
    unsigned char *v4 = nullptr, *v4s = nullptr;  // fp4 rounding residuals of v and their row scales (bf16)
};

constexpr int ELT_RING = 10;      // bf16 residual-gradient buffers (see layer_backward)

// A byte range of the workspace, as an offset from its base.
struct Span {
    size_t off = 0, bytes = 0;
};

struct BwdWs {
    float *p32 = nullptr, *q32 = nullptr, *dn = nullptr, *delta = nullptr, *dmem32 = nullptr;
    void* ring[ELT_RING] = {};  // dL/dx in the partition dtype, rotating across layers
    void *dc = nullptr;
    void *dz[2] = {}, *dqkv[2] = {}, *dxq[2] = {}, *dxkv[2] = {};  // by layer parity
    double *loss_partial = nullptr, *loss_acc = nullptr;
    int* flag = nullptr;
    int* bad_label = nullptr;  // set by the cross-entropy head on a label outside [0, V)
    float* splitk = nullptr;   // split-K partial tiles (the call's stream)
    float* splitk_side = nullptr;  // split-K partial tiles of the weight-gradient stream
    float* splitk_remat = nullptr; // split-K partial tiles of the recompute-ahead stream
    // the feed-forward input in fp16 (Linear::f16): read only by the GEMM right
    // after the LayerNorm that writes it, so one buffer per stream that runs
    // forward passes (rows of a recompute unit), not one per layer and set
    void *v16_main = nullptr, *v16_remat = nullptr;
    long splitk_elems = 0;
    // loss head
    float* sth = nullptr;
    void *h = nullptr, *z = nullptr;
};

// Grouped weight gradients: the weight-gradient GEMMs of micro-batches
// Gi .. Gi + G - 1 (G = 2 or 4) run as one GEMM with a reduction over the
// group's token rows (one fp32 read-modify-write of the accumulator, one
// launch, per group).  Their operands must then stay until the last backward
// call of the group (its lowest micro-batch) and sit back to back: per layer,
// the bf16 gradients a layer's weight-gradient GEMMs take as dY live here, G
// micro-batches' rows each (member h = micro-batch Gi + h), instead of in the
// recycled ring and parity buffers; the activations come from workspace sets
// allocated in groups.
struct DyStore {
    void* gin = nullptr;    // dL/dx_out of the layer (dY of the ffn2 weight gradient)
    void* gffn = nullptr;   // after the feed-forward block's LayerNorm backward (dY of o / xo)
    void* gcross = nullptr; // decoder: after the cross-attention block's LayerNorm backward (dY of o)
    void* dz = nullptr;     // dY of the ffn1 weight gradient
    void* dqkv = nullptr;   // dY of the qkv weight gradient
    void* dxq = nullptr;    // decoder: dY of the cross-attention query weight gradient
    void* dxkv = nullptr;   // decoder: dY of the cross-attention key/value weight gradient (memory rows)
};

// The working memory of a first forward pass (re-materialisation off: one
// layer slot and two ping-pong residual buffers, nothing kept).  There are two,
// taken by micro-batch parity, so that consecutive forwards issued on two
// streams run side by side.  The even one uses the split-K partials and the
// fp16 buffer of the caller's stream (those of the backward, which starts after
// every forward); the odd one has its own.
struct FirstPass {
    LayerWs w;
    float* xs[2] = {};
    std::vector<Span> span;  // the layer slot and the residual buffers
    float* splitk = nullptr; // odd slot: split-K partials (the most one forward writes)
    void* v16 = nullptr;     // odd slot: the feed-forward input in fp16 (Linear::f16)
    Span splitk_span;
    // The last forward in this slot: its stream, events recorded on it after
    // the boundary input was stashed and at its end (from the event ring), and
    // the capture its recordings belong to (0: none).
    hipStream_t stream = nullptr;
    hipEvent_t stashed = nullptr, done = nullptr;
    unsigned long long capture = 0;
};

} // namespace gp

using namespace gp;

// Event pairs around the launches of the selected role(s), with the roles'
// algorithmic FLOPs and bytes.
struct LaunchTimer {
    int selected = GP_K_NONE;
    bool markers = false;  // GP_TIMER_MARKERS=1: also launch role_marker around each timed launch
    int every = 1;         // time one launch in `every` of a selected role
    long seen[GP_K_COUNT] = {};  // launches of each selected role since the last reset
    std::vector<std::pair<hipEvent_t, hipEvent_t>> recs[GP_K_COUNT];
    double flops[GP_K_COUNT] = {}, bytes[GP_K_COUNT] = {};
    std::vector<hipEvent_t> pool;  // created events not in use
    std::vector<hipEvent_t> all;   // every created event (destroyed with the partition)

    bool on(int role) const {
        return role > GP_K_NONE && role < GP_K_COUNT && (selected == GP_K_COUNT || selected == role);
    }
    gp_status take(hipEvent_t& e) {
        if (pool.empty()) {
            GP_HIP(hipEventCreate(&e));
            all.push_back(e);
        } else {
            e = pool.back();
            pool.pop_back();
        }
        return GP_OK;
    }
    void reset() {
        for (int r = 0; r < GP_K_COUNT; ++r) {
            for (auto& pr : recs[r]) {
                pool.push_back(pr.first);
                pool.push_back(pr.second);
            }
            recs[r].clear();
            flops[r] = bytes[r] = 0.0;
            seen[r] = 0;
        }
    }
};

struct gp_partition {
    Dims d;
    Geometry g;
    Sched sched;
    ParamPlan plan;
    size_t esz = 4;
    float* master = nullptr;
    float* grads = nullptr;
    char* welt = nullptr;
    char* stash_x = nullptr;
    char* stash_m = nullptr;
    char* ws = nullptr;
    // workspace sets: set s holds a residual stream xs[s][0..L] and layer slots lw[s][0..L-1]
    std::vector<std::vector<float*>> xs;
    std::vector<std::vector<LayerWs>> lw;
    int nsets = 1;
    // grouped weight gradients (GP_PAIR_DW=0 turns them off): workspace sets
    // are allocated in groups of `group` micro-batches (2 or 4) whose buffers
    // hold the group's micro-batches back to back
    bool pair_dw = true;
    int group = 1;
    std::vector<DyStore> dys;  // per layer (grouping only)
    // micro-batches re-materialised together in one pass over their rows
    // (1, or 2 within a group of sets)
    int remat_group = 1;
    // the first passes' own working memory (no set's), by micro-batch parity
    // (one when M = 1 or GP_FWD_LANES=1)
    FirstPass fpass[2];
    int fp_lanes = 1;
    int lane_of(int m) const { return fp_lanes > 1 ? m & 1 : 0; }
    // Backward lanes: the two members of a recompute pair are
    // back-propagated side by side when the caller issues them on two streams.
    // The odd member (whose call comes first) uses `bw1` and its own split-K
    // partials; it records hi_ev[l] after each layer l, and the even member
    // waits for it before its first LayerNorm backward of layer l (so the
    // LayerNorm partial sums accumulate in micro-batch order, as with one
    // lane) and before launching the pair's weight gradients of layer l.
    // A pair starts after the previous pair's even member (its weight
    // gradients and recompute-ahead fork included); each call waits for the
    // previous call in its lane.  GP_BWD_LANES=1 turns this off.
    int bwd_lanes = 1;
    int blane(int m) const { return bwd_lanes > 1 ? m & 1 : 0; }
    std::vector<hipEvent_t> hi_ev;
    hipEvent_t lane_end[2] = {};
    hipStream_t lane_stream[2] = {};
    unsigned long long lane_capture[2] = {};
    hipEvent_t unit_ready = nullptr;  // the pair's recompute available (on its first call's stream)
    hipStream_t unit_ready_stream = nullptr;
    unsigned long long unit_ready_capture = 0;
    Span bwd1_span, splitk1_span, loss1_span, head1_span;
    // the odd member's loss head done (its loss sum and head gradient come
    // first; the even member's head waits for it)
    hipEvent_t head_ev = nullptr;
    // Per-layer update: the mini-batch's last backward call records, per layer
    // l, an event on its stream after layer l (every read of layer l's weights
    // by the backward is behind it) and the weight-gradient stream's event
    // after layer l's last weight-gradient GEMM; the update then refreshes
    // layer l on the recompute stream (idle by then) as soon as both have
    // passed, beside the backward of the layers below.
    std::vector<hipEvent_t> lay_main, lay_side;
    bool lay_ready = false;
    bool layer_update = true;  // GP_LAYER_UPDATE=0: the whole update after the last backward
    // the last update's stream and an event recorded at its end, with its
    // capture: a forward issued on another stream waits for it
    hipStream_t tail_stream = nullptr;
    hipEvent_t tail_done = nullptr;
    unsigned long long tail_capture = 0;
    bool dw_started = false;   // a weight-gradient GEMM of this mini-batch was launched
    float* opt_ms = nullptr;  // RMSProp: running mean square of every gradient [n32]
    // bf16 partitions whose linears are whole 64 x 64 tiles update each
    // linear's weights fused with the refresh of its working copies, and the
    // rest (biases, LayerNorm parameters) from a table of float ranges
    bool fused_update = false;
    long* upd_ranges = nullptr;  // device: (offset, count) pairs
    int n_upd_ranges = 0;
    // GP_POISON=1 (test mode): every workspace region is filled with NaN
    // right before the phase that (re)writes it, so that a read of a stale or
    // never-written value shows up in the results.  Regions, per set: the
    // residual stream, each layer slot; and the backward scratch, the LayerNorm
    // partial sums, the split-K partials of each stream, the loss partials.
    bool poison = false;
    std::vector<std::vector<Span>> slot_span; // per set: its residual stream and every buffer of its layer slots
    std::vector<std::vector<Span>> dys_span;  // per member: its rows of every grouped-gradient buffer
    Span bwd_span, lnpart_span, loss_span, loss_acc_span, head_span;
    Span splitk_span[3];                      // caller's stream, weight-gradient stream, recompute stream
    // gp_forward_microbatch_noalloc: this device's address of the static
    // scratch array (nullptr if it could not be resolved) and the most
    // split-K partial floats one first forward pass writes
    float* noalloc_scratch = nullptr;
    std::string noalloc_error;
    long fwd_ws_need = 0;
    // per LayerNorm: block partial sums of its gamma/beta gradients, added up
    // over the micro-batches of a mini-batch and reduced after the last one
    std::vector<float*> lnpart;
    BwdWs bw;
    BwdWs bw1;  // the odd backward lane's scratch (p32, q32, dn, dc, delta, dmem32, splitk, v16)
    size_t bytes_params = 0, bytes_grads = 0, bytes_stash = 0, bytes_ws = 0;
    // GEMM tile-shape override (GP_GEMM_TILE = 0..10, GP_GEMM_SPLITS), read at
    // configure; -1 lets the library choose per problem.
    int gemm_tile = -1, gemm_splits = 0;
    LaunchTimer timer;
    // Weight-gradient GEMMs run on a second stream (GP_SIDE_STREAM=0 turns it
    // off), ordered against the caller's stream by events from a ring.
    // Fork/join events come from a ring of distinct event objects: a stream
    // wait must refer to the recording made just before it, and a recorded
    // event is not recorded again until the ring has gone round (the host can
    // run many calls ahead of the device).
    std::vector<hipEvent_t> evring;
    size_t ev_next = 0;
    bool events() const { return !evring.empty(); }
    hipEvent_t next_event() {
        hipEvent_t e = evring[ev_next];
        ev_next = (ev_next + 1) % evring.size();
        return e;
    }
    bool use_side = true;
    // when weight-gradient GEMMs are handed to the side stream (GP_DW_FLUSH):
    // 0 each as soon as its inputs are enqueued, 1 after the feed-forward
    // block and at the end of the layer, 2 at the end of the layer
    int dw_flush = 0;
    hipStream_t side = nullptr;
    hipEvent_t side_done[4] = {};  // side stream's last event of layer l % 4 (from evring)
    // Recompute-ahead (GP_REMAT_AHEAD=0 turns it off): while micro-batch m is
    // back-propagated, micro-batch m - 1 is re-materialised on a third stream
    // into the other workspace set.
    bool remat_ahead = true;
    // Early recompute of the last micro-batch (GP_REMAT_EARLY=0 turns it off):
    // its backward comes first, so its re-materialising forward is started on
    // the recompute stream by the last forward call itself, right after the
    // boundary input is stashed, and runs beside that forward.
    bool remat_early = true;
    // split-K reduce of a residual GEMM fused into the next LayerNorm (GP_FUSE_RES_LN)
    bool fuse_res_ln = true;
    // two-wave attention kernels where they apply (GP_ATTN_KSPLIT)
    bool attn_split = true;
    // attention waves per workgroup (GP_ATTN_WAVES = 1, 2 or 4; 0: by grid size)
    int attn_waves = 0;
    hipStream_t remat = nullptr;
    hipEvent_t remat_done = nullptr;  // from evring
    int remat_pending = -1;  // micro-batch whose recompute-ahead is enqueued

    // Workspace set of micro-batch m: its own set when activations are kept;
    // else the sets rotate group by group -- micro-batch m takes member m % group
    // of group (m / group) mod (nsets / group) -- so that with recompute-ahead
    // the set being rebuilt is never one the backward or a pending grouped
    // weight gradient still reads.
    int set_of(int m) const {
        if (g.keep_act) return m;
        return group * ((m / group) % (nsets / group)) + m % group;
    }
    // grouped weight gradients: micro-batches in m's group, and whether m's
    // backward launches them (the lowest member; the others run first and defer)
    int group_size(int m) const { return std::min(group, g.M - (m - m % group)); }
    bool launches_dw(int m) const { return m % group == 0; }
    bool ahead_on = false;  // recompute-ahead / early-recompute stream in use
    bool ahead() const { return ahead_on; }
    void* W(size_t elt_off) const { return welt + elt_off * esz; }
    char* stash_x_mb(int m) const { return stash_x + (size_t)m * g.T() * d.D * esz; }
    char* stash_m_mb(int m) const { return stash_m + (size_t)m * g.Tm() * d.D * esz; }
    void* off_elt(void* p, long elems) const { return static_cast<char*>(p) + elems * (long)esz; }
    const void* off_elt(const void* p, long elems) const { return static_cast<const char*>(p) + elems * (long)esz; }
};

namespace {

// Carve the workspace; with a.base == nullptr only measures it.
long forward_workspace_need(const gp_partition* p);

void plan_workspace(gp_partition* p, Arena& a) {
    const Dims& d = p->d;
    const Geometry& g = p->g;
    const long T = g.T(), Tm = g.Tm(), D = d.D, F = d.F;
    const long lse_n = (long)g.n * d.H * g.S;
    const size_t e = p->esz;
    const bool dec = g.kind == GP_DECODER_CROSS;
    const bool f16 = !p->plan.layers.empty() && p->plan.layers[0].ffn1.f16;
    p->xs.assign(p->nsets, std::vector<float*>(d.L + 1, nullptr));
    p->lw.assign(p->nsets, std::vector<LayerWs>(d.L, LayerWs{}));
    p->slot_span.assign(p->nsets, std::vector<Span>{});
    auto span_from = [&](size_t start) { return Span{start, a.off - start}; };
    // Residual streams and layer slots, one group of sets at a time: each
    // buffer holds the rows of the group's members back to back (member h at
    // row h * rows), so that a pass can cover the whole group.
    const int G = p->group;
    for (int g0 = 0; g0 < p->nsets; g0 += G) {
        for (int li = 0; li <= d.L; ++li) {
            const size_t off = a.mark();
            float* base = a.take<float>((size_t)T * D * G);
            for (int h = 0; h < G; ++h) {
                p->xs[g0 + h][li] = base + (size_t)h * T * D;
                p->slot_span[g0 + h].push_back(Span{off + (size_t)h * T * D * 4, (size_t)T * D * 4});
            }
        }
    }
    // the first passes' slots: one layer of one micro-batch, and two residuals
    for (int ln = 0; ln < 2; ++ln) {
        FirstPass& f = p->fpass[ln];
        f.w = LayerWs{};
        f.xs[0] = f.xs[1] = nullptr;
        f.span.clear();
        if (ln >= p->fp_lanes) continue;
        auto take1 = [&](auto LayerWs::*field, long count, size_t esz) {
            const size_t off = a.mark();
            f.w.*field = reinterpret_cast<typename std::remove_reference<decltype(f.w.*field)>::type>(
                a.take_elt((size_t)count, esz));
            f.span.push_back(Span{off, (size_t)count * esz});
        };
        take1(&LayerWs::st1, 2 * T, 4);
        take1(&LayerWs::u, T * D, e);
        take1(&LayerWs::qkv, T * 3 * D, e);
        take1(&LayerWs::c, T * D, e);
        take1(&LayerWs::lse, lse_n, 4);
        take1(&LayerWs::x1, T * D, 4);
        if (dec) {
            take1(&LayerWs::stc, 2 * T, 4);
            take1(&LayerWs::uc, T * D, e);
            take1(&LayerWs::xq, T * D, e);
            take1(&LayerWs::xkv, Tm * 2 * D, e);
            take1(&LayerWs::xc, T * D, e);
            take1(&LayerWs::xlse, lse_n, 4);
            take1(&LayerWs::x2, T * D, 4);
        }
        take1(&LayerWs::stf, 2 * T, 4);
        take1(&LayerWs::v, T * D, e);
        if (!f16 && p->g.dtype == GP_BF16) {
            take1(&LayerWs::v4, T * D / 2, 1);
            take1(&LayerWs::v4s, T, 1);
        }
        take1(&LayerWs::a, T * F, e);
        for (float*& x : f.xs) {
            const size_t off = a.mark();
            x = a.take<float>((size_t)T * D);
            f.span.push_back(Span{off, (size_t)T * D * 4});
        }
    }
    for (int g0 = 0; g0 < p->nsets; g0 += G) {
        for (int li = 0; li < d.L; ++li) {
            // one buffer of `count` elements of `esz` bytes per member
            auto take = [&](auto LayerWs::*field, long count, size_t esz) {
                const size_t off = a.mark();
                char* base = static_cast<char*>(a.take_elt((size_t)count * G, esz));
                for (int h = 0; h < G; ++h) {
                    p->lw[g0 + h][li].*field = reinterpret_cast<typename std::remove_reference<
                        decltype(p->lw[0][0].*field)>::type>(base + (size_t)h * count * esz);
                    p->slot_span[g0 + h].push_back(Span{off + (size_t)h * count * esz, (size_t)count * esz});
                }
            };
            take(&LayerWs::st1, 2 * T, 4);
            take(&LayerWs::u, T * D, e);
            take(&LayerWs::qkv, T * 3 * D, e);
            take(&LayerWs::c, T * D, e);
            take(&LayerWs::lse, lse_n, 4);
            take(&LayerWs::x1, T * D, 4);
            if (dec) {
                take(&LayerWs::stc, 2 * T, 4);
                take(&LayerWs::uc, T * D, e);
                take(&LayerWs::xq, T * D, e);
                take(&LayerWs::xkv, Tm * 2 * D, e);
                take(&LayerWs::xc, T * D, e);
                take(&LayerWs::xlse, lse_n, 4);
                take(&LayerWs::x2, T * D, 4);
            }
            take(&LayerWs::stf, 2 * T, 4);
            take(&LayerWs::v, T * D, e);
            if (!f16 && p->g.dtype == GP_BF16) {  // see Linear::split
                take(&LayerWs::v4, T * D / 2, 1);
                take(&LayerWs::v4s, T, 1);
            }
            take(&LayerWs::a, T * F, e);
        }
    }
    // grouped weight-gradient operands: per layer, the group's micro-batches' rows
    p->dys.assign(G > 1 ? d.L : 0, DyStore{});
    p->dys_span.assign(G > 1 ? G : 0, std::vector<Span>{});
    for (auto& y : p->dys) {
        auto take = [&](void*& field, long count) {
            const size_t off = a.mark();
            field = a.take_elt((size_t)count * G, e);
            for (int h = 0; h < G; ++h) p->dys_span[h].push_back(Span{off + (size_t)h * count * e, (size_t)count * e});
        };
        take(y.gin, T * D);
        take(y.gffn, T * D);
        take(y.dz, T * F);
        take(y.dqkv, T * 3 * D);
        if (dec) {
            take(y.gcross, T * D);
            take(y.dxq, T * D);
            take(y.dxkv, Tm * 2 * D);
        }
    }
    BwdWs& b = p->bw;
    const size_t b0 = a.mark();
    b.p32 = a.take<float>(T * D);
    b.q32 = a.take<float>(T * D);
    b.dn = a.take<float>(T * D);
    b.dc = a.take_elt(T * D, e);
    if (G == 1) {
        for (auto& r : b.ring) r = a.take_elt(T * D, e);
        for (int i = 0; i < 2; ++i) {
            b.dz[i] = a.take_elt(T * F, e);
            b.dqkv[i] = a.take_elt(T * 3 * D, e);
            if (dec) {
                b.dxq[i] = a.take_elt(T * D, e);
                b.dxkv[i] = a.take_elt(Tm * 2 * D, e);
            }
        }
    }
    b.delta = a.take<float>(lse_n);
    if (dec) b.dmem32 = a.take<float>(Tm * D);
    p->bwd_span = span_from(b0);
    const std::vector<const Norm*> norms = p->plan.norms();
    p->lnpart.assign(norms.size(), nullptr);
    const size_t n0 = a.mark();
    for (const Norm* n : norms) p->lnpart[n->id] = a.take<float>((size_t)layernorm_bwd_blocks(T) * 2 * n->n);
    p->lnpart_span = span_from(n0);
    // split-K partials: up to 8 splits of a T x D activation GEMM or of the
    // D x 3D packed-QKV weight gradient (with its bias column sums)
    b.splitk_elems = std::max<long>(8 * T * D, 8 * (3 * D * D + 3 * D));
    const size_t sk_bytes = (size_t)b.splitk_elems * sizeof(float);
    // a grouped recompute runs the single micro-batch's splits over its
    // members' rows; it can run on the caller's stream too (no early recompute)
    const size_t main_elems = (size_t)b.splitk_elems * p->remat_group;
    p->splitk_span[0] = Span{a.mark(), main_elems * sizeof(float)};
    b.splitk = a.take<float>(main_elems);
    p->splitk_span[1] = Span{a.mark(), sk_bytes};
    b.splitk_side = a.take<float>((size_t)b.splitk_elems);
    p->splitk_span[2] = Span{};
    if (p->ahead()) {
        const size_t rm = main_elems;
        p->splitk_span[2] = Span{a.mark(), rm * sizeof(float)};
        b.splitk_remat = a.take<float>(rm);
    }
    if (f16) {
        const size_t n16 = (size_t)p->remat_group * T * D;
        b.v16_main = a.take_elt(n16, 2);
        if (p->ahead()) b.v16_remat = a.take_elt(n16, 2);
    }
    // the odd backward lane's scratch
    p->bw1 = BwdWs{};
    p->bwd1_span = p->splitk1_span = Span{};
    if (p->bwd_lanes > 1) {
        BwdWs& q = p->bw1;
        const size_t q0 = a.mark();
        q.p32 = a.take<float>(T * D);
        q.q32 = a.take<float>(T * D);
        q.dn = a.take<float>(T * D);
        q.dc = a.take_elt(T * D, e);
        q.delta = a.take<float>(lse_n);
        if (dec) q.dmem32 = a.take<float>(Tm * D);
        p->bwd1_span = span_from(q0);
        q.splitk_elems = b.splitk_elems;
        p->splitk1_span = Span{a.mark(), main_elems * sizeof(float)};
        q.splitk = a.take<float>(main_elems);
        if (f16) q.v16_main = a.take_elt((size_t)p->remat_group * T * D, 2);
    }
    // the odd first-pass slot's own partials and fp16 buffer (one micro-batch)
    for (int ln = 1; ln < 2; ++ln) {
        FirstPass& f = p->fpass[ln];
        f.splitk = nullptr;
        f.v16 = nullptr;
        f.splitk_span = Span{};
        if (ln >= p->fp_lanes) continue;
        const size_t need = (size_t)std::max<long>(1, forward_workspace_need(p));
        f.splitk_span = Span{a.mark(), need * sizeof(float)};
        f.splitk = a.take<float>(need);
        if (f16) f.v16 = a.take_elt((size_t)T * D, 2);
    }
    size_t lp = (size_t)loss_blocks();
    if (g.loss == GP_LOSS_XENT_LS && (size_t)xent_partials(T) > lp) lp = xent_partials(T);
    p->loss_span = Span{a.mark(), lp * sizeof(double)};
    b.loss_partial = a.take<double>(lp);
    p->loss_acc_span = Span{a.mark(), sizeof(double)};
    b.loss_acc = a.take<double>(1);
    b.flag = a.take<int>(1);
    b.bad_label = a.take<int>(1);
    p->head_span = Span{};
    if (g.loss == GP_LOSS_XENT_LS) {
        const size_t h0 = a.mark();
        b.sth = a.take<float>(2 * T);
        b.h = a.take_elt(T * D, e);
        b.z = a.take_elt(T * (long)g.V, e);
        p->head_span = span_from(h0);
    }
    // the odd backward lane's loss partials and head scratch; the loss sum and
    // the flags stay shared (the odd member's head runs first)
    p->loss1_span = p->head1_span = Span{};
    if (p->bwd_lanes > 1) {
        BwdWs& q = p->bw1;
        p->loss1_span = Span{a.mark(), lp * sizeof(double)};
        q.loss_partial = a.take<double>(lp);
        q.loss_acc = b.loss_acc;
        q.flag = b.flag;
        q.bad_label = b.bad_label;
        if (g.loss == GP_LOSS_XENT_LS) {
            const size_t h0 = a.mark();
            q.sth = a.take<float>(2 * T);
            q.h = a.take_elt(T * D, e);
            q.z = a.take_elt(T * (long)g.V, e);
            p->head1_span = span_from(h0);
        }
    }
}

// GP_POISON: fill one workspace region with NaN on stream st.
gp_status poison_span(const gp_partition* p, const Span& sp, hipStream_t st) {
    if (!p->poison || sp.bytes == 0) return GP_OK;
    return poison_fill(p->ws + sp.off, sp.bytes, st);
}

// GP_POISON: a first-pass slot's layer slot and residual buffers.
gp_status poison_first_pass_slot(const gp_partition* p, int lane, hipStream_t st) {
    if (!p->poison) return GP_OK;
    gp_status s = GP_OK;
    for (const Span& sp : p->fpass[lane].span)
        if (s == GP_OK) s = poison_span(p, sp, st);
    return s;
}

// GP_POISON: a whole workspace set (residual stream and every layer slot),
// before a pass that rewrites all of it.
gp_status poison_set(const gp_partition* p, int set, hipStream_t st) {
    if (!p->poison) return GP_OK;
    gp_status s = GP_OK;
    for (const Span& sp : p->slot_span[set])
        if (s == GP_OK) s = poison_span(p, sp, st);
    return s;
}

// A GEMM launched split-K whose reduce is left to the LayerNorm that takes its
// output, the next launch on the same stream: a residual GEMM of a forward pass
// (EPI_RES_F32; layernorm_fwd_res runs both in one kernel), or an fp32 input-
// gradient GEMM of the backward (EPI_F32; the LayerNorm backward sums the
// partials as it loads them).  splits == 0: nothing pending.
struct PendingRes {
    int splits = 0;
    int epi = 0;
    GemmArgs g;  // the GEMM's arguments: partials (ws), bias, residual (aux), outputs
};

struct Ctx {
    gp_partition* p;
    hipStream_t st;
    int dt;
    float* ws = nullptr;        // split-K partials for launches on st
    bool last = false;          // the mini-batch's last backward micro-batch
    PendingRes* pend = nullptr; // forward passes: a deferred split-K reduce
    int nseq = 0;               // sequences of a forward pass (0: one micro-batch; 2n: a pair's recompute)
    void* v16 = nullptr;        // the feed-forward input in fp16 for passes on st (Linear::f16)
    int lane = 0;               // first forward passes: the slot (FirstPass) they run in
    BwdWs* bw = nullptr;        // backward scratch of the call's lane (nullptr: p->bw)
    const hipEvent_t* ln_gate = nullptr;  // even backward lane: the odd member's per-layer events
};

enum class Lane { Main, Side, Remat };

Ctx make_ctx(gp_partition* p, hipStream_t st, Lane lane = Lane::Main) {
    Ctx c{p, st, p->g.dtype};
    c.ws = lane == Lane::Side ? p->bw.splitk_side : lane == Lane::Remat ? p->bw.splitk_remat : p->bw.splitk;
    c.v16 = lane == Lane::Side ? nullptr : lane == Lane::Remat ? p->bw.v16_remat : p->bw.v16_main;
    return c;
}

#define GP_TRY(x)                    \
    do {                             \
        gp_status s_ = (x);          \
        if (s_ != GP_OK) return s_;  \
    } while (0)

// Run `launch` (which enqueues on c.st); when `role` is being timed (and this
// is a sampled launch of it), bracket it with two events on c.st and add its
// algorithmic work.
template <class F>
gp_status timed(const Ctx& c, int role, double flops, double bytes, F&& launch) {
    LaunchTimer& t = c.p->timer;
    if (!t.on(role)) return launch();
    if (t.seen[role]++ % t.every != 0) return launch();
    hipEvent_t e0, e1;
    GP_TRY(t.take(e0));
    GP_TRY(t.take(e1));
    if (t.markers) GP_TRY(role_marker(role, 0, c.st));
    // the events ride on the role's own kernel dispatches (klaunch)
    LaunchEvents& ev = launch_events();
    ev.start = e0;
    ev.stop = e1;
    ev.started = false;
    const gp_status s = launch();
    const bool launched = ev.started;
    ev = LaunchEvents();
    if (t.markers) GP_TRY(role_marker(role, 1, c.st));
    if (launched) {
        t.recs[role].emplace_back(e0, e1);
        t.flops[role] += flops;
        t.bytes[role] += bytes;
    } else {
        t.pool.push_back(e0);
        t.pool.push_back(e1);
    }
    return s;
}

// Algorithmic bytes of a GEMM: operands read once, outputs written once (and
// read once where the epilogue reads them).
double gemm_bytes(const GemmArgs& g, int epi, size_t esz) {
    const double mn = (double)g.M * g.N;
    double b = ((double)g.M * g.K + (double)g.N * g.K) * (double)esz;
    switch (epi) {
    case EPI_STORE: b += mn * esz; break;
    case EPI_RES_F32: b += mn * 8.0 + (g.C2 ? mn * esz : 0.0); break;
    case EPI_F32: b += mn * 4.0; break;
    case EPI_RELU_MASK: b += mn * 2.0 * esz; break;
    case EPI_ACC_F32: b += mn * 4.0 * (g.accumulate ? 2.0 : 1.0) + (g.colsum ? g.N * 4.0 * (g.accumulate ? 2.0 : 1.0) : 0.0); break;
    default: break;
    }
    return b;
}

gp_status timed_gemm(const Ctx& c, int role, const GemmArgs& g, int epi, bool kmaj) {
    return timed(c, role, 2.0 * g.M * g.N * (double)g.K, gemm_bytes(g, epi, c.p->esz),
                 [&] { return gemm(g, epi, kmaj, kmaj, c.dt, c.st); });
}

gp_status timed_attention(const Ctx& c, int role, const AttnArgs& a, bool bwd) {
    const double f = 4.0 * a.n * a.H * (double)a.Sq * a.Sk * a.dh * (a.causal ? 0.5 : 1.0) * (bwd ? 2.0 : 1.0);
    const double D = (double)a.H * a.dh, esz = (double)c.p->esz;
    const double qo = (double)a.n * a.Sq * D * esz, kv = (double)a.n * a.Sk * D * esz;
    const double stats = (double)a.n * a.H * a.Sq * 4.0;
    // forward: Q, K, V in, O and the log-sum-exp out; backward: Q, K, V, O, dO
    // and the log-sum-exp in, dQ, dK, dV out
    const double by = bwd ? 3.0 * qo + 4.0 * kv + stats : 2.0 * qo + 2.0 * kv + stats;
    return timed(c, role, f, by, [&] { return bwd ? attention_bwd(c.dt, a, c.st) : attention_fwd(c.dt, a, c.st); });
}

// The reduce of a deferred split-K GEMM on its own (when no LayerNorm takes it).
gp_status flush_pending(const Ctx& c) {
    if (!c.pend || c.pend->splits < 2) return GP_OK;
    const int sp = c.pend->splits;
    c.pend->splits = 0;
    return gemm_reduce(c.pend->g, c.pend->epi, sp, c.st);
}

gp_status timed_ln_fwd(const Ctx& c, const float* x, long rows, int D, const float* gamma, const float* beta,
                       float eps, void* out, float* stats, unsigned char* lo4 = nullptr, unsigned char* lo_sc = nullptr,
                       void* out16 = nullptr) {
    if (c.pend && c.pend->splits > 1) {
        const GemmArgs& g = c.pend->g;
        if (c.pend->epi == EPI_RES_F32 && g.C == x && g.M == rows && g.N == D) {
            // x is the pending GEMM's output: its reduce and this LayerNorm in one kernel
            const int sp = c.pend->splits;
            c.pend->splits = 0;
            const double plane = (double)rows * D;
            const double by =
                plane * (4.0 * sp + 4.0 + 4.0 + (g.C2 ? 2.0 : 0.0) + c.p->esz + (lo4 ? 0.5 : 0.0) + (out16 ? 2.0 : 0.0)) +
                rows * 8.0 + D * 12.0;
            return timed(c, GP_K_LN_FWD, 0.0, by, [&] {
                return layernorm_fwd_res(c.dt, g.ws, sp, (long)rows * D, g.bias, static_cast<const float*>(g.aux),
                                         static_cast<float*>(g.C), g.C2, rows, D, gamma, beta, eps, out, stats, lo4,
                                         lo_sc, c.st, out16);
            });
        }
        GP_TRY(flush_pending(c));
    }
    const double by = (double)rows * D * (4.0 + c.p->esz + (lo4 ? 0.5 : 0.0) + (out16 ? 2.0 : 0.0)) + rows * 8.0 +
                      D * 8.0;
    return timed(c, GP_K_LN_FWD, 0.0, by, [&] {
        return layernorm_fwd(c.dt, x, rows, D, gamma, beta, eps, out, stats, lo4, lo_sc, c.st, out16);
    });
}

// Y = A W + b with an epilogue; A [M, K] k-contiguous, W^T working copy [N, K].
// A4 / A4s: fp4 rounding residuals of A and their row scales (split layers).
// defer: the next launch on c.st is the LayerNorm of C, which may then take
// over a split-K reduce (EPI_RES_F32, see PendingRes).
gp_status linear_fwd(const Ctx& c, const Linear& L, const void* A, long M, void* C, long ldc, int epi, int relu,
                     const float* res, void* C2, const unsigned char* A4 = nullptr, const unsigned char* A4s = nullptr,
                     bool defer = false) {
    GP_TRY(flush_pending(c));
    GemmArgs g;
    g.M = (int)M;
    g.N = L.out;
    g.K = L.in;
    g.A = A;
    g.lda = L.in;
    g.B = c.p->W(L.nk);
    g.ldb = L.in;
    if (L.split && A4) {
        g.a4 = A4;
        g.sa4 = A4s;
        g.b4 = c.p->W(L.q4);
        g.sb4 = static_cast<const unsigned char*>(c.p->W(L.q4s));
    }
    g.C = C;
    g.ldc = ldc;
    g.C2 = C2;
    g.ldc2 = ldc;
    g.bias = c.p->master + L.b;
    g.aux = res;
    g.ldaux = ldc;
    g.relu = relu;
    g.ws = c.ws;
    g.ws_elems = c.p->bw.splitk_elems;
    g.force_cfg = c.p->gemm_tile;
    g.force_splits = c.p->gemm_splits;
    g.f16 = L.f16 ? 1 : 0;  // A is then the fp16 copy of the input, nk holds fp16
    // a pass over a pair's rows takes one micro-batch's tile and split choice
    // (same rounding as two single passes; the recompute workspace holds the
    // pair's partials)
    if (c.nseq && c.nseq != c.p->g.n) g.split_rows = (int)(M * c.p->g.n / c.nseq);
    int splits = 1;
    if (defer && c.pend && c.p->fuse_res_ln && epi == EPI_RES_F32 && ldc == L.out &&
        layernorm_fwd_res_ok(c.dt, L.out, c.ws, g.bias, res, static_cast<const float*>(C), C2))
        g.deferred = &splits;
    GP_TRY(timed_gemm(c, L.role, g, epi, true));
    if (splits > 1) {
        c.pend->splits = splits;
        c.pend->epi = epi;
        c.pend->g = g;
        c.pend->g.deferred = nullptr;
    }
    return GP_OK;
}

// The most split-K partial floats one first forward pass of a micro-batch
// writes: the largest need among its GEMMs, with the tile and split choice
// linear_fwd's arguments lead to (they depend on the shape, the epilogue, the
// fp4 correction and the workspace size, not on the operands' addresses).
long forward_workspace_need(const gp_partition* p) {
    static const unsigned char with_fp4 = 0;
    long need = 0;
    auto one = [&](const Linear& L, long M, int epi) {
        if (!L.present) return;
        GemmArgs g;
        g.M = (int)M;
        g.N = L.out;
        g.K = L.in;
        g.ws = p->bw.splitk;
        g.ws_elems = p->bw.splitk_elems;
        g.force_cfg = p->gemm_tile;
        g.force_splits = p->gemm_splits;
        if (L.split) g.a4 = &with_fp4;
        need = std::max(need, gemm_workspace_need(g, epi, true, p->g.dtype));
    };
    const long T = p->g.T(), Tm = p->g.Tm();
    for (const LayerPlan& P : p->plan.layers) {
        one(P.qkv, T, EPI_STORE);
        one(P.o, T, EPI_RES_F32);
        one(P.xq, T, EPI_STORE);
        one(P.xkv, Tm, EPI_STORE);
        one(P.xo, T, EPI_RES_F32);
        one(P.ffn1, T, EPI_STORE);
        one(P.ffn2, T, EPI_RES_F32);
    }
    return need;
}

// dX = dY W^T with an epilogue; dY [M, out] k-contiguous, W working copy [in, out].
gp_status linear_dx(const Ctx& c, const Linear& L, const void* dY, long M, void* C, int epi, const void* aux,
                    int accumulate, bool defer = false) {
    GP_TRY(flush_pending(c));
    GemmArgs g;
    g.M = (int)M;
    g.N = L.in;
    g.K = L.out;
    g.A = dY;
    g.lda = L.out;
    g.B = c.p->W(L.kn);
    g.ldb = L.out;
    g.C = C;
    g.ldc = L.in;
    g.aux = aux;
    g.ldaux = L.in;
    g.accumulate = accumulate;
    g.ws = c.ws;
    g.ws_elems = c.p->bw.splitk_elems;
    g.force_cfg = c.p->gemm_tile;
    g.force_splits = c.p->gemm_splits;
    int splits = 1;
    if (defer && c.pend && c.p->fuse_res_ln && epi == EPI_F32 && c.dt == GP_BF16 && L.in % 256 == 0 &&
        L.in <= 2048)
        g.deferred = &splits;
    GP_TRY(timed_gemm(c, L.role + 1, g, epi, true));
    if (splits > 1) {
        c.pend->splits = splits;
        c.pend->epi = epi;
        c.pend->g = g;
        c.pend->g.deferred = nullptr;
    }
    return GP_OK;
}

// G_W (+)= X^T dY and G_b (+)= sum_rows dY (one kernel).  X [rows, in], dY [rows, out].
gp_status linear_dw(const Ctx& c, const Linear& L, const void* X, const void* dY, long rows, int accumulate) {
    GP_TRY(flush_pending(c));
    GemmArgs g;
    g.M = L.in;
    g.N = L.out;
    g.K = (int)rows;
    g.A = X;
    g.lda = L.in;
    g.B = dY;
    g.ldb = L.out;
    g.C = c.p->grads + L.w;
    g.ldc = L.out;
    g.accumulate = accumulate;
    g.ws = c.ws;
    g.ws_elems = c.p->bw.splitk_elems;
    g.force_cfg = c.p->gemm_tile;
    g.force_splits = c.p->gemm_splits;
    g.colsum = c.p->grads + L.b;  // bias gradient fused into the GEMM
    return timed_gemm(c, L.role + 2, g, EPI_ACC_F32, false);
}

// A weight-gradient GEMM of one layer, collected while the layer's input-
// gradient chain is enqueued and launched afterwards (on the side stream when
// there is one).
struct DwJob {
    const Linear* L;
    const void* X;
    const void* dY;
    long rows;
};

// LayerNorm backward: dx, and the gamma/beta gradient partials added into
// the norm's partial buffer (overwritten on the first backward micro-batch);
// after the last micro-batch they are reduced into the gradients.
gp_status norm_bwd(const Ctx& c, const Norm& N, const float* dn, const float* x, const float* stats, long rows,
                   const float* dres, float* dx32, void* dxe, int accumulate) {
    int nblk = 0;
    float* part = c.p->lnpart[N.id];
    // dn still as the split-K partials of the GEMM that produced it: summed while loading
    int sp = 1;
    if (c.pend && c.pend->splits > 1) {
        const GemmArgs& g = c.pend->g;
        if (c.pend->epi == EPI_F32 && g.C == dn && g.M == rows && g.N == N.n && g.ldc == N.n) {
            sp = c.pend->splits;
            dn = g.ws;
            c.pend->splits = 0;
        } else {
            GP_TRY(flush_pending(c));
        }
    }
    const double rd = (double)rows * N.n;
    const double by = rd * (4.0 * sp + 4.0 + (dres ? 4.0 : 0.0) + (dx32 ? 4.0 : 0.0) + (dxe ? (double)c.p->esz : 0.0)) +
                      rows * 8.0 + (double)layernorm_bwd_blocks(rows) * 2 * N.n * 4.0 * (accumulate ? 2.0 : 1.0);
    return timed(c, GP_K_LN_BWD, 0.0, by, [&] {
        GP_TRY(layernorm_bwd(c.dt, dn, x, stats, c.p->master + N.g, rows, N.n, dres, dx32, dxe, part, accumulate,
                             &nblk, c.st, sp, rd > 0 ? (long)rd : 0));
        if (!c.last) return GP_OK;
        return colsum_finalize(part, nblk, 2 * N.n, c.p->grads + N.g, 0, c.st);
    });
}

AttnArgs attn_args(const gp_partition* p, int Sk, int causal, int nseq = 0) {
    AttnArgs a;
    a.n = nseq ? nseq : p->g.n;
    a.hint_n = a.n != p->g.n ? p->g.n : 0;  // a pair's pass takes one micro-batch's kernel variant
    a.H = p->d.H;
    a.Sq = p->g.S;
    a.Sk = Sk;
    a.dh = p->d.D / p->d.H;
    a.causal = causal;
    a.scale = 1.f / sqrtf((float)a.dh);
    a.split = p->attn_split ? 1 : 0;
    a.waves = p->attn_waves;
    return a;
}

// One layer's forward.  `ws` holds its intermediates, x_in/x_out the residual
// stream; mem is the decoder memory (elt [Tm, D]); y_out (optional) receives
// the output rounded to the partition dtype.
gp_status layer_forward(const Ctx& c, int l, LayerWs& w, const float* x_in, float* x_out, const void* mem,
                        void* y_out) {
    gp_partition* p = c.p;
    const LayerPlan& P = p->plan.layers[l];
    const int ns = c.nseq ? c.nseq : p->g.n;
    const long T = (long)ns * p->g.S, Tm = (long)ns * p->g.Smem, D = p->d.D;
    const bool dec = p->g.kind == GP_DECODER_CROSS;
    const float eps = p->g.eps;
    // self-attention block
    GP_TRY(timed_ln_fwd(c, x_in, T, (int)D, p->master + P.ln1.g, p->master + P.ln1.b, eps, w.u, w.st1));
    GP_TRY(linear_fwd(c, P.qkv, w.u, T, w.qkv, 3 * D, EPI_STORE, 0, nullptr, nullptr));
    AttnArgs a = attn_args(p, p->g.S, dec ? 1 : 0, ns);
    a.q = w.qkv;
    a.k = p->off_elt(w.qkv, D);
    a.v = p->off_elt(w.qkv, 2 * D);
    a.ldq = a.ldk = a.ldv = 3 * D;
    a.o = w.c;
    a.ldo = D;
    a.lse = w.lse;
GP_TRY(timed_attention(c, GP_K_ATTN_FWD, a, false));
    GP_TRY(linear_fwd(c, P.o, w.c, T, w.x1, D, EPI_RES_F32, 0, x_in, nullptr, nullptr, nullptr, true));
    const float* xf = w.x1;
    if (dec) {
        // cross-attention block: queries from LN2(x1), keys/values from the memory
        GP_TRY(timed_ln_fwd(c, w.x1, T, (int)D, p->master + P.ln2.g, p->master + P.ln2.b, eps, w.uc, w.stc));
        GP_TRY(linear_fwd(c, P.xq, w.uc, T, w.xq, D, EPI_STORE, 0, nullptr, nullptr));
        GP_TRY(linear_fwd(c, P.xkv, mem, Tm, w.xkv, 2 * D, EPI_STORE, 0, nullptr, nullptr));
        AttnArgs x = attn_args(p, p->g.Smem, 0, ns);
        x.q = w.xq;
        x.ldq = D;
        x.k = w.xkv;
        x.v = p->off_elt(w.xkv, D);
        x.ldk = x.ldv = 2 * D;
        x.o = w.xc;
        x.ldo = D;
        x.lse = w.xlse;
        GP_TRY(timed_attention(c, GP_K_XATTN_FWD, x, false));
        GP_TRY(linear_fwd(c, P.xo, w.xc, T, w.x2, D, EPI_RES_F32, 0, w.x1, nullptr, nullptr, nullptr, true));
        xf = w.x2;
    }
    // feed-forward block
    const Norm& nf = dec ? P.ln3 : P.ln2;
    // The fp4 correction of the bf16-rounded LayerNorm output runs in the
    // first pass and in the recompute alike, so that the recompute reproduces
    // the first pass bit for bit (the backward differentiates the very F_k
    // whose output left the partition).
    const bool s4 = P.ffn1.split, h16 = P.ffn1.f16;
    if (h16 && !c.v16) return set_error(GP_ERR_INVALID_ARG, "fp16 feed-forward input buffer missing on this stream");
    GP_TRY(timed_ln_fwd(c, xf, T, (int)D, p->master + nf.g, p->master + nf.b, eps, w.v, w.stf, s4 ? w.v4 : nullptr,
                        s4 ? w.v4s : nullptr, h16 ? c.v16 : nullptr));
    GP_TRY(linear_fwd(c, P.ffn1, h16 ? c.v16 : w.v, T, w.a, p->d.F, EPI_STORE, 1, nullptr, nullptr,
                      s4 ? w.v4 : nullptr, s4 ? w.v4s : nullptr));
    // the next layer begins with the LayerNorm of x_out
    GP_TRY(linear_fwd(c, P.ffn2, w.a, T, x_out, D, EPI_RES_F32, 0, xf, y_out, nullptr, nullptr, l + 1 < p->d.L));
    return GP_OK;
}

// Forward of micro-batch m through all layers.  keep = false: a first pass
// in the first-pass slot, intermediates discarded (one layer slot, ping-pong
// residuals); keep = true: every layer's intermediates kept in workspace set
// `set`, for c.nseq sequences (2n: micro-batches m and m + 1 together, in the
// group whose first member is `set`).  x != nullptr: x (and mem) go into the
// stash unless skip_intake, and y (optional) receives the output;
// x == nullptr: the re-materialisation from the stash.
gp_status partition_forward(const Ctx& c, int m, bool keep, const void* x, const void* mem, void* y, int set = 0,
                            bool skip_intake = false) {
    gp_partition* p = c.p;
    const int ns = c.nseq ? c.nseq : p->g.n;
    const long T = (long)ns * p->g.S, Tm = (long)ns * p->g.Smem, D = p->d.D;
    const int L = p->d.L;
    FirstPass& f = p->fpass[c.lane];
    float* x0 = keep ? p->xs[set][0] : f.xs[0];
    if (x) {
        if (!skip_intake) {
            GP_TRY(intake(c.dt, x, p->stash_x_mb(m), x0, T * D, c.st));
            if (mem) GP_TRY(intake(c.dt, mem, p->stash_m_mb(m), nullptr, Tm * D, c.st));
        }
    } else {
        GP_TRY(intake(c.dt, p->stash_x_mb(m), nullptr, x0, T * D, c.st));
    }
    const void* mem_m = p->g.kind == GP_DECODER_CROSS ? p->stash_m_mb(m) : nullptr;
    PendingRes pend;
    Ctx cf = c;
    cf.pend = &pend;
    for (int l = 0; l < L; ++l) {
        LayerWs& w = keep ? p->lw[set][l] : f.w;
        const float* xi = keep ? p->xs[set][l] : f.xs[l & 1];
        float* xo = keep ? p->xs[set][l + 1] : f.xs[(l + 1) & 1];
        GP_TRY(layer_forward(cf, l, w, xi, xo, mem_m, l == L - 1 ? y : nullptr));
    }
    return flush_pending(cf);
}

// The re-materialisation unit of micro-batch m: the micro-batches one
// recompute pass covers -- {lo, ..., lo + r - 1} with lo = m - m % r for a
// recompute group of r, cut at the last micro-batch -- as its first
// micro-batch and count.  Its recompute must be done before the backward of
// its highest member, which comes first.
void remat_unit(const gp_partition* p, int m, int& lo, int& cnt) {
    const int r = p->remat_group;
    lo = m - m % r;
    cnt = std::min(r, p->g.M - lo);
}

// Recompute the forward of a unit from the stash into its workspace set(s),
// keeping every intermediate, on c's stream.  A pair is one pass over both
// micro-batches' rows, with each kernel's variant chosen as for one
// micro-batch, so that every value equals its first-pass value bit for bit.
gp_status remat_pass(const Ctx& c, int lo, int cnt) {
    gp_partition* p = c.p;
    const int set = p->set_of(lo);
    for (int i = 0; i < cnt; ++i) GP_TRY(poison_set(p, p->set_of(lo + i), c.st));
    Ctx cr = c;
    cr.nseq = cnt * p->g.n;
    return partition_forward(cr, lo, true, nullptr, nullptr, nullptr, set);
}

// The capture a stream is recording into (0: none).
unsigned long long capture_of(hipStream_t st) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    unsigned long long id = 0;
    if (hipStreamGetCaptureInfo(st, &cs, &id) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return cs == hipStreamCaptureStatusActive ? id : 0;
}

// Make st wait for an event an earlier call recorded on stream `from`, unless
// there is none, it was st itself (stream order covers it), or the two belong
// to different captures (a graph is ordered by its own edges, and a capture
// cannot wait on work outside it).
gp_status wait_recorded(hipStream_t st, hipStream_t from, hipEvent_t ev, unsigned long long cap) {
    if (!ev || from == st || cap != capture_of(st)) return GP_OK;
    GP_HIP(hipStreamWaitEvent(st, ev, 0));
    return GP_OK;
}

// Context of a first forward pass in slot `lane`: the odd slot has its own
// split-K partials and fp16 buffer.
Ctx first_pass_ctx(gp_partition* p, hipStream_t st, int lane) {
    Ctx c = make_ctx(p, st);
    c.lane = lane;
    if (lane) {
        c.ws = p->fpass[lane].splitk;
        c.v16 = p->fpass[lane].v16;
    }
    return c;
}

// Order a first forward pass on c.st after the previous forward in its slot
// (and, with `both`, in the other slot) and after the last update, whose
// weights it reads and whose mini-batch's backward used the even slot's
// partials.  Calls on one stream are ordered by the stream already.
gp_status order_first_pass(gp_partition* p, const Ctx& c, bool both) {
    for (int ln = 0; ln < p->fp_lanes; ++ln) {
        if (ln != c.lane && !both) continue;
        const FirstPass& f = p->fpass[ln];
        GP_TRY(wait_recorded(c.st, f.stream, f.done, f.capture));
    }
    return wait_recorded(c.st, p->tail_stream, p->tail_done, p->tail_capture);
}

// Record the end of a first forward pass in its slot.
gp_status record_first_pass(gp_partition* p, const Ctx& c) {
    if (!p->events()) return GP_OK;
    FirstPass& f = p->fpass[c.lane];
    f.done = p->next_event();
    GP_HIP(hipEventRecord(f.done, c.st));
    f.stream = c.st;
    f.capture = capture_of(c.st);
    return GP_OK;
}

// Backward of one layer.  dY arrives in (in32, ine); dX leaves in the pair
// returned through out32/oute.  The fp32 halves ping-pong between the two
// backward buffers; every bf16 gradient the layer writes takes the next
// buffer of the ring (`ri`), and dz / dQKV (and the cross-attention dQ, dKV)
// alternate by layer parity, so that the layer's weight-gradient GEMMs -- which
// read ine, the LayerNorm outputs, dz and dQKV -- can run while the next layer
// down is processed.  They are appended to `jobs` and launched by `flush`
// at the granularity the partition is set to (the caller flushes the rest).
template <class Flush>
gp_status layer_backward(const Ctx& c, int set, int half, int l, bool first, float* in32, void* ine, float* sc32,
                         int& ri, float*& out32, void*& oute, float* dx32_final, void* dxe_final, const void* mem,
                         std::vector<DwJob>& jobs, Flush&& flush) {
    gp_partition* p = c.p;
    const LayerPlan& P = p->plan.layers[l];
    LayerWs& w = p->lw[set][l];
    BwdWs& b = c.bw ? *c.bw : p->bw;
    const long T = p->g.T(), Tm = p->g.Tm(), D = p->d.D, F = p->d.F;
    const bool dec = p->g.kind == GP_DECODER_CROSS;
    const int acc = first ? 0 : 1;
    const int par = l & 1;
    auto next_elt = [&]() {
        void* r = b.ring[ri];
        ri = (ri + 1) % ELT_RING;
        return r;
    };
    // The weight gradients' dY operands: with grouping, this micro-batch's rows
    // of the layer's grouped buffers (kept for the group's one GEMM); else the
    // parity buffers and the ring.
    const bool pr = p->group > 1;
    auto hrow = [&](void* base, long rows, long width) { return p->off_elt(base, (long)half * rows * width); };
    void* dz = pr ? hrow(p->dys[l].dz, T, F) : b.dz[par];
    void* dqkv = pr ? hrow(p->dys[l].dqkv, T, 3 * D) : b.dqkv[par];
    void* dxq = pr && dec ? hrow(p->dys[l].dxq, T, D) : b.dxq[par];
    void* dxkv = pr && dec ? hrow(p->dys[l].dxkv, Tm, 2 * D) : b.dxkv[par];
    const float* xf = dec ? w.x2 : w.x1;
    const Norm& nf = dec ? P.ln3 : P.ln2;
    // feed-forward block:  dz = dY W2^T * [a > 0];  dv = dz W1^T;  dW2, dW1 (and biases) as jobs
    // flush(0): after each weight-gradient job; flush(1): after the feed-forward block
    jobs.push_back({&P.ffn2, w.a, ine, T});
    GP_TRY(flush(0));
    GP_TRY(linear_dx(c, P.ffn2, ine, T, dz, EPI_RELU_MASK, w.a, 0));
    jobs.push_back({&P.ffn1, w.v, dz, T});
    GP_TRY(flush(0));
    GP_TRY(linear_dx(c, P.ffn1, dz, T, b.dn, EPI_F32, nullptr, 0, true));
    GP_TRY(flush(1));
    void* sce = pr ? hrow(p->dys[l].gffn, T, D) : next_elt();
    // the other lane's layer l first: the LayerNorm partial sums accumulate in micro-batch order
    if (c.ln_gate) GP_HIP(hipStreamWaitEvent(c.st, c.ln_gate[l], 0));
    GP_TRY(norm_bwd(c, nf, b.dn, xf, w.stf, T, in32, sc32, sce, acc));
    // (sc) = dL/d(xf)
    float* cur32 = sc32;
    void* cure = sce;
    float* oth32 = in32;
    if (dec) {
        // cross-attention block
        jobs.push_back({&P.xo, w.xc, cure, T});
        GP_TRY(flush(0));
        GP_TRY(linear_dx(c, P.xo, cure, T, b.dc, EPI_STORE, nullptr, 0));
        AttnArgs x = attn_args(p, p->g.Smem, 0);
        x.q = w.xq;
        x.ldq = D;
        x.k = w.xkv;
        x.v = p->off_elt(w.xkv, D);
        x.ldk = x.ldv = 2 * D;
        x.o = w.xc;
        x.ldo = D;
        x.lse = w.xlse;
        x.dout = b.dc;
        x.lddo = D;
        x.dq = dxq;
        x.lddq = D;
        x.dk = dxkv;
        x.dv = p->off_elt(dxkv, D);
        x.lddk = x.lddv = 2 * D;
        x.delta = b.delta;
        GP_TRY(timed_attention(c, GP_K_XATTN_BWD, x, true));
        jobs.push_back({&P.xq, w.uc, dxq, T});
        GP_TRY(flush(0));
        GP_TRY(linear_dx(c, P.xq, dxq, T, b.dn, EPI_F32, nullptr, 0));
        jobs.push_back({&P.xkv, mem, dxkv, Tm});
        GP_TRY(flush(0));
        GP_TRY(linear_dx(c, P.xkv, dxkv, Tm, b.dmem32, EPI_ACC_F32, nullptr, l == p->d.L - 1 ? 0 : 1));
        void* e2 = pr ? hrow(p->dys[l].gcross, T, D) : next_elt();
        GP_TRY(norm_bwd(c, P.ln2, b.dn, w.x1, w.stc, T, cur32, oth32, e2, acc));
        std::swap(cur32, oth32);
        cure = e2;
    }
    // self-attention block
    jobs.push_back({&P.o, w.c, cure, T});
    GP_TRY(flush(0));
    GP_TRY(linear_dx(c, P.o, cure, T, b.dc, EPI_STORE, nullptr, 0));
    AttnArgs a = attn_args(p, p->g.S, dec ? 1 : 0);
    a.q = w.qkv;
    a.k = p->off_elt(w.qkv, D);
    a.v = p->off_elt(w.qkv, 2 * D);
    a.ldq = a.ldk = a.ldv = 3 * D;
    a.o = w.c;
    a.ldo = D;
    a.lse = w.lse;
    a.dout = b.dc;
    a.lddo = D;
    a.dq = dqkv;
    a.dk = p->off_elt(dqkv, D);
    a.dv = p->off_elt(dqkv, 2 * D);
    a.lddq = a.lddk = a.lddv = 3 * D;
    a.delta = b.delta;
    GP_TRY(timed_attention(c, GP_K_ATTN_BWD, a, true));
    jobs.push_back({&P.qkv, w.u, dqkv, T});
    GP_TRY(flush(0));
    GP_TRY(linear_dx(c, P.qkv, dqkv, T, b.dn, EPI_F32, nullptr, 0, true));
    const float* x_in = p->xs[set][l];
    if (dxe_final || dx32_final || l == 0) {
        GP_TRY(norm_bwd(c, P.ln1, b.dn, x_in, w.st1, T, cur32, dx32_final, dxe_final, acc));
        out32 = dx32_final;
        oute = dxe_final;
    } else {
        void* oe = pr ? hrow(p->dys[l - 1].gin, T, D) : next_elt();
        GP_TRY(norm_bwd(c, P.ln1, b.dn, x_in, w.st1, T, cur32, oth32, oe, acc));
        out32 = oth32;
        oute = oe;
    }
    return GP_OK;
}

gp_status head_backward(const Ctx& c, int set, bool first, const int* labels, void* dy_elt) {
    gp_partition* p = c.p;
    const HeadPlan& Hd = p->plan.head;
    BwdWs& b = c.bw ? *c.bw : p->bw;
    const long T = p->g.T(), D = p->d.D, V = p->g.V;
    const int acc = first ? 0 : 1;
    const float* y = p->xs[set][p->d.L];
    GP_TRY(timed_ln_fwd(c, y, T, (int)D, p->master + Hd.lnf.g, p->master + Hd.lnf.b, p->g.eps, b.h, b.sth));
    GP_TRY(linear_fwd(c, Hd.out, b.h, T, b.z, V, EPI_STORE, 0, nullptr, nullptr));
    const double norm = (double)p->g.n * p->g.M * p->g.S;
    GP_TRY(xent_ls(c.dt, b.z, T, (int)V, labels, p->g.ls, p->g.logit_clip, norm, b.loss_partial, b.bad_label, c.st));
    GP_TRY(loss_finalize(b.loss_partial, (int)T, b.loss_acc, acc, c.st));
    GP_TRY(linear_dw(c, Hd.out, b.h, b.z, T, acc));
    GP_TRY(linear_dx(c, Hd.out, b.z, T, b.dn, EPI_F32, nullptr, 0));
    return norm_bwd(c, Hd.lnf, b.dn, y, b.sth, T, nullptr, b.p32, dy_elt, acc);
}

gp_status upload_param_block(gp_partition* p, const ParamRef& r, const float* host) {
    GP_HIP(hipMemcpy2D(p->master + r.off, (size_t)r.ld * 4, host, (size_t)r.cols * 4, (size_t)r.cols * 4, r.rows,
                       hipMemcpyHostToDevice));
    if (r.lin) {
        GP_TRY(refresh_linear(p->g.dtype, p->master + r.lin->w, r.lin->in, r.lin->out, p->W(r.lin->kn),
                              p->W(r.lin->nk), r.lin->split ? p->W(r.lin->q4) : nullptr,
                              r.lin->split ? p->W(r.lin->q4s) : nullptr, nullptr, r.lin->f16));
        GP_HIP(hipDeviceSynchronize());
    }
    return GP_OK;
}

void free_all(gp_partition* p) {
    for (hipEvent_t e : p->evring)
        if (e) (void)hipEventDestroy(e);
    p->evring.clear();
    p->ev_next = 0;
    for (hipEvent_t& e : p->side_done) e = nullptr;
    if (p->side) (void)hipStreamDestroy(p->side);
    p->side = nullptr;
    if (p->remat) (void)hipStreamDestroy(p->remat);
    p->remat = nullptr;
    p->remat_done = nullptr;
    p->remat_pending = -1;
    for (hipEvent_t e : p->timer.all) (void)hipEventDestroy(e);
    const bool markers = p->timer.markers;
    p->timer = LaunchTimer();
    p->timer.markers = markers;
    for (void* x : {(void*)p->master, (void*)p->grads, (void*)p->welt, (void*)p->stash_x, (void*)p->stash_m,
                    (void*)p->ws, (void*)p->opt_ms, (void*)p->upd_ranges})
        if (x) (void)hipFree(x);
    p->master = p->grads = p->opt_ms = nullptr;
    p->upd_ranges = nullptr;
    p->n_upd_ranges = 0;
    p->fused_update = false;
    p->welt = p->stash_x = p->stash_m = p->ws = nullptr;
}

gp_status alloc(void** ptr, size_t bytes) {
    if (bytes == 0) bytes = 256;
    hipError_t e = hipMalloc(ptr, bytes);
    if (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        return set_error(GP_ERR_OOM, "device allocation failed (out of memory)");
    }
    if (e != hipSuccess) return hip_fail(e, __FILE__, __LINE__);
    return GP_OK;
}

} // namespace

// Scratch of gp_forward_microbatch_noalloc: the split-K partial tiles of the
// GEMMs of its forward pass live in this file-scope device array instead of
// the partition's workspace, so that a caller can run that pass with no
// allocation anywhere.  Each device the library runs on holds its own copy
// until the process ends; every such call on a device shares it, so calls
// that overlap on one device race.  Nothing in it needs clearing: a GEMM
// writes every partial tile it later reads.
constexpr size_t NOALLOC_SCRATCH_FLOATS = (size_t)8 << 20;  // 32 MiB
static __device__ __align__(256) float scratch[NOALLOC_SCRATCH_FLOATS];

namespace {
// Host code cannot use `scratch` itself (its host-side name is a stand-in,
// not a device address): the address is resolved once per device, with that
// device current, and kept here.
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[MAX_DEVICES] = {};
bool g_scratch_done[MAX_DEVICES] = {};
hipError_t g_scratch_err[MAX_DEVICES] = {};

// This device's address of `scratch` (nullptr and *err set on failure).
float* scratch_for_device(int dev, hipError_t* err) {
    if (dev < 0 || dev >= MAX_DEVICES) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_done[dev]) {
        void* ptr = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? static_cast<float*>(ptr) : nullptr;
        g_scratch_done[dev] = true;
    }
    *err = g_scratch_err[dev];
    return g_scratch_ptr[dev];
}
} // namespace

namespace {
// Geometry, schedule knobs, parameter plan and byte counts of a partition for
// cfg (already validated); host arithmetic only, no device is touched.
void plan_partition(gp_partition* p, const gp_config* cfg) {
    Geometry& g = p->g;
    g.S = cfg->seq_len;
    g.n = cfg->seqs_per_microbatch;
    g.M = cfg->num_microbatches;
    g.dtype = cfg->dtype;
    g.kind = cfg->kind;
    g.Smem = cfg->mem_seq_len;
    g.loss = cfg->loss;
    g.V = cfg->vocab;
    g.ls = cfg->label_smoothing;
    g.eps = cfg->ln_eps;
    g.check_finite = cfg->check_finite;
    g.keep_act = cfg->keep_activations;
    g.optimizer = cfg->optimizer;
    g.rms_decay = cfg->rms_decay;
    g.rms_eps = cfg->rms_eps;
    g.logit_clip = cfg->logit_clip;
    p->esz = g.dtype == GP_BF16 ? 2 : 4;
    if (const char* e = std::getenv("GP_TIMER_MARKERS")) p->timer.markers = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_SIDE_STREAM")) p->use_side = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_LAYER_UPDATE")) p->layer_update = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_REMAT_AHEAD")) p->remat_ahead = std::atoi(e) != 0;
    // Early recompute by default where a micro-batch has at most 1024 rows:
    // with 2048 (enc1024, M = 8) the recompute of the last pair competes with
    // the last two forwards and the step was 0.45 ms slower with it; at 512
    // rows (M = 32) it was 0.5 ms faster, at 1024 and 4096 even.
    p->remat_early = g.T() <= 1024;
    if (const char* e = std::getenv("GP_REMAT_EARLY")) p->remat_early = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_FUSE_RES_LN")) p->fuse_res_ln = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_ATTN_KSPLIT")) p->attn_split = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_ATTN_WAVES")) p->attn_waves = std::atoi(e);
    if (const char* e = std::getenv("GP_POISON")) p->poison = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_DW_FLUSH")) p->dw_flush = std::atoi(e);
    if (const char* e = std::getenv("GP_PAIR_DW")) p->pair_dw = std::atoi(e) != 0;
    // Workspace sets in groups of the micro-batches whose weight gradients
    // run as one GEMM: two, or four with GP_DW_GROUP=4 (GP_DW_GROUP=1 or
    // GP_PAIR_DW=0: none); one set per micro-batch when activations are kept,
    // else two groups (recompute-ahead) or one.  Groups of four halve the
    // accumulator passes again but hold twice the re-materialised sets
    // (enc1024: M = 32 1.8% faster with 3.9 instead of 2.2 GB of workspace,
    // M = 16 0.6% with 7.1 instead of 3.8 GB), so two is the default: the
    // workspace keeps shrinking as M grows.
    int grp = 2;
    if (const char* e = std::getenv("GP_DW_GROUP")) grp = std::atoi(e);
    if (grp != 1 && grp != 2 && grp != 4) grp = 2;
    p->group = p->pair_dw ? std::max(1, std::min(grp, g.M >= 4 ? 4 : g.M >= 2 ? 2 : 1)) : 1;
    // Recompute pairs in one pass where a micro-batch has at most 2048 rows:
    // the pass's GEMMs fill more of the chip, and (without a loss head) the
    // pair's backwards can then run side by side in two lanes.  Measured at
    // enc1024 with both: M = 32 -14%, M = 16 -8%, M = 8 -1.4%; at M = 4
    // (4096 rows) +1%.  GP_PAIR_REMAT=0/1 forces it.
    bool pair_remat = g.T() <= 2048;
    if (const char* e = std::getenv("GP_PAIR_REMAT")) pair_remat = std::atoi(e) != 0;
    p->remat_group = pair_remat && p->group >= 2 && !g.keep_act ? 2 : 1;
    p->ahead_on = !g.keep_act && p->remat_ahead && g.M >= 2;
    // two first-pass slots (GP_FWD_LANES=1: one), so that forwards issued on
    // two streams overlap
    int lanes = 2;
    if (const char* e = std::getenv("GP_FWD_LANES")) lanes = std::atoi(e) == 1 ? 1 : 2;
    p->fp_lanes = g.M >= 2 ? lanes : 1;
    p->nsets = g.keep_act ? (g.M + p->group - 1) / p->group * p->group : p->group * (p->ahead_on ? 2 : 1);
    // two backward lanes for recompute pairs
    int blanes = 2;
    if (const char* e = std::getenv("GP_BWD_LANES")) blanes = std::atoi(e) == 1 ? 1 : 2;
    p->bwd_lanes = blanes > 1 && p->group == 2 && p->remat_group == 2 && p->ahead_on && p->use_side ? 2 : 1;
    if (const char* e = std::getenv("GP_GEMM_TILE")) p->gemm_tile = std::atoi(e);
    if (const char* e = std::getenv("GP_GEMM_SPLITS")) p->gemm_splits = std::atoi(e);
    if (const char* e = std::getenv("GP_FFN_FP4")) g.ffn_fp4 = std::atoi(e) != 0;
    if (const char* e = std::getenv("GP_FFN_F16")) g.ffn_f16 = std::atoi(e) != 0;
    p->plan = plan_params(p->d, g);
    Arena measure;
    plan_workspace(p, measure);
    const bool rms = g.optimizer == GP_OPT_RMSPROP;
    p->bytes_params = p->plan.n32 * 4 * (rms ? 2 : 1) + p->plan.nelt * p->esz;
    p->bytes_grads = p->plan.n32 * 4;
    p->bytes_stash = (size_t)g.M * (g.T() + g.Tm()) * p->d.D * p->esz;
    p->bytes_ws = measure.off;
}
} // namespace

extern "C" {

const char* gp_last_error(void) { return g_err.c_str(); }

gp_status gp_partition_create(int layers, int d_model, int d_ff, int heads, gp_partition** out) {
    if (!out) return set_error(GP_ERR_INVALID_ARG, "out must not be NULL");
    *out = nullptr;
    std::string msg;
    gp_status s = check_dims(layers, d_model, d_ff, heads, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    gp_partition* p = new (std::nothrow) gp_partition();
    if (!p) return set_error(GP_ERR_OOM, "host allocation failed");
    p->d.L = layers;
    p->d.D = d_model;
    p->d.F = d_ff;
    p->d.H = heads;
    *out = p;
    return GP_OK;
}

gp_status gp_memory_plan(int layers, int d_model, int d_ff, int heads, const gp_config* cfg, size_t* params,
                         size_t* grads, size_t* stash, size_t* workspace) {
    if (!cfg) return set_error(GP_ERR_INVALID_ARG, "config must not be NULL");
    std::string msg;
    gp_status s = check_dims(layers, d_model, d_ff, heads, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    gp_partition p;
    p.d.L = layers;
    p.d.D = d_model;
    p.d.F = d_ff;
    p.d.H = heads;
    s = check_config(p.d, *cfg, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    plan_partition(&p, cfg);
    if (params) *params = p.bytes_params;
    if (grads) *grads = p.bytes_grads;
    if (stash) *stash = p.bytes_stash;
    if (workspace) *workspace = p.bytes_ws;
    return GP_OK;
}

gp_status gp_partition_configure(gp_partition* p, const gp_config* cfg) {
    if (!p || !cfg) return set_error(GP_ERR_INVALID_ARG, "partition and config must not be NULL");
    std::string msg;
    if (p->sched.configured()) return set_error(GP_ERR_STATE, "partition already configured");
    gp_status s = check_config(p->d, *cfg, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    plan_partition(p, cfg);
    const Geometry& g = p->g;
    const bool rms = g.optimizer == GP_OPT_RMSPROP;
    void *m = nullptr, *gr = nullptr, *we = nullptr, *sx = nullptr, *sm = nullptr, *ws = nullptr;
    s = alloc(&m, p->plan.n32 * 4);
    if (s == GP_OK) s = alloc(&gr, p->plan.n32 * 4);
    if (s == GP_OK) s = alloc(&we, p->plan.nelt * p->esz);
    if (s == GP_OK) s = alloc(&sx, (size_t)g.M * g.T() * p->d.D * p->esz);
    if (s == GP_OK && g.Tm() > 0) s = alloc(&sm, (size_t)g.M * g.Tm() * p->d.D * p->esz);
    if (s == GP_OK) s = alloc(&ws, p->bytes_ws);
    void* ms = nullptr;
    if (s == GP_OK && rms) s = alloc(&ms, p->plan.n32 * 4);
    p->opt_ms = (float*)ms;
    p->master = (float*)m;
    p->grads = (float*)gr;
    p->welt = (char*)we;
    p->stash_x = (char*)sx;
    p->stash_m = (char*)sm;
    p->ws = (char*)ws;
    if (s != GP_OK) {
        free_all(p);
        return s;
    }
    Arena real;
    real.base = p->ws;
    plan_workspace(p, real);
    // parameters: zero, LayerNorm gains 1; accumulators zero
    std::vector<float> init(p->plan.n32, 0.f);
    for (const Norm* n : p->plan.norms())
        for (int i = 0; i < n->n; ++i) init[n->g + i] = 1.f;
    hipError_t e = hipMemcpy(p->master, init.data(), p->plan.n32 * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(p->grads, 0, p->plan.n32 * 4);
    if (e == hipSuccess) e = hipMemset(p->ws, 0, p->bytes_ws);
    if (e == hipSuccess && p->opt_ms) e = hipMemset(p->opt_ms, 0, p->plan.n32 * 4);
    if (e == hipSuccess && g.dtype == GP_BF16) {
        std::vector<long> ranges;
        if (plan_update_ranges(p->plan, ranges)) {
            e = hipMalloc((void**)&p->upd_ranges, ranges.size() * sizeof(long));
            if (e == hipSuccess)
                e = hipMemcpy(p->upd_ranges, ranges.data(), ranges.size() * sizeof(long), hipMemcpyHostToDevice);
            p->n_upd_ranges = (int)(ranges.size() / 2);
            p->fused_update = e == hipSuccess;
        }
    }
    if (e != hipSuccess) {
        free_all(p);
        return hip_fail(e, __FILE__, __LINE__);
    }
    for (const Linear* l : p->plan.linears()) {
        s = refresh_linear(g.dtype, p->master + l->w, l->in, l->out, p->W(l->kn), p->W(l->nk),
                           l->split ? p->W(l->q4) : nullptr, l->split ? p->W(l->q4s) : nullptr, nullptr, l->f16);
        if (s != GP_OK) {
            free_all(p);
            return s;
        }
    }
    // default priority, like every stream of the library
    if (p->use_side) e = hipStreamCreateWithFlags(&p->side, hipStreamNonBlocking);
    if (e == hipSuccess && p->ahead()) e = hipStreamCreateWithFlags(&p->remat, hipStreamNonBlocking);
    p->hi_ev.assign(p->d.L, nullptr);
    p->lay_main.assign(p->d.L, nullptr);
    p->lay_side.assign(p->d.L, nullptr);
    // events that order the library's streams and the calls a caller issues
    // on different streams
    if (e == hipSuccess) {
        p->evring.assign(4096, nullptr);
        for (size_t i = 0; e == hipSuccess && i < p->evring.size(); ++i)
            e = hipEventCreateWithFlags(&p->evring[i], hipEventDisableTiming);
    }
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        free_all(p);
        return hip_fail(e, __FILE__, __LINE__);
    }
    // the no-allocation forward's scratch on this device, and its need
    int dev = 0;
    hipError_t se = hipGetDevice(&dev);
    if (se == hipSuccess) p->noalloc_scratch = scratch_for_device(dev, &se);
    if (se != hipSuccess) {
        (void)hipGetLastError();
        p->noalloc_scratch = nullptr;
        p->noalloc_error = std::string("the static scratch array has no address on this device: ") +
                           hipGetErrorString(se);
    }
    p->fwd_ws_need = forward_workspace_need(p);
    p->sched.configure(g.M, msg);
    return GP_OK;
}

gp_status gp_partition_destroy(gp_partition* p) {
    if (!p) return GP_OK;
    if (p->sched.configured()) (void)hipDeviceSynchronize();
    free_all(p);
    delete p;
    return GP_OK;
}

static gp_status param_io(gp_partition* p, int layer, int id, float* host, size_t count, int what) {
    if (!p || !host) return set_error(GP_ERR_INVALID_ARG, "partition and host buffer must not be NULL");
    std::string msg;
    if (!p->sched.configured()) return set_error(GP_ERR_STATE, "partition not configured");
    if (what == 0) {
        gp_status s = p->sched.can_set_param(msg);
        if (s != GP_OK) return set_error(s, msg.c_str());
    }
    ParamRef r;
    gp_status s = resolve_param(p->plan, p->d, layer, id, r, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    if (count != (size_t)r.rows * r.cols) return set_error(GP_ERR_INVALID_ARG, "count does not match the parameter's size");
    if (what == 0) return upload_param_block(p, r, host);
    GP_HIP(hipDeviceSynchronize());
    const float* src = (what == 1 ? p->master : p->grads) + r.off;
    GP_HIP(hipMemcpy2D(host, (size_t)r.cols * 4, src, (size_t)r.ld * 4, (size_t)r.cols * 4, r.rows,
                       hipMemcpyDeviceToHost));
    return GP_OK;
}

gp_status gp_set_param(gp_partition* p, int layer, int id, const float* host, size_t count) {
    return param_io(p, layer, id, const_cast<float*>(host), count, 0);
}
gp_status gp_get_param(gp_partition* p, int layer, int id, float* host, size_t count) {
    return param_io(p, layer, id, host, count, 1);
}
gp_status gp_get_grad(gp_partition* p, int layer, int id, float* host, size_t count) {
    return param_io(p, layer, id, host, count, 2);
}

gp_status gp_timer_select(gp_partition* p, int role) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    if (role < GP_K_NONE || role > GP_K_COUNT) return set_error(GP_ERR_INVALID_ARG, "timer role out of range");
    p->timer.selected = role;
    return GP_OK;
}

gp_status gp_timer_sample(gp_partition* p, int every) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    if (every < 1) return set_error(GP_ERR_INVALID_ARG, "timer sampling stride must be >= 1");
    p->timer.every = every;
    return GP_OK;
}

gp_status gp_timer_read(gp_partition* p, int role, double* ms, long* launches, double* flops, double* bytes) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    if (role <= GP_K_NONE || role >= GP_K_COUNT) return set_error(GP_ERR_INVALID_ARG, "timer role out of range");
    const auto& recs = p->timer.recs[role];
    double total = 0.0;
    if (!recs.empty()) GP_HIP(hipEventSynchronize(recs.back().second));
    for (const auto& pr : recs) {
        float t = 0.f;
        GP_HIP(hipEventElapsedTime(&t, pr.first, pr.second));
        total += t;
    }
    if (ms) *ms = total;
    if (launches) *launches = (long)recs.size();
    if (flops) *flops = p->timer.flops[role];
    if (bytes) *bytes = p->timer.bytes[role];
    return GP_OK;
}

gp_status gp_mfma_peak(void* stream, double* tflops) {
    if (!tflops) return set_error(GP_ERR_INVALID_ARG, "tflops must not be NULL");
    return mfma_peak(static_cast<hipStream_t>(stream), tflops);
}

gp_status gp_timer_reset(gp_partition* p) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    p->timer.reset();
    return GP_OK;
}

gp_status gp_partition_memory(gp_partition* p, size_t* params, size_t* grads, size_t* stash, size_t* workspace) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    if (!p->sched.configured()) return set_error(GP_ERR_STATE, "partition not configured");
    if (params) *params = p->bytes_params;
    if (grads) *grads = p->bytes_grads;
    if (stash) *stash = p->bytes_stash;
    if (workspace) *workspace = p->bytes_ws;
    return GP_OK;
}

gp_status gp_param_count(gp_partition* p, size_t* count) {
    if (!p || !count) return set_error(GP_ERR_INVALID_ARG, "partition and count must not be NULL");
    if (!p->sched.configured()) return set_error(GP_ERR_STATE, "partition not configured");
    *count = p->plan.count;
    return GP_OK;
}

gp_status gp_forward_microbatch(gp_partition* p, int mb, const void* x, const void* mem, void* y, gp_stream stream) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    std::string msg;
    gp_status s = p->sched.can_forward(mb, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    if (!x) return set_error(GP_ERR_INVALID_ARG, "x must not be NULL");
    const bool dec = p->g.kind == GP_DECODER_CROSS;
    if (dec && !mem) return set_error(GP_ERR_INVALID_ARG, "decoder partitions need the memory input");
    if (!dec && mem) return set_error(GP_ERR_INVALID_ARG, "encoder partitions take no memory input");
    const int lane = p->lane_of(mb);
    Ctx c = first_pass_ctx(p, (hipStream_t)stream, lane);
    GP_TRY(order_first_pass(p, c, false));
    const int set = p->g.keep_act ? p->set_of(mb) : 0;
    if (p->poison) {
        GP_TRY(poison_span(p, lane ? p->fpass[lane].splitk_span : p->splitk_span[0], c.st));
        if (p->g.keep_act) {
            GP_TRY(poison_set(p, set, c.st));
        } else {
            GP_TRY(poison_first_pass_slot(p, lane, c.st));
        }
    }
    const long T = p->g.T(), D = p->d.D;
    FirstPass& f = p->fpass[lane];
    GP_TRY(intake(c.dt, x, p->stash_x_mb(mb), p->g.keep_act ? p->xs[set][0] : f.xs[0], T * D, c.st));
    if (mem) GP_TRY(intake(c.dt, mem, p->stash_m_mb(mb), nullptr, p->g.Tm() * D, c.st));
    // The last micro-batch's backward comes first, so the recompute of its
    // unit starts on the recompute stream as soon as its boundary inputs are
    // stashed; the first pass runs in its own slot beside it.
    const bool early_on = p->remat_early && p->ahead();
    int lo = mb, cnt = 1;
    remat_unit(p, p->g.M - 1, lo, cnt);
    if (early_on && mb >= lo && mb < p->g.M - 1 && p->events()) {
        // a lower member of that unit: the early recompute reads its stash
        f.stashed = p->next_event();
        GP_HIP(hipEventRecord(f.stashed, c.st));
    }
    if (early_on && mb == p->g.M - 1) {
        const hipEvent_t fork = p->next_event();
        GP_HIP(hipEventRecord(fork, c.st));
        Ctx cr = make_ctx(p, p->remat, Lane::Remat);
        GP_HIP(hipStreamWaitEvent(cr.st, fork, 0));
        for (int m2 = lo; m2 < mb; ++m2) {
            const FirstPass& o = p->fpass[p->lane_of(m2)];
            GP_TRY(wait_recorded(cr.st, o.stream, o.stashed, o.capture));
        }
        GP_TRY(poison_span(p, p->splitk_span[2], cr.st));
        s = remat_pass(cr, lo, cnt);
        if (s != GP_OK) return s;
        p->remat_done = p->next_event();
        GP_HIP(hipEventRecord(p->remat_done, cr.st));
        p->remat_pending = lo;
    }
    // stored-activation mode: this micro-batch's intermediates stay in its own set
    s = partition_forward(c, mb, p->g.keep_act != 0, x, mem, y, set, true);
    if (s != GP_OK) return s;
    GP_TRY(record_first_pass(p, c));
    p->sched.did_forward();
    return GP_OK;
}

gp_status gp_forward_microbatch_noalloc(gp_partition* p, int mb, const void* x, const void* mem, void* y,
                                       gp_stream stream) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    std::string msg;
    gp_status s = p->sched.can_forward(mb, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    if (!x) return set_error(GP_ERR_INVALID_ARG, "x must not be NULL");
    const bool dec = p->g.kind == GP_DECODER_CROSS;
    if (dec && !mem) return set_error(GP_ERR_INVALID_ARG, "decoder partitions need the memory input");
    if (!dec && mem) return set_error(GP_ERR_INVALID_ARG, "encoder partitions take no memory input");
    if (!p->noalloc_scratch) return set_error(GP_ERR_HIP, p->noalloc_error.c_str());
    if ((size_t)p->fwd_ws_need > NOALLOC_SCRATCH_FLOATS) {
        const std::string m = "forward pass needs " + std::to_string(p->fwd_ws_need * 4 >> 20) +
                              " MiB of split-K scratch; the static scratch holds " +
                              std::to_string(NOALLOC_SCRATCH_FLOATS * 4 >> 20) + " MiB";
        return set_error(GP_ERR_UNSUPPORTED, m.c_str());
    }
    // Same tile and split choices as gp_forward_microbatch (the workspace size
    // the chooser sees is unchanged); the partials go to the static scratch,
    // so this pass also waits for the other slot's last forward (two of these
    // in flight would share the array).
    const int lane = p->lane_of(mb);
    Ctx c = first_pass_ctx(p, (hipStream_t)stream, lane);
    c.ws = p->noalloc_scratch;
    GP_TRY(order_first_pass(p, c, true));
    if (p->poison) {
        GP_TRY(poison_fill(p->noalloc_scratch, (size_t)p->fwd_ws_need * 4, c.st));
        if (p->g.keep_act) {
            GP_TRY(poison_set(p, p->set_of(mb), c.st));
        } else {
            GP_TRY(poison_first_pass_slot(p, lane, c.st));
        }
    }
    // No early recompute on the library's recompute stream: the backward of
    // the last micro-batch re-materialises it itself.
    if (p->g.keep_act)
        s = partition_forward(c, mb, true, x, mem, y, p->set_of(mb));
    else
        s = partition_forward(c, mb, false, x, mem, y);
    if (s != GP_OK) return s;
    GP_TRY(record_first_pass(p, c));
    p->sched.did_forward();
    return GP_OK;
}

gp_status gp_backward_microbatch_remat(gp_partition* p, int mb, const void* dy_or_target, void* dx, void* dmem,
                                       gp_stream stream) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    std::string msg;
    gp_status s = p->sched.can_backward(mb, msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    if (!dy_or_target) return set_error(GP_ERR_INVALID_ARG, "dy_or_target must not be NULL");
    const bool dec = p->g.kind == GP_DECODER_CROSS;
    if (!dec && dmem) return set_error(GP_ERR_INVALID_ARG, "encoder partitions have no memory gradient");
    const bool lanes = p->bwd_lanes > 1;
    const int bl = p->blane(mb);
    Ctx c = make_ctx(p, (hipStream_t)stream);
    c.last = mb == 0;
    if (bl) {
        c.bw = &p->bw1;
        c.ws = p->bw1.splitk;
        c.v16 = p->bw1.v16_main;
    }
    Ctx cs = make_ctx(p, p->side, Lane::Side);
    const bool side = p->use_side && p->side;
    const bool first = p->sched.first_backward();
    const long T = p->g.T(), D = p->d.D;
    const int set = p->set_of(mb);
    if (first) {
        // every forward of the mini-batch, on whatever stream, precedes its backward
        for (FirstPass& f : p->fpass) {
            GP_TRY(wait_recorded(c.st, f.stream, f.done, f.capture));
            f.done = f.stashed = nullptr;
        }
    }
    // The backward of a unit's highest micro-batch (which comes first) needs
    // the unit re-materialised; the unit's other member then finds it done.
    int lo = mb, cnt = 1;
    remat_unit(p, mb, lo, cnt);
    const bool unit_first = mb == lo + cnt - 1;
    // The previous call in this lane (with one lane: the previous backward
    // call, whatever stream it was given); with two lanes a unit's first call
    // also waits for the previous unit's last call, which waited for that
    // unit's weight gradients (they read the grouped rows this unit rewrites,
    // and the recompute-ahead forked below rebuilds their sets).
    GP_TRY(wait_recorded(c.st, p->lane_stream[bl], p->lane_end[bl], p->lane_capture[bl]));
    if (lanes && unit_first)
        GP_TRY(wait_recorded(c.st, p->lane_stream[bl ^ 1], p->lane_end[bl ^ 1], p->lane_capture[bl ^ 1]));
    if (p->poison) {
        const Span* sk_side = lanes ? nullptr : &p->splitk_span[1];  // lanes: poisoned on the side stream
        const Span* own_bwd = bl ? &p->bwd1_span : &p->bwd_span;
        const Span* own_sk = bl ? &p->splitk1_span : &p->splitk_span[0];
        const Span* own_loss = bl ? &p->loss1_span : &p->loss_span;
        const Span* own_head = bl ? &p->head1_span : &p->head_span;
        for (const Span* sp : {own_bwd, own_sk, sk_side, own_loss, own_head})
            if (sp) GP_TRY(poison_span(p, *sp, c.st));
        // this micro-batch's rows of the grouped weight-gradient operands (the
        // other members' rows may hold later micro-batches, not yet consumed)
        if (p->group > 1)
            for (const Span& sp : p->dys_span[mb % p->group]) GP_TRY(poison_span(p, sp, c.st));
        if (first) {
            // overwritten (not accumulated into) by the first backward micro-batch
            GP_TRY(poison_span(p, p->lnpart_span, c.st));
            GP_TRY(poison_span(p, p->loss_acc_span, c.st));
            GP_TRY(poison_fill(p->grads, p->plan.n32 * 4, c.st));
        }
    }
    // Everything this call's stream is ordered after so far (all forwards,
    // the previous units' backwards, which read the other workspace sets, and
    // their weight gradients) precedes a recompute-ahead launched from this
    // call.
    hipEvent_t remat_fork = nullptr;
    const bool ahead = p->ahead() && !p->g.keep_act && unit_first && lo > 0;
    if (ahead) {
        remat_fork = p->next_event();
        GP_HIP(hipEventRecord(remat_fork, c.st));
    }
    // re-materialise the unit's forward from the stash, unless an earlier call
    // already did so on the recompute stream
    if (p->g.keep_act || !unit_first) {
        // the forward kept every intermediate (stored-activation mode), or the
        // unit's first backward had it recomputed
        if (lanes && !unit_first)
            GP_TRY(wait_recorded(c.st, p->unit_ready_stream, p->unit_ready, p->unit_ready_capture));
    } else if (p->remat_pending == lo) {
        GP_HIP(hipStreamWaitEvent(c.st, p->remat_done, 0));
        p->remat_pending = -1;
    } else {
        s = remat_pass(c, lo, cnt);
        if (s != GP_OK) return s;
    }
    if (lanes && unit_first && cnt > 1) {
        p->unit_ready = p->next_event();
        GP_HIP(hipEventRecord(p->unit_ready, c.st));
        p->unit_ready_stream = c.st;
        p->unit_ready_capture = capture_of(c.st);
    }
    // lanes: the unit's first call records the end of each layer; its other
    // member follows it layer by layer
    const bool record_hi = lanes && unit_first && cnt > 1;
    if (lanes && !unit_first) c.ln_gate = p->hi_ev.data();
    if (ahead) {
        // re-materialise the next unit (the micro-batches below) meanwhile
        // (GPipe, Section 2.3: the recompute can be scheduled earlier)
        Ctx cr = make_ctx(p, p->remat, Lane::Remat);
        GP_HIP(hipStreamWaitEvent(cr.st, remat_fork, 0));
        GP_TRY(poison_span(p, p->splitk_span[2], cr.st));
        int lo2 = 0, cnt2 = 1;
        remat_unit(p, lo - 1, lo2, cnt2);
        s = remat_pass(cr, lo2, cnt2);
        if (s != GP_OK) return s;
        p->remat_done = p->next_event();
        GP_HIP(hipEventRecord(p->remat_done, cr.st));
        p->remat_pending = lo2;
    }
    BwdWs& b = bl ? p->bw1 : p->bw;
    // dL/dy of the partition output into (p32, top): top is the ring's first
    // buffer, or with grouped weight gradients this micro-batch's rows of the
    // last layer's incoming-gradient buffer
    const bool pr = p->group > 1;
    const int half = pr ? mb % p->group : 0;
    void* top = pr ? p->off_elt(p->dys[p->d.L - 1].gin, (long)half * T * D) : b.ring[0];
    // lanes: the loss sum and the head's gradient accumulate in micro-batch order
    const bool head_order = lanes && p->g.loss != GP_LOSS_NONE;
    if (head_order && !unit_first) GP_HIP(hipStreamWaitEvent(c.st, p->head_ev, 0));
    if (p->g.loss == GP_LOSS_NONE) {
        s = intake(c.dt, dy_or_target, top, b.p32, T * D, c.st);
    } else if (p->g.loss == GP_LOSS_MSE) {
        int nb = 0;
        const double norm = (double)p->g.n * p->g.M * p->g.S * D;
        s = mse_grad(c.dt, p->xs[set][p->d.L], dy_or_target, T * D, norm, b.p32, top, b.loss_partial, &nb, c.st);
        if (s == GP_OK) s = loss_finalize(b.loss_partial, nb, b.loss_acc, first ? 0 : 1, c.st);
    } else {
        s = head_backward(c, set, first, reinterpret_cast<const int*>(dy_or_target), top);
    }
    if (s != GP_OK) return s;
    if (head_order && record_hi) {
        p->head_ev = p->next_event();
        GP_HIP(hipEventRecord(p->head_ev, c.st));
    }
    const void* mem_m = dec ? p->stash_m_mb(mb) : nullptr;
    // Layer l's weight-gradient GEMMs run on the side stream while layer l - 1
    // is processed.  Without grouping, layer l - 2 rewrites parity and ring
    // buffers that layer l's GEMMs read, so it first waits for them
    // (side_done[l % 4]); the grouped buffers are per layer.
    // With grouping the higher members of a group (whose backwards come first)
    // leave their weight gradients to the lowest one, which runs each as one
    // GEMM over all the members' rows.  The first weight-gradient GEMMs of the
    // mini-batch overwrite the accumulators.
    if (first) p->dw_started = false;
    const bool run_dw = p->launches_dw(mb);
    const int dw_acc = p->dw_started ? 1 : 0;
    const long dw_rows = pr ? p->group_size(mb) : 1;
    float* in32 = b.p32;
    void* ine = top;
    float* sc32 = b.q32;
    int ri = 1;
    std::vector<DwJob> jobs;
    hipEvent_t last_done = nullptr;  // latest side-stream event of this call
    PendingRes pend;                 // a dX GEMM's split-K reduce left to the next LayerNorm backward
    Ctx cb = c;
    cb.pend = &pend;
    auto fail = [&](gp_status st) {
        if (last_done) (void)hipStreamWaitEvent(c.st, last_done, 0);
        return st;
    };
    for (int l = p->d.L - 1; l >= 0; --l) {
        if (side && !pr && l + 2 <= p->d.L - 1) GP_HIP(hipStreamWaitEvent(c.st, p->side_done[(l + 2) % 4], 0));
        float* out32 = nullptr;
        void* oute = nullptr;
        jobs.clear();
        // launch the collected weight-gradient GEMMs (after everything enqueued on main so far)
        auto flush = [&](int level) -> gp_status {
            if (!run_dw) jobs.clear();  // the group's lowest member runs them
            if (jobs.empty() || level < p->dw_flush) return GP_OK;
            if (side) {
                const hipEvent_t fork = p->next_event();
                GP_HIP(hipEventRecord(fork, c.st));
                GP_HIP(hipStreamWaitEvent(cs.st, fork, 0));
                // lanes: the group's other member's rows of layer l
                if (c.ln_gate) GP_HIP(hipStreamWaitEvent(cs.st, c.ln_gate[l], 0));
                if (lanes) GP_TRY(poison_span(p, p->splitk_span[1], cs.st));
            }
            for (const DwJob& j : jobs)
                GP_TRY(linear_dw(side ? cs : cb, *j.L, j.X, j.dY, j.rows * dw_rows, dw_acc));
            jobs.clear();
            return GP_OK;
        };
        s = layer_backward(cb, set, half, l, first, in32, ine, sc32, ri, out32, oute, nullptr, l == 0 ? dx : nullptr,
                           mem_m, jobs, flush);
        if (s == GP_OK) s = flush(2);
        if (s != GP_OK) return fail(s);
        if (side && (run_dw || !lanes)) {
            p->side_done[l % 4] = p->next_event();
            GP_HIP(hipEventRecord(p->side_done[l % 4], cs.st));
            last_done = p->side_done[l % 4];
        }
        if (record_hi) {
            p->hi_ev[l] = p->next_event();
            GP_HIP(hipEventRecord(p->hi_ev[l], c.st));
        }
        if (c.last && p->remat && p->layer_update) {
            p->lay_main[l] = p->next_event();
            GP_HIP(hipEventRecord(p->lay_main[l], c.st));
            p->lay_side[l] = side ? p->side_done[l % 4] : nullptr;
        }
        if (l > 0) {
            sc32 = (out32 == b.p32) ? b.q32 : b.p32;
            in32 = out32;
            ine = oute;
        }
    }
    if (s == GP_OK) s = flush_pending(cb);
    if (s != GP_OK) return fail(s);
    if (run_dw) p->dw_started = true;
    p->lay_ready = p->layer_update && c.last && p->remat && side && run_dw;
    // the caller's stream resumes only after the last weight-gradient GEMM
    // (lanes: the one of the call that launched them; the other member's
    // next call waits for that call)
    if (side && (run_dw || !lanes)) GP_HIP(hipStreamWaitEvent(c.st, p->side_done[0], 0));
    if (dec && dmem) {
        s = cast_out(c.dt, b.dmem32, dmem, p->g.Tm() * D, c.st);
        if (s != GP_OK) return s;
    }
    if (p->events()) {
        p->lane_end[bl] = p->next_event();
        GP_HIP(hipEventRecord(p->lane_end[bl], c.st));
        p->lane_stream[bl] = c.st;
        p->lane_capture[bl] = capture_of(c.st);
    }
    p->sched.did_backward();
    return GP_OK;
}

gp_status gp_stream_create(gp_stream* out) {
    if (!out) return set_error(GP_ERR_INVALID_ARG, "out must not be NULL");
    hipStream_t st = nullptr;
    GP_HIP(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));  // default priority
    *out = st;
    return GP_OK;
}

gp_status gp_stream_destroy(gp_stream stream) {
    if (!stream) return set_error(GP_ERR_INVALID_ARG, "stream must not be NULL");
    GP_HIP(hipStreamDestroy((hipStream_t)stream));
    return GP_OK;
}

gp_status gp_recomputed_output(gp_partition* p, void* y, gp_stream stream) {
    if (!p || !y) return set_error(GP_ERR_INVALID_ARG, "partition and y must not be NULL");
    if (!p->sched.configured()) return set_error(GP_ERR_STATE, "partition not configured");
    const int mb = p->sched.last_backward();
    if (mb < 0) return set_error(GP_ERR_STATE, "no backward micro-batch has run in this mini-batch");
    const int set = p->set_of(mb);
    return cast_out(p->g.dtype, p->xs[set][p->d.L], y, p->g.T() * p->d.D, (hipStream_t)stream);
}

gp_status gp_accumulate_and_step(gp_partition* p, float lr, double* loss_out, gp_stream stream) {
    if (!p) return set_error(GP_ERR_INVALID_ARG, "partition must not be NULL");
    std::string msg;
    gp_status s = p->sched.can_step(msg);
    if (s != GP_OK) return set_error(s, msg.c_str());
    hipStream_t st = (hipStream_t)stream;
    const int dt = p->g.dtype;
    // both backward lanes' last calls (their weight gradients included)
    for (int ln = 0; ln < 2; ++ln) {
        GP_TRY(wait_recorded(st, p->lane_stream[ln], p->lane_end[ln], p->lane_capture[ln]));
        p->lane_end[ln] = nullptr;
    }
    // Labels outside [0, V) were read as class 0 and flagged on the device; a
    // step that synchronises anyway reports them and skips the update.
    if (p->g.loss == GP_LOSS_XENT_LS && (loss_out || p->g.check_finite)) {
        int bad = 0;
        GP_HIP(hipMemcpyAsync(&bad, p->bw.bad_label, sizeof(int), hipMemcpyDeviceToHost, st));
        GP_HIP(hipStreamSynchronize(st));
        if (bad) {
            GP_HIP(hipMemsetAsync(p->bw.bad_label, 0, sizeof(int), st));
            p->sched.did_step();
            return set_error(GP_ERR_INVALID_ARG, "a label was outside [0, vocab): update skipped");
        }
    }
    if (p->g.check_finite) {
        GP_HIP(hipMemsetAsync(p->bw.flag, 0, sizeof(int), st));
        GP_TRY(finite_check(p->grads, (long)p->plan.n32, p->bw.flag, st));
        int flag = 0;
        GP_HIP(hipMemcpyAsync(&flag, p->bw.flag, sizeof(int), hipMemcpyDeviceToHost, st));
        GP_HIP(hipStreamSynchronize(st));
        if (flag) {
            p->sched.did_step();
            return set_error(GP_ERR_NONFINITE, "non-finite gradient: update skipped");
        }
    }
    const bool rms = p->g.optimizer == GP_OPT_RMSPROP;
    auto update_linear = [&](const Linear* l, hipStream_t us) {
        return update_refresh_linear(p->master + l->w, p->grads + l->w, rms ? p->opt_ms + l->w : nullptr, lr,
                                     p->g.rms_decay, p->g.rms_eps, l->in, l->out, p->W(l->kn), p->W(l->nk),
                                     l->split ? p->W(l->q4) : nullptr, l->split ? p->W(l->q4s) : nullptr, us,
                                     l->f16);
    };
    if (p->fused_update && p->lay_ready) {
        // each layer's linears as soon as the last backward is past that layer
        // (top layer first, as the backward goes), then the head's linear, the
        // biases and LayerNorm parameters on the caller's stream
        const hipStream_t us = p->remat;
        const int L = p->d.L;
        for (int l = L - 1; l >= 0; --l) {
            GP_HIP(hipStreamWaitEvent(us, p->lay_main[l], 0));
            if (p->lay_side[l]) GP_HIP(hipStreamWaitEvent(us, p->lay_side[l], 0));
            const LayerPlan& P = p->plan.layers[l];
            for (const Linear* x : {&P.qkv, &P.o, &P.ffn1, &P.ffn2, &P.xq, &P.xkv, &P.xo})
                if (x->present) GP_TRY(update_linear(x, us));
        }
        const hipEvent_t upd = p->next_event();
        GP_HIP(hipEventRecord(upd, us));
        GP_HIP(hipStreamWaitEvent(st, upd, 0));
        if (p->plan.head.out.present) GP_TRY(update_linear(&p->plan.head.out, st));
        GP_TRY(update_ranges(p->master, p->grads, rms ? p->opt_ms : nullptr, lr, p->g.rms_decay, p->g.rms_eps,
                             p->upd_ranges, p->n_upd_ranges, st));
    } else if (p->fused_update) {
        // one pass over each linear's W and G that also rewrites its working
        // copies, then the biases and LayerNorm parameters
        for (const Linear* l : p->plan.linears()) GP_TRY(update_linear(l, st));
        GP_TRY(update_ranges(p->master, p->grads, rms ? p->opt_ms : nullptr, lr, p->g.rms_decay, p->g.rms_eps,
                             p->upd_ranges, p->n_upd_ranges, st));
    } else {
        if (rms)
            GP_TRY(rmsprop_update(p->master, p->grads, p->opt_ms, lr, p->g.rms_decay, p->g.rms_eps,
                                  (long)p->plan.n32, st));
        else
            GP_TRY(sgd_update(p->master, p->grads, lr, (long)p->plan.n32, st));
        for (const Linear* l : p->plan.linears())
            GP_TRY(refresh_linear(dt, p->master + l->w, l->in, l->out, p->W(l->kn), p->W(l->nk),
                                  l->split ? p->W(l->q4) : nullptr, l->split ? p->W(l->q4s) : nullptr, st, l->f16));
    }
    if (loss_out) {
        double v = 0.0;
        if (p->g.loss != GP_LOSS_NONE)
            GP_HIP(hipMemcpyAsync(&v, p->bw.loss_acc, sizeof(double), hipMemcpyDeviceToHost, st));
        GP_HIP(hipStreamSynchronize(st));
        *loss_out = v;
    }
    p->lay_ready = false;
    if (p->events()) {
        p->tail_done = p->next_event();
        GP_HIP(hipEventRecord(p->tail_done, st));
        p->tail_stream = st;
        p->tail_capture = capture_of(st);
    }
    p->sched.did_step();
    return GP_OK;
}

} // extern "C"
