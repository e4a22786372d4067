// C ABI of the MoE layer library: argument validation, workspace layout and
// the launch sequence of each entry point.  Pure host code; every kernel is
// enqueued on the caller's stream and nothing here synchronises.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>

#include "../../include/moe.h"
#include "kernels.h"

namespace {

constexpr size_t ALIGN = 256;

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// Byte offsets of every workspace region; depends only on the shape and, for
// bounded-memory execution, on the ring size.  The prefix (error word, plan
// scratch, W_r^T, position tables, zero page) is the same in every layout,
// so moe_route and moe_plan work with any of them.
struct Layout {
    size_t err, blockcounts, blockbase, blockflags, wrt, rpart, rowidx, wperm, zeros, fused;
    size_t prefix_total;
    size_t acc, coff;          // ring only: fp32 per-token accumulator, window regions
    size_t A, B, H, Yexp, As, Bs, Hs, Ysh;
    size_t fwd_total;
    size_t dA, dB, Hw, dgpart, dg, dZ, dXperm, dAs, dBs, dXsh, dwr_part, dzs, wrs, xtt;
    size_t dytt;
    long xt_ld;
    size_t bwd_total;
    size_t xq, xs, hq, hsc;   // MXFP8 forward: quantised X and H (over the backward regions)
    size_t mx_total;
    size_t dyq, dys, daq, das, dbq, dbs;   // MXFP8 backward: quantised dY, dA, dB
    size_t a32, b32;                       // MXFP8: the fp32 pre-activations kept for the backward
    size_t mxb_total;
    // MXFP8 weight gradients: padded expert offsets and the token-axis codes
    // and scales of X, dY, dA, dB and w h, [C][tpad] and [C][tpad / 32]
    size_t poff, xt, xts, dyt, dyts, dat, dats, dbt, dbts, hwt, hwts;
    size_t da32, db32, hw32;   // their fp32 sources dA, dB, w h (plan order)
    size_t mxw_total;
    long tpad;                 // their row pitch: the padded token positions' bound
    long act_rows;             // rows of the per-route activation buffers
    int dg_parts;
};

// ring_rows < 0: per-route activations for all T*k routes; otherwise a ring
// of ring_rows rows (bounded-memory execution).
Layout make_layout(const moe_shape &s, long ring_rows = -1) {
    const size_t T = s.T, d = s.d, E = s.E, f = s.f, fs = s.f_shared;
    const size_t R = T * (size_t)s.k;
    const size_t nb = (size_t)plan_nblocks((long)R);
    const size_t epad = (size_t)route_epad((int)E);
    const size_t Ra = ring_rows < 0 ? R : (size_t)ring_rows;
    Layout L{};
    L.act_rows = (long)Ra;
    size_t o = 0;
    auto take = [&](size_t bytes) { const size_t at = o; o += up(bytes > 0 ? bytes : 1); return at; };
    L.err = take(4);
    L.blockcounts = take(nb * E * 4);
    L.blockbase = take(nb * E * 4);
    L.blockflags = take(nb * 4);
    L.wrt = take(epad * d * 2);
    L.rpart = take(route_part_bytes((long)T, (int)d, (int)E));
    L.rowidx = take(R * 4);
    L.wperm = take(R * 4);
    L.zeros = take(ZERO_PAGE_ELEMS * 2);
    L.fused = take((size_t)fused_counter_ints((long)T, (long)R, (int)E) * 4);
    L.prefix_total = o;
    if (ring_rows >= 0) {
        L.acc = take(T * d * 4);
        L.coff = take(2 * (E + 1) * 4);
    }
    L.A = take(Ra * f * 2);
    L.B = take(Ra * f * 2);
    L.H = take(Ra * f * 2);
    L.Yexp = take(Ra * d * 2);
    L.As = take(T * fs * 2);
    L.Bs = take(T * fs * 2);
    L.Hs = take(T * fs * 2);
    L.Ysh = take(T * d * 2);
    L.fwd_total = o;
    L.dg_parts = (int)(f / (size_t)gemm_tile_n());
    L.dA = take(Ra * f * 2);
    L.Hw = take(Ra * f * 2);
    L.dB = take(Ra * f * 2);
    L.dgpart = take(R * (size_t)L.dg_parts * 4);
    L.dg = take(R * 4);
    L.dZ = take(T * E * 4);
    L.dXperm = take(Ra * d * 2);
    L.dAs = take(T * fs * 2);
    L.dBs = take(T * fs * 2);
    L.dXsh = take(T * d * 2);
    L.dwr_part = take((size_t)dwr_nchunks((long)T) * d * E * 4);
    L.dzs = take(T * 64 * 2);   // dense routing: router-term rows of dX
    L.wrs = take(d * 64 * 2);
    // X^T and dY^T rows: the tokens rounded up to a K step, plus one more
    // (zero) K step, so a window of the bounded-memory backward that starts
    // mid-expert (an unaligned first column) still reads inside the row
    L.xt_ld = (long)((T + 63) / 64 * 64 + 64);
    L.xtt = take(s.k == s.E ? d * (size_t)L.xt_ld * 2 : 0);   // dense routing: X^T [d][xt_ld]
    L.dytt = take(s.k == s.E ? d * (size_t)L.xt_ld * 2 : 0);  // dense routing: dY^T likewise
    L.bwd_total = o;
    o = L.fwd_total;
    L.xq = take(T * d);
    L.xs = take(T * d / 32);
    L.hq = take(R * f);
    L.hsc = take(R * f / 32);
    L.mx_total = o;
    o = L.bwd_total;
    L.dyq = take(T * d);
    L.dys = take(T * d / 32);
    L.daq = take(R * f);
    L.das = take(R * f / 32);
    L.dbq = take(R * f);
    L.dbs = take(R * f / 32);
    L.a32 = take(R * f * 4);
    L.b32 = take(R * f * 4);
    L.mxb_total = o;
    // each expert's rows padded to 128 positions: at most R + 127 E in all
    L.tpad = (long)((R + 128 * E + 127) / 128 * 128);
    const size_t P = (size_t)L.tpad;
    L.poff = take((E + 1) * 4);
    L.xt = take(d * P);
    L.xts = take(d * P / 32);
    L.dyt = take(d * P);
    L.dyts = take(d * P / 32);
    L.dat = take(f * P);
    L.dats = take(f * P / 32);
    L.dbt = take(f * P);
    L.dbts = take(f * P / 32);
    L.hwt = take(f * P);
    L.hwts = take(f * P / 32);
    L.da32 = take(R * f * 4);
    L.db32 = take(R * f * 4);
    L.hw32 = take(R * f * 4);
    L.mxw_total = o;
    return L;
}

bool aligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool ptr_ok(const void *p) { return p != nullptr && aligned(p); }
bool opt_ok(const void *p) { return p == nullptr || aligned(p); }

moe_status check_shape(const moe_shape *s) {
    if (!s) return MOE_EINVAL;
    if (s->T < 0 || s->d <= 0 || s->E <= 0 || s->k <= 0 || s->f <= 0 || s->f_shared < 0)
        return MOE_EINVAL;
    if (s->k > s->E) return MOE_EINVAL;
    if (s->d % 256 || s->f % 256 || s->f_shared % 256) return MOE_EUNSUPPORTED;
    if (s->k > 16 || s->E > 256) return MOE_EUNSUPPORTED;
    if (s->T * s->k >= (int64_t(1) << 31)) return MOE_EUNSUPPORTED;
    if (s->d > (int64_t(1) << 20) || s->f > (int64_t(1) << 20) || s->f_shared > (int64_t(1) << 20))
        return MOE_EUNSUPPORTED;
    return MOE_OK;
}

moe_status check_weights(const moe_shape *s, const moe_weights *w) {
    if (!w) return MOE_EINVAL;
    if (!ptr_ok(w->W_gate) || !ptr_ok(w->W_up) || !ptr_ok(w->W_down)) return MOE_EINVAL;
    const bool shared = s->f_shared > 0;
    const bool any = w->Wg_s || w->Wu_s || w->Wd_s;
    if (shared) {
        if (!ptr_ok(w->Wg_s) || !ptr_ok(w->Wu_s) || !ptr_ok(w->Wd_s)) return MOE_EINVAL;
    } else if (any) {
        return MOE_EINVAL;
    }
    return MOE_OK;
}

moe_status check_plan(const moe_plan_bufs *p) {
    if (!p) return MOE_EINVAL;
    if (!ptr_ok(p->counts) || !ptr_ok(p->offsets) || !ptr_ok(p->perm) || !ptr_ok(p->route_pos))
        return MOE_EINVAL;
    return MOE_OK;
}

moe_status check_ws(const moe_shape *s, const void *ws, size_t ws_bytes, int with_backward) {
    if (!ptr_ok(ws)) return MOE_EINVAL;
    const Layout L = make_layout(*s);
    if (ws_bytes < (with_backward ? L.bwd_total : L.fwd_total)) return MOE_ENOSPACE;
    return MOE_OK;
}

// moe_route and moe_plan touch only the layout prefix.
moe_status check_ws_prefix(const moe_shape *s, const void *ws, size_t ws_bytes) {
    if (!ptr_ok(ws)) return MOE_EINVAL;
    if (ws_bytes < make_layout(*s).prefix_total) return MOE_ENOSPACE;
    return MOE_OK;
}

// Multi-rank schedule: validation and workspace (error word, per-chunk
// flags, per-(row, chunk, expert) counts that become ordinal bases).
moe_status check_schedule_dims(int64_t R, int64_t NK, int64_t L, int64_t c) {
    if (R <= 0 || L <= 0 || NK < 0 || c < 0 || c >= R) return MOE_EINVAL;
    if (R > 1024 || L > 256) return MOE_EUNSUPPORTED;
    if (L * sched_rpad((int)R) > SCHED_MAX_TABLE) return MOE_EUNSUPPORTED;
    if (R * NK >= (int64_t(1) << 31)) return MOE_EUNSUPPORTED;
    return MOE_OK;
}

struct SchedLayout {
    size_t err, flags, counts, total;
};

SchedLayout schedule_layout(int64_t R, int64_t NK, int64_t L) {
    const size_t C = (size_t)sched_nchunks((long)NK);
    SchedLayout SL{};
    size_t o = 0;
    auto take = [&](size_t bytes) { const size_t at = o; o += up(bytes > 0 ? bytes : 1); return at; };
    SL.err = take(4);
    SL.flags = take((size_t)R * C * 4);
    SL.counts = take((size_t)R * C * (size_t)L * 4);
    SL.total = o;
    return SL;
}

template <typename T>
T *at(void *ws, size_t off) { return reinterpret_cast<T *>(static_cast<char *>(ws) + off); }

// Plan scratch of moe_plan_noalloc: a device array the library owns, one
// copy per GPU, held until the process ends.  In host code `scratch` is only
// a stand-in for the symbol: its device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is ever handed to a kernel.
constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(MOE_PLAN_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) uint8_t scratch[NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void *scratch_ptr[MAX_DEVICES] = {};

// The current device's copy of `scratch` (nullptr if its address cannot be had).
void *device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        scratch_ptr[dev] = p;
    }
    return scratch_ptr[dev];
}

// Bytes of plan scratch for R routes over E experts (per-chunk histograms,
// their scanned bases and flags, each region 256-byte aligned).
size_t plan_scratch_bytes(long R, long E) {
    const size_t nb = (size_t)plan_nblocks(R);
    return 2 * up(nb * (size_t)E * 4) + up(nb * 4 > 0 ? nb * 4 : 1);
}

// MXFP8 path: every fp8 operand is addressed with 32-bit offsets.
moe_status check_mx_shape(const moe_shape *s) {
    const int64_t lim = int64_t(1) << 32;
    if (s->T * s->d >= lim || s->T * s->k * s->f >= lim || s->E * s->f * s->d >= lim)
        return MOE_EUNSUPPORTED;
    return MOE_OK;
}

// MXFP8 weight gradients: their token-axis operands too.
moe_status check_mx_wgrad_shape(const moe_shape *s) {
    const int64_t lim = int64_t(1) << 32;
    const int64_t tpad = (s->T * s->k + 128 * s->E + 127) / 128 * 128;
    if (s->d * tpad >= lim || s->f * tpad >= lim) return MOE_EUNSUPPORTED;
    return MOE_OK;
}

moe_status check_mx_weights(const moe_shape *s, const moe_weights *w, const moe_mx_weights *q) {
    if (!w || !q) return MOE_EINVAL;
    if (!ptr_ok(q->Wg_q) || !ptr_ok(q->Wu_q) || !ptr_ok(q->Wd_q) || !ptr_ok(q->Wg_s) ||
        !ptr_ok(q->Wu_s) || !ptr_ok(q->Wd_s))
        return MOE_EINVAL;
    const bool any = w->Wg_s || w->Wu_s || w->Wd_s;
    if (s->f_shared > 0) {
        if (!ptr_ok(w->Wg_s) || !ptr_ok(w->Wu_s) || !ptr_ok(w->Wd_s)) return MOE_EINVAL;
    } else if (any) {
        return MOE_EINVAL;
    }
    return MOE_OK;
}

// Records stage event i (if requested) on the stream.
struct StageMarks {
    const moe_stage_events *ev;
    hipStream_t s;
    hipError_t mark(int i) const {
        if (!ev || i >= MOE_MAX_STAGE_EVENTS || !ev->ev[i]) return hipSuccess;
        return hipEventRecord(static_cast<hipEvent_t>(ev->ev[i]), s);
    }
};

#define MOE_TRY(expr)                                      \
    do {                                                   \
        if ((expr) != hipSuccess) return MOE_EHIP;         \
    } while (0)

// Shared expert (BF16 in both precisions): up/gate + SwiGLU into Hs, then
// down into Ysh.
GemmArgs shared_up_args(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                        const moe_weights *w, bool save) {
    const int T = (int)sh.T, d = (int)sh.d, fs = (int)sh.f_shared;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = X; g.lda = d; g.a_nrows = T > 0 ? T : 1; g.M = T;
    g.B = w->Wg_s; g.B2 = w->Wu_s; g.ldb = fs;
    g.N = fs; g.K = d;
    g.C = at<uint16_t>(ws, L.Hs); g.ldc = fs;
    if (save) { g.C2 = at<uint16_t>(ws, L.As); g.C3 = at<uint16_t>(ws, L.Bs); }
    return g;
}

hipError_t shared_up(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                     const moe_weights *w, bool save, hipStream_t s) {
    return launch_gemm_fwd_up(shared_up_args(sh, L, ws, X, w, save), sh.T, 1, s);
}

GemmArgs shared_down_args(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w) {
    const int T = (int)sh.T, d = (int)sh.d, fs = (int)sh.f_shared;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = at<uint16_t>(ws, L.Hs); g.lda = fs; g.a_nrows = T > 0 ? T : 1; g.M = T;
    g.B = w->Wd_s; g.ldb = d;
    g.N = d; g.K = fs;
    g.C = at<uint16_t>(ws, L.Ysh); g.ldc = d;
    return g;
}

hipError_t shared_down(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                       hipStream_t s) {
    return launch_gemm_fwd_down(shared_down_args(sh, L, ws, w), sh.T, 1, s);
}

// Dense routing (k == E): every token routes to every local expert (see
// down_cmb_args).  Expert e's plan rows are then the tokens in order, so in
// any window that starts at position 0 (its regions start where the plan's
// do) a gathered row is the position minus the region's start.
bool dense_routing(const moe_shape &sh) { return sh.k == sh.E; }

// Positions [w0, w1) of the routed buffer, with the expert regions clipped
// to it.  Per-route activation rows live at row p - w0 of their region, so
// kernels keep indexing by the global position p through a shifted base.
// The one-pass path is the single window [0, T k) with the plan's offsets.
struct Window {
    const int *offs;
    int w0, w1;
    template <class T> T *rows(void *ws, size_t region, long ld) const {
        return at<T>(ws, region) - (long)w0 * ld;
    }
    int span() const { return w1 > 1 ? w1 : 1; }   // clamp bound of position-indexed rows
    long count() const { return (long)w1 - w0; }
};

// Routed up/gate + SwiGLU over a window: H (optional) and, for the backward,
// the pre-activations A and B.
GemmArgs up_args(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                 const moe_weights *w, const Window &win, bool keep_h, bool save) {
    const int T = (int)sh.T, d = (int)sh.d, f = (int)sh.f;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = X; g.lda = d; g.a_rows = at<int>(ws, L.rowidx); g.a_nrows = T > 0 ? T : 1;
    g.B = w->W_gate; g.B2 = w->W_up; g.ldb = f; g.b_estride = (long)d * f;
    g.N = f; g.K = d; g.offsets = win.offs; g.E = (int)sh.E;
    if (keep_h) g.C = win.rows<uint16_t>(ws, L.H, f);
    g.ldc = f;
    if (save) { g.C2 = win.rows<uint16_t>(ws, L.A, f); g.C3 = win.rows<uint16_t>(ws, L.B, f); }
    return g;
}

hipError_t routed_up(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                     const moe_weights *w, const Window &win, bool keep_h, bool save, hipStream_t s) {
    return launch_gemm_fwd_up(up_args(sh, L, ws, X, w, win, keep_h, save), win.count(), (int)sh.E, s);
}

GemmArgs down_args(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                   const Window &win) {
    const int d = (int)sh.d, f = (int)sh.f;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = win.rows<uint16_t>(ws, L.H, f); g.lda = f; g.a_nrows = win.span();
    g.B = w->W_down; g.ldb = d; g.b_estride = (long)f * d;
    g.N = d; g.K = f; g.offsets = win.offs; g.E = (int)sh.E;
    g.C = win.rows<uint16_t>(ws, L.Yexp, d); g.ldc = d;
    return g;
}

hipError_t routed_down(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                       const Window &win, hipStream_t s) {
    return launch_gemm_fwd_down(down_args(sh, L, ws, w, win), win.count(), (int)sh.E, s);
}

// dh' = dY W_down^T with the SwiGLU backward and the dg partials.
hipError_t routed_dgrad(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *dY,
                        const moe_weights *w, const Window &win, hipStream_t s) {
    const int T = (int)sh.T, d = (int)sh.d, f = (int)sh.f;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = dY; g.lda = d; g.a_rows = at<int>(ws, L.rowidx); g.a_nrows = T > 0 ? T : 1;
    g.B = w->W_down; g.ldb = d; g.b_estride = (long)f * d;
    g.N = f; g.K = d; g.offsets = win.offs; g.E = (int)sh.E;
    g.E1 = win.rows<uint16_t>(ws, L.A, f); g.E2 = win.rows<uint16_t>(ws, L.B, f); g.ldc = f;
    g.rowscale = at<float>(ws, L.wperm);
    g.a_local = win.w0 == 0 && dense_routing(sh) ? 1 : 0;   // dY row = position - offsets[e]
    g.C = win.rows<uint16_t>(ws, L.dA, f); g.C2 = win.rows<uint16_t>(ws, L.dB, f);
    g.C3 = win.rows<uint16_t>(ws, L.Hw, f);
    g.dgpart = at<float>(ws, L.dgpart); g.dg_ld = L.dg_parts;
    return launch_gemm_bwd_dgrad(g, win.count(), (int)sh.E, s);
}

// dXperm = dA W_gate^T + dB W_up^T.
hipError_t routed_dx(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                     const Window &win, hipStream_t s) {
    const int d = (int)sh.d, f = (int)sh.f;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = win.rows<uint16_t>(ws, L.dA, f); g.A2 = win.rows<uint16_t>(ws, L.dB, f);
    g.lda = f; g.a_nrows = win.span();
    g.B = w->W_gate; g.B2 = w->W_up; g.ldb = f; g.b_estride = (long)d * f;
    g.N = d; g.K = f; g.offsets = win.offs; g.E = (int)sh.E;
    g.C = win.rows<uint16_t>(ws, L.dXperm, d); g.ldc = d;
    return launch_gemm_bwd_dx(g, win.count(), (int)sh.E, s);
}

// Weight gradients over the window's rows of each expert (added to the
// previous windows' sums when accumulate):
//   which 0: dW_gate[e] = Xperm_e^T dA_e   1: dW_up[e] = Xperm_e^T dB_e
//   which 2: dW_down[e] = (w H_e)^T dYperm_e
GemmArgs wgrad_args(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                    const moe_bf16 *dY, const moe_grads *gr, const Window &win, bool accumulate,
                    int which) {
    const int T = (int)sh.T, d = (int)sh.d, f = (int)sh.f;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.offsets = win.offs; g.E = (int)sh.E;
    g.accumulate = accumulate ? 1 : 0;
    const bool dense_rows = dense_routing(sh) && win.w0 == 0;   // rows = tokens in order
    if (which < 2) {
        g.A = X; g.lda = d; g.a_rows = at<int>(ws, L.rowidx); g.a_nrows = T > 0 ? T : 1;
        g.a_local = dense_rows ? 1 : 0;
        g.B = win.rows<uint16_t>(ws, which == 0 ? L.dA : L.dB, f); g.ldb = f; g.b_nrows = win.span();
        g.M = d; g.N = f;
        g.Cf = which == 0 ? gr->dW_gate : gr->dW_up; g.c_estride = (long)d * f; g.ldc = f;
    } else {
        g.A = win.rows<uint16_t>(ws, L.Hw, f); g.lda = f; g.a_nrows = win.span();
        g.B = dY; g.ldb = d; g.b_rows = at<int>(ws, L.rowidx); g.b_nrows = T > 0 ? T : 1;
        g.b_local = dense_rows ? 1 : 0;
        g.M = f; g.N = d;
        g.Cf = gr->dW_down; g.c_estride = (long)f * d; g.ldc = d;
    }
    return g;
}

// Dense routing: X^T and dY^T ([d][xt_ld], zero-padded), made once per
// backward.  The weight gradients of every expert (and of the shared expert)
// contract X and dY over the tokens in order, so they read them as
// K-contiguous rows instead of column tiles of 2d-byte rows.
hipError_t dense_transposes(const moe_shape &sh, const Layout &L, const moe_bf16 *X,
                            const moe_bf16 *dY, uint16_t *xt, uint16_t *dyt, hipStream_t s) {
    hipError_t e = launch_transpose_rows(X, (int)sh.T, (int)sh.d, xt, L.xt_ld, s);
    if (e != hipSuccess) return e;
    return launch_transpose_rows(dY, (int)sh.T, (int)sh.d, dyt, L.xt_ld, s);
}

// Routed weight gradients which0 .. which1 - 1 (0 dW_gate, 1 dW_up, 2 dW_down)
// of a one-pass backward with dense routing, on X^T / dY^T.
hipError_t dense_wgrads(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *X,
                        const moe_bf16 *dY, const moe_grads *gr, const int *offsets,
                        const uint16_t *xt, const uint16_t *dyt, int which0, int which1,
                        hipStream_t s) {
    const Window all{offsets, 0, (int)(sh.T * sh.k)};
    for (int which = which0; which < which1; ++which) {
        GemmArgs g = wgrad_args(sh, L, ws, X, dY, gr, all, false, which);
        hipError_t e;
        if (which < 2) {
            g.A = xt; g.lda = L.xt_ld; g.a_rows = nullptr; g.a_local = 1;
            e = launch_gemm_wgrad_t(g, (int)sh.E, s);
        } else {
            g.B = dyt; g.ldb = L.xt_ld; g.b_rows = nullptr; g.b_local = 1;
            e = launch_gemm_wgrad_tb(g, (int)sh.E, s);
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Shared-expert backward, in three parts: dAs/dBs (the gated-activation
// backward on the saved As, Bs), dXsh, and the three weight gradients.
hipError_t shared_dgrad(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *dY,
                        const moe_weights *w, hipStream_t s) {
    const int T = (int)sh.T, d = (int)sh.d, fs = (int)sh.f_shared;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = dY; g.lda = d; g.a_nrows = T > 0 ? T : 1; g.M = T;
    g.B = w->Wd_s; g.ldb = d;
    g.N = fs; g.K = d;
    g.E1 = at<uint16_t>(ws, L.As); g.E2 = at<uint16_t>(ws, L.Bs); g.ldc = fs;
    g.C = at<uint16_t>(ws, L.dAs); g.C2 = at<uint16_t>(ws, L.dBs);
    return launch_gemm_bwd_dgrad(g, T, 1, s);
}

hipError_t shared_dx(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                     hipStream_t s) {
    const int T = (int)sh.T, d = (int)sh.d, fs = (int)sh.f_shared;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = at<uint16_t>(ws, L.dAs); g.A2 = at<uint16_t>(ws, L.dBs); g.lda = fs;
    g.a_nrows = T > 0 ? T : 1; g.M = T;
    g.B = w->Wg_s; g.B2 = w->Wu_s; g.ldb = fs;
    g.N = d; g.K = fs;
    g.C = at<uint16_t>(ws, L.dXsh); g.ldc = d;
    return launch_gemm_bwd_dx(g, T, 1, s);
}

// xt, dyt: X^T and dY^T [d][L.xt_ld] when the caller made them (dense
// routing): the products then read them K-contiguous.
hipError_t shared_wgrads(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *dY,
                         const moe_bf16 *X, const moe_grads *gr, hipStream_t s,
                         const uint16_t *xt = nullptr, const uint16_t *dyt = nullptr) {
    const int T = (int)sh.T, d = (int)sh.d, fs = (int)sh.f_shared;
    const int Tn = T > 0 ? T : 1;
    hipError_t e;
    {
        GemmArgs g;
        g.zeros = at<uint16_t>(ws, L.zeros);
        g.A = X; g.lda = d; g.a_nrows = Tn;
        g.B = at<uint16_t>(ws, L.dAs); g.ldb = fs; g.b_nrows = Tn;
        g.M = d; g.N = fs; g.K = T;
        g.Cf = gr->dWg_s; g.ldc = fs;
        if (xt) { g.A = xt; g.lda = L.xt_ld; }
        auto wg = [&]() { return xt ? launch_gemm_wgrad_t(g, 1, s) : launch_gemm_wgrad(g, 1, s); };
        if ((e = wg()) != hipSuccess) return e;
        g.B = at<uint16_t>(ws, L.dBs); g.Cf = gr->dWu_s;
        if ((e = wg()) != hipSuccess) return e;
    }
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = at<uint16_t>(ws, L.Hs); g.lda = fs; g.a_nrows = Tn;
    g.B = dY; g.ldb = d; g.b_nrows = Tn;
    g.M = fs; g.N = d; g.K = T;
    g.Cf = gr->dWd_s; g.ldc = d;
    if (dyt) {
        g.B = dyt; g.ldb = L.xt_ld;
        return launch_gemm_wgrad_tb(g, 1, s);
    }
    return launch_gemm_wgrad(g, 1, s);
}

// The whole shared-expert backward.  Marks stages 7 and 8 of the stage
// events between its GEMMs.
hipError_t shared_backward(const moe_shape &sh, const Layout &L, void *ws, const moe_bf16 *dY,
                           const moe_bf16 *X, const moe_weights *w, const moe_grads *gr,
                           const StageMarks &mk, hipStream_t s, const uint16_t *xt = nullptr,
                           const uint16_t *dyt = nullptr) {
    hipError_t e;
    if ((e = shared_dgrad(sh, L, ws, dY, w, s)) != hipSuccess) return e;
    if ((e = mk.mark(7)) != hipSuccess) return e;
    if ((e = shared_dx(sh, L, ws, w, s)) != hipSuccess) return e;
    if ((e = mk.mark(8)) != hipSuccess) return e;
    return shared_wgrads(sh, L, ws, dY, X, gr, s, xt, dyt);
}

// Dense routing (k == E): every token routes to every local expert, so its
// route to expert e sits at row offsets[e] + t of the plan, and the combine
// (sum over the token's experts in ascending id, plus the shared expert) is a
// contraction over the experts' concatenated intermediate columns.  The down
// product then writes Y directly from fp32, with no per-route output and no
// combine pass; the dX product likewise writes dX with the shared expert's
// and the router's terms.

// Y = sum_e (w h)_e W_down[e] + Hs Wd_s over K segments (H holds w h).
GemmArgs down_cmb_args(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                       const int *offsets, moe_bf16 *Y) {
    const int T = (int)sh.T, d = (int)sh.d, f = (int)sh.f, fs = (int)sh.f_shared;
    const long R = (long)T * sh.k;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = at<uint16_t>(ws, L.H); g.lda = f; g.a_nrows = R > 0 ? (int)R : 1;
    g.B = w->W_down; g.ldb = d; g.b_estride = (long)f * d;
    g.M = T; g.N = d;
    g.seg_offsets = offsets; g.nseg = (int)sh.E; g.segK = f;
    if (fs > 0) {
        g.segK_s = fs;
        g.As = at<uint16_t>(ws, L.Hs); g.lda_s = fs;
        g.Bs = w->Wd_s; g.ldb_s = d;
    }
    g.C = Y; g.ldc = d;
    return g;
}

// dX = sum_e (dA W_gate[e]^T + dB W_up[e]^T) + dAs Wg_s^T + dBs Wu_s^T +
// dZ W_r^T over K segments (the router term from the split rows).
GemmArgs dx_cmb_args(const moe_shape &sh, const Layout &L, void *ws, const moe_weights *w,
                     const int *offsets, moe_bf16 *dX) {
    const int T = (int)sh.T, d = (int)sh.d, f = (int)sh.f, fs = (int)sh.f_shared;
    const long R = (long)T * sh.k;
    GemmArgs g;
    g.zeros = at<uint16_t>(ws, L.zeros);
    g.A = at<uint16_t>(ws, L.dA); g.A2 = at<uint16_t>(ws, L.dB); g.lda = f;
    g.a_nrows = R > 0 ? (int)R : 1;
    g.B = w->W_gate; g.B2 = w->W_up; g.ldb = f; g.b_estride = (long)d * f;
    g.M = T; g.N = d;
    g.seg_offsets = offsets; g.nseg = (int)sh.E; g.segK = f;
    if (fs > 0) {
        g.segK_s = fs;
        g.As = at<uint16_t>(ws, L.dAs); g.As2 = at<uint16_t>(ws, L.dBs); g.lda_s = fs;
        g.Bs = w->Wg_s; g.Bs2 = w->Wu_s; g.ldb_s = fs;
    }
    g.Ar = at<uint16_t>(ws, L.dzs); g.Br = at<uint16_t>(ws, L.wrs);
    g.C = dX; g.ldc = d;
    return g;
}

moe_status check_backward_args(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                               const moe_bf16 *W_r, const moe_weights *weights,
                               const int32_t *topk_idx, const float *topk_w,
                               const moe_plan_bufs *plan, const moe_bf16 *dX,
                               const moe_grads *grads) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(dY) || !ptr_ok(X) || !ptr_ok(W_r) || !ptr_ok(topk_idx) || !ptr_ok(topk_w) ||
        !ptr_ok(dX))
        return MOE_EINVAL;
    if ((st = check_weights(shape, weights)) != MOE_OK) return st;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if (!grads || !ptr_ok(grads->dW_gate) || !ptr_ok(grads->dW_up) || !ptr_ok(grads->dW_down) ||
        !ptr_ok(grads->dW_r) || !opt_ok(grads->dZ))
        return MOE_EINVAL;
    if (shape->f_shared > 0) {
        if (!ptr_ok(grads->dWg_s) || !ptr_ok(grads->dWu_s) || !ptr_ok(grads->dWd_s)) return MOE_EINVAL;
    } else if (grads->dWg_s || grads->dWu_s || grads->dWd_s) {
        return MOE_EINVAL;
    }
    return MOE_OK;
}

// Bounded-memory execution: ring size and window count.
moe_status check_ring(int64_t ring_rows) {
    if (ring_rows < 1) return MOE_EINVAL;
    if (ring_rows >= (int64_t(1) << 31)) return MOE_EUNSUPPORTED;
    return MOE_OK;
}

long ring_act_rows(const moe_shape &sh, int64_t ring_rows) {
    const long R = (long)sh.T * sh.k;
    return ring_rows < R ? (long)ring_rows : R;
}

int ring_windows(const moe_shape &sh, int64_t ring_rows) {
    const long R = (long)sh.T * sh.k;
    const long m = (R + ring_rows - 1) / ring_rows;
    return m > 0 ? (int)m : 1;   // an empty batch still runs one (empty) window
}

// Dense routing whose windows hold whole experts (every expert's region is T
// rows, so a window of a multiple of T rows, or of the whole batch, cuts
// none): the ring then runs the folded down and dX products of one-pass
// dense routing on each window's experts, keeping a running fp32 sum per
// token across windows instead of per-route outputs and a combine pass.
bool ring_folds(const moe_shape &sh, int64_t ring_rows) {
    const long R = (long)sh.T * sh.k;
    return dense_routing(sh) && sh.T > 0 && (ring_rows % sh.T == 0 || ring_rows >= R);
}

// The folded product of window [w0, w1) (whole experts w0 / T .. w1 / T - 1)
// of a pass over nwin windows, `first` / `last` in processing order: the
// first writes the running sum (or, alone, the output), later ones add to
// it, the last writes the output.
void fold_window(GemmArgs &g, const moe_shape &sh, long w0, long w1, int nwin, bool first,
                 bool last, float *acc, moe_bf16 *out) {
    const long T = sh.T;
    const long e0 = w0 / T;
    g.a_row0 = (int)w0;
    g.a_nrows = (int)w1;
    g.seg_offsets += e0;
    g.nseg = (int)(w1 / T - e0);
    g.B += e0 * g.b_estride;
    if (g.B2) g.B2 += e0 * g.b_estride;
    if (nwin > 1) {
        g.Cf = acc;
        g.accumulate = first ? 0 : 1;
        g.C = last ? out : nullptr;
    }
}

}  // namespace

extern "C" {

size_t moe_workspace_bytes(const moe_shape *shape, int with_backward) {
    if (check_shape(shape) != MOE_OK) return 0;
    const Layout L = make_layout(*shape);
    return with_backward ? L.bwd_total : L.fwd_total;
}

moe_status moe_workspace_region(const moe_shape *shape, int with_backward, moe_ws_tensor which,
                                size_t *offset, size_t *bytes) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!offset || !bytes) return MOE_EINVAL;
    const Layout L = make_layout(*shape);
    const size_t R = (size_t)(shape->T * shape->k);
    const size_t T = shape->T, d = shape->d, f = shape->f;
    switch (which) {
        case MOE_WS_ERROR: *offset = L.err; *bytes = 4; break;
        case MOE_WS_A: *offset = L.A; *bytes = R * f * 2; break;
        case MOE_WS_B: *offset = L.B; *bytes = R * f * 2; break;
        case MOE_WS_H: *offset = L.H; *bytes = R * f * 2; break;
        case MOE_WS_YEXP: *offset = L.Yexp; *bytes = R * d * 2; break;
        case MOE_WS_YSH: *offset = L.Ysh; *bytes = T * d * 2; break;
        case MOE_WS_DG: *offset = L.dg; *bytes = R * 4; break;
        case MOE_WS_DA: *offset = L.dA; *bytes = R * f * 2; break;
        case MOE_WS_DB: *offset = L.dB; *bytes = R * f * 2; break;
        case MOE_WS_DXPERM: *offset = L.dXperm; *bytes = R * d * 2; break;
        case MOE_WS_HW: *offset = L.Hw; *bytes = R * f * 2; break;
        default: return MOE_EINVAL;
    }
    if (!with_backward && *offset >= L.fwd_total) return MOE_EINVAL;
    return MOE_OK;
}

moe_status moe_route(const moe_shape *shape, const moe_bf16 *X, const moe_bf16 *W_r,
                     const float *bias, float *logits, int32_t *topk_idx, float *topk_w, void *ws,
                     size_t ws_bytes, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(W_r) || !opt_ok(bias) || !ptr_ok(logits) || !ptr_ok(topk_idx) ||
        !ptr_ok(topk_w))
        return MOE_EINVAL;
    if ((st = check_ws_prefix(shape, ws, ws_bytes)) != MOE_OK) return st;
    const Layout L = make_layout(*shape);
    hipStream_t s = static_cast<hipStream_t>(stream);
    MOE_TRY(launch_route(X, W_r, bias, logits, topk_idx, topk_w, at<uint16_t>(ws, L.wrt),
                         at<float>(ws, L.rpart),
                         (int)shape->T, (int)shape->d, (int)shape->E, (int)shape->k, s));
    return MOE_OK;
}

moe_status moe_plan(const moe_shape *shape, const int32_t *topk_idx, const moe_plan_bufs *plan,
                    void *ws, size_t ws_bytes, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(topk_idx)) return MOE_EINVAL;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if ((st = check_ws_prefix(shape, ws, ws_bytes)) != MOE_OK) return st;
    const Layout L = make_layout(*shape);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int R = (int)(shape->T * shape->k);
    MOE_TRY(launch_plan(topk_idx, R, (int)shape->E, plan->counts, plan->offsets, plan->perm,
                        plan->route_pos, at<int>(ws, L.blockcounts), at<int>(ws, L.blockbase),
                        at<int>(ws, L.blockflags), at<int>(ws, L.err), s));
    return MOE_OK;
}

moe_status moe_plan_noalloc(const moe_shape *shape, const int32_t *topk_idx,
                            const moe_plan_bufs *plan, int32_t *error_word, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(topk_idx) || !ptr_ok(error_word)) return MOE_EINVAL;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    const long R = (long)(shape->T * shape->k);
    const size_t need = plan_scratch_bytes(R, shape->E);
    if (need > NOALLOC_SCRATCH_BYTES) return MOE_EUNSUPPORTED;
    uint8_t *sp = static_cast<uint8_t *>(device_scratch());
    if (!sp) return MOE_EHIP;
    const size_t nb = (size_t)plan_nblocks(R);
    const size_t cnt_bytes = up(nb * (size_t)shape->E * 4);
    int *blockcounts = reinterpret_cast<int *>(sp);
    int *blockbase = reinterpret_cast<int *>(sp + cnt_bytes);
    int *blockflags = reinterpret_cast<int *>(sp + 2 * cnt_bytes);
    // every scratch word is written before it is read, so nothing is cleared
    MOE_TRY(launch_plan(topk_idx, (int)R, (int)shape->E, plan->counts, plan->offsets, plan->perm,
                        plan->route_pos, blockcounts, blockbase, blockflags, error_word,
                        static_cast<hipStream_t>(stream)));
    return MOE_OK;
}

size_t moe_schedule_workspace_bytes(int64_t R, int64_t NK, int64_t L) {
    if (check_schedule_dims(R, NK, L, 0) != MOE_OK) return 0;
    return schedule_layout(R, NK, L).total;
}

moe_status moe_schedule(int64_t R, int64_t NK, int64_t L, int64_t c, const int32_t *A, int32_t *M,
                        int32_t *S, int32_t *phi, int64_t phi_rows, void *ws, size_t ws_bytes,
                        moe_stream stream) {
    moe_status st = check_schedule_dims(R, NK, L, c);
    if (st != MOE_OK) return st;
    if (!ptr_ok(A) || !ptr_ok(M) || !ptr_ok(S) || !ptr_ok(phi) || !ptr_ok(ws) || phi_rows < 0)
        return MOE_EINVAL;
    const SchedLayout SL = schedule_layout(R, NK, L);
    if (ws_bytes < SL.total) return MOE_ENOSPACE;
    MOE_TRY(launch_schedule(A, (int)R, (int)NK, (int)L, (int)c, M, S, phi, (long)phi_rows,
                            at<int>(ws, SL.counts), at<int>(ws, SL.flags), at<int>(ws, SL.err),
                            static_cast<hipStream_t>(stream)));
    return MOE_OK;
}

moe_status moe_dispatch(const moe_shape *shape, const moe_bf16 *X, const moe_plan_bufs *plan,
                        moe_bf16 *Xperm, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(Xperm)) return MOE_EINVAL;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    MOE_TRY(launch_gather(X, plan->perm, plan->offsets, (int)shape->E, (int)shape->k,
                          (int)shape->T, (int)shape->d, Xperm, s));
    return MOE_OK;
}

moe_status moe_forward(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                       const int32_t *topk_idx, const float *topk_w, const moe_plan_bufs *plan,
                       moe_bf16 *Y, int save_for_backward, void *ws, size_t ws_bytes,
                       moe_stream stream, const moe_stage_events *events) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(topk_idx) || !ptr_ok(topk_w) || !ptr_ok(Y)) return MOE_EINVAL;
    if ((st = check_weights(shape, weights)) != MOE_OK) return st;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if ((st = check_ws(shape, ws, ws_bytes, 0)) != MOE_OK) return st;
    const Layout L = make_layout(*shape);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const int fs = (int)shape->f_shared;
    const Window all{plan->offsets, 0, (int)((long)T * k)};
    const StageMarks mk{events, s};

    MOE_TRY(mk.mark(0));
    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    MOE_TRY(mk.mark(1));
    if (dense_routing(*shape)) {
        // H keeps w h; the down product adds every expert and the shared
        // expert into Y (stages 4 and 5 are empty)
        GemmArgs gu = up_args(*shape, L, ws, X, weights, all, true, save_for_backward != 0);
        gu.rowscale = at<float>(ws, L.wperm);
        MOE_TRY(launch_gemm_fwd_up(gu, all.count(), E, s));
        MOE_TRY(mk.mark(2));
        if (fs > 0) MOE_TRY(shared_up(*shape, L, ws, X, weights, save_for_backward != 0, s));
        MOE_TRY(mk.mark(3));
        MOE_TRY(launch_gemm_fwd_down_cmb(down_cmb_args(*shape, L, ws, weights, plan->offsets, Y), s));
        MOE_TRY(mk.mark(4));
        MOE_TRY(mk.mark(5));
        MOE_TRY(mk.mark(6));
        return MOE_OK;
    }
    MOE_TRY(routed_up(*shape, L, ws, X, weights, all, true, save_for_backward != 0, s));
    MOE_TRY(mk.mark(2));
    if (fs > 0) MOE_TRY(shared_up(*shape, L, ws, X, weights, save_for_backward != 0, s));
    MOE_TRY(mk.mark(3));
    MOE_TRY(routed_down(*shape, L, ws, weights, all, s));
    MOE_TRY(mk.mark(4));
    if (fs > 0) MOE_TRY(shared_down(*shape, L, ws, weights, s));
    MOE_TRY(mk.mark(5));
    MOE_TRY(launch_combine(at<uint16_t>(ws, L.Yexp), fs > 0 ? at<uint16_t>(ws, L.Ysh) : nullptr,
                           topk_w, plan->route_pos, T, d, k, Y, s));
    MOE_TRY(mk.mark(6));
    return MOE_OK;
}

moe_status moe_forward_fused(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                             const int32_t *topk_idx, const float *topk_w, const moe_plan_bufs *plan,
                             moe_bf16 *Y, int save_for_backward, void *ws, size_t ws_bytes,
                             moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(topk_idx) || !ptr_ok(topk_w) || !ptr_ok(Y)) return MOE_EINVAL;
    if ((st = check_weights(shape, weights)) != MOE_OK) return st;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if ((st = check_ws(shape, ws, ws_bytes, 0)) != MOE_OK) return st;
    const Layout L = make_layout(*shape);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const bool shared = shape->f_shared > 0;
    const long R = (long)T * k;
    const Window all{plan->offsets, 0, (int)R};
    const bool save = save_for_backward != 0;

    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    const GemmArgs none;
    const bool dense = dense_routing(*shape);
    GemmArgs gu = up_args(*shape, L, ws, X, weights, all, true, save);
    if (dense) gu.rowscale = at<float>(ws, L.wperm);
    MOE_TRY(launch_fused_forward(shared ? shared_up_args(*shape, L, ws, X, weights, save) : none, gu,
                                 shared && !dense ? shared_down_args(*shape, L, ws, weights) : none,
                                 dense ? down_cmb_args(*shape, L, ws, weights, plan->offsets, Y)
                                       : down_args(*shape, L, ws, weights, all),
                                 shared, dense, T, R, E,
                                 at<uint16_t>(ws, L.Yexp), at<uint16_t>(ws, L.Ysh), topk_w,
                                 plan->route_pos, topk_idx, plan->offsets, d, k, Y,
                                 at<int>(ws, L.fused), at<int>(ws, L.err), s));
    return MOE_OK;
}

moe_status moe_backward(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                        const moe_bf16 *W_r, const moe_weights *weights, const int32_t *topk_idx,
                        const float *topk_w, const moe_plan_bufs *plan, moe_bf16 *dX,
                        const moe_grads *grads, void *ws, size_t ws_bytes, moe_stream stream,
                        const moe_stage_events *events) {
    moe_status st = check_backward_args(shape, dY, X, W_r, weights, topk_idx, topk_w, plan, dX, grads);
    if (st != MOE_OK) return st;
    if ((st = check_ws(shape, ws, ws_bytes, 1)) != MOE_OK) return st;
    const Layout L = make_layout(*shape);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const Window all{plan->offsets, 0, (int)((long)T * k)};
    float *dZ = grads->dZ ? grads->dZ : at<float>(ws, L.dZ);
    const StageMarks mk{events, s};

    const bool shared = shape->f_shared > 0;

    MOE_TRY(mk.mark(0));
    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    MOE_TRY(mk.mark(1));
    MOE_TRY(routed_dgrad(*shape, L, ws, dY, weights, all, s));
    MOE_TRY(mk.mark(2));
    MOE_TRY(launch_softmax_bwd(at<float>(ws, L.dgpart), L.dg_parts, plan->route_pos, topk_w, topk_idx,
                               T, k, E, at<float>(ws, L.dg), dZ, s));
    if (dense_routing(*shape)) {
        // dX in one product over every expert, the shared expert and the
        // router term (stage 3, the routed dX, and stage 10, the reverse
        // combine, are empty; stage 7 is the whole dX)
        MOE_TRY(launch_router_split(dZ, W_r, T, d, E, at<uint16_t>(ws, L.dzs), at<uint16_t>(ws, L.wrs), s));
        MOE_TRY(mk.mark(3));
        uint16_t *xt = at<uint16_t>(ws, L.xtt), *dyt = at<uint16_t>(ws, L.dytt);
        MOE_TRY(dense_transposes(*shape, L, X, dY, xt, dyt, s));
        MOE_TRY(mk.mark(4));
        MOE_TRY(dense_wgrads(*shape, L, ws, X, dY, grads, plan->offsets, xt, dyt, 0, 2, s));
        MOE_TRY(mk.mark(5));
        MOE_TRY(dense_wgrads(*shape, L, ws, X, dY, grads, plan->offsets, xt, dyt, 2, 3, s));
        MOE_TRY(mk.mark(6));
        if (shared) MOE_TRY(shared_dgrad(*shape, L, ws, dY, weights, s));
        MOE_TRY(mk.mark(7));
        MOE_TRY(launch_gemm_bwd_dx_cmb(dx_cmb_args(*shape, L, ws, weights, plan->offsets, dX), s));
        MOE_TRY(mk.mark(8));
        if (shared) MOE_TRY(shared_wgrads(*shape, L, ws, dY, X, grads, s, xt, dyt));
        MOE_TRY(mk.mark(9));
        MOE_TRY(launch_dwr(X, dZ, T, d, E, at<float>(ws, L.dwr_part), grads->dW_r, s));
        MOE_TRY(mk.mark(10));
        MOE_TRY(mk.mark(11));
        return MOE_OK;
    }
    MOE_TRY(mk.mark(3));
    MOE_TRY(routed_dx(*shape, L, ws, weights, all, s));
    MOE_TRY(mk.mark(4));
    MOE_TRY(launch_gemm_wgrad(wgrad_args(*shape, L, ws, X, dY, grads, all, false, 0), E, s));
    MOE_TRY(launch_gemm_wgrad(wgrad_args(*shape, L, ws, X, dY, grads, all, false, 1), E, s));
    MOE_TRY(mk.mark(5));
    MOE_TRY(launch_gemm_wgrad(wgrad_args(*shape, L, ws, X, dY, grads, all, false, 2), E, s));
    MOE_TRY(mk.mark(6));
    if (shared) {
        MOE_TRY(shared_backward(*shape, L, ws, dY, X, weights, grads, mk, s));
    } else {
        MOE_TRY(mk.mark(7));
        MOE_TRY(mk.mark(8));
    }
    MOE_TRY(mk.mark(9));
    MOE_TRY(launch_dwr(X, dZ, T, d, E, at<float>(ws, L.dwr_part), grads->dW_r, s));
    MOE_TRY(mk.mark(10));
    MOE_TRY(launch_reverse_combine(at<uint16_t>(ws, L.dXperm), shared ? at<uint16_t>(ws, L.dXsh) : nullptr,
                                   dZ, W_r, plan->route_pos, T, d, k, E, nullptr, dX, s));
    MOE_TRY(mk.mark(11));
    return MOE_OK;
}

size_t moe_ring_workspace_bytes(const moe_shape *shape, int64_t ring_rows, int with_backward) {
    if (check_shape(shape) != MOE_OK || check_ring(ring_rows) != MOE_OK) return 0;
    const Layout L = make_layout(*shape, ring_act_rows(*shape, ring_rows));
    return with_backward ? L.bwd_total : L.fwd_total;
}

moe_status moe_forward_ring(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                            const int32_t *topk_idx, const float *topk_w, const moe_plan_bufs *plan,
                            moe_bf16 *Y, int64_t ring_rows, int save_for_backward, void *ws,
                            size_t ws_bytes, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(topk_idx) || !ptr_ok(topk_w) || !ptr_ok(Y)) return MOE_EINVAL;
    if ((st = check_weights(shape, weights)) != MOE_OK) return st;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if ((st = check_ring(ring_rows)) != MOE_OK) return st;
    if (!ptr_ok(ws)) return MOE_EINVAL;
    const Layout L = make_layout(*shape, ring_act_rows(*shape, ring_rows));
    if (ws_bytes < L.fwd_total) return MOE_ENOSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const int fs = (int)shape->f_shared;
    const long R = (long)T * k;
    const int nwin = ring_windows(*shape, ring_rows);
    int *coff = at<int>(ws, L.coff);

    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    if (ring_folds(*shape, ring_rows)) {
        // per window: up/gate (H keeps w h) and the folded down product of
        // its experts; the first window processed also takes the shared
        // expert's segment
        if (fs > 0) MOE_TRY(shared_up(*shape, L, ws, X, weights, save_for_backward != 0, s));
        for (int m = nwin - 1; m >= 0; --m) {
            const int w0 = (int)(m * ring_rows);
            const int w1 = (int)(R < w0 + ring_rows ? R : w0 + ring_rows);
            const Window win{coff, w0, w1};
            MOE_TRY(launch_clip_offsets(plan->offsets, E, w0, w1, coff, s));
            GemmArgs gu = up_args(*shape, L, ws, X, weights, win, true, save_for_backward != 0);
            gu.rowscale = at<float>(ws, L.wperm);
            MOE_TRY(launch_gemm_fwd_up(gu, win.count(), E, s));
            GemmArgs gd = down_cmb_args(*shape, L, ws, weights, plan->offsets, Y);
            gd.A = win.rows<uint16_t>(ws, L.H, (int)shape->f);
            if (m != nwin - 1) gd.segK_s = 0;
            fold_window(gd, *shape, w0, w1, nwin, m == nwin - 1, m == 0, at<float>(ws, L.acc), Y);
            MOE_TRY(launch_gemm_fwd_down_cmb(gd, s));
        }
        return MOE_OK;
    }
    if (fs > 0) {   // first: its output seeds every token's accumulator
        MOE_TRY(shared_up(*shape, L, ws, X, weights, save_for_backward != 0, s));
        MOE_TRY(shared_down(*shape, L, ws, weights, s));
    }
    // reverse window order: the ring ends up holding the first window, the
    // one the backward consumes first
    for (int m = nwin - 1; m >= 0; --m) {
        const int w0 = (int)(m * ring_rows);
        const int w1 = (int)(R < w0 + ring_rows ? R : w0 + ring_rows);
        const Window win{coff, w0, w1};
        MOE_TRY(launch_clip_offsets(plan->offsets, E, w0, w1, coff, s));
        MOE_TRY(routed_up(*shape, L, ws, X, weights, win, true, save_for_backward != 0, s));
        MOE_TRY(routed_down(*shape, L, ws, weights, win, s));
        MOE_TRY(launch_window_accum(at<uint16_t>(ws, L.Yexp), w0, w1, topk_w,
                                    plan->route_pos, T, d, k, at<float>(ws, L.acc), m == nwin - 1,
                                    fs > 0 ? at<uint16_t>(ws, L.Ysh) : nullptr, m == 0 ? Y : nullptr,
                                    s));
    }
    return MOE_OK;
}

moe_status moe_backward_ring(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                             const moe_bf16 *W_r, const moe_weights *weights, const int32_t *topk_idx,
                             const float *topk_w, const moe_plan_bufs *plan, moe_bf16 *dX,
                             const moe_grads *grads, int64_t ring_rows, void *ws, size_t ws_bytes,
                             moe_stream stream) {
    moe_status st = check_backward_args(shape, dY, X, W_r, weights, topk_idx, topk_w, plan, dX, grads);
    if (st != MOE_OK) return st;
    if ((st = check_ring(ring_rows)) != MOE_OK) return st;
    if (!ptr_ok(ws)) return MOE_EINVAL;
    const Layout L = make_layout(*shape, ring_act_rows(*shape, ring_rows));
    if (ws_bytes < L.bwd_total) return MOE_ENOSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const long R = (long)T * k;
    const int nwin = ring_windows(*shape, ring_rows);
    const bool shared = shape->f_shared > 0;
    int *coff = at<int>(ws, L.coff);
    float *acc = at<float>(ws, L.acc);
    float *dZ = grads->dZ ? grads->dZ : at<float>(ws, L.dZ);
    const StageMarks none{nullptr, s};

    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    // dense routing: the weight gradients of every window read X^T and dY^T
    // (made once) as K-contiguous rows, each expert's rows of the window
    // being the tokens from (first row - the expert's first plan row)
    const bool dense = dense_routing(*shape);
    uint16_t *xt = dense ? at<uint16_t>(ws, L.xtt) : nullptr;
    uint16_t *dyt = dense ? at<uint16_t>(ws, L.dytt) : nullptr;
    if (dense) MOE_TRY(dense_transposes(*shape, L, X, dY, xt, dyt, s));
    const bool fold = ring_folds(*shape, ring_rows);
    if (shared && fold) {
        // dXsh is folded into the first window's dX product
        MOE_TRY(shared_dgrad(*shape, L, ws, dY, weights, s));
        MOE_TRY(shared_wgrads(*shape, L, ws, dY, X, grads, s, xt, dyt));
    } else if (shared) {
        MOE_TRY(shared_backward(*shape, L, ws, dY, X, weights, grads, none, s, xt, dyt));
    }
    // windows alternate between two clipped-offset arrays, so the replay of
    // window m + 1 can share a launch with the weight gradients of window m
    auto window = [&](int m) {
        const int w0 = (int)(m * ring_rows);
        const int w1 = (int)(R < w0 + ring_rows ? R : w0 + ring_rows);
        return Window{coff + (m & 1) * (E + 1), w0, w1};
    };
    auto clip = [&](int m) {
        const Window w = window(m);
        return launch_clip_offsets(plan->offsets, E, w.w0, w.w1, coff + (m & 1) * (E + 1), s);
    };
    MOE_TRY(clip(0));
    for (int m = 0; m < nwin; ++m) {
        const Window win = window(m);
        // window 0 uses the activations the forward left in the ring; the
        // pre-activations of every later window were recomputed in the
        // previous window's weight-gradient launch
        MOE_TRY(routed_dgrad(*shape, L, ws, dY, weights, win, s));
        if (fold) {
            // the folded dX product of the window's experts; the first also
            // takes the shared expert's segments, the last the router term
            // (every dg is known once the last window's dgrad has run)
            if (m == nwin - 1) {
                MOE_TRY(launch_softmax_bwd(at<float>(ws, L.dgpart), L.dg_parts, plan->route_pos, topk_w,
                                           topk_idx, T, k, E, at<float>(ws, L.dg), dZ, s));
                MOE_TRY(launch_router_split(dZ, W_r, T, d, E, at<uint16_t>(ws, L.dzs),
                                            at<uint16_t>(ws, L.wrs), s));
            }
            GemmArgs gx = dx_cmb_args(*shape, L, ws, weights, plan->offsets, dX);
            gx.A = win.rows<uint16_t>(ws, L.dA, (int)shape->f);
            gx.A2 = win.rows<uint16_t>(ws, L.dB, (int)shape->f);
            if (m != 0) gx.segK_s = 0;
            if (m != nwin - 1) gx.Ar = nullptr;
            fold_window(gx, *shape, win.w0, win.w1, nwin, m == 0, m == nwin - 1, acc, dX);
            MOE_TRY(launch_gemm_bwd_dx_cmb(gx, s));
        } else {
            MOE_TRY(routed_dx(*shape, L, ws, weights, win, s));
            MOE_TRY(launch_window_accum(at<uint16_t>(ws, L.dXperm), win.w0, win.w1, nullptr,
                                        plan->route_pos, T, d, k, acc, m == 0,
                                        shared ? at<uint16_t>(ws, L.dXsh) : nullptr, nullptr, s));
        }
        GemmArgs wg[3];
        int modes[3] = {0, 0, 0};
        for (int i = 0; i < 3; ++i) {
            wg[i] = wgrad_args(*shape, L, ws, X, dY, grads, win, m > 0, i);
            if (!dense) continue;
            wg[i].tok_offsets = plan->offsets;
            if (i < 2) {
                wg[i].A = xt; wg[i].lda = L.xt_ld; wg[i].a_rows = nullptr; wg[i].a_local = 1;
                modes[i] = 1;
            } else {
                wg[i].B = dyt; wg[i].ldb = L.xt_ld; wg[i].b_rows = nullptr; wg[i].b_local = 1;
                modes[i] = 2;
            }
        }
        if (m + 1 < nwin) {
            // recompute only A and B of the next window (no H, no down
            // projection): its dgrad reads nothing else
            const Window nxt = window(m + 1);
            MOE_TRY(clip(m + 1));
            const GemmArgs up = up_args(*shape, L, ws, X, weights, nxt, false, true);
            MOE_TRY(launch_gemm_wgrad_batch(wg, 3, E, &up, nxt.count(), s, modes));
        } else {
            MOE_TRY(launch_gemm_wgrad_batch(wg, 3, E, nullptr, 0, s, modes));
        }
    }
    if (fold) {
        MOE_TRY(launch_dwr(X, dZ, T, d, E, at<float>(ws, L.dwr_part), grads->dW_r, s));
        return MOE_OK;
    }
    MOE_TRY(launch_softmax_bwd(at<float>(ws, L.dgpart), L.dg_parts, plan->route_pos, topk_w, topk_idx,
                               T, k, E, at<float>(ws, L.dg), dZ, s));
    MOE_TRY(launch_dwr(X, dZ, T, d, E, at<float>(ws, L.dwr_part), grads->dW_r, s));
    MOE_TRY(launch_reverse_combine(nullptr, nullptr, dZ, W_r, plan->route_pos, T, d, k, E, acc, dX, s));
    return MOE_OK;
}

size_t moe_mx_workspace_bytes(const moe_shape *shape, int with_backward) {
    if (check_shape(shape) != MOE_OK || check_mx_shape(shape) != MOE_OK) return 0;
    if (with_backward < 0 || with_backward > 2) return 0;
    const Layout L = make_layout(*shape);
    if (!with_backward) return L.mx_total;
    if (with_backward == 2) return check_mx_wgrad_shape(shape) == MOE_OK ? L.mxw_total : 0;
    return L.mxb_total > L.mx_total ? L.mxb_total : L.mx_total;
}

moe_status moe_mx_workspace_region(const moe_shape *shape, moe_ws_tensor which, size_t *offset,
                                   size_t *bytes) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if ((st = check_mx_shape(shape)) != MOE_OK) return st;
    if (!offset || !bytes) return MOE_EINVAL;
    const Layout L = make_layout(*shape);
    const size_t R = (size_t)(shape->T * shape->k);
    const size_t T = shape->T, d = shape->d, f = shape->f;
    switch (which) {
        case MOE_WS_ERROR: *offset = L.err; *bytes = 4; break;
        case MOE_WS_YEXP: *offset = L.Yexp; *bytes = R * d * 2; break;
        case MOE_WS_YSH: *offset = L.Ysh; *bytes = T * d * 2; break;
        case MOE_WS_XQ: *offset = L.xq; *bytes = T * d; break;
        case MOE_WS_XS: *offset = L.xs; *bytes = T * d / 32; break;
        case MOE_WS_HQ: *offset = L.hq; *bytes = R * f; break;
        case MOE_WS_HS: *offset = L.hsc; *bytes = R * f / 32; break;
        case MOE_WS_DYQ: *offset = L.dyq; *bytes = T * d; break;
        case MOE_WS_DYS: *offset = L.dys; *bytes = T * d / 32; break;
        case MOE_WS_DAQ: *offset = L.daq; *bytes = R * f; break;
        case MOE_WS_DAS: *offset = L.das; *bytes = R * f / 32; break;
        case MOE_WS_DBQ: *offset = L.dbq; *bytes = R * f; break;
        case MOE_WS_DBS: *offset = L.dbs; *bytes = R * f / 32; break;
        case MOE_WS_POFF: *offset = L.poff; *bytes = (size_t)(shape->E + 1) * 4; break;
        case MOE_WS_XTQ: *offset = L.xt; *bytes = d * (size_t)L.tpad; break;
        case MOE_WS_XTS: *offset = L.xts; *bytes = d * (size_t)L.tpad / 32; break;
        case MOE_WS_DYTQ: *offset = L.dyt; *bytes = d * (size_t)L.tpad; break;
        case MOE_WS_DYTS: *offset = L.dyts; *bytes = d * (size_t)L.tpad / 32; break;
        case MOE_WS_AF: *offset = L.a32; *bytes = R * f * 4; break;
        case MOE_WS_BF: *offset = L.b32; *bytes = R * f * 4; break;
        case MOE_WS_DAF: *offset = L.da32; *bytes = R * f * 4; break;
        case MOE_WS_DBF: *offset = L.db32; *bytes = R * f * 4; break;
        case MOE_WS_HWF: *offset = L.hw32; *bytes = R * f * 4; break;
        default: return moe_workspace_region(shape, 1, which, offset, bytes);
    }
    return MOE_OK;
}

moe_status moe_mx_quantize_weights(const moe_shape *shape, const moe_weights *weights,
                                   const moe_mx_weights *mx, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if ((st = check_mx_shape(shape)) != MOE_OK) return st;
    if (!weights || !ptr_ok(weights->W_gate) || !ptr_ok(weights->W_up) || !ptr_ok(weights->W_down))
        return MOE_EINVAL;
    if (!mx || !ptr_ok(mx->Wg_q) || !ptr_ok(mx->Wu_q) || !ptr_ok(mx->Wd_q) || !ptr_ok(mx->Wg_s) ||
        !ptr_ok(mx->Wu_s) || !ptr_ok(mx->Wd_s))
        return MOE_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int E = (int)shape->E, d = (int)shape->d, f = (int)shape->f;
    MOE_TRY(launch_mx_quant_weights(weights->W_gate, E, d, f, mx->Wg_q, mx->Wg_s, s));
    MOE_TRY(launch_mx_quant_weights(weights->W_up, E, d, f, mx->Wu_q, mx->Wu_s, s));
    MOE_TRY(launch_mx_quant_weights(weights->W_down, E, f, d, mx->Wd_q, mx->Wd_s, s));
    return MOE_OK;
}

moe_status moe_forward_mx(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                          const moe_mx_weights *mx, const int32_t *topk_idx, const float *topk_w,
                          const moe_plan_bufs *plan, moe_bf16 *Y, int save_for_backward, void *ws,
                          size_t ws_bytes, moe_stream stream, const moe_stage_events *events) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if ((st = check_mx_shape(shape)) != MOE_OK) return st;
    if (!ptr_ok(X) || !ptr_ok(topk_idx) || !ptr_ok(topk_w) || !ptr_ok(Y)) return MOE_EINVAL;
    if ((st = check_mx_weights(shape, weights, mx)) != MOE_OK) return st;
    if ((st = check_plan(plan)) != MOE_OK) return st;
    if (!ptr_ok(ws)) return MOE_EINVAL;
    const Layout L = make_layout(*shape);
    if (ws_bytes < L.mx_total) return MOE_ENOSPACE;
    if (save_for_backward && ws_bytes < L.mxb_total) return MOE_ENOSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const int f = (int)shape->f, fs = (int)shape->f_shared;
    const long R = (long)T * k;
    int *rowidx = at<int>(ws, L.rowidx);
    uint8_t *xq = at<uint8_t>(ws, L.xq), *xs = at<uint8_t>(ws, L.xs);
    uint8_t *hq = at<uint8_t>(ws, L.hq), *hs = at<uint8_t>(ws, L.hsc);
    const StageMarks mk{events, s};

    MOE_TRY(mk.mark(0));
    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, rowidx, at<float>(ws, L.wperm),
                        at<uint16_t>(ws, L.zeros), s));
    // activation quantisation of the dispatch: each token once, before the gather
    MOE_TRY(launch_mx_quant_rows(X, T, d, xq, xs, s));
    MOE_TRY(mk.mark(1));
    {   // routed up/gate + SwiGLU, H quantised in the epilogue
        MxGemmArgs g;
        g.A = xq; g.As = xs; g.a_rows = rowidx; g.a_nrows = T > 0 ? T : 1;
        g.B = mx->Wg_q; g.Bs = mx->Wg_s; g.B2 = mx->Wu_q; g.Bs2 = mx->Wu_s;
        g.K = d; g.N = f; g.offsets = plan->offsets; g.E = E;
        g.C = hq; g.Cs = hs;
        if (save_for_backward) { g.Sa = at<float>(ws, L.a32); g.Sb = at<float>(ws, L.b32); }
        g.a_bytes = (uint32_t)((long)(T > 0 ? T : 1) * d);
        g.as_bytes = (uint32_t)((long)(T > 0 ? T : 1) * d / 32);
        g.b_bytes = (uint32_t)((long)E * f * d);
        g.bs_bytes = (uint32_t)((long)E * f * d / 32);
        MOE_TRY(launch_gemm_mx_up(g, R, E, s));
    }
    MOE_TRY(mk.mark(2));
    if (fs > 0) MOE_TRY(shared_up(*shape, L, ws, X, weights, save_for_backward != 0, s));
    MOE_TRY(mk.mark(3));
    {   // routed down
        MxGemmArgs g;
        g.A = hq; g.As = hs; g.a_nrows = R > 0 ? (int)R : 1;
        g.B = mx->Wd_q; g.Bs = mx->Wd_s;
        g.K = f; g.N = d; g.offsets = plan->offsets; g.E = E;
        g.Cb = at<uint16_t>(ws, L.Yexp);
        g.a_bytes = (uint32_t)((R > 0 ? R : 1) * f);
        g.as_bytes = (uint32_t)((R > 0 ? R : 1) * f / 32);
        g.b_bytes = (uint32_t)((long)E * d * f);
        g.bs_bytes = (uint32_t)((long)E * d * f / 32);
        MOE_TRY(launch_gemm_mx_down(g, R, E, s));
    }
    MOE_TRY(mk.mark(4));
    if (fs > 0) MOE_TRY(shared_down(*shape, L, ws, weights, s));
    MOE_TRY(mk.mark(5));
    MOE_TRY(launch_combine(at<uint16_t>(ws, L.Yexp), fs > 0 ? at<uint16_t>(ws, L.Ysh) : nullptr,
                           topk_w, plan->route_pos, T, d, k, Y, s));
    MOE_TRY(mk.mark(6));
    return MOE_OK;
}

moe_status moe_mx_quantize_weights_bwd(const moe_shape *shape, const moe_weights *weights,
                                       const moe_mx_bwd_weights *mx, moe_stream stream) {
    moe_status st = check_shape(shape);
    if (st != MOE_OK) return st;
    if ((st = check_mx_shape(shape)) != MOE_OK) return st;
    if (!weights || !ptr_ok(weights->W_gate) || !ptr_ok(weights->W_up) || !ptr_ok(weights->W_down))
        return MOE_EINVAL;
    if (!mx || !ptr_ok(mx->Wg_q) || !ptr_ok(mx->Wu_q) || !ptr_ok(mx->Wd_q) || !ptr_ok(mx->Wg_s) ||
        !ptr_ok(mx->Wu_s) || !ptr_ok(mx->Wd_s))
        return MOE_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const long E = shape->E, d = shape->d, f = shape->f;
    // each weight row is already contiguous along the axis its backward
    // product contracts: W_gate / W_up [E, d, f] along f, W_down [E, f, d] along d
    MOE_TRY(launch_mx_quant_rows(weights->W_gate, E * d, (int)f, mx->Wg_q, mx->Wg_s, s));
    MOE_TRY(launch_mx_quant_rows(weights->W_up, E * d, (int)f, mx->Wu_q, mx->Wu_s, s));
    MOE_TRY(launch_mx_quant_rows(weights->W_down, E * f, (int)d, mx->Wd_q, mx->Wd_s, s));
    return MOE_OK;
}

moe_status moe_backward_mx(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                           const moe_bf16 *W_r, const moe_weights *weights,
                           const moe_mx_bwd_weights *mx, const int32_t *topk_idx, const float *topk_w,
                           const moe_plan_bufs *plan, moe_bf16 *dX, const moe_grads *grads,
                           int wgrad_mxfp8, void *ws, size_t ws_bytes, moe_stream stream) {
    moe_status st = check_backward_args(shape, dY, X, W_r, weights, topk_idx, topk_w, plan, dX, grads);
    if (st != MOE_OK) return st;
    if ((st = check_mx_shape(shape)) != MOE_OK) return st;
    if (wgrad_mxfp8 != 0 && wgrad_mxfp8 != 1) return MOE_EINVAL;
    if (wgrad_mxfp8 && (st = check_mx_wgrad_shape(shape)) != MOE_OK) return st;
    if (!mx || !ptr_ok(mx->Wg_q) || !ptr_ok(mx->Wu_q) || !ptr_ok(mx->Wd_q) || !ptr_ok(mx->Wg_s) ||
        !ptr_ok(mx->Wu_s) || !ptr_ok(mx->Wd_s))
        return MOE_EINVAL;
    if (!ptr_ok(ws)) return MOE_EINVAL;
    const Layout L = make_layout(*shape);
    if (ws_bytes < L.mxb_total || ws_bytes < L.mx_total) return MOE_ENOSPACE;
    if (wgrad_mxfp8 && ws_bytes < L.mxw_total) return MOE_ENOSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = (int)shape->T, d = (int)shape->d, E = (int)shape->E, k = (int)shape->k;
    const int f = (int)shape->f;
    const long R = (long)T * k;
    const long Tn = T > 0 ? T : 1, Rn = R > 0 ? R : 1;
    const Window all{plan->offsets, 0, (int)R};
    const bool shared = shape->f_shared > 0;
    float *dZ = grads->dZ ? grads->dZ : at<float>(ws, L.dZ);
    uint8_t *dyq = at<uint8_t>(ws, L.dyq), *dys = at<uint8_t>(ws, L.dys);
    uint8_t *daq = at<uint8_t>(ws, L.daq), *das = at<uint8_t>(ws, L.das);
    uint8_t *dbq = at<uint8_t>(ws, L.dbq), *dbs = at<uint8_t>(ws, L.dbs);

    MOE_TRY(launch_prep(plan->perm, plan->offsets, E, topk_w, k, T, at<int>(ws, L.rowidx),
                        at<float>(ws, L.wperm), at<uint16_t>(ws, L.zeros), s));
    // the reverse-combine's activation quantisation: dY once per token, before the gather
    MOE_TRY(launch_mx_quant_rows(dY, T, d, dyq, dys, s));
    {   // dh' = Q(dY) Q(W_down)^T with the gated-activation backward; dA, dB quantised along f
        MxGemmArgs g;
        g.A = dyq; g.As = dys; g.a_rows = at<int>(ws, L.rowidx); g.a_nrows = (int)Tn;
        g.B = mx->Wd_q; g.Bs = mx->Wd_s;
        g.K = d; g.N = f; g.offsets = plan->offsets; g.E = E;
        g.C = daq; g.Cs = das; g.C2 = dbq; g.Cs2 = dbs;
        if (wgrad_mxfp8) {   // the token-axis quantisers read dA, dB, w h at fp32
            g.Cf1 = at<float>(ws, L.da32); g.Cf2 = at<float>(ws, L.db32); g.Cf3 = at<float>(ws, L.hw32);
        } else {
            g.Cb = at<uint16_t>(ws, L.dA); g.Cb2 = at<uint16_t>(ws, L.dB); g.Cb3 = at<uint16_t>(ws, L.Hw);
        }
        g.E1 = at<float>(ws, L.a32); g.E2 = at<float>(ws, L.b32);
        g.rowscale = at<float>(ws, L.wperm);
        g.dgpart = at<float>(ws, L.dgpart); g.dg_ld = L.dg_parts;
        g.a_bytes = (uint32_t)(Tn * d);
        g.as_bytes = (uint32_t)(Tn * d / 32);
        g.b_bytes = (uint32_t)((long)E * f * d);
        g.bs_bytes = (uint32_t)((long)E * f * d / 32);
        MOE_TRY(launch_gemm_mx_dgrad(g, R, E, s));
    }
    MOE_TRY(launch_softmax_bwd(at<float>(ws, L.dgpart), L.dg_parts, plan->route_pos, topk_w, topk_idx,
                               T, k, E, at<float>(ws, L.dg), dZ, s));
    {   // dXperm = Q(dA) Q(W_gate)^T + Q(dB) Q(W_up)^T
        MxGemmArgs g;
        g.A = daq; g.As = das; g.A2 = dbq; g.As2 = dbs; g.a_nrows = (int)Rn;
        g.B = mx->Wg_q; g.Bs = mx->Wg_s; g.B2 = mx->Wu_q; g.Bs2 = mx->Wu_s;
        g.K = f; g.N = d; g.offsets = plan->offsets; g.E = E;
        g.Cb = at<uint16_t>(ws, L.dXperm);
        g.a_bytes = (uint32_t)(Rn * f);
        g.as_bytes = (uint32_t)(Rn * f / 32);
        g.b_bytes = (uint32_t)((long)E * d * f);
        g.bs_bytes = (uint32_t)((long)E * d * f / 32);
        MOE_TRY(launch_gemm_mx_dx(g, R, E, s));
    }
    if (wgrad_mxfp8) {
        // weight gradients in MXFP8: the operands quantised along the token
        // axis per expert (blocks of 32 from each expert's first row, each
        // expert's region padded to 128 positions), then dW = A . B^T over
        // the expert's padded range on the block-scaled matrix cores
        int *poff = at<int>(ws, L.poff);
        const long P = L.tpad;
        const int *rowidx = at<int>(ws, L.rowidx);
        MOE_TRY(launch_mx_pad_offsets(plan->offsets, E, poff, s));
        // With dense routing every expert's range holds tokens 0 .. T-1 in
        // order, so the token-axis codes of X and dY are the same for every
        // expert: quantise expert 0's range only and let the weight-gradient
        // products read it from position 0 (bitwise the same operands).
        const bool dense = dense_routing(*shape);
        const int qE = dense ? 1 : E;
        MOE_TRY(launch_mx_quant_tokens(X, d, T, rowidx, plan->offsets, poff, qE, d, P, P,
                                       at<uint8_t>(ws, L.xt), at<uint8_t>(ws, L.xts), s));
        MOE_TRY(launch_mx_quant_tokens(dY, d, T, rowidx, plan->offsets, poff, qE, d, P, P,
                                       at<uint8_t>(ws, L.dyt), at<uint8_t>(ws, L.dyts), s));
        MOE_TRY(launch_mx_quant_tokens_f32(at<float>(ws, L.da32), f, R, plan->offsets, poff, E, f, P,
                                           P, at<uint8_t>(ws, L.dat), at<uint8_t>(ws, L.dats), s));
        MOE_TRY(launch_mx_quant_tokens_f32(at<float>(ws, L.db32), f, R, plan->offsets, poff, E, f, P,
                                           P, at<uint8_t>(ws, L.dbt), at<uint8_t>(ws, L.dbts), s));
        MOE_TRY(launch_mx_quant_tokens_f32(at<float>(ws, L.hw32), f, R, plan->offsets, poff, E, f, P,
                                           P, at<uint8_t>(ws, L.hwt), at<uint8_t>(ws, L.hwts), s));
        auto wg = [&](size_t a, size_t as, int M, size_t b, size_t bs, int N, float *out, int a_sh,
                      int b_sh) {
            MxGemmArgs g;
            g.a_shared = a_sh; g.b_shared = b_sh;
            g.A = at<uint8_t>(ws, a); g.As = at<uint8_t>(ws, as); g.a_nrows = M;
            g.B = at<uint8_t>(ws, b); g.Bs = at<uint8_t>(ws, bs);
            g.M = M; g.N = N; g.K = (int)P; g.offsets = poff; g.E = E; g.Cf = out;
            g.a_bytes = (uint32_t)((long)M * P);
            g.as_bytes = (uint32_t)((long)M * P / 32);
            g.b_bytes = (uint32_t)((long)N * P);
            g.bs_bytes = (uint32_t)((long)N * P / 32);
            return launch_gemm_mx_wgrad(g, E, s);
        };
        MOE_TRY(wg(L.xt, L.xts, d, L.dat, L.dats, f, grads->dW_gate, dense, 0));
        MOE_TRY(wg(L.xt, L.xts, d, L.dbt, L.dbts, f, grads->dW_up, dense, 0));
        MOE_TRY(wg(L.hwt, L.hwts, f, L.dyt, L.dyts, d, grads->dW_down, 0, dense));
    } else if (dense_routing(*shape)) {
        // weight gradients in BF16 on the unquantised operands, X and dY
        // read transposed (dense routing; see dense_transposes)
        uint16_t *xt = at<uint16_t>(ws, L.xtt), *dyt = at<uint16_t>(ws, L.dytt);
        MOE_TRY(dense_transposes(*shape, L, X, dY, xt, dyt, s));
        MOE_TRY(dense_wgrads(*shape, L, ws, X, dY, grads, plan->offsets, xt, dyt, 0, 3, s));
        if (shared) {
            MOE_TRY(shared_dgrad(*shape, L, ws, dY, weights, s));
            MOE_TRY(shared_dx(*shape, L, ws, weights, s));
            MOE_TRY(shared_wgrads(*shape, L, ws, dY, X, grads, s, xt, dyt));
        }
    } else {
        // weight gradients in BF16 on the unquantised operands
        for (int i = 0; i < 3; ++i)
            MOE_TRY(launch_gemm_wgrad(wgrad_args(*shape, L, ws, X, dY, grads, all, false, i), E, s));
    }
    if (shared && (wgrad_mxfp8 || !dense_routing(*shape)))
        MOE_TRY(shared_backward(*shape, L, ws, dY, X, weights, grads, StageMarks{nullptr, s}, s));
    MOE_TRY(launch_dwr(X, dZ, T, d, E, at<float>(ws, L.dwr_part), grads->dW_r, s));
    MOE_TRY(launch_reverse_combine(at<uint16_t>(ws, L.dXperm), shared ? at<uint16_t>(ws, L.dXsh) : nullptr,
                                   dZ, W_r, plan->route_pos, T, d, k, E, nullptr, dX, s));
    return MOE_OK;
}

const char *moe_status_string(moe_status status) {
    switch (status) {
        case MOE_OK: return "ok";
        case MOE_EINVAL: return "invalid argument";
        case MOE_EUNSUPPORTED: return "unsupported shape";
        case MOE_ENOSPACE: return "workspace too small";
        case MOE_EHIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

const char *moe_version(void) { return "moe-mi355x 0.1 (gfx950)"; }

}  // extern "C"
