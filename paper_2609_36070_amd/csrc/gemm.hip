// Grouped bf16 GEMMs of the expert FFNs on CDNA4 MFMA (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation, with the SwiGLU forward/backward fused into the
// epilogues (§2.1 FFN; §3.4 router-weight gradient fused into the gated
// activation backward).
//
// One kernel template serves five products; per expert e and buffer
// positions p of e's region [offsets[e], offsets[e+1]):
//
//   FWD_UP     A_e = X[tok(p)] W_gate[e], B_e = X[tok(p)] W_up[e],
//              H = silu(A) * B      (A, B kept for backward; H may be skipped
//                                    when only A, B are recomputed)
//   FWD_DOWN   Yexp = H W_down[e]
//   BWD_DGRAD  dh' = dY[tok(p)] W_down[e]^T, then dg partials <dh', h>,
//              dA = w dh' * B * silu'(A), dB = w dh' * silu(A), Hw = w * h
//   BWD_DX     dXperm = dA W_gate[e]^T + dB W_up[e]^T  (one K loop over both)
//   WGRAD      dW[e] = P_e^T Q_e (or dW[e] += P_e^T Q_e), K = the expert's
//              ragged route count
//
// The dispatch gather is fused into the operand loads: A rows (or WGRAD k
// rows) are read through the plan's token index, so no expert-contiguous
// copy of X or dY is ever written.  The shared expert runs through the same
// kernel as one ungrouped problem of T rows.
//
// Pipeline: 256 x 256 block tile, K step 64, two LDS stages (2 x 64 KB)
// filled by direct global->LDS loads (global_load_lds_dwordx4, no staging
// registers): the next tile streams in while the current one is multiplied,
// one fence-free barrier per K step.  8 waves as 2 (M) x 4 (N), 128 x 64 per
// wave (4 x 2 MFMA tiles).  Tiles are rastered XCD-aware.
//
// LDS tile formats:
//   K-contiguous ("row" tiles: A rows, B rows of an [N][K] weight): 128-byte
//     rows, the 16-byte chunk index XOR (row >> 1) & 7; fragments are read
//     with ds_read_b128.
//   MN-contiguous ("col" tiles: [K][N] weights, both WGRAD operands): 512-byte
//     k rows, the 32-byte block index XOR 2 * (k & 3); fragments are read
//     with ds_read_b64_tr_b16, which hands each lane one column of a 4 x 16
//     block, so no operand is ever transposed in registers.
// Both swizzles keep fragment reads free of bank conflicts and are applied
// on the global side of the direct loads.
//
// Each output element is owned by exactly one block and its K loop runs in
// a fixed order: results are bitwise deterministic (§3.4 "Determinism").
#include "common.h"
#include "kernels.h"

#include <type_traits>

#define LDSP __attribute__((address_space(3)))

namespace {

#ifndef MOE_GEMM_BK
#define MOE_GEMM_BK 64
#endif
constexpr int BM = 256, BN = 256, BK = MOE_GEMM_BK;
static_assert(BK == 32 || BK == 64, "K step is 32 or 64");
#ifndef MOE_GEMM_WAVES_M
#define MOE_GEMM_WAVES_M 2
#endif
#ifndef MOE_GEMM_WAVES_N
#define MOE_GEMM_WAVES_N 4
#endif
constexpr int WAVES_M = MOE_GEMM_WAVES_M, WAVES_N = MOE_GEMM_WAVES_N;
constexpr int NWAVES = WAVES_M * WAVES_N;
constexpr int NTHREADS = 64 * NWAVES;
constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
constexpr int TM = WM / 32, TN = WN / 32;
constexpr int TILE_ELEMS = BM * BK;        // per operand per stage (bf16 elements)
constexpr int ROWS_PER_LD = 512 / BK;      // row-tile rows covered by one 1 KB wave load
constexpr int LD_PER_OP = (BK / 2) / NWAVES;  // 1 KB direct loads per operand per wave per K step
constexpr int LOADS_PER_K = 2 * LD_PER_OP; // direct-load instructions per thread per K step
static_assert(WN == 64 || WN == 128, "gate/up column pairs and the epilogue need 64- or 128-column wave tiles");

enum Mode { FWD_UP = 0, FWD_DOWN = 1, BWD_DGRAD = 2, BWD_DX = 3, WGRAD = 4, FWD_DOWN_CMB = 5,
            BWD_DX_CMB = 6, WGRAD_T = 7, WGRAD_TB = 8 };

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

template <int MODE>
struct Traits {
    static constexpr bool A_COL = (MODE == WGRAD || MODE == WGRAD_TB);   // A stored [K][M]
    static constexpr bool B_COL = (MODE == FWD_UP || MODE == FWD_DOWN || MODE == WGRAD ||
                                   MODE == FWD_DOWN_CMB || MODE == WGRAD_T);
    static constexpr bool WG = (MODE == WGRAD || MODE == WGRAD_T || MODE == WGRAD_TB);  // K = tokens
    static constexpr bool GROUPED_ROWS = !WG;
    static constexpr bool CMB = (MODE == FWD_DOWN_CMB || MODE == BWD_DX_CMB);   // K segments
};

// Row tiles: 16-byte chunk c of row r lives at chunk c ^ ((r >> 2) & 3)
// (64-byte rows) or c ^ ((r >> 1) & 7) (128-byte rows).
DEV int row_swz(int r, int c) { return BK == 32 ? c ^ ((r >> 2) & 3) : c ^ ((r >> 1) & 7); }
// Col tiles: 32-byte block b of k row kr lives at block b ^ (2 * (kr & 3)).
DEV int col_swz(int kr, int b) { return b ^ (2 * (kr & 3)); }

DEV void load_lds16(const uint16_t *src, uint16_t *lds_dst) {
    __builtin_amdgcn_global_load_lds(src, (LDSP void *)lds_dst, 16, 0, 0);
}

DEV int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Workgroup barrier without the memory fence __syncthreads() carries: the
// fence would wait for every in-flight direct load (vmcnt(0)) and undo the
// prefetch.  Ordering is explicit instead: each wave waits for its own tile
// loads (wait_vmcnt) before the barrier, and every LDS read of the previous
// K step has been consumed by an MFMA before the wave reaches it.
DEV void barrier_no_fence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n) leaving lgkm/exp counters alone (gfx9 encoding).
template <int N>
DEV void wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Fragment for MFMA operand rows [r0, r0+32) from a row tile, k step ks.
DEV bf16x8_t frag_row(const uint16_t *t, int r0, int ks, int lane) {
    const int r = r0 + (lane & 31);
    const int c = 2 * ks + (lane >> 5);
    return __builtin_bit_cast(bf16x8_t, ld_u32x4(t + r * BK + 8 * row_swz(r, c)));
}

// Fragment for MFMA operand columns [n0, n0+32) from a col tile, k step ks.
// Lane l gets column n0 + (l & 31) at k = 16 ks + 8 (l >> 5) + 0..7, built
// from two transposing reads of 4 k rows each.
DEV bf16x8_t frag_col(const uint16_t *t, int n0, int ks, int lane) {
    const int i = lane & 15, grp = lane >> 4;
    const int n = n0 + 16 * (grp & 1) + 4 * (i & 3);
    const int kb = 16 * ks + 8 * (grp >> 1) + (i >> 2);
    bf16x4_t v[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int kr = kb + 4 * q;
        const int off = kr * BN + 16 * col_swz(kr, n >> 4) + (n & 15);
        v[q] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDSP bf16x4_t *)(t + off));
    }
    return bf16x8_t{v[0][0], v[0][1], v[0][2], v[0][3], v[1][0], v[1][1], v[1][2], v[1][3]};
}



// Two LDS stages, each operand its own object: the compiler then knows the
// tile being read never aliases the tile being filled and does not stall the
// reads on the in-flight direct loads.  They live at file scope so that one
// kernel can run tiles of several products (each product's tile code uses
// the same arrays).
__shared__ __attribute__((aligned(16))) uint16_t lds_a0[TILE_ELEMS];
__shared__ __attribute__((aligned(16))) uint16_t lds_b0[TILE_ELEMS];
__shared__ __attribute__((aligned(16))) uint16_t lds_a1[TILE_ELEMS];
__shared__ __attribute__((aligned(16))) uint16_t lds_b1[TILE_ELEMS];
__shared__ int s_info[2];
// fused forward: first m-tile slot of every expert in the grouped raster
// (entry E: the total), and the plan's offsets [E+1]
__shared__ int s_tilebase[257];
__shared__ int s_offs[257];

// One output tile of product MODE: workgroup vb of a grid of nvb (a multiple
// of 8, so vb % 8 is the XCD the tile runs on).
// Fused forward: the longest a workgroup waits for a counter, in ticks of
// the 100 MHz real-time clock (0.2 s; a legitimate wait lasts a few tile
// times, well under 10 ms).  A wait that runs out sets bit 1 of the error
// word; once that bit is set every later wait returns at once, so a launch
// always ends soon after.
#ifndef MOE_FUSED_WAIT_TICKS
#define MOE_FUSED_WAIT_TICKS 20000000ull
#endif

// Poll *ctr until it reaches need (one thread).  Counters are written by
// other workgroups of the same launch with agent-scope release adds after
// their data; the data a waiter then reads was never read before in this
// launch by any workgroup, so no cache level can hold a stale copy of it.
DEV void poll_count(const int *ctr, int need, int *err) {
    const unsigned long long t0 = wall_clock64();
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < need) {
        if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 2) return;
        if (wall_clock64() - t0 > MOE_FUSED_WAIT_TICKS) {
            __hip_atomic_fetch_or(err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

DEV void wait_count(const int *ctr, int need, int *err) {
    if (threadIdx.x == 0) poll_count(ctr, need, err);
    __syncthreads();
}

// Publish a finished tile: every wave waits for its own stores, then one
// release add (which writes this XCD's L2 back) makes them visible to all XCDs.
// When every waiter runs on this XCD (local), the stores are already in the
// L2 they read through, so the add skips the write-back.
DEV void signal_done(int *ctr, bool local) {
    wait_vmcnt<0>();
    __syncthreads();
    if (threadIdx.x == 0) {
        if (local) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Four consecutive plan indices; plan positions carry no alignment beyond 4 bytes.
typedef int idx4_t __attribute__((ext_vector_type(4), aligned(4)));

// Epilogue outputs are streamed out with non-temporal stores: they are
// read by a later launch, not by this one, and allocating them in L2 would
// evict operand panels that concurrently running tiles still share.
DEV void st_nt(void *p, u32x4_t v) { __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(p)); }

template <int MODE, bool GROUPED, bool PERSISTENT = false>
DEV void gemm_tile(const GemmArgs &g, const int *__restrict__ a_rows, const int *__restrict__ b_rows,
                   int vb, int nvb) {
    using Tr = Traits<MODE>;
    int slot = 0;   // m-tile slot of a row product (fused forward dependencies)

    // In a persistent loop the thread index passes through an empty asm, so
    // the compiler cannot hoist this tile's per-thread addressing out of the
    // loop (holding it in registers across tiles spills).
    int tid_v = threadIdx.x;
    if constexpr (PERSISTENT) asm volatile("" : "+v"(tid_v));
    const int tid = tid_v;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // ---------------- tile assignment ----------------
    int e = 0, row0 = 0, row_end = 0, n0 = 0, ntile = 0;
    int m0 = 0, kbeg = 0, klen = 0;
    int ebase = 0;   // grouped row products: the expert's first plan row
    int tok_base = 0;   // weight gradients: the expert's first plan row of the whole plan
    if constexpr (Tr::GROUPED_ROWS) {
        const int ntn = (MODE == FWD_UP) ? g.N / (BN / 2) : g.N / BN;
        int mt = 0;
        if (!map_tile(vb, g.tiles_m, ntn, mt, ntile)) return;
        n0 = ntile * ((MODE == FWD_UP) ? BN / 2 : BN);
        if constexpr (GROUPED && PERSISTENT) {
            // the fused kernel keeps the grouped raster's prefix and the
            // offsets in LDS: each wave finds the expert of m-tile slot mt by
            // a ballot over them (no global loads, no barrier)
            e = -1;
            for (int base = 0; base < g.E && e < 0; base += 64) {
                const int ee = base + lane;
                const bool hit = ee < g.E && mt >= s_tilebase[ee] && mt < s_tilebase[ee + 1];
                const unsigned long long m = __ballot(hit);
                if (m) e = base + __builtin_ctzll(m);
            }
            e = uniform(e);
            if (e < 0) return;
            ebase = uniform(s_offs[e]);
            row0 = ebase + (mt - uniform(s_tilebase[e])) * BM;
            row_end = uniform(s_offs[e + 1]);
        } else if constexpr (GROUPED) {
            if (tid == 0) s_info[0] = -1;
            __syncthreads();
            if (tid < 64) {
                int cum = 0;
                for (int base = 0; base < g.E; base += 64) {
                    const int ee = base + lane;
                    const int cnt = ee < g.E ? g.offsets[ee + 1] - g.offsets[ee] : 0;
                    const int tiles = cnt > 0 ? (cnt + BM - 1) / BM : 0;
                    int x = tiles;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const int y = __shfl_up(x, off, 64);
                        if (lane >= off) x += y;
                    }
                    const int excl = cum + x - tiles;
                    if (ee < g.E && mt >= excl && mt < excl + tiles) {
                        s_info[0] = ee;
                        s_info[1] = mt - excl;
                    }
                    cum += __shfl(x, 63, 64);
                }
            }
            __syncthreads();
            e = uniform(s_info[0]);
            if (e < 0) return;
            ebase = uniform(g.offsets[e]);
            row0 = ebase + uniform(s_info[1]) * BM;
            row_end = uniform(g.offsets[e + 1]);
        } else {
            row0 = mt * BM;
            row_end = g.M;
            if (row0 >= row_end) return;
        }
        klen = g.K;
        slot = mt;
        if constexpr (Tr::CMB) {
            // fused dense forward: this token tile needs the up/gate tile of
            // its tokens in every expert, and the shared expert's
            if (g.dep) {
                if (tid < g.nseg)
                    poll_count(g.dep + min(s_tilebase[tid] + mt, g.dep_slots - 1), g.dep_need, g.err);
                else if (tid == g.nseg && g.dep2) poll_count(g.dep2 + mt, g.dep_need2, g.err);
                __syncthreads();
            }
        } else {
            if (g.dep) wait_count(g.dep + mt, g.dep_need, g.err);
        }
    } else {
        const int ntn = g.N / BN, ntm = g.M / BM;
        int cm = 0;   // (expert, m-tile) pair
        if (!map_tile_wgrad(vb, g.tiles_m / ntm, ntm, ntn, cm, ntile)) return;
        m0 = (cm % ntm) * BM;
        e = cm / ntm;
        n0 = ntile * BN;
        if constexpr (GROUPED) {
            kbeg = uniform(g.offsets[e]);
            klen = uniform(g.offsets[e + 1]) - kbeg;
            tok_base = g.tok_offsets ? uniform(g.tok_offsets[e]) : kbeg;
        } else {
            kbeg = 0;
            klen = g.K;
        }
        // an expert with no rows adds nothing to a running sum
        if (klen == 0 && g.accumulate) return;
    }

    // ---------------- direct-load set-up ----------------
    // Each thread issues LD_PER_OP (4) loads per operand per K step.  Load i
    // of wave w is wave-instruction q = LD_PER_OP w + i (0..31), writing 1 KB
    // of the stage's tile.
    //   row tile: instruction q covers rows 8 q .. 8 q + 7; lane -> row
    //             8 q + lane / 8, physical 16-byte chunk lane & 7.
    //   col tile: instruction q covers k rows 2 q, 2 q + 1; lane -> k row
    //             2 q + lane / 32, physical 16-byte slot lane & 31.
    const uint16_t *a_row[LD_PER_OP];   // row tile: row base (+ chunk), K offset added per step
    const uint16_t *a2_row[LD_PER_OP];
    const uint16_t *b_row[LD_PER_OP];
    const uint16_t *b2_row[LD_PER_OP];
    long a_col_off = 0, b_col_off = 0;              // col tile: column offset of this lane
    const uint16_t *b_col_base = nullptr;
    int lds_off[LD_PER_OP];
#pragma unroll
    for (int i = 0; i < LD_PER_OP; ++i) lds_off[i] = (LD_PER_OP * wave + i) * 512;   // bf16 elements (1 KB)

    // dense-routing products: element offsets of each load inside its
    // segment's operand, for the three row pitches a segment can have (routed,
    // shared, router); the segment only adds its base and K offset.  Every
    // operand here holds fewer than 2^31 elements.
    // token / output row of each load, its chunk, and (B col tiles) its column
    uint32_t cm_t[LD_PER_OP], cm_c[LD_PER_OP], cm_b[LD_PER_OP];   // filled once col_of exists
    if constexpr (Tr::CMB) {
    } else if constexpr (MODE == WGRAD_T) {
        // A^T rows m0 + r; its columns are the expert's positions (from
        // kbeg), or with a_local the tokens (from the token of plan row kbeg)
        const long acol0 = g.a_local ? kbeg - tok_base : kbeg;
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int r = ROWS_PER_LD * (LD_PER_OP * wave + i) + lane / (BK / 8);
            const int c = row_swz(r, lane % (BK / 8));
            a_row[i] = g.A + (long)(m0 + r) * g.lda + acol0 + 8 * c;
        }
    } else if constexpr (!Tr::A_COL) {
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int r = ROWS_PER_LD * (LD_PER_OP * wave + i) + lane / (BK / 8);
            const int c = row_swz(r, lane % (BK / 8));
            // rows past the region's end load its last row; their results are never stored
            const int p = min(row0 + r, row_end - 1);
            int phys = g.a_local ? p - ebase : a_rows ? a_rows[p] : p;
            phys = min(max(phys, 0), g.a_nrows - 1);
            a_row[i] = g.A + (long)phys * g.lda + 8 * c;
            if (MODE == BWD_DX) a2_row[i] = g.A2 + (long)phys * g.lda + 8 * c;
        }
    } else {
        a_col_off = m0;
    }
    if constexpr (Tr::CMB) {
        // set above
    } else if constexpr (MODE == WGRAD_TB) {
        // B^T rows n0 + r; its columns are the expert's positions (from
        // kbeg), or with b_local the tokens (from the token of plan row kbeg)
        const long bcol0 = g.b_local ? kbeg - tok_base : kbeg;
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int r = ROWS_PER_LD * (LD_PER_OP * wave + i) + lane / (BK / 8);
            const int c = row_swz(r, lane % (BK / 8));
            b_row[i] = g.B + (long)(n0 + r) * g.ldb + bcol0 + 8 * c;
        }
    } else if constexpr (!Tr::B_COL) {
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int r = ROWS_PER_LD * (LD_PER_OP * wave + i) + lane / (BK / 8);
            const int c = row_swz(r, lane % (BK / 8));
            const long n = n0 + r;
            b_row[i] = g.B + (long)e * g.b_estride + n * g.ldb + 8 * c;
            if (MODE == BWD_DX) b2_row[i] = g.B2 + (long)e * g.b_estride + n * g.ldb + 8 * c;
        }
    } else {
        b_col_base = g.B + (long)e * g.b_estride;
        b_col_off = n0;
    }

    // column (within the 256-wide tile) that this lane's 16-byte col-tile load covers
    auto col_of = [&](int kr) {
        const int slot = lane & 31;
        const int b = col_swz(kr, slot >> 1);       // logical 32-byte block
        return 16 * b + 8 * (slot & 1);
    };

    // dense routing: steps per routed segment, routed steps (E segments, two
    // per expert for dX), shared steps, and the router step of dX
    constexpr int CM_H = (MODE == BWD_DX_CMB) ? 2 : 1;
    const int cm_sr = Tr::CMB ? g.segK / BK : 1;
    const int cm_nr = Tr::CMB ? g.nseg * CM_H * cm_sr : 0;
    const int cm_ss = Tr::CMB ? g.segK_s / BK : 1;
    const int cm_ns = (Tr::CMB && g.segK_s > 0) ? CM_H * cm_ss : 0;
    const int cm_nrt = (MODE == BWD_DX_CMB && g.Ar) ? 1 : 0;
    if constexpr (Tr::CMB) {
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int r = ROWS_PER_LD * (LD_PER_OP * wave + i) + lane / (BK / 8);
            // rows past the last token load the last token; they are never stored
            cm_t[i] = (uint32_t)min(row0 + r, row_end - 1);
            cm_c[i] = 8u * (uint32_t)row_swz(r, lane % (BK / 8));
            if constexpr (Tr::B_COL) {
                // the routed and shared down weights share the row pitch d
                const int kr = 2 * (LD_PER_OP * wave + i) + (lane >> 5);
                cm_b[i] = (uint32_t)(kr * g.ldb + n0 + col_of(kr));
            } else {
                cm_b[i] = (uint32_t)(n0 + r);
            }
        }
    }
    // segment sg: routed (expert sg / CM_H, half sg % CM_H), then shared
    // (half), then the router step; bases at the segment's first K step
    struct CmbSeg {
        const uint16_t *ab, *bb;
        uint32_t lda, ldb;
        int len;
    };
    const int cm_nsr = Tr::CMB ? g.nseg * CM_H : 0;
    const int cm_nsegs = cm_nsr + (cm_ns ? CM_H : 0) + cm_nrt;
    auto cmb_enter = [&](int sg) {
        CmbSeg c;
        if (sg < cm_nsr) {
            const int ex = sg / CM_H, half = sg - ex * CM_H;
            // the tokens' rows in expert ex's region; an offset that a
            // malformed plan would push past the buffer is clamped into it
            const int off = min(max(uniform(g.seg_offsets[ex]), g.a_row0), g.a_nrows - g.M);
            c.ab = (half ? g.A2 : g.A) + (long)off * g.lda;
            c.bb = (half ? g.B2 : g.B) + (long)ex * g.b_estride;
            c.lda = (uint32_t)g.lda;
            c.ldb = (uint32_t)g.ldb;
            c.len = cm_sr;
        } else if (sg < cm_nsr + (cm_ns ? CM_H : 0)) {
            const int half = sg - cm_nsr;
            c.ab = half ? g.As2 : g.As;
            c.bb = half ? g.Bs2 : g.Bs;
            c.lda = (uint32_t)g.lda_s;
            c.ldb = (uint32_t)g.ldb_s;
            c.len = cm_ss;
        } else {
            c.ab = g.Ar;
            c.bb = g.Br;
            c.lda = 64u;
            c.ldb = 64u;
            c.len = 1;
        }
        return c;
    };
    int cs_sg = 0, cs_st = 0;
    CmbSeg cs{};
    if constexpr (Tr::CMB) cs = cmb_enter(0);
    const int nk = Tr::CMB ? cm_nr + cm_ns + cm_nrt
                 : (MODE == BWD_DX) ? 2 * (g.K / BK) : (klen + BK - 1) / BK;
    const int nk_half = g.K / BK;

    // Forward col tiles: this lane's source for each of its loads at K step
    // 0, so the K loop only adds kt * BK rows (and never re-reads the weight
    // pointers, which a persistent kernel would otherwise reload every step).
    const long ldb = g.ldb;
    const uint16_t *bcol[LD_PER_OP];
    if constexpr (MODE == FWD_UP || MODE == FWD_DOWN) {
#pragma unroll
        for (int i = 0; i < LD_PER_OP; ++i) {
            const int kr = 2 * (LD_PER_OP * wave + i) + (lane >> 5);
            const int col = col_of(kr);
            if constexpr (MODE == FWD_UP) {
                // tile columns: 32-column groups alternate gate / up over the same f range
                const int fcol = (int)b_col_off + (col >> 6) * 32 + (col & 31);
                bcol[i] = (((col >> 5) & 1) ? g.B2 : g.B) + (long)e * g.b_estride + (long)kr * ldb + fcol;
            } else {
                bcol[i] = b_col_base + (long)kr * ldb + b_col_off + col;
            }
        }
    }

    // issue() in parts: the WGRAD k-row index fetch, the A loads, the B loads
    constexpr int LD_IDX = 1, LD_A = 2, LD_B = 4, LD_ALL = 7;
    int pa[LD_PER_OP], pb[LD_PER_OP];
    auto issue = [&](int kt, uint16_t *la, uint16_t *lb, int parts) {
        // WGRAD k rows come through the plan's token index: fetch every index
        // this K step needs first (scalar loads, one wait), then issue the
        // direct loads.  A wave's k rows are consecutive plan positions, so
        // inside the expert's range they take one 4-index load per 4 rows.
        if constexpr (Tr::CMB) {
            // steps run in order: the current segment's bases advance by one
            // K step per call, and a new segment is entered when one ends
            const int kl = cs_st * BK;
            // row offsets in 32 bits (token < 2^24, pitch < 2^21)
            if (parts & LD_A) {
#pragma unroll
                for (int i = 0; i < LD_PER_OP; ++i)
                    load_lds16(cs.ab + kl + (cm_t[i] * cs.lda + cm_c[i]), la + lds_off[i]);
            }
            if (!(parts & LD_B)) return;   // the step advances with its B loads
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                if constexpr (Tr::B_COL)
                    load_lds16(cs.bb + (long)kl * cs.ldb + cm_b[i], lb + lds_off[i]);
                else
                    load_lds16(cs.bb + kl + (cm_b[i] * cs.ldb + cm_c[i]), lb + lds_off[i]);
            }
            if (++cs_st == cs.len) {
                cs_st = 0;
                if (++cs_sg < cm_nsegs) cs = cmb_enter(cs_sg);
            }
            return;
        }
        if constexpr (Tr::WG) if (parts & LD_IDX) {
            int ia[2 * LD_PER_OP], ib[2 * LD_PER_OP];
            // this wave's k rows are the 2 LD_PER_OP consecutive positions from r0
            const int r0 = kt * BK + 2 * LD_PER_OP * wave;
            if (kt * BK + BK <= klen) {
                // the whole step lies in the expert's range: one scalar load per operand
                static_assert(LD_PER_OP % 2 == 0, "4-index scalar loads");
                const int abase = g.a_local ? 0 : kbeg, bbase = g.b_local ? 0 : kbeg;
#pragma unroll
                for (int q = 0; q < 2 * LD_PER_OP; q += 4) {
                    if (a_rows && !g.a_local) {
                        const idx4_t v = *reinterpret_cast<const idx4_t *>(a_rows + kbeg + r0 + q);
                        ia[q] = v[0]; ia[q + 1] = v[1]; ia[q + 2] = v[2]; ia[q + 3] = v[3];
                    } else {
#pragma unroll
                        for (int u = 0; u < 4; ++u) ia[q + u] = abase + r0 + q + u;
                    }
                    if (b_rows && !g.b_local) {
                        const idx4_t v = *reinterpret_cast<const idx4_t *>(b_rows + kbeg + r0 + q);
                        ib[q] = v[0]; ib[q + 1] = v[1]; ib[q + 2] = v[2]; ib[q + 3] = v[3];
                    } else {
#pragma unroll
                        for (int u = 0; u < 4; ++u) ib[q + u] = bbase + r0 + q + u;
                    }
                }
            } else {
                // the expert's last step: positions past its end are clamped to
                // its last row (their loads read zeros instead)
#pragma unroll
                for (int q = 0; q < 2 * LD_PER_OP; ++q) {
                    const int p = kbeg + min(r0 + q, klen - 1);
                    ia[q] = g.a_local ? p - kbeg : a_rows ? a_rows[p] : p;
                    ib[q] = g.b_local ? p - kbeg : b_rows ? b_rows[p] : p;
                }
            }
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                pa[i] = min(max((lane >> 5) ? ia[2 * i + 1] : ia[2 * i], 0), g.a_nrows - 1);
                pb[i] = min(max((lane >> 5) ? ib[2 * i + 1] : ib[2 * i], 0), g.b_nrows - 1);
            }
        }
        // ---- operand A ----
        if (!(parts & LD_A)) {
        } else if constexpr (!Tr::A_COL) {
            const bool second = (MODE == BWD_DX) && kt >= nk_half;
            const int kk = (second ? kt - nk_half : kt) * BK;
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i)
                load_lds16((second ? a2_row[i] : a_row[i]) + kk, la + lds_off[i]);
        } else {
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                const int kr = 2 * (LD_PER_OP * wave + i) + (lane >> 5);
                const int kk = kt * BK + kr;
                const int col = col_of(kr);
                const uint16_t *src = kk < klen ? g.A + (long)pa[i] * g.lda + a_col_off + col
                                                : g.zeros + col;
                load_lds16(src, la + lds_off[i]);
            }
        }
        // ---- operand B ----
        if (!(parts & LD_B)) {
        } else if constexpr (!Tr::B_COL) {
            const bool second = (MODE == BWD_DX) && kt >= nk_half;
            const int kk = (second ? kt - nk_half : kt) * BK;
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i)
                load_lds16((second ? b2_row[i] : b_row[i]) + kk, lb + lds_off[i]);
        } else {
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                const int kr = 2 * (LD_PER_OP * wave + i) + (lane >> 5);
                const int kk = kt * BK + kr;
                const int col = col_of(kr);
                const uint16_t *src;
                if constexpr (Tr::WG) {
                    src = kk < klen ? b_col_base + (long)pb[i] * ldb + b_col_off + col
                                    : g.zeros + col;
                } else {
                    src = bcol[i] + (long)(kt * BK) * ldb;
                }
                load_lds16(src, lb + lds_off[i]);
            }
        }
    };

    // FWD_UP with dense routing: the gate weights of this lane's epilogue
    // rows, loaded now so that their round trips are long over by then
    float wrow[TM][2];
    if constexpr (MODE == FWD_UP) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int p = min(row0 + wm * WM + 32 * i + (lane >> 2) + 16 * t, row_end - 1);
                wrow[i][t] = g.rowscale ? g.rowscale[p] : 1.0f;
            }
    }

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    auto load_frags = [&](const uint16_t *la, const uint16_t *lb, int ks, bf16x8_t (&af)[TM],
                          bf16x8_t (&bfr)[TN]) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if constexpr (Tr::A_COL) af[i] = frag_col(la, wm * WM + 32 * i, ks, lane);
            else af[i] = frag_row(la, wm * WM + 32 * i, ks, lane);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            if constexpr (Tr::B_COL) bfr[j] = frag_col(lb, wn * WN + 32 * j, ks, lane);
            else bfr[j] = frag_row(lb, wn * WN + 32 * j, ks, lane);
        }
    };
    // Fragments are double-buffered in registers: the reads of k sub-step
    // ks + 1 are issued before the MFMAs of sub-step ks (the scheduling
    // barrier stops the compiler from sinking them to their uses), so LDS
    // latency hides behind the matrix cores.
    //
    // The next tile's direct loads (step nkt, into stages nla / nlb) go out in
    // two halves, one operand ahead of the MFMAs of sub-step 0 and the other
    // ahead of sub-step 1, instead of all at the step's start: every wave of
    // every CU of an XCD reaches the step's barrier together, and 64 KB per CU
    // requested at once queue in L2.  The K-contiguous row tile goes first.
    // Measured on the training step: 3-6 % per GEMM; later halves (sub-steps
    // 0 and 2, or 1 and 2) were slower, and so was the column tile first.
    // The gathered WGRAD (index fetch and both operands as column tiles)
    // keeps all its loads at the step's start.
    constexpr int SPLIT = (MODE == WGRAD) ? 0 : (Tr::A_COL && !Tr::B_COL) ? 2 : 1;
    auto compute = [&](const uint16_t *la, const uint16_t *lb, int nkt, uint16_t *nla, uint16_t *nlb) {
        bf16x8_t af[2][TM], bfr[2][TN];
        load_frags(la, lb, 0, af[0], bfr[0]);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int cur = ks & 1;
            if (ks + 1 < BK / 16) load_frags(la, lb, ks + 1, af[cur ^ 1], bfr[cur ^ 1]);
            if (SPLIT != 0 && nkt >= 0 && ks < 2) {
                const int first = SPLIT == 1 ? LD_A : LD_B;
                asm volatile("" ::: "memory");   // after this sub-step's LDS reads
                issue(nkt, nla, nlb, ks == 0 ? (LD_IDX | first) : (LD_A | LD_B) ^ first);
                asm volatile("" ::: "memory");
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j],
                                                                        acc[i][j], 0, 0, 0);
        }
    };

    // Double-buffered K loop, unrolled by two so each half names its stages:
    // wait for this wave's loads of the tile about to be read, barrier (all
    // waves' loads landed, all reads of the other stage done), then compute on
    // this stage while the next tile streams into the other one.
    if (nk > 0) issue(0, lds_a0, lds_b0, LD_ALL);
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        wait_vmcnt<0>();
        barrier_no_fence();
        if constexpr (SPLIT == 0) {
            issue(kt + 1, lds_a1, lds_b1, LD_ALL);
            asm volatile("" ::: "memory");   // keep the loads ahead of this step's LDS reads
        }
        compute(lds_a0, lds_b0, kt + 1, lds_a1, lds_b1);
        wait_vmcnt<0>();
        barrier_no_fence();
        if constexpr (SPLIT == 0) {
            if (kt + 2 < nk) issue(kt + 2, lds_a0, lds_b0, LD_ALL);
            asm volatile("" ::: "memory");
        }
        compute(lds_a1, lds_b1, kt + 2 < nk ? kt + 2 : -1, lds_a0, lds_b0);
    }
    if (kt < nk) {
        wait_vmcnt<0>();
        barrier_no_fence();
        compute(lds_a0, lds_b0, -1, nullptr, nullptr);
    }
    __syncthreads();

    // ---------------- epilogues ----------------
    // 32x32 accumulator layout: lane l, register q -> row 8*(q/4) + 4*(l/32) + q%4, column l%32.
    // Row-tile outputs go through a per-wave LDS scratch (32 rows x WN fp32,
    // pitch SP) so every global access of the epilogue is a 16-byte vector of
    // 8 consecutive columns of one row.
    const int lrow = lane & 31, lhalf = lane >> 5;
    constexpr int SP = WN + 4;                   // scratch pitch in floats (16-byte rows, few bank conflicts)
    constexpr int LPR = WN / 8;                  // lanes per staged row
    constexpr int RPP = 64 / LPR;                // staged rows per pass
    constexpr int WPA = NWAVES / 4;              // waves sharing one 32 KB stage array
    static_assert(WPA * 32 * SP + WAVES_N * BM <= TILE_ELEMS / 2, "epilogue scratch fits a stage array");
    uint16_t *scr_base = (wave / WPA) == 0 ? lds_a0 : (wave / WPA) == 1 ? lds_b0
                       : (wave / WPA) == 2 ? lds_a1 : lds_b1;
    float *scr = reinterpret_cast<float *>(scr_base) + (wave % WPA) * 32 * SP;
    auto stage = [&](int i) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q)
                scr[(8 * (q >> 2) + 4 * lhalf + (q & 3)) * SP + 32 * j + lrow] = acc[i][j][q];
    };
    auto read8 = [&](int row, int c) {
        const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(scr + row * SP + c);
        const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(scr + row * SP + c + 4);
        return f32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    };
    if constexpr (MODE == FWD_UP) {
        // staged columns 64 jp + 0..31 hold the gate, 64 jp + 32..63 the up
        // projection of the same 32 f columns.  With dense routing each row
        // is scaled by its gate weight (loaded before the K loop).
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            stage(i);
#pragma unroll
            for (int jp = 0; jp < TN / 2; ++jp) {
                const long fcol0 = n0 + (wn * WN / 64 + jp) * 32;
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int row = (lane >> 2) + 16 * t, c = 8 * (lane & 3);
                    const int p = row0 + wm * WM + 32 * i + row;
                    const f32x8 a = read8(row, 64 * jp + c), b = read8(row, 64 * jp + 32 + c);
                    if (p < row_end) {
                        // dense routing keeps w h for the folded combine
                        const float ws = wrow[i][t];
                        f32x8 h;
#pragma unroll
                        for (int k = 0; k < 8; ++k) h[k] = ws * (silu_f(a[k]) * b[k]);
                        const long o = (long)p * g.ldc + fcol0 + c;
                        if (g.C) st_nt(g.C + o, pack_bf8(h));
                        if (g.C2) {
                            st_nt(g.C2 + o, pack_bf8(a));
                            st_nt(g.C3 + o, pack_bf8(b));
                        }
                    }
                }
            }
        }
    } else if constexpr (MODE == FWD_DOWN || MODE == BWD_DX || MODE == FWD_DOWN_CMB ||
                         MODE == BWD_DX_CMB) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            stage(i);
#pragma unroll
            for (int t = 0; t < 32 / RPP; ++t) {
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const int p = row0 + wm * WM + 32 * i + row;
                f32x8 v = read8(row, c);
                if (p >= row_end) continue;
                const long o = (long)p * g.ldc + n0 + wn * WN + c;
                if (Tr::CMB && g.Cf) {
                    if (g.accumulate) {
                        const f32x8 prev = ld_f32x8(g.Cf + o);
#pragma unroll
                        for (int q = 0; q < 8; ++q) v[q] = prev[q] + v[q];
                    }
                    if (!g.C) {
                        st_f32x8(g.Cf + o, v);
                        continue;
                    }
                }
                st_nt(g.C + o, pack_bf8(v));
            }
        }
    } else if constexpr (MODE == BWD_DGRAD) {
        float *red = reinterpret_cast<float *>(lds_a0) + WPA * 32 * SP;  // [WAVES_N][BM]
        // The forward's a and b (and the row's gate weight) of each 32-row
        // group are loaded one group ahead, so their round trips overlap the
        // previous group's work instead of each waiting in turn.  Rows past
        // the region's end load its last row and are never stored.
        constexpr int NP = 32 / RPP;
        u32x4_t av[2][NP], bv[2][NP];
        float wvs[2][NP];
        auto fetch_ab = [&](int i, u32x4_t (&a)[NP], u32x4_t (&b)[NP], float (&wv)[NP]) {
#pragma unroll
            for (int t = 0; t < NP; ++t) {
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const int p = min(row0 + wm * WM + 32 * i + row, row_end - 1);
                const long o = (long)p * g.ldc + n0 + wn * WN + c;
                a[t] = ld_u32x4(g.E1 + o);
                b[t] = ld_u32x4(g.E2 + o);
                wv[t] = g.rowscale ? g.rowscale[p] : 1.0f;
            }
        };
        fetch_ab(0, av[0], bv[0], wvs[0]);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if (i + 1 < TM) fetch_ab(i + 1, av[(i + 1) & 1], bv[(i + 1) & 1], wvs[(i + 1) & 1]);
            stage(i);
#pragma unroll
            for (int t = 0; t < NP; ++t) {
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const int rl = wm * WM + 32 * i + row;
                const int p = row0 + rl;
                const f32x8 dhp = read8(row, c);
                float prod = 0.f;
                if (p < row_end) {
                    const float wv = wvs[i & 1][t];
                    const long o = (long)p * g.ldc + n0 + wn * WN + c;
                    const u32x4_t ap = av[i & 1][t], bp = bv[i & 1][t];
                    f32x8 da, db, hw;
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const float a = (k & 1) ? bf_hi(ap[k >> 1]) : bf_lo(ap[k >> 1]);
                        const float b = (k & 1) ? bf_hi(bp[k >> 1]) : bf_lo(bp[k >> 1]);
                        const float sg = sigmoid_f(a);
                        const float sl = a * sg;
                        const float h = sl * b;
                        prod = prod + dhp[k] * h;
                        const float dh = wv * dhp[k];
                        da[k] = dh * b * (sg * (1.0f + a * (1.0f - sg)));
                        db[k] = dh * sl;
                        hw[k] = wv * h;
                    }
                    st_nt(g.C + o, pack_bf8(da));
                    st_nt(g.C2 + o, pack_bf8(db));
                    if (g.C3) st_nt(g.C3 + o, pack_bf8(hw));
                }
                // sum over the LPR lanes holding this row's WN columns (fixed butterfly order)
#pragma unroll
                for (int m = 1; m < LPR; m <<= 1) prod = prod + shfl_xor_f(prod, m);
                if (lane % LPR == 0) red[wn * BM + rl] = prod;
            }
        }
        __syncthreads();
        if (g.dgpart && tid < BM) {
            const int p = row0 + tid;
            if (p < row_end) {
                float sum = red[tid];
#pragma unroll
                for (int w = 1; w < WAVES_N; ++w) sum = sum + red[w * BM + tid];
                g.dgpart[(long)p * g.dg_ld + ntile] = sum;
            }
        }
    } else {  // WGRAD, WGRAD_T, WGRAD_TB
        // accumulator q of MFMA tile (i, j) is row 8 (q >> 2) + 4 lhalf + (q & 3)
        // of the 32-row block, column lrow
        float *out = g.Cf + (long)e * g.c_estride + (long)(m0 + wm * WM + 4 * lhalf) * g.ldc
                   + n0 + wn * WN + lrow;
        const long ld = g.ldc;
        if (g.accumulate) {
            // read all 16 old values of an MFMA tile before adding, so the
            // loads overlap instead of each waiting for its own round trip
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    float *o = out + (long)(32 * i) * ld + 32 * j;
                    float old[16];
#pragma unroll
                    for (int q = 0; q < 16; ++q) old[q] = o[(8 * (q >> 2) + (q & 3)) * ld];
#pragma unroll
                    for (int q = 0; q < 16; ++q) __builtin_nontemporal_store(old[q] + acc[i][j][q], &o[(8 * (q >> 2) + (q & 3)) * ld]);
                }
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    float *o = out + (long)(32 * i) * ld + 32 * j;
#pragma unroll
                    for (int q = 0; q < 16; ++q) __builtin_nontemporal_store(acc[i][j][q], &o[(8 * (q >> 2) + (q & 3)) * ld]);
                }
        }
    }
    if constexpr (Tr::GROUPED_ROWS) {
        if (g.sig) signal_done(g.sig + slot, g.sig_local);
    }
}

template <int MODE, bool GROUPED>
__global__ __launch_bounds__(NTHREADS, 1) void gemm_kernel(GemmArgs g, const int *__restrict__ a_rows,
                                                          const int *__restrict__ b_rows) {
    gemm_tile<MODE, GROUPED>(g, a_rows, b_rows, blockIdx.x, gridDim.x);
}

// Several grouped weight-gradient products, optionally followed by one
// grouped up/gate product, in one launch.  Product i owns workgroups
// [start[i], start[i+1]) (each start a multiple of 8, so its XCD raster is
// the one a launch of its own would have).  Workgroups are dispatched in
// order: the long weight-gradient tiles go first and the short up/gate tiles
// fill the tail.
constexpr int MAX_BATCH = 4;
struct GemmBatch {
    GemmArgs g[MAX_BATCH];
    int start[MAX_BATCH + 1];
    int mode[MAX_BATCH];   // weight-gradient products: 0 WGRAD, 1 WGRAD_T, 2 WGRAD_TB
    int n;          // products
    int up_last;    // the last product is FWD_UP
};

__global__ __launch_bounds__(NTHREADS, 1) void gemm_batch_kernel(GemmBatch bt) {
    const int b = blockIdx.x;
    int i = 0;
#pragma unroll
    for (int j = 1; j < MAX_BATCH; ++j)
        if (j < bt.n && b >= bt.start[j]) i = j;
    const int vb = b - bt.start[i], nvb = bt.start[i + 1] - bt.start[i];
    if (bt.up_last && i == bt.n - 1)
        gemm_tile<FWD_UP, true>(bt.g[i], bt.g[i].a_rows, bt.g[i].b_rows, vb, nvb);
    else if (bt.mode[i] == 1)
        gemm_tile<WGRAD_T, true>(bt.g[i], bt.g[i].a_rows, bt.g[i].b_rows, vb, nvb);
    else if (bt.mode[i] == 2)
        gemm_tile<WGRAD_TB, true>(bt.g[i], bt.g[i].a_rows, bt.g[i].b_rows, vb, nvb);
    else
        gemm_tile<WGRAD, true>(bt.g[i], bt.g[i].a_rows, bt.g[i].b_rows, vb, nvb);
}

template <int MODE>
hipError_t launch_mode(GemmArgs g, int tiles_m, int ntn, hipStream_t st, long grid_blocks = 0) {
    const long tiles = (long)tiles_m * ntn;
    if (tiles <= 0) return hipSuccess;
    g.tiles_m = tiles_m;
    const unsigned grid = (unsigned)(grid_blocks > 0 ? grid_blocks : raster_grid(tiles_m, ntn));
    if (g.offsets)
        gemm_kernel<MODE, true><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g, g.a_rows, g.b_rows);
    else
        gemm_kernel<MODE, false><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g, g.a_rows, g.b_rows);
    return hipGetLastError();
}

}  // namespace

int gemm_tile_m() { return BM; }
int gemm_tile_n() { return BN; }

// m-tile slots of a row problem.  Grouped: an upper bound on
// sum_e ceil(M_e / BM), which is at most rows / BM + groups; slots past the
// actual tiles return at once.
static int mtiles(const GemmArgs &g, long rows, int groups) {
    return g.offsets ? (int)(rows / BM + (groups > 0 ? groups : 1)) : (int)((rows + BM - 1) / BM);
}

hipError_t launch_gemm_fwd_up(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mode<FWD_UP>(g, mtiles(g, rows, groups), g.N / (BN / 2), st);
}
hipError_t launch_gemm_fwd_down(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mode<FWD_DOWN>(g, mtiles(g, rows, groups), g.N / BN, st);
}
hipError_t launch_gemm_bwd_dgrad(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mode<BWD_DGRAD>(g, mtiles(g, rows, groups), g.N / BN, st);
}
hipError_t launch_gemm_bwd_dx(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mode<BWD_DX>(g, mtiles(g, rows, groups), g.N / BN, st);
}
hipError_t launch_gemm_fwd_down_cmb(const GemmArgs &g, hipStream_t st) {
    if (g.offsets) return hipErrorInvalidValue;   // token tiles are not grouped
    return launch_mode<FWD_DOWN_CMB>(g, (g.M + BM - 1) / BM, g.N / BN, st);
}
hipError_t launch_gemm_bwd_dx_cmb(const GemmArgs &g, hipStream_t st) {
    if (g.offsets) return hipErrorInvalidValue;
    return launch_mode<BWD_DX_CMB>(g, (g.M + BM - 1) / BM, g.N / BN, st);
}
hipError_t launch_gemm_wgrad_tb(const GemmArgs &g, int groups, hipStream_t st) {
    return launch_mode<WGRAD_TB>(g, groups * (g.M / BM), g.N / BN, st,
                                 wgrad_grid(groups, g.M / BM, g.N / BN));
}
hipError_t launch_gemm_wgrad_t(const GemmArgs &g, int groups, hipStream_t st) {
    return launch_mode<WGRAD_T>(g, groups * (g.M / BM), g.N / BN, st,
                                wgrad_grid(groups, g.M / BM, g.N / BN));
}
hipError_t launch_gemm_wgrad(const GemmArgs &g, int groups, hipStream_t st) {
    return launch_mode<WGRAD>(g, groups * (g.M / BM), g.N / BN, st,
                              wgrad_grid(groups, g.M / BM, g.N / BN));
}

hipError_t launch_gemm_wgrad_batch(const GemmArgs *wg, int nw, int groups, const GemmArgs *up,
                                   long up_rows, hipStream_t st, const int *modes) {
    GemmBatch bt{};
    if (nw < 0 || nw + (up ? 1 : 0) > MAX_BATCH) return hipErrorInvalidValue;
    long at = 0;
    bt.n = 0;
    for (int i = 0; i < nw; ++i) {
        GemmArgs g = wg[i];
        if (!g.offsets) return hipErrorInvalidValue;
        const int ntm = g.M / BM, ntn = g.N / BN;
        g.tiles_m = groups * ntm;
        const long blocks = wgrad_grid(groups, ntm, ntn);
        if ((long)g.tiles_m * ntn <= 0) continue;
        bt.g[bt.n] = g;
        bt.mode[bt.n] = modes ? modes[i] : 0;
        if (bt.mode[bt.n] < 0 || bt.mode[bt.n] > 2) return hipErrorInvalidValue;
        bt.start[bt.n] = (int)at;
        at += blocks;
        ++bt.n;
    }
    if (up) {
        GemmArgs g = *up;
        if (!g.offsets) return hipErrorInvalidValue;
        const int ntn = g.N / (BN / 2);
        g.tiles_m = mtiles(g, up_rows, groups);
        const long tiles = (long)g.tiles_m * ntn;
        if (tiles > 0) {
            bt.g[bt.n] = g;
            bt.start[bt.n] = (int)at;
            at += raster_grid(g.tiles_m, ntn);
            ++bt.n;
            bt.up_last = 1;
        }
    }
    if (bt.n == 0) return hipSuccess;
    bt.start[bt.n] = (int)at;
    gemm_batch_kernel<<<dim3((unsigned)at), dim3(NTHREADS), 0, st>>>(bt);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fused persistent forward.
//
// One workgroup per CU loops over a work queue until it is empty.  Work
// items, in queue order: the shared expert's up/gate tiles (first: they
// need nothing), the routed up/gate tiles, the shared down tiles, the
// routed down tiles, and the combine of blocks of FUSED_TB tokens.  There is
// one queue per XCD (workgroup index mod 8); queue x holds, for each GEMM,
// exactly the tiles the XCD-aware raster gives XCD x in a launch of its own,
// in the same order, so every tile keeps its L2 neighbours.  A down tile
// waits until all up/gate tiles of its m-tile slot have been published; a
// combine block waits for the down tiles holding its tokens' routes.  Items
// are taken in queue order and wait only on items earlier in some queue,
// which running workgroups hold and finish without waiting on later ones:
// the launch cannot deadlock (and every wait is bounded besides).
//
// Each tile is computed by the same code as in the separate launches and
// the combine adds in the same order, so results are bitwise those of the
// unfused forward.
namespace {

constexpr int FUSED_TB = 16;   // tokens per combine item (k <= 16: <= 256 route checks)

struct FusedFwd {
    GemmArgs g[4];       // shared up, routed up, shared down, routed down (dense: folded down)
    int dense;           // every token routes to every expert: no combine phase
    int grid[4];         // workgroups of each product's own launch (multiple of 8)
    int base[6];         // queue item index where each phase starts (5 phases)
    int *queue;          // [8] tickets
    int *err;
    const uint16_t *Yexp, *Ysh;
    const float *topk_w;
    const int *route_pos, *topk_idx, *offsets;
    const int *down_done_r, *down_done_s;
    int need_r, need_s;  // n-tiles per m-tile of the routed / shared down products
    // dense routing with every expert's m-tiles a multiple of 32: an XCD's
    // routed up/gate items are taken token group first (groups_x token groups
    // of 4 m-tiles per expert on each XCD), so the folded down tiles of its
    // first token group are ready long before the up/gate phase ends; 0 keeps
    // the raster's expert-major order
    int groups_x;
    int tpg_up;          // routed up/gate tiles per group (4 m-tiles x its n-tiles)
    int xcc_queues;      // the device is 8 XCDs: serve the queue of the XCD read from XCC_ID
    int T, d, k, E, R;
    uint16_t *Y;
};

__shared__ int s_ticket;
__shared__ int s_cpos[FUSED_TB * 16];     // combine item: route positions (-1: none)
__shared__ float s_cwt[FUSED_TB * 16];    // and gate weights, [token][slot]

DEV void fused_combine(const FusedFwd &fa, int blk) {
    const int t0 = blk * FUSED_TB;
    if (t0 >= fa.T) return;
    const int t1 = min(fa.T, t0 + FUSED_TB);
    const int tid = threadIdx.x;
    // dependencies: the routed down m-tile of every route of these tokens,
    // and the shared down m-tiles of the tokens (one thread each)
    const int npairs = (t1 - t0) * fa.k;
    if (tid < npairs) {
        const long j = (long)t0 * fa.k + tid;
        const int p = fa.route_pos[j], e = fa.topk_idx[j];
        // the item's positions and weights, read once for all its column chunks
        s_cpos[tid] = (p >= 0 && p < fa.R) ? p : -1;
        s_cwt[tid] = fa.topk_w[j];
        if (p >= 0 && p < fa.R && e >= 0 && e < fa.E)
            poll_count(fa.down_done_r + s_tilebase[e] + (p - fa.offsets[e]) / BM, fa.need_r, fa.err);
    } else if (fa.Ysh && tid < npairs + 2) {
        poll_count(fa.down_done_s + (tid == npairs ? t0 : t1 - 1) / BM, fa.need_s, fa.err);
    }
    __syncthreads();
    // the combine of the unfused path: fp32 from Ysh, + w * Yexp in slot
    // order.  Work unit u = (token, 8-column chunk); each thread takes two
    // units per pass with all of their loads in flight together (one
    // workgroup per CU leaves few waves to hide memory latency).
    const int nc = fa.d / 8;
    const int units = (t1 - t0) * nc;
    for (int u0 = tid; u0 < units; u0 += 2 * NTHREADS) {
        int tt[2], cc[2], pos[2][16];
        float wt[2][16];
        u32x4_t rows[2][16], sh[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int u = min(u0 + h * NTHREADS, units - 1);
            tt[h] = t0 + u / nc;
            cc[h] = u % nc;
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                pos[h][s] = -1;
                wt[h][s] = 0.f;
                if (s < fa.k) {
                    pos[h][s] = s_cpos[(tt[h] - t0) * fa.k + s];
                    wt[h][s] = s_cwt[(tt[h] - t0) * fa.k + s];
                }
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int s = 0; s < 16; ++s)
                if (s < fa.k) rows[h][s] = ld_u32x4(fa.Yexp + (long)max(pos[h][s], 0) * fa.d + 8 * cc[h]);
            if (fa.Ysh) sh[h] = ld_u32x4(fa.Ysh + (long)tt[h] * fa.d + 8 * cc[h]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (h == 1 && u0 + NTHREADS >= units) break;
            float acc[8];
            if (fa.Ysh) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[2 * q] = bf_lo(sh[h][q]);
                    acc[2 * q + 1] = bf_hi(sh[h][q]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = 0.f;
            }
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                if (s < fa.k && pos[h][s] >= 0) {
                    const u32x4_t v = rows[h][s];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc[2 * q] = acc[2 * q] + wt[h][s] * bf_lo(v[q]);
                        acc[2 * q + 1] = acc[2 * q + 1] + wt[h][s] * bf_hi(v[q]);
                    }
                }
            }
            u32x4_t o;
#pragma unroll
            for (int q = 0; q < 4; ++q) o[q] = pack_bf2(acc[2 * q], acc[2 * q + 1]);
            st_u32x4(fa.Y + (long)tt[h] * fa.d + 8 * cc[h], o);
        }
    }
}

// The XCD this wave runs on (hardware register XCC_ID, bits 3:0).
DEV int xcc_id() { return __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 7; }

__global__ __launch_bounds__(NTHREADS, 1) void fused_forward_kernel(FusedFwd fa) {
    const int tid = threadIdx.x;
    // every workgroup serves the queue of the XCD it runs on, so a tile and
    // the items that wait for it share that XCD's L2 (on a device of another
    // shape, workgroup b serves queue b mod 8 and nothing is XCD-local)
    const int q = fa.xcc_queues ? xcc_id() : (int)(blockIdx.x & 7);
    // first m-tile slot of every expert (the grouped raster's prefix)
    if (tid < 64) {
        const int lane = tid;
        int cum = 0;
        for (int base = 0; base < fa.E; base += 64) {
            const int ee = base + lane;
            const int cnt = ee < fa.E ? fa.offsets[ee + 1] - fa.offsets[ee] : 0;
            const int tiles = cnt > 0 ? (cnt + BM - 1) / BM : 0;
            int x = tiles;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int y = __shfl_up(x, off, 64);
                if (lane >= off) x += y;
            }
            if (ee < fa.E) s_tilebase[ee] = cum + x - tiles;
            cum += __shfl(x, 63, 64);
        }
        if (lane == 0) s_tilebase[fa.E] = cum;
    }
    for (int i = tid; i <= fa.E; i += NTHREADS) s_offs[i] = fa.offsets[i];
    __syncthreads();
    // the next ticket is requested when an item starts, so its round trip
    // overlaps the item instead of stalling the workgroup between items
    if (tid == 0) s_ticket = __hip_atomic_fetch_add(fa.queue + q, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    int t = s_ticket;
    for (;;) {
        if (t >= fa.base[5]) break;
        int next = 0;
        if (tid == 0) next = __hip_atomic_fetch_add(fa.queue + q, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int P = 0;
#pragma unroll
        for (int i = 1; i < 5; ++i)
            if (t >= fa.base[i]) P = i;
        int j = t - fa.base[P];
        if (P == 1 && fa.groups_x > 0) {
            const int gi = j / fa.tpg_up, w = j % fa.tpg_up;   // this XCD's gi-th group
            if (gi < fa.E * fa.groups_x) j = ((gi % fa.E) * fa.groups_x + gi / fa.E) * fa.tpg_up + w;
        }
        const int vb = 8 * j + q;
        if (P == 0) gemm_tile<FWD_UP, false, true>(fa.g[0], fa.g[0].a_rows, fa.g[0].b_rows, vb, fa.grid[0]);
        else if (P == 1) gemm_tile<FWD_UP, true, true>(fa.g[1], fa.g[1].a_rows, fa.g[1].b_rows, vb, fa.grid[1]);
        else if (P == 2) gemm_tile<FWD_DOWN, false, true>(fa.g[2], fa.g[2].a_rows, fa.g[2].b_rows, vb, fa.grid[2]);
        else if (P == 3 && fa.dense) gemm_tile<FWD_DOWN_CMB, false, true>(fa.g[3], nullptr, nullptr, vb, fa.grid[3]);
        else if (P == 3) gemm_tile<FWD_DOWN, true, true>(fa.g[3], fa.g[3].a_rows, fa.g[3].b_rows, vb, fa.grid[3]);
        else fused_combine(fa, vb);
        __syncthreads();   // LDS of this item is free for the next
        if (tid == 0) s_ticket = next;
        __syncthreads();
        t = s_ticket;
    }
}

__global__ void fill_zero_kernel(int *p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

int cu_count() {
    static int n = 0;
    if (n == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            n = v;
        else
            n = 256;
    }
    return n;
}

}  // namespace

// counters: queue[8], up_done_s[tm_s], up_done_r[tm_r], down_done_s[tm_s], down_done_r[tm_r]
int fused_counter_ints(long T, long R, int E) {
    const long tm_s = (T + BM - 1) / BM, tm_r = R / BM + (E > 0 ? E : 1);
    return (int)(8 + 2 * tm_s + 2 * tm_r);
}

hipError_t launch_fused_forward(const GemmArgs &up_s, const GemmArgs &up_r, const GemmArgs &down_s,
                                const GemmArgs &down_r, bool shared, bool dense, long T, long R, int E,
                                const uint16_t *Yexp, const uint16_t *Ysh, const float *topk_w,
                                const int *route_pos, const int *topk_idx, const int *offsets, int d,
                                int k, uint16_t *Y, int *counters, int *err, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    if (k > 16 || E > 256) return hipErrorInvalidValue;
    const long tm_s = (T + BM - 1) / BM, tm_r = R / BM + (E > 0 ? E : 1);
    const int n = fused_counter_ints(T, R, E);
    int *queue = counters;
    int *up_done_s = counters + 8, *up_done_r = up_done_s + tm_s;
    int *down_done_s = up_done_r + tm_r, *down_done_r = down_done_s + tm_s;
    fill_zero_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(counters, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    if (dense && (down_r.offsets || down_r.nseg != E || E > 256)) return hipErrorInvalidValue;
    FusedFwd fa{};
    fa.dense = dense ? 1 : 0;
    fa.g[0] = up_s; fa.g[1] = up_r; fa.g[2] = down_s; fa.g[3] = down_r;
    const int ntn_up_s = shared ? up_s.N / (BN / 2) : 0, ntn_up_r = up_r.N / (BN / 2);
    const int ntn_dn_s = (shared && !dense) ? down_s.N / BN : 0, ntn_dn_r = down_r.N / BN;
    fa.g[0].tiles_m = shared ? (int)tm_s : 0;
    fa.g[1].tiles_m = (int)tm_r;
    fa.g[2].tiles_m = (shared && !dense) ? (int)tm_s : 0;
    // dense: the folded down product runs over token tiles
    fa.g[3].tiles_m = dense ? (int)tm_s : (int)tm_r;
    const long tiles[4] = {(long)fa.g[0].tiles_m * ntn_up_s, (long)tm_r * ntn_up_r,
                           (long)fa.g[2].tiles_m * ntn_dn_s, (long)fa.g[3].tiles_m * ntn_dn_r};
    fa.g[0].sig = up_done_s; fa.g[1].sig = up_done_r;
    fa.g[2].dep = up_done_s; fa.g[2].dep_need = ntn_up_s; fa.g[2].sig = down_done_s;
    fa.g[3].dep = up_done_r; fa.g[3].dep_need = ntn_up_r;
    if (dense) {
        // a token tile waits for its up/gate tile in every expert and in the
        // shared expert; nothing waits for it
        fa.g[3].dep2 = shared ? up_done_s : nullptr;
        fa.g[3].dep_need2 = ntn_up_s;
        fa.g[3].dep_slots = (int)tm_r;
    } else {
        fa.g[3].sig = down_done_r;
    }
    for (int i = 0; i < 4; ++i) fa.g[i].err = err;
    long at = 0;
    const int ntns[4] = {ntn_up_s, ntn_up_r, ntn_dn_s, ntn_dn_r};
    for (int i = 0; i < 4; ++i) {
        fa.grid[i] = tiles[i] > 0 ? (int)raster_grid(fa.g[i].tiles_m, ntns[i]) : 0;
        fa.base[i] = (int)at;
        at += fa.grid[i] / 8;
    }
    const long nblk = dense ? 0 : (T + FUSED_TB - 1) / FUSED_TB;
    fa.base[4] = (int)at;
    at += (nblk + 7) / 8;
    fa.base[5] = (int)at;
    fa.queue = queue;
    fa.err = err;
    fa.Yexp = Yexp; fa.Ysh = shared ? Ysh : nullptr;
    fa.topk_w = topk_w; fa.route_pos = route_pos; fa.topk_idx = topk_idx; fa.offsets = offsets;
    fa.down_done_r = down_done_r; fa.down_done_s = down_done_s;
    fa.need_r = ntn_dn_r; fa.need_s = ntn_dn_s;
    fa.T = (int)T; fa.d = d; fa.k = k; fa.E = E; fa.R = (int)R;
    fa.Y = Y;
    // Dense routing with T a multiple of 32 tiles: expert e's m-tile t is the
    // raster's slot e (T / BM) + t, in group (e T / BM + t) / 4, which goes
    // to the same XCD as the shared tile t and the token tile t of the folded
    // down product (group t / 4): every wait is XCD-local.
    // an MI355X in its 8-XCD mode: 256 CUs, 32 per XCD
    fa.xcc_queues = cu_count() == 256 ? 1 : 0;
    const bool local = fa.xcc_queues && dense && T % (32 * BM) == 0;
    fa.groups_x = local ? (int)(T / BM / 32) : 0;
    fa.tpg_up = RASTER_GM * ntn_up_r;
    fa.g[0].sig_local = fa.g[1].sig_local = local ? 1 : 0;
    const int grid = cu_count() / 8 * 8 > 0 ? cu_count() / 8 * 8 : 8;
    fused_forward_kernel<<<dim3(grid), dim3(NTHREADS), 0, st>>>(fa);
    return hipGetLastError();
}
