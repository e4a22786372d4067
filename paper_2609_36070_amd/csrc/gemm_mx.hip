// Grouped MXFP8 GEMMs of the routed experts (§3.4 "MXFP8 Support") on the
// gfx950 block-scaled MFMA v_mfma_scale_f32_32x32x64_f8f6f4 (E4M3 x E4M3,
// fp32 accumulation).  Per expert e and buffer positions p of e's region:
//
//   MX_UP    g = Xq[tok(p)] . Wg_q[e][n], u = Xq[tok(p)] . Wu_q[e][n];
//            H = silu(g) * u, quantised to MXFP8 along f (the activation
//            quantisation fused into the gated activation) -> Hq, Hs; g and
//            u kept in fp32 for the backward on request
//   MX_DOWN  Yexp = Hq[p] . Wd_q[e][n] -> bf16
//   MX_DGRAD dh' = dYq[tok(p)] . Wd_qd[e][n] (W_down rows quantised along d),
//            then the gated-activation backward on the saved fp32 A, B: dg
//            partials <dh', h>, dA = w dh' B silu'(A), dB = w dh' silu(A),
//            Hw = w h; dA, dB and Hw go out for the weight gradients (bf16,
//            or fp32 when the weight gradients quantise them) and dA, dB
//            quantised to MXFP8 along f (for the dX product)
//   MX_DX    dXperm = dAq[p] . Wg_qf[e][n] + dBq[p] . Wu_qf[e][n] (one K loop
//            over both halves; W_gate / W_up rows quantised along f) -> bf16
//   MX_WGRAD dW[e][m][n] = sum over e's padded token positions t of
//            A[m][t] B[n][t]: both operands quantised along the token axis
//            (X^T or (w h)^T, and dA^T, dB^T or dY^T) -> fp32, one tile per
//            (expert, m tile, n tile), K = the expert's padded range
//
// Every operand is a matrix of K-contiguous byte rows (A: token or position
// rows; B: one row per output column, the pre-quantised weight layout) with
// one E8M0 scale byte per row per 32 k.  The MFMA takes each row's two
// 32-blocks of a 64-wide k step as bytes 0-15 (block 0) and 16-31 (block 1)
// of every lane, lane l serving row l % 32 and supplying the scale of block
// l / 32; a lane therefore reads k [16h, 16h + 16) and [32 + 16h, 48 + 16h)
// of its row (h = l / 32), which matches what the other operand holds.
//
// Pipeline as in the BF16 kernels: 256 x 256 block tile, K step 128 bytes,
// two LDS stages filled by direct global->LDS loads (128-byte rows, chunk
// XOR (row >> 1) & 7), 8 waves of 128 x 64 (two per SIMD), tiles
// rastered XCD-aware.  The scale words of a K step (4 blocks of a row) go
// to LDS by the same direct loads, one stage ahead, together with the tiles.
#include "common.h"
#include "kernels.h"
#include "mx_common.h"

#define LDSP __attribute__((address_space(3)))

namespace {

constexpr int BM = 256, BN = 256, BK = 128;
#ifndef MOE_MX_WAVES_N
#define MOE_MX_WAVES_N 4
#endif
// 2 x 4 waves of 128 x 64 (two waves per SIMD, so one can issue matrix
// instructions while the other waits on its loads or the barrier); 2 x 2
// waves of 128 x 128 (one per SIMD, accumulators in AGPRs) with
// MOE_MX_WAVES_N=2.
constexpr int WAVES_M = 2, WAVES_N = MOE_MX_WAVES_N, NWAVES = WAVES_M * WAVES_N;
constexpr int NTHREADS = 64 * NWAVES;
constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N, TM = WM / 32, TN = WN / 32;
constexpr int TILE = BM * BK;                      // bytes per operand per stage
constexpr int LD_PER_OP = TILE / 1024 / NWAVES;    // 1 KB direct loads per operand per wave per step
static_assert(WN == 64 || WN == 128, "gate/up column pairs need 64- or 128-column wave tiles");

enum MxMode { MX_UP = 0, MX_DOWN = 1, MX_DGRAD = 2, MX_DX = 3, MX_WGRAD = 4 };

typedef int i32x8_t __attribute__((ext_vector_type(8)));

DEV int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

DEV int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Raw buffer resource over [p, p + bytes) (gfx9 word 3: 32-bit data format).
DEV __amdgpu_buffer_rsrc_t make_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

DEV void barrier_no_fence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int N>
DEV void wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// MFMA operand for rows [r0, r0 + 32) at k step ks (64 wide) of a stage tile.
DEV i32x8_t frag(const uint8_t *t, int r0, int ks, int lane) {
    const int r = r0 + (lane & 31), h = lane >> 5;
    const u32x4_t lo = ld_u32x4(t + r * BK + 16 * swz(r, 4 * ks + h));
    const u32x4_t hi = ld_u32x4(t + r * BK + 16 * swz(r, 4 * ks + 2 + h));
    return i32x8_t{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                   (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
}

template <int MODE>
__global__ __launch_bounds__(NTHREADS, 1) void gemm_mx_kernel(MxGemmArgs g, const int *__restrict__ a_rows) {
    // one LDS object for both stages of both operands: the K loop picks the
    // stage by a wave-uniform offset at run time (see there)
    __shared__ __attribute__((aligned(16))) uint8_t lds_all[4 * TILE];
    uint8_t *const lds_a0 = lds_all, *const lds_a1 = lds_all + TILE;
    uint8_t *const lds_b0 = lds_all + 2 * TILE, *const lds_b1 = lds_all + 3 * TILE;
    // scale words of the K step per stage: A tile rows; B tile columns (MX_UP:
    // 128 gate then 128 up columns of the tile's f range)
    __shared__ uint32_t sc_all[2 * BM + 2 * BN];
    uint32_t *const sc_a0 = sc_all, *const sc_a1 = sc_all + BM;
    uint32_t *const sc_b0 = sc_all + 2 * BM, *const sc_b1 = sc_all + 2 * BM + BN;
    __shared__ int s_info[2];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // ---------------- tile: expert region and rows ----------------
    int e = 0, row0 = 0, row_end = 0, n0 = 0, ntile = 0;
    uint32_t kbase = 0;   // MX_WGRAD: byte offset of the expert's padded token range
    int nk_w = 0;         // MX_WGRAD: K steps over that range
    if constexpr (MODE == MX_WGRAD) {
        const int ntm = g.M / BM;
        int cm = 0;
        if (!map_tile_wgrad(blockIdx.x, g.E, ntm, g.N / BN, cm, ntile)) return;
        e = cm / ntm;
        row0 = (cm % ntm) * BM;
        row_end = g.M;
        n0 = ntile * BN;
        kbase = (uint32_t)uniform(g.offsets[e]);
        nk_w = (uniform(g.offsets[e + 1]) - (int)kbase) / BK;
    } else {
        const int ntn = (MODE == MX_UP) ? g.N / (BN / 2) : g.N / BN;
        int mt = 0;
        if (!map_tile(blockIdx.x, g.tiles_m, ntn, mt, ntile)) return;
        n0 = ntile * ((MODE == MX_UP) ? BN / 2 : BN);
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
        row0 = uniform(g.offsets[e] + uniform(s_info[1]) * BM);
        row_end = uniform(g.offsets[e + 1]);
    }
    const long ks_row = g.K / 32;     // scale bytes per row

    // physical A row of tile row r (rows past the region's end repeat its last
    // row; their results are never stored)
    auto a_phys = [&](int r) {
        const int p = min(row0 + r, row_end - 1);
        const int phys = a_rows ? a_rows[p] : p;
        return min(max(phys, 0), g.a_nrows - 1);
    };
    // ---------------- direct-load set-up ----------------
    // Every operand is read through a buffer resource (base and size in
    // SGPRs): a load takes a 32-bit VGPR offset, the K step and any
    // wave-uniform row offset go in the scalar offset, and the hardware
    // returns zeros for any access past the operand's end.
    // Tile load i of wave w is wave instruction q = LD_PER_OP w + i: 1 KB = 8
    // rows of 128 bytes; lane -> row 8 q + lane / 8, physical chunk
    // (lane & 7) ^ ((4 (q & 1) + lane / 16) & 7).  Rows of B (and of an
    // ungathered A) are linear in q, so one VGPR per parity of q serves all
    // loads; a gathered A needs one per load.
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(g.A, g.a_bytes);
    // (B resources are built per load from the selected base: a conditional
    // between two resource values is not accepted by the host compilation)
    const int l8 = lane >> 3;
    const uint32_t col_even = 16u * (uint32_t)((lane & 7) ^ ((l8 >> 1) & 7));
    const uint32_t col_odd = 16u * (uint32_t)((lane & 7) ^ ((4 + (l8 >> 1)) & 7));
    const uint32_t K = (uint32_t)g.K;
    const uint32_t b_lane_even = (uint32_t)l8 * K + col_even, b_lane_odd = (uint32_t)l8 * K + col_odd;
    constexpr bool GATHER = (MODE == MX_UP || MODE == MX_DGRAD);
    uint32_t a_off[LD_PER_OP];   // gathered A only
#pragma unroll
    for (int i = 0; i < LD_PER_OP; ++i) {
        const int q = LD_PER_OP * wave + i;
        a_off[i] = GATHER ? (uint32_t)a_phys(8 * q + l8) * K + ((q & 1) ? col_odd : col_even) : 0u;
    }
    // scale DMA: 8 instructions of 64 words per K step (A rows 64 c + lane for
    // c < 4; B words 64 (c - 4) + lane), spread over the waves
    constexpr int SC_PER_WAVE = 8 / NWAVES;
    uint32_t sc_off[SC_PER_WAVE];
#pragma unroll
    for (int i = 0; i < SC_PER_WAVE; ++i) {
        const int c = SC_PER_WAVE * wave + i;
        if (c < 4) {
            sc_off[i] = (uint32_t)a_phys(64 * c + lane) * (uint32_t)ks_row;
        } else {
            const int wd = 64 * (c - 4) + lane;               // B scale word
            const uint32_t brow = (MODE == MX_UP)      ? (uint32_t)(e * g.N + n0 + (wd & 127))
                                : (MODE == MX_WGRAD) ? (uint32_t)(n0 + wd)
                                                     : (uint32_t)(e * g.N + n0 + wd);
            sc_off[i] = brow * (uint32_t)ks_row;
        }
    }

    const int nk_half = g.K / BK;
    const int nk = (MODE == MX_DX) ? 2 * nk_half : (MODE == MX_WGRAD) ? nk_w : nk_half;
    // parts: 1 = the A tile and the scale words, 2 = the B tile
    auto issue = [&](int kt_all, uint8_t *la, uint8_t *lb, uint32_t *sa, uint32_t *sb, int parts) {
        // MX_DX: the second half of the K loop reads dBq against the W_up rows
        const bool second = (MODE == MX_DX) && kt_all >= nk_half;
        const int kt = second ? kt_all - nk_half : kt_all;
        // MX_WGRAD: an operand shared by all experts starts at position 0
        const uint32_t kb = kbase + (uint32_t)kt * BK;
        const uint32_t kb_a = (MODE == MX_WGRAD && g.a_shared) ? (uint32_t)kt * BK : kb;
        const uint32_t kb_b = (MODE == MX_WGRAD && g.b_shared) ? (uint32_t)kt * BK : kb;
        if (parts & 1) {
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                const int q = LD_PER_OP * wave + i;
                if constexpr (GATHER) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (LDSP void *)(la + q * 1024), 16, a_off[i],
                                                             kb, 0, 0);
                } else {
                    // rows past the region (or the operand) hold results that are never stored
                    const uint32_t arow = (uint32_t)(row0 + 8 * q);
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(second ? g.A2 : g.A, g.a_bytes),
                                                             (LDSP void *)(la + q * 1024), 16,
                                                             (q & 1) ? b_lane_odd : b_lane_even,
                                                             arow * K + kb_a, 0, 0);
                }
            }
        }
        if (parts & 2) {
#pragma unroll
            for (int i = 0; i < LD_PER_OP; ++i) {
                const int q = LD_PER_OP * wave + i;
                // B row of instruction q less the lane part l8 (uniform); MX_UP: tile
                // rows 8 q .. 8 q + 7 lie in column group q / 4, gate or up
                const bool up = ((MODE == MX_UP) && ((q >> 2) & 1)) || second;
                const uint32_t brow = (MODE == MX_UP)
                    ? (uint32_t)(e * g.N + n0 + (q >> 3) * 32 + 8 * (q & 3))
                    : (uint32_t)((MODE == MX_WGRAD ? 0 : e * g.N) + n0 + 8 * q);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(up ? g.B2 : g.B, g.b_bytes),
                                                         (LDSP void *)(lb + q * 1024), 16,
                                                         (q & 1) ? b_lane_odd : b_lane_even,
                                                         brow * K + kb_b, 0, 0);
            }
        }
        if (!(parts & 1)) return;
#pragma unroll
        for (int i = 0; i < SC_PER_WAVE; ++i) {
            const int c = SC_PER_WAVE * wave + i;
            if (c < 4) {
                __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(second ? g.As2 : g.As, g.as_bytes),
                                                         (LDSP void *)(sa + 64 * c), 4, sc_off[i],
                                                         (MODE == MX_WGRAD ? kb_a / 32 : kbase / 32 + 4 * kt), 0, 0);
            } else {
                const bool up = ((MODE == MX_UP) && (c - 4 >= 2)) || second;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(up ? g.Bs2 : g.Bs, g.bs_bytes),
                                                         (LDSP void *)(sb + 64 * (c - 4)), 4,
                                                         sc_off[i], (MODE == MX_WGRAD ? kb_b / 32 : kbase / 32 + 4 * kt), 0, 0);
            }
        }
    };

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    const int h = lane >> 5;
    // Fragments one step ahead of their MFMAs: the A fragment of row tile
    // i + 1 (or of the next k sub-step's row tile 0) is read before the MFMAs
    // of row tile i, and each B fragment of the next k sub-step right after
    // its last MFMA of this one, into the same registers, so the LDS round
    // trips overlap the matrix unit with no extra registers.  The fragments
    // and scale words live here, across the two sub-step calls of a K step.
    constexpr int KS = BK / 64;
    static_assert(KS == 2, "two 64-wide k sub-steps per K step");
    uint32_t wa[TM], wb[TN];
    i32x8_t bfr[TN], a_cur;
    auto compute_ks = [&](const uint8_t *la, const uint8_t *lb, const uint32_t *sa, const uint32_t *sb,
                          int ks) {
        if (ks == 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i) wa[i] = sa[wm * WM + 32 * i + (lane & 31)];
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                // scale word of tile column wn WN + 32 j + lane % 32 (MX_UP: gate
                // words 0..127, up words 128..255 of the tile's f range)
                const int wd = (MODE == MX_UP) ? (j & 1) * 128 + (wn * WN / 64 + j / 2) * 32 + (lane & 31)
                                               : wn * WN + 32 * j + (lane & 31);
                wb[j] = sb[wd];
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[j] = frag(lb, wn * WN + 32 * j, 0, lane);
            a_cur = frag(la, wm * WM, 0, lane);
        }
        // this lane's scales: block 2 ks + h of its row / column
        const int sh = 8 * (2 * ks + h);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            i32x8_t a_nxt = a_cur;
            if (i + 1 < TM) a_nxt = frag(la, wm * WM + 32 * (i + 1), ks, lane);
            else if (ks + 1 < KS) a_nxt = frag(la, wm * WM, ks + 1, lane);
            const int sai = (int)((wa[i] >> sh) & 0xffu);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int sbj = (int)((wb[j] >> sh) & 0xffu);
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    a_cur, bfr[j], acc[i][j], 0, 0, 0, sai, 0, sbj);
                if (i == TM - 1 && ks + 1 < KS) bfr[j] = frag(lb, wn * WN + 32 * j, ks + 1, lane);
            }
            a_cur = a_nxt;
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Double-buffered K loop with the stage as a wave-uniform run-time
    // offset.  With both stages named in an unrolled pair of steps the
    // compiler keeps a lane address register per stage for every fragment
    // read, which at two waves per SIMD (256 registers, 128 of them
    // accumulators) spills inside the loop; with the offset added at each
    // read it needs 195-238 registers and none spill.
    //
    // The next step's B tile goes out before the MFMAs of sub-step 0 and its
    // A tile and scale words before those of sub-step 1 (the row products:
    // down 2.20 -> 2.12 ms, training step -0.9 %; A first was slower).  The
    // weight gradients keep all their loads at the step's start (split, they
    // were 0.5 % slower).
    constexpr int FIRST = (MODE == MX_WGRAD) ? 3 : 2;
    if (nk > 0) issue(0, lds_a0, lds_b0, sc_a0, sc_b0, 3);
    int cur = 0;
#pragma clang loop unroll(disable)
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<0>();
        barrier_no_fence();
        const int nxt = uniform(cur ^ 1);
        uint8_t *nla = lds_all + nxt * TILE, *nlb = lds_all + (2 + nxt) * TILE;
        uint32_t *nsa = sc_all + nxt * BM, *nsb = sc_all + 2 * BM + nxt * BN;
        const uint8_t *la = lds_all + cur * TILE, *lb = lds_all + (2 + cur) * TILE;
        const uint32_t *sa = sc_all + cur * BM, *sb = sc_all + 2 * BM + cur * BN;
        if (kt + 1 < nk) issue(kt + 1, nla, nlb, nsa, nsb, FIRST);
        asm volatile("" ::: "memory");   // keep the loads ahead of this step's LDS reads
        compute_ks(la, lb, sa, sb, 0);
        if (FIRST != 3 && kt + 1 < nk) {
            asm volatile("" ::: "memory");
            issue(kt + 1, nla, nlb, nsa, nsb, 3 ^ FIRST);
            asm volatile("" ::: "memory");
        }
        compute_ks(la, lb, sa, sb, 1);
        cur = nxt;
    }
    __syncthreads();

    // ---------------- epilogue ----------------
    // accumulator layout: lane l, register q -> row 8 (q / 4) + 4 (l / 32) + q % 4,
    // column l % 32; rows go through a per-wave LDS scratch (32 x WN fp32)
    const int lrow = lane & 31, lhalf = lane >> 5;
    constexpr int SP = WN + 4;
    constexpr int WPA = NWAVES >= 4 ? NWAVES / 4 : 1;
    uint8_t *scr_base = (wave / WPA) == 0 ? lds_a0 : (wave / WPA) == 1 ? lds_b0
                      : (wave / WPA) == 2 ? lds_a1 : lds_b1;
    float *scr = reinterpret_cast<float *>(scr_base) + (wave % WPA) * 32 * SP;
    static_assert(WPA * 32 * SP * 4 <= TILE, "epilogue scratch fits a stage array");
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
    if constexpr (MODE == MX_UP) {
        // staged columns 64 jp + 0..31 hold the gate, 64 jp + 32..63 the up
        // projection of the same 32 f columns: one MXFP8 block of H per row
        // and pair, spread over 4 lanes
        const long hs_row = g.N / 32;
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
                    float hv[8];
                    float amax = 0.f;
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        hv[k] = silu_f(a[k]) * b[k];
                        amax = fmaxf(amax, fabsf(hv[k]));
                    }
                    amax = fmaxf(amax, shfl_xor_f(amax, 1));
                    amax = fmaxf(amax, shfl_xor_f(amax, 2));
                    const int s = mx_shared_exp(amax);
                    if (p < row_end) {
                        *reinterpret_cast<u32x2_t *>(g.C + (long)p * g.N + fcol0 + c) =
                            e4m3_pack8(hv, s);
                        if ((lane & 3) == 0) g.Cs[(long)p * hs_row + fcol0 / 32] = (uint8_t)(s + 127);
                        if (g.Sa) {   // pre-activations for the backward, fp32
                            float *sa = g.Sa + (long)p * g.N + fcol0 + c;
                            float *sb = g.Sb + (long)p * g.N + fcol0 + c;
                            st_f32x8(sa, a);
                            st_f32x8(sb, b);
                        }
                    }
                }
            }
        }
    } else if constexpr (MODE == MX_DGRAD) {
        // per row: the gated-activation backward on the saved A, B, then dA
        // and dB out in bf16 and quantised along f (a 32-column block is 4
        // neighbouring lanes of one row); <dh', h> summed over the row's
        // columns in a fixed order (lanes, then waves)
        constexpr int LPR = WN / 8, RPP = 64 / LPR;
        static_assert(WAVES_N <= 4, "one dg partial array per wave column");
        auto red_of = [&](int w) {
            return reinterpret_cast<float *>(w == 0 ? sc_a0 : w == 1 ? sc_b0 : w == 2 ? sc_a1 : sc_b1);
        };
        const long fs_row = g.N / 32;
        // The saved a, b and the row's gate weight of pass u = (i, t) are
        // loaded PF passes ahead through a small register queue, so their
        // round trips overlap the passes in between instead of each pass
        // waiting for its own.  Rows past the region's end read its last row.
        constexpr int NP = 32 / RPP, NU = TM * NP, PF = 4;
        f32x8 qa[PF], qb[PF];
        float qw[PF];
        auto fetch = [&](int u, f32x8 &a, f32x8 &b, float &w) {
            const int row = lane / LPR + RPP * (u % NP), c = 8 * (lane % LPR);
            const int pl = min(row0 + wm * WM + 32 * (u / NP) + row, row_end - 1);
            const long o = (long)pl * g.N + n0 + wn * WN + c;
            a = ld_f32x8(g.E1 + o);
            b = ld_f32x8(g.E2 + o);
            w = g.rowscale[pl];
        };
#pragma unroll
        for (int q = 0; q < PF; ++q)
            if (q < NU) fetch(q, qa[q], qb[q], qw[q]);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            stage(i);
            // not unrolled: a body this size unrolled 8 x 4 times makes the
            // compiler keep i dynamic and the accumulators in scratch
#pragma unroll 1
            for (int t = 0; t < NP; ++t) {
                const int u = i * NP + t;
                const f32x8 av = qa[0], bv = qb[0];
                const float wv = qw[0];
#pragma unroll
                for (int q = 0; q + 1 < PF; ++q) { qa[q] = qa[q + 1]; qb[q] = qb[q + 1]; qw[q] = qw[q + 1]; }
                if (u + PF < NU) fetch(u + PF, qa[PF - 1], qb[PF - 1], qw[PF - 1]);
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const int rl = wm * WM + 32 * i + row;
                const int p = row0 + rl;
                const int pl = min(p, row_end - 1);
                const f32x8 dhp = read8(row, c);
                const int col = n0 + wn * WN + c;
                const long o = (long)pl * g.N + col;
                f32x8 dav, dbv, hw;
                float prod = 0.f, amax_a = 0.f, amax_b = 0.f;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const float a = av[k], b = bv[k];
                    const float sg = sigmoid_f(a);
                    const float sl = a * sg;
                    const float h = sl * b;
                    prod = prod + dhp[k] * h;
                    const float dh = wv * dhp[k];
                    dav[k] = dh * b * (sg * (1.0f + a * (1.0f - sg)));
                    dbv[k] = dh * sl;
                    hw[k] = wv * h;
                    amax_a = fmaxf(amax_a, fabsf(dav[k]));
                    amax_b = fmaxf(amax_b, fabsf(dbv[k]));
                }
                amax_a = fmaxf(amax_a, shfl_xor_f(amax_a, 1));
                amax_a = fmaxf(amax_a, shfl_xor_f(amax_a, 2));
                amax_b = fmaxf(amax_b, shfl_xor_f(amax_b, 1));
                amax_b = fmaxf(amax_b, shfl_xor_f(amax_b, 2));
                const int sa = mx_shared_exp(amax_a), sb = mx_shared_exp(amax_b);
                if (p < row_end) {
                    if (g.Cf1) {   // fp32 for the token-axis quantisers
                        st_f32x8(g.Cf1 + o, dav);
                        st_f32x8(g.Cf2 + o, dbv);
                        st_f32x8(g.Cf3 + o, hw);
                    } else {
                        st_u32x4(g.Cb + o, pack_bf8(dav));
                        st_u32x4(g.Cb2 + o, pack_bf8(dbv));
                        st_u32x4(g.Cb3 + o, pack_bf8(hw));
                    }
                    *reinterpret_cast<u32x2_t *>(g.C + o) = e4m3_pack8(dav, sa);
                    *reinterpret_cast<u32x2_t *>(g.C2 + o) = e4m3_pack8(dbv, sb);
                    if ((lane & 3) == 0) {
                        g.Cs[(long)p * fs_row + col / 32] = (uint8_t)(sa + 127);
                        g.Cs2[(long)p * fs_row + col / 32] = (uint8_t)(sb + 127);
                    }
                } else {
                    prod = 0.f;
                }
#pragma unroll
                for (int m = 1; m < LPR; m <<= 1) prod = prod + shfl_xor_f(prod, m);
                if (lane % LPR == 0) red_of(wn)[rl] = prod;
            }
        }
        __syncthreads();
        if (g.dgpart && tid < BM) {
            const int p = row0 + tid;
            if (p < row_end) {
                float sum = red_of(0)[tid];
#pragma unroll
                for (int w = 1; w < WAVES_N; ++w) sum = sum + red_of(w)[tid];
                g.dgpart[(long)p * g.dg_ld + ntile] = sum;
            }
        }
    } else if constexpr (MODE == MX_WGRAD) {
        // fp32 rows of dW[e]; M and N are multiples of the tile, so every
        // staged row is a real one
        constexpr int LPR = WN / 8, RPP = 64 / LPR;
        float *out = g.Cf + (long)e * g.M * g.N;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            stage(i);
#pragma unroll
            for (int t = 0; t < 32 / RPP; ++t) {
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const f32x8 v = read8(row, c);
                float *o = out + (long)(row0 + wm * WM + 32 * i + row) * g.N + n0 + wn * WN + c;
                *reinterpret_cast<f32x4_t *>(o) = f32x4_t{v[0], v[1], v[2], v[3]};
                *reinterpret_cast<f32x4_t *>(o + 4) = f32x4_t{v[4], v[5], v[6], v[7]};
            }
        }
    } else {   // MX_DOWN, MX_DX: bf16 rows
        constexpr int LPR = WN / 8, RPP = 64 / LPR;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            stage(i);
#pragma unroll
            for (int t = 0; t < 32 / RPP; ++t) {
                const int row = lane / LPR + RPP * t, c = 8 * (lane % LPR);
                const int p = row0 + wm * WM + 32 * i + row;
                const f32x8 v = read8(row, c);
                if (p < row_end)
                    st_u32x4(g.Cb + (long)p * g.N + n0 + wn * WN + c, pack_bf8(v));
            }
        }
    }
}

template <int MODE>
hipError_t launch_mx_mode(MxGemmArgs g, int tiles_m, int ntn, hipStream_t st) {
    const long tiles = (long)tiles_m * ntn;
    if (tiles <= 0) return hipSuccess;
    g.tiles_m = tiles_m;
    const unsigned grid = (unsigned)raster_grid(tiles_m, ntn);
    gemm_mx_kernel<MODE><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g, g.a_rows);
    return hipGetLastError();
}

int mx_mtiles(long rows, int groups) { return (int)(rows / BM + (groups > 0 ? groups : 1)); }

}  // namespace

hipError_t launch_gemm_mx_up(const MxGemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mx_mode<MX_UP>(g, mx_mtiles(rows, groups), g.N / (BN / 2), st);
}
hipError_t launch_gemm_mx_down(const MxGemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mx_mode<MX_DOWN>(g, mx_mtiles(rows, groups), g.N / BN, st);
}

hipError_t launch_gemm_mx_dgrad(const MxGemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mx_mode<MX_DGRAD>(g, mx_mtiles(rows, groups), g.N / BN, st);
}

hipError_t launch_gemm_mx_dx(const MxGemmArgs &g, long rows, int groups, hipStream_t st) {
    return launch_mx_mode<MX_DX>(g, mx_mtiles(rows, groups), g.N / BN, st);
}

hipError_t launch_gemm_mx_wgrad(const MxGemmArgs &g, int groups, hipStream_t st) {
    if (groups <= 0 || g.M <= 0 || g.N <= 0 || g.E != groups) return hipSuccess;
    const unsigned grid = (unsigned)wgrad_grid(groups, g.M / BM, g.N / BN);
    gemm_mx_kernel<MX_WGRAD><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g, nullptr);
    return hipGetLastError();
}
