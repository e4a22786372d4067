// Grouped bf16 GEMMs of the expert FFNs on CDNA4 MFMA (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation, with the SwiGLU forward/backward fused into the
// epilogues (§2.1 FFN; §3.4 router-weight gradient fused into the gated
// activation backward).
//
// One kernel template serves five products; per expert e and buffer
// positions p of e's region [offsets[e], offsets[e+1]):
//
//   FWD_UP     A_e = X[tok(p)] W_gate[e], B_e = X[tok(p)] W_up[e],
//              H = silu(A) * B                         (A, B kept for backward)
//   FWD_DOWN   Yexp = H W_down[e]
//   BWD_DGRAD  dh' = dY[tok(p)] W_down[e]^T, then dg partials <dh', h>,
//              dA = w dh' * B * silu'(A), dB = w dh' * silu(A)
//   BWD_DX     dXperm = dA W_gate[e]^T + dB W_up[e]^T  (one K loop over both)
//   WGRAD      dW[e] = P_e^T Q_e, K = the expert's ragged route count
//
// The dispatch gather is fused into the operand loads: A rows (or WGRAD k
// rows) are read through the plan's token index, so no expert-contiguous
// copy of X or dY is ever written.  The shared expert runs through the same
// kernel as one ungrouped problem of T rows.
//
// Tiling: 256 x 256 x 64 block tile, 8 waves as 2 (M) x 4 (N), 128 x 64 per
// wave (4 x 2 MFMA tiles), double-buffered LDS (2 x 64 KB).  Operands live in
// LDS K-contiguous, 128-byte rows with the 16-byte chunk index XOR-swizzled
// by (row >> 1) & 7, so fragment reads and staging writes hit distinct banks.
// Operands stored N- or M-contiguous in HBM (W_gate/W_up/W_down in the
// forward, both operands of WGRAD) are transposed in registers during
// staging (8 k-rows x 4 columns per thread, v_perm byte selects).
//
// Tile order: n-tile fastest, so the blocks resident together share A panels
// and the whole B panel set of one expert stays cache-resident.  Each output
// element is owned by exactly one block and its K loop runs in a fixed
// order: results are bitwise deterministic (§3.4 "Determinism").
#include "common.h"
#include "kernels.h"

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NTHREADS = 512;
constexpr int WAVES_N = 4;
constexpr int WM = 128, WN = 64;
constexpr int TM = WM / 32, TN = WN / 32;
constexpr int TILE_ELEMS = BM * BK;  // per operand per stage (bf16 elements)

enum Mode { FWD_UP = 0, FWD_DOWN = 1, BWD_DGRAD = 2, BWD_DX = 3, WGRAD = 4 };

DEV int swz(int row, int c) { return c ^ ((row >> 1) & 7); }

// 8 k-rows x 4 columns (2 dwords per row) -> 4 columns x 8 k (16 bytes each).
DEV void transpose_8x4(const u32x2_t (&v)[8], u32x4_t (&o)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t lo0 = v[2 * q][0], hi0 = v[2 * q + 1][0];
        const uint32_t lo1 = v[2 * q][1], hi1 = v[2 * q + 1][1];
        o[0][q] = __builtin_amdgcn_perm(hi0, lo0, 0x05040100u);
        o[1][q] = __builtin_amdgcn_perm(hi0, lo0, 0x07060302u);
        o[2][q] = __builtin_amdgcn_perm(hi1, lo1, 0x05040100u);
        o[3][q] = __builtin_amdgcn_perm(hi1, lo1, 0x07060302u);
    }
}

template <int MODE>
struct Traits {
    static constexpr bool A_KM = (MODE == WGRAD);                       // A transposed in staging
    static constexpr bool B_KN = (MODE == FWD_UP || MODE == FWD_DOWN || MODE == WGRAD);
    static constexpr bool GROUPED_ROWS = (MODE != WGRAD);
};

template <int MODE, bool GROUPED>
__global__ __launch_bounds__(NTHREADS, 1) void gemm_kernel(GemmArgs g) {
    using Tr = Traits<MODE>;
    __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][TILE_ELEMS];  // [stage][A/B]
    __shared__ int s_info[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // ---------------- tile assignment ----------------
    int e = 0, row0 = 0, row_end = 0, n0 = 0, ntile = 0;
    int m0 = 0, kbeg = 0, klen = 0;
    if constexpr (Tr::GROUPED_ROWS) {
        const int ntn = (MODE == FWD_UP) ? g.N / (BN / 2) : g.N / BN;
        ntile = blockIdx.x % ntn;
        const int mt = blockIdx.x / ntn;
        n0 = ntile * ((MODE == FWD_UP) ? BN / 2 : BN);
        if constexpr (GROUPED) {
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
            if (s_info[0] < 0) return;
            e = s_info[0];
            row0 = g.offsets[e] + s_info[1] * BM;
            row_end = g.offsets[e + 1];
        } else {
            row0 = mt * BM;
            row_end = g.M;
            if (row0 >= row_end) return;
        }
        klen = g.K;
    } else {
        const int ntn = g.N / BN, ntm = g.M / BM;
        ntile = blockIdx.x % ntn;
        const int rest = blockIdx.x / ntn;
        m0 = (rest % ntm) * BM;
        e = rest / ntm;
        n0 = ntile * BN;
        if constexpr (GROUPED) {
            kbeg = g.offsets[e];
            klen = g.offsets[e + 1] - kbeg;
        } else {
            kbeg = 0;
            klen = g.K;
        }
    }

    // ---------------- staging set-up ----------------
    // MK / NK operands: thread -> chunk c = tid % 8 of rows tid/8 + 64*i.
    const int st_c = tid & 7, st_r = tid >> 3;
    // KN / KM operands: thread -> k-group kg = tid / 64 (8 k rows), column group cg = tid % 64.
    const int kg = tid >> 6, cg = tid & 63;

    const uint16_t *a_ptr[4];
    const uint16_t *a2_ptr[4];
    bool a_ok[4];
    const uint16_t *b_ptr[4];
    const uint16_t *b2_ptr[4];
    const uint16_t *bkn_base = nullptr;   // KN: column base of this thread (row 0)
    const uint16_t *akm_base = nullptr;   // KM: column base of this thread (row 0)

    if constexpr (!Tr::A_KM) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = row0 + st_r + 64 * i;
            a_ok[i] = p < row_end;
            int phys = a_ok[i] ? (g.a_rows ? g.a_rows[p] : p) : 0;
            phys = min(max(phys, 0), g.a_nrows - 1);
            a_ptr[i] = g.A + (long)phys * g.lda + 8 * st_c;
            a2_ptr[i] = (MODE == BWD_DX) ? g.A2 + (long)phys * g.lda + 8 * st_c : nullptr;
        }
    } else {
        akm_base = g.A + m0 + 4 * cg;
    }
    if constexpr (!Tr::B_KN) {
        // NK: row n of B is output column n0 + n, K contiguous.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int n = n0 + st_r + 64 * i;
            b_ptr[i] = g.B + (long)e * g.b_estride + (long)n * g.ldb + 8 * st_c;
            b2_ptr[i] = (MODE == BWD_DX) ? g.B2 + (long)e * g.b_estride + (long)n * g.ldb + 8 * st_c
                                         : nullptr;
        }
    } else {
        if constexpr (MODE == FWD_UP) {
            const int nn = 4 * cg;                       // B tile row (0..255)
            const int which = (nn >> 5) & 1;             // 0 gate, 1 up
            const int fcol = n0 + (nn >> 6) * 32 + (nn & 31);
            bkn_base = (which ? g.B2 : g.B) + (long)e * g.b_estride + fcol;
        } else {
            bkn_base = g.B + (long)e * g.b_estride + n0 + 4 * cg;
        }
    }

    u32x4_t ra[4];
    u32x2_t rkm[8];
    u32x4_t rb[4];
    u32x2_t rkn[8];

    const int nk = (MODE == BWD_DX) ? 2 * (g.K / BK) : (klen + BK - 1) / BK;
    const int nk_half = g.K / BK;

    auto load_global = [&](int kt) {
        if constexpr (!Tr::A_KM) {
            const bool second = (MODE == BWD_DX) && kt >= nk_half;
            const int kk = (second ? kt - nk_half : kt) * BK;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint16_t *src = (second ? a2_ptr[i] : a_ptr[i]) + kk;
                ra[i] = a_ok[i] ? ld_u32x4(src) : u32x4_t{0, 0, 0, 0};
            }
        } else {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int kr = kt * BK + 8 * kg + r;
                if (kr < klen) {
                    const int p = kbeg + kr;
                    int phys = g.a_rows ? g.a_rows[p] : p;
                    phys = min(max(phys, 0), g.a_nrows - 1);
                    u32x2_t v = ld_u32x2(akm_base + (long)phys * g.lda);
                    if (g.a_kscale) {
                        const float s = g.a_kscale[p];
                        v[0] = pack_bf2(bf_lo(v[0]) * s, bf_hi(v[0]) * s);
                        v[1] = pack_bf2(bf_lo(v[1]) * s, bf_hi(v[1]) * s);
                    }
                    rkm[r] = v;
                } else {
                    rkm[r] = u32x2_t{0, 0};
                }
            }
        }
        if constexpr (!Tr::B_KN) {
            const bool second = (MODE == BWD_DX) && kt >= nk_half;
            const int kk = (second ? kt - nk_half : kt) * BK;
#pragma unroll
            for (int i = 0; i < 4; ++i) rb[i] = ld_u32x4((second ? b2_ptr[i] : b_ptr[i]) + kk);
        } else {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int kr = kt * BK + 8 * kg + r;
                if constexpr (MODE == WGRAD) {
                    if (kr < klen) {
                        const int p = kbeg + kr;
                        int phys = g.b_rows ? g.b_rows[p] : p;
                        phys = min(max(phys, 0), g.b_nrows - 1);
                        rkn[r] = ld_u32x2(bkn_base + (long)phys * g.ldb);
                    } else {
                        rkn[r] = u32x2_t{0, 0};
                    }
                } else {
                    rkn[r] = ld_u32x2(bkn_base + (long)kr * g.ldb);
                }
            }
        }
    };

    auto store_lds = [&](int stage) {
        uint16_t *la = lds[stage][0];
        uint16_t *lb = lds[stage][1];
        if constexpr (!Tr::A_KM) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = st_r + 64 * i;
                st_u32x4(la + row * BK + 8 * swz(row, st_c), ra[i]);
            }
        } else {
            u32x4_t o[4];
            transpose_8x4(rkm, o);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int j = (q + (cg >> 2)) & 3;
                const int row = 4 * cg + j;
                st_u32x4(la + row * BK + 8 * swz(row, kg), o[j]);
            }
        }
        if constexpr (!Tr::B_KN) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = st_r + 64 * i;
                st_u32x4(lb + row * BK + 8 * swz(row, st_c), rb[i]);
            }
        } else {
            u32x4_t o[4];
            transpose_8x4(rkn, o);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int j = (q + (cg >> 2)) & 3;
                const int row = 4 * cg + j;
                st_u32x4(lb + row * BK + 8 * swz(row, kg), o[j]);
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

    if (nk > 0) {
        load_global(0);
        store_lds(0);
        __syncthreads();
    }
    const int lrow = lane & 31, lhalf = lane >> 5;
    for (int kt = 0; kt < nk; ++kt) {
        const int stage = kt & 1;
        if (kt + 1 < nk) load_global(kt + 1);
        const uint16_t *la = lds[stage][0];
        const uint16_t *lb = lds[stage][1];
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int c = 2 * ks + lhalf;
            bf16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wm * WM + 32 * i + lrow;
                af[i] = __builtin_bit_cast(bf16x8_t, ld_u32x4(la + row * BK + 8 * swz(row, c)));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int row = wn * WN + 32 * j + lrow;
                bfr[j] = __builtin_bit_cast(bf16x8_t, ld_u32x4(lb + row * BK + 8 * swz(row, c)));
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) store_lds(stage ^ 1);
        __syncthreads();
    }

    // ---------------- epilogues ----------------
    // 32x32 accumulator layout: lane l, register q -> row 8*(q/4) + 4*(l/32) + q%4, column l%32.
    if constexpr (MODE == FWD_UP) {
        const int fcol = n0 + wn * 32 + lrow;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int p = row0 + wm * WM + 32 * i + 8 * (q >> 2) + 4 * lhalf + (q & 3);
                if (p < row_end) {
                    const float a = acc[i][0][q], b = acc[i][1][q];
                    const long o = (long)p * g.ldc + fcol;
                    g.C[o] = f2bf(silu_f(a) * b);
                    if (g.C2) {
                        g.C2[o] = f2bf(a);
                        g.C3[o] = f2bf(b);
                    }
                }
            }
    } else if constexpr (MODE == FWD_DOWN || MODE == BWD_DX) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = n0 + wn * WN + 32 * j + lrow;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int p = row0 + wm * WM + 32 * i + 8 * (q >> 2) + 4 * lhalf + (q & 3);
                    if (p < row_end) g.C[(long)p * g.ldc + col] = f2bf(acc[i][j][q]);
                }
            }
    } else if constexpr (MODE == BWD_DGRAD) {
        float *red = reinterpret_cast<float *>(&lds[0][0][0]);  // [WAVES_N][BM]
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int rl = wm * WM + 32 * i + 8 * (q >> 2) + 4 * lhalf + (q & 3);
                const int p = row0 + rl;
                const bool ok = p < row_end;
                const float wv = (ok && g.rowscale) ? g.rowscale[p] : 1.0f;
                float prod = 0.f;
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int col = n0 + wn * WN + 32 * j + lrow;
                    if (ok) {
                        const long o = (long)p * g.ldc + col;
                        const float a = bf2f(g.E1[o]), b = bf2f(g.E2[o]);
                        const float sg = 1.0f / (1.0f + expf(-a));
                        const float sl = a * sg;
                        const float dhp = acc[i][j][q];
                        prod = prod + dhp * (sl * b);
                        const float dh = wv * dhp;
                        g.C[o] = f2bf(dh * b * (sg * (1.0f + a * (1.0f - sg))));
                        g.C2[o] = f2bf(dh * sl);
                    }
                }
                // sum over the 32 columns held by this half-wave (fixed butterfly order)
#pragma unroll
                for (int off = 16; off >= 1; off >>= 1) prod = prod + shfl_xor_f(prod, off);
                if (lrow == 0) red[wn * BM + rl] = prod;
            }
        __syncthreads();
        if (g.dgpart && tid < BM) {
            const int p = row0 + tid;
            if (p < row_end) {
                float s = red[0 * BM + tid] + red[1 * BM + tid];
                s = s + red[2 * BM + tid];
                s = s + red[3 * BM + tid];
                g.dgpart[(long)p * g.dg_ld + ntile] = s;
            }
        }
    } else {  // WGRAD
        float *out = g.Cf + (long)e * g.c_estride;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = n0 + wn * WN + 32 * j + lrow;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int m = m0 + wm * WM + 32 * i + 8 * (q >> 2) + 4 * lhalf + (q & 3);
                    out[(long)m * g.ldc + col] = acc[i][j][q];
                }
            }
    }
}

template <int MODE>
hipError_t launch_mode(const GemmArgs &g, unsigned grid, hipStream_t st) {
    if (grid == 0) return hipSuccess;
    if (g.offsets)
        gemm_kernel<MODE, true><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g);
    else
        gemm_kernel<MODE, false><<<dim3(grid), dim3(NTHREADS), 0, st>>>(g);
    return hipGetLastError();
}

}  // namespace

int gemm_tile_m() { return BM; }
int gemm_tile_n() { return BN; }

// Upper bound on the m-tiles of a grouped problem with `rows` total rows over
// `groups` groups: sum_e ceil(M_e / BM) <= rows / BM + groups.
static unsigned grouped_mtiles(long rows, int groups) {
    return (unsigned)(rows / BM + (groups > 0 ? groups : 1));
}

hipError_t launch_gemm_fwd_up(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    const unsigned mt = g.offsets ? grouped_mtiles(rows, groups) : (unsigned)((rows + BM - 1) / BM);
    return launch_mode<FWD_UP>(g, mt * (unsigned)(g.N / (BN / 2)), st);
}
hipError_t launch_gemm_fwd_down(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    const unsigned mt = g.offsets ? grouped_mtiles(rows, groups) : (unsigned)((rows + BM - 1) / BM);
    return launch_mode<FWD_DOWN>(g, mt * (unsigned)(g.N / BN), st);
}
hipError_t launch_gemm_bwd_dgrad(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    const unsigned mt = g.offsets ? grouped_mtiles(rows, groups) : (unsigned)((rows + BM - 1) / BM);
    return launch_mode<BWD_DGRAD>(g, mt * (unsigned)(g.N / BN), st);
}
hipError_t launch_gemm_bwd_dx(const GemmArgs &g, long rows, int groups, hipStream_t st) {
    const unsigned mt = g.offsets ? grouped_mtiles(rows, groups) : (unsigned)((rows + BM - 1) / BM);
    return launch_mode<BWD_DX>(g, mt * (unsigned)(g.N / BN), st);
}
hipError_t launch_gemm_wgrad(const GemmArgs &g, int groups, hipStream_t st) {
    const unsigned tiles = (unsigned)(groups * (g.M / BM) * (g.N / BN));
    return launch_mode<WGRAD>(g, tiles, st);
}
