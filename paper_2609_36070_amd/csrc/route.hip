// Router: logits = X W_r + bias on MFMA, then per-token top-k and the
// renormalised softmax weights (§2.1: the router scores every expert for a
// token, keeps the k best and gives each a weight).
//
// Layout: 16 MT tokens per block, NW waves (8, or 4 when 256 experts make
// the partial sums large).  The d axis is cut into 64-wide chunks dealt
// round-robin to the waves (split-K); each wave accumulates 16 MT x EPAD
// partial logits with v_mfma_f32_16x16x32_bf16 reading X rows straight from
// HBM and the transposed router W_r^T from L2.  The partial sums are added in
// wave order, so the result is deterministic.  The selection then runs on
// groups of lanes per token (up to 64 experts) or as a radix search per
// token (128 or more).
#include "common.h"
#include "kernels.h"

namespace {

// WrT[e][kk] = W_r[kk][e] (zero rows for E <= e < EPAD).
__global__ __launch_bounds__(256) void wr_transpose_kernel(const uint16_t *__restrict__ Wr,
                                                           uint16_t *__restrict__ WrT,
                                                           int d, int E, int EPAD) {
    long i = (long)blockIdx.x * 256 + threadIdx.x;
    if (i >= (long)EPAD * d) return;
    int e = (int)(i / d), kk = (int)(i % d);
    WrT[i] = e < E ? Wr[(long)kk * E + e] : (uint16_t)0;
}

// Top-k of one token's logits.  Each logit maps to an unsigned key with the
// same order (-0 and +0 share one key; a NaN ranks as -inf; every real key
// is above 0), and an entry (key, id) ranks above another when its key is
// larger or, for equal keys, its id is smaller: ties go to the lower expert
// id.  L = EPAD / 16 lanes share a token, 16 experts each.  Each lane keeps
// its best KP entries (KP = k rounded up to a power of two) sorted by rank,
// inserting its experts in ascending id; the L lists are then merged in
// log2 L rounds with the lane at distance s (the elementwise better of one
// list and the other reversed holds the best KP of both, as a bitonic
// sequence, which log2 KP half-cleaner stages sort).  Every lane of the
// group ends with the token's best KP entries; the first k are the
// selection.  Lane 0 of the group puts them in ascending id order and writes
// ids and weights exp(z - zmax) / sum, the sum taken in ascending id order.
DEV uint32_t logit_key(float z) {
    z = z == z ? z : -INFINITY;
    z = z == 0.f ? 0.f : z;
    const uint32_t u = __float_as_uint(z);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
DEV float key_logit(uint32_t key) {
    return __uint_as_float((key & 0x80000000u) ? (key ^ 0x80000000u) : ~key);
}
DEV bool ranks_above(uint32_t ka, int ia, uint32_t kb, int ib) {
    return ka > kb || (ka == kb && ia < ib);
}
// put the better of slots a, b first
DEV void order2(uint32_t &ka, int &ia, uint32_t &kb, int &ib) {
    const bool sw = ranks_above(kb, ib, ka, ia);
    const uint32_t k0 = ka, k1 = kb;
    const int i0 = ia, i1 = ib;
    ka = sw ? k1 : k0;
    kb = sw ? k0 : k1;
    ia = sw ? i1 : i0;
    ib = sw ? i0 : i1;
}

template <int EPAD, int KP>
DEV void select_topk(const float *zs, int ld, int BT, int NW, int t0, int T, int E, int k,
                     int *__restrict__ topk_idx, float *__restrict__ topk_w) {
    constexpr int PE = EPAD < 16 ? EPAD : 16;      // experts per lane
    constexpr int L = EPAD / PE;                    // lanes per token
    constexpr int TW = 64 / L;                      // tokens per wave
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int sub = l % L;
    for (int tb = w * TW; tb < BT; tb += NW * TW) {
        const int tt = min(tb + l / L, BT - 1), t = t0 + tb + l / L;
        float zr[PE];
#pragma unroll
        for (int i = 0; i < PE; ++i) zr[i] = zs[tt * ld + sub * PE + i];
        uint32_t bk[KP];
        int bi[KP];
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            bk[j] = 0u;
            bi[j] = 0;
        }
#pragma unroll
        for (int i = 0; i < PE; ++i) {
            uint32_t key = sub * PE + i < E ? logit_key(zr[i]) : 0u;
            int id = sub * PE + i;
#pragma unroll
            for (int j = 0; j < KP; ++j) order2(bk[j], bi[j], key, id);
        }
#pragma unroll
        for (int st = 1; st < L; st <<= 1) {
            uint32_t pk[KP];
            int pi[KP];
#pragma unroll
            for (int j = 0; j < KP; ++j) {
                pk[j] = (uint32_t)__shfl_xor((int)bk[j], st, 64);
                pi[j] = __shfl_xor(bi[j], st, 64);
            }
#pragma unroll
            for (int j = 0; j < KP; ++j) order2(bk[j], bi[j], pk[KP - 1 - j], pi[KP - 1 - j]);
#pragma unroll
            for (int len = KP / 2; len >= 1; len >>= 1)
#pragma unroll
                for (int j = 0; j < KP; ++j)
                    if ((j & len) == 0) order2(bk[j], bi[j], bk[j + len], bi[j + len]);
        }
        if (sub != 0 || tb + l / L >= BT || t >= T) continue;
        const float zmax = key_logit(bk[0]);
        // the k kept entries in ascending id order (adjacent swaps)
#pragma unroll
        for (int i = 1; i < KP; ++i)
#pragma unroll
            for (int j = i; j >= 1; --j) {
                if (i < k && bi[j - 1] > bi[j]) {
                    const uint32_t kt = bk[j - 1];
                    const int it = bi[j - 1];
                    bk[j - 1] = bk[j];
                    bi[j - 1] = bi[j];
                    bk[j] = kt;
                    bi[j] = it;
                }
            }
        float ex[KP];
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            ex[j] = expf(key_logit(bk[j]) - zmax);
            if (j < k) sum = sum + ex[j];
        }
        const float inv = 1.0f / sum;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            if (j < k) {
                topk_idx[(long)t * k + j] = bi[j];
                topk_w[(long)t * k + j] = ex[j] * inv;
            }
        }
    }
}

// Top-k by a bitwise radix search, for many experts (128 or more): wave w
// selects for tokens TPW w .. TPW w + TPW - 1; lane l holds experts l + 64 m.
template <int EPAD, int BT, int NW>
DEV void select_topk_radix(const float *zs, int ld, int t0, int T, int E, int k,
                           int *__restrict__ topk_idx, float *__restrict__ topk_w) {
    constexpr int PER = (EPAD + 63) / 64;
    constexpr int TPW = BT / NW;
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    // top-k: wave w selects for tokens TPW w .. TPW w + TPW - 1 (rows past
    // the batch hold finite logits too and are computed, not stored); lane
    // l holds experts
    // l + 64 m.  Each logit maps to an unsigned key with the same order (-0
    // and +0 share one key; a NaN ranks as -inf; padding entries get key 0,
    // below every logit), so that the k-th largest key and the largest key
    // fall out of a bitwise radix search whose counts are ballots: every
    // step is wave-uniform and no lane exchanges values.  The kept set is
    // every key above the k-th largest plus, among keys equal to it, the
    // lowest ids up to k (ties go to the lower expert id).  Each lane writes
    // its own kept experts at their rank among the kept ids, so the ids come
    // out ascending; the weights are exp(z - zmax) over their sum taken in
    // ascending id order.
    const unsigned long long lt = (l == 0) ? 0ull : (~0ull >> (64 - l));
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
        const int tt = TPW * w + q, t = t0 + tt;
        float v[PER];
        uint32_t key[PER];
        uint32_t lane_max = 0;
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int e = l + 64 * m;
            float z = e < E ? zs[tt * ld + e] : -INFINITY;
            z = z == z ? z : -INFINITY;
            z = z == 0.f ? 0.f : z;
            v[m] = z;
            const uint32_t u = __float_as_uint(z);
            key[m] = e < E ? ((u & 0x80000000u) ? ~u : (u | 0x80000000u)) : 0u;
            lane_max = max(lane_max, key[m]);
        }
        uint32_t kth = 0, top = 0;
#pragma unroll
        for (int b = 31; b >= 0; --b) {
            const uint32_t ck = kth | (1u << b), ct = top | (1u << b);
            int n = 0;
#pragma unroll
            for (int m = 0; m < PER; ++m) n += __popcll(__ballot(key[m] >= ck));
            if (n >= k) kth = ck;
            if (__ballot(lane_max >= ct)) top = ct;
        }
        unsigned long long sel[PER];
        int need = k;
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            sel[m] = __ballot(key[m] > kth);
            need -= __popcll(sel[m]);
        }
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            unsigned long long eq = __ballot(key[m] == kth);
            const int c = __popcll(eq);
            if (c <= need) {
                sel[m] |= eq;
                need -= c;
            } else {
                for (; need > 0; --need) {
                    sel[m] |= eq & (~eq + 1);
                    eq &= eq - 1;
                }
            }
        }
        const uint32_t ut = (top & 0x80000000u) ? (top ^ 0x80000000u) : ~top;
        const float zmax = __uint_as_float(ut);
        float ex[PER];
#pragma unroll
        for (int m = 0; m < PER; ++m) ex[m] = expf(v[m] - zmax);
        float sum = 0.f;
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            for (unsigned long long s = sel[m]; s; s &= s - 1) {
                const int src = __builtin_ctzll(s);
                sum = sum + __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ex[m]), src));
            }
        }
        const float inv = 1.0f / sum;
        int before = 0;   // kept ids in lower blocks of 64
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            if (t < T && ((sel[m] >> l) & 1ull)) {
                const int rank = before + __popcll(sel[m] & lt);
                topk_idx[(long)t * k + rank] = l + 64 * m;
                topk_w[(long)t * k + rank] = ex[m] * inv;
            }
            before += __popcll(sel[m]);
        }
    }
}

template <int EPAD, int NW, int MT>
__global__ __launch_bounds__(64 * NW) void route_kernel(const uint16_t *__restrict__ X,
                                                    const uint16_t *__restrict__ WrT,
                                                    const float *__restrict__ bias,
                                                    float *__restrict__ logits,
                                                    int *__restrict__ topk_idx,
                                                    float *__restrict__ topk_w,
                                                    int T, int d, int E, int k) {
    constexpr int NT = EPAD / 16;
    constexpr int BT = 16 * MT;             // tokens per block
    __shared__ float red[NW][BT][EPAD + 1];
    __shared__ float zs[BT][EPAD + 1];

    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int g = l >> 4, r = l & 15;
    const int t0 = blockIdx.x * BT;

    f32x4_t acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // CU chunks per pass: all their loads first, then the MFMAs in chunk
    // order (so the sums are those of one chunk at a time).  Each W_r^T
    // fragment serves the MT token tiles of the wave.
    constexpr int CU = 24 / (2 * MT + 2 * NT) < 1 ? 1 : 24 / (2 * MT + 2 * NT) > 4 ? 4
                                                     : 24 / (2 * MT + 2 * NT);
    const int nchunks = d / 64;
    for (int c0 = w; c0 < nchunks; c0 += NW * CU) {
        u32x4_t a0[CU][MT], a1[CU][MT], b0[CU][NT], b1[CU][NT];
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            const int c = c0 + NW * u;
            const int kb = min(c, nchunks - 1) * 64 + 16 * g;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int tok = t0 + 16 * mt + r;
                a0[u][mt] = u32x4_t{0, 0, 0, 0};
                a1[u][mt] = u32x4_t{0, 0, 0, 0};
                if (tok < T && c < nchunks) {
                    const uint16_t *xrow = X + (long)tok * d + kb;
                    a0[u][mt] = ld_u32x4(xrow);
                    a1[u][mt] = ld_u32x4(xrow + 8);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const uint16_t *wrow = WrT + (long)(16 * nt + r) * d + kb;
                b0[u][nt] = ld_u32x4(wrow);
                b1[u][nt] = ld_u32x4(wrow + 8);
            }
        }
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            if (c0 + NW * u < nchunks) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8_t, a0[u][mt]),
                            __builtin_bit_cast(bf16x8_t, b0[u][nt]), acc[mt][nt], 0, 0, 0);
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8_t, a1[u][mt]),
                            __builtin_bit_cast(bf16x8_t, b1[u][nt]), acc[mt][nt], 0, 0, 0);
                    }
            }
        }
    }
    // 16x16 accumulator layout: lane (g, r) register q holds row 4g+q, column r.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int q = 0; q < 4; ++q) red[w][16 * mt + 4 * g + q][16 * nt + r] = acc[mt][nt][q];
    __syncthreads();

    for (int i = threadIdx.x; i < BT * EPAD; i += 64 * NW) {
        const int tt = i / EPAD, e = i % EPAD;
        float z = red[0][tt][e] + red[1][tt][e];
#pragma unroll
        for (int v = 2; v < NW; ++v) z = z + red[v][tt][e];
        if (e < E) {
            if (bias) z = z + bias[e];
            if (t0 + tt < T) logits[(long)(t0 + tt) * E + e] = z;
            zs[tt][e] = z;
        }
    }
    __syncthreads();

    // top-k (ties to the lower expert id), ids ascending, renormalised
    // softmax weights; see select_topk.
    if constexpr (EPAD >= 128) {
        select_topk_radix<EPAD, BT, NW>(&zs[0][0], EPAD + 1, t0, T, E, k, topk_idx, topk_w);
        return;
    }
    switch (k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : 16) {
        case 1: select_topk<EPAD, 1>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 2: select_topk<EPAD, 2>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 4: select_topk<EPAD, 4>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 8: select_topk<EPAD, 8>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        default: select_topk<EPAD, 16>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
    }
}

}  // namespace

int route_epad(int E) {
    int p = 16;
    while (p < E) p *= 2;
    return p;
}

hipError_t launch_route(const uint16_t *X, const uint16_t *W_r, const float *bias, float *logits,
                        int *topk_idx, float *topk_w, uint16_t *WrT, int T, int d, int E, int k,
                        hipStream_t st) {
    const int EPAD = route_epad(E);
    const long n = (long)EPAD * d;
    wr_transpose_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(W_r, WrT, d, E, EPAD);
    if (T == 0) return hipGetLastError();
    // token tiles per wave: each W_r^T fragment a wave loads serves MT tiles
    // of 16 tokens, as many as keep about one block per compute unit (the
    // partial sums of 8 waves must fit the 160 KiB of LDS)
    const int mt_max = EPAD <= 64 ? 4 : EPAD == 128 ? 2 : 1;
    int mt = 1;
    while (mt < mt_max && (T + 32 * mt - 1) / (32 * mt) >= 256) mt *= 2;
    const dim3 b8(512), b4(256);
    auto grid = [&](int m) { return dim3((unsigned)((T + 16 * m - 1) / (16 * m))); };
#define ROUTE_LAUNCH(EP, NW, M) \
    route_kernel<EP, NW, M><<<grid(M), NW == 8 ? b8 : b4, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k)
    switch (EPAD * 8 + mt) {
        case 16 * 8 + 1: ROUTE_LAUNCH(16, 8, 1); break;
        case 16 * 8 + 2: ROUTE_LAUNCH(16, 8, 2); break;
        case 16 * 8 + 4: ROUTE_LAUNCH(16, 8, 4); break;
        case 32 * 8 + 1: ROUTE_LAUNCH(32, 8, 1); break;
        case 32 * 8 + 2: ROUTE_LAUNCH(32, 8, 2); break;
        case 32 * 8 + 4: ROUTE_LAUNCH(32, 8, 4); break;
        case 64 * 8 + 1: ROUTE_LAUNCH(64, 8, 1); break;
        case 64 * 8 + 2: ROUTE_LAUNCH(64, 8, 2); break;
        case 64 * 8 + 4: ROUTE_LAUNCH(64, 8, 4); break;
        case 128 * 8 + 1: ROUTE_LAUNCH(128, 8, 1); break;
        case 128 * 8 + 2: ROUTE_LAUNCH(128, 8, 2); break;
        case 256 * 8 + 1: ROUTE_LAUNCH(256, 4, 1); break;
        default: return hipErrorInvalidValue;
    }
#undef ROUTE_LAUNCH
    return hipGetLastError();
}
