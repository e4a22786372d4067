// Router: logits = X W_r + bias on MFMA, then per-token top-k and the
// renormalised softmax weights (§2.1: the router scores every expert for a
// token, keeps the k best and gives each a weight).
//
// Up to 64 experts (route_kernel): 16 MT tokens per block, 8 waves.  The d
// axis is cut into 64-wide chunks dealt round-robin to the waves (split-K);
// each wave accumulates 16 MT x EPAD partial logits with
// v_mfma_f32_16x16x32_bf16 reading X rows straight from HBM and the
// transposed router W_r^T from L2.  The partial sums are added in wave
// order, so the result is deterministic.  128 or more experts
// (route_split_kernel, route_reduce_kernel): 128-token tiles over slices of
// the d axis staged through LDS, partial tiles added in slice order by a
// second kernel.  The selection runs on groups of lanes per token.
#include "common.h"
#include "kernels.h"

namespace {

// WrT[e][kk] = W_r[kk][e] (zero rows for E <= e < EPAD), through a 32 x 64
// LDS tile so that both the reads (along e) and the writes (along kk) are
// contiguous.  Block (x, y) covers kk in [32 x, 32 x + 32), e in [64 y, ...).
__global__ __launch_bounds__(256) void wr_transpose_kernel(const uint16_t *__restrict__ Wr,
                                                           uint16_t *__restrict__ WrT,
                                                           int d, int E, int EPAD) {
    __shared__ uint16_t tile[32][66];
    const int kk0 = blockIdx.x * 32, e0 = blockIdx.y * 64;
    uint16_t v[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const int r = (threadIdx.x >> 6) + 4 * m, kk = kk0 + r, e = e0 + (threadIdx.x & 63);
        v[m] = (kk < d && e < E) ? Wr[(long)kk * E + e] : (uint16_t)0;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) tile[(threadIdx.x >> 6) + 4 * m][threadIdx.x & 63] = v[m];
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const int c = (threadIdx.x >> 5) + 8 * m, e = e0 + c, kk = kk0 + (threadIdx.x & 31);
        if (e < EPAD && kk < d) WrT[(long)e * d + kk] = tile[threadIdx.x & 31][c];
    }
}

// Top-k of one token's logits.  Each logit maps to an unsigned key with the
// same order (-0 and +0 share one key; a NaN ranks as -inf; every real key
// is above 0), and an entry (key, id) ranks above another when its key is
// larger or, for equal keys, its id is smaller: ties go to the lower expert
// id.  An entry is packed as key * 2^32 + (0xffff - id), so that rank order
// is plain unsigned 64-bit order and a compare-exchange is one 64-bit
// compare and four selects; padding entries are 0, below every real one.
// L = EPAD / PE lanes share a token, PE experts each (16, or all of them
// for 16 experts or fewer).  Each lane finds its best KP entries (KP = k
// rounded up to a power of two) sorted by rank: it sorts its experts in
// groups of KP with a bitonic network and merges the groups; the L lists
// are then merged in log2 L rounds with the lane at distance s.  A merge of
// two sorted lists takes the elementwise better of one list and the other
// reversed, which holds the best KP of both as a bitonic sequence, and
// sorts it with log2 KP half-cleaner stages.  Every lane of the group ends with the
// token's best KP entries; the first k are the selection.  Lane 0 of the
// group puts them in ascending id order and writes ids and weights
// exp(z - zmax) / sum, the sum taken in ascending id order.
DEV uint32_t logit_key(float z) {
    z = z == z ? z : -INFINITY;
    z = z == 0.f ? 0.f : z;
    const uint32_t u = __float_as_uint(z);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
DEV float key_logit(uint32_t key) {
    return __uint_as_float((key & 0x80000000u) ? (key ^ 0x80000000u) : ~key);
}
DEV uint64_t pack_entry(uint32_t key, int id) {
    return ((uint64_t)key << 32) | (uint32_t)(0xffff - id);
}
DEV int entry_id(uint64_t v) { return 0xffff - (int)(uint32_t)v; }
// put the better of a, b first
DEV void order2(uint64_t &a, uint64_t &b) {
    const bool sw = b > a;
    const uint64_t x = a, y = b;
    a = sw ? y : x;
    b = sw ? x : y;
}
DEV uint64_t shfl_xor_u64(uint64_t v, int m) {
    const int lo = __shfl_xor((int)(uint32_t)v, m, 64);
    const int hi = __shfl_xor((int)(uint32_t)(v >> 32), m, 64);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}
// Sort N entries best first (bitonic network, N a power of two).
template <int N>
DEV void sort_desc(uint64_t (&a)[N]) {
#pragma unroll
    for (int size = 2; size <= N; size <<= 1)
#pragma unroll
        for (int stride = size / 2; stride > 0; stride >>= 1)
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int j = i ^ stride;
                if (j > i) {
                    if ((i & size) == 0 || size == N) order2(a[i], a[j]);
                    else order2(a[j], a[i]);
                }
            }
}
// a, b sorted best first: a becomes the best N of both, sorted (the
// elementwise better of a and reversed b is bitonic; half-cleaners sort it).
template <int N>
DEV void merge_best(uint64_t (&a)[N], uint64_t (&b)[N]) {
#pragma unroll
    for (int j = 0; j < N; ++j) order2(a[j], b[N - 1 - j]);
#pragma unroll
    for (int len = N / 2; len >= 1; len >>= 1)
#pragma unroll
        for (int j = 0; j < N; ++j)
            if ((j & len) == 0) order2(a[j], a[j + len]);
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
        // the lane's best KP: its PE entries in groups of KP, each sorted by
        // a bitonic network, merged pairwise into the running best KP
        constexpr int G = PE < KP ? PE : KP;     // group size
        uint64_t bk[KP];
#pragma unroll
        for (int j = 0; j < KP; ++j) bk[j] = 0ull;
#pragma unroll
        for (int g0 = 0; g0 < PE; g0 += G) {
            uint64_t v[KP];
#pragma unroll
            for (int j = 0; j < KP; ++j) {
                const int id = sub * PE + g0 + j;
                v[j] = (j < G && id < E) ? pack_entry(logit_key(zr[g0 + (j < G ? j : 0)]), id) : 0ull;
            }
            sort_desc<KP>(v);
            if (g0 == 0) {
#pragma unroll
                for (int j = 0; j < KP; ++j) bk[j] = v[j];
            } else {
                merge_best<KP>(bk, v);
            }
        }
#pragma unroll
        for (int st = 1; st < L; st <<= 1) {
            uint64_t pk[KP];
#pragma unroll
            for (int j = 0; j < KP; ++j) pk[j] = shfl_xor_u64(bk[j], st);
            merge_best<KP>(bk, pk);
        }
        if (sub != 0 || tb + l / L >= BT || t >= T) continue;
        const float zmax = key_logit((uint32_t)(bk[0] >> 32));
        // the k kept entries in ascending id order (adjacent swaps)
#pragma unroll
        for (int i = 1; i < KP; ++i)
#pragma unroll
            for (int j = i; j >= 1; --j) {
                if (i < k && entry_id(bk[j - 1]) > entry_id(bk[j])) {
                    const uint64_t x = bk[j - 1];
                    bk[j - 1] = bk[j];
                    bk[j] = x;
                }
            }
        float ex[KP];
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            ex[j] = expf(key_logit((uint32_t)(bk[j] >> 32)) - zmax);
            if (j < k) sum = sum + ex[j];
        }
        const float inv = 1.0f / sum;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            if (j < k) {
                topk_idx[(long)t * k + j] = entry_id(bk[j]);
                topk_w[(long)t * k + j] = ex[j] * inv;
            }
        }
    }
}

// The selection for a block's BT tokens, dispatched on KP.
template <int EPAD>
DEV void select_block(const float *zs, int ld, int BT, int NW, int t0, int T, int E, int k,
                      int *__restrict__ topk_idx, float *__restrict__ topk_w) {
    switch (k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : 16) {
        case 1: select_topk<EPAD, 1>(zs, ld, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 2: select_topk<EPAD, 2>(zs, ld, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 4: select_topk<EPAD, 4>(zs, ld, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        case 8: select_topk<EPAD, 8>(zs, ld, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
        default: select_topk<EPAD, 16>(zs, ld, BT, NW, t0, T, E, k, topk_idx, topk_w); break;
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

    // 64 NW is a multiple of EPAD: each thread keeps one expert column, so
    // its bias is loaded once, ahead of the loop
    static_assert((64 * NW) % EPAD == 0, "one expert column per thread");
    const int ecol = threadIdx.x % EPAD;
    const float bz = (bias && ecol < E) ? bias[ecol] : 0.f;
    for (int i = threadIdx.x; i < BT * EPAD; i += 64 * NW) {
        const int tt = i / EPAD, e = i % EPAD;
        float z = red[0][tt][e] + red[1][tt][e];
#pragma unroll
        for (int v = 2; v < NW; ++v) z = z + red[v][tt][e];
        if (e < E) {
            if (bias) z = z + bz;
            if (t0 + tt < T) logits[(long)(t0 + tt) * E + e] = z;
            zs[tt][e] = z;
        }
    }
    __syncthreads();

    // top-k (ties to the lower expert id), ids ascending, renormalised
    // softmax weights; see select_topk.
    select_block<EPAD>(&zs[0][0], EPAD + 1, BT, NW, t0, T, E, k, topk_idx, topk_w);
}


// ---------------------------------------------------------------------------
// Router for many experts (E_pad >= 64): a split-K tile kernel.
//
// With many experts the transposed router is as large as a block's share of
// X (512 KB at 128 experts and d = 2048), so a block of few tokens spends
// most of its time streaming W_r^T from L2.  Here a block owns RT = 128
// tokens and one of S slices of the d axis (S chosen so the grid fills the
// device), and stages X and W_r^T chunks of 64 columns through LDS with
// direct loads, double-buffered: per block (RT + E_pad) * d / S * 2 bytes.
// 8 waves as 4 (tokens) x 2 (experts), each 32 tokens x E_pad / 2 experts on
// v_mfma_f32_32x32x16_bf16.  With S > 1 each block stores its fp32 partial
// tile and route_reduce_kernel adds the S partials in slice order, adds the
// bias, writes the logits and runs the selection; with S = 1 the block does
// that itself.
constexpr int RT = 128;            // tokens per block
#define LDS_AS __attribute__((address_space(3)))

DEV void r_load_lds16(const uint16_t *src, uint16_t *lds_dst) {
    __builtin_amdgcn_global_load_lds(src, (LDS_AS void *)lds_dst, 16, 0, 0);
}
DEV void r_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
// s_waitcnt vmcnt(N) leaving the other counters alone (gfx9 encoding)
template <int N>
DEV void r_wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
// 16-byte chunk c of LDS row r (128-byte rows) lives at chunk c ^ ((r >> 1) & 7)
DEV int r_swz(int r, int c) { return c ^ ((r >> 1) & 7); }

template <int EPAD>
__global__ __launch_bounds__(512) void route_split_kernel(const uint16_t *__restrict__ X,
                                                          const uint16_t *__restrict__ WrT,
                                                          const float *__restrict__ bias,
                                                          float *__restrict__ logits,
                                                          int *__restrict__ topk_idx,
                                                          float *__restrict__ topk_w,
                                                          float *__restrict__ part,
                                                          int T, int d, int E, int k, int S) {
    static_assert(EPAD == 64 || EPAD == 128 || EPAD == 256, "split router: 64, 128 or 256 experts");
    constexpr int TN = EPAD / 64;                         // 32-wide expert tiles per wave
    constexpr int XT = RT * 64, WT = EPAD * 64;           // stage elements (bf16)
    // stages of the chunk pipeline (NST - 1 chunks in flight): 4, or 3 where
    // 4 would not fit the 160 KiB of LDS
    constexpr int NST = 2 * (XT + WT) * 4 <= 160 * 1024 - 4096 ? 4 : 3;
    constexpr int STAGE_BYTES = NST * 2 * (XT + WT);
    constexpr int ZS_BYTES = RT * (EPAD + 1) * 4;
    constexpr int LDS_BYTES = STAGE_BYTES > ZS_BYTES ? STAGE_BYTES : ZS_BYTES;
    __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
    // stage st: X tile at st (XT + WT), W_r^T tile right after it (bf16 elements)
    uint16_t *const stg = reinterpret_cast<uint16_t *>(lds);
    float *zs = reinterpret_cast<float *>(lds);

    const int tile = blockIdx.x / S, slice = blockIdx.x % S;
    const int t0 = tile * RT;
    const int dS = d / S, k0 = slice * dS, nch = dS / 64;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave >> 1, wc = wave & 1;

    // direct loads: wave instruction q covers 8 rows of 128 bytes; lane ->
    // row 8 q + lane / 8, physical chunk lane & 7 (logical r_swz of it).
    // X: 16 instructions (2 per wave); W_r^T: EPAD / 8 (EPAD / 64 per wave).
    const uint16_t *xsrc[2];
    int xdst[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = 2 * wave + i, r = 8 * q + (lane >> 3);
        const int t = min(t0 + r, T - 1);          // rows past the batch load its last token
        xsrc[i] = X + (long)t * d + k0 + 8 * r_swz(r, lane & 7);
        xdst[i] = q * 512;
    }
    const uint16_t *wsrc[TN];
    int wdst[TN];
#pragma unroll
    for (int i = 0; i < TN; ++i) {
        const int q = TN * wave + i, r = 8 * q + (lane >> 3);
        wsrc[i] = WrT + (long)r * d + k0 + 8 * r_swz(r, lane & 7);
        wdst[i] = q * 512;
    }
    auto issue = [&](int c, int st) {
#pragma unroll
        for (int i = 0; i < 2; ++i) r_load_lds16(xsrc[i] + 64 * c, stg + st * (XT + WT) + xdst[i]);
#pragma unroll
        for (int i = 0; i < TN; ++i) r_load_lds16(wsrc[i] + 64 * c, stg + st * (XT + WT) + XT + wdst[i]);
    };

    f32x16_t acc[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;

    const int arow = 32 * wr + (lane & 31);
    // chunk c goes to stage c % NST; the first NST - 1 chunks are issued
    // ahead, and each step waits only for its own chunk (the later chunks'
    // loads, LPC per chunk, stay in flight)
    constexpr int LPC = 2 + TN;
    for (int c = 0; c < NST - 1 && c < nch; ++c) issue(c, c);
    for (int c = 0; c < nch; ++c) {
        const int st = c % NST;
        const int after = min(NST - 2, nch - 1 - c);
        if (after >= 2) r_wait_vmcnt<2 * LPC>();
        else if (after == 1) r_wait_vmcnt<LPC>();
        else r_wait_vmcnt<0>();
        r_barrier();
        if (c + NST - 1 < nch) issue(c + NST - 1, (c + NST - 1) % NST);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int ch = 2 * ks + (lane >> 5);
            const bf16x8_t a = __builtin_bit_cast(
                bf16x8_t, ld_u32x4(stg + st * (XT + WT) + arow * 64 + 8 * r_swz(arow, ch)));
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int brow = (EPAD / 2) * wc + 32 * j + (lane & 31);
                const bf16x8_t b = __builtin_bit_cast(
                    bf16x8_t, ld_u32x4(stg + st * (XT + WT) + XT + brow * 64 + 8 * r_swz(brow, ch)));
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
            }
        }
    }
    __syncthreads();   // every wave is done with the stages: zs reuses them

    // 32x32 accumulator layout: lane l, register q -> row 8 (q / 4) + 4 (l / 32) + q % 4, column l % 32
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int r = 32 * wr + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
            const int e = (EPAD / 2) * wc + 32 * j + (lane & 31);
            zs[r * (EPAD + 1) + e] = acc[j][q];
            if (S > 1 && t0 + r < T) part[((long)slice * T + t0 + r) * EPAD + e] = acc[j][q];
        }
    if (S > 1) return;   // route_reduce_kernel adds the slices
    __syncthreads();
    // logits: the bias added to the sums (one expert column per thread)
    const float bz = (bias && tid % EPAD < E) ? bias[tid % EPAD] : 0.f;
    for (int i = tid; i < RT * EPAD; i += 512) {
        const int r = i / EPAD, e = i % EPAD, t = t0 + r;
        float z = zs[r * (EPAD + 1) + e];
        if (e < E) {
            if (bias) z = z + bz;
            if (t < T) logits[(long)t * E + e] = z;
        }
        zs[r * (EPAD + 1) + e] = z;
    }
    __syncthreads();
    select_block<EPAD>(zs, EPAD + 1, RT, 8, t0, T, E, k, topk_idx, topk_w);
}


// The S partial tiles of the split router added in slice order, the bias,
// the logits and the selection: 32 tokens per block of 4 waves.
constexpr int RR_BT = 32;
template <int EPAD, int S>
__global__ __launch_bounds__(256) void route_reduce_kernel(const float *__restrict__ part,
                                                           const float *__restrict__ bias,
                                                           float *__restrict__ logits,
                                                           int *__restrict__ topk_idx,
                                                           float *__restrict__ topk_w, int T, int E,
                                                           int k) {
    __shared__ float zs[RR_BT][EPAD + 1];
    const int t0 = blockIdx.x * RR_BT;
    // every thread loads its 16-byte pieces of all S slices before adding
    constexpr int NV = RR_BT * EPAD / 4 / 256;   // pieces per slice per thread
    static_assert(NV >= 1, "32 tokens x E_pad fp32 cover the block");
    f32x4_t v[S][NV];
    // 256 is a multiple of E_pad / 4: each thread keeps columns c .. c + 3
    const int c4 = 4 * (threadIdx.x % (EPAD / 4));
    float bz[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) bz[q] = (bias && c4 + q < E) ? bias[c4 + q] : 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + 256 * j, r = i / (EPAD / 4), c = 4 * (i % (EPAD / 4));
        const int t = min(t0 + r, T - 1);
#pragma unroll
        for (int sl = 0; sl < S; ++sl)
            v[sl][j] = *reinterpret_cast<const f32x4_t *>(part + ((long)sl * T + t) * EPAD + c);
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + 256 * j, r = i / (EPAD / 4), c = 4 * (i % (EPAD / 4));
        const int t = t0 + r;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float z = v[0][j][q];
#pragma unroll
            for (int sl = 1; sl < S; ++sl) z = z + v[sl][j][q];
            const int e = c + q;
            if (e < E) {
                if (bias) z = z + bz[q];
                if (t < T) logits[(long)t * E + e] = z;
            }
            zs[r][e] = z;
        }
    }
    __syncthreads();
    select_block<EPAD>(&zs[0][0], EPAD + 1, RR_BT, 4, t0, T, E, k, topk_idx, topk_w);
}

}  // namespace

int route_epad(int E) {
    int p = 16;
    while (p < E) p *= 2;
    return p;
}

// Padded expert counts from which the split router runs.
constexpr int ROUTE_SPLIT_MIN = 128;

// Slices of the d axis the split router uses for T tokens (1: no partials);
// 0 when the shape takes the one-pass router.
int route_split_slices(long T, int d, int E) {
    if (route_epad(E) < ROUTE_SPLIT_MIN) return 0;
    const long ntiles = (T + RT - 1) / RT;
    int S = 1;
    while (S < 8 && ntiles * S < 256 && (d / 64) % (2 * S) == 0) S *= 2;
    return S;
}

size_t route_part_bytes(long T, int d, int E) {
    const int S = route_split_slices(T, d, E);
    return S > 1 ? (size_t)S * (size_t)T * (size_t)route_epad(E) * 4 : 0;
}

hipError_t launch_route(const uint16_t *X, const uint16_t *W_r, const float *bias, float *logits,
                        int *topk_idx, float *topk_w, uint16_t *WrT, float *part, int T,
                        int d, int E, int k, hipStream_t st) {
    const int EPAD = route_epad(E);
    const int S = route_split_slices(T, d, E);
    wr_transpose_kernel<<<dim3((unsigned)((d + 31) / 32), (unsigned)((EPAD + 63) / 64)), dim3(256), 0,
                          st>>>(W_r, WrT, d, E, EPAD);
    if (T == 0) return hipGetLastError();
    if (S > 0) {
        const dim3 grid((unsigned)(((T + RT - 1) / RT) * S)), block(512);
        switch (EPAD) {
            case 64:
                route_split_kernel<64><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w,
                                                               part, T, d, E, k, S);
                break;
            case 128:
                route_split_kernel<128><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w,
                                                                part, T, d, E, k, S);
                break;
            case 256:
                route_split_kernel<256><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w,
                                                                part, T, d, E, k, S);
                break;
            default: return hipErrorInvalidValue;
        }
        if (S > 1) {
            const dim3 rg((unsigned)((T + RR_BT - 1) / RR_BT)), rb(256);
#define ROUTE_REDUCE(EP, SL) \
    route_reduce_kernel<EP, SL><<<rg, rb, 0, st>>>(part, bias, logits, topk_idx, topk_w, T, E, k)
            switch (EPAD * 16 + S) {
                case 64 * 16 + 2: ROUTE_REDUCE(64, 2); break;
                case 64 * 16 + 4: ROUTE_REDUCE(64, 4); break;
                case 64 * 16 + 8: ROUTE_REDUCE(64, 8); break;
                case 128 * 16 + 2: ROUTE_REDUCE(128, 2); break;
                case 128 * 16 + 4: ROUTE_REDUCE(128, 4); break;
                case 128 * 16 + 8: ROUTE_REDUCE(128, 8); break;
                case 256 * 16 + 2: ROUTE_REDUCE(256, 2); break;
                case 256 * 16 + 4: ROUTE_REDUCE(256, 4); break;
                case 256 * 16 + 8: ROUTE_REDUCE(256, 8); break;
                default: return hipErrorInvalidValue;
            }
#undef ROUTE_REDUCE
        }
        return hipGetLastError();
    }
    // token tiles per wave: each W_r^T fragment a wave loads serves MT tiles
    // of 16 tokens, as many as keep about one block per compute unit (the
    // partial sums of 8 waves must fit the 160 KiB of LDS)
    const int mt_max = 4;
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
        default: return hipErrorInvalidValue;
    }
#undef ROUTE_LAUNCH
    return hipGetLastError();
}
