// Router: logits = X W_r + bias on MFMA, then per-token top-k and the
// renormalised softmax weights (§2.1: a router projection selects the top-k
// routed experts and assigns each a router weight).
//
// Layout: 16 tokens per block, 4 waves.  The d axis is cut into 64-wide
// chunks dealt round-robin to the waves (split-K); each wave accumulates
// 16 x EPAD partial logits with v_mfma_f32_16x16x32_bf16 reading X rows
// straight from HBM and the transposed router W_r^T from L2.  The four
// partial sums are added in wave order, so the result is deterministic.
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

template <int EPAD>
__global__ __launch_bounds__(256) void route_kernel(const uint16_t *__restrict__ X,
                                                    const uint16_t *__restrict__ WrT,
                                                    const float *__restrict__ bias,
                                                    float *__restrict__ logits,
                                                    int *__restrict__ topk_idx,
                                                    float *__restrict__ topk_w,
                                                    int T, int d, int E, int k) {
    constexpr int NT = EPAD / 16;
    constexpr int PER = (EPAD + 63) / 64;
    __shared__ float red[4][16][EPAD + 1];
    __shared__ float zs[16][EPAD + 1];

    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int g = l >> 4, r = l & 15;
    const int t0 = blockIdx.x * 16;
    const int tok = t0 + r;
    const bool tok_ok = tok < T;
    const uint16_t *xrow = X + (long)(tok_ok ? tok : 0) * d;

    f32x4_t acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // CU chunks per pass: all their loads first, then the MFMAs in chunk
    // order (so the sums are those of one chunk at a time)
    constexpr int CU = NT <= 2 ? 4 : NT <= 4 ? 2 : 1;
    const int nchunks = d / 64;
    for (int c0 = w; c0 < nchunks; c0 += 4 * CU) {
        u32x4_t a0[CU], a1[CU], b0[CU][NT], b1[CU][NT];
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            const int c = c0 + 4 * u;
            const int kb = min(c, nchunks - 1) * 64 + 16 * g;
            a0[u] = u32x4_t{0, 0, 0, 0};
            a1[u] = u32x4_t{0, 0, 0, 0};
            if (tok_ok && c < nchunks) {
                a0[u] = ld_u32x4(xrow + kb);
                a1[u] = ld_u32x4(xrow + kb + 8);
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
            if (c0 + 4 * u < nchunks) {
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, a0[u]), __builtin_bit_cast(bf16x8_t, b0[u][nt]),
                        acc[nt], 0, 0, 0);
                    acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, a1[u]), __builtin_bit_cast(bf16x8_t, b1[u][nt]),
                        acc[nt], 0, 0, 0);
                }
            }
        }
    }
    // 16x16 accumulator layout: lane (g, r) register q holds row 4g+q, column r.
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int q = 0; q < 4; ++q) red[w][4 * g + q][16 * nt + r] = acc[nt][q];
    __syncthreads();

    for (int i = threadIdx.x; i < 16 * EPAD; i += 256) {
        const int tt = i / EPAD, e = i % EPAD;
        float z = red[0][tt][e] + red[1][tt][e];
        z = z + red[2][tt][e];
        z = z + red[3][tt][e];
        if (e < E) {
            if (bias) z = z + bias[e];
            if (t0 + tt < T) logits[(long)(t0 + tt) * E + e] = z;
            zs[tt][e] = z;
        }
    }
    __syncthreads();

    // top-k: wave w selects for tokens 4w .. 4w+3.
    for (int q = 0; q < 4; ++q) {
        const int tt = 4 * w + q, t = t0 + tt;
        if (t >= T) break;
        float v[PER];
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int e = l + 64 * m;
            v[m] = e < E ? zs[tt][e] : -INFINITY;
        }
        uint32_t taken = 0;
        int sel[16];
        float selz[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            sel[s] = 0x7fffffff;
            selz[s] = 0.f;
            if (s < k) {
                float bv = -INFINITY;
                int bi = 0x7fffffff;
#pragma unroll
                for (int m = 0; m < PER; ++m) {
                    const int e = l + 64 * m;
                    if (e < E && !((taken >> m) & 1u)) {
                        if (v[m] > bv || (v[m] == bv && e < bi)) { bv = v[m]; bi = e; }
                    }
                }
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    const float ov = shfl_xor_f(bv, off);
                    const int oi = shfl_xor_i(bi, off);
                    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
                }
                sel[s] = bi;
                selz[s] = bv;
                if ((bi & 63) == l) taken |= 1u << (bi >> 6);
            }
        }
        const float zmax = selz[0];
        // ascending expert order (entries past k hold INT_MAX and stay last)
#pragma unroll
        for (int a = 0; a < 15; ++a)
#pragma unroll
            for (int b = 0; b < 15 - a; ++b)
                if (sel[b] > sel[b + 1]) {
                    int ti = sel[b]; sel[b] = sel[b + 1]; sel[b + 1] = ti;
                    float tz = selz[b]; selz[b] = selz[b + 1]; selz[b + 1] = tz;
                }
        float ex[16];
        float sum = 0.f;
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            ex[s] = s < k ? expf(selz[s] - zmax) : 0.f;
            sum = sum + ex[s];
        }
        const float inv = 1.0f / sum;
        if (l == 0) {
#pragma unroll
            for (int s = 0; s < 16; ++s)
                if (s < k) {
                    topk_idx[(long)t * k + s] = sel[s];
                    topk_w[(long)t * k + s] = ex[s] * inv;
                }
        }
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
    dim3 grid((unsigned)((T + 15) / 16)), block(256);
    switch (EPAD) {
        case 16: route_kernel<16><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k); break;
        case 32: route_kernel<32><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k); break;
        case 64: route_kernel<64><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k); break;
        case 128: route_kernel<128><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k); break;
        case 256: route_kernel<256><<<grid, block, 0, st>>>(X, WrT, bias, logits, topk_idx, topk_w, T, d, E, k); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}
