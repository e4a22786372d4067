// MXFP8 quantisation (§3.4 "MXFP8 Support"): OCP FP8 E4M3 elements with one
// E8M0 scale per 32 consecutive elements along the contraction axis of the
// GEMM that consumes the tensor.
//
// For a block with largest magnitude amax the scale is 2^s with
// s = floor(log2(amax)) - 8 (8 = the largest E4M3 exponent), clamped to
// [-127, 127] (s = -127 for an all-zero block), stored as the byte s + 127.
// Each element is v * 2^-s clamped to +-448 and rounded to the nearest E4M3
// value, ties to even (v_cvt_pk_fp8_f32 rounds to nearest even; it does not
// saturate, hence the clamp).  Multiplying by 2^-s is exact, so the codes
// depend only on the input values.
//
//   mx_quant_rows:    rows of a K-contiguous bf16 matrix (tokens of X); each
//                     lane takes 8 elements, 4 lanes share a block.
//   mx_quant_weights: [E][K][N] bf16 weights -> K-contiguous [E][N][K] codes
//                     and [E][N][K/32] scales (128 x 256 tiles transposed
//                     through LDS), the operand layout of the fp8 GEMMs.
//   mx_quant_tokens:  the weight-gradient operands, which contract over an
//                     expert's tokens: rows of the expert's plan region in
//                     32-row blocks from its first row, written transposed
//                     (token-contiguous) at the expert's region padded to
//                     128 positions, the K step of the fp8 GEMM.  The source
//                     is bf16 (X, dY, gathered by token) or fp32 (dA, dB and
//                     w h as the gated-activation backward produced them).
#include "common.h"
#include "kernels.h"
#include "mx_common.h"

namespace {

// One thread per 8 elements: thread i of a row covers columns 8 i .. 8 i + 7,
// so the 4 threads of a 32-block are consecutive lanes.
__global__ __launch_bounds__(256) void mx_quant_rows_kernel(const uint16_t *__restrict__ X, long rows,
                                                            int K, uint8_t *__restrict__ q,
                                                            uint8_t *__restrict__ sc) {
    const long i = (long)blockIdx.x * 256 + threadIdx.x;
    const int per_row = K / 8;
    const long total = rows * per_row;
    const bool live = i < total;
    const long row = live ? i / per_row : 0;
    const int c8 = live ? (int)(i - row * per_row) : 0;
    float v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (live) {
        const u32x4_t w = ld_u32x4(X + row * K + 8 * c8);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = bf_lo(w[j]);
            v[2 * j + 1] = bf_hi(w[j]);
        }
    }
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[j]));
    // K % 32 == 0 and rows start at multiples of K/8 threads: the 4 threads of
    // a block are lanes 4g .. 4g + 3 of one wave
    amax = fmaxf(amax, shfl_xor_f(amax, 1));
    amax = fmaxf(amax, shfl_xor_f(amax, 2));
    const int s = mx_shared_exp(amax);
    if (!live) return;
    const u32x2_t codes = e4m3_pack8(v, s);
    *reinterpret_cast<u32x2_t *>(q + row * K + 8 * c8) = codes;
    if ((c8 & 3) == 0) sc[row * (K / 32) + c8 / 4] = (uint8_t)(s + 127);
}

constexpr int WQ_TN = 256;            // output rows (weight columns) per block
constexpr int WQ_PITCH = WQ_TN + 8;   // LDS pitch in bf16 (16-byte rows)

// Padded expert regions: poff[e] = sum over e' < e of count(e') rounded up
// to 128; poff[E] = the padded total.  One wave, a scan per 64 experts.
__global__ __launch_bounds__(64) void mx_pad_offsets_kernel(const int *__restrict__ offsets, int E,
                                                           int *__restrict__ poff) {
    const int lane = threadIdx.x;
    int cum = 0;
    for (int base = 0; base < E; base += 64) {
        const int e = base + lane;
        const int n = e < E ? offsets[e + 1] - offsets[e] : 0;
        const int padded = (n + 127) / 128 * 128;
        int x = padded;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (e < E) poff[e] = cum + x - padded;
        cum += __shfl(x, 63, 64);
    }
    if (lane == 0) poff[E] = cum;
}

// Quantisation along the rows of a bf16 matrix, 128 rows x 256 columns per
// workgroup: thread t owns column c0 + t and quantises its four 32-row MX
// blocks.  Each block is staged through LDS (32 rows x 256 columns; the next
// block's rows are loaded into registers meanwhile).  The codes stay in
// registers until all four blocks are done; then they go through LDS once
// more, so that every store instruction writes whole 128-byte row segments
// (8 columns per wave instruction) instead of 16 bytes in each of 64 rows.
constexpr int TQ_OPITCH = 144;   // LDS bytes per column of codes (+16: conflict-free 16-byte writes)
constexpr int TQ_LDS = 256 * TQ_OPITCH;
static_assert(32 * WQ_PITCH * 2 <= TQ_LDS, "the input block fits the code buffer");

// Element formats of the column quantiser's source: PER elements per 16-byte
// chunk, CH chunks per thread per 32-row block, LDS pitch in elements.
template <typename S> struct TqFmt;
template <> struct TqFmt<uint16_t> {
    static constexpr int PER = 8, CH = 4, PITCH = WQ_PITCH;
    static DEV float val(uint16_t v) { return bf2f(v); }
};
template <> struct TqFmt<float> {
    static constexpr int PER = 4, CH = 8, PITCH = 256 + 4;
    static DEV float val(float v) { return v; }
};
static_assert(32 * TqFmt<uint16_t>::PITCH * 2 <= TQ_LDS, "a bf16 input block fits the code buffer");
static_assert(32 * TqFmt<float>::PITCH * 4 <= TQ_LDS, "an fp32 input block fits the code buffer");

// Rows 32 sb .. 32 sb + 31 of the 128 (s_row: source row, < 0 for zeros),
// one 16-byte chunk of the 256 columns per load, CH loads per thread.
template <typename S>
DEV void tq_fetch(const S *__restrict__ src, long ld, const int *s_row, int sb, int c0, int t,
                  u32x4_t *v) {
    using F = TqFmt<S>;
    constexpr int RC = 256 / F::PER;   // chunks per row
#pragma unroll
    for (int it = 0; it < F::CH; ++it) {
        const int ch = it * 256 + t;
        const int r = ch / RC, c = F::PER * (ch % RC);
        const int row = s_row[32 * sb + r];
        v[it] = u32x4_t{0, 0, 0, 0};
        if (row >= 0) v[it] = ld_u32x4(src + (long)row * ld + c0 + c);
    }
}

// The 128 source rows are s_row[0..127] (written before the call, visible
// after its first barrier).  Column c's 128 codes go to q + c * pitch (c
// counted from c0) and its 4 scales to the 4 bytes at sc + c * spitch.
template <typename S>
DEV void quant_cols128(const S *__restrict__ src, long ld, const int *s_row, int c0, int t,
                       uint8_t *lds, uint8_t *__restrict__ q, long pitch, uint8_t *__restrict__ sc,
                       long spitch) {
    using F = TqFmt<S>;
    constexpr int RC = 256 / F::PER;
    S *tile = reinterpret_cast<S *>(lds);
    __syncthreads();
    u32x4_t pf[F::CH];
    tq_fetch(src, ld, s_row, 0, c0, t, pf);
    uint32_t codes[32];
    uint32_t scw = 0;
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
        if (sb > 0) __syncthreads();            // the previous block's column reads are done
#pragma unroll
        for (int it = 0; it < F::CH; ++it) {
            const int ch = it * 256 + t;
            st_u32x4(tile + (ch / RC) * F::PITCH + F::PER * (ch % RC), pf[it]);
        }
        __syncthreads();
        if (sb < 3) tq_fetch(src, ld, s_row, sb + 1, c0, t, pf);
        float v[32];
        float amax = 0.f;
#pragma unroll
        for (int r = 0; r < 32; ++r) {
            v[r] = F::val(tile[r * F::PITCH + t]);
            amax = fmaxf(amax, fabsf(v[r]));
        }
        const int s = mx_shared_exp(amax);
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            float part[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) part[j] = v[8 * h + j];
            const u32x2_t w = e4m3_pack8(part, s);
            codes[8 * sb + 2 * h] = w[0];
            codes[8 * sb + 2 * h + 1] = w[1];
        }
        scw |= (uint32_t)(s + 127) << (8 * sb);
    }
    __syncthreads();                            // every column read of the last block is done
#pragma unroll
    for (int w = 0; w < 8; ++w)
        st_u32x4(lds + t * TQ_OPITCH + 16 * w,
                 u32x4_t{codes[4 * w], codes[4 * w + 1], codes[4 * w + 2], codes[4 * w + 3]});
    __syncthreads();
    // pass i: thread t writes bytes 16 (t % 8) .. + 15 of column 32 i + t / 8
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int cr = 32 * i + (t >> 3), chunk = t & 7;
        st_u32x4(q + (long)cr * pitch + 16 * chunk, ld_u32x4(lds + cr * TQ_OPITCH + 16 * chunk));
    }
    *reinterpret_cast<uint32_t *>(sc + (long)t * spitch) = scw;
}

// Grid (N / 256, K / 128, E): W [E][K][N] -> K-contiguous codes [E][N][K] and
// scales [E][N][K / 32], the operand layout of the fp8 GEMMs.
__global__ __launch_bounds__(256) void mx_quant_weights_kernel(const uint16_t *__restrict__ W, int K,
                                                               int N, uint8_t *__restrict__ q,
                                                               uint8_t *__restrict__ sc) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[TQ_LDS];
    __shared__ int s_row[128];
    const int t = threadIdx.x;
    const int c0 = blockIdx.x * WQ_TN, k0 = blockIdx.y * 128, e = blockIdx.z;
    if (t < 128) s_row[t] = k0 + t;
    const long col0 = (long)e * N + c0;
    quant_cols128(W + (long)e * K * N, N, s_row, c0, t, lds, q + col0 * K + k0, K,
                  sc + col0 * (K / 32) + k0 / 32, K / 32);
}

// Grid (C / 256, max_pos / 128): the 128 padded positions [p0, p0 + 128) of
// one expert, rows of its plan region (gathered through `rows` when GATHER)
// or zeros past its count.
template <bool GATHER, typename S>
__global__ __launch_bounds__(256) void mx_quant_tokens_kernel(const S *__restrict__ src, long ld,
                                                              long nsrc, const int *__restrict__ rows,
                                                              const int *__restrict__ offsets,
                                                              const int *__restrict__ poff, int E,
                                                              long pitch, uint8_t *__restrict__ q,
                                                              uint8_t *__restrict__ sc) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[TQ_LDS];
    __shared__ int s_row[128];
    const int t = threadIdx.x;
    const int c0 = blockIdx.x * WQ_TN;
    const int p0 = blockIdx.y * 128;
    if (p0 >= poff[E]) return;                 // past the padded total (uniform)
    // the expert whose padded region holds p0: the last e with poff[e] <= p0
    int lo = 0, hi = E - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (poff[mid] <= p0) lo = mid;
        else hi = mid - 1;
    }
    const int base = offsets[lo], cnt = offsets[lo + 1] - base;
    if (t < 128) {
        const int local = p0 - poff[lo] + t;
        int r = -1;                             // padding: zeros
        if (local < cnt) {
            r = GATHER ? rows[base + local] : base + local;
            r = r < 0 ? 0 : (r >= nsrc ? (int)nsrc - 1 : r);   // a malformed plan stays in bounds
        }
        s_row[t] = r;
    }
    quant_cols128(src, ld, s_row, c0, t, lds, q + (long)c0 * pitch + p0, pitch,
                  sc + (long)c0 * (pitch / 32) + p0 / 32, pitch / 32);
}

}  // namespace

hipError_t launch_mx_quant_rows(const uint16_t *X, long rows, int K, uint8_t *q, uint8_t *sc,
                                hipStream_t st) {
    const long threads = rows * (K / 8);
    if (threads <= 0) return hipSuccess;
    mx_quant_rows_kernel<<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st>>>(X, rows, K, q,
                                                                                       sc);
    return hipGetLastError();
}

hipError_t launch_mx_quant_weights(const uint16_t *W, int E, int K, int N, uint8_t *q, uint8_t *sc,
                                   hipStream_t st) {
    if (E <= 0) return hipSuccess;
    mx_quant_weights_kernel<<<dim3(N / WQ_TN, K / 128, E), dim3(256), 0, st>>>(W, K, N, q, sc);
    return hipGetLastError();
}

hipError_t launch_mx_pad_offsets(const int *offsets, int E, int *poff, hipStream_t st) {
    mx_pad_offsets_kernel<<<dim3(1), dim3(64), 0, st>>>(offsets, E, poff);
    return hipGetLastError();
}

hipError_t launch_mx_quant_tokens(const uint16_t *src, long ld, long nsrc, const int *rows,
                                  const int *offsets, const int *poff, int E, int C, long pitch,
                                  long max_pos, uint8_t *q, uint8_t *sc, hipStream_t st) {
    if (max_pos <= 0 || C <= 0 || E <= 0 || nsrc <= 0) return hipSuccess;
    const dim3 grid((unsigned)(C / WQ_TN), (unsigned)(max_pos / 128));
    if (rows)
        mx_quant_tokens_kernel<true, uint16_t><<<grid, dim3(256), 0, st>>>(src, ld, nsrc, rows, offsets, poff, E, pitch, q, sc);
    else
        mx_quant_tokens_kernel<false, uint16_t><<<grid, dim3(256), 0, st>>>(src, ld, nsrc, rows, offsets, poff, E, pitch, q, sc);
    return hipGetLastError();
}

hipError_t launch_mx_quant_tokens_f32(const float *src, long ld, long nsrc, const int *offsets,
                                      const int *poff, int E, int C, long pitch, long max_pos,
                                      uint8_t *q, uint8_t *sc, hipStream_t st) {
    if (max_pos <= 0 || C <= 0 || E <= 0 || nsrc <= 0) return hipSuccess;
    const dim3 grid((unsigned)(C / WQ_TN), (unsigned)(max_pos / 128));
    mx_quant_tokens_kernel<false, float><<<grid, dim3(256), 0, st>>>(src, ld, nsrc, nullptr, offsets, poff, E, pitch, q, sc);
    return hipGetLastError();
}
