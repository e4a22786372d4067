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
//                     and [E][N][K/32] scales (a 32 x 256 tile transposed
//                     through LDS), the operand layout of the fp8 GEMMs.
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

// Grid (N / 256, K / 32, E).  Block: 256 threads, thread t owns weight column
// n0 + t for the 32 k rows of this block.
__global__ __launch_bounds__(256) void mx_quant_weights_kernel(const uint16_t *__restrict__ W, int K,
                                                               int N, uint8_t *__restrict__ q,
                                                               uint8_t *__restrict__ sc) {
    __shared__ __attribute__((aligned(16))) uint16_t tile[32 * WQ_PITCH];
    const int t = threadIdx.x;
    const int n0 = blockIdx.x * WQ_TN, k0 = blockIdx.y * 32, e = blockIdx.z;
    const uint16_t *src = W + ((long)e * K + k0) * N + n0;
    // 32 rows x 256 columns: 1024 chunks of 8 bf16, 4 per thread, coalesced
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int ch = it * 256 + t;
        const int r = ch / 32, c = 8 * (ch % 32);
        st_u32x4(tile + r * WQ_PITCH + c, ld_u32x4(src + (long)r * N + c));
    }
    __syncthreads();
    float v[32];
    float amax = 0.f;
#pragma unroll
    for (int r = 0; r < 32; ++r) {
        v[r] = bf2f(tile[r * WQ_PITCH + t]);
        amax = fmaxf(amax, fabsf(v[r]));
    }
    const int s = mx_shared_exp(amax);
    const long n = n0 + t;
    uint8_t *dst = q + ((long)e * N + n) * K + k0;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        float part[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) part[j] = v[8 * h + j];
        *reinterpret_cast<u32x2_t *>(dst + 8 * h) = e4m3_pack8(part, s);
    }
    sc[((long)e * N + n) * (K / 32) + k0 / 32] = (uint8_t)(s + 127);
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
    mx_quant_weights_kernel<<<dim3(N / WQ_TN, K / 32, E), dim3(256), 0, st>>>(W, K, N, q, sc);
    return hipGetLastError();
}
