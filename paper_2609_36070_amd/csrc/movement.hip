// HBM-bound steps around the expert GEMMs: dispatch gather, plan-order
// prologue, the fixed-order weighted combine and its backward counterpart,
// the restricted-softmax backward and the router-weight gradient.
//
// Every row copy moves 16-byte vectors; every sum over a token's routes runs
// in slot order (ascending expert id) in fp32, so results are bitwise
// repeatable (§3.4 "Determinism").
#include "common.h"
#include "kernels.h"

namespace {

// Xperm[p] = X[perm[p] / k]; rows past the placed total are zero-filled.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint16_t *__restrict__ X,
                                                          const int *__restrict__ perm,
                                                          const int *__restrict__ offsets, int E,
                                                          int k, int T, int d, int R,
                                                          uint16_t *__restrict__ out) {
    const int total = offsets[E];
    const int nc = d / 8;
    for (int p = blockIdx.x; p < R; p += gridDim.x) {
        int t = -1;
        if (p < total) {
            const int j = perm[p];
            t = (j >= 0 && j < R) ? j / k : -1;
        }
        u32x4_t *dst = reinterpret_cast<u32x4_t *>(out + (long)p * d);
        if (t < 0 || t >= T) {
            for (int c = threadIdx.x; c < nc; c += 256) dst[c] = u32x4_t{0, 0, 0, 0};
        } else {
            const u32x4_t *src = reinterpret_cast<const u32x4_t *>(X + (long)t * d);
            for (int c = threadIdx.x; c < nc; c += 256) dst[c] = src[c];
        }
    }
}

// Plan-order prologue: token row and router weight of every buffer position,
// and the zero page the weight-gradient GEMMs read past an expert's count.
__global__ __launch_bounds__(256) void prep_kernel(const int *__restrict__ perm,
                                                   const int *__restrict__ offsets, int E,
                                                   const float *__restrict__ topk_w, int k, int T,
                                                   int R, int *__restrict__ rowidx,
                                                   float *__restrict__ wperm,
                                                   uint16_t *__restrict__ zeros) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p < ZERO_PAGE_ELEMS) zeros[p] = 0;
    if (p >= R) return;
    const int total = offsets[E];
    int t = 0;
    float wv = 0.f;
    if (p < total) {
        const int j = perm[p];
        if (j >= 0 && j < R) {
            t = j / k;
            wv = topk_w[j];
        }
    }
    rowidx[p] = t < T ? t : 0;
    wperm[p] = wv;
}

// Y[t] = Ysh[t] + sum_slot w[t,slot] * Yexp[route_pos[t*k+slot]]  (fp32, one rounding)
__global__ __launch_bounds__(256) void combine_kernel(const uint16_t *__restrict__ Yexp,
                                                      const uint16_t *__restrict__ Ysh,
                                                      const float *__restrict__ topk_w,
                                                      const int *__restrict__ route_pos, int T,
                                                      int d, int k, int R,
                                                      uint16_t *__restrict__ Y) {
    const int nc = d / 8;
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        int pos[16];
        float wt[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            pos[s] = -1;
            wt[s] = 0.f;
            if (s < k) {
                const int p = route_pos[(long)t * k + s];
                pos[s] = (p >= 0 && p < R) ? p : -1;
                wt[s] = topk_w[(long)t * k + s];
            }
        }
        for (int c = threadIdx.x; c < nc; c += 256) {
            // every load first (slots past k or without a position read row 0
            // and are not added), so they are in flight together
            u32x4_t rows[16];
#pragma unroll
            for (int s = 0; s < 16; ++s)
                if (s < k) rows[s] = ld_u32x4(Yexp + (long)max(pos[s], 0) * d + 8 * c);
            float acc[8];
            if (Ysh) {
                const u32x4_t v = ld_u32x4(Ysh + (long)t * d + 8 * c);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[2 * q] = bf_lo(v[q]);
                    acc[2 * q + 1] = bf_hi(v[q]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = 0.f;
            }
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                if (s < k && pos[s] >= 0) {
                    const u32x4_t v = rows[s];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc[2 * q] = acc[2 * q] + wt[s] * bf_lo(v[q]);
                        acc[2 * q + 1] = acc[2 * q + 1] + wt[s] * bf_hi(v[q]);
                    }
                }
            }
            u32x4_t o;
#pragma unroll
            for (int q = 0; q < 4; ++q) o[q] = pack_bf2(acc[2 * q], acc[2 * q + 1]);
            st_u32x4(Y + (long)t * d + 8 * c, o);
        }
    }
}

// dg[p] = sum over n-tiles of the partial <dh', h> (fixed order), then the
// restricted-softmax backward per token:
//   dZ[t,e_s] = w_s (dg_s - sum_s' w_s' dg_s'),  zero for unselected experts.
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const float *__restrict__ dgpart,
                                                          int nparts,
                                                          const int *__restrict__ route_pos,
                                                          const float *__restrict__ topk_w,
                                                          const int *__restrict__ topk_idx, int T,
                                                          int k, int E, int R,
                                                          float *__restrict__ dg_out,
                                                          float *__restrict__ dZ) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= T) return;
    float dg[16], wt[16];
    float swdg = 0.f;
#pragma unroll
    for (int s = 0; s < 16; ++s) {
        dg[s] = 0.f;
        wt[s] = 0.f;
        if (s < k) {
            const int p = route_pos[(long)t * k + s];
            wt[s] = topk_w[(long)t * k + s];
            if (p >= 0 && p < R) {
                float acc = 0.f;
                for (int q = 0; q < nparts; ++q) acc = acc + dgpart[(long)p * nparts + q];
                dg[s] = acc;
                dg_out[p] = acc;
            }
            swdg = swdg + wt[s] * dg[s];
        }
    }
    for (int e = 0; e < E; ++e) dZ[(long)t * E + e] = 0.f;
#pragma unroll
    for (int s = 0; s < 16; ++s) {
        if (s < k) {
            const int e = topk_idx[(long)t * k + s];
            if (e >= 0 && e < E) dZ[(long)t * E + e] = wt[s] * (dg[s] - swdg);
        }
    }
}

// dX[t] = dXsh[t] + sum_slot dXperm[route_pos[t*k+slot]] + sum_e dZ[t,e] W_r[:,e]
__global__ __launch_bounds__(256) void reverse_combine_kernel(const uint16_t *__restrict__ dXperm,
                                                              const uint16_t *__restrict__ dXsh,
                                                              const float *__restrict__ dZ,
                                                              const uint16_t *__restrict__ Wr,
                                                              const int *__restrict__ route_pos,
                                                              int T, int d, int k, int E, int R,
                                                              const float *__restrict__ dXacc,
                                                              uint16_t *__restrict__ dX) {
    __shared__ float dz[256];
    const int nc = d / 8;
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        __syncthreads();
        for (int e = threadIdx.x; e < E; e += 256) dz[e] = dZ[(long)t * E + e];
        __syncthreads();
        int pos[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            pos[s] = -1;
            if (s < k) {
                const int p = route_pos[(long)t * k + s];
                pos[s] = (p >= 0 && p < R) ? p : -1;
            }
        }
        for (int c = threadIdx.x; c < nc; c += 256) {
            float acc[8];
            if (dXacc) {
                // shared-expert and routed terms already summed per token
                // (bounded-memory backward)
                const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(dXacc + (long)t * d + 8 * c);
                const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(dXacc + (long)t * d + 8 * c + 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[q] = lo[q];
                    acc[4 + q] = hi[q];
                }
            } else if (dXsh) {
                const u32x4_t v = ld_u32x4(dXsh + (long)t * d + 8 * c);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[2 * q] = bf_lo(v[q]);
                    acc[2 * q + 1] = bf_hi(v[q]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = 0.f;
            }
            if (!dXacc) {
                u32x4_t rows[16];   // all loads first, as in the combine
#pragma unroll
                for (int s = 0; s < 16; ++s)
                    if (s < k) rows[s] = ld_u32x4(dXperm + (long)max(pos[s], 0) * d + 8 * c);
#pragma unroll
                for (int s = 0; s < 16; ++s) {
                    if (s < k && pos[s] >= 0) {
                        const u32x4_t v = rows[s];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            acc[2 * q] = acc[2 * q] + bf_lo(v[q]);
                            acc[2 * q + 1] = acc[2 * q + 1] + bf_hi(v[q]);
                        }
                    }
                }
            }
            // router term: rows 8c..8c+7 of W_r, all experts
            float racc[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) racc[q] = 0.f;
            if ((E & 7) == 0) {
                for (int e0 = 0; e0 < E; e0 += 8) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const u32x4_t wv = ld_u32x4(Wr + (long)(8 * c + q) * E + e0);
#pragma unroll
                        for (int h = 0; h < 4; ++h) {
                            racc[q] = racc[q] + dz[e0 + 2 * h] * bf_lo(wv[h]);
                            racc[q] = racc[q] + dz[e0 + 2 * h + 1] * bf_hi(wv[h]);
                        }
                    }
                }
            } else {
                for (int e = 0; e < E; ++e) {
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        racc[q] = racc[q] + dz[e] * bf2f(Wr[(long)(8 * c + q) * E + e]);
                }
            }
            u32x4_t o;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                o[q] = pack_bf2(acc[2 * q] + racc[2 * q], acc[2 * q + 1] + racc[2 * q + 1]);
            st_u32x4(dX + (long)t * d + 8 * c, o);
        }
    }
}

// The same sum for a small expert count (E = 8 EG, EG <= 2): one thread owns
// an 8-column chunk of dX for a group of tokens and keeps the 8 x E router
// weights of its chunk in registers, so W_r is read once per group instead of
// once per token; dZ rows are uniform loads.  The arithmetic and its order
// are those of reverse_combine_kernel, so the results are identical.
constexpr int RC_TG = 8;      // tokens per block
constexpr int RC_BT = 128;    // threads per block, one column chunk each

template <int EG>
__global__ __launch_bounds__(RC_BT) void reverse_combine_small_e_kernel(
        const uint16_t *__restrict__ dXperm, const uint16_t *__restrict__ dXsh,
        const float *__restrict__ dZ, const uint16_t *__restrict__ Wr,
        const int *__restrict__ route_pos, int T, int d, int k, int R,
        const float *__restrict__ dXacc, uint16_t *__restrict__ dX) {
    constexpr int E = 8 * EG;
    const int nc = d / 8;
    const int c = blockIdx.y * RC_BT + threadIdx.x;
    if (c >= nc) return;   // nothing below synchronises the block
    u32x4_t w[8][EG];
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
        for (int g = 0; g < EG; ++g) w[q][g] = ld_u32x4(Wr + (long)(8 * c + q) * E + 8 * g);
    const int t0 = blockIdx.x * RC_TG;
    const int t1 = min(T, t0 + RC_TG);
    for (int t = t0; t < t1; ++t) {
        float dz[E];
#pragma unroll
        for (int e = 0; e < E; ++e) dz[e] = dZ[(long)t * E + e];
        float acc[8];
        if (dXacc) {
            const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(dXacc + (long)t * d + 8 * c);
            const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(dXacc + (long)t * d + 8 * c + 4);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc[q] = lo[q];
                acc[4 + q] = hi[q];
            }
        } else {
            int pos[16];
#pragma unroll
            for (int s2 = 0; s2 < 16; ++s2) {
                pos[s2] = -1;
                if (s2 < k) {
                    const int p = route_pos[(long)t * k + s2];
                    pos[s2] = (p >= 0 && p < R) ? p : -1;
                }
            }
            u32x4_t rows[16];
#pragma unroll
            for (int s2 = 0; s2 < 16; ++s2)
                if (s2 < k) rows[s2] = ld_u32x4(dXperm + (long)max(pos[s2], 0) * d + 8 * c);
            if (dXsh) {
                const u32x4_t v = ld_u32x4(dXsh + (long)t * d + 8 * c);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[2 * q] = bf_lo(v[q]);
                    acc[2 * q + 1] = bf_hi(v[q]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = 0.f;
            }
#pragma unroll
            for (int s2 = 0; s2 < 16; ++s2) {
                if (s2 < k && pos[s2] >= 0) {
                    const u32x4_t v = rows[s2];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc[2 * q] = acc[2 * q] + bf_lo(v[q]);
                        acc[2 * q + 1] = acc[2 * q + 1] + bf_hi(v[q]);
                    }
                }
            }
        }
        float racc[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            racc[q] = 0.f;
#pragma unroll
            for (int g = 0; g < EG; ++g)
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    racc[q] = racc[q] + dz[8 * g + 2 * h] * bf_lo(w[q][g][h]);
                    racc[q] = racc[q] + dz[8 * g + 2 * h + 1] * bf_hi(w[q][g][h]);
                }
        }
        u32x4_t o;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            o[q] = pack_bf2(acc[2 * q] + racc[2 * q], acc[2 * q + 1] + racc[2 * q + 1]);
        st_u32x4(dX + (long)t * d + 8 * c, o);
    }
}

// Bounded-memory execution: per-route rows of the positions [w0, w1) live in
// a ring (row p at ring row p - w0).  For every token, the routes that fall
// in the window are added to an fp32 per-token accumulator in ascending slot
// order (optionally weighted by the gate weight); windows are visited in a
// fixed order, so the sums are deterministic.  `init` starts the accumulator
// at `add` (a bf16 row per token, the shared-expert term) or at zero; with
// `out` the result is rounded once into out instead of being stored in acc.
// A single window covering every route therefore adds in exactly the order
// of the one-pass combine.
__global__ __launch_bounds__(256) void window_accum_kernel(const uint16_t *__restrict__ ring, int w0,
                                                           int w1, const float *__restrict__ topk_w,
                                                           const int *__restrict__ route_pos, int T,
                                                           int d, int k, float *__restrict__ acc,
                                                           int init, const uint16_t *__restrict__ add,
                                                           uint16_t *__restrict__ out) {
    const int nc = d / 8;
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        int pos[16];
        float wt[16];
        bool any = false;
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            pos[s] = -1;
            wt[s] = 1.f;
            if (s < k) {
                const int p = route_pos[(long)t * k + s];
                pos[s] = (p >= w0 && p < w1) ? p - w0 : -1;
                if (topk_w) wt[s] = topk_w[(long)t * k + s];
                any = any || pos[s] >= 0;
            }
        }
        if (!any && !init && !out) continue;   // nothing of this token in the window
        for (int c = threadIdx.x; c < nc; c += 256) {
            float a[8];
            float *ap = acc + (long)t * d + 8 * c;
            if (init && add) {
                const u32x4_t v = ld_u32x4(add + (long)t * d + 8 * c);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[2 * q] = bf_lo(v[q]);
                    a[2 * q + 1] = bf_hi(v[q]);
                }
            } else if (init) {
#pragma unroll
                for (int q = 0; q < 8; ++q) a[q] = 0.f;
            } else {
                const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(ap);
                const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(ap + 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[q] = lo[q];
                    a[4 + q] = hi[q];
                }
            }
            u32x4_t rows[16];   // all loads first, as in the combine
#pragma unroll
            for (int s = 0; s < 16; ++s)
                if (s < k) rows[s] = ld_u32x4(ring + (long)max(pos[s], 0) * d + 8 * c);
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                if (s < k && pos[s] >= 0) {
                    const u32x4_t v = rows[s];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        a[2 * q] = a[2 * q] + wt[s] * bf_lo(v[q]);
                        a[2 * q + 1] = a[2 * q + 1] + wt[s] * bf_hi(v[q]);
                    }
                }
            }
            if (out) {
                u32x4_t o;
#pragma unroll
                for (int q = 0; q < 4; ++q) o[q] = pack_bf2(a[2 * q], a[2 * q + 1]);
                st_u32x4(out + (long)t * d + 8 * c, o);
            } else {
                *reinterpret_cast<f32x4_t *>(ap) = f32x4_t{a[0], a[1], a[2], a[3]};
                *reinterpret_cast<f32x4_t *>(ap + 4) = f32x4_t{a[4], a[5], a[6], a[7]};
            }
        }
    }
}

// Expert regions restricted to the window [w0, w1).
__global__ __launch_bounds__(256) void clip_offsets_kernel(const int *__restrict__ offsets, int E,
                                                           int w0, int w1, int *__restrict__ out) {
    for (int e = threadIdx.x; e <= E; e += 256) out[e] = min(max(offsets[e], w0), w1);
}

// dW_r = X^T dZ in two fixed-order stages.  Stage 1: block (256 columns,
// chunk of DWR_TC tokens) -> part[chunk][i][e]; stage 2 sums the chunks in
// order.
constexpr int DWR_TC = 256;             // tokens per chunk

// Stage 1 on MFMA.  dZ is split into bf16 hi + lo (hi = dZ rounded to bf16,
// lo = the rest rounded again; each bf16 x bf16 product is exact in fp32), so
// dW_r[i][e] = sum_t X[t][i] hi[t][e] + sum_t X[t][i] lo[t][e] with fp32
// accumulation, and the contraction over tokens runs as
// v_mfma_f32_16x16x32_bf16 with M = 16 columns of X, N = 8 experts x
// {hi, lo}, K = 32 tokens.  A block owns 256 columns and one chunk of
// DWR_TC tokens (4 steps of 64); each wave owns 64 columns (4 m-tiles).
// X[64][256] tiles reach LDS by direct loads (global_load_lds_dwordx4, two
// stages, the next step in flight while one is multiplied); the chunk's
// split dZ is staged once per group of 8 experts.  X fragments come from the
// transposing ds_read_b64_tr_b16, which hands each lane one column of a
// 4 x 16 block.  X's LDS rows are 512 bytes with the 32-byte block index XOR
// s(k) = (k & 3) | ((k >> 3) & 3) << 2, so the 16 rows one transposing read
// touches sit at 16 different block positions; the swizzle is applied on the
// global side of the loads.  74 KB of LDS: two blocks per CU.
constexpr int DWM_COLS = 256;            // columns per block
constexpr int DWM_STEP = 64;             // tokens per LDS stage
constexpr int DWM_ZLD = DWR_TC + 8;      // padded row of the split-dZ tile

typedef __bf16 dwm_bf16x4_t __attribute__((ext_vector_type(4)));
#define DWM_LDS __attribute__((address_space(3)))

DEV int dwm_swz(int k) { return (k & 3) | (((k >> 3) & 3) << 2); }

// Workgroup barrier without the fence __syncthreads() carries (which would
// wait for the direct loads still in flight); each wave waits for its own
// loads first, and LDS reads before it have all been consumed.
DEV void dwm_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(N), other counters untouched (gfx9 encoding).
template <int N>
DEV void dwm_wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__global__ __launch_bounds__(256) void dwr_mfma_kernel(const uint16_t *__restrict__ X,
                                                       const float *__restrict__ dZ, int T, int d,
                                                       int E, float *__restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint16_t xa[DWM_STEP * DWM_COLS];
    __shared__ __attribute__((aligned(16))) uint16_t xb[DWM_STEP * DWM_COLS];
    __shared__ __attribute__((aligned(16))) uint16_t zsh[16 * DWM_ZLD];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r = lane & 15;
    const int i0 = blockIdx.x * DWM_COLS;
    const int ch = blockIdx.y;
    const int tc0 = ch * DWR_TC, tc1 = min(T, tc0 + DWR_TC);
    const int n = (tc1 - tc0 + DWM_STEP - 1) / DWM_STEP;

    // this lane's 8 direct loads of a step: LDS row 16 wave + 2p + lane / 32,
    // 16-byte position lane % 32, which holds global chunk lcol (swizzle)
    int lrow[8], lcol[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const int row = 16 * wave + 2 * p + (lane >> 5), pos = lane & 31;
        lrow[p] = row;
        lcol[p] = i0 + 8 * (2 * ((pos >> 1) ^ dwm_swz(row)) + (pos & 1));
    }
    // rows past the chunk re-read its last token; their dZ entries are 0
    auto issue = [&](uint16_t *buf, int st) {
        const int tb = tc0 + st * DWM_STEP;
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const int t = min(tb + lrow[p], tc1 - 1);
            __builtin_amdgcn_global_load_lds(X + (long)t * d + lcol[p],
                                             (DWM_LDS void *)(buf + (8 * wave + p) * 512), 16, 0, 0);
        }
    };
    auto compute = [&](const uint16_t *buf, int st, f32x4_t (&acc)[4]) {
#pragma unroll
        for (int ks = 0; ks < DWM_STEP / 32; ++ks) {
            const bf16x8_t bz = __builtin_bit_cast(
                bf16x8_t, *reinterpret_cast<const u32x4_t *>(
                              &zsh[r * DWM_ZLD + DWM_STEP * st + 32 * ks + 8 * g]));
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int cb = wave * 64 + 16 * mt;   // first column of the m-tile
                dwm_bf16x4_t v[2];
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int k = 32 * ks + 8 * g + 4 * q + (r >> 2);
                    const int off = k * DWM_COLS + (((cb >> 4) ^ dwm_swz(k)) << 4) + 4 * (r & 3);
                    v[q] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((DWM_LDS dwm_bf16x4_t *)(buf + off));
                }
                const bf16x8_t a = bf16x8_t{v[0][0], v[0][1], v[0][2], v[0][3],
                                            v[1][0], v[1][1], v[1][2], v[1][3]};
                acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bz, acc[mt], 0, 0, 0);
            }
        }
    };

    for (int eg0 = 0; eg0 < E; eg0 += 8) {
        // the chunk's dZ for experts eg0 .. eg0 + 7, split: rows 0-7 hi, 8-15 lo
        {
            // all 8 loads issued together (clamped in bounds), then masked
            const int t = tc0 + tid;   // 256 threads = DWR_TC tokens
            const float *zrow = dZ + (long)min(t, tc1 - 1) * E;
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = zrow[min(eg0 + e, E - 1)];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float z = (t < tc1 && eg0 + e < E) ? v[e] : 0.f;
                const uint16_t hi = f2bf(z);
                zsh[e * DWM_ZLD + tid] = hi;
                zsh[(8 + e) * DWM_ZLD + tid] = f2bf(z - bf2f(hi));
            }
        }
        __syncthreads();
        f32x4_t acc[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        issue(xa, 0);
        if (n > 1) issue(xb, 1);
        for (int st = 0; st < n; st += 2) {
            // step st from xa: in flight are st and, if it exists, st + 1
            if (st + 1 < n) dwm_wait_vmcnt<8>(); else dwm_wait_vmcnt<0>();
            dwm_barrier();
            compute(xa, st, acc);
            dwm_barrier();
            if (st + 2 < n) issue(xa, st + 2);
            if (st + 1 < n) {
                if (st + 2 < n) dwm_wait_vmcnt<8>(); else dwm_wait_vmcnt<0>();
                dwm_barrier();
                compute(xb, st + 1, acc);
                dwm_barrier();
                if (st + 3 < n) issue(xb, st + 3);
            }
        }
        // lane (g, r) holds columns 4g + q of each m-tile for n = r: hi for
        // r < 8, lo for r >= 8; hi + lo, then the lane with r < 8 stores
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float lo = __shfl_xor(acc[mt][q], 8);
                const int e = eg0 + r;
                if (r < 8 && e < E) {
                    const int i = i0 + wave * 64 + 16 * mt + 4 * g + q;
                    part[((long)ch * d + i) * E + e] = acc[mt][q] + lo;
                }
            }
    }
}

__global__ __launch_bounds__(256) void dwr_reduce_kernel(const float *__restrict__ part, int nch,
                                                         long n, float *__restrict__ dWr) {
    const long q = (long)blockIdx.x * 256 + threadIdx.x;
    if (q >= n) return;
    // 16 chunk loads in flight at a time, added in chunk order
    float acc = 0.f;
    for (int c0 = 0; c0 < nch; c0 += 16) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = c0 + u < nch ? part[(long)(c0 + u) * n + q] : 0.f;
#pragma unroll
        for (int u = 0; u < 16; ++u)
            if (c0 + u < nch) acc = acc + v[u];
    }
    dWr[q] = acc;
}

inline unsigned rows_grid(long rows) { return (unsigned)(rows < 16384 ? (rows > 0 ? rows : 1) : 16384); }

// Transpose of a [T][d] bf16 matrix into [d][ldt] through 64 x 64 LDS tiles;
// columns T .. ldt - 1 of the result are written as zeros.  Grid (ldt / 64,
// d / 64); each thread moves two 16-byte chunks each way.
__global__ __launch_bounds__(256) void transpose_rows_kernel(const uint16_t *__restrict__ X, int T,
                                                             int d, uint16_t *__restrict__ XT,
                                                             long ldt) {
    __shared__ uint16_t tile[64][64 + 8];
    const int t0 = blockIdx.x * 64, c0 = blockIdx.y * 64, tid = threadIdx.x;
    X += (long)blockIdx.z * T * d;       // matrix z of a batch
    XT += (long)blockIdx.z * d * ldt;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int ch = h * 256 + tid, r = ch >> 3, c = 8 * (ch & 7);   // row t0 + r, columns c0 + c ..
        u32x4_t v = u32x4_t{0, 0, 0, 0};
        if (t0 + r < T) v = ld_u32x4(X + (long)(t0 + r) * d + c0 + c);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            tile[r][c + 2 * q] = (uint16_t)(v[q] & 0xffffu);
            tile[r][c + 2 * q + 1] = (uint16_t)(v[q] >> 16);
        }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int ch = h * 256 + tid, r = ch >> 3, c = 8 * (ch & 7);   // XT row c0 + r, columns t0 + c ..
        u32x4_t v;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            v[q] = (uint32_t)tile[c + 2 * q][r] | ((uint32_t)tile[c + 2 * q + 1][r] << 16);
        st_u32x4(XT + (long)(c0 + r) * ldt + t0 + c, v);
    }
}

// Rows of 64 bf16 for the router term of the dense dX product: row t < T
// holds the high and low bf16 parts of dZ[t][e] (hi = RNE(v), lo = RNE(v - hi),
// so hi + lo carries about 16 significant bits) in columns e and 32 + e; row
// T + n holds W_r[n][e] in both.  Multiplying the two row sets over the 64
// columns gives sum_e dZ[t][e] W_r[n][e] (hi W + lo W).  One thread per row.
__global__ __launch_bounds__(256) void router_split_kernel(const float *__restrict__ dZ,
                                                           const uint16_t *__restrict__ Wr, int T,
                                                           int d, int E, uint16_t *__restrict__ dzs,
                                                           uint16_t *__restrict__ wrs) {
    const long i = (long)blockIdx.x * 256 + threadIdx.x;
    if (i >= (long)T + d) return;
    uint32_t w[32];
#pragma unroll
    for (int q = 0; q < 32; ++q) w[q] = 0u;
    uint16_t *dst;
    if (i < T) {
#pragma unroll
        for (int e = 0; e < 32; ++e) {
            if (e < E) {
                const float v = dZ[i * E + e];
                const uint16_t hi = f2bf(v);
                const uint16_t lo = f2bf(v - bf2f(hi));
                w[e >> 1] |= (uint32_t)hi << (16 * (e & 1));
                w[16 + (e >> 1)] |= (uint32_t)lo << (16 * (e & 1));
            }
        }
        dst = dzs + i * 64;
    } else {
        const long n = i - T;
#pragma unroll
        for (int e = 0; e < 32; ++e) {
            if (e < E) {
                const uint32_t v = Wr[n * E + e];
                w[e >> 1] |= v << (16 * (e & 1));
                w[16 + (e >> 1)] |= v << (16 * (e & 1));
            }
        }
        dst = wrs + n * 64;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
        st_u32x4(dst + 8 * q, u32x4_t{w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]});
}

}  // namespace

int dwr_nchunks(long T) { return (int)((T + DWR_TC - 1) / DWR_TC); }

hipError_t launch_gather(const uint16_t *X, const int *perm, const int *offsets, int E, int k, int T,
                         int d, uint16_t *Xperm, hipStream_t st) {
    const long R = (long)T * k;
    if (R == 0) return hipSuccess;
    gather_rows_kernel<<<dim3(rows_grid(R)), dim3(256), 0, st>>>(X, perm, offsets, E, k, T, d, (int)R, Xperm);
    return hipGetLastError();
}

hipError_t launch_prep(const int *perm, const int *offsets, int E, const float *topk_w, int k, int T,
                       int *rowidx, float *wperm, uint16_t *zeros, hipStream_t st) {
    const long R = (long)T * k;
    const long n = R > ZERO_PAGE_ELEMS ? R : ZERO_PAGE_ELEMS;
    prep_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(perm, offsets, E, topk_w, k, T,
                                                                         (int)R, rowidx, wperm, zeros);
    return hipGetLastError();
}

hipError_t launch_combine(const uint16_t *Yexp, const uint16_t *Ysh, const float *topk_w,
                          const int *route_pos, int T, int d, int k, uint16_t *Y, hipStream_t st) {
    if (T == 0) return hipSuccess;
    combine_kernel<<<dim3(rows_grid(T)), dim3(256), 0, st>>>(Yexp, Ysh, topk_w, route_pos, T, d, k,
                                                              T * k, Y);
    return hipGetLastError();
}

hipError_t launch_softmax_bwd(const float *dgpart, int nparts, const int *route_pos,
                              const float *topk_w, const int *topk_idx, int T, int k, int E,
                              float *dg_out, float *dZ, hipStream_t st) {
    if (T == 0) return hipSuccess;
    softmax_bwd_kernel<<<dim3((unsigned)((T + 255) / 256)), dim3(256), 0, st>>>(
        dgpart, nparts, route_pos, topk_w, topk_idx, T, k, E, T * k, dg_out, dZ);
    return hipGetLastError();
}

hipError_t launch_reverse_combine(const uint16_t *dXperm, const uint16_t *dXsh, const float *dZ,
                                  const uint16_t *W_r, const int *route_pos, int T, int d, int k,
                                  int E, const float *dXacc, uint16_t *dX, hipStream_t st) {
    if (T == 0) return hipSuccess;
    if (E == 8 || E == 16) {
        const dim3 grid((unsigned)((T + RC_TG - 1) / RC_TG), (unsigned)((d / 8 + RC_BT - 1) / RC_BT));
        if (E == 8)
            reverse_combine_small_e_kernel<1><<<grid, dim3(RC_BT), 0, st>>>(
                dXperm, dXsh, dZ, W_r, route_pos, T, d, k, T * k, dXacc, dX);
        else
            reverse_combine_small_e_kernel<2><<<grid, dim3(RC_BT), 0, st>>>(
                dXperm, dXsh, dZ, W_r, route_pos, T, d, k, T * k, dXacc, dX);
        return hipGetLastError();
    }
    reverse_combine_kernel<<<dim3(rows_grid(T)), dim3(256), 0, st>>>(dXperm, dXsh, dZ, W_r, route_pos,
                                                                      T, d, k, E, T * k, dXacc, dX);
    return hipGetLastError();
}

hipError_t launch_window_accum(const uint16_t *ring, int w0, int w1, const float *topk_w,
                               const int *route_pos, int T, int d, int k, float *acc, int init,
                               const uint16_t *add, uint16_t *out, hipStream_t st) {
    if (T == 0) return hipSuccess;
    window_accum_kernel<<<dim3(rows_grid(T)), dim3(256), 0, st>>>(ring, w0, w1, topk_w, route_pos, T, d,
                                                                   k, acc, init, add, out);
    return hipGetLastError();
}

hipError_t launch_clip_offsets(const int *offsets, int E, int w0, int w1, int *out, hipStream_t st) {
    clip_offsets_kernel<<<dim3(1), dim3(256), 0, st>>>(offsets, E, w0, w1, out);
    return hipGetLastError();
}

hipError_t launch_dwr(const uint16_t *X, const float *dZ, int T, int d, int E, float *part,
                      float *dWr, hipStream_t st) {
    if (d % DWM_COLS) return hipErrorInvalidValue;   // the layer requires d % 256 == 0
    const int nch = dwr_nchunks(T);
    const long n = (long)d * E;
    if (nch > 0) {
        dim3 grid((unsigned)(d / DWM_COLS), (unsigned)nch);
        dwr_mfma_kernel<<<grid, dim3(256), 0, st>>>(X, dZ, T, d, E, part);
    }
    dwr_reduce_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(part, nch, n, dWr);
    return hipGetLastError();
}

hipError_t launch_router_split(const float *dZ, const uint16_t *W_r, int T, int d, int E,
                               uint16_t *dz_split, uint16_t *wr_split, hipStream_t st) {
    if (E > 32) return hipErrorInvalidValue;
    const long n = (long)T + d;
    if (n <= 0) return hipSuccess;
    router_split_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(dZ, W_r, T, d, E,
                                                                                  dz_split, wr_split);
    return hipGetLastError();
}

hipError_t launch_transpose_rows(const uint16_t *X, int T, int d, uint16_t *XT, long ldt,
                                 hipStream_t st, int batch) {
    if (ldt % 64 || ldt < T || d % 64 || batch < 1) return hipErrorInvalidValue;
    if (ldt == 0 || d == 0) return hipSuccess;
    transpose_rows_kernel<<<dim3((unsigned)(ldt / 64), (unsigned)(d / 64), (unsigned)batch), dim3(256), 0,
                            st>>>(X, T, d, XT, ldt);
    return hipGetLastError();
}
