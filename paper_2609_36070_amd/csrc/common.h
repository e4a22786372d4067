// Shared device helpers for the gfx950 MoE kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

#define DEV __device__ __forceinline__

// bf16 bits -> fp32 (exact)
DEV float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
DEV float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
DEV float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (gfx950 converts natively).
DEV uint16_t f2bf(float x) {
    __bf16 b = (__bf16)x;
    return __builtin_bit_cast(uint16_t, b);
}
// Two at once: one v_cvt_pk_bf16_f32 with both sources (the scalar
// conversions above take one each, plus a shift and an OR to combine them).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
DEV uint32_t pack_bf2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// The gated activation's logistic function from the hardware base-2
// exponential and reciprocal (v_exp_f32, v_rcp_f32, each within about 1 ulp,
// plus the rounding of -a log2(e)): a handful of instructions where expf and
// an IEEE division take about twenty, which matters in the SwiGLU epilogues,
// whose per-element arithmetic is a large part of their time.  Limits:
// a -> +inf gives 1, a -> -inf gives 0, NaN stays NaN.
DEV float sigmoid_f(float a) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-a * 1.4426950408889634f));
}
DEV float silu_f(float a) { return a * sigmoid_f(a); }

typedef float f32x8 __attribute__((ext_vector_type(8)));

DEV int wave_lane() { return threadIdx.x & 63; }

// 32-bit wave shuffles
DEV float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, 64); }
DEV int shfl_xor_i(int v, int m) { return __shfl_xor(v, m, 64); }

DEV u32x4_t ld_u32x4(const void *p) { return *reinterpret_cast<const u32x4_t *>(p); }
DEV void st_u32x4(void *p, u32x4_t v) { *reinterpret_cast<u32x4_t *>(p) = v; }
DEV u32x2_t ld_u32x2(const void *p) { return *reinterpret_cast<const u32x2_t *>(p); }
// 8 consecutive floats (two 16-byte accesses)
DEV f32x8 ld_f32x8(const float *p) {
    const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(p);
    const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(p + 4);
    return f32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}
DEV void st_f32x8(float *p, const f32x8 &v) {
    *reinterpret_cast<f32x4_t *>(p) = f32x4_t{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4_t *>(p + 4) = f32x4_t{v[4], v[5], v[6], v[7]};
}

// 8 floats -> 8 bf16 (round to nearest even) packed in 16 bytes
DEV u32x4_t pack_bf8(const f32x8 &v) {
    return u32x4_t{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                   pack_bf2(v[6], v[7])};
}

// XCD-aware raster of the grouped GEMMs.  Workgroups are dealt to the 8 XCDs
// round-robin (workgroup b runs on XCD b % 8).  The tiles are cut into groups
// of RASTER_GM m-tiles x all n-tiles, walked m-tile fastest; group g goes to
// XCD g % 8, and each XCD walks its groups in order.  The ~32 workgroups an
// XCD runs at once then share RASTER_GM A panels and ~8 B panels in its L2,
// and at any time the 8 XCDs work on 8 neighbouring groups, which read the
// same expert's weights: those reads hit in the Infinity Cache instead of
// each XCD streaming a different expert from HBM (3-7 % faster than giving
// each XCD one contiguous run of groups).  Slots past the tiles return at once.
constexpr int RASTER_GM = 4;

DEV bool map_tile(int b, int tiles_m, int ntn, int &mt, int &nt) {
    constexpr int NX = 8, GM = RASTER_GM;
    const int x = b % NX, j = b / NX;
    const int tpg = GM * ntn;
    const int group = (j / tpg) * NX + x;
    const int within = j % tpg;
    const int first = group * GM;
    if (first >= tiles_m) return false;
    const int gm = min(GM, tiles_m - first);
    if (within >= gm * ntn) return false;
    mt = first + within % gm;
    nt = within / gm;
    return true;
}

// Workgroups of a launch whose tiles map_tile places.
inline long raster_grid(long tiles_m, int ntn) {
    const long groups = (tiles_m + RASTER_GM - 1) / RASTER_GM;
    return 8 * ((groups + 7) / 8) * RASTER_GM * ntn;
}

// Weight-gradient raster.  A tile's cost is its expert's route count, so
// XCDs that each ran whole experts would wait for the heaviest one (or idle
// outright when a window of the bounded-memory backward holds only some of
// the experts).  Instead each expert's ntm x ntn tiles are cut into blocks of
// 4 x 4 tiles, the blocks of all experts are numbered expert by expert, and
// block h goes to XCD h % 8: every XCD gets an equal share of each expert
// (up to one block), and the 32 tiles an XCD runs at once are two such
// blocks, each sharing 4 A and 4 B panels in that XCD's L2.
// Grid: 8 * 16 * ceil(groups * blocks_per_expert / 8) workgroups.
constexpr int WG_BM = 4, WG_BN = 4;
__host__ __device__ __forceinline__ int wgrad_blocks_per_expert(int ntm, int ntn) {
    return ((ntm + WG_BM - 1) / WG_BM) * ((ntn + WG_BN - 1) / WG_BN);
}
DEV bool map_tile_wgrad(int b, int groups, int ntm, int ntn, int &cm, int &nt) {
    constexpr int NX = 8, PER = WG_BM * WG_BN;
    const int nbm = (ntm + WG_BM - 1) / WG_BM;
    const int nb = wgrad_blocks_per_expert(ntm, ntn);
    const int j = b / NX;                        // position in this XCD's sequence
    const int h = (j / PER) * NX + b % NX;       // block
    const int t = j % PER;                       // tile within the block, m fastest
    const int e = h / nb, lb = h % nb;
    if (e >= groups) return false;
    const int mt = (lb % nbm) * WG_BM + t % WG_BM;
    nt = (lb / nbm) * WG_BN + t / WG_BM;
    if (mt >= ntm || nt >= ntn) return false;
    cm = e * ntm + mt;
    return true;
}

// Workgroups of a launch whose tiles map_tile_wgrad places.
inline long wgrad_grid(long groups, int ntm, int ntn) {
    const long nblk = groups * wgrad_blocks_per_expert(ntm, ntn);
    return 8L * WG_BM * WG_BN * ((nblk + 7) / 8);
}
