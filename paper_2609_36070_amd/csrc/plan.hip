// Dispatch plan: Algorithm 1 of §3.1 with a single source rank, built on the
// device with no host readback.  With one rank the position of route j in
// expert e's region is the number of earlier routes to e, so the plan is a
// stable counting sort of the routes by expert:
//
//   1. plan_hist:    per-chunk expert histograms (LDS integer counters),
//                    stored expert-major ([E][chunks]) so that the scan's
//                    lanes, one chunk each, read and write consecutive words;
//   2. plan_scan:    exclusive scans over chunks (per expert) and experts;
//   3. plan_scatter: each chunk walks its routes in order in 64-lane groups;
//                    lanes with equal expert ids are matched with ballots, so
//                    ranks come from popcounts, never from position atomics.
//
// Every step is integer-exact and independent of scheduling.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int MAXE = 256;

__global__ __launch_bounds__(64) void plan_hist_kernel(const int *__restrict__ idx, int R, int E,
                                                       int *__restrict__ blockcounts,
                                                       int *__restrict__ blockflags) {
    __shared__ int cnt[MAXE];
    const int b = blockIdx.x, l = threadIdx.x;
    for (int e = l; e < E; e += 64) cnt[e] = 0;
    __syncthreads();
    const int j0 = b * PLAN_CHUNK;
    const int j1 = min(R, j0 + PLAN_CHUNK);
    // all of the lane's ids first (their loads overlap), then the counts
    constexpr int PER = PLAN_CHUNK / 64;
    int ev[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int j = j0 + l + 64 * q;
        ev[q] = j < j1 ? idx[j] : 0;
    }
    int bad = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        if (j0 + l + 64 * q >= j1) break;
        const int e = ev[q];
        if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
        else bad = 1;
    }
    __syncthreads();
    for (int e = l; e < E; e += 64) blockcounts[(long)e * gridDim.x + b] = cnt[e];
    const unsigned long long anybad = __ballot(bad);
    if (l == 0) blockflags[b] = anybad != 0ull;
}

DEV int wave_incl_scan(int v, int l) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(v, off, 64);
        if (l >= off) v += y;
    }
    return v;
}

__global__ __launch_bounds__(1024) void plan_scan_kernel(int nb, int E,
                                                         const int *__restrict__ blockcounts,
                                                         int *__restrict__ blockbase,
                                                         int *__restrict__ counts,
                                                         int *__restrict__ offsets,
                                                         const int *__restrict__ blockflags,
                                                         int *__restrict__ err) {
    __shared__ int tot[MAXE];
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    if (nb <= 256) {
        // up to 256 chunks: lane l holds chunks l + 64 m of each of the
        // wave's experts (e = w + 16 q), all loaded before any scan
        constexpr int QN = MAXE / 16;
        int v[QN][4];
        const int nm = (nb + 63) / 64;   // 64-chunk groups in use
#pragma unroll
        for (int q = 0; q < QN; ++q)
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int e = w + 16 * q, b = l + 64 * m;
                v[q][m] = (e < E && m < nm && b < nb) ? blockcounts[(long)e * nb + b] : 0;
            }
#pragma unroll
        for (int q = 0; q < QN; ++q) {
            const int e = w + 16 * q;
            if (e >= E) break;
            int run = 0;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                if (m >= nm) break;
                const int b = l + 64 * m;
                const int x = wave_incl_scan(v[q][m], l);
                if (b < nb) blockbase[(long)e * nb + b] = run + x - v[q][m];
                run += __shfl(x, 63, 64);
            }
            if (l == 0) tot[e] = run;
        }
    } else {
        for (int e = w; e < E; e += 16) {
            int run = 0;
            for (int base = 0; base < nb; base += 64) {
                const int b = base + l;
                const int v = b < nb ? blockcounts[(long)e * nb + b] : 0;
                const int x = wave_incl_scan(v, l);
                if (b < nb) blockbase[(long)e * nb + b] = run + x - v;
                run += __shfl(x, 63, 64);
            }
            if (l == 0) tot[e] = run;
        }
    }
    __syncthreads();
    if (w == 0) {
        int run = 0;
        for (int base = 0; base < E; base += 64) {
            const int e = base + l;
            const int v = e < E ? tot[e] : 0;
            const int x = wave_incl_scan(v, l);
            if (e < E) {
                offsets[e] = run + x - v;
                counts[e] = v;
            }
            run += __shfl(x, 63, 64);
        }
        if (l == 0) offsets[E] = run;
    } else if (w == 1) {
        int f = 0;
        for (int b = l; b < nb; b += 64) f |= blockflags[b];
        const unsigned long long any = __ballot(f != 0);
        if (l == 0) err[0] = any != 0ull;
    }
}

__global__ __launch_bounds__(64) void plan_scatter_kernel(const int *__restrict__ idx, int R, int E,
                                                          int ebits,
                                                          const int *__restrict__ blockbase,
                                                          const int *__restrict__ offsets,
                                                          int *__restrict__ perm,
                                                          int *__restrict__ route_pos) {
    __shared__ int run[MAXE];
    const int b = blockIdx.x, l = threadIdx.x;
    for (int e = l; e < E; e += 64) run[e] = offsets[e] + blockbase[(long)e * gridDim.x + b];
    __syncthreads();
    const int j0 = b * PLAN_CHUNK;
    const int j1 = min(R, j0 + PLAN_CHUNK);
    const unsigned long long lt = (l == 0) ? 0ull : (~0ull >> (64 - l));
    // all of the lane's ids first (their loads overlap), then the ranks
    constexpr int PER = PLAN_CHUNK / 64;
    int ev[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int j = j0 + l + 64 * q;
        ev[q] = j < j1 ? idx[j] : -1;
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int base = j0 + 64 * q;
        if (base >= j1) break;
        const int j = base + l;
        const bool valid = j < j1;
        const int e = valid ? ev[q] : -1;
        const bool ok = valid && e >= 0 && e < E;
        unsigned long long m = __ballot(ok);
        for (int bit = 0; bit < ebits; ++bit) {
            const bool on = ok && ((e >> bit) & 1);
            const unsigned long long bb = __ballot(on);
            m &= on ? bb : ~bb;
        }
        if (!ok) m = 0ull;
        const int rank = __popcll(m & lt);
        const int grp = __popcll(m);
        const int pos = ok ? run[e] + rank : -1;
        __syncthreads();
        if (ok && rank == grp - 1) run[e] += grp;
        __syncthreads();
        if (valid) route_pos[j] = (ok && pos < R) ? pos : -1;
        if (ok && pos >= 0 && pos < R) perm[pos] = j;
    }
}

}  // namespace

int plan_nblocks(long R) { return (int)((R + PLAN_CHUNK - 1) / PLAN_CHUNK); }

hipError_t launch_plan(const int *topk_idx, int R, int E, int *counts, int *offsets, int *perm,
                       int *route_pos, int *blockcounts, int *blockbase, int *blockflags,
                       int *err, hipStream_t st) {
    const int nb = plan_nblocks(R);
    int ebits = 0;
    while ((1 << ebits) < E) ++ebits;
    if (nb > 0)
        plan_hist_kernel<<<dim3(nb), dim3(64), 0, st>>>(topk_idx, R, E, blockcounts, blockflags);
    plan_scan_kernel<<<dim3(1), dim3(1024), 0, st>>>(nb, E, blockcounts, blockbase, counts, offsets,
                                                      blockflags, err);
    if (nb > 0)
        plan_scatter_kernel<<<dim3(nb), dim3(64), 0, st>>>(topk_idx, R, E, ebits, blockbase, offsets,
                                                            perm, route_pos);
    return hipGetLastError();
}
