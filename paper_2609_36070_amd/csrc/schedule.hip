// Pull-based dispatch schedule for R source ranks: Algorithm 1 of §3.1.
//
// Input: the all-gathered routes A[R, NK] (global expert id of route j on
// source rank r).  For the current rank c with L local experts the schedule
// lists, region by region, which (source rank, route) lands at each position
// of the local expert-contiguous buffer.  Within local expert l's region the
// routes are ordered by (ordinal o, source rank r), o = the number of earlier
// routes of row r to the same expert, so the source ranks interleave
// round-robin.  The position inside the region is
//
//     p = sum_{r'} min(M[r', l], o) + #{r' < r : M[r', l] > o},
//
// i.e. the routes of all earlier ordinal rounds, then the ranks before r that
// still have a route in round o.
//
//   1. sched_hist:    per (row, chunk) local-expert histograms in LDS;
//   2. sched_scan:    per (row, expert) exclusive scan over chunks, in place
//                     (ordinal base of each chunk) and the totals M[r, l];
//   3. sched_scatter: region starts S[l] = sum_{l' < l} sum_r M[r, l'] (each
//                     block rebuilds them from M), then one lane per route:
//                     equal expert ids are matched with ballots, so ordinals
//                     come from popcounts and per-wave counts, then p from
//                     the formula above.
//
// Integer-exact, no atomics beyond LDS histogram counters, independent of
// scheduling order.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int MAXL = 256;

constexpr int HIST_THREADS = 256;

// Grid (chunks, R).  counts[(r * C + ch) * L + l] = local routes of row r,
// chunk ch, to local expert l; flags[r * C + ch] = the chunk holds an id
// outside [0, R * L).
__global__ __launch_bounds__(HIST_THREADS) void sched_hist_kernel(const int *__restrict__ A, int NK,
                                                                  int L, int lo, int nexp, int C,
                                                                  int *__restrict__ counts,
                                                                  int *__restrict__ flags) {
    __shared__ int cnt[MAXL];
    __shared__ int anybad;
    const int ch = blockIdx.x, r = blockIdx.y, t = threadIdx.x;
    for (int e = t; e < L; e += HIST_THREADS) cnt[e] = 0;
    if (t == 0) anybad = 0;
    __syncthreads();
    const int j0 = ch * SCHED_CHUNK;
    const int j1 = min(NK, j0 + SCHED_CHUNK);
    const int *row = A + (long)r * NK;
    int bad = 0;
    for (int j = j0 + t; j < j1; j += HIST_THREADS) {
        const int a = row[j];
        if (a < 0 || a >= nexp) bad = 1;
        else if (a >= lo && a < lo + L) atomicAdd(&cnt[a - lo], 1);
    }
    if (__ballot(bad) != 0ull && (t & 63) == 0) anybad = 1;
    __syncthreads();
    const long cb = ((long)r * C + ch) * L;
    for (int e = t; e < L; e += HIST_THREADS) counts[cb + e] = cnt[e];
    if (t == 0) flags[(long)r * C + ch] = anybad;
}

DEV int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(v, off, 64);
        if (lane >= off) v += y;
    }
    return v;
}

// One wave per (r, l): exclusive prefix over the row's chunks, in place
// (64 chunks per wave scan), and the row total M[r, l].
__global__ __launch_bounds__(256) void sched_scan_kernel(int R, int L, int C,
                                                         int *__restrict__ counts,
                                                         int *__restrict__ M) {
    const long i = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (i >= (long)R * L) return;
    const long r = i / L, l = i - r * L;
    int run = 0;
    for (int base = 0; base < C; base += 64) {
        const int ch = base + lane;
        int *p = counts + ((r * C + ch) * L + l);
        const int v = ch < C ? *p : 0;
        const int x = wave_incl_scan(v, lane);
        if (ch < C) *p = run + x - v;
        run += __shfl(x, 63, 64);
    }
    if (lane == 0) M[i] = run;
}

// Grid (chunks, R), SCHED_WAVES waves per block, wave w taking the
// SCHED_GROUPS consecutive 64-route groups that start at route
// 64 * SCHED_GROUPS * w of the chunk.  Every block first rebuilds, in LDS,
// the transposed zero-padded count table MT[l][r'] = M[r', l] (RP = R
// rounded up to 4) and the region starts S (column sums of M, then a scan
// over l); the first block also publishes S and the error word.
//
// A route's ordinal is the chunk's ordinal base + the same-expert routes of
// earlier waves (a per-wave count table) + those of earlier groups of its
// own wave + its rank among equal ids in its group.  Matches come from
// per-group ballots of the key bits: for group i, keybit[i][b] has lane x
// set iff route x is local with bit b of its expert set, so the lanes of
// group i holding expert e are  local[i] & AND_b (e_b ? keybit : ~keybit).
#ifndef MOE_SCHED_WAVES
#define MOE_SCHED_WAVES 8
#endif
constexpr int SCHED_WAVES = MOE_SCHED_WAVES;
constexpr int SCHED_GROUPS = SCHED_CHUNK / (64 * SCHED_WAVES);
static_assert(SCHED_GROUPS * 64 * SCHED_WAVES == SCHED_CHUNK, "chunk = waves x groups x 64");
constexpr int MAXLBITS = 8;

__global__ __launch_bounds__(64 * SCHED_WAVES) void sched_scatter_kernel(
    const int *__restrict__ A, int R, int NK, int L, int lo, int lbits, int C, int RP,
    const int *__restrict__ obase, const int *__restrict__ M, const int *__restrict__ flags,
    int *__restrict__ S, int *__restrict__ phi, long phi_rows, int *__restrict__ err) {
    constexpr int NT = 64 * SCHED_WAVES;
    __shared__ int base[MAXL];               // ordinal base of this chunk
    __shared__ int start[MAXL + 1];          // region starts
    __shared__ int wcnt[SCHED_WAVES][MAXL];  // per-wave expert counts
    __shared__ int badflag;
    extern __shared__ int4 mt4[];            // [L][RP] ints, 16-byte aligned
    int *mt = reinterpret_cast<int *>(mt4);
    const int ch = blockIdx.x, r = blockIdx.y;
    const int t = threadIdx.x, w = t >> 6, lane = t & 63;
    const bool first = ch == 0 && r == 0;
    const long cb = ((long)r * C + ch) * L;
    // this wave's routes first: they do not depend on the tables
    const int jw = ch * SCHED_CHUNK + 64 * SCHED_GROUPS * w + lane;
    int av[SCHED_GROUPS];
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i) {
        const int j = jw + 64 * i;
        av[i] = j < NK ? A[(long)r * NK + j] : -1;
    }
    if (t == 0) badflag = 0;
    for (int e = t; e < L; e += NT) base[e] = ch < C ? obase[cb + e] : 0;
    for (int i = t; i < SCHED_WAVES * MAXL; i += NT) (&wcnt[0][0])[i] = 0;
    for (int i = t; i < L * RP; i += NT) {
        const int l = i / RP, rp = i - l * RP;
        mt[i] = rp < R ? M[(long)rp * L + l] : 0;
    }
    int key[SCHED_GROUPS];
    bool loc[SCHED_GROUPS];
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i) {
        loc[i] = av[i] >= lo && av[i] < lo + L;
        key[i] = loc[i] ? av[i] - lo : 0;
    }
    // per-group ballots of locality and of each key bit
    unsigned long long lmask[SCHED_GROUPS], kb[SCHED_GROUPS][MAXLBITS];
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i) {
        lmask[i] = __ballot(loc[i]);
#pragma unroll
        for (int b = 0; b < MAXLBITS; ++b)
            kb[i][b] = b < lbits ? __ballot(loc[i] && ((key[i] >> b) & 1)) : 0ull;
    }
    // lanes of group g holding expert e
    auto match = [&](int g, int e) {
        unsigned long long m = lmask[g];
#pragma unroll
        for (int b = 0; b < MAXLBITS; ++b)
            if (b < lbits) m &= ((e >> b) & 1) ? kb[g][b] : ~kb[g][b];
        return m;
    };
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int before[SCHED_GROUPS];   // same-expert routes before this one inside the wave
    bool last[SCHED_GROUPS];    // the wave's last route to its expert
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i) {
        int n = 0, after = 0;
#pragma unroll
        for (int g = 0; g < SCHED_GROUPS; ++g) {
            const unsigned long long m = match(g, key[i]);
            if (g < i) n += __popcll(m);
            else if (g == i) n += __popcll(m & lt), after += __popcll(m & ~lt) - 1;
            else after += __popcll(m);
        }
        before[i] = n;
        last[i] = loc[i] && after == 0;
    }
    __syncthreads();   // the tables are staged and wcnt is zero
    // the wave's last route to each expert publishes the wave's count
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i)
        if (last[i]) wcnt[w][key[i]] = before[i] + 1;
    // region starts: per-expert totals (one wave per expert), then a scan
    for (int l = w; l < L; l += SCHED_WAVES) {
        int sum = 0;
        for (int rp = lane; rp < RP; rp += 64) sum += mt[l * RP + rp];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
        if (lane == 0) start[l] = sum;
    }
    if (first) {
        int f = 0;
        for (int i = t; i < R * C; i += NT) f |= flags[i];
        if (__ballot(f != 0) != 0ull && lane == 0) badflag = 1;
    }
    __syncthreads();
    if (w == 0) {
        int run = 0;
        for (int b0 = 0; b0 < L; b0 += 64) {
            const int l = b0 + lane;
            const int v = l < L ? start[l] : 0;
            const int x = wave_incl_scan(v, lane);
            if (l < L) start[l] = run + x - v;
            run += __shfl(x, 63, 64);
        }
        if (lane == 0) start[L] = run;
    }
    __syncthreads();
    if (first) {
        for (int l = t; l <= L; l += NT) S[l] = start[l];
        if (t == 0) err[0] = (badflag ? 1 : 0) | ((long)start[L] > phi_rows ? 2 : 0);
    }
#pragma unroll
    for (int i = 0; i < SCHED_GROUPS; ++i) {
        if (!loc[i]) continue;
        const int e = key[i];
        int o = base[e] + before[i];
        for (int g = 0; g < w; ++g) o += wcnt[g][e];
        // p = sum_r' min(M[r', e], o) + #{r' < r : M[r', e] > o}
        const int4 *col = mt4 + ((e * RP) >> 2);
        int p = 0;
#pragma unroll 4
        for (int q = 0; q < (RP >> 2); ++q) {
            const int4 v = col[q];
            const int r0 = 4 * q;
            p += min(v.x, o) + ((r0 + 0 < r && v.x > o) ? 1 : 0);
            p += min(v.y, o) + ((r0 + 1 < r && v.y > o) ? 1 : 0);
            p += min(v.z, o) + ((r0 + 2 < r && v.z > o) ? 1 : 0);
            p += min(v.w, o) + ((r0 + 3 < r && v.w > o) ? 1 : 0);
        }
        const long pos = (long)start[e] + p;
        if (pos < phi_rows) {
            int2 v;
            v.x = r;
            v.y = jw + 64 * i;
            reinterpret_cast<int2 *>(phi)[pos] = v;
        }
    }
}

}  // namespace

int sched_nchunks(long NK) { return (int)((NK + SCHED_CHUNK - 1) / SCHED_CHUNK); }

int sched_rpad(int R) { return (R + 3) & ~3; }

hipError_t launch_schedule(const int *A, int R, int NK, int L, int c, int *M, int *S, int *phi,
                           long phi_rows, int *counts, int *flags, int *err, hipStream_t st) {
    const int C = sched_nchunks(NK);
    const int RP = sched_rpad(R);
    int lbits = 0;
    while ((1 << lbits) < L) ++lbits;
    const int lo = c * L, nexp = R * L;
    if (C > 0) {
        sched_hist_kernel<<<dim3(C, R), dim3(HIST_THREADS), 0, st>>>(A, NK, L, lo, nexp, C, counts,
                                                                     flags);
    }
    const long pairs = (long)R * L;
    sched_scan_kernel<<<dim3((unsigned)((pairs + 3) / 4)), dim3(256), 0, st>>>(R, L, C, counts, M);
    // with no routes one scatter block still publishes S and the error word
    const size_t lds = (size_t)L * RP * 4;
    sched_scatter_kernel<<<dim3(C > 0 ? C : 1, R), dim3(64 * SCHED_WAVES), lds, st>>>(
        A, R, NK, L, lo, lbits, C, RP, counts, M, flags, S, phi, phi_rows, err);
    return hipGetLastError();
}
