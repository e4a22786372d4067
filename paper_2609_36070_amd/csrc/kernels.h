// Internal launcher declarations of the gfx950 MoE kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

constexpr int PLAN_CHUNK = 1024;  // routes per plan block
#ifndef MOE_SCHED_CHUNK
#define MOE_SCHED_CHUNK 512
#endif
constexpr int SCHED_CHUNK = MOE_SCHED_CHUNK;  // routes of one source rank per schedule block

// Grouped-GEMM problem description (see gemm.hip for the five modes).
struct GemmArgs {
    // operand A
    const uint16_t *A = nullptr;
    const uint16_t *A2 = nullptr;      // second K half (BWD_DX)
    long lda = 0;
    const int *a_rows = nullptr;       // row gather (MK rows / KM k-rows)
    int a_nrows = 1;                   // rows addressable through A (clamp bound)
    const uint16_t *zeros = nullptr;   // >= 512 zero bytes: source of k rows past a WGRAD count
    // operand B
    const uint16_t *B = nullptr;
    const uint16_t *B2 = nullptr;      // W_up (FWD_UP, BWD_DX)
    long ldb = 0;
    long b_estride = 0;                // elements between experts' weights
    const int *b_rows = nullptr;       // WGRAD: k-row gather
    int b_nrows = 1;
    // problem
    int M = 0, N = 0, K = 0;
    const int *offsets = nullptr;      // per-expert row ranges (device), or null
    int E = 0;
    // outputs
    uint16_t *C = nullptr, *C2 = nullptr, *C3 = nullptr;   // BWD_DGRAD: dA, dB, w*h
    long ldc = 0;
    float *Cf = nullptr;
    long c_estride = 0;
    const uint16_t *E1 = nullptr, *E2 = nullptr;  // BWD_DGRAD: saved A, B
    const float *rowscale = nullptr;              // BWD_DGRAD: router weight per row
    float *dgpart = nullptr;
    int dg_ld = 0;
    int accumulate = 0;                // WGRAD: add to Cf instead of overwriting it
    int tiles_m = 0;                   // set by the launcher: m-tile slots of the raster
    // fused forward (row products only): before loading, wait until
    // dep[m-tile slot] >= dep_need; after storing, add 1 to sig[m-tile slot]
    const int *dep = nullptr;
    int dep_need = 0;
    int *sig = nullptr;
    int sig_local = 0;                 // every waiter on sig runs on this tile's XCD
    int *err = nullptr;                // bit 1 set when a wait gave up
    // Dense routing (every token routes to every one of the E experts): the
    // K loop of a token tile runs over segments.  Routed segment e reads the
    // plan rows of the tile's tokens in expert e's region (seg_offsets[e] +
    // token) through A (and A2), against expert e's B (and B2); then the
    // shared expert's segments (As / Bs, As2 / Bs2, width segK_s); BWD_DX_CMB
    // ends with one 64-wide step of the router term (Ar, Br rows of 64).
    const int *seg_offsets = nullptr;  // the plan's offsets [E+1]
    int nseg = 0, segK = 0, segK_s = 0;
    // a segment's first row is clamped into [a_row0, a_nrows - M] (a window
    // of the plan held in a ring: its first row)
    int a_row0 = 0;
    // With Cf set, the token tiles keep a running fp32 sum over the windows
    // of a bounded-memory pass: Cf [M][ldc] holds the earlier windows' sum
    // (added first when accumulate), and the result goes to C (bf16, the
    // last window) or back to Cf.
    const uint16_t *As = nullptr, *As2 = nullptr, *Bs = nullptr, *Bs2 = nullptr;
    long lda_s = 0, ldb_s = 0;
    const uint16_t *Ar = nullptr, *Br = nullptr;
    // fused dense forward: a token tile also waits for dep2[m-tile] >= dep_need2
    // (the shared expert's up/gate tiles); dep is then indexed per expert
    const int *dep2 = nullptr;
    int dep_need2 = 0;
    int dep_slots = 0;                 // counters in dep (per-expert indices are clamped to it)
    // Dense routing: expert e's plan rows are all tokens in order, so a
    // gathered operand's row is the position minus offsets[e] (no index
    // loads); a_local for A (rows of a row product, k rows of WGRAD), b_local
    // for WGRAD's B.  The gather pointers are then ignored.
    int a_local = 0, b_local = 0;
    // The plan's offsets that turn such a row into a token (row minus the
    // expert's first plan row) when `offsets` are clipped to a window of the
    // plan (bounded-memory execution); null: `offsets` themselves.
    const int *tok_offsets = nullptr;
};

int gemm_tile_m();
int gemm_tile_n();
hipError_t launch_gemm_fwd_up(const GemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_fwd_down(const GemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_bwd_dgrad(const GemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_bwd_dx(const GemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_wgrad(const GemmArgs &g, int groups, hipStream_t st);
// The weight gradient with A given transposed: A [M][lda] row-major with its
// columns the expert's positions (from offsets[e]; with a_local the tokens,
// from 0), K-contiguous like the row products' operands; B as for WGRAD.  A's
// columns past an expert's last row must hold finite values (a padded pitch).
hipError_t launch_gemm_wgrad_t(const GemmArgs &g, int groups, hipStream_t st);
// ... and with B given transposed instead: B [N][ldb], columns as A's above.
hipError_t launch_gemm_wgrad_tb(const GemmArgs &g, int groups, hipStream_t st);
// X [T][d] -> XT [d][ldt] (ldt >= T rounded up to 64; columns T .. ldt-1 zero),
// for `batch` matrices stored one after the other on both sides.
hipError_t launch_transpose_rows(const uint16_t *X, int T, int d, uint16_t *XT, long ldt,
                                 hipStream_t st, int batch = 1);
// Dense routing (k == E): Y = sum over experts of (w h) W_down[e], plus the
// shared expert, over one token tile's K segments (the combine folded into the
// down product); dX likewise with dA W_gate^T + dB W_up^T per expert, the
// shared expert and the router term.  g.M = T, g.N = d.
hipError_t launch_gemm_fwd_down_cmb(const GemmArgs &g, hipStream_t st);
hipError_t launch_gemm_bwd_dx_cmb(const GemmArgs &g, hipStream_t st);
// Rows of 64 bf16 for the router term of the dense dX product: for dZ (fp32
// [T][E]) the high and low bf16 parts of each value in columns e and 32 + e;
// for W_r (bf16 [d][E]) the value in both.  E <= 32; other columns zero.
hipError_t launch_router_split(const float *dZ, const uint16_t *W_r, int T, int d, int E,
                               uint16_t *dz_split, uint16_t *wr_split, hipStream_t st);
// Up to 4 grouped weight-gradient products (same groups), optionally with one
// grouped up/gate product over `up_rows` plan rows, in one launch.
// Fused persistent forward: shared up/gate, routed up/gate, shared down,
// routed down and the combine in one launch (see gemm.hip).  `counters`
// holds fused_counter_ints(...) ints; the launcher clears them first.  A
// wait that gives up sets bit 1 of *err.
int fused_counter_ints(long T, long R, int E);
// With dense routing (down_r's mode is the folded down product: dense =
// true) there is no combine phase: down_r's token tiles write Y.
hipError_t launch_fused_forward(const GemmArgs &up_s, const GemmArgs &up_r, const GemmArgs &down_s,
                                const GemmArgs &down_r, bool shared, bool dense, long T, long R, int E,
                                const uint16_t *Yexp, const uint16_t *Ysh, const float *topk_w,
                                const int *route_pos, const int *topk_idx, const int *offsets, int d,
                                int k, uint16_t *Y, int *counters, int *err, hipStream_t st);
// modes[i] (null: all 0): 0 the weight gradient on column tiles, 1 with A
// read as the K-contiguous X^T (as launch_gemm_wgrad_t), 2 with B read as
// dY^T (as launch_gemm_wgrad_tb).
hipError_t launch_gemm_wgrad_batch(const GemmArgs *wg, int nw, int groups, const GemmArgs *up,
                                   long up_rows, hipStream_t st, const int *modes = nullptr);

int route_epad(int E);
// Scratch of the split router (many experts): fp32 partial logits of its d
// slices; 0 for shapes on the one-pass router.
size_t route_part_bytes(long T, int d, int E);
hipError_t launch_route(const uint16_t *X, const uint16_t *W_r, const float *bias, float *logits,
                        int *topk_idx, float *topk_w, uint16_t *WrT, float *part, int T,
                        int d, int E, int k, hipStream_t st);

int plan_nblocks(long R);
hipError_t launch_plan(const int *topk_idx, int R, int E, int *counts, int *offsets, int *perm,
                       int *route_pos, int *blockcounts, int *blockbase, int *blockflags, int *err,
                       hipStream_t st);

constexpr int SCHED_MAX_TABLE = 8192;  // L * (R rounded up to 4): the count table staged in LDS
// MXFP8 routed-expert GEMM problem (see gemm_mx.hip).
struct MxGemmArgs {
    const uint8_t *A = nullptr;        // [a_nrows][K] E4M3 rows
    const uint8_t *As = nullptr;       // [a_nrows][K/32] E8M0 scales
    const int *a_rows = nullptr;       // position -> A row (NULL: identity)
    int a_nrows = 1;
    const uint8_t *B = nullptr;        // [E][N or N/2][K] weight rows (gate for MX_UP)
    const uint8_t *Bs = nullptr;
    const uint8_t *B2 = nullptr;       // up weight rows (MX_UP)
    const uint8_t *Bs2 = nullptr;
    int K = 0, N = 0;                  // MX_UP: N = f (tile columns pair gate and up)
    const int *offsets = nullptr;      // [E+1] expert regions
    int E = 0;
    const uint8_t *A2 = nullptr;       // MX_DX: second K half of A (dBq) and its scales
    const uint8_t *As2 = nullptr;
    uint8_t *C = nullptr;              // MX_UP: Hq [rows][N]; MX_DGRAD: dAq
    uint8_t *Cs = nullptr;             // MX_UP: Hs [rows][N/32]; MX_DGRAD: dAs
    uint8_t *C2 = nullptr;             // MX_DGRAD: dBq, dBs
    uint8_t *Cs2 = nullptr;
    uint16_t *Cb = nullptr;            // MX_DOWN, MX_DX: bf16 [rows][N]; MX_DGRAD: dA bf16
    uint16_t *Cb2 = nullptr;           // MX_DGRAD: dB bf16
    uint16_t *Cb3 = nullptr;           // MX_DGRAD: w * h bf16
    float *Cf1 = nullptr;              // MX_DGRAD: dA, dB, w * h in fp32 instead of bf16
    float *Cf2 = nullptr;              //   (the token-axis quantisers of the MXFP8 weight
    float *Cf3 = nullptr;              //   gradients read them)
    float *Sa = nullptr;               // MX_UP: keep the gate / up pre-activations (fp32)
    float *Sb = nullptr;
    const float *E1 = nullptr;         // MX_DGRAD: saved pre-activations A, B (fp32)
    const float *E2 = nullptr;
    const float *rowscale = nullptr;   // MX_DGRAD: router weight per row
    float *dgpart = nullptr;           // MX_DGRAD: <dh', h> partial per row and n-tile
    int dg_ld = 0;
    uint32_t a_bytes = 0, as_bytes = 0, b_bytes = 0, bs_bytes = 0;   // operand extents (< 4 GiB)
    int tiles_m = 0;
    // MX_WGRAD: dW[e] = A[:, k_e] . B[:, k_e]^T over expert e's padded token
    // range k_e = [offsets[e], offsets[e+1]) (multiples of 128); A [M][K] and
    // B [N][K] hold token-axis codes, K is their row pitch in bytes
    int M = 0;
    float *Cf = nullptr;               // MX_WGRAD: fp32 [E][M][N]
    // MX_WGRAD with dense routing: every expert's token range holds the same
    // tokens, so X^T (A of dW_gate, dW_up) or dY^T (B of dW_down) is quantised
    // once, as expert 0's range, and read from position 0 for every expert
    int a_shared = 0, b_shared = 0;
};
hipError_t launch_gemm_mx_up(const MxGemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_mx_down(const MxGemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_mx_dgrad(const MxGemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_mx_dx(const MxGemmArgs &g, long rows, int groups, hipStream_t st);
hipError_t launch_gemm_mx_wgrad(const MxGemmArgs &g, int groups, hipStream_t st);
// Token-axis MXFP8 operands of the weight gradients: for each expert, the rows
// of its plan region (through `rows`: position -> source row, or the position
// itself) in 32-row blocks from the region's start, written transposed as
// [C][pitch] codes and [C][pitch / 32] scales at the expert's padded offset
// poff[e] (multiples of 128; positions past the region's rows are zeros).
// src has nsrc rows of pitch ld; max_pos (a multiple of 128) bounds poff[E].
hipError_t launch_mx_pad_offsets(const int *offsets, int E, int *poff, hipStream_t st);
hipError_t launch_mx_quant_tokens(const uint16_t *src, long ld, long nsrc, const int *rows,
                                  const int *offsets, const int *poff, int E, int C, long pitch,
                                  long max_pos, uint8_t *q, uint8_t *sc, hipStream_t st);
// The same for an fp32 source in plan order (no gather).
hipError_t launch_mx_quant_tokens_f32(const float *src, long ld, long nsrc, const int *offsets,
                                      const int *poff, int E, int C, long pitch, long max_pos,
                                      uint8_t *q, uint8_t *sc, hipStream_t st);
hipError_t launch_mx_quant_rows(const uint16_t *X, long rows, int K, uint8_t *q, uint8_t *sc,
                                hipStream_t st);
hipError_t launch_mx_quant_weights(const uint16_t *W, int E, int K, int N, uint8_t *q, uint8_t *sc,
                                   hipStream_t st);

int sched_nchunks(long NK);
int sched_rpad(int R);
hipError_t launch_schedule(const int *A, int R, int NK, int L, int c, int *M, int *S, int *phi,
                           long phi_rows, int *counts, int *flags, int *err, hipStream_t st);

int dwr_nchunks(long T);
hipError_t launch_gather(const uint16_t *X, const int *perm, const int *offsets, int E, int k, int T,
                         int d, uint16_t *Xperm, hipStream_t st);
hipError_t launch_prep(const int *perm, const int *offsets, int E, const float *topk_w, int k, int T,
                       int *rowidx, float *wperm, uint16_t *zeros, hipStream_t st);
constexpr int ZERO_PAGE_ELEMS = 512;  // bf16 elements of the zero page (1 KB)
hipError_t launch_combine(const uint16_t *Yexp, const uint16_t *Ysh, const float *topk_w,
                          const int *route_pos, int T, int d, int k, uint16_t *Y, hipStream_t st);
hipError_t launch_softmax_bwd(const float *dgpart, int nparts, const int *route_pos,
                              const float *topk_w, const int *topk_idx, int T, int k, int E,
                              float *dg_out, float *dZ, hipStream_t st);
hipError_t launch_reverse_combine(const uint16_t *dXperm, const uint16_t *dXsh, const float *dZ,
                                  const uint16_t *W_r, const int *route_pos, int T, int d, int k,
                                  int E, const float *dXacc, uint16_t *dX, hipStream_t st);
hipError_t launch_window_accum(const uint16_t *ring, int w0, int w1, const float *topk_w,
                               const int *route_pos, int T, int d, int k, float *acc, int init,
                               const uint16_t *add, uint16_t *out, hipStream_t st);
hipError_t launch_clip_offsets(const int *offsets, int E, int w0, int w1, int *out, hipStream_t st);
hipError_t launch_dwr(const uint16_t *X, const float *dZ, int T, int d, int E, float *part,
                      float *dWr, hipStream_t st);
