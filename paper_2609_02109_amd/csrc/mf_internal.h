// Internal declarations of libmf: device-side layouts, kernel argument blocks
// and the host-side launchers each .hip file provides.  Not installed; the C
// ABI is include/mf.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mf.h"

namespace mfi {

constexpr int kMaxN = MF_MAX_MODELS;
constexpr int kSearchWaves = 8;          // waves per workgroup of the fast search kernel (base)
constexpr int kSearchWavesWide = 16;     // ... when registers and LDS allow 4 waves per SIMD
constexpr int kCertWaves = 4;            // waves per workgroup of the canonical kernels
constexpr int kDefaultWorklist = 1 << 20; // certification list capacity (entries)
constexpr int kFastPar = 160;            // floats of per-model parameters after the fp32 fast image in LDS
constexpr int kFastLdsMax = 163840 - 512; // dynamic LDS of the fp32 fast kernel (its static LDS takes < 512 bytes)
constexpr int kBf16Waves = 8;            // waves per workgroup of the bf16 fast kernel
constexpr int kBf16Tiles = 8;            // 32-configuration tiles per wave and model staging
constexpr int kBf16Par = 128;            // floats of per-model parameters after the bf16 tables in LDS

// ---------------------------------------------------------------------------
// Fast-path LDS image.  The device copy of the image is laid out exactly as
// the fast kernel wants it in LDS, so its prologue is one straight copy.
// Offsets are in floats from the image start; every block is 16-byte aligned.
// Model i's layer-1 rows (w1a, p) are scaled by 2^e1[i], b2 by 2^(e1+e2),
// W2 by 2^e2 and W3 by 2^-(e1+e2): exact power-of-two scalings that keep the
// binary16 pieces of layer 2 in range and leave every fp32 rounding as it
// would be unscaled.
//   w1a[i][mb][lane][j]            A operand of layer 1 (aggregate columns):
//                                  binary16 w1 (j < ns) and w2 (j >= ns) of
//                                  2^(e1 - ex) W1[32 mb + lane%32][slot
//                                  2 (j%ns) + lane/32]; ns = 4 slots (16
//                                  bytes per lane), 2 when A <= 4 (8 bytes)
//   b2 [i][H]                      layer-2 bias (accumulator init)
//   w2 [i][mb2][mb1][kh][pc][lane][j]  A operands of layer 2: binary16 pieces
//                                  pc = 0 (w1), 1 (w2) of W2[32 mb2 + lane%32]
//                                  [32 mb1 + 16 kh + 8 (j/4) + 4 (lane/32) + j%4],
//                                  8 per lane (16 bytes; one float slot per weight)
//   w3 [i][o][mb2][q][half][j]     layer-3 weights in accumulator row order
//   b3 [i][2]  (padded to 4)
//   p  [row][pst]                  per-option first-layer precompute
//                                  b1 + W1_local x (fp64, rounded to fp32),
//                                  row = global option row
//   g  [row][half][4]              aggregate columns of each option row in
//                                  internal slot order (slot 0 = the VRAM
//                                  slot); internal slot 2s+half at [half][s]
//   c  [half][4]                   aggregate centre in the same order: layer 1
//                                  takes a - c (exact on the 2^-14 grid) and
//                                  P carries W1_agg c
//   c1 [i][c1_stride]              (when it fits) each model's canonical block
//                                  (W1T, b1, W2T, b2, W3, b3 as given), for
//                                  canonical evaluation
//   feat [row][L]                  (with c1) the option table
// ---------------------------------------------------------------------------
struct FastLayout {
    int H, A, AP, MB, S1, PST;
    int off_w1a, off_b2, off_w2, off_w3, off_b3, off_p, off_g, off_c;
    int off_c1, c1_stride;     // canonical block per model, W1T b1 W2T b2 W3 b3 as in the canonical image (-1: not in the image)
    int off_feat;              // the option table [sumK][L] (with the c1 block; -1: not in the image)
    int total_floats;          // multiple of 4
};

// The fp32 fast kernel's per-wave candidate lists are merged after the scan,
// when the image's blocks before g (weights and the per-option precompute)
// are no longer read: they take that space when it is large enough, else
// they follow the parameter block.
inline bool fast_lists_in_image(const FastLayout &ly, int waves, int kp)
{
    return (size_t)waves * kp * 8 <= (size_t)ly.off_g * 4;
}
inline size_t fast_dyn_lds(const FastLayout &ly, int waves, int kp, size_t ep_bytes)
{
    return (size_t)ly.total_floats * 4 + kFastPar * 4 +
           (fast_lists_in_image(ly, waves, kp) ? 0 : (size_t)waves * kp * 8) + ep_bytes;
}

// Per-problem constants of the fast kernels (kernel-argument block).
struct FastConst {
    int32_t n_models;
    int32_t act;                // output activation: 0 identity, 1 sigmoid (bounds below are then
                                // pre-activation for the latency, post-activation for the throughput)
    int32_t K[kMaxN];
    int32_t opt_off[kMaxN];     // first global option row of model i
    uint32_t magic[kMaxN];      // floor(2^32 / K) + 1 (K > 1), 0 for K == 1
    float vram_cap;
    // power-of-two scale 2^ex of internal aggregate slot 2s + half at
    // [half][s] (the fast kernel's binary16 layer-1 operand; 1 past A)
    float agg_scale[2][4];
    // a-priori bound on |fast - canonical| for (lat, thr) of model i, and on |thr|
    double bound_lat[kMaxN], bound_thr[kMaxN], mag_thr[kMaxN];
};

// Objective of a search (the full utility of Eq. 3 when kind == 1).  vrow
// holds two float4 per option row: (fmin, fmax, 1/(fmax - fmin) rounded to
// fp32, Q) and (variant as int bits, reload cost of the row's model, 0, 0).
struct ObjArgs {
    int32_t kind;
    float alpha, beta, delta;
    float tau[kMaxN];
    int32_t prev[kMaxN];
    const float4 *vrow;
};

// Counters and results the search kernels fill in device memory.
struct DevResult {
    unsigned long long n_vram, n_feas_sure, n_work, n_collect;
    unsigned long long n_feas_cert, n_cand;
    unsigned int status;        // see kStat*
    int n_top;
    unsigned long long top_idx[MF_MAX_TOPK];
    double top_J[MF_MAX_TOPK];
    double theta;               // fallback collect threshold on the upper bound U
    double eJ;                  // global bound on |fast J - canonical J| (fp32 path)
    double tail_U;              // upper bound U of the last fast candidate (list full)
    double check_max_dJ;        // max (U - canonical J) seen on candidates
    double ck_cand;             // k-th canonical J among the fast candidates
    unsigned long long fast_ticks;  // small ranges: wall-clock ticks from the first workgroup's start
                                    // to the last one's end of the fast kernel
    unsigned long long done_seq;    // small ranges, host copy: the call's sequence number, written last
};
constexpr unsigned kStatVerified = 1u;      // top-k exactness condition held
constexpr unsigned kStatSelfCheck = 2u;     // a fast decision disagreed with canonical
constexpr unsigned kStatWorkOverflow = 4u;
constexpr unsigned kStatCollectOverflow = 8u;
constexpr unsigned kStatListFull = 16u;

// Entry flags written by the canonical kernel (besides bit0 VRAM, bit1 all
// latency bounds, bit2 feasible, bit 8+i model i misses its bound).
constexpr unsigned kEntNoJ = 32u;   // feasible, but fast J proves it outside the top-k band

// 128-bit selection key: (order-preserving bits of an fp64 J, bitwise-not of
// the joint index), so that a larger key is better and equal J prefers the
// lower index; 0 is "no entry".
struct K128 {
    unsigned long long hi, lo;
};

// Kernel mode of the fast kernel.
enum FastMode { kModeSearch = 0, kModeCollect = 1, kModeList = 2 };

struct FastArgs {
    const float4 *image;
    int image_f4;
    FastLayout lay;
    uint64_t lo, n;             // range [lo, lo+n); list mode: n entries of idx_list
    const uint64_t *idx_list;   // list mode only
    uint32_t stride_digits[kMaxN]; // mixed-radix digits of (total waves * 32) mod |Lambda|
    int total_waves;
    int waves;                  // waves per workgroup (kSearchWaves or kSearchWavesWide)
    const float *sla;           // device [N]
    const float *omega;         // device [N]
    DevResult *res;
    unsigned long long *work;   // certification list: offset | (uncertain-model mask << 32)
    float *work_J;              // upper bound U >= canonical J of each certification entry
    uint32_t work_cap;
    uint32_t *collect;          // fallback candidate list
    uint32_t collect_cap;
    double theta;               // collect mode threshold on U
    unsigned long long *wg_lists; // [grid][KP] top-KP keys (U, lowest index) per workgroup
    unsigned long long *wg_counts; // [grid][2] VRAM-feasible and surely feasible counts per workgroup
    uint8_t *mask;              // dump (optional)
    float *pred;                // dump (optional)
    ObjArgs obj;
    int ep_bytes;               // LDS bytes after the workgroup lists for the small-range certification
    int lst_off;                // floats from the LDS start to the per-wave lists (0: over the fast weights)
    const float *canon;         // canonical fp32 image [N][wstride] (W1T[nin][H1], b1, ...)
    // Small ranges (search mode, completed by the finish kernel): no global
    // counter.  Certification entries go to a segment of seg_cap entries per
    // workgroup; after its scan each workgroup evaluates canonically its first
    // eval_top list entries and its segment, and writes its wg_k best
    // canonical keys (wg_top [grid][wg_k], sorted, zeros past the last) and
    // wg_rec[8 g] = {entries offered (may exceed seg_cap), start and end
    // wall-clock ticks, status bits << 32 | the order-preserving bits of the
    // upper bound U of list entry eval_top (0: none), segment entries found
    // feasible, -, -, -}.
    int small;
    uint32_t seg_cap;
    unsigned long long *seg;
    float *seg_J;
    unsigned long long *wg_rec;
    int eval_top, wg_k;
    K128 *wg_top;
    int64_t wstride;
    const float *features;      // [sumK][n_local]
    const int32_t *agg_cols;    // [A] (original slot order)
    int n_local, vram_slot;
};

// ---------------------------------------------------------------------------
// bf16 fast path.  Per model, one block staged into LDS (offsets in floats):
//   w2a [mb2][ks][lane][8 bf16]   A operand of layer 2: lane l, element j holds
//                                 W2[32 mb2 + l%32][32 (ks/2) + 16 (ks%2) + 8 (j/4) + 4 (l/32) + j%4]
//   w1a [mb][s][lane]             A operand of layer 1 (aggregate slot 2s + l/32)
//   b2  [H]
//   w3  [o][mb][q][half][4]       W3[o][32 mb + 8 q + 4 half + j]
//   cst [12]                      b3[0], b3[1], then per output (lat, thr):
//                                 k0 (fixed bound terms), |W3||b2|, max_u (|W3||W2|)_u,
//                                 max_v |W3[o][v]|
// Resident in LDS for the whole launch: g [sumK][half][4] aggregate slots of
// every option row (slot 2s + half at [half][s], original slot order) and the
// VRAM column gv [sumK].  In global memory: phat [sumK][PST], the fp32 chain
// of each option's local columns from b1.
// ---------------------------------------------------------------------------
struct Bf16Layout {
    int H, A, MB, KS, S1, PST;
    int off_w2a, off_w1a, off_b2, off_w3, off_cst;
    int model_floats;          // multiple of 256 (1 KB)
    int sumK, gv_floats;       // gv_floats: sumK rounded up to a multiple of 4
};

constexpr Bf16Layout bf16_layout(int H, int A, int sumK)
{
    Bf16Layout l{};
    l.H = H;
    l.A = A;
    l.MB = H / 32;
    l.KS = H / 16;
    l.S1 = A / 2;
    l.PST = H;
    l.off_w2a = 0;
    l.off_w1a = l.off_w2a + l.MB * l.KS * 64 * 4;
    l.off_b2 = l.off_w1a + l.MB * l.S1 * 64;
    l.off_w3 = l.off_b2 + H;
    l.off_cst = l.off_w3 + 2 * H;
    l.model_floats = (l.off_cst + 12 + 255) & ~255;   // whole 1 KB chunks (direct LDS loads)
    l.sumK = sumK;
    l.gv_floats = (sumK + 3) & ~3;
    return l;
}

struct Bf16Const {
    float g2, g3, gN;          // gamma_{2 KS}, gamma_{H/8+4}, gamma_N at fp32 unit roundoff
    int32_t act;               // output activation: 0 identity, 1 sigmoid
    float mag_thr[kMaxN];      // a-priori bound on |thr| of model i
};

struct Bf16Args {
    const float4 *models;      // [N][model_floats / 4]
    const float4 *g_image;     // [(sumK * 8 + gv_floats) / 4]
    const float *phat;         // [sumK][PST]
    Bf16Layout lay;
    uint64_t lo, n;
    const uint64_t *idx_list;  // list mode only
    const float *sla, *omega;
    DevResult *res;
    unsigned long long *work;
    float *work_J;
    uint32_t work_cap;
    uint32_t *collect;
    uint32_t collect_cap;
    double theta;
    unsigned long long *wg_lists;
    unsigned long long *wg_counts;
    uint8_t *mask;
    float *pred;
    ObjArgs obj;
};

// Canonical (fp64) evaluation of entries.
struct CanonArgs {
    int n_models, L, A, H1, H2, bf16, act;
    int32_t K[kMaxN];
    int32_t opt_off[kMaxN];
    const int32_t *agg_cols;    // device [A] (original order)
    int vram_slot;
    float vram_cap;
    const float *features;      // device [sumK][L]
    const float *weights;       // device [N][stride]
    int64_t wstride;
    const float *sla, *omega;   // device [N]
    uint64_t lo;                // entries hold offsets from lo (search) ...
    const uint64_t *idx64;      // ... or absolute indices (list mode) when non-null
    // search mode entry sources: fast candidates (keys) then the work list then the collect list
    const unsigned long long *cand_keys; int n_cand_keys;
    const unsigned long long *work; const float *work_J; uint32_t work_cap;
    const uint32_t *collect; uint32_t collect_cap;
    DevResult *res;             // counters, eJ, collect threshold
    int top_k;
    int collect_mode;
    int phase;                  // search mode: 0 fast candidates, 1 certification (+ collect) entries
    int64_t n_list;             // list mode entry count
    // outputs per entry
    double *ent_J;
    uint32_t *ent_flags;
    double *pred;               // list mode optional [n][N][2]
    uint8_t *mask;              // search dump: patch worklist entries
    ObjArgs obj;
};

// The rest of a small-range search after the fast kernel, in one workgroup:
// sum the workgroups' counts and records, select the exact top-k among the
// workgroups' best canonical keys (drawn from each workgroup's first eval_top
// list entries and its certification segment) and fill the result block.  The top-k is exact when
// its k-th canonical J exceeds every workgroup's first unevaluated upper
// bound; otherwise the status asks for the fallback (collect) pass.
struct FinishArgs {
    DevResult *res;
    DevResult *res_host;            // optional copy in pinned host memory (counts, status, top-k)
    unsigned long long seq;         // written to res_host->done_seq after everything else
    const float *omega;
    int top_k, n_wg;
    uint32_t seg_cap, work_cap;
    const unsigned long long *wg_counts;  // [n_wg][2]
    const unsigned long long *wg_rec;     // [n_wg][8]
    const K128 *wg_top;                   // [n_wg][top_k]
};

// Small ranges, fallback only: the workgroups' certification segments
// gathered into one list for the collect pass.
struct GatherArgs {
    int n_wg;
    uint32_t seg_cap;
    const unsigned long long *wg_rec, *seg;
    const float *seg_J;
    unsigned long long *work_out;
    float *work_J_out;
};

// One workgroup's share of the exact top-k selection over a long entry list.
struct SelPart {
    K128 keys[MF_MAX_TOPK];     // sorted, zeros past k
    unsigned long long feas;    // certified feasible work entries
    double maxd;                // largest U - J over the fast candidates
    uint32_t stat, pad;         // self-check bits
};

struct SelectArgs {
    SelPart *parts;             // [n_parts] when the selection runs in two levels
    int n_parts;                // <= 1: one workgroup
    int top_k, kp;
    const unsigned long long *cand_keys;   // [kp] fast candidates (0 = empty)
    const unsigned long long *work; const uint32_t *collect;
    uint32_t work_cap, collect_cap;
    const double *ent_J;
    const uint32_t *ent_flags;
    uint64_t lo;
    int collect_mode;           // 1: the collect pass ran; candidates = collect list
    DevResult *res;
};

// Fixed observed state (Section III-B): per option row, the canonical terms
// of the row's model under the fixed aggregate input.  FixedRow (16 bytes):
// q (thr for the linear objective, Q f under Eq. 3), the row's VRAM value and
// flags: kRowBad (the sign bit, so that an OR over a configuration's rows is
// tested by one signed compare) the latency bound or floor fails, kRowP /
// kRowPen subtract FixedPen's P / pen after J = fma(omega, q, J) (Eq. 3 only).
constexpr int kFixedWaves = 8;               // waves per workgroup of the fixed-state scan
constexpr int kFixedMaxWgsPerCu = 4;         // resident scan workgroups per CU at most (grid = CUs x that)
constexpr unsigned kRowBad = 0x80000000u, kRowP = 2u, kRowPen = 4u;
struct FixedRow {
    double q;
    float vram;
    uint32_t flags;
};
struct FixedPen {
    double P, pen;
};

// The scan splits the models into an outer prefix 0..n_outer-1 and the inner
// models n_outer..N-1 (inner space of `inner` configurations, at least 256
// unless the whole space is smaller).  Joint index = block * inner + u; a
// wave takes blocks_per_wave consecutive blocks, computes the outer prefix of
// the canonical chain once per block and the inner models per lane.
struct FixedArgs {
    int n_models, L, A, H1, H2, bf16, sumK, act;
    int32_t K[kMaxN];
    int32_t opt_off[kMaxN];
    uint32_t magic[kMaxN];
    int n_outer;
    uint32_t inner;
    int32_t in_K[kMaxN];             // K, first row and magic of inner model n_outer + t
    int32_t in_off[kMaxN];
    uint32_t in_magic[kMaxN];
    uint64_t block0, n_blocks, blocks_per_wave;
    uint64_t part_block_lo, part_block_hi;   // blocks holding the range ends mid-block (~0: none)
    int lc_shift;                    // >= 0: two inner models, the last with 2^lc_shift options
                                     // dividing 64 and a block of whole 128-configuration pairs
                                     // of tiles (its digit is lane-constant); -1: general decode
    const int32_t *row_model;        // device [sumK]
    const float *features;           // device [sumK][L]
    const float *weights;            // device canonical image [N][wstride]
    int64_t wstride;
    float state[kMaxN];              // observed aggregate, original slot order ([A])
    int vram_col;                    // feature column of the VRAM slot
    float vram_cap;
    const float *sla, *omega;        // device [N]
    uint64_t lo, n;                  // index range [lo, lo + n)
    int top_k;
    FixedRow *rows;                  // [sumK]
    FixedPen *pens;                  // [sumK]
    float2 *pred_rows;               // [sumK] canonical (lat, thr) rounded to fp32
    K128 *wg_lists;                  // [grid][top_k]
    unsigned long long *wg_counts;   // [grid][2] VRAM-feasible and feasible counts per workgroup
    DevResult *res;
    uint8_t *mask;                   // dump (optional)
    float *pred;                     // dump (optional)
    ObjArgs obj;
};

// Static (multi-step) search: one configuration held over T steps.  f
// carries the shape, the block split, the range and the outputs; per step t
// the table kernel fills rows_steps[t][sumK] (and pens_steps) from the
// step's observed state, bounds and previous deployment.
struct StaticArgs {
    FixedArgs f;
    int n_steps;
    const float *omega_steps;        // device [T][N]
    FixedRow *rows_steps;            // [T][sumK]
    FixedPen *pens_steps;            // [T][sumK]
    // list mode
    const uint64_t *idx;
    int64_t n_list;
    double *out_J;                   // [n][T] or null
    double *out_S;                   // [n] or null
    uint32_t *out_flags;             // [n][T] or null
};

// GA problem constants (kernel-argument block).
struct GAConst {
    int N, L, A, H1, H2, bf16, act;
    int32_t K[kMaxN];
    int32_t opt_off[kMaxN];
    int vram_col;               // option column of the VRAM aggregate slot
    int vram_slot;
    float vram_cap;
    uint64_t space;
    const float *features;      // [sumK][L]
    const int32_t *agg_cols;    // [A]
    const double *w64;          // [N][stride] packed weights (W1 b1 W2 b2 W3 b3) as fp64
    const double *pre;          // [sumK][H1] canonical layer-1 chain over each option's local features
    int sumK;
    const float *canon;         // [N][stride] canonical image (W1^T b1 W2^T b2 W3 b3)
    int64_t wstride;
    int fixed;                  // the surrogates see state[] instead of the candidate's aggregate
    float state[kMaxN];
    ObjArgs obj;
    // the run's memo of canonical predictions per joint index (null: none):
    // memo[idx][N][2] (lat, thr) and tag[idx] = 2 g' + vram_ok, g' - 1 the
    // generation that wrote it (0: not yet evaluated in this run)
    double *memo;
    uint32_t *memo_tag;
    unsigned long long *n_forwards;   // individuals whose fitness ran the surrogates (with the memo)
};

// Raise a kernel's dynamic-LDS limit to at least `bytes` on the current
// device; the attribute stays set, so it is applied once per kernel, device
// and size increase (a call that changes nothing costs a table lookup).
hipError_t ensure_dyn_lds(const void *fn, size_t bytes);

// Per-model power-of-two exponents (kernel argument).
struct Pow2Scales {
    int32_t e[kMaxN];
};

// launchers (return hipError_t of the launch)
hipError_t launch_precompute_p(const float *features, const float *weights, const float *centre,
                               int n_rows, int L, int A, int H, int64_t wstride,
                               const int32_t *row_model, float *image_p, int pst, const Pow2Scales &sc,
                               hipStream_t s);
hipError_t launch_fast_impl(const FastArgs &a, const FastConst &fc, int grid, int kp, int mode, hipStream_t s);
int fast_waves_for(int n_models, const FastLayout &lay, int kp, int act);
int fast_kernel_supported(int n_models, int A, int H, int kp);
int bf16_kernel_supported(int n_models, int A, int H);
size_t bf16_lds_bytes(const Bf16Layout &lay, int kp);
hipError_t launch_bf16_impl(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                            hipStream_t s);
hipError_t launch_bf16_h64(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                           hipStream_t s);
hipError_t launch_bf16_h128(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                            hipStream_t s);
hipError_t launch_bf16_h256(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                            hipStream_t s);
hipError_t launch_precompute_phat(const float *features, const float *canon_w, int n_rows, int L, int A, int H,
                                  int64_t wstride, const int32_t *row_model, float *phat, int pst, hipStream_t s);
hipError_t launch_merge_lists(const unsigned long long *lists, int n_lists, int kp, unsigned long long *out,
                              const unsigned long long *wg_counts, unsigned long long *counts_out, hipStream_t s);
hipError_t launch_canonical(const CanonArgs &a, int n_entries_max, bool search_mode, hipStream_t s);
hipError_t launch_kth_candidate(const unsigned long long *cand_keys, const double *ent_J, const uint32_t *ent_flags,
                                int kp, int k, DevResult *res, hipStream_t s);
hipError_t launch_select(const SelectArgs &a, hipStream_t s);
hipError_t launch_gather_small(const GatherArgs &g, hipStream_t s);
hipError_t launch_finish_small(const FinishArgs &f, const FastConst &fc, hipStream_t s);
size_t fast_small_epilogue_bytes(int n_models);
constexpr uint64_t kSmallRange = 1ull << 20;   // fp32 ranges up to this size finish in one workgroup
size_t fixed_lds_bytes(int sumK, bool eq3);
size_t static_lds_bytes(int n_steps, int sumK, int n_models, bool eq3);
hipError_t launch_fixed_table(const FixedArgs &a, hipStream_t s);
hipError_t launch_static(const StaticArgs &a, int grid, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_static_eval(const StaticArgs &a, hipStream_t s);
int static_wgs_per_cu(const StaticArgs &a);
int fixed_wgs_per_cu(const FixedArgs &a);
hipError_t launch_fixed(const FixedArgs &a, int grid, bool table, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
constexpr int64_t kGaWideMax = 8192;   // populations (S x P) up to this size take the wide fitness kernel
constexpr int kSelParts = 128;            // workgroups of the two-level selection over long entry lists
constexpr uint64_t kSelSingleMax = 1ull << 20;   // ranges up to this size select in one workgroup
constexpr int kCanonMaxGrid = 8192;        // certification workgroups (one wave each): 8 per SIMD
constexpr int kCanonWaves = 8;             // certification of few entries: waves (models) per workgroup, at most
constexpr int kCanonFewEntries = 1024;     // index lists up to this length count as few
constexpr int kGaWideWaves = 8;             // ... with up to this many waves (models) per workgroup
constexpr size_t kGaStageBytes = 64 * 1024;   // ... copying the weights to LDS when they fit in this
constexpr int kGaFitThreads = 512;             // large populations: lanes (individuals) per fitness workgroup
constexpr int kGaMemoThreads = 256;            // ... after the first generation: individuals per memo workgroup
constexpr uint64_t kGaMemoMaxBytes = 256ull << 20;   // the run's memo of predictions, at most this large
constexpr size_t kGaPreLdsBytes = 96 * 1024;   // ... continuing the local-feature chains staged in this much LDS
constexpr int64_t kGaWideStagedWgs = 512;    // ... and then running this many workgroups at most
int ga_fitness_supported(int nin, int h1, int h2);
hipError_t launch_ga_feasible(const GAConst &c, uint32_t *blk_count, uint64_t *blk_off, unsigned long long *n_fl,
                              uint32_t *fl, hipStream_t st);
hipError_t launch_ga_init(uint64_t seed, int S, int P, const uint32_t *fl, const unsigned long long *n_fl,
                          uint64_t *pop, double *best_J, uint64_t *best_idx, hipStream_t st);
hipError_t launch_ga_fitness(const GAConst &c, int S, int P, const uint64_t *pop, const float *sla,
                             const float *omega, double *fit, hipStream_t st, uint32_t memo_gen = 0);
// Whether generation 0's fitness takes the one-lane kernel that continues the
// local chains (the kernel that fills the run's memo for the later ones).
bool ga_memo_supported(const GAConst &c, int S, int P);
hipError_t launch_ga_memo_clear(uint32_t *tag, uint64_t n, unsigned long long *n_forwards,
                                unsigned long long first, hipStream_t st);
hipError_t launch_ga_ops(const GAConst &c, uint64_t seed, int S, int P, int gen, int gens, int tk, float p_cx,
                         float p_swap, float p_mut, const uint32_t *fl, const unsigned long long *n_fl,
                         const uint64_t *pop, const double *fit, uint64_t *next, double *best_J,
                         uint64_t *best_idx, uint64_t *final_pop, hipStream_t st);

}  // namespace mfi
