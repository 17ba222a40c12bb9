// Exhaustive search with the observed state held fixed (Section III-B: the
// aggregate GPU state the surrogates see is observed by the runtime monitor
// and held fixed during the search, the paper's own semantics).
//
// With the aggregate input fixed, model i's prediction depends on its own
// option only, so the surrogates run once per option row (sum_i K_i canonical
// forwards, `fixed_table_kernel`) and the joint search sums table entries
// under the VRAM cap (`fixed_scan_kernel`).  Every value the scan combines is
// canonical and it combines them in the canonical order (model 0 first), so
// the search is exact without any certification.  The scan shares the chain's
// prefix: per block of configurations that agree on the outer models, the
// outer part of the chain (J, VRAM sum, service flag) is computed once, and
// each lane adds the inner models of its own configuration (two LDS rows per
// configuration at the usual shapes).  Top-k are selected on 128-bit (J,
// index) keys, per wave, per workgroup, then over the grid.
#include "mf_canon.h"

namespace mfi {

// ---------------------------------------------------------------------------
// Table: one 64-thread workgroup per option row.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ void __launch_bounds__(64) fixed_table_kernel(const FixedArgs a)
{
    __shared__ double h1s[kCanonMaxH];
    __shared__ double h2s[kCanonMaxH];
    __shared__ double zs[kCanonMaxIn];
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    const int lane = threadIdx.x;
#pragma unroll
    for (int i = 0; i < kMaxN; i++)   // compile-time index into the argument block
        if (lane == i) {
            s_tau[i] = a.obj.tau[i];
            s_prev[i] = a.obj.prev[i];
        }
    const int nin = a.L + a.A;
    for (int r = blockIdx.x; r < a.sumK; r += gridDim.x) {
        const int i = a.row_model[r];
        const float *x = a.features + (int64_t)r * a.L;
        __syncthreads();
        for (int k = lane; k < nin; k += 64) zs[k] = k < a.L ? (double)x[k] : (double)a.state[k - a.L];
        __syncthreads();
        double lat, thr;
        canon_model<BF16>(a.weights + (int64_t)i * a.wstride, nin, a.H1, a.H2, zs, h1s, h2s, lane, lat, thr, a.act);
        if (lane == 0) {
            FixedRow row;
            FixedPen pp = {0.0, 0.0};
            uint32_t fl = lat <= (double)a.sla[i] ? 0u : kRowBad;
            row.q = thr;
            if (a.obj.kind != 0) {
                bool do_P, do_pen;
                if (!canon_eq3(a.obj, r, thr, s_tau[i], s_prev[i], row.q, pp.P, do_P, pp.pen, do_pen)) fl = kRowBad;
                fl |= (do_P ? kRowP : 0u) | (do_pen ? kRowPen : 0u);
            }
            row.vram = x[a.vram_col];
            row.flags = fl;
            a.rows[r] = row;
            a.pens[r] = pp;
            a.pred_rows[r] = make_float2((float)lat, (float)thr);
        }
    }
}

// One model's step of the canonical chain: VRAM sum, service flags (ORed;
// kRowBad is the sign bit), J.
template <bool EQ3>
__device__ __forceinline__ void chain_step(const FixedRow &r, const FixedPen *pens, uint32_t row, double om,
                                           double &J, float &v, uint32_t &fl)
{
    v += r.vram;
    fl |= r.flags;
    J = fma(om, r.q, J);
    if (EQ3) {
        const FixedPen pp = pens[row];
        if (r.flags & kRowP) J = J - pp.P;
        if (r.flags & kRowPen) J = J - pp.pen;
    }
}

template <bool EQ3>
__device__ __forceinline__ void chain_row(const FixedRow *rows, const FixedPen *pens, uint32_t row, double om,
                                          double &J, float &v, uint32_t &fl)
{
    chain_step<EQ3>(rows[row], pens, row, om, J, v, fl);
}

template <bool B>
struct BoolC {
    static constexpr bool value = B;
};

// Wave ballot of a lane predicate, straight into a scalar mask.
__device__ __forceinline__ unsigned long long ballot64(bool b) { return __builtin_amdgcn_ballot_w64(b); }

// Offer the lanes of candidate mask cm to the wave's top-k list, and refresh
// thrJ, the J of the list's k-th key (-inf while the list is not full): a key
// can only enter if its J is at least thrJ, so that test screens lanes before
// any 128-bit key is formed.
__device__ __forceinline__ void offer_mask(K128 &slot, K128 &thr, double &thrJ, unsigned long long cm, double J,
                                        uint64_t idx, int lane, int k)
{
    const bool mine = ((cm >> lane) & 1ull) != 0ull;
    list128_offer(slot, key_if(mine, K128{ord_f64(J), ~idx}), lane, k, thr);
    thrJ = nz128(thr) ? unord_f64(thr.hi) : -INFINITY;
}

// One 64-configuration tile of a block: inner rows, and the chain from the
// block's outer prefix.
template <int NI>
struct Tile {
    double J;
    float v;
    uint32_t fl;
    uint32_t rr[NI];
};

template <int NI, bool EQ3, bool LC, bool EXACT>
__device__ __forceinline__ Tile<NI> eval_tile(const FixedArgs &a, const FixedRow *rows, const FixedPen *pens,
                                              uint32_t u, uint32_t t0, int ni, uint32_t M, const double *omi,
                                              double Jp, float vp, uint32_t flp, const FixedRow &rb,
                                              uint32_t row_a0, uint32_t row_b)
{
    Tile<NI> o;
    o.J = Jp;
    o.v = vp;
    o.fl = flp;
    if (LC) {
        o.rr[0] = row_a0 + (t0 >> a.lc_shift);
        o.rr[1] = row_b;
        chain_row<EQ3>(rows, pens, o.rr[0], omi[0], o.J, o.v, o.fl);
        chain_step<EQ3>(rb, pens, row_b, omi[1], o.J, o.v, o.fl);
    } else if (EXACT) {
        // exactly NI inner models, each but the first with at least two
        // options, and u < M: the digits with no guards
        uint32_t uu = u;
#pragma unroll
        for (int t = NI - 1; t > 0; t--) {
            const uint32_t q = __umulhi(uu, a.in_magic[t]);
            o.rr[t] = (uint32_t)a.in_off[t] + (uu - q * (uint32_t)a.in_K[t]);
            uu = q;
        }
        o.rr[0] = (uint32_t)a.in_off[0] + uu;
#pragma unroll
        for (int t = 0; t < NI; t++) chain_row<EQ3>(rows, pens, o.rr[t], omi[t], o.J, o.v, o.fl);
    } else {
        uint32_t uu = u < M ? u : 0u;
#pragma unroll
        for (int t = NI - 1; t >= 0; t--) {
            o.rr[t] = 0;
            if (t < ni) {
                // the first inner digit is what remains (uu < K there)
                const uint32_t q = (t > 0 && a.in_magic[t]) ? __umulhi(uu, a.in_magic[t]) : (t > 0 ? uu : 0u);
                o.rr[t] = (uint32_t)a.in_off[t] + (uu - q * (uint32_t)a.in_K[t]);
                uu = q;
            }
        }
#pragma unroll
        for (int t = 0; t < NI; t++)
            if (t < ni) chain_row<EQ3>(rows, pens, o.rr[t], omi[t], o.J, o.v, o.fl);
    }
    return o;
}

template <int NI>
__device__ __forceinline__ void dump_tile(const FixedArgs &a, const Tile<NI> &x, bool valid, float cap, uint64_t idx,
                                          const int32_t *s_off, const uint32_t *od, uint32_t dl, int nout, int ni)
{
    if (!valid) return;
    const bool vram_ok = x.v <= cap, ok = (int32_t)x.fl >= 0;
    const int N = a.n_models;
    const uint64_t off = idx - a.lo;
    a.mask[off] = (uint8_t)((vram_ok ? 1u : 0u) | (ok ? 2u : 0u) | (vram_ok && ok ? 4u : 0u));
    float *pd = a.pred + off * (uint64_t)N * 2u;
#pragma unroll 1
    for (int j = 0; j < nout; j++) {
        const float2 pr = a.pred_rows[s_off[j] + (j == nout - 1 ? dl : od[j])];
        pd[2 * j] = pr.x;
        pd[2 * j + 1] = pr.y;
    }
#pragma unroll
    for (int t = 0; t < NI; t++)
        if (t < ni) {
            const float2 pr = a.pred_rows[x.rr[t]];
            pd[2 * (nout + t)] = pr.x;
            pd[2 * (nout + t) + 1] = pr.y;
        }
}

// ---------------------------------------------------------------------------
// Scan: per wave a run of consecutive blocks; per block the outer prefix once
// (wave-uniform, from LDS), then the inner configurations two 64-tiles at a
// time, one configuration per lane and tile.  Decisions become wave masks at
// once (counts by popcount, candidates by mask).  NI: compile-time bound on
// the number of inner models.  LC (NI = 2 only): the last model's digit is
// lane-constant (its row lives in registers) and the other inner digit is a
// shift of the tile offset.
// ---------------------------------------------------------------------------
template <int NI, bool EQ3, bool LC, bool EXACT = false>
__global__ void __launch_bounds__(kFixedWaves * 64) fixed_scan_kernel(const FixedArgs a)
{
    extern __shared__ float4 smem4[];
    __shared__ double s_om[kMaxN];
    __shared__ int32_t s_off[kMaxN], s_K[kMaxN];
    __shared__ uint32_t s_od[kFixedWaves][kMaxN];   // outer digits of each wave's current block
    FixedRow *rows = reinterpret_cast<FixedRow *>(smem4);
    FixedPen *pens = reinterpret_cast<FixedPen *>(rows + a.sumK);
    K128 *lst = reinterpret_cast<K128 *>(pens + (EQ3 ? a.sumK : 0));
    const int N = a.n_models, nout = a.n_outer, ni = N - nout, k = a.top_k;
#pragma unroll 1
    for (int t = threadIdx.x; t < a.sumK; t += blockDim.x) {   // not unrolled: keeps registers for the scan
        rows[t] = a.rows[t];
        if (EQ3) pens[t] = a.pens[t];
    }
    if (threadIdx.x < (unsigned)N) s_om[threadIdx.x] = (double)a.omega[threadIdx.x];
#pragma unroll
    for (int j = 0; j < kMaxN; j++)   // compile-time index into the argument block
        if (threadIdx.x == (unsigned)j) {
            s_off[j] = a.opt_off[j];
            s_K[j] = a.K[j];
        }
    double omi[NI];
#pragma unroll
    for (int t = 0; t < NI; t++) omi[t] = t < ni ? (double)a.omega[nout + t] : 0.0;

    const int lane = threadIdx.x & 63;
    // the wave index is wave-uniform: say so, so that everything derived from
    // it (blocks, digits, masks) stays in scalar registers
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint64_t gw = (uint64_t)blockIdx.x * kFixedWaves + wv;
    const uint64_t b_first = gw * a.blocks_per_wave;
    const uint64_t b_begin = a.block0 + (b_first < a.n_blocks ? b_first : a.n_blocks);
    const uint64_t b_end = a.block0 + (b_first + a.blocks_per_wave < a.n_blocks ? b_first + a.blocks_per_wave
                                                                                : a.n_blocks);
    const uint64_t idx_lo = a.lo, idx_hi = a.lo + a.n;
    const uint32_t M = a.inner;
    const float cap = a.vram_cap;
    uint32_t *od = s_od[wv];
    if (lane == 0) {
        uint64_t x = b_begin;
        for (int j = nout - 1; j >= 0; j--) {
            od[j] = (uint32_t)(x % (uint64_t)a.K[j]);
            x /= (uint64_t)a.K[j];
        }
    }
    __syncthreads();

    // LC: the last model's row of this lane, and the first row of the other
    // inner model this lane starts at
    FixedRow rb = {0.0, 0.f, 0u};
    uint32_t row_b = 0, row_a0 = 0;
    if (LC) {
        const int sh = a.lc_shift;
        row_b = (uint32_t)a.in_off[1] + ((uint32_t)lane & ((1u << sh) - 1u));
        rb = rows[row_b];
        row_a0 = (uint32_t)a.in_off[0] + ((uint32_t)lane >> sh);
    }

    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    double thrJ = -INFINITY;
    unsigned long long c_vram = 0, c_feas = 0;   // wave-uniform
    double Jc = 0.0;      // chain over outer models 0..nout-2
    float vc = 0.f;
    uint32_t flc = 0u;
    bool need_full = true;
    // the last outer model: its digit dl lives in a scalar register (the
    // odometer in LDS is touched only when dl wraps)
    uint32_t dl = nout > 0 ? od[nout - 1] : 0u;
    const uint32_t K_last = nout > 0 ? (uint32_t)a.K[nout - 1] : 1u;
    const uint32_t off_last = nout > 0 ? (uint32_t)a.opt_off[nout - 1] : 0u;
    const double om_last = nout > 0 ? (double)a.omega[nout - 1] : 0.0;

    for (uint64_t b = b_begin; b < b_end; b++) {
        if (need_full) {
            Jc = 0.0;
            vc = 0.f;
            flc = 0u;
#pragma unroll 1
            for (int j = 0; j < nout - 1; j++) chain_row<EQ3>(rows, pens, (uint32_t)s_off[j] + od[j], s_om[j], Jc, vc, flc);
            need_full = false;
        }
        double Jp = Jc;
        float vp = vc;
        uint32_t flp = flc;
        if (nout > 0) chain_row<EQ3>(rows, pens, off_last + dl, om_last, Jp, vp, flp);

        const uint64_t base = b * (uint64_t)M;
        // every lane of every tile valid unless the block holds a range end
        // (or a partial last tile)
        const bool whole = b != a.part_block_lo && b != a.part_block_hi && (M & 63u) == 0u;
        const uint32_t u_lo = whole ? 0u : (base < idx_lo ? (uint32_t)(idx_lo - base) : 0u);
        const uint32_t u_hi = whole ? M : (idx_hi - base < (uint64_t)M ? (uint32_t)(idx_hi - base) : M);
        const uint32_t u_span = u_hi - u_lo;

        // the block's tiles, two at a time; WHOLE and DUMP are compile-time
        auto tiles = [&](auto whole_c, auto dump_c) {
            constexpr bool WHOLE = decltype(whole_c)::value, DUMP = decltype(dump_c)::value;
            uint32_t cv = 0, cf = 0;
#pragma unroll 1
            for (uint32_t t0 = 0; t0 < M; t0 += 128) {
                // second tile: past the block end it repeats the first with no
                // valid lane (LC blocks are whole 128-tiles)
                const bool two = LC || t0 + 64 < M;
                const uint32_t t1 = two ? t0 + 64 : t0;
                const uint32_t ux = t0 + (uint32_t)lane, uy = t1 + (uint32_t)lane;
                const Tile<NI> x = eval_tile<NI, EQ3, LC, EXACT>(a, rows, pens, ux, t0, ni, M, omi, Jp, vp, flp, rb, row_a0, row_b);
                const Tile<NI> y = eval_tile<NI, EQ3, LC, EXACT>(a, rows, pens, uy, t1, ni, M, omi, Jp, vp, flp, rb, row_a0, row_b);
                unsigned long long mvx = ~0ull, mvy = two ? ~0ull : 0ull;   // valid lanes
                if (!WHOLE) {
                    mvx = ballot64(ux - u_lo < u_span);
                    mvy = two ? ballot64(uy - u_lo < u_span) : 0ull;
                }
                const unsigned long long vx = mvx & ballot64(x.v <= cap), vy = mvy & ballot64(y.v <= cap);
                const unsigned long long fx = vx & ballot64((int32_t)x.fl >= 0), fy = vy & ballot64((int32_t)y.fl >= 0);
                const unsigned long long cx = fx & ballot64(x.J >= thrJ), cy = fy & ballot64(y.J >= thrJ);
                cv += (uint32_t)(__popcll(vx) + __popcll(vy));
                cf += (uint32_t)(__popcll(fx) + __popcll(fy));
                if (cx) offer_mask(slot, thr, thrJ, cx, x.J, base + ux, lane, k);
                if (cy) offer_mask(slot, thr, thrJ, cy, y.J, base + uy, lane, k);
                if (DUMP) {
                    dump_tile<NI>(a, x, ((mvx >> lane) & 1ull) != 0ull, cap, base + ux, s_off, od, dl, nout, ni);
                    dump_tile<NI>(a, y, ((mvy >> lane) & 1ull) != 0ull, cap, base + uy, s_off, od, dl, nout, ni);
                }
            }
            c_vram += cv;
            c_feas += cf;
        };
        if (a.mask) {
            if (whole) tiles(BoolC<true>{}, BoolC<true>{});
            else tiles(BoolC<false>{}, BoolC<true>{});
        } else {
            if (whole) tiles(BoolC<true>{}, BoolC<false>{});
            else tiles(BoolC<false>{}, BoolC<false>{});
        }

        // next block: the last outer digit, and on its wrap the odometer of
        // the others (lane 0 writes the wave's digits; the wave reads them
        // back after the write), which invalidates the cached prefix
        if (nout > 0 && ++dl == K_last) {
            dl = 0u;
            bool carry = true;
            for (int j = nout - 2; j >= 0 && carry; j--) {
                uint32_t d = od[j] + 1u;
                carry = d == (uint32_t)s_K[j];
                if (carry) d = 0u;
                __builtin_amdgcn_wave_barrier();
                if (lane == 0) od[j] = d;
                __builtin_amdgcn_wave_barrier();
            }
            need_full = true;
        }
    }

    // counts and list per workgroup (the merge kernel sums and merges them)
    __shared__ unsigned long long s_cnt[2 * kFixedWaves];
    if (lane == 0) {
        s_cnt[wv] = c_vram;
        s_cnt[kFixedWaves + wv] = c_feas;
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
#pragma unroll 1
        for (int w = 1; w < kFixedWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        if (lane < k) a.wg_lists[(uint64_t)blockIdx.x * k + lane] = slot;
        if (lane < 2) {
            unsigned long long t = 0;
            for (int w = 0; w < kFixedWaves; w++) t += s_cnt[lane * kFixedWaves + w];
            a.wg_counts[2 * (uint64_t)blockIdx.x + lane] = t;
        }
    }
}

// ---------------------------------------------------------------------------
// Scan with a periodic last digit: two inner models a (first) and b (last),
// K_b options for b.  Over the inner configurations u = 64 t + lane of a
// block, b = u mod K_b depends on the lane and on t mod P only, with
// P = K_b / gcd(64, K_b), and a = G (t div P) + A_p(lane), G = 64 P / K_b.
// Each lane keeps its P rows of model b in registers and its P first rows of
// model a as LDS addresses; a tile is then one row read, the chain steps of
// a and b in model order, and three compares.  Taken when the inner block is
// a whole number of P-tile groups, every block of the range is whole and no
// dump is asked for.  Under Eq. 3 the penalties are staged with zeros where a
// row's flags do not apply them (subtracting +0 changes no value), so the
// chain needs no test.  NG > 0: the block is exactly NG groups, unrolled
// (row offsets then differ by constants); NG = 0: a loop over the groups.
// ---------------------------------------------------------------------------
template <int P, bool EQ3, int NG = 0>
__global__ void __launch_bounds__(kFixedWaves * 64) fixed_periodic_kernel(const FixedArgs a)
{
    extern __shared__ float4 smem4[];
    __shared__ double s_om[kMaxN];
    __shared__ int32_t s_off[kMaxN], s_K[kMaxN];
    __shared__ uint32_t s_od[kFixedWaves][kMaxN];
    FixedRow *rows = reinterpret_cast<FixedRow *>(smem4);
    FixedPen *pens = reinterpret_cast<FixedPen *>(rows + a.sumK);   // Eq. 3: zero where not applied
    K128 *lst = reinterpret_cast<K128 *>(pens + (EQ3 ? a.sumK : 0));
    const int N = a.n_models, nout = a.n_outer, k = a.top_k;
#pragma unroll 1
    for (int t = threadIdx.x; t < a.sumK; t += blockDim.x) {
        const FixedRow r = a.rows[t];
        rows[t] = r;
        if (EQ3) {
            const FixedPen pp = a.pens[t];
            pens[t] = FixedPen{(r.flags & kRowP) ? pp.P : 0.0, (r.flags & kRowPen) ? pp.pen : 0.0};
        }
    }
    if (threadIdx.x < (unsigned)N) s_om[threadIdx.x] = (double)a.omega[threadIdx.x];
#pragma unroll
    for (int j = 0; j < kMaxN; j++)   // compile-time index into the argument block
        if (threadIdx.x == (unsigned)j) {
            s_off[j] = a.opt_off[j];
            s_K[j] = a.K[j];
        }
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint64_t gw = (uint64_t)blockIdx.x * kFixedWaves + wv;
    const uint64_t b_first = gw * a.blocks_per_wave;
    const uint64_t b_begin = a.block0 + (b_first < a.n_blocks ? b_first : a.n_blocks);
    const uint64_t b_end = a.block0 + (b_first + a.blocks_per_wave < a.n_blocks ? b_first + a.blocks_per_wave
                                                                                : a.n_blocks);
    const uint32_t M = a.inner, Kb = (uint32_t)a.in_K[1];
    const uint32_t n_grp = M / (64u * P);              // P-tile groups per block
    const uint32_t G = 64u * P / Kb;                   // rows of model a per group
    const float cap = a.vram_cap;
    uint32_t *od = s_od[wv];
    if (lane == 0) {
        uint64_t x = b_begin;
        for (int j = nout - 1; j >= 0; j--) {
            od[j] = (uint32_t)(x % (uint64_t)a.K[j]);
            x /= (uint64_t)a.K[j];
        }
    }
    __syncthreads();

    // this lane's rows: model b for each phase p (registers), model a's first
    // row for each phase (an LDS index, advanced by G per group)
    const double oma = (double)a.omega[nout], omb = (double)a.omega[nout + 1];
    double bq[P], bP[P], bpen[P];
    float bv[P];
    uint32_t bf[P], ra0[P];
#pragma unroll
    for (int p = 0; p < P; p++) {
        const uint32_t u = 64u * p + (uint32_t)lane;
        const uint32_t rb = (uint32_t)a.in_off[1] + u % Kb;
        const FixedRow r = rows[rb];
        bq[p] = r.q;
        bv[p] = r.vram;
        bf[p] = r.flags;
        bP[p] = EQ3 ? pens[rb].P : 0.0;
        bpen[p] = EQ3 ? pens[rb].pen : 0.0;
        ra0[p] = (uint32_t)a.in_off[0] + u / Kb;
    }
    // the rows of a and of b with the largest omega q (the largest q for
    // omega >= 0, the smallest otherwise) and, under Eq. 3, the smallest
    // staged P and pen of each.  RN and fma are monotone, J falls as P or pen
    // grows, and the chain below applies them in the kernel's own order, so
    // it bounds the J of every configuration of a block from above, bit for
    // bit (a NaN extreme gives a NaN bound, which prunes nothing)
    double qa_star = 0.0, qb_star = 0.0, Pa_min = 0.0, pena_min = 0.0, Pb_min = 0.0, penb_min = 0.0;
    for (int t = 0; t < 2; t++) {
        const int K = a.in_K[t], off = a.in_off[t];
        const bool up = (t == 0 ? oma : omb) >= 0.0;
        double best = rows[off].q;
        double Pm = EQ3 ? pens[off].P : 0.0, pm = EQ3 ? pens[off].pen : 0.0;
        for (int r = 1; r < K; r++) {
            const double q = rows[off + r].q;
            if (up ? q > best : q < best) best = q;
            if (EQ3) {
                const FixedPen pp = pens[off + r];
                if (pp.P < Pm) Pm = pp.P;
                if (pp.pen < pm) pm = pp.pen;
            }
        }
        if (t == 0) {
            qa_star = best;
            Pa_min = Pm;
            pena_min = pm;
        } else {
            qb_star = best;
            Pb_min = Pm;
            penb_min = pm;
        }
    }
    uint32_t aoff[P];   // byte offsets of this lane's first rows of model a (rows and penalties alike)
#pragma unroll
    for (int p = 0; p < P; p++) aoff[p] = ra0[p] * (uint32_t)sizeof(FixedRow);
    static_assert(sizeof(FixedRow) == sizeof(FixedPen), "one offset serves both tables");

    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    double thrJ = -INFINITY;
    unsigned long long c_vram = 0, c_feas = 0;   // wave-uniform
    double Jc = 0.0;   // chain over outer models 0..nout-2
    float vc = 0.f;
    uint32_t flc = 0u;
    bool need_full = true;
    uint32_t dl = nout > 0 ? od[nout - 1] : 0u;
    const uint32_t K_last = nout > 0 ? (uint32_t)a.K[nout - 1] : 1u;
    const uint32_t off_last = nout > 0 ? (uint32_t)a.opt_off[nout - 1] : 0u;
    const double om_last = nout > 0 ? (double)a.omega[nout - 1] : 0.0;

    // counts in 32 bits over the whole run (the host keeps a run below 2^32
    // configurations); the block's first joint index advances by M
    const uint32_t n_blk = (uint32_t)(b_end - b_begin);
    uint32_t cv = 0, cf = 0;
    uint64_t base = b_begin * (uint64_t)M;
#pragma unroll 1
    for (uint32_t bi = 0; bi < n_blk; bi++, base += M) {
        if (need_full) {
            Jc = 0.0;
            vc = 0.f;
            flc = 0u;
#pragma unroll 1
            for (int j = 0; j < nout - 1; j++)
                chain_row<EQ3>(rows, pens, (uint32_t)s_off[j] + od[j], s_om[j], Jc, vc, flc);
            need_full = false;
        }
        double Jp = Jc;
        float vp = vc;
        uint32_t flp = flc;
        if (nout > 0) chain_row<EQ3>(rows, pens, off_last + dl, om_last, Jp, vp, flp);
        // model a's rows of group g: each lane's first rows (its byte
        // offsets) plus one uniform offset per group
        const char *grow = reinterpret_cast<const char *>(rows);
        const char *gpen = reinterpret_cast<const char *>(pens);
        uint64_t ibase = base;   // joint index of the group's first configuration
        // one tile: phase p of a group whose model-a rows start at grow
        // no configuration of the block can enter the wave's list when its
        // prefix fails a bound or its largest J is under the k-th J: then
        // only the counts are formed
        double Jub = fma(oma, qa_star, Jp);
        if (EQ3) Jub = (Jub - Pa_min) - pena_min;
        Jub = fma(omb, qb_star, Jub);
        if (EQ3) Jub = (Jub - Pb_min) - penb_min;
        const bool counts_only = (int32_t)flp < 0 || Jub < thrJ;
        auto tile = [&](const char *gr, const char *gp, uint64_t ib, int p, auto co) {
            constexpr bool CO = decltype(co)::value;
            const FixedRow x = *reinterpret_cast<const FixedRow *>(gr + aoff[p]);
            const float v = (vp + x.vram) + bv[p];
            const uint32_t fl = flp | x.flags | bf[p];
            if constexpr (CO) {
                const unsigned long long mv = ballot64(v <= cap);
                cv += (uint32_t)__popcll(mv);
                cf += (uint32_t)__popcll(mv & ballot64((int32_t)fl >= 0));
                return;
            }
            double J = fma(oma, x.q, Jp);
            if (EQ3) {
                const FixedPen pa = *reinterpret_cast<const FixedPen *>(gp + aoff[p]);
                J = (J - pa.P) - pa.pen;
            }
            J = fma(omb, bq[p], J);
            if (EQ3) J = (J - bP[p]) - bpen[p];
            const unsigned long long mv = ballot64(v <= cap);
            const unsigned long long mf = mv & ballot64((int32_t)fl >= 0);
            const unsigned long long mc = mf & ballot64(J >= thrJ);
            cv += (uint32_t)__popcll(mv);
            cf += (uint32_t)__popcll(mf);
            if (mc) offer_mask(slot, thr, thrJ, mc, J, ib + (uint64_t)(p * 64 + lane), lane, k);
        };
        auto groups = [&](auto co) {
            if constexpr (NG > 0) {
#pragma unroll
                for (int g = 0; g < NG; g++)
#pragma unroll
                    for (int p = 0; p < P; p++)
                        tile(grow + g * G * sizeof(FixedRow), gpen + g * G * sizeof(FixedPen),
                             base + (uint64_t)g * 64u * P, p, co);
            } else {
#pragma unroll 1
                for (uint32_t g = 0; g < n_grp; g++) {
#pragma unroll
                    for (int p = 0; p < P; p++) tile(grow, gpen, ibase, p, co);
                    grow += G * sizeof(FixedRow);
                    gpen += G * sizeof(FixedPen);
                    ibase += 64u * P;
                }
            }
        };
        if (counts_only) groups(BoolC<true>{});
        else groups(BoolC<false>{});
        // next block: the last outer digit, and on its wrap the odometer of
        // the others (lane 0 writes the wave's digits)
        if (nout > 0 && ++dl == K_last) {
            dl = 0u;
            bool carry = true;
            for (int j = nout - 2; j >= 0 && carry; j--) {
                uint32_t d = od[j] + 1u;
                carry = d == (uint32_t)s_K[j];
                if (carry) d = 0u;
                __builtin_amdgcn_wave_barrier();
                if (lane == 0) od[j] = d;
                __builtin_amdgcn_wave_barrier();
            }
            need_full = true;
        }
    }

    c_vram = cv;
    c_feas = cf;
    // counts and list per workgroup (the merge kernel sums and merges them)
    __shared__ unsigned long long s_cnt[2 * kFixedWaves];
    if (lane == 0) {
        s_cnt[wv] = c_vram;
        s_cnt[kFixedWaves + wv] = c_feas;
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
#pragma unroll 1
        for (int w = 1; w < kFixedWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        if (lane < k) a.wg_lists[(uint64_t)blockIdx.x * k + lane] = slot;
        if (lane < 2) {
            unsigned long long t = 0;
            for (int w = 0; w < kFixedWaves; w++) t += s_cnt[lane * kFixedWaves + w];
            a.wg_counts[2 * (uint64_t)blockIdx.x + lane] = t;
        }
    }
}

// ---------------------------------------------------------------------------
// Merge: the workgroup lists into the final top-k (one workgroup).  Each list
// is sorted and holds k keys, so the largest k-th key of any list bounds the
// final k-th key from below: keys under it are dropped before selection.
// Keys are loaded several per lane ahead of their selection.
// ---------------------------------------------------------------------------
constexpr int kFixedMergeWaves = 16;
constexpr int kMergeAhead = 4;

__global__ void __launch_bounds__(kFixedMergeWaves * 64)
fixed_merge_kernel(const K128 *lists, const unsigned long long *wg_counts, int n_lists, int k, DevResult *R)
{
    __shared__ K128 lst[kFixedMergeWaves * 64];
    __shared__ unsigned long long s_cnt[2 * kFixedMergeWaves];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    // the workgroups' counts
    unsigned long long cv = 0, cf = 0;
    for (int l = threadIdx.x; l < n_lists; l += blockDim.x) {
        cv += wg_counts[2 * (int64_t)l];
        cf += wg_counts[2 * (int64_t)l + 1];
    }
    cv = wave_sum64(cv);
    cf = wave_sum64(cf);
    if (lane == 0) {
        s_cnt[wv] = cv;
        s_cnt[kFixedMergeWaves + wv] = cf;
    }
    // the largest k-th key over the lists
    K128 lb = {0ull, 0ull};
    for (int l = threadIdx.x; l < n_lists; l += blockDim.x) {
        const K128 x = lists[(int64_t)l * k + (k - 1)];
        if (gt128(x, lb)) lb = x;
    }
    lst[threadIdx.x] = lb;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s && gt128(lst[threadIdx.x + s], lst[threadIdx.x])) lst[threadIdx.x] = lst[threadIdx.x + s];
        __syncthreads();
    }
    lb = lst[0];
    __syncthreads();

    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    const int64_t n_keys = (int64_t)n_lists * k;
    const int64_t per_wave = (n_keys + kFixedMergeWaves - 1) / kFixedMergeWaves;
    const int64_t e0 = (int64_t)wv * per_wave;
    const int64_t e1 = e0 + per_wave < n_keys ? e0 + per_wave : n_keys;
    for (int64_t base = e0; base < e1; base += 64 * kMergeAhead) {
        K128 key[kMergeAhead];
#pragma unroll
        for (int q = 0; q < kMergeAhead; q++) {
            const int64_t e = base + q * 64 + lane;
            key[q] = K128{0ull, 0ull};
            if (e < e1) key[q] = lists[e];
        }
#pragma unroll
        for (int q = 0; q < kMergeAhead; q++)
            list128_offer(slot, key_if(!gt128(lb, key[q]), key[q]), lane, k, thr);
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
        for (int w = 1; w < kFixedMergeWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        const int n_top = __popcll(__ballot(lane < k && nz128(slot)));
        if (lane < MF_MAX_TOPK) {
            const bool ok = lane < n_top;
            R->top_idx[lane] = ok ? ~slot.lo : ~0ull;
            R->top_J[lane] = ok ? unord_f64(slot.hi) : -INFINITY;
        }
        if (lane == 0) {
            R->n_top = n_top;
            R->status |= kStatVerified;
        }
        if (lane < 2) {
            unsigned long long t = 0;
            for (int w = 0; w < kFixedMergeWaves; w++) t += s_cnt[lane * kFixedMergeWaves + w];
            (lane == 0 ? R->n_vram : R->n_feas_sure) = t;
        }
    }
}

size_t fixed_lds_bytes(int sumK, bool eq3)
{
    return (size_t)sumK * sizeof(FixedRow) + (eq3 ? (size_t)sumK * sizeof(FixedPen) : 0) +
           (size_t)kFixedWaves * 64 * sizeof(K128);
}

using ScanFn = void (*)(const FixedArgs);

static ScanFn scan_fn(const FixedArgs &a)
{
    const bool eq3 = a.obj.kind != 0;
    const int ni = a.n_models - a.n_outer;
    // two inner models, a periodic last digit, whole blocks, no dump
    if (ni == 2 && !a.mask && a.part_block_lo == ~0ull && a.part_block_hi == ~0ull && a.in_K[1] >= 1 &&
        a.blocks_per_wave * (uint64_t)a.inner < (1ull << 32)) {
        const uint32_t kb = (uint32_t)a.in_K[1];
        uint32_t g = 64, x = kb;
        while (x) {
            const uint32_t t = g % x;
            g = x;
            x = t;
        }
        const uint32_t per = kb / g;
        // option counts up to 255 give P = 1 (powers of two), 2 (128) or 3
        // (3 times a power of two)
        if (per <= 3 && a.inner % (64u * per) == 0) {
            // blocks of 3 groups of 3 tiles (24 x 24 options) and of 4
            // single tiles (16 x 16) unrolled
            const uint32_t ng = a.inner / (64u * per);
            if (per == 3 && ng == 3) return eq3 ? fixed_periodic_kernel<3, true, 3> : fixed_periodic_kernel<3, false, 3>;
            if (per == 1 && ng == 4) return eq3 ? fixed_periodic_kernel<1, true, 4> : fixed_periodic_kernel<1, false, 4>;
            switch (per) {
                case 1: return eq3 ? fixed_periodic_kernel<1, true> : fixed_periodic_kernel<1, false>;
                case 2: return eq3 ? fixed_periodic_kernel<2, true> : fixed_periodic_kernel<2, false>;
                case 3: return eq3 ? fixed_periodic_kernel<3, true> : fixed_periodic_kernel<3, false>;
            }
        }
    }
    if (a.lc_shift >= 0) return eq3 ? fixed_scan_kernel<2, true, true> : fixed_scan_kernel<2, false, true>;
    // two inner models, the second with at least two options, whole 64-tiles
    if (ni == 2 && a.in_K[1] >= 2 && a.inner % 64 == 0)
        return eq3 ? fixed_scan_kernel<2, true, false, true> : fixed_scan_kernel<2, false, false, true>;
    return ni <= 2 ? (eq3 ? fixed_scan_kernel<2, true, false> : fixed_scan_kernel<2, false, false>)
         : ni <= 4 ? (eq3 ? fixed_scan_kernel<4, true, false> : fixed_scan_kernel<4, false, false>)
                   : (eq3 ? fixed_scan_kernel<kMaxN, true, false> : fixed_scan_kernel<kMaxN, false, false>);
}

int fixed_wgs_per_cu(const FixedArgs &a)
{
    const ScanFn fn = scan_fn(a);
    const size_t lds = fixed_lds_bytes(a.sumK, a.obj.kind != 0);
    if (ensure_dyn_lds((const void *)fn, lds) != hipSuccess)
        return 1;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kFixedWaves * 64, lds) != hipSuccess || n < 1) return 1;
    return n < kFixedMaxWgsPerCu ? n : kFixedMaxWgsPerCu;
}

hipError_t launch_fixed(const FixedArgs &a, int grid, bool table, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1)
{
    hipError_t e;
    if (table && (e = launch_fixed_table(a, s)) != hipSuccess) return e;
    const size_t lds = fixed_lds_bytes(a.sumK, a.obj.kind != 0);
    const ScanFn fn = scan_fn(a);
    e = ensure_dyn_lds((const void *)fn, lds);
    if (e != hipSuccess) return e;
    if (ev0 && (e = hipEventRecord(ev0, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kFixedWaves * 64), lds, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev1 && (e = hipEventRecord(ev1, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fixed_merge_kernel, dim3(1), dim3(kFixedMergeWaves * 64), 0, s, a.wg_lists, a.wg_counts, grid,
                       a.top_k, a.res);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Static (multi-step) search: S = sum over steps of J_t, one configuration
// for all steps.  Per step t the table kernel has filled rows_steps[t]; the
// VRAM sum is the same at every step.
// ---------------------------------------------------------------------------

// One model's step of step t's chain: service flags and J (VRAM apart).
template <bool EQ3>
__device__ __forceinline__ void chain_J(const FixedRow &r, const FixedPen *pens, uint32_t row, double om, double &J,
                                        uint32_t &fl)
{
    fl |= r.flags;
    J = fma(om, r.q, J);
    if (EQ3) {
        const FixedPen pp = pens[row];
        if (r.flags & kRowP) J = J - pp.P;
        if (r.flags & kRowPen) J = J - pp.pen;
    }
}

__host__ __device__ constexpr size_t static_om_doubles(int n_steps, int n_models)
{
    return ((size_t)n_steps * n_models + 1) & ~(size_t)1;   // 16-byte multiple
}

size_t static_lds_bytes(int n_steps, int sumK, int n_models, bool eq3)
{
    const size_t rows = (size_t)n_steps * sumK;
    return rows * sizeof(FixedRow) + (eq3 ? rows * sizeof(FixedPen) : 0) +
           static_om_doubles(n_steps, n_models) * 8 + (size_t)kFixedWaves * 64 * sizeof(K128);
}

template <int NI, bool EQ3>
__global__ void __launch_bounds__(kFixedWaves * 64) static_scan_kernel(const StaticArgs sa)
{
    const FixedArgs &a = sa.f;
    extern __shared__ float4 smem4[];
    __shared__ int32_t s_off[kMaxN], s_K[kMaxN];
    __shared__ uint32_t s_od[kFixedWaves][kMaxN];
    __shared__ double s_preJ[kFixedWaves][MF_MAX_STEPS];     // outer prefix of each step's chain
    __shared__ uint32_t s_preF[kFixedWaves][MF_MAX_STEPS];
    const int T = sa.n_steps, sumK = a.sumK, N = a.n_models, nout = a.n_outer, ni = N - nout, k = a.top_k;
    const int TR = T * sumK;
    FixedRow *rows = reinterpret_cast<FixedRow *>(smem4);                    // [T][sumK]
    FixedPen *pens = reinterpret_cast<FixedPen *>(rows + TR);                // [T][sumK] (Eq. 3)
    double *om = reinterpret_cast<double *>(pens + (EQ3 ? TR : 0));          // [T][N]
    K128 *lst = reinterpret_cast<K128 *>(om + static_om_doubles(T, N));
#pragma unroll 1
    for (int t = threadIdx.x; t < TR; t += blockDim.x) {
        rows[t] = sa.rows_steps[t];
        if (EQ3) pens[t] = sa.pens_steps[t];
    }
    for (int t = threadIdx.x; t < T * N; t += blockDim.x) om[t] = (double)sa.omega_steps[t];
#pragma unroll
    for (int j = 0; j < kMaxN; j++)
        if (threadIdx.x == (unsigned)j) {
            s_off[j] = a.opt_off[j];
            s_K[j] = a.K[j];
        }

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint64_t gw = (uint64_t)blockIdx.x * kFixedWaves + wv;
    const uint64_t b_first = gw * a.blocks_per_wave;
    const uint64_t b_begin = a.block0 + (b_first < a.n_blocks ? b_first : a.n_blocks);
    const uint64_t b_end = a.block0 + (b_first + a.blocks_per_wave < a.n_blocks ? b_first + a.blocks_per_wave
                                                                                : a.n_blocks);
    const uint64_t idx_lo = a.lo, idx_hi = a.lo + a.n;
    const uint32_t M = a.inner;
    const float cap = a.vram_cap;
    uint32_t *od = s_od[wv];
    if (lane == 0) {
        uint64_t x = b_begin;
        for (int j = nout - 1; j >= 0; j--) {
            od[j] = (uint32_t)(x % (uint64_t)a.K[j]);
            x /= (uint64_t)a.K[j];
        }
    }
    __syncthreads();

    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    double thrS = -INFINITY;
    unsigned long long c_vram = 0, c_feas = 0;

    for (uint64_t b = b_begin; b < b_end; b++) {
        // outer prefix: the VRAM sum once, each step's chain (wave-uniform)
        float vp = 0.f;
#pragma unroll 1
        for (int j = 0; j < nout; j++) vp += rows[s_off[j] + od[j]].vram;
#pragma unroll 1
        for (int t = 0; t < T; t++) {
            double J = 0.0;
            uint32_t fl = 0u;
#pragma unroll 1
            for (int j = 0; j < nout; j++) {
                const uint32_t row = (uint32_t)(t * sumK + s_off[j]) + od[j];
                chain_J<EQ3>(rows[row], pens, row, om[t * N + j], J, fl);
            }
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) {
                s_preJ[wv][t] = J;
                s_preF[wv][t] = fl;
            }
            __builtin_amdgcn_wave_barrier();
        }
        const uint64_t base = b * (uint64_t)M;
        const uint32_t u_lo = base < idx_lo ? (uint32_t)(idx_lo - base) : 0u;
        const uint32_t u_hi = idx_hi - base < (uint64_t)M ? (uint32_t)(idx_hi - base) : M;
        const uint32_t u_span = u_hi - u_lo;
        uint32_t cv = 0, cf = 0;
#pragma unroll 1
        for (uint32_t t0 = 0; t0 < M; t0 += 64) {
            const uint32_t u = t0 + (uint32_t)lane;
            uint32_t uu = u < M ? u : 0u;
            uint32_t rr[NI];
#pragma unroll
            for (int q = NI - 1; q >= 0; q--) {
                rr[q] = 0;
                if (q < ni) {
                    const uint32_t qq = (q > 0 && a.in_magic[q]) ? __umulhi(uu, a.in_magic[q]) : (q > 0 ? uu : 0u);
                    rr[q] = (uint32_t)a.in_off[q] + (uu - qq * (uint32_t)a.in_K[q]);
                    uu = qq;
                }
            }
            float v = vp;
#pragma unroll
            for (int q = 0; q < NI; q++)
                if (q < ni) v += rows[rr[q]].vram;
            double S = 0.0;
            uint32_t fall = 0u;
#pragma unroll 1
            for (int t = 0; t < T; t++) {
                double J = s_preJ[wv][t];
                uint32_t fl = s_preF[wv][t];
#pragma unroll
                for (int q = 0; q < NI; q++)
                    if (q < ni) {
                        const uint32_t row = (uint32_t)(t * sumK) + rr[q];
                        chain_J<EQ3>(rows[row], pens, row, om[t * N + nout + q], J, fl);
                    }
                S = t == 0 ? J : S + J;
                fall |= fl;
            }
            const unsigned long long mv = ballot64(u - u_lo < u_span);
            const unsigned long long vm = mv & ballot64(v <= cap);
            const unsigned long long fm = vm & ballot64((int32_t)fall >= 0);
            const unsigned long long cm = fm & ballot64(S >= thrS);
            cv += (uint32_t)__popcll(vm);
            cf += (uint32_t)__popcll(fm);
            if (cm) offer_mask(slot, thr, thrS, cm, S, base + u, lane, k);
            if (a.mask && ((mv >> lane) & 1ull)) {
                const bool vok = v <= cap, sok = (int32_t)fall >= 0;
                a.mask[base + u - idx_lo] = (uint8_t)((vok ? 1u : 0u) | (sok ? 2u : 0u) | (vok && sok ? 4u : 0u));
            }
        }
        c_vram += cv;
        c_feas += cf;
        bool carry = true;
        for (int j = nout - 1; j >= 0 && carry; j--) {
            uint32_t d = od[j] + 1u;
            carry = d == (uint32_t)s_K[j];
            if (carry) d = 0u;
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) od[j] = d;
            __builtin_amdgcn_wave_barrier();
        }
    }

    // counts and list per workgroup (the merge kernel sums and merges them)
    __shared__ unsigned long long s_cnt[2 * kFixedWaves];
    if (lane == 0) {
        s_cnt[wv] = c_vram;
        s_cnt[kFixedWaves + wv] = c_feas;
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
#pragma unroll 1
        for (int w = 1; w < kFixedWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        if (lane < k) a.wg_lists[(uint64_t)blockIdx.x * k + lane] = slot;
        if (lane < 2) {
            unsigned long long t = 0;
            for (int w = 0; w < kFixedWaves; w++) t += s_cnt[lane * kFixedWaves + w];
            a.wg_counts[2 * (uint64_t)blockIdx.x + lane] = t;
        }
    }
}

// List mode: one thread per index, every model decoded, each step's chain.
template <bool EQ3>
__global__ void __launch_bounds__(256) static_eval_kernel(const StaticArgs sa)
{
    const FixedArgs &a = sa.f;
    const int T = sa.n_steps, sumK = a.sumK, N = a.n_models;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < sa.n_list;
         e += (int64_t)gridDim.x * blockDim.x) {
        uint64_t x = sa.idx[e];
        uint32_t row[kMaxN];
#pragma unroll
        for (int j = kMaxN - 1; j >= 0; j--) {
            row[j] = 0;
            if (j < N) {
                row[j] = (uint32_t)a.opt_off[j] + (uint32_t)(x % (uint64_t)a.K[j]);
                x /= (uint64_t)a.K[j];
            }
        }
        float v = 0.f;
#pragma unroll
        for (int j = 0; j < kMaxN; j++)
            if (j < N) v += sa.rows_steps[row[j]].vram;
        const uint32_t vok = v <= a.vram_cap ? 1u : 0u;
        double S = 0.0;
        for (int t = 0; t < T; t++) {
            double J = 0.0;
            uint32_t fl = 0u;
#pragma unroll
            for (int j = 0; j < kMaxN; j++)
                if (j < N) {
                    const uint32_t r = (uint32_t)(t * sumK) + row[j];
                    chain_J<EQ3>(sa.rows_steps[r], sa.pens_steps, r, (double)sa.omega_steps[t * N + j], J, fl);
                }
            S = t == 0 ? J : S + J;
            if (sa.out_J) sa.out_J[e * T + t] = J;
            if (sa.out_flags) sa.out_flags[e * T + t] = vok | ((int32_t)fl >= 0 ? 2u : 0u);
        }
        if (sa.out_S) sa.out_S[e] = S;
    }
}

using StaticFn = void (*)(const StaticArgs);

static StaticFn static_fn(const StaticArgs &a)
{
    const bool eq3 = a.f.obj.kind != 0;
    const int ni = a.f.n_models - a.f.n_outer;
    return ni <= 2 ? (eq3 ? static_scan_kernel<2, true> : static_scan_kernel<2, false>)
         : ni <= 4 ? (eq3 ? static_scan_kernel<4, true> : static_scan_kernel<4, false>)
                   : (eq3 ? static_scan_kernel<kMaxN, true> : static_scan_kernel<kMaxN, false>);
}

int static_wgs_per_cu(const StaticArgs &a)
{
    const StaticFn fn = static_fn(a);
    const size_t lds = static_lds_bytes(a.n_steps, a.f.sumK, a.f.n_models, a.f.obj.kind != 0);
    if (ensure_dyn_lds((const void *)fn, lds) != hipSuccess)
        return 1;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kFixedWaves * 64, lds) != hipSuccess || n < 1) return 1;
    return n < kFixedMaxWgsPerCu ? n : kFixedMaxWgsPerCu;
}

hipError_t launch_fixed_table(const FixedArgs &a, hipStream_t s)
{
    if (a.bf16)
        hipLaunchKernelGGL(fixed_table_kernel<true>, dim3(a.sumK), dim3(64), 0, s, a);
    else
        hipLaunchKernelGGL(fixed_table_kernel<false>, dim3(a.sumK), dim3(64), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_static(const StaticArgs &a, int grid, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1)
{
    const size_t lds = static_lds_bytes(a.n_steps, a.f.sumK, a.f.n_models, a.f.obj.kind != 0);
    const StaticFn fn = static_fn(a);
    hipError_t e = ensure_dyn_lds((const void *)fn, lds);
    if (e != hipSuccess) return e;
    if (ev0 && (e = hipEventRecord(ev0, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kFixedWaves * 64), lds, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev1 && (e = hipEventRecord(ev1, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fixed_merge_kernel, dim3(1), dim3(kFixedMergeWaves * 64), 0, s, a.f.wg_lists, a.f.wg_counts,
                       grid, a.f.top_k, a.f.res);
    return hipGetLastError();
}

hipError_t launch_static_eval(const StaticArgs &a, hipStream_t s)
{
    const int64_t blocks = (a.n_list + 255) / 256;
    const int grid = (int)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
    if (a.f.obj.kind != 0)
        hipLaunchKernelGGL(static_eval_kernel<true>, dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(static_eval_kernel<false>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace mfi
