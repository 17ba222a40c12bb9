// Canonical fp64 evaluation and the exact top-k selection.
//
// Results of the search are defined by canonical fp64 semantics (each dot
// product one fused multiply-add chain, ascending inputs, starting from the
// bias; relu(x) = x > 0 ? x : +0; J the fma chain over models; in bf16 mode
// the first hidden layer accumulates in fp32 and is rounded to bfloat16).  The fast
// fp32 MFMA path settles every latency decision whose margin exceeds its
// a-priori error bound; the rest, and every top-k candidate, are evaluated
// here with that exact chain (v_fma_f64 is correctly rounded, so the values
// are the canonical ones bit for bit).
//
// One workgroup per entry, lanes over hidden units.  The long certification
// lists run one wave per entry, model after model.  Few entries (the top-k
// candidates, short index lists) are latency-bound: there (FEW) wave w runs
// the forward of the entry's models w, w + W, ... on its own scratch, and
// wave 0 combines them in model order.
#include <algorithm>

#include "mf_canon.h"

namespace mfi {


// Canonical image per model (fp32 values, exact in fp64):
//   W1T[nin][H1], b1[H1], W2T[H1][H2], b2[H2], W3[2][H2], b3[2]
template <bool BF16, bool FEW>
__global__ void __launch_bounds__(FEW ? 64 * kCanonWaves : 64)
canon_kernel(const CanonArgs a, const int search_mode)
{
    extern __shared__ double canon_dyn[];   // FEW: [W][H1 + H2 + nin]
    __shared__ double h1s_1[FEW ? 1 : kCanonMaxH];
    __shared__ double h2s_1[FEW ? 1 : kCanonMaxH];
    __shared__ double zs_1[FEW ? 1 : kCanonMaxIn];
    __shared__ int32_t ds[kMaxN];
    __shared__ float aggs[16];
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    __shared__ double s_lat[FEW ? kMaxN : 1], s_thr[FEW ? kMaxN : 1];
    const int lane = threadIdx.x & 63;
    const int wave = FEW ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
    const int W = FEW ? (int)(blockDim.x >> 6) : 1;
#pragma unroll
    for (int i = 0; i < kMaxN; i++)   // compile-time index into the argument block
        if (threadIdx.x == (unsigned)i) {
            s_tau[i] = a.obj.tau[i];
            s_prev[i] = a.obj.prev[i];
        }
    const bool eq3 = a.obj.kind != 0;
    const int N = a.n_models, L = a.L, A = a.A, H1 = a.H1, H2 = a.H2, nin = L + A;
    double *h1s = h1s_1, *h2s = h2s_1, *zs = zs_1;
    if (FEW) {
        h1s = canon_dyn + (int64_t)wave * (H1 + H2 + nin);
        h2s = h1s + H1;
        zs = h2s + H2;
    }
    __syncthreads();

    int64_t n_cand = 0, n_work = 0, n_coll = 0, n_ent, e0 = 0;
    double jthr = -INFINITY;   // certification entries need the full J only from here up
    if (search_mode) {
        n_cand = a.collect_mode ? 0 : a.n_cand_keys;
        n_work = (int64_t)min(a.res->n_work, (unsigned long long)a.work_cap);
        n_coll = a.collect_mode ? (int64_t)min(a.res->n_collect, (unsigned long long)a.collect_cap) : 0;
        // phase 0: the fast candidates; phase 1: certification (+ collected) entries
        if (a.phase == 0) {
            n_ent = n_cand;
        } else {
            e0 = n_cand;
            n_ent = n_cand + n_work + n_coll;
            // an entry whose upper bound U is below the k-th canonical J of
            // the candidates (the collect threshold in the fallback pass)
            // cannot enter the top-k: only its uncertain models are needed
            jthr = a.collect_mode ? a.res->theta : a.res->ck_cand;
        }
    } else {
        n_ent = a.n_list;
    }

    for (int64_t e = e0 + blockIdx.x; e < n_ent; e += gridDim.x) {
        uint64_t idx, off = 0;
        uint32_t models = 0xFFFFFFFFu;   // models to evaluate
        bool work_entry = false, need_J = true;
        if (search_mode) {
            if (e < n_cand) {
                const unsigned long long key = a.cand_keys[e];
                if (key == 0ull) {
                    if (threadIdx.x == 0) { a.ent_J[e] = -INFINITY; a.ent_flags[e] = 0; }
                    continue;
                }
                off = 0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull);
            } else if (e < n_cand + n_work) {
                const unsigned long long w = a.work[e - n_cand];
                off = (uint32_t)(w & 0xFFFFFFFFull);
                work_entry = true;
                need_J = (double)a.work_J[e - n_cand] >= jthr;
                if (!need_J) models = (uint32_t)(w >> 32);
            } else {
                off = a.collect[e - n_cand - n_work];
            }
            idx = a.lo + off;
        } else {
            idx = a.idx64[e];
        }
        // decode (model N-1 least significant): thread i < N takes digit i
        if (FEW) __syncthreads();   // the previous entry's combine has read ds and aggs
        if (threadIdx.x < (unsigned)N) {
            uint64_t stride = 1;
            for (int j = N - 1; j > lane; j--) stride *= (uint64_t)a.K[j];
            ds[lane] = (int32_t)((idx / stride) % (uint64_t)a.K[lane]);
        }
        __syncthreads();
        // aggregate field: thread k < A sums slot k in fp32, model order
        if (threadIdx.x < (unsigned)A) {
            float s = 0.f;
            for (int i = 0; i < N; i++)
                s = s + a.features[(int64_t)(a.opt_off[i] + ds[i]) * L + a.agg_cols[lane]];
            aggs[lane] = s;
        }
        __syncthreads();
        if (FEW) {
            // the entry's models, W at a time: every wave takes part in every
            // round (the forward has barriers); a wave past the last model
            // repeats the first one and drops the result
            const uint32_t need = models & ((1u << N) - 1u);
            const int n_need = __popc(need);
            for (int r0 = 0; r0 < n_need; r0 += W) {
                const int q = r0 + wave;
                uint32_t m = need;
                for (int j = 0; j < q && m; j++) m &= m - 1u;
                const bool act = q < n_need;
                const int i = act ? __ffs(m) - 1 : __ffs(need) - 1;
                const float *x = a.features + (int64_t)(a.opt_off[i] + ds[i]) * L;
                for (int k = lane; k < nin; k += 64) zs[k] = k < L ? (double)x[k] : (double)aggs[k - L];
                __syncthreads();
                double lat, thr;
                canon_model<BF16>(a.weights + (int64_t)i * a.wstride, nin, H1, H2, zs, h1s, h2s, lane, lat, thr, a.act);
                if (act && lane == 0) {
                    s_lat[i] = lat;
                    s_thr[i] = thr;
                }
            }
            __syncthreads();
            if (wave != 0) continue;
        }
        const bool vram_ok = (double)aggs[a.vram_slot] <= (double)a.vram_cap;
        bool sla_ok = true;
        uint32_t fl = 0;
        double J = 0.0;
        for (int i = 0; i < N; i++) {
            if (!((models >> i) & 1u)) continue;
            double lat, thr;
            if (FEW) {
                lat = s_lat[i];
                thr = s_thr[i];
            } else {
                const float *x = a.features + (int64_t)(a.opt_off[i] + ds[i]) * L;
                for (int k = lane; k < nin; k += 64) zs[k] = k < L ? (double)x[k] : (double)aggs[k - L];
                __syncthreads();
                canon_model<BF16>(a.weights + (int64_t)i * a.wstride, nin, H1, H2, zs, h1s, h2s, lane, lat, thr, a.act);
            }
            if (!(lat <= (double)a.sla[i])) { sla_ok = false; fl |= 1u << (8 + i); }
            if (eq3) {
                // Eq. 3 (Section II): per-variant min-max throughput, quality,
                // reload penalty, soft SLA penalty; the throughput floor
                const int64_t row = (int64_t)a.opt_off[i] + ds[i];
                double q, P, pen;
                bool do_P, do_pen;
                const bool floor_ok = canon_eq3(a.obj, row, thr, s_tau[i], s_prev[i], q, P, do_P, pen, do_pen);
                if (!floor_ok) { sla_ok = false; fl |= 1u << (8 + i); }
                J = fma((double)a.omega[i], q, J);
                if (do_P) J = J - P;
                if (do_pen) J = J - pen;
            } else {
                J = fma((double)a.omega[i], thr, J);
            }
            if (a.pred && lane == 0) {
                a.pred[(e * N + i) * 2 + 0] = lat;
                a.pred[(e * N + i) * 2 + 1] = thr;
            }
            if (!FEW) __syncthreads();
        }
        const bool feas = vram_ok && sla_ok;
        fl |= (vram_ok ? 1u : 0u) | (sla_ok ? 2u : 0u) | (feas ? 4u : 0u);
        if (feas && !need_J) fl |= kEntNoJ;
        if (lane == 0) {
            if (a.ent_J) a.ent_J[e] = (feas && need_J) ? J : -INFINITY;
            if (a.ent_flags) a.ent_flags[e] = fl;
            if (search_mode && a.mask && work_entry)
                a.mask[off] = (uint8_t)((a.mask[off] & 1u) | (sla_ok ? 2u : 0u) | (feas ? 4u : 0u) | 8u);
        }
    }
}

hipError_t launch_canonical(const CanonArgs &a, int n_entries_max, bool search_mode, hipStream_t s)
{
    int grid = n_entries_max < 1 ? 1 : n_entries_max;
    if (grid > kCanonMaxGrid) grid = kCanonMaxGrid;
    const int sm = search_mode ? 1 : 0;
    const bool few = search_mode ? a.phase == 0 : n_entries_max <= kCanonFewEntries;
    if (!few) {
        if (a.bf16)
            hipLaunchKernelGGL((canon_kernel<true, false>), dim3(grid), dim3(64), 0, s, a, sm);
        else
            hipLaunchKernelGGL((canon_kernel<false, false>), dim3(grid), dim3(64), 0, s, a, sm);
        return hipGetLastError();
    }
    // a wave per model
    const int W = a.n_models < kCanonWaves ? a.n_models : kCanonWaves;
    const size_t lds = (size_t)W * (a.H1 + a.H2 + a.L + a.A) * 8;
    auto fn = a.bf16 ? canon_kernel<true, true> : canon_kernel<false, true>;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(64 * W), lds, s, a, sm);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Exact top-k over the canonically evaluated entries (128-bit keys K128).
// ---------------------------------------------------------------------------
constexpr int kSelWaves = 16;

// k-th canonical J among the fast candidates (by J desc, index asc); -inf if
// fewer than k are feasible.  One workgroup; kp <= 1024.
__global__ void __launch_bounds__(1024) kth_candidate_kernel(const unsigned long long *cand, const double *ent_J,
                                                             const uint32_t *ent_flags, int kp, int k, DevResult *R)
{
    const int e = threadIdx.x;
    if (e == 0) R->ck_cand = -INFINITY;
    __syncthreads();
    if (e >= kp) return;
    const bool ok = cand[e] != 0ull && (ent_flags[e] & 4u);
    const double v = ok ? ent_J[e] : -INFINITY;
    const uint64_t iv = ok ? (uint64_t)(0xFFFFFFFFu - (uint32_t)(cand[e] & 0xFFFFFFFFull)) : ~0ull;
    int rank = 0;
    for (int f = 0; f < kp; f++) {
        const bool okf = cand[f] != 0ull && (ent_flags[f] & 4u);
        const double vf = okf ? ent_J[f] : -INFINITY;
        const uint64_t ivf = okf ? (uint64_t)(0xFFFFFFFFu - (uint32_t)(cand[f] & 0xFFFFFFFFull)) : ~0ull;
        rank += (vf > v || (vf == v && ivf < iv) || (vf == v && ivf == iv && f < e)) ? 1 : 0;
    }
    if (ok && rank == k - 1) R->ck_cand = v;
}

hipError_t launch_kth_candidate(const unsigned long long *cand_keys, const double *ent_J, const uint32_t *ent_flags,
                                int kp, int k, DevResult *res, hipStream_t s)
{
    hipLaunchKernelGGL(kth_candidate_kernel, dim3(1), dim3(1024), 0, s, cand_keys, ent_J, ent_flags, kp, k, res);
    return hipGetLastError();
}


// MODE 0: one workgroup over every entry, then the result.  MODE 1: each
// workgroup of a grid over a stride of the entries, its top-k, count and
// checks to parts[blockIdx.x].  MODE 2: one workgroup merges the parts, then
// the result.
template <int MODE>
__global__ void __launch_bounds__(kSelWaves * 64)
select_kernel(const SelectArgs a, SelPart *parts, int n_parts)
{
    __shared__ K128 lst[kSelWaves * 64];
    __shared__ unsigned long long s_feas;
    __shared__ unsigned int s_stat;
    __shared__ double s_maxd;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    DevResult *R = a.res;
    if (threadIdx.x == 0) { s_feas = 0; s_stat = 0; s_maxd = 0.0; }
    __syncthreads();
    const int64_t n_cand = a.collect_mode ? 0 : a.kp;
    const int64_t n_work = (int64_t)min(R->n_work, (unsigned long long)a.work_cap);
    const int64_t n_coll = a.collect_mode ? (int64_t)min(R->n_collect, (unsigned long long)a.collect_cap) : 0;
    const int64_t n_ent = n_cand + n_work + n_coll;
    const int k = a.top_k;
    K128 slot = {0, 0}, thr = {0, 0};
    unsigned long long my_feas = 0;
    if (MODE == 2) {
        // the parts: lists (sorted, zeros past k), counts, checks
        for (int p = wv; p < n_parts; p += kSelWaves) list128_offer(slot, parts[p].keys[lane], lane, k, thr);
        for (int p = threadIdx.x; p < n_parts; p += kSelWaves * 64) {
            my_feas += parts[p].feas;
            if (parts[p].stat) atomicOr(&s_stat, parts[p].stat);
            atomicMax((unsigned long long *)&s_maxd, (unsigned long long)__double_as_longlong(parts[p].maxd));
        }
    }
    const int64_t e_first = MODE == 1 ? ((int64_t)blockIdx.x * kSelWaves + wv) * 64 : (int64_t)wv * 64;
    const int64_t e_step = MODE == 1 ? (int64_t)gridDim.x * kSelWaves * 64 : kSelWaves * 64;
    for (int64_t base = MODE == 2 ? n_ent : e_first; base < n_ent; base += e_step) {
        const int64_t e = base + lane;
        K128 key = {0, 0};
        if (e < n_ent) {
            const uint32_t fl = a.ent_flags[e];
            uint64_t off = 0;
            bool have = true;
            if (e < n_cand) {
                const unsigned long long ck = a.cand_keys[e];
                have = ck != 0ull;
                off = 0xFFFFFFFFu - (uint32_t)(ck & 0xFFFFFFFFull);
                if (have) {
                    // a sure-feasible fast decision must be canonically
                    // feasible, and the key's U must bound the canonical J
                    if (!(fl & 4u)) atomicOr(&s_stat, kStatSelfCheck);
                    const double U = (double)unord_f32((uint32_t)(ck >> 32));
                    const double dj = U - a.ent_J[e];
                    if (!(dj >= 0.0)) atomicOr(&s_stat, kStatSelfCheck);
                    if (dj >= 0.0)
                        atomicMax((unsigned long long *)&s_maxd, (unsigned long long)__double_as_longlong(dj));
                }
            } else if (e < n_cand + n_work) {
                off = (uint32_t)(a.work[e - n_cand] & 0xFFFFFFFFull);
                if (fl & 4u) my_feas++;
                have = !(fl & kEntNoJ);
            } else {
                off = a.collect[e - n_cand - n_work];
            }
            if (have && (fl & 4u)) key = {ord_f64(a.ent_J[e]), ~(a.lo + off)};
        }
        list128_offer(slot, key, lane, k, thr);
    }
    if (my_feas) atomicAdd(&s_feas, my_feas);
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (MODE == 1) {
        if (wv == 0) {
            for (int w = 1; w < kSelWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
            SelPart &pt = parts[blockIdx.x];
            pt.keys[lane] = key_if(lane < k, slot);
            if (lane == 0) {
                pt.feas = s_feas;
                pt.stat = s_stat;
                pt.maxd = s_maxd;
            }
        }
        return;
    }
    if (wv == 0) {
        for (int w = 1; w < kSelWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        const int n_top = __popcll(__ballot(lane < k && nz128(slot)));
        const uint64_t kth_hi = readlane64(slot.hi, k - 1);
        if (lane < MF_MAX_TOPK) {
            const bool ok = lane < n_top;
            R->top_idx[lane] = ok ? ~slot.lo : ~0ull;
            const uint64_t o = slot.hi;
            const uint64_t b = (o & 0x8000000000000000ull) ? (o & 0x7FFFFFFFFFFFFFFFull) : ~o;
            R->top_J[lane] = ok ? __longlong_as_double((long long)b) : -INFINITY;
        }
        if (lane == 0) {
            R->n_top = n_top;
            unsigned stat = s_stat;
            if (!a.collect_mode) {
                R->n_feas_cert = s_feas;
                R->check_max_dJ = s_maxd;
                const unsigned long long tail = a.cand_keys[a.kp - 1];
                const bool full = tail != 0ull;
                if (full) stat |= kStatListFull;
                // every sure-feasible configuration outside the list has an
                // upper bound U <= tail_U: exact when the k-th canonical J
                // exceeds it; otherwise the fallback collects all U >= C_k
                const double tailU = full ? (double)unord_f32((uint32_t)(tail >> 32)) : -INFINITY;
                R->tail_U = tailU;
                bool verified = !full;
                if (full && n_top >= k) {
                    const uint64_t b = (kth_hi & 0x8000000000000000ull) ? (kth_hi & 0x7FFFFFFFFFFFFFFFull) : ~kth_hi;
                    const double Ck = __longlong_as_double((long long)b);
                    verified = Ck > tailU;
                    R->theta = Ck;
                }
                if (verified) stat |= kStatVerified;
            } else {
                stat |= kStatVerified;
            }
            if (R->n_work > a.work_cap) stat |= kStatWorkOverflow;
            if (a.collect_mode && R->n_collect > a.collect_cap) stat |= kStatCollectOverflow;
            R->status |= stat;
        }
    }
}

hipError_t launch_select(const SelectArgs &a, hipStream_t s)
{
    if (a.n_parts <= 1) {
        hipLaunchKernelGGL(select_kernel<0>, dim3(1), dim3(kSelWaves * 64), 0, s, a, (SelPart *)nullptr, 0);
    } else {
        hipLaunchKernelGGL(select_kernel<1>, dim3(a.n_parts), dim3(kSelWaves * 64), 0, s, a, a.parts, a.n_parts);
        hipLaunchKernelGGL(select_kernel<2>, dim3(1), dim3(kSelWaves * 64), 0, s, a, a.parts, a.n_parts);
    }
    return hipGetLastError();
}

}  // namespace mfi

// ---------------------------------------------------------------------------
// Small ranges: the rest of the search in one workgroup.  The fast kernel's
// workgroups have already evaluated canonically their first list entries and
// their certification segments; this kernel sums counts and selects.
// ---------------------------------------------------------------------------
namespace mfi {

constexpr int kFinWaves = 8;

// Segment of certification entry e: the last workgroup whose exclusive
// prefix is <= e (empty segments share their offset with the next).
__device__ __forceinline__ int seg_of(const uint32_t *off, int n_wg, uint32_t e)
{
    int lo = 0, hi = n_wg;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ unsigned long long wave_max64(unsigned long long x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const unsigned long long o = shfl_xor64(x, m);
        x = o > x ? o : x;
    }
    return x;
}

__device__ __forceinline__ unsigned long long wave_min64(unsigned long long x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const unsigned long long o = shfl_xor64(x, m);
        x = o < x ? o : x;
    }
    return x;
}

__device__ __forceinline__ unsigned long long wave_or64(unsigned long long x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x |= shfl_xor64(x, m);
    return x;
}

// The last store of a finish kernel to the host copy: the call's sequence
// number, after a system-scope fence.
__device__ __forceinline__ void publish_done(const FinishArgs &f)
{
    __threadfence_system();
    *reinterpret_cast<volatile unsigned long long *>(&f.res_host->done_seq) = f.seq;
}

// STAGED: the workgroups' keys are copied to LDS first (when they fit).
template <bool STAGED>
__global__ void __launch_bounds__(kFinWaves * 64) finish_small_kernel(const FinishArgs f, const FastConst fc)
{
    extern __shared__ K128 lkeys[];   // [n_wg][k] the workgroups' best canonical keys, sorted
    const K128 *ckeys = STAGED ? lkeys : f.wg_top;
    __shared__ unsigned long long s_red[8][kFinWaves];
    __shared__ K128 klst[kFinWaves * 64];
    __shared__ K128 s_floor;
    constexpr int W = kFinWaves;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k = f.top_k, n_wg = f.n_wg;
    DevResult *R = f.res;

    // ---- one round trip: every workgroup's keys (all loads in flight
    // together, then staged in LDS) and its records
    const uint32_t n_cand = (uint32_t)n_wg * (uint32_t)k;
    constexpr int kCpt = 8;   // keys per thread per pass
    for (uint32_t base = 0; STAGED && base < n_cand; base += kCpt * blockDim.x) {
        K128 v[kCpt];
#pragma unroll
        for (int q = 0; q < kCpt; q++) {
            const uint32_t t = base + q * blockDim.x + tid;
            v[q] = t < n_cand ? f.wg_top[t] : K128{0ull, 0ull};
        }
#pragma unroll
        for (int q = 0; q < kCpt; q++) {
            const uint32_t t = base + q * blockDim.x + tid;
            if (t < n_cand) lkeys[t] = v[q];
        }
    }
    // counts, certification entries (offered, kept, found feasible), the
    // wall-clock span, status bits and the largest unevaluated upper bound
    unsigned long long nv = 0, nf = 0, nw = 0, ovf = 0, nfc = 0, t0 = ~0ull, t1 = 0, st = 0, rest = 0;
    if (tid < n_wg) {
        const unsigned long long *r = f.wg_rec + 8 * (uint64_t)tid;
        const unsigned long long off = r[0];
        ovf = off > f.seg_cap ? 1u : 0u;
        nw = off > f.seg_cap ? f.seg_cap : off;
        t0 = r[1];
        t1 = r[2];
        st = r[3] >> 32;
        rest = r[3] & 0xFFFFFFFFull;
        nfc = r[4];
        nv = f.wg_counts[2 * (uint64_t)tid];
        nf = f.wg_counts[2 * (uint64_t)tid + 1];
    }
    nv = wave_sum64(nv);
    nf = wave_sum64(nf);
    nw = wave_sum64(nw);
    ovf = wave_sum64(ovf);
    nfc = wave_sum64(nfc);
    t0 = wave_min64(t0);
    t1 = wave_max64(t1);
    rest = wave_max64(rest);
    st = wave_or64(st);
    if (lane == 0) {
        s_red[0][wv] = nv;
        s_red[1][wv] = nf;
        s_red[2][wv] = nw;
        s_red[3][wv] = ovf;
        s_red[4][wv] = nfc;
        s_red[5][wv] = t0;
        s_red[6][wv] = t1;
        s_red[7][wv] = (rest << 32) | st;
    }
    __syncthreads();
    unsigned long long tnv = 0, tnf = 0, tnw = 0, tovf = 0, tnfc = 0, tt0 = ~0ull, tt1 = 0, trest = 0, tst = 0;
    for (int w = 0; w < W; w++) {
        tnv += s_red[0][w];
        tnf += s_red[1][w];
        tnw += s_red[2][w];
        tovf += s_red[3][w];
        tnfc += s_red[4][w];
        tt0 = s_red[5][w] < tt0 ? s_red[5][w] : tt0;
        tt1 = s_red[6][w] > tt1 ? s_red[6][w] : tt1;
        const unsigned long long rs = s_red[7][w] >> 32;
        trest = rs > trest ? rs : trest;
        tst |= s_red[7][w] & 0xFFFFFFFFull;
    }
    if (tovf || tnw > f.work_cap) {
        if (tid == 0) {
            R->status = kStatWorkOverflow;
            R->n_work = (unsigned long long)f.work_cap + 1;
            if (f.res_host) {
                f.res_host->status = kStatWorkOverflow;
                f.res_host->n_work = (unsigned long long)f.work_cap + 1;
                publish_done(f);
            }
        }
        return;
    }

    // ---- a lower bound of the k-th largest key: the k-th largest of up to
    // 64 maxima of the workgroups' first (largest) keys, distinct candidates
    if (wv == 0) {
        K128 m = {0ull, 0ull};
        for (int g = lane; g < n_wg; g += 64) {
            const K128 x = ckeys[(uint32_t)g * (uint32_t)k];
            if (gt128(x, m)) m = x;
        }
        const K128 srt = sort128_desc(m, lane);
        const K128 fk = {readlane64(srt.hi, k - 1), readlane64(srt.lo, k - 1)};
        if (lane == 0) s_floor = fk;
    }
    __syncthreads();
    const K128 floor_key = s_floor;

    // ---- the exact top-k: the keys at or above the bound, offered per wave,
    // the waves' lists merged in a tree
    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    for (uint32_t b0 = (uint32_t)wv * 64; b0 < n_cand; b0 += W * 64) {
        const uint32_t t = b0 + lane;
        K128 mine = {0ull, 0ull};
        if (t < n_cand) {
            const K128 x = ckeys[t];
            if (!gt128(floor_key, x)) mine = x;
        }
        list128_offer_many(slot, mine, lane, k, thr);
    }
    klst[wv * 64 + lane] = key_if(lane < k, slot);
#pragma unroll
    for (int h = W / 2; h >= 1; h >>= 1) {
        __syncthreads();
        if (wv < h) {
            list128_merge_sorted(slot, klst[(wv + h) * 64 + lane], lane, k, thr);
            if (h > 1) klst[wv * 64 + lane] = slot;
        }
    }
    if (wv == 0) {
        const int n_top = __popcll(__ballot(lane < k && nz128(slot)));
        const uint64_t kth_hi = readlane64(slot.hi, k - 1);
        const bool ok = lane < n_top;
        const unsigned long long tidx = ok ? ~slot.lo : ~0ull;
        const double tJ = ok ? unord_f64(slot.hi) : -INFINITY;
        R->top_idx[lane] = tidx;
        R->top_J[lane] = tJ;
        if (f.res_host) {
            f.res_host->top_idx[lane] = tidx;
            f.res_host->top_J[lane] = tJ;
        }
        if (lane == 0) {
            // every sure-feasible configuration not evaluated has an upper
            // bound U <= the largest first unevaluated list bound: exact when
            // the k-th canonical J exceeds it (or nothing is unevaluated);
            // otherwise the fallback collects every U >= C_k (every
            // sure-feasible configuration when fewer than k were found)
            const double restU = trest ? (double)unord_f32((uint32_t)trest) : -INFINITY;
            unsigned stat = (unsigned)tst;
            double Ck = -INFINITY;
            bool verified;
            if (n_top >= k) {
                Ck = unord_f64(kth_hi);
                verified = Ck > restU;
            } else {
                verified = trest == 0ull;
            }
            if (verified) stat |= kStatVerified;
            R->n_vram = tnv;
            R->n_feas_sure = tnf;
            R->n_work = tnw;
            R->n_collect = 0;
            R->n_feas_cert = tnfc;
            R->n_cand = 0;
            R->status = stat;
            R->n_top = n_top;
            R->theta = Ck;
            R->eJ = bound_eJ(fc, f.omega);
            R->tail_U = restU;
            R->check_max_dJ = 0.0;
            R->ck_cand = Ck;
            R->fast_ticks = tt1 > tt0 ? tt1 - tt0 : 0ull;
            if (DevResult *H = f.res_host) {
                // the host reads this copy after the sequence number appears
                H->n_vram = tnv;
                H->n_feas_sure = tnf;
                H->n_work = tnw;
                H->n_collect = 0;
                H->n_feas_cert = tnfc;
                H->n_cand = 0;
                H->status = stat;
                H->n_top = n_top;
                H->theta = Ck;
                H->tail_U = restU;
                H->ck_cand = Ck;
                H->fast_ticks = R->fast_ticks;
            }
        }
        if (f.res_host) {
            // every lane's stores to the host copy are ordered before the
            // sequence number the host waits for
            __threadfence_system();
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) publish_done(f);
        }
    }
}

hipError_t launch_finish_small(const FinishArgs &f, const FastConst &fc, hipStream_t s)
{
    if (f.n_wg < 1 || f.n_wg >= kFinWaves * 64 || f.top_k < 1 || f.top_k > 64) return hipErrorInvalidValue;
    // the keys are staged in LDS up to 128 KiB (8192 keys), read from global
    // memory beyond
    const size_t lds = (size_t)f.n_wg * f.top_k * sizeof(K128);
    if (lds <= 131072) {
        hipError_t e = ensure_dyn_lds((const void *)finish_small_kernel<true>, lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(finish_small_kernel<true>, dim3(1), dim3(kFinWaves * 64), lds, s, f, fc);
    } else {
        hipLaunchKernelGGL(finish_small_kernel<false>, dim3(1), dim3(kFinWaves * 64), 0, s, f, fc);
    }
    return hipGetLastError();
}

// The fallback's certification list: segment g's first min(offered, seg_cap)
// entries at the exclusive prefix of those lengths.  Dynamic LDS: [n_wg + 1].
__global__ void __launch_bounds__(1024) gather_small_kernel(const GatherArgs a)
{
    extern __shared__ uint32_t woff[];
    if (threadIdx.x == 0) {
        uint32_t o = 0;
        for (int g = 0; g < a.n_wg; g++) {
            woff[g] = o;
            const unsigned long long off = a.wg_rec[8 * (uint64_t)g];
            o += (uint32_t)(off > a.seg_cap ? a.seg_cap : off);
        }
        woff[a.n_wg] = o;
    }
    __syncthreads();
    const uint32_t n = woff[a.n_wg];
    for (uint32_t e = threadIdx.x; e < n; e += blockDim.x) {
        const int g = seg_of(woff, a.n_wg, e);
        const uint64_t at = (uint64_t)g * a.seg_cap + (e - woff[g]);
        a.work_out[e] = a.seg[at];
        a.work_J_out[e] = a.seg_J[at];
    }
}

hipError_t launch_gather_small(const GatherArgs &g, hipStream_t s)
{
    if (g.n_wg < 1 || g.n_wg >= 65536) return hipErrorInvalidValue;
    const size_t lds = ((size_t)g.n_wg + 1) * 4;
    hipError_t e = ensure_dyn_lds((const void *)gather_small_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(gather_small_kernel, dim3(1), dim3(1024), lds, s, g);
    return hipGetLastError();
}

}  // namespace mfi
