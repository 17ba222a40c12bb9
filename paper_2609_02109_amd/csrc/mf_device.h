// Device helpers shared by the kernels of libmf (HIP translation units only).
#pragma once

#include "mf_internal.h"

namespace mfi {

// Bound on |fast J - canonical J| for objective weights omega: each model's
// throughput bound, plus the rounding of the fp32 fma chain over N models
// (gamma_N relative to sum |omega_i thr_i|) and of the fp64 canonical chain.
__device__ inline double bound_eJ(const FastConst &fc, const float *omega)
{
    const int N = fc.n_models;
    const double g = N * 0x1p-24 / (1.0 - N * 0x1p-24);
    double e = 0.0, m = 0.0;
    for (int i = 0; i < N; i++) {
        const double w = fabs((double)omega[i]);
        e += w * (fc.bound_thr[i] + g * (fc.mag_thr[i] + fc.bound_thr[i]));
        m += w * fc.mag_thr[i];
    }
    return (e + m * 0x1p-48) * (1.0 + 0x1p-20) + 1e-30;
}

// Fast-path term of the full utility (Section II, Eq. 3) for one model.
// r0 = (fmin, fmax, 1/(fmax - fmin) in fp32, Q), r1 = (variant bits, reload
// cost); thr is the fast fp32 throughput and e_thr a bound on its distance
// from the canonical one.  Returns the term c (omega Q f - alpha c eta -
// beta max(0, tau + delta - f)^2 in fp32), e with |c - canonical term| <= e,
// mag >= |c| (for the rounding of the sum over models), and the floor
// decision f >= tau: pass / fail when the bound settles it.
struct Eq3Term {
    float c, e, mag;
    bool pass, fail;
};

__device__ __forceinline__ Eq3Term eq3_term(const float4 r0, const float4 r1, float thr, float e_thr, float omega,
                                            float tau, int prev, float alpha, float beta, float delta)
{
    const float fmin = r0.x, inv = r0.z, Q = r0.w;
    const int var = __float_as_int(r1.x);
    const float num = thr - fmin;
    const float f = num * inv;
    // the throughput error through 1/range, and the fp32 rounding of the
    // subtraction, of 1/range and of the product (3 u relative < 2^-22)
    const float e_f = (e_thr + fabsf(num) * 0x1p-22f) * fabsf(inv) * 1.001f + 1e-30f;
    const float w = omega * Q;
    const float P = (prev >= 0 && var != prev) ? alpha * r1.y : 0.f;
    Eq3Term t;
    float pen = 0.f, epen = 0.f;
    if (tau == -INFINITY) {
        t.pass = true;
        t.fail = false;
    } else {
        const float slack = e_f + (fabsf(f) + fabsf(tau)) * 0x1p-22f;
        t.pass = f - slack >= tau;
        t.fail = f + slack < tau;
        const float d = (tau + delta) - f;
        const float e_d = e_f + (fabsf(tau) + fabsf(delta) + fabsf(f)) * 0x1p-22f;
        const float dp = d > 0.f ? d : 0.f;
        pen = beta * (dp * dp);
        // max(0, d)^2 moves by at most (2 max(0, d) + e_d) e_d when d moves by e_d
        epen = beta * (2.f * dp + e_d) * e_d;
    }
    const float wf = w * f;
    t.c = (wf - P) - pen;
    t.mag = fabsf(wf) + P + pen;
    t.e = fabsf(w) * e_f + epen + t.mag * 0x1p-20f + 1e-30f;
    return t;
}

// Fast-path sigmoid in fp32.  Against the exact sigmoid of the same input its
// error stays below 2^-21: the exponential's relative error e (from rounding
// the scaled argument, |y| 2^-24, and the instruction's own) moves the
// result by s (1 - s) e <= max(|y| e^-|y|) 2^-24 + 2^-23, and the add and
// divide round twice more.  The bound used for it is 2^-20.
__device__ __forceinline__ float sigmoid_f32(float y) { return 1.0f / (1.0f + __expf(-y)); }

// relu of a finite fp32 value as one integer max: negative values (and -0)
// have a negative bit pattern and map to +0, the rest are unchanged
__device__ __forceinline__ float relu_f32(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

__device__ __forceinline__ uint32_t ord_f32(float f)
{
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ unsigned long long readlane64(unsigned long long x, int src)
{
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)x, src);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), src);
    return ((unsigned long long)hi << 32) | lo;
}

// x of lane - 1 (lane 0: unspecified), by the DPP whole-wave shift; the
// whole wave must be active.
__device__ __forceinline__ double readlane_f64(double x, int src)
{
    return __longlong_as_double((long long)readlane64((unsigned long long)__double_as_longlong(x), src));
}

__device__ __forceinline__ unsigned long long shfl_up1_64(unsigned long long x)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)x, 0x138, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(x >> 32), 0x138, 0xF, 0xF, false);
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ unsigned long long wave_sum64(unsigned long long x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const uint32_t lo = __shfl_xor((int)(uint32_t)x, m);
        const uint32_t hi = __shfl_xor((int)(uint32_t)(x >> 32), m);
        x += ((unsigned long long)hi << 32) | lo;
    }
    return x;
}

// A wave's descending list of up to 64*NS distinct 64-bit keys in registers:
// slot q = j*64 + lane lives in s[j].  thr is the smallest key while the
// list is full (kp entries), 0 before.  Keys of 0 are never inserted.
template <int NS>
struct WaveList {
    unsigned long long s[NS];
    unsigned long long thr;
};

template <int NS>
__device__ __forceinline__ void wl_init(WaveList<NS> &L)
{
#pragma unroll
    for (int j = 0; j < NS; j++) L.s[j] = 0ull;
    L.thr = 0ull;
}

template <int NS>
__device__ __forceinline__ void wl_insert(WaveList<NS> &L, unsigned long long nk, int lane, int kp)
{
    int pos = 0;
#pragma unroll
    for (int j = 0; j < NS; j++) pos += __popcll(__ballot(j * 64 + lane < kp && L.s[j] > nk));
    unsigned long long prev[NS];
#pragma unroll
    for (int j = 0; j < NS; j++) {
        prev[j] = shfl_up1_64(L.s[j]);
        if (j > 0) {
            const unsigned long long last = readlane64(L.s[j - 1], 63);
            if (lane == 0) prev[j] = last;
        }
    }
#pragma unroll
    for (int j = 0; j < NS; j++) {
        const int q = j * 64 + lane;
        if (q < kp) L.s[j] = q < pos ? L.s[j] : (q == pos ? nk : prev[j]);
    }
    const int t = kp - 1;
    unsigned long long th = 0ull;
#pragma unroll
    for (int j = 0; j < NS; j++)
        if (t / 64 == j) th = readlane64(L.s[j], t % 64);
    L.thr = th;
}

__device__ __forceinline__ unsigned long long shfl64(unsigned long long x, int src)
{
    const uint32_t lo = __shfl((int)(uint32_t)x, src);
    const uint32_t hi = __shfl((int)(uint32_t)(x >> 32), src);
    return ((unsigned long long)hi << 32) | lo;
}

// x of lane (lane ^ m), m in {1, 2, 4, 8, 16, 32} (a constant after
// unrolling): DPP moves within rows of 16 lanes (quad permutations, the
// half-row mirror, a rotation by 8) and the gfx950 permlane swaps across
// rows, all VALU operations.  The whole wave must be active.
__device__ __forceinline__ uint32_t xor_lane32(uint32_t x, int m)
{
    switch (m) {
        case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
        case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
        case 4: {   // half-row mirror, then quad_perm [3,2,1,0]
            const int h = __builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, false);
            return (uint32_t)__builtin_amdgcn_mov_dpp(h, 0x1B, 0xF, 0xF, false);
        }
        case 8: return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x128, 0xF, 0xF, false);  // row_ror:8
        case 16: {
            const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
            return (__lane_id() & 16) ? r[0] : r[1];
        }
        default: {
            const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
            return (__lane_id() & 32) ? r[0] : r[1];
        }
    }
}

__device__ __forceinline__ unsigned long long shfl_xor64(unsigned long long x, int m)
{
    const uint32_t lo = xor_lane32((uint32_t)x, m);
    const uint32_t hi = xor_lane32((uint32_t)(x >> 32), m);
    return ((unsigned long long)hi << 32) | lo;
}

// x of lane 63 - lane: mirror within rows of 16, then swap the rows (lane ^ 48).
__device__ __forceinline__ unsigned long long reverse64(unsigned long long x)
{
    uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)x, 0x140, 0xF, 0xF, false);
    uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(x >> 32), 0x140, 0xF, 0xF, false);
    lo = xor_lane32(xor_lane32(lo, 16), 32);
    hi = xor_lane32(xor_lane32(hi, 16), 32);
    return ((unsigned long long)hi << 32) | lo;
}

// Compare-exchange with the lane j apart: the lower lane of the pair keeps
// the larger key when `desc`, the smaller otherwise.
__device__ __forceinline__ unsigned long long cx_lane(unsigned long long x, int j, int lane, bool desc)
{
    const unsigned long long o = shfl_xor64(x, j);
    const bool keep_max = ((lane & j) == 0) == desc;
    const unsigned long long hi = x > o ? x : o, lo = x > o ? o : x;
    return keep_max ? hi : lo;
}

// Merge a sorted list b (the layout of WaveList, zeros past its end) into L:
// L keeps the kp largest keys of both, sorted.  With both sides descending,
// the elementwise max of L and b reversed holds the 64 NS largest keys of the
// union as a bitonic sequence; the half-cleaner cascade sorts it.
template <int NS>
__device__ __forceinline__ void wl_merge_sorted(WaveList<NS> &L, const unsigned long long (&b)[NS], int lane,
                                                int kp)
{
    unsigned long long c[NS];
#pragma unroll
    for (int j = 0; j < NS; j++) {
        const unsigned long long r = reverse64(b[NS - 1 - j]);
        c[j] = L.s[j] > r ? L.s[j] : r;
    }
    if constexpr (NS == 2) {   // stride 64: the two registers of a lane
        const unsigned long long hi = c[0] > c[1] ? c[0] : c[1], lo = c[0] > c[1] ? c[1] : c[0];
        c[0] = hi;
        c[1] = lo;
    }
#pragma unroll
    for (int j = 32; j > 0; j >>= 1)
#pragma unroll
        for (int r = 0; r < NS; r++) c[r] = cx_lane(c[r], j, lane, true);
    unsigned long long th = 0ull;
#pragma unroll
    for (int j = 0; j < NS; j++) {
        L.s[j] = j * 64 + lane < kp ? c[j] : 0ull;
        if ((kp - 1) / 64 == j) th = readlane64(L.s[j], (kp - 1) % 64);
    }
    L.thr = th;
}

// Tree merge of a workgroup's per-wave lists: list w sits at lst + w stride
// (slot q at q, zeros from kp on).  WAVES is a power of two; the result ends
// in wave 0's L.  Every thread of the workgroup calls this.
template <int NS, int WAVES>
__device__ __forceinline__ void wl_tree_merge(WaveList<NS> &L, unsigned long long *lst, int stride, int wv,
                                              int lane, int kp)
{
#pragma unroll
    for (int h = WAVES / 2; h >= 1; h >>= 1) {
        __syncthreads();
        if (wv < h) {
            unsigned long long b[NS];
#pragma unroll
            for (int j = 0; j < NS; j++) b[j] = j * 64 + lane < kp ? lst[(wv + h) * stride + j * 64 + lane] : 0ull;
            wl_merge_sorted(L, b, lane, kp);
            if (h > 1)
#pragma unroll
                for (int j = 0; j < NS; j++)
                    if (j * 64 + lane < kp) lst[wv * stride + j * 64 + lane] = L.s[j];
        }
    }
}

// Offer every lane's key (0 = none) to the list, one key at a time (the
// form for hot loops: it holds no extra registers).
template <int NS>
__device__ __forceinline__ void wl_offer(WaveList<NS> &L, unsigned long long mykey, int lane, int kp)
{
    unsigned long long cm = __ballot(mykey > L.thr);
    while (cm) {
        const int src = __ffsll((long long)cm) - 1;
        cm &= cm - 1;
        const unsigned long long nk = readlane64(mykey, src);
        if (nk > L.thr) wl_insert(L, nk, lane, kp);
    }
}

// wl_offer for one-register lists when many keys may pass at once (a list
// still filling): above four passing keys the wave's keys are sorted
// descending by a bitonic network and merged into the list in one step.
__device__ __forceinline__ void wl_offer_many(WaveList<1> &L, unsigned long long mykey, int lane, int kp)
{
    const bool pass = mykey > L.thr;
    if (__popcll(__ballot(pass)) <= 4) {
        wl_offer(L, mykey, lane, kp);
        return;
    }
    unsigned long long x = pass ? mykey : 0ull;
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) x = cx_lane(x, j, lane, (lane & k) == 0);
    const unsigned long long b[1] = {x};
    wl_merge_sorted(L, b, lane, kp);
}

// Selection on 128-bit keys (K128): a wave keeps the best k <= 64 keys
// sorted, slot lane in lane (thr: the k-th key once the list is full, 0
// before).
__device__ __forceinline__ bool gt128(const K128 &x, const K128 &y)
{
    return x.hi > y.hi || (x.hi == y.hi && x.lo > y.lo);
}
__device__ __forceinline__ bool nz128(const K128 &x) { return (x.hi | x.lo) != 0ull; }
__device__ __forceinline__ K128 key_if(bool c, const K128 &x)
{
    return K128{c ? x.hi : 0ull, c ? x.lo : 0ull};
}

__device__ __forceinline__ uint64_t ord_f64(double x)
{
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    return (b & 0x8000000000000000ull) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double unord_f64(uint64_t o)
{
    const uint64_t b = (o & 0x8000000000000000ull) ? (o & 0x7FFFFFFFFFFFFFFFull) : ~o;
    return __longlong_as_double((long long)b);
}

__device__ __forceinline__ void list128_offer(K128 &slot, const K128 &mine, int lane, int k, K128 &thr)
{
    unsigned long long cm = __ballot(nz128(mine) && gt128(mine, thr));
    while (cm) {
        const int src = __ffsll((long long)cm) - 1;
        cm &= cm - 1;
        const K128 nk = {readlane64(mine.hi, src), readlane64(mine.lo, src)};
        if (!gt128(nk, thr)) continue;
        const int pos = __popcll(__ballot(lane < k && gt128(slot, nk)));
        const K128 prev = {shfl_up1_64(slot.hi), shfl_up1_64(slot.lo)};
        if (lane < k) {   // per field: a select of whole structs goes through scratch
            slot.hi = lane < pos ? slot.hi : (lane == pos ? nk.hi : prev.hi);
            slot.lo = lane < pos ? slot.lo : (lane == pos ? nk.lo : prev.lo);
        }
        thr = {readlane64(slot.hi, k - 1), readlane64(slot.lo, k - 1)};
    }
}

__device__ __forceinline__ K128 shfl_xor128(const K128 &x, int m) { return {shfl_xor64(x.hi, m), shfl_xor64(x.lo, m)}; }

// Compare-exchange of 128-bit keys with the lane m apart (the lower lane
// of the pair keeps the larger key when desc).
__device__ __forceinline__ K128 cx128(const K128 &x, int m, int lane, bool desc)
{
    const K128 o = shfl_xor128(x, m);
    const bool xg = gt128(x, o);
    const bool keep_max = ((lane & m) == 0) == desc;
    const bool take_x = keep_max == xg;
    return K128{take_x ? x.hi : o.hi, take_x ? x.lo : o.lo};
}

// list128_offer when many keys may pass at once: above four passing keys the
// wave's keys are sorted descending (bitonic) and merged into the list (the
// elementwise maximum of the list and the sorted keys reversed is bitonic;
// six half-cleaner stages sort it); the list keeps its k best.
// Bitonic sort of one key per lane, descending (lane 0 the largest).
__device__ __forceinline__ K128 sort128_desc(K128 x, int lane)
{
#pragma unroll
    for (int kk = 2; kk <= 64; kk <<= 1)
#pragma unroll
        for (int j = kk >> 1; j > 0; j >>= 1) x = cx128(x, j, lane, (lane & kk) == 0);
    return x;
}

__device__ __forceinline__ void list128_offer_many(K128 &slot, const K128 &mine, int lane, int k, K128 &thr)
{
    const bool pass = nz128(mine) && gt128(mine, thr);
    if (__popcll(__ballot(pass)) <= 4) {
        list128_offer(slot, mine, lane, k, thr);
        return;
    }
    const K128 x = sort128_desc(key_if(pass, mine), lane);
    const K128 r = {reverse64(x.hi), reverse64(x.lo)};
    K128 c = gt128(slot, r) ? slot : r;
#pragma unroll
    for (int j = 32; j > 0; j >>= 1) c = cx128(c, j, lane, true);
    slot = key_if(lane < k, c);
    thr = {readlane64(slot.hi, k - 1), readlane64(slot.lo, k - 1)};
}

// Merge another wave's sorted list b (slot lane, zeros past its end) into
// this wave's list.
__device__ __forceinline__ void list128_merge_sorted(K128 &slot, const K128 &b, int lane, int k, K128 &thr)
{
    const K128 r = {reverse64(b.hi), reverse64(b.lo)};
    K128 c = gt128(slot, r) ? slot : r;
#pragma unroll
    for (int j = 32; j > 0; j >>= 1) c = cx128(c, j, lane, true);
    slot = key_if(lane < k, c);
    thr = {readlane64(slot.hi, k - 1), readlane64(slot.lo, k - 1)};
}

// Append flagged lanes' values to a device list; the counter keeps counting
// past cap so the host can see an overflow.
__device__ __forceinline__ unsigned long long list_reserve(bool flag, int lane, unsigned long long *count,
                                                           unsigned long long &slot_out)
{
    const unsigned long long m = __ballot(flag);
    if (m == 0) return 0;
    unsigned long long base = 0;
    if (lane == 0) base = atomicAdd(count, (unsigned long long)__popcll(m));
    base = readlane64(base, 0);
    slot_out = base + (unsigned long long)__popcll(m & ((1ull << lane) - 1ull));
    return m;
}

__device__ __forceinline__ void list_append(bool flag, uint32_t value, int lane, unsigned long long *count,
                                            uint32_t *list, uint32_t cap)
{
    unsigned long long slot = 0;
    if (list_reserve(flag, lane, count, slot) && flag && slot < cap) list[slot] = value;
}

__device__ __forceinline__ void work_append(bool flag, unsigned long long entry, float fj, int lane,
                                            unsigned long long *count, unsigned long long *list, float *list_J,
                                            uint32_t cap)
{
    unsigned long long slot = 0;
    if (list_reserve(flag, lane, count, slot) && flag && slot < cap) {
        list[slot] = entry;
        list_J[slot] = fj;
    }
}

// A wave's certification entries buffered in registers, one per lane
// (lanes [0, n) hold entries; n is wave-uniform), written to the device list
// 64 at a time: one reservation and contiguous stores instead of a partial
// line per append.  The list's order carries no meaning.
struct WorkBuf {
    unsigned long long e;
    float j;
    int n;
};

__device__ __forceinline__ void wb_flush(WorkBuf &b, int lane, unsigned long long *count, unsigned long long *list,
                                         float *list_J, uint32_t cap)
{
    if (b.n == 0) return;
    unsigned long long base = 0;
    if (lane == 0) base = atomicAdd(count, (unsigned long long)b.n);
    base = readlane64(base, 0);
    if (lane < b.n) {
        const unsigned long long slot = base + (unsigned long long)lane;
        if (slot < cap) {
            list[slot] = b.e;
            list_J[slot] = b.j;
        }
    }
    b.n = 0;
}

// Append the flagged lanes' (entry, fj).  Each flagged lane's values move to
// buffer lane n + (its rank among the flagged lanes); the other lanes move to
// the remaining lanes, so the move is a permutation of the wave.
__device__ __forceinline__ void wb_append(WorkBuf &b, bool flag, unsigned long long entry, float fj, int lane,
                                          unsigned long long *count, unsigned long long *list, float *list_J,
                                          uint32_t cap)
{
    const unsigned long long m = __ballot(flag);
    if (m == 0ull) return;
    const int c = __popcll(m);
    if (b.n + c > 64) wb_flush(b, lane, count, list, list_J, cap);
    const unsigned long long lt = (1ull << lane) - 1ull;
    const int r = flag ? __popcll(m & lt) : c + __popcll(~m & lt);
    const int dst = ((b.n + r) & 63) * 4;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_permute(dst, (int)(uint32_t)entry);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_permute(dst, (int)(uint32_t)(entry >> 32));
    const uint32_t jj = (uint32_t)__builtin_amdgcn_ds_permute(dst, __float_as_int(fj));
    if (lane >= b.n && lane < b.n + c) {
        b.e = (unsigned long long)lo | ((unsigned long long)hi << 32);
        b.j = __int_as_float((int)jj);
    }
    b.n += c;
}

// Smallest float >= x (x finite double).
__device__ __forceinline__ float f32_up(double x)
{
    float f = (float)x;
    if ((double)f < x) f = __uint_as_float(f >= 0.f ? __float_as_uint(f) + 1u
                                                     : (f == -0.f ? 1u : __float_as_uint(f) - 1u));
    return f;
}

__device__ __forceinline__ float unord_f32(uint32_t o)
{
    const uint32_t b = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(b);
}

}  // namespace mfi
