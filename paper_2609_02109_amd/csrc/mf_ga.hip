// Genetic-algorithm scheduler (Section IV-C) on the GPU.
//
// Per generation two launches: the fitness of every individual of every
// scenario (the canonical fp64 surrogate chain, so every tournament compares
// exactly the values the results are defined by: one lane per individual for
// large populations, one workgroup per individual for small ones), then the
// operators, 64 parent pairs per workgroup: elitism (slot 0), tournaments of
// k draws with replacement, uniform crossover, per-gene mutation, repair of
// VRAM-infeasible children from the feasible list.
//
// Random draws: Philox4x64-10 (Salmon et al., SC'11), key (seed, 0), counter
// (item, generation, scenario, purpose), one 64-bit word per draw;
// uniform(r) = (r >> 11) 2^-53, int(r, n) = ((r >> 32) n) >> 32.  Counter
// assignment (item = pair q for selection / crossover, child slot j for
// mutation / repair, slot for initialisation):
//   INIT 1 (gen 0), SEL 2 + m/4 (draw m of 2k), CX 8, SWAP 9 + i/4 (gene i),
//   MUT 16 + w/4 (word w = 2i: mutate?, 2i+1: new value), REP 32.
#include "mf_canon.h"

namespace mfi {

enum { kPInit = 1, kPSel = 2, kPCx = 8, kPSwap = 9, kPMut = 16, kPRep = 32 };

struct Philox4 {
    uint64_t w[4];
};

// The 128-bit product a b: its high and low 64 bits from four 32 x 32 -> 64
// multiply-adds (no partial sum overflows 64 bits).
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t b, uint64_t &hi, uint64_t &lo)
{
    const uint64_t a0 = (uint32_t)a, a1 = a >> 32, b0 = (uint32_t)b, b1 = b >> 32;
    const uint64_t p00 = a0 * b0;
    const uint64_t t1 = a0 * b1 + (p00 >> 32);
    const uint64_t t2 = a1 * b0 + (t1 & 0xFFFFFFFFull);
    hi = a1 * b1 + (t1 >> 32) + (t2 >> 32);
    lo = (t2 << 32) | (p00 & 0xFFFFFFFFull);
}

__device__ __forceinline__ Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                                 uint64_t k1)
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        if (r) { k0 += W0; k1 += W1; }
        uint64_t h0, l0, h1, l1;
        mulhilo64(M0, c0, h0, l0);
        mulhilo64(M1, c2, h1, l1);
        const uint64_t y0 = h1 ^ c1 ^ k0, y2 = h0 ^ c3 ^ k1;
        c0 = y0; c1 = l1; c2 = y2; c3 = l0;
    }
    return Philox4{{c0, c1, c2, c3}};
}

__device__ __forceinline__ uint64_t ga_draw(uint64_t seed, uint64_t item, uint64_t gen, uint64_t scen,
                                            uint64_t purpose, int word)
{
    const Philox4 p = philox4x64_10(item, gen, scen, purpose, seed, 0);
    return p.w[word & 3];
}
__device__ __forceinline__ double ga_uni(uint64_t r) { return (double)(r >> 11) * 0x1p-53; }
__device__ __forceinline__ uint64_t ga_below(uint64_t r, uint64_t n) { return ((r >> 32) * n) >> 32; }

// ---------------------------------------------------------------- feasible list

// Mixed-radix digits of a joint index, model 0 most significant (the decode of
// Eq. 1's configuration vector); 32-bit divisions when the space fits 32 bits.
__device__ __forceinline__ void ga_digits(const GAConst &c, uint64_t idx, int32_t *d)
{
    if (c.space <= 0x100000000ull) {
        uint32_t x = (uint32_t)idx;
        for (int i = c.N - 1; i >= 0; i--) {
            const uint32_t k = (uint32_t)c.K[i], q = x / k;
            d[i] = (int32_t)(x - q * k);
            x = q;
        }
    } else {
        for (int i = c.N - 1; i >= 0; i--) {
            d[i] = (int32_t)(idx % (uint64_t)c.K[i]);
            idx /= (uint64_t)c.K[i];
        }
    }
}

__device__ __forceinline__ bool vram_feasible(const GAConst &c, uint64_t idx)
{
    // fp32 sum of the VRAM column in model order (the aggregate slot's value)
    int32_t d[kMaxN];
    ga_digits(c, idx, d);
    float s = 0.f;
    for (int i = 0; i < c.N; i++) s = s + c.features[(int64_t)(c.opt_off[i] + d[i]) * c.L + c.vram_col];
    return (double)s <= (double)c.vram_cap;
}

constexpr int kFlBlock = 256;

__global__ void __launch_bounds__(kFlBlock) fl_count_kernel(const GAConst c, uint32_t *blk_count)
{
    const uint64_t idx = (uint64_t)blockIdx.x * kFlBlock + threadIdx.x;
    const bool f = idx < c.space && vram_feasible(c, idx);
    const int n = __syncthreads_count(f);
    if (threadIdx.x == 0) blk_count[blockIdx.x] = (uint32_t)n;
}

// exclusive scan of the block counts (one workgroup); total to *n_fl
__global__ void __launch_bounds__(1024) fl_scan_kernel(const uint32_t *blk_count, uint64_t n_blk, uint64_t *blk_off,
                                                       unsigned long long *n_fl)
{
    __shared__ uint64_t part[1024];
    __shared__ uint64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (uint64_t base = 0; base < n_blk; base += 1024) {
        const uint64_t i = base + threadIdx.x;
        const uint64_t v = i < n_blk ? blk_count[i] : 0;
        part[threadIdx.x] = v;
        __syncthreads();
        for (int o = 1; o < 1024; o <<= 1) {
            const uint64_t t = threadIdx.x >= (unsigned)o ? part[threadIdx.x - o] : 0;
            __syncthreads();
            part[threadIdx.x] += t;
            __syncthreads();
        }
        if (i < n_blk) blk_off[i] = carry + part[threadIdx.x] - v;
        __syncthreads();
        if (threadIdx.x == 1023) carry += part[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0) *n_fl = carry;
}

__global__ void __launch_bounds__(kFlBlock) fl_write_kernel(const GAConst c, const uint64_t *blk_off, uint32_t *fl)
{
    __shared__ uint32_t wcount[kFlBlock / 64];
    const uint64_t idx = (uint64_t)blockIdx.x * kFlBlock + threadIdx.x;
    const bool f = idx < c.space && vram_feasible(c, idx);
    const unsigned long long m = __ballot(f);
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    if (lane == 0) wcount[wv] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t before = 0;
    for (int w = 0; w < wv; w++) before += wcount[w];
    const uint32_t rank = before + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
    if (f) fl[blk_off[blockIdx.x] + rank] = (uint32_t)idx;
}

// ---------------------------------------------------------------- population

__global__ void ga_init_kernel(uint64_t seed, int S, int P, const uint32_t *fl, const unsigned long long *n_fl,
                               uint64_t *pop, double *best_J, uint64_t *best_idx)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)S * P) return;
    const int s = (int)(t / P), j = (int)(t % P);
    // no VRAM-feasible configuration: index 0 throughout (every fitness is
    // -inf, the best stays unset and the final population reads all ones)
    const unsigned long long nf = *n_fl;
    pop[t] = nf ? fl[ga_below(ga_draw(seed, (uint64_t)j, 0, (uint64_t)s, kPInit, 0), nf)] : 0;
    if (j == 0) {
        best_J[s] = -INFINITY;
        best_idx[s] = ~0ull;
    }
}

// Canonical fp64 fitness, one lane per individual.  Weights are uniform across
// the wave and reach the FMAs through scalar loads.
template <int NIN, int H1, int H2, bool BF16>
__global__ void __launch_bounds__(256) ga_fitness_kernel(const GAConst c, int S, int P, const uint64_t *pop,
                                                         const float *sla, const float *omega, double *fit)
{
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
#pragma unroll
    for (int j = 0; j < kMaxN; j++)   // compile-time index into the argument block
        if (threadIdx.x == (unsigned)j) {
            s_tau[j] = c.obj.tau[j];
            s_prev[j] = c.obj.prev[j];
        }
    __syncthreads();
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)S * P) return;
    const int s = (int)(t / P);
    const int N = c.N, L = c.L;
    int32_t d[kMaxN];
    ga_digits(c, pop[t], d);
    double z[NIN];
    // aggregate: fp32, model order, each slot
#pragma unroll
    for (int k = 0; k < NIN; k++) z[k] = 0.0;
    float agg_v = 0.f;
#pragma unroll
    for (int k = 0; k < NIN; k++) {
        if (k >= L) {
            const int col = c.agg_cols[k - L];
            float a = 0.f;
            for (int i = 0; i < N; i++) a = a + c.features[(int64_t)(c.opt_off[i] + d[i]) * L + col];
            // the surrogates' aggregate input: the candidate's, or the
            // observed state held fixed (the VRAM cap still sees the candidate)
            z[k] = c.fixed ? (double)c.state[k - L] : (double)a;
            if (k - L == c.vram_slot) agg_v = a;
        }
    }
    const bool vram_ok = (double)agg_v <= (double)c.vram_cap;
    bool sla_ok = true;
    double J = 0.0;
    for (int i = 0; i < N; i++) {
        const float *x = c.features + (int64_t)(c.opt_off[i] + d[i]) * L;
#pragma unroll
        for (int k = 0; k < NIN; k++)
            if (k < L) z[k] = (double)x[k];
        const double *w = c.w64 + (int64_t)i * c.wstride;
        const double *W1 = w, *b1 = W1 + H1 * NIN, *W2 = b1 + H1, *b2 = W2 + H2 * H1, *W3 = b2 + H2, *b3 = W3 + 2 * H2;
        double h1[H1];
#pragma unroll
        for (int u = 0; u < H1; u++) {
            if (BF16) {
                // fp32 accumulation in input order, relu, round to bfloat16
                float a = (float)b1[u];
#pragma unroll
                for (int k = 0; k < NIN; k++) a = fmaf((float)W1[u * NIN + k], (float)z[k], a);
                a = a > 0.f ? a : 0.f;
                const uint32_t bits = __float_as_uint(a);
                const uint32_t r = (bits + 0x7FFFu + ((bits >> 16) & 1u)) & 0xFFFF0000u;
                h1[u] = (double)__uint_as_float(r);
            } else {
                double a = b1[u];
#pragma unroll
                for (int k = 0; k < NIN; k++) a = fma(W1[u * NIN + k], z[k], a);
                h1[u] = a > 0.0 ? a : 0.0;
            }
        }
        double y0 = b3[0], y1 = b3[1];
        // four layer-2 chains in flight (each still in input order; the
        // layer-3 chains take them in unit order)
#pragma unroll 4
        for (int v = 0; v < H2; v++) {
            double a = b2[v];
#pragma unroll
            for (int u = 0; u < H1; u++) a = fma(W2[v * H1 + u], h1[u], a);
            a = a > 0.0 ? a : 0.0;
            y0 = fma(W3[v], a, y0);
            y1 = fma(W3[H2 + v], a, y1);
        }
        if (c.act) {   // the predictor's sigmoid output
            y0 = canon_sigmoid(y0);
            y1 = canon_sigmoid(y1);
        }
        if (!(y0 <= (double)sla[(int64_t)s * N + i])) sla_ok = false;
        const double om = (double)omega[(int64_t)s * N + i];
        if (c.obj.kind != 0) {
            // the full utility of Eq. 3, canonical term order
            double q, Pr, pen;
            bool do_P, do_pen;
            if (!canon_eq3(c.obj, c.opt_off[i] + d[i], y1, s_tau[i], s_prev[i], q, Pr, do_P, pen, do_pen))
                sla_ok = false;
            J = fma(om, q, J);
            if (do_P) J = J - Pr;
            if (do_pen) J = J - pen;
        } else {
            J = fma(om, y1, J);
        }
    }
    fit[t] = (vram_ok && sla_ok) ? J : -INFINITY;
}

// Canonical fitness, one lane per individual, layer 1 continued from each
// option's precomputed local-feature chain (only the A aggregate steps are
// left per individual).  Dynamic LDS: [sumK][H1 + 2] doubles of that chain
// (rows padded by 16 bytes against bank conflicts), then [sumK][A] floats:
// each option row's aggregate columns.  The workgroup's waves take the
// models together (a barrier per model), so that the model's weights, read
// through scalar loads, stay in the scalar cache.
template <int A, int H1, int H2, bool BF16>
__global__ void __launch_bounds__(kGaFitThreads) ga_fitness_pre_kernel(const GAConst c, int S, int P,
                                                                       const uint64_t *pop, const float *sla,
                                                                       const float *omega, double *fit,
                                                                       uint32_t memo_gen)
{
    extern __shared__ __align__(16) double pre_s[];
    constexpr int PS = H1 + 2;
    float *agg_s = reinterpret_cast<float *>(pre_s + (size_t)c.sumK * PS);
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < kMaxN; j++)   // compile-time index into the argument block
        if (tid == j) {
            s_tau[j] = c.obj.tau[j];
            s_prev[j] = c.obj.prev[j];
        }
    for (int t = tid; t < c.sumK * H1; t += blockDim.x) {
        const int r = t / H1;
        pre_s[r * PS + (t - r * H1)] = c.pre[t];
    }
    for (int t = tid; t < c.sumK * A; t += blockDim.x) {
        const int r = t / A;
        agg_s[t] = c.features[(int64_t)r * c.L + c.agg_cols[t - r * A]];
    }
    __syncthreads();
    const int64_t n = (int64_t)S * P;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + tid;
    // lanes past the population leave: a wave that has ended no longer
    // counts at the barriers below (and one that is partly done still
    // executes them)
    if (t >= n) return;
    const int64_t tt = t;
    const int s = (int)(tt / P);
    const int N = c.N, L = c.L, NIN = L + A;
    int32_t d[kMaxN];
    const uint64_t idx = pop[tt];
    ga_digits(c, idx, d);
    // aggregate slots: fp32 sums in model order; the surrogates see them, or
    // the observed state held fixed (the VRAM cap still sees the candidate)
    double za[A];
    float agg_v = 0.f;
#pragma unroll
    for (int a = 0; a < A; a++) {
        float x = 0.f;
        for (int i = 0; i < N; i++) x = x + agg_s[(c.opt_off[i] + d[i]) * A + a];
        za[a] = c.fixed ? (double)c.state[a] : (double)x;
        if (a == c.vram_slot) agg_v = x;
    }
    const bool vram_ok = (double)agg_v <= (double)c.vram_cap;
    bool sla_ok = true;
    double J = 0.0;
    for (int i = 0; i < N; i++) {
        // a bare barrier: it orders no memory, so the weights below stay
        // scalar loads (read-only for the whole kernel, in the constant
        // address space)
        __builtin_amdgcn_s_barrier();
        typedef const __attribute__((address_space(4))) double cdouble;
        const cdouble *w = (const cdouble *)(c.w64 + (int64_t)i * c.wstride);
        const cdouble *W1a = w + L, *W2 = w + (int64_t)H1 * NIN + H1, *b2 = W2 + H2 * H1, *W3 = b2 + H2,
                      *b3 = W3 + 2 * H2;
        const double *pr = pre_s + (c.opt_off[i] + d[i]) * PS;
        double h1[H1];
#pragma unroll
        for (int u = 0; u < H1; u += 2) {
            const double2 v = *reinterpret_cast<const double2 *>(pr + u);
            h1[u] = v.x;
            h1[u + 1] = v.y;
        }
#pragma unroll
        for (int u = 0; u < H1; u++) {
            if (BF16) {
                // the fp32 chain continues over the aggregate inputs, relu,
                // round to bfloat16
                float a = (float)h1[u];
#pragma unroll
                for (int k = 0; k < A; k++) a = fmaf((float)W1a[u * NIN + k], (float)za[k], a);
                a = a > 0.f ? a : 0.f;
                const uint32_t bits = __float_as_uint(a);
                const uint32_t r = (bits + 0x7FFFu + ((bits >> 16) & 1u)) & 0xFFFF0000u;
                h1[u] = (double)__uint_as_float(r);
            } else {
                double a = h1[u];
#pragma unroll
                for (int k = 0; k < A; k++) a = fma(W1a[u * NIN + k], za[k], a);
                h1[u] = a > 0.0 ? a : 0.0;
            }
        }
        double y0 = b3[0], y1 = b3[1];
        // four layer-2 chains in flight (each in input order; the layer-3
        // chains take them in unit order)
#pragma unroll 4
        for (int v = 0; v < H2; v++) {
            double a = b2[v];
#pragma unroll
            for (int u = 0; u < H1; u++) a = fma(W2[v * H1 + u], h1[u], a);
            a = a > 0.0 ? a : 0.0;
            y0 = fma(W3[v], a, y0);
            y1 = fma(W3[H2 + v], a, y1);
        }
        if (c.act) {   // the predictor's sigmoid output
            y0 = canon_sigmoid(y0);
            y1 = canon_sigmoid(y1);
        }
        if (memo_gen) {   // into the run's memo (equal values where two lanes share an index)
            c.memo[(idx * (uint64_t)N + (uint64_t)i) * 2u] = y0;
            c.memo[(idx * (uint64_t)N + (uint64_t)i) * 2u + 1u] = y1;
        }
        if (!(y0 <= (double)sla[(int64_t)s * N + i])) sla_ok = false;
        const double om = (double)omega[(int64_t)s * N + i];
        if (c.obj.kind != 0) {
            // the full utility of Eq. 3, canonical term order
            double q, Pr, pen;
            bool do_P, do_pen;
            if (!canon_eq3(c.obj, c.opt_off[i] + d[i], y1, s_tau[i], s_prev[i], q, Pr, do_P, pen, do_pen))
                sla_ok = false;
            J = fma(om, q, J);
            if (do_P) J = J - Pr;
            if (do_pen) J = J - pen;
        } else {
            J = fma(om, y1, J);
        }
    }
    fit[t] = (vram_ok && sla_ok) ? J : -INFINITY;
    if (memo_gen) c.memo_tag[idx] = 2u * memo_gen + (vram_ok ? 1u : 0u);
}

// One model's term of the canonical fitness, in the order every fitness
// kernel takes it: the service constraint (Eq. 4), then J = fma(omega, thr,
// J) or, under Eq. 3, the utility's terms (throughput floor as a constraint).
__device__ __forceinline__ void ga_term(const GAConst &c, int s, int i, int64_t row, double lat, double thr,
                                        const float *sla, const float *omega, const float *tau,
                                        const int32_t *prev, double &J, bool &ok)
{
    if (!(lat <= (double)sla[(int64_t)s * c.N + i])) ok = false;
    const double om = (double)omega[(int64_t)s * c.N + i];
    if (c.obj.kind != 0) {
        double q, Pr, pen;
        bool do_P, do_pen;
        if (!canon_eq3(c.obj, row, thr, tau[i], prev[i], q, Pr, do_P, pen, do_pen)) ok = false;
        J = fma(om, q, J);
        if (do_P) J = J - Pr;
        if (do_pen) J = J - pen;
    } else {
        J = fma(om, thr, J);
    }
}

// Generations after the first (large populations): the canonical fitness
// from the run's memo of per-model predictions, which depend on the joint
// index only (not on the scenario).  An individual whose index an earlier
// generation evaluated (tag 2 g' + v, g' below this launch's) reads its
// models' (lat, thr) there and combines them with its scenario's bounds and
// weights.  The workgroup's other individuals (configurations new to the
// run) are evaluated here, one wave per individual with lanes over hidden
// units (the canonical forward, weights staged in LDS when they fit), and
// written to the memo.  Entries written by this launch are not read by it
// (evaluating an index twice gives equal values), so no workgroup waits on
// another.  Dynamic LDS: [staged weights][W x (nin + H1 + H2) doubles].
template <bool BF16, bool STAGE>
__global__ void __launch_bounds__(kGaMemoThreads) ga_fitness_memo_kernel(const GAConst c, int S, int P,
                                                                         const uint64_t *pop, const float *sla,
                                                                         const float *omega, double *fit,
                                                                         uint32_t memo_gen, int stage_floats)
{
    extern __shared__ float4 dyn4[];
    __shared__ int s_miss[kGaMemoThreads];
    __shared__ int s_nmiss;
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    constexpr int W = kGaMemoThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (tid < kMaxN) {
        s_tau[tid] = c.obj.tau[tid];
        s_prev[tid] = c.obj.prev[tid];
    }
    if (tid == 0) s_nmiss = 0;
    __syncthreads();
    const int N = c.N, L = c.L, A = c.A, nin = L + A;
    const int64_t n = (int64_t)S * P;
    const int64_t t = (int64_t)blockIdx.x * kGaMemoThreads + tid;
    if (t < n) {
        const uint64_t idx = pop[t];
        const uint32_t tg = c.memo_tag[idx];
        // the entry's values are read beside its tag (used only on a hit)
        double m[2 * kMaxN];
        const double *mp = c.memo + idx * (uint64_t)N * 2u;
#pragma unroll
        for (int j = 0; j < 2 * kMaxN; j++)
            if (j < 2 * N) m[j] = mp[j];
        if ((tg >> 1) != 0u && (tg >> 1) < memo_gen) {
            int32_t d[kMaxN];
            ga_digits(c, idx, d);
            const int s = (int)(t / P);
            bool ok = (tg & 1u) != 0u;
            double J = 0.0;
#pragma unroll
            for (int i = 0; i < kMaxN; i++)
                if (i < N)
                    ga_term(c, s, i, c.opt_off[i] + d[i], m[2 * i], m[2 * i + 1], sla, omega, s_tau, s_prev, J, ok);
            fit[t] = ok ? J : -INFINITY;
        } else {
            s_miss[atomicAdd(&s_nmiss, 1)] = tid;
        }
    }
    __syncthreads();
    const int nm = s_nmiss;
    if (nm == 0) return;   // uniform: the workgroup had no new configuration
    if (tid == 0) atomicAdd(c.n_forwards, (unsigned long long)nm);
    const float *wbase = c.canon;
    if (STAGE) {
        const int n4 = (stage_floats + 3) / 4;
        const float4 *src = reinterpret_cast<const float4 *>(c.canon);
        for (int q = tid; q < n4; q += blockDim.x) dyn4[q] = src[q];
        wbase = reinterpret_cast<const float *>(dyn4);
        __syncthreads();
    }
    double *zs = reinterpret_cast<double *>(dyn4 + (STAGE ? (stage_floats + 3) / 4 : 0)) +
                 (int64_t)wave * (nin + c.H1 + c.H2);
    double *h1s = zs + nin, *h2s = h1s + c.H1;
    for (int q = wave; q < nm; q += W) {
        const int64_t tt = (int64_t)blockIdx.x * kGaMemoThreads + s_miss[q];
        const uint64_t idx = pop[tt];
        const int s = (int)(tt / P);
        int32_t d[kMaxN];
        ga_digits(c, idx, d);
        // aggregate slot `lane` (fp32, model order); the VRAM slot decides the cap
        float a = 0.f;
        if (lane < A)
            for (int i = 0; i < N; i++) a = a + c.features[(int64_t)(c.opt_off[i] + d[i]) * L + c.agg_cols[lane]];
        const float av = __shfl(a, c.vram_slot);
        const bool vram_ok = (double)av <= (double)c.vram_cap;
        if (lane < A) zs[L + lane] = c.fixed ? (double)c.state[lane] : (double)a;
        bool ok = vram_ok;
        double J = 0.0;
        for (int i = 0; i < N; i++) {
            const float *x = c.features + (int64_t)(c.opt_off[i] + d[i]) * L;
            for (int k = lane; k < L; k += 64) zs[k] = (double)x[k];
            __builtin_amdgcn_wave_barrier();
            double lat, thr;
            canon_model<BF16, true>(wbase + (int64_t)i * c.wstride, nin, c.H1, c.H2, zs, h1s, h2s, lane, lat, thr,
                                    c.act);
            if (lane == 0) {
                c.memo[(idx * (uint64_t)N + (uint64_t)i) * 2u] = lat;
                c.memo[(idx * (uint64_t)N + (uint64_t)i) * 2u + 1u] = thr;
            }
            ga_term(c, s, i, c.opt_off[i] + d[i], lat, thr, sla, omega, s_tau, s_prev, J, ok);
            __builtin_amdgcn_wave_barrier();
        }
        if (lane == 0) {
            fit[tt] = ok ? J : -INFINITY;
            c.memo_tag[idx] = 2u * memo_gen + (vram_ok ? 1u : 0u);
        }
    }
}

// Zero a run's memo tags; the forward count starts at `first` (the
// generations that do not read the memo).
__global__ void ga_memo_clear_kernel(uint32_t *tag, uint64_t n, unsigned long long *n_forwards,
                                     unsigned long long first)
{
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) tag[i] = 0u;
    if (i == 0) *n_forwards = first;
}

// Canonical fp64 fitness, one workgroup per individual (small populations,
// and shapes the one-lane kernel does not take): wave w runs the canonical
// forward of models w, w + W, ... (W waves), each on its own LDS scratch; lane
// 0 then combines the models' predictions in model order, so J equals the
// one-lane kernel's bit for bit.  STAGE: the
// canonical weights of every model are first copied to LDS.  Dynamic LDS:
// [staged weights][W x (H1 + H2 + nin) doubles].
template <bool BF16, bool STAGE>
__global__ void __launch_bounds__(64 * kGaWideWaves) ga_fitness_wide_kernel(const GAConst c, int S, int P,
                                                                             const uint64_t *pop, const float *sla,
                                                                             const float *omega, double *fit,
                                                                             int stage_floats)
{
    extern __shared__ float4 dyn4[];
    __shared__ double aggs[kMaxN];
    __shared__ double s_lat[kMaxN], s_thr[kMaxN];
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    __shared__ int32_t d[kMaxN];
    __shared__ int s_vram_ok;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int W = (int)(blockDim.x >> 6);
    if (tid < kMaxN) {
        s_tau[tid] = c.obj.tau[tid];
        s_prev[tid] = c.obj.prev[tid];
        aggs[tid] = (double)c.state[tid];
    }
    const int N = c.N, L = c.L, A = c.A, nin = L + A, H1 = c.H1, H2 = c.H2;
    const float *wbase = c.canon;
    if (STAGE) {
        const int n4 = (stage_floats + 3) / 4;
        const float4 *src = reinterpret_cast<const float4 *>(c.canon);
        for (int q = tid; q < n4; q += blockDim.x) dyn4[q] = src[q];
        wbase = reinterpret_cast<const float *>(dyn4);
    }
    double *scr = reinterpret_cast<double *>(dyn4 + (STAGE ? (stage_floats + 3) / 4 : 0)) +
                  (int64_t)wave * (H1 + H2 + nin);
    double *h1s = scr, *h2s = scr + H1, *zs = scr + H1 + H2;
    const int rounds = (N + W - 1) / W;
    for (int64_t t = blockIdx.x; t < (int64_t)S * P; t += gridDim.x) {
        const int s = (int)(t / P);
        __syncthreads();
        if (tid == 0) ga_digits(c, pop[t], d);
        __syncthreads();
        // aggregate slot k (fp32, model order); the VRAM slot decides the cap
        if (tid < A) {
            float a = 0.f;
            for (int i = 0; i < N; i++) a = a + c.features[(int64_t)(c.opt_off[i] + d[i]) * L + c.agg_cols[tid]];
            if (!c.fixed) aggs[tid] = (double)a;
            if (tid == c.vram_slot) s_vram_ok = a <= c.vram_cap;
        }
        // every wave takes part in every round (the forward has barriers); a
        // wave past the last model repeats it and drops the result
        for (int r = 0; r < rounds; r++) {
            const int i = r * W + wave, ii = i < N ? i : N - 1;
            __syncthreads();
            const float *x = c.features + (int64_t)(c.opt_off[ii] + d[ii]) * L;
            for (int k = lane; k < nin; k += 64) zs[k] = k < L ? (double)x[k] : aggs[k - L];
            __syncthreads();
            double lat, thr;
            canon_model<BF16>(wbase + (int64_t)ii * c.wstride, nin, H1, H2, zs, h1s, h2s, lane, lat, thr, c.act);
            if (i < N && lane == 0) {
                s_lat[i] = lat;
                s_thr[i] = thr;
            }
        }
        __syncthreads();
        if (tid == 0) {
            bool ok = s_vram_ok != 0;
            double J = 0.0;
            for (int i = 0; i < N; i++) {
                const double lat = s_lat[i], thr = s_thr[i];
                if (!(lat <= (double)sla[(int64_t)s * N + i])) ok = false;
                const double om = (double)omega[(int64_t)s * N + i];
                if (c.obj.kind != 0) {
                    double q, Pr, pen;
                    bool do_P, do_pen;
                    if (!canon_eq3(c.obj, c.opt_off[i] + d[i], thr, s_tau[i], s_prev[i], q, Pr, do_P, pen, do_pen))
                        ok = false;
                    J = fma(om, q, J);
                    if (do_P) J = J - Pr;
                    if (do_pen) J = J - pen;
                } else {
                    J = fma(om, thr, J);
                }
            }
            fit[t] = ok ? J : -INFINITY;
        }
    }
}

__device__ __forceinline__ bool ga_better(double fa, uint64_t ia, double fb, uint64_t ib)
{
    return fa > fb || (fa == fb && ia < ib);
}

constexpr int kOpThreads = 256;                   // threads per operator workgroup
constexpr int kOpTeam = 4;                        // lanes per parent pair
constexpr int kOpPairs = kOpThreads / kOpTeam;    // parent pairs per operator workgroup

// The Philox blocks of a parent pair kept in LDS, in a fixed order: the
// selection blocks (2k draws), the crossover block, the swap blocks (one
// word per gene), the mutation blocks of child 1 + 2q and of child 2 + 2q
// (two words per gene).  A child's repair block is drawn where it is needed.
struct OpBlocks {
    int nsel, nswap, nmut, total;
    __host__ __device__ OpBlocks(int tk, int N)
        : nsel((2 * tk + 3) / 4), nswap((N + 3) / 4), nmut((N + 1) / 2), total(nsel + 1 + nswap + 2 * nmut)
    {
    }
    __host__ __device__ int cx() const { return nsel; }
    __host__ __device__ int swap() const { return nsel + 1; }
    __host__ __device__ int mut(int t) const { return nsel + 1 + nswap + t * nmut; }
};

// Dynamic LDS of the operator kernel: the pairs' Philox words, the parents'
// genes.
inline size_t ops_lds_bytes(int tk, int N)
{
    return (size_t)kOpPairs * OpBlocks(tk, N).total * 32 + (size_t)kOpPairs * 2 * N * 4;
}

// Operators: a scenario's pairs are spread over ceil((P/2) / kOpPairs)
// workgroups; tournaments read fitness and population from global memory.
// The elite (slot 0 of the next generation, which no child writes) and the
// best ever are found by one more workgroup beside a scenario's operator
// workgroups (elite_wg = 1), off their critical path; with elite_wg = 0 the
// first operator workgroup finds them.  At g == gens the final population is
// copied out.  The pairs'
// Philox blocks are first computed by all threads together (each block once,
// its four words used in order); then, in each team of lanes, lane t runs
// tournament t and decodes parent t, and builds child t (crossover,
// mutation, repair).
__global__ void __launch_bounds__(kOpThreads) ga_ops_kernel(const GAConst c, uint64_t seed, int P, int gen, int gens,
                                                            int tk, float p_cx, float p_swap, float p_mut,
                                                            const uint32_t *fl, const unsigned long long *n_fl_ptr,
                                                            const uint64_t *pop, const double *fit, uint64_t *next,
                                                            double *best_J, uint64_t *best_idx, uint64_t *final_pop,
                                                            int wgs_per_scen, int elite_wg)
{
    extern __shared__ uint64_t ops_dyn[];
    __shared__ int red[kOpThreads];
    __shared__ double red_f[kOpThreads];
    __shared__ uint64_t red_i[kOpThreads];
    // per scenario: wgs_per_scen operator workgroups, then (elite_wg) one
    // workgroup for the elite alone; otherwise operator workgroup 0 finds it
    const int wgs_all = wgs_per_scen + elite_wg;
    const int s = blockIdx.x / wgs_all, pb = blockIdx.x % wgs_all, tid = threadIdx.x;
    const int N = c.N;
    const OpBlocks ob(tk, N);
    uint64_t *words = ops_dyn;                                                                // [kOpPairs][total][4]
    int32_t *genes = reinterpret_cast<int32_t *>(words + (int64_t)kOpPairs * ob.total * 4);   // [kOpPairs][2][N]
    const uint64_t *ps = pop + (int64_t)s * P;
    const double *fs = fit + (int64_t)s * P;
    uint64_t *ns = next + (int64_t)s * P;
    const unsigned long long n_fl = *n_fl_ptr;
    if (gen == gens && pb < wgs_per_scen) {
        if (final_pop)
            for (int j = pb * kOpThreads + tid; j < P; j += wgs_per_scen * kOpThreads)
                final_pop[(int64_t)s * P + j] = n_fl ? ps[j] : ~0ull;
    }
    if (pb == (elite_wg ? wgs_per_scen : 0)) {
        // elite: best (f desc, index asc, slot asc), reduced in LDS
        int b = -1;
        double fb = 0.0;
        uint64_t ib = 0;
        for (int j = tid; j < P; j += kOpThreads) {
            const double f = fs[j];
            const uint64_t i = ps[j];
            if (b < 0 || ga_better(f, i, fb, ib)) {
                b = j;
                fb = f;
                ib = i;
            }
        }
        red[tid] = b;
        red_f[tid] = fb;
        red_i[tid] = ib;
        __syncthreads();
        for (int o = kOpThreads / 2; o > 0; o >>= 1) {
            if (tid < o) {
                const int x = red[tid], y = red[tid + o];
                const double fx = red_f[tid], fy = red_f[tid + o];
                const uint64_t ix = red_i[tid], iy = red_i[tid + o];
                if (y >= 0 && (x < 0 || ga_better(fy, iy, fx, ix) || (fy == fx && iy == ix && y < x))) {
                    red[tid] = y;
                    red_f[tid] = fy;
                    red_i[tid] = iy;
                }
            }
            __syncthreads();
        }
        if (tid == 0) {
            const double fe = red_f[0];
            const uint64_t ie = red_i[0];
            if (fe > -INFINITY && ga_better(fe, ie, best_J[s], best_idx[s])) {
                best_J[s] = fe;
                best_idx[s] = ie;
            }
            if (gen != gens) ns[0] = ie;
        }
        if (elite_wg) return;
    }
    if (gen == gens) return;
    const uint64_t g1 = (uint64_t)gen + 1, sc = (uint64_t)s;
    const int q0 = pb * kOpPairs;
    const int np = P / 2 - q0 < kOpPairs ? P / 2 - q0 : kOpPairs;
    // the Philox blocks of this workgroup's pairs, each computed once by one
    // thread: first the selection and crossover blocks, then the swap blocks
    // of the pairs that cross over and the mutation blocks; a child's repair
    // block only when it is needed (every draw is counter-addressed, so the
    // values do not depend on which are computed)
    const int nA = ob.nsel + 1, nB = ob.nswap + 2 * ob.nmut;
    for (int jb = tid; jb < np * nA; jb += kOpThreads) {
        const int ql = jb / nA, k = jb - ql * nA;
        const Philox4 r = philox4x64_10((uint64_t)(q0 + ql), g1, sc, k < ob.cx() ? kPSel + k : kPCx, seed, 0);
        uint64_t *w = words + ((int64_t)ql * ob.total + k) * 4;
#pragma unroll
        for (int x = 0; x < 4; x++) w[x] = r.w[x];
    }
    __syncthreads();
    for (int jb = tid; jb < np * nB; jb += kOpThreads) {
        const int ql = jb / nB, k = ob.swap() + (jb - ql * nB);
        const uint64_t q = (uint64_t)(q0 + ql);
        uint64_t item = q, purpose;
        if (k < ob.mut(0)) {
            if (!(ga_uni(words[((int64_t)ql * ob.total + ob.cx()) * 4]) < (double)p_cx)) continue;
            purpose = kPSwap + (k - ob.swap());
        } else {
            const int t = (k - ob.mut(0)) / ob.nmut;
            item = 1 + 2 * q + t;
            purpose = kPMut + (k - ob.mut(t));
        }
        const Philox4 r = philox4x64_10(item, g1, sc, purpose, seed, 0);
        uint64_t *w = words + ((int64_t)ql * ob.total + k) * 4;
#pragma unroll
        for (int x = 0; x < 4; x++) w[x] = r.w[x];
    }
    __syncthreads();
    const int ql = tid / kOpTeam, t = tid % kOpTeam;
    const bool act = ql < np && t < 2;
    const uint64_t *pw = words + (int64_t)ql * ob.total * 4;
    int32_t *pg = genes + (ql * 2) * N;
    if (act) {
        // tournament t: draws t k .. t k + k - 1 of the selection words
        int par = -1;
        double fpar = 0.0;
        uint64_t ipar = 0;
        for (int m = t * tk; m < t * tk + tk; m++) {
            const int dj = (int)ga_below(pw[m], (uint64_t)P);
            const double f = fs[dj];
            const uint64_t i = ps[dj];
            if (par < 0 || ga_better(f, i, fpar, ipar)) {
                par = dj;
                fpar = f;
                ipar = i;
            }
        }
        int32_t dp[kMaxN];
        ga_digits(c, ipar, dp);
        for (int i = 0; i < N; i++) pg[t * N + i] = dp[i];
    }
    __syncthreads();
    if (!act) return;
    const int j = 1 + 2 * (q0 + ql) + t;
    if (j >= P) return;
    // child t starts as parent t; uniform crossover gives it the other
    // parent's gene wherever the pair's swap draw falls below p_swap; gene i
    // mutates with words 2i (mutate?) and 2i + 1 (new value).  Gene by gene
    // in model order, with a compile-time model index (no per-lane array).
    const bool cx = ga_uni(pw[ob.cx() * 4]) < (double)p_cx;
    const uint64_t *mw = pw + ob.mut(t) * 4;
    float vs = 0.f;
    uint64_t idx = 0;
#pragma unroll
    for (int i = 0; i < kMaxN; i++) {
        if (i < N) {
            const bool sw = cx && ga_uni(pw[ob.swap() * 4 + i]) < (double)p_swap;
            int32_t g = pg[(sw ? 1 - t : t) * N + i];
            if (ga_uni(mw[2 * i]) < (double)p_mut) g = (int32_t)ga_below(mw[2 * i + 1], (uint64_t)c.K[i]);
            vs = vs + c.features[(int64_t)(c.opt_off[i] + g) * c.L + c.vram_col];
            idx = idx * (uint64_t)c.K[i] + (uint64_t)g;
        }
    }
    if (!((double)vs <= (double)c.vram_cap))
        idx = n_fl ? fl[ga_below(philox4x64_10((uint64_t)j, g1, sc, kPRep, seed, 0).w[0], n_fl)] : 0;
    ns[j] = idx;
}

// ---------------------------------------------------------------- launchers

template <int NIN, int H1, int H2>
static hipError_t launch_fit_t(const GAConst &c, int S, int P, const uint64_t *pop, const float *sla,
                               const float *omega, double *fit, hipStream_t st)
{
    const int64_t n = (int64_t)S * P;
    const int grid = (int)((n + 255) / 256);
    if (c.bf16)
        hipLaunchKernelGGL((ga_fitness_kernel<NIN, H1, H2, true>), dim3(grid), dim3(256), 0, st, c, S, P, pop, sla, omega, fit);
    else
        hipLaunchKernelGGL((ga_fitness_kernel<NIN, H1, H2, false>), dim3(grid), dim3(256), 0, st, c, S, P, pop, sla, omega, fit);
    return hipGetLastError();
}

int ga_fitness_supported(int nin, int h1, int h2)
{
    return (h1 == 32 && h2 == 32 && (nin == 10 || nin == 12 || nin == 14 || nin == 16)) ||
           (h1 == 64 && h2 == 32 && (nin == 10 || nin == 12 || nin == 14 || nin == 16)) ||
           (h1 == 64 && h2 == 64 && (nin == 12 || nin == 16 || nin == 22));
}

template <int A, int H1, int H2>
static hipError_t launch_fit_pre_t(const GAConst &c, int S, int P, const uint64_t *pop, const float *sla,
                                   const float *omega, double *fit, size_t lds, hipStream_t st, uint32_t memo_gen)
{
    const int64_t n = (int64_t)S * P;
    const int grid = (int)((n + kGaFitThreads - 1) / kGaFitThreads);
    auto fn = c.bf16 ? ga_fitness_pre_kernel<A, H1, H2, true> : ga_fitness_pre_kernel<A, H1, H2, false>;
    const hipError_t e = ensure_dyn_lds((const void *)fn, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kGaFitThreads), lds, st, c, S, P, pop, sla, omega, fit, memo_gen);
    return hipGetLastError();
}

static size_t ga_pre_lds(const GAConst &c)
{
    return (size_t)c.sumK * (c.H1 + 2) * 8 + (size_t)c.sumK * c.A * 4;
}

static bool ga_pre_shape(int A, int H1, int H2)
{
    return (A == 2 || A == 4 || A == 6 || A == 8) && ((H1 == 32 && H2 == 32) || (H1 == 64 && (H2 == 32 || H2 == 64)));
}

bool ga_memo_supported(const GAConst &c, int S, int P)
{
    return (int64_t)S * P > kGaWideMax && c.pre && ga_pre_lds(c) <= kGaPreLdsBytes && ga_pre_shape(c.A, c.H1, c.H2);
}

hipError_t launch_ga_memo_clear(uint32_t *tag, uint64_t n, unsigned long long *n_forwards,
                                unsigned long long first, hipStream_t st)
{
    const uint64_t m = n > 0 ? n : 1;
    hipLaunchKernelGGL(ga_memo_clear_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, st, tag, n,
                       n_forwards, first);
    return hipGetLastError();
}

hipError_t launch_ga_fitness(const GAConst &c, int S, int P, const uint64_t *pop, const float *sla, const float *omega,
                             double *fit, hipStream_t st, uint32_t memo_gen)
{
    const int nin = c.L + c.A;
    if (c.memo && memo_gen >= 2) {
        // later generations with the run's memo
        const int64_t n = (int64_t)S * P;
        const int64_t wfloats = (int64_t)c.N * c.wstride;
        const bool stage = ((wfloats + 3) / 4) * 16 <= (int64_t)kGaStageBytes;
        const size_t lds = (stage ? (size_t)((wfloats + 3) / 4) * 16 : 0) +
                           (size_t)(kGaMemoThreads / 64) * (nin + c.H1 + c.H2) * 8;
        auto fn = c.bf16 ? (stage ? ga_fitness_memo_kernel<true, true> : ga_fitness_memo_kernel<true, false>)
                         : (stage ? ga_fitness_memo_kernel<false, true> : ga_fitness_memo_kernel<false, false>);
        const hipError_t e = ensure_dyn_lds((const void *)fn, lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(fn, dim3((unsigned)((n + kGaMemoThreads - 1) / kGaMemoThreads)), dim3(kGaMemoThreads),
                           lds, st, c, S, P, pop, sla, omega, fit, memo_gen, stage ? (int)wfloats : 0);
        return hipGetLastError();
    }
    // large populations: the kernel that continues each option's local chain,
    // when the chain table and the aggregate columns fit in LDS
    const size_t pre_lds = ga_pre_lds(c);
    const uint32_t mg = c.memo ? memo_gen : 0u;
    if ((int64_t)S * P > kGaWideMax && c.pre && pre_lds <= kGaPreLdsBytes) {
#define MF_GA_PRE(AA, HA, HB) \
    if (c.A == AA && c.H1 == HA && c.H2 == HB) return launch_fit_pre_t<AA, HA, HB>(c, S, P, pop, sla, omega, fit, pre_lds, st, mg);
        MF_GA_PRE(2, 32, 32) MF_GA_PRE(4, 32, 32) MF_GA_PRE(6, 32, 32) MF_GA_PRE(8, 32, 32)
        MF_GA_PRE(2, 64, 32) MF_GA_PRE(4, 64, 32) MF_GA_PRE(6, 64, 32) MF_GA_PRE(8, 64, 32)
        MF_GA_PRE(2, 64, 64) MF_GA_PRE(4, 64, 64) MF_GA_PRE(6, 64, 64) MF_GA_PRE(8, 64, 64)
#undef MF_GA_PRE
    }
    if ((int64_t)S * P <= kGaWideMax || !ga_fitness_supported(nin, c.H1, c.H2)) {
        const int64_t n = (int64_t)S * P;
        // every model's weights in LDS when they fit (the canonical image is
        // 16-byte aligned per problem and padded to 256 bytes)
        const int W = c.N < kGaWideWaves ? c.N : kGaWideWaves;
        const int64_t wfloats = (int64_t)c.N * c.wstride;
        const bool stage = ((wfloats + 3) / 4) * 16 <= (int64_t)kGaStageBytes;
        const size_t lds = (stage ? (size_t)((wfloats + 3) / 4) * 16 : 0) + (size_t)W * (c.H1 + c.H2 + nin) * 8;
        const int64_t cap = stage ? kGaWideStagedWgs : 65536;
        const int grid = (int)(n < cap ? n : cap);
        auto fn = c.bf16 ? (stage ? ga_fitness_wide_kernel<true, true> : ga_fitness_wide_kernel<true, false>)
                         : (stage ? ga_fitness_wide_kernel<false, true> : ga_fitness_wide_kernel<false, false>);
        const hipError_t e = ensure_dyn_lds((const void *)fn, lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(fn, dim3(grid), dim3(64 * W), lds, st, c, S, P, pop, sla, omega, fit,
                           stage ? (int)wfloats : 0);
        return hipGetLastError();
    }
#define MF_GA_FIT(NI, HA, HB) \
    if (nin == NI && c.H1 == HA && c.H2 == HB) return launch_fit_t<NI, HA, HB>(c, S, P, pop, sla, omega, fit, st);
    MF_GA_FIT(10, 32, 32) MF_GA_FIT(12, 32, 32) MF_GA_FIT(14, 32, 32) MF_GA_FIT(16, 32, 32)
    MF_GA_FIT(10, 64, 32) MF_GA_FIT(12, 64, 32) MF_GA_FIT(14, 64, 32) MF_GA_FIT(16, 64, 32)
    MF_GA_FIT(12, 64, 64) MF_GA_FIT(16, 64, 64) MF_GA_FIT(22, 64, 64)
#undef MF_GA_FIT
    return hipErrorInvalidValue;
}

hipError_t launch_ga_feasible(const GAConst &c, uint32_t *blk_count, uint64_t *blk_off, unsigned long long *n_fl,
                              uint32_t *fl, hipStream_t st)
{
    const uint64_t n_blk = (c.space + kFlBlock - 1) / kFlBlock;
    hipLaunchKernelGGL(fl_count_kernel, dim3((unsigned)n_blk), dim3(kFlBlock), 0, st, c, blk_count);
    hipLaunchKernelGGL(fl_scan_kernel, dim3(1), dim3(1024), 0, st, blk_count, n_blk, blk_off, n_fl);
    hipLaunchKernelGGL(fl_write_kernel, dim3((unsigned)n_blk), dim3(kFlBlock), 0, st, c, blk_off, fl);
    return hipGetLastError();
}

hipError_t launch_ga_init(uint64_t seed, int S, int P, const uint32_t *fl, const unsigned long long *n_fl,
                          uint64_t *pop, double *best_J, uint64_t *best_idx, hipStream_t st)
{
    const int64_t n = (int64_t)S * P;
    hipLaunchKernelGGL(ga_init_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, seed, S, P, fl, n_fl, pop,
                       best_J, best_idx);
    return hipGetLastError();
}

hipError_t launch_ga_ops(const GAConst &c, uint64_t seed, int S, int P, int gen, int gens, int tk, float p_cx,
                         float p_swap, float p_mut, const uint32_t *fl, const unsigned long long *n_fl,
                         const uint64_t *pop, const double *fit, uint64_t *next, double *best_J, uint64_t *best_idx,
                         uint64_t *final_pop, hipStream_t st)
{
    const int wgs = (P / 2 + kOpPairs - 1) / kOpPairs > 0 ? (P / 2 + kOpPairs - 1) / kOpPairs : 1;
    const size_t lds = ops_lds_bytes(tk, c.N);
    const hipError_t e = ensure_dyn_lds((const void *)ga_ops_kernel, lds);
    if (e != hipSuccess) return e;
    const int elite_wg = 1;   // the elite's reduction in a workgroup of its own
    hipLaunchKernelGGL(ga_ops_kernel, dim3(S * (wgs + elite_wg)), dim3(kOpThreads), lds, st, c, seed, P, gen, gens, tk,
                       p_cx, p_swap, p_mut, fl, n_fl, pop, fit, next, best_J, best_idx, final_pop, wgs, elite_wg);
    return hipGetLastError();
}

}  // namespace mfi
