// Genetic-algorithm scheduler (Section IV-C) on the GPU.
//
// Per generation two launches: the fitness of every individual of every
// scenario (one lane per individual, the canonical fp64 surrogate chain, so
// every tournament compares exactly the values the results are defined by),
// then one workgroup per scenario applies the operators: elitism (slot 0),
// tournaments of k draws with replacement, uniform crossover, per-gene
// mutation, repair of VRAM-infeasible children from the feasible list.
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

__device__ __forceinline__ Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                                 uint64_t k1)
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        if (r) { k0 += W0; k1 += W1; }
        const uint64_t h0 = __umul64hi(M0, c0), l0 = M0 * c0;
        const uint64_t h1 = __umul64hi(M1, c2), l1 = M1 * c2;
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

__device__ __forceinline__ bool vram_feasible(const GAConst &c, uint64_t idx)
{
    // fp32 sum of the VRAM column in model order (the aggregate slot's value)
    int32_t d[kMaxN];
    for (int i = c.N - 1; i >= 0; i--) {
        d[i] = (int32_t)(idx % (uint64_t)c.K[i]);
        idx /= (uint64_t)c.K[i];
    }
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
    pop[t] = fl[ga_below(ga_draw(seed, (uint64_t)j, 0, (uint64_t)s, kPInit, 0), *n_fl)];
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
    uint64_t idx = pop[t];
    int32_t d[kMaxN];
    for (int i = N - 1; i >= 0; i--) {
        d[i] = (int32_t)(idx % (uint64_t)c.K[i]);
        idx /= (uint64_t)c.K[i];
    }
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

__device__ __forceinline__ bool ga_better(double fa, uint64_t ia, double fb, uint64_t ib)
{
    return fa > fb || (fa == fb && ia < ib);
}

constexpr int kOpPairs = 256;     // parent pairs (threads) per operator workgroup
constexpr int kGaMaxPop = 4096;

// Operators: a scenario's pairs are spread over ceil((P/2) / kOpPairs)
// workgroups, each holding the scenario's population and fitness in LDS and
// computing the elite itself; the first of them updates the best ever.  At
// g == gens the final population is copied out.  Every Philox block is
// computed once and its four words used in order.
__global__ void __launch_bounds__(kOpPairs) ga_ops_kernel(const GAConst c, uint64_t seed, int P, int gen, int gens,
                                                          int tk, float p_cx, float p_swap, float p_mut,
                                                          const uint32_t *fl, const unsigned long long *n_fl_ptr,
                                                          const uint64_t *pop, const double *fit, uint64_t *next,
                                                          double *best_J, uint64_t *best_idx, uint64_t *final_pop,
                                                          int wgs_per_scen)
{
    __shared__ double sf[kGaMaxPop];
    __shared__ uint64_t si[kGaMaxPop];
    __shared__ int red[kOpPairs];
    const int s = blockIdx.x / wgs_per_scen, pb = blockIdx.x % wgs_per_scen, tid = threadIdx.x;
    const int N = c.N;
    const uint64_t *ps = pop + (int64_t)s * P;
    const double *fs = fit + (int64_t)s * P;
    for (int j = tid; j < P; j += kOpPairs) {
        sf[j] = fs[j];
        si[j] = ps[j];
    }
    __syncthreads();
    // elite: best (f desc, index asc, slot asc)
    int b = -1;
    for (int j = tid; j < P; j += kOpPairs)
        if (b < 0 || ga_better(sf[j], si[j], sf[b], si[b])) b = j;
    red[tid] = b;
    __syncthreads();
    for (int o = kOpPairs / 2; o > 0; o >>= 1) {
        if (tid < o) {
            const int x = red[tid], y = red[tid + o];
            if (y >= 0 && (x < 0 || ga_better(sf[y], si[y], sf[x], si[x]) ||
                           (sf[y] == sf[x] && si[y] == si[x] && y < x)))
                red[tid] = y;
        }
        __syncthreads();
    }
    const int e = red[0];
    if (pb == 0 && tid == 0) {
        if (sf[e] > -INFINITY && ga_better(sf[e], si[e], best_J[s], best_idx[s])) {
            best_J[s] = sf[e];
            best_idx[s] = si[e];
        }
    }
    if (gen == gens) {
        if (final_pop)
            for (int j = pb * kOpPairs + tid; j < P; j += wgs_per_scen * kOpPairs) final_pop[(int64_t)s * P + j] = si[j];
        return;
    }
    uint64_t *ns = next + (int64_t)s * P;
    if (pb == 0 && tid == 0) ns[0] = si[e];
    const uint64_t g1 = (uint64_t)gen + 1, sc = (uint64_t)s, n_fl = *n_fl_ptr;
    const int q = pb * kOpPairs + tid;
    if (q >= P / 2) return;
    // tournaments: draws 0..tk-1 choose parent A, tk..2tk-1 parent B
    int pa = -1, pbest = -1;
    const int nsel = 2 * tk;
    for (int bl = 0; 4 * bl < nsel; bl++) {
        const Philox4 r = philox4x64_10((uint64_t)q, g1, sc, kPSel + bl, seed, 0);
#pragma unroll
        for (int w = 0; w < 4; w++) {
            const int m = 4 * bl + w;
            if (m < nsel) {
                const int dj = (int)ga_below(r.w[w], (uint64_t)P);
                if (m < tk) {
                    if (pa < 0 || ga_better(sf[dj], si[dj], sf[pa], si[pa])) pa = dj;
                } else {
                    if (pbest < 0 || ga_better(sf[dj], si[dj], sf[pbest], si[pbest])) pbest = dj;
                }
            }
        }
    }
    int32_t ch[2][kMaxN];
    {
        uint64_t x0 = si[pa], x1 = si[pbest];
        for (int i = N - 1; i >= 0; i--) {
            ch[0][i] = (int32_t)(x0 % (uint64_t)c.K[i]);
            x0 /= (uint64_t)c.K[i];
            ch[1][i] = (int32_t)(x1 % (uint64_t)c.K[i]);
            x1 /= (uint64_t)c.K[i];
        }
    }
    if (ga_uni(ga_draw(seed, (uint64_t)q, g1, sc, kPCx, 0)) < (double)p_cx) {
        for (int bl = 0; 4 * bl < N; bl++) {
            const Philox4 r = philox4x64_10((uint64_t)q, g1, sc, kPSwap + bl, seed, 0);
#pragma unroll
            for (int w = 0; w < 4; w++) {
                const int i = 4 * bl + w;
                if (i < N && ga_uni(r.w[w]) < (double)p_swap) {
                    const int32_t tmp = ch[0][i];
                    ch[0][i] = ch[1][i];
                    ch[1][i] = tmp;
                }
            }
        }
    }
    for (int t = 0; t < 2; t++) {
        const int j = 1 + 2 * q + t;
        if (j >= P) break;
        // mutation: gene i reads words 2i and 2i+1 of consecutive blocks,
        // so block bl holds genes 2 bl (words 0, 1) and 2 bl + 1 (words 2, 3)
        for (int bl = 0; 2 * bl < N; bl++) {
            const Philox4 r = philox4x64_10((uint64_t)j, g1, sc, kPMut + bl, seed, 0);
            const int i0 = 2 * bl, i1 = 2 * bl + 1;
            if (ga_uni(r.w[0]) < (double)p_mut) ch[t][i0] = (int32_t)ga_below(r.w[1], (uint64_t)c.K[i0]);
            if (i1 < N && ga_uni(r.w[2]) < (double)p_mut) ch[t][i1] = (int32_t)ga_below(r.w[3], (uint64_t)c.K[i1]);
        }
        float vs = 0.f;
        uint64_t idx = 0;
        for (int i = 0; i < N; i++) {
            vs = vs + c.features[(int64_t)(c.opt_off[i] + ch[t][i]) * c.L + c.vram_col];
            idx = idx * (uint64_t)c.K[i] + (uint64_t)ch[t][i];
        }
        if (!((double)vs <= (double)c.vram_cap))
            idx = fl[ga_below(ga_draw(seed, (uint64_t)j, g1, sc, kPRep, 0), n_fl)];
        ns[j] = idx;
    }
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

hipError_t launch_ga_fitness(const GAConst &c, int S, int P, const uint64_t *pop, const float *sla, const float *omega,
                             double *fit, hipStream_t st)
{
    const int nin = c.L + c.A;
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
    hipLaunchKernelGGL(ga_ops_kernel, dim3(S * wgs), dim3(kOpPairs), 0, st, c, seed, P, gen, gens, tk, p_cx, p_swap,
                       p_mut, fl, n_fl, pop, fit, next, best_J, best_idx, final_pop, wgs);
    return hipGetLastError();
}

}  // namespace mfi
