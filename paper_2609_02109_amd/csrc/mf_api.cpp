// Host side of libmf: argument validation, the fast path's a-priori error
// bounds, device tables, the search driver (range chunking, splitting on a
// full certification list, the top-k fallback pass) and result merging.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <atomic>
#include <cstring>
#include <limits>
#include <map>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "mf_internal.h"

using namespace mfi;

namespace {
// What one search call holds while it runs: the start and end events of its
// timed kernel, and a pinned host copy of the small-range result block.
struct EventPair {
    hipEvent_t a = nullptr, b = nullptr;
    mfi::DevResult *h_res = nullptr;
};
}  // namespace

struct mf_problem {
    int N = 0, L = 0, A = 0, H1 = 0, H2 = 0;
    bool bf16 = false;
    int act = MF_ACT_IDENTITY;   // output activation of both surrogate outputs
    std::vector<int32_t> K, agg_cols, opt_off;
    int vram_slot = 0;
    float vram_cap = 0.f;
    uint64_t space = 0;
    int64_t wstride = 0;
    int sumK = 0;
    bool fast_ok = false;
    int num_cus = 0;
    int device = 0;
    double wall_khz = 0.0;      // device wall-clock ticks per millisecond
    // device tables: pointers into the caller's buffer (borrowed until destroy)
    void *d_tables = nullptr;
    void *d_scratch = nullptr;   // this device's copy of the no-allocation scratch
    float4 *d_image = nullptr;
    float *d_canon = nullptr, *d_features = nullptr, *d_zeros = nullptr, *d_centre = nullptr;
    double *d_w64 = nullptr;     // packed weights as fp64 (GA fitness)
    double *d_pre = nullptr;     // [sumK][H1] canonical layer-1 chain over the local features (GA fitness)
    std::vector<float> centre;   // aggregate centre per slot (original slot order)
    int32_t *d_agg_cols = nullptr, *d_row_model = nullptr;
    FastLayout lay{};
    FastConst fc{};
    int fast_e1[kMaxN] = {}, fast_e2[kMaxN] = {};   // fast image scales: layer 1 by 2^e1, W2 by 2^e2
    // variant metadata of the full utility (Eq. 3)
    bool has_var = false;
    std::vector<int32_t> n_var;
    float4 *d_vrow = nullptr;    // [sumK][2]: (fmin, fmax, 1/range, Q), (variant bits, reload cost, 0, 0)
    // bf16 fast path
    bool bf_ok = false;
    Bf16Layout blay{};
    Bf16Const bcst{};
    float4 *d_bmodels = nullptr, *d_bg = nullptr;
    float *d_phat = nullptr;
    std::atomic<unsigned long long> call_seq{0};   // sequence numbers of small-range searches
    // timing events: created with the problem, handed to one call at a time
    std::mutex ev_mu;
    std::vector<EventPair> ev_free, ev_all;
};

namespace mfi {

hipError_t ensure_dyn_lds(const void *fn, size_t bytes)
{
    static std::mutex mu;
    static std::map<std::pair<const void *, int>, size_t> done;   // (kernel, device) -> limit set
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> g(mu);
    const auto key = std::make_pair(fn, dev);
    const auto it = done.find(key);
    if (it != done.end() && it->second >= bytes) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) done[key] = bytes;
    return e;
}

}  // namespace mfi

// Device scratch of mf_search_noalloc: a file-scope array, one copy per GPU,
// held until the process ends.  Host code never uses the array's name as an
// address: each device's address comes from hipGetSymbolAddress (scratch_ptr).
static __device__ __align__(256) unsigned char scratch[MF_NOALLOC_SCRATCH_BYTES];

namespace {

// The device address of `scratch` on device `dev` (the current device),
// looked up once per device.
hipError_t scratch_ptr(int dev, void **out)
{
    static std::mutex mu;
    static std::map<int, void *> ptrs;
    std::lock_guard<std::mutex> g(mu);
    const auto it = ptrs.find(dev);
    if (it != ptrs.end()) {
        *out = it->second;
        return hipSuccess;
    }
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    ptrs[dev] = ptr;
    *out = ptr;
    return hipSuccess;
}

bool create_event_pair(EventPair &e)
{
    if (hipEventCreate(&e.a) != hipSuccess) return false;
    if (hipEventCreate(&e.b) != hipSuccess) {
        (void)hipEventDestroy(e.a);
        e.a = nullptr;
        return false;
    }
    // coherent: the finish kernel's stores reach the host while it runs
    if (hipHostMalloc((void **)&e.h_res, sizeof(DevResult), hipHostMallocCoherent) != hipSuccess) e.h_res = nullptr;
    return true;
}

// A pair of the problem's timing events held by one call.  A call finding
// none free creates one more pair for the pool when it may (concurrent calls
// on several streams); otherwise it runs untimed.
class EventLease {
public:
    EventLease(mf_problem *p, bool may_create) : p_(p)
    {
        std::lock_guard<std::mutex> g(p->ev_mu);
        if (!p->ev_free.empty()) {
            ev_ = p->ev_free.back();
            p->ev_free.pop_back();
        } else if (may_create && create_event_pair(ev_)) {
            p->ev_all.push_back(ev_);
        }
    }
    ~EventLease()
    {
        if (!ev_.a) return;
        std::lock_guard<std::mutex> g(p_->ev_mu);
        p_->ev_free.push_back(ev_);
    }
    EventLease(const EventLease &) = delete;
    EventLease &operator=(const EventLease &) = delete;
    hipEvent_t start() const { return ev_.a; }
    hipEvent_t stop() const { return ev_.b; }
    DevResult *host_result() const { return ev_.h_res; }

private:
    mf_problem *p_;
    EventPair ev_{};
};


constexpr double kU32 = 0x1p-24;   // fp32 unit roundoff (round to nearest)
constexpr double kU64 = 0x1p-53;   // fp64 unit roundoff

double gam(double n, double u) { return n * u / (1.0 - n * u); }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool all_finite(const std::vector<float> &v)
{
    for (float x : v)
        if (!std::isfinite(x)) return false;
    return true;
}

bool bf16_exact(float x)
{
    uint32_t b;
    std::memcpy(&b, &x, 4);
    return (b & 0xFFFFu) == 0u;
}

// x rounded to the nearest binary16 value (ties to even), as a double; x
// finite with |x| < 65504.  Subnormal binary16 values are spaced 2^-24.
double f16_rne(double x)
{
    const double a = std::fabs(x);
    if (a == 0.0) return 0.0;
    int e;
    (void)std::frexp(a, &e);                                  // a in [2^(e-1), 2^e)
    const double q = std::ldexp(1.0, std::max(e - 1, -14) - 10);   // spacing at a
    const double r = std::nearbyint(a / q) * q;               // default rounding: to nearest even
    return x < 0 ? -r : r;
}

// IEEE binary16 encoding of a value f16_rne returned.
uint16_t f16_bits(double v)
{
    const uint16_t sign = v < 0 ? 0x8000u : 0u;
    const double a = std::fabs(v);
    if (a < 0x1p-14) return (uint16_t)(sign | (uint16_t)std::lround(a * 0x1p24));   // subnormal (or zero)
    int e;
    const double f = std::frexp(a, &e);                       // a = f 2^e, f in [0.5, 1)
    const int ex = e - 1 + 15;
    const uint32_t mant = (uint32_t)std::lround((2.0 * f - 1.0) * 1024.0);
    return (uint16_t)(sign | (uint16_t)(ex << 10) | (uint16_t)mant);
}

// A weight w (already scaled) as two binary16 pieces w1 = RNE(w), w2 =
// RNE(w - w1); *ew = |w - w1 - w2| (exact).  The matrix cores take binary16
// subnormals as they are (a probe on the MI355X: every product with a
// subnormal operand exact), so subnormal pieces count at their value.
void split_w_f16(double w, double *w1, double *w2, double *ew)
{
    *w1 = f16_rne(w);
    *w2 = f16_rne(w - *w1);   // w - w1 is exact in double
    *ew = std::fabs(w - *w1 - *w2);
}

// Per model: a-priori bounds on |fast fp32 path - canonical fp64| for both
// outputs, and a magnitude bound on throughput.  Each dot product of n terms
// computed as any sequence of n correctly rounded fused multiply-adds (the
// measured behaviour of v_mfma_f32_32x32x2f32 and of v_fma_f32/f64) has error
// <= gamma_n * (|bias| + sum |w||x|) (Higham, Accuracy and Stability of
// Numerical Algorithms, 2nd ed., Sec. 3.1).  Errors of a layer's input
// propagate through |W| (relu is 1-Lipschitz).  Magnitudes use the largest
// |input| over all options and all joint configurations.
//
// Fast path, layer 1: P'[o] = b1 + W1_loc x_o + W1_agg c (fp64 chain of L+A
// terms, rounded to fp32), then A fp32 fmas W1_agg (a - c) onto it, with
// a - c rounded to fp32 (exact on the generator's grid).
// Per aggregate column k (original order): amax[k] bounds |a_k| and amaxc[k]
// bounds |a_k - c_k| over the joint space.
void agg_ranges(const mf_problem &p, const std::vector<float> &F, std::vector<double> &amax,
                std::vector<double> &amaxc)
{
    const int L = p.L, A = p.A;
    amax.assign(A, 0.0);
    amaxc.assign(A, 0.0);
    for (int k = 0; k < A; k++) {
        double smax = 0.0, smin = 0.0, sabs = 0.0;
        for (int j = 0; j < p.N; j++) {
            double mx = -INFINITY, mn = INFINITY, ma = 0.0;
            for (int o = 0; o < p.K[j]; o++) {
                const double v = F[(int64_t)(p.opt_off[j] + o) * L + p.agg_cols[k]];
                mx = std::max(mx, v);
                mn = std::min(mn, v);
                ma = std::max(ma, std::fabs(v));
            }
            smax += mx;
            smin += mn;
            sabs += ma;
        }
        amax[k] = sabs;
        // the fp32 aggregate (model order) is within N u sabs of the exact sum
        amaxc[k] = (std::max(std::fabs(smax - p.centre[k]), std::fabs(smin - p.centre[k])) + 2.0 * p.N * kU32 * sabs) *
                   (1 + 1e-12);
    }
}

// Power-of-two scale 2^ex[k] of each aggregate column's binary16 layer-1
// operand: |2^ex (a - c)| <= 2^14.
std::vector<int> agg_exponents(const std::vector<double> &amaxc)
{
    std::vector<int> ex(amaxc.size(), 0);
    for (size_t k = 0; k < amaxc.size(); k++) {
        if (amaxc[k] > 0.0) ex[k] = (int)std::floor(std::log2(0x1p14 / amaxc[k]));
        ex[k] = std::min(std::max(ex[k], -60), 60);
        while (ex[k] > -60 && amaxc[k] * (1 + kU32) * std::ldexp(1.0, ex[k]) > 0x1p14) ex[k]--;
    }
    return ex;
}

bool model_bounds(const mf_problem &p, const std::vector<float> &F, const std::vector<float> &W, int i,
                  const std::vector<int> &ex, double *b_lat, double *b_thr, double *m_thr, int *e1_out, int *e2_out)
{
    const int L = p.L, A = p.A, H1 = p.H1, H2 = p.H2, nin = L + A;
    const float *w = W.data() + (int64_t)i * p.wstride;
    const float *W1 = w, *b1 = W1 + (int64_t)H1 * nin, *W2 = b1 + H1, *b2 = W2 + (int64_t)H2 * H1, *W3 = b2 + H2,
                *b3 = W3 + 2 * H2;
    std::vector<double> xmax(L, 0.0), amax, amaxc;
    for (int o = 0; o < p.K[i]; o++)
        for (int k = 0; k < L; k++)
            xmax[k] = std::max(xmax[k], (double)std::fabs(F[(int64_t)(p.opt_off[i] + o) * L + k]));
    agg_ranges(p, F, amax, amaxc);
    std::vector<double> M1(H1), e1f(H1), e1c(H1), M2(H2), e2f(H2), e2c(H2), pmax_h(H1);
    for (int h = 0; h < H1; h++) {
        // |P'| over this model's options, and the magnitudes of its fp64 chain
        double pmax = 0.0, pchain = 0.0;
        double cpart = 0.0, cabs = std::fabs((double)b1[h]);
        for (int k = 0; k < A; k++) {
            cpart += (double)W1[(int64_t)h * nin + L + k] * p.centre[k];
            cabs += std::fabs((double)W1[(int64_t)h * nin + L + k] * p.centre[k]);
        }
        for (int o = 0; o < p.K[i]; o++) {
            double v = (double)b1[h] + cpart, va = cabs;
            for (int k = 0; k < L; k++) {
                const double t = (double)W1[(int64_t)h * nin + k] * F[(int64_t)(p.opt_off[i] + o) * L + k];
                v += t;
                va += std::fabs(t);
            }
            pmax = std::max(pmax, std::fabs(v) + 1e-12 * va);
            pchain = std::max(pchain, va);
        }
        double am = 0.0, aw = 0.0, am_full = std::fabs((double)b1[h]);
        for (int k = 0; k < A; k++) {
            const double wa = std::fabs((double)W1[(int64_t)h * nin + L + k]);
            am += wa * amaxc[k];
            aw += wa * amaxc[k];
            am_full += wa * amax[k];
        }
        for (int k = 0; k < L; k++) am_full += std::fabs((double)W1[(int64_t)h * nin + k]) * xmax[k];
        M1[h] = pmax + am;
        pmax_h[h] = pmax;
        e1f[h] = gam(L + A, kU64) * pchain            // fp64 precompute
                 + kU32 * pmax                         // rounding P' to fp32
                 + kU32 * aw                           // rounding a - c to fp32
                 + 0x1p-80;                            // fp32 subnormals under the layer-1 scale
        e1c[h] = gam(nin, kU64) * am_full;             // canonical chain on uncentred inputs
    }
    // Layer 1's aggregate part on binary16 pieces, in scaled units: x_k =
    // 2^ex_k (a_k - c_k) (|x| <= X_k) as x1 + x2 (|x - x1 - x2| <= 2^-21 |x| +
    // 2^-24), w = 2^(e1 - ex_k) W1_agg as w1 + w2 (|w - w1 - w2| = ew), all
    // four cross products on two v_mfma_f32_32x32x16_f16 (one when A <= 4)
    // onto P' = 2^e1 P, each counted as 17 u (|C| + sum |products|) (see
    // layer 2 below).  The
    // scale 2^e1 keeps |2^e1 h1| <= 2^14 and the weight pieces in range.
    std::vector<double> e1m(H1, 0.0);
    double w1a_max = 0.0, x_max0 = 0.0;
    for (int h = 0; h < H1; h++) {
        x_max0 = std::max(x_max0, M1[h] + e1f[h]);
        for (int k = 0; k < A; k++)
            w1a_max = std::max(w1a_max, std::fabs((double)W1[(int64_t)h * nin + L + k]) * std::ldexp(1.0, -ex[k]));
    }
    int e1 = x_max0 > 0.0 ? (int)std::floor(std::log2(0x1p13 / x_max0)) : 0;
    if (w1a_max > 0.0) e1 = std::min(e1, (int)std::floor(std::log2(0x1p14 / w1a_max)));
    e1 = std::min(std::max(e1, -60), 60);
    auto layer1_terms = [&](int e) {
        const double s1 = std::ldexp(1.0, e);
        for (int h = 0; h < H1; h++) {
            double er = 0.0, sp = 0.0;
            for (int k = 0; k < A; k++) {
                const double X = std::ldexp(amaxc[k] * (1 + kU32), ex[k]);
                double w1, w2, ew;
                const double wk = s1 * std::ldexp((double)W1[(int64_t)h * nin + L + k], -ex[k]);
                split_w_f16(wk, &w1, &w2, &ew);
                er += (0x1p-21 * X + 0x1p-24) * (std::fabs(wk) + ew) + X * ew;
                sp += (X * (1.0 + 0x1p-10) + 0x1p-23) * (std::fabs(w1) + std::fabs(w2));
            }
            e1m[h] = (er + gam(A <= 4 ? 17.0 : 34.0, kU32) * (s1 * pmax_h[h] + sp)) / s1;
        }
    };
    for (;;) {
        layer1_terms(e1);
        double xm = 0.0;
        for (int h = 0; h < H1; h++) xm = std::max(xm, M1[h] + e1f[h] + e1m[h]);
        if (xm * std::ldexp(1.0, e1) <= 0x1p14 || e1 <= -60) break;
        e1--;
    }
    for (int h = 0; h < H1; h++) e1f[h] += e1m[h];
    // Layer 2 runs on binary16 pieces in scaled units: x = 2^e1 h1 (fast h1,
    // |x| <= X = 2^e1 (M1 + e1f) <= 2^14) as x1 = x truncated and x2 = (x -
    // x1) rounded to nearest (|x2| <= 2^-10 |x| + 2^-23, |x - x1 - x2| <=
    // 2^-21 |x| + 2^-24, the absolute parts for binary16 subnormals) and
    // w = 2^e2 W2 as w1 + w2 (rounded on the host, |w - w1 - w2| = ew);
    // x w - (x1 w1 + x1 w2 + x2 w1) = x2 w2 + (x - x1 - x2) w + (x1 + x2) ew.
    // Accumulation, 3 H1 / 16 v_mfma_f32_32x32x16_f16 per output: each is
    // counted as 17 u (|C| + sum |products|), what 17 terms aligned to the
    // largest within a window of at least 24 bits, truncated, then rounded
    // once, can lose (a probe on the MI355X over 8 M outputs, exponents of
    // the products spread over 2^30 and cancelling accumulators included,
    // found at most 5.8 u; the matrix core does not round each product sum
    // separately, so the error is not that of one rounding).  The kernel
    // issues the 2 nb small cross products first (nb = H1 / 16 K-blocks),
    // onto the bias B = 2^(e1+e2) |b2| (|C| <= B + Tc, Tc the corrections'
    // magnitude), then the leading products of K-blocks j = 0 .. nb - 1
    // (|C| <= B + Tc + T_0 + ... + T_(j-1)): in all
    // 17 u (3 nb (B + Tc) + Tc + sum_j (nb - j) T_j), the accumulated errors
    // inside C taken by a factor 1 + 2^-10.
    double x_max = 0.0, w_max = 0.0;
    for (int h = 0; h < H1; h++) x_max = std::max(x_max, M1[h] + e1f[h]);
    for (int64_t t = 0; t < (int64_t)H2 * H1; t++) w_max = std::max(w_max, (double)std::fabs(W2[t]));
    if (x_max * std::ldexp(1.0, e1) > 0x1p14) return false;
    int e2 = 0;
    if (w_max > 0.0) e2 = (int)std::floor(std::log2(0x1p14 / w_max));
    e2 = std::min(std::max(e2, -60), 60);
    while (e2 > -60 && w_max * std::ldexp(1.0, e2) > 0x1p14) e2--;
    // W3 / 2^(e1+e2) and b2 2^(e1+e2) must stay normal and finite in fp32
    auto scaled_ok = [&](int es) {
        for (int t = 0; t < 2 * H2; t++) {
            const double a = std::fabs((double)W3[t]) * std::ldexp(1.0, -es);
            if (W3[t] != 0.f && (a < 0x1p-126 || a > 0x1p127)) return false;
        }
        for (int v = 0; v < H2; v++) {
            const double a = std::fabs((double)b2[v]) * std::ldexp(1.0, es);
            if (b2[v] != 0.f && (a < 0x1p-126 || a > 0x1p127)) return false;
        }
        return true;
    };
    // a smaller W2 scale only costs binary16 range at the small end
    while (!scaled_ok(e1 + e2) && e2 > -60 && e1 + e2 > 0) e2--;
    if (!scaled_ok(e1 + e2)) return false;
    *e1_out = e1;
    *e2_out = e2;
    const double s1 = std::ldexp(1.0, e1), s2 = std::ldexp(1.0, e2), S = s1 * s2;
    const int nb = H1 / 16;
    for (int v = 0; v < H2; v++) {
        double m = std::fabs((double)b2[v]), pf = 0.0, pc = 0.0, mc = m, er = 0.0, tc = 0.0, tj[16] = {};
        for (int h = 0; h < H1; h++) {
            const double w = (double)W2[(int64_t)v * H1 + h], aw = std::fabs(w);
            double w1, w2, ew;
            split_w_f16(s2 * w, &w1, &w2, &ew);
            const double X = s1 * (M1[h] + e1f[h]);       // |x1| <= |x| <= X
            const double X2 = 0x1p-10 * (1.0 + 0x1p-10) * X + 0x1p-23;   // |x2|
            er += X2 * std::fabs(w2) + (0x1p-21 * X + 0x1p-24) * s2 * aw + (X * (1.0 + 0x1p-20) + 0x1p-24) * ew;
            tc += std::fabs(w2) * X + std::fabs(w1) * X2;
            tj[h / 16] += std::fabs(w1) * X;
            m += aw * M1[h];
            pf += aw * e1f[h];
            pc += aw * e1c[h];
            mc += aw * (M1[h] + e1c[h]);
        }
        const double B = S * std::fabs((double)b2[v]);
        double acc = 3.0 * nb * (B + tc) + tc;
        for (int j = 0; j < nb; j++) acc += (double)(nb - j) * tj[j];
        M2[v] = m;
        e2f[v] = pf + (er + 17.0 * kU32 * (1.0 + 0x1p-10) * acc) / S;
        e2c[v] = pc + gam(H1, kU64) * mc;
    }
    double out_b[2], out_m = 0.0;
    for (int o = 0; o < 2; o++) {
        double pf = 0.0, pc = 0.0, mf = std::fabs((double)b3[o]), mc = mf, m = mf;
        for (int v = 0; v < H2; v++) {
            const double aw = std::fabs((double)W3[o * H2 + v]);
            pf += aw * e2f[v];
            pc += aw * e2c[v];
            mf += aw * (M2[v] + e2f[v]);
            mc += aw * (M2[v] + e2c[v]);
            m += aw * M2[v];
        }
        // fast layer 3: per-half fma chains of H2/2 terms, one cross add, + b3
        const double ef = pf + gam(H2 / 2 + 2, kU32) * mf;
        const double ec = pc + gam(H2, kU64) * mc;
        out_b[o] = (ef + ec) * 1.01 + 1e-30;
        if (o == 1) out_m = m + ef;
    }
    *b_lat = out_b[0];
    *b_thr = out_b[1];
    *m_thr = out_m;
    return true;
}

// Smallest float >= x.
float f32_up_host(double x)
{
    float f = (float)x;
    if ((double)f < x) f = std::nextafter(f, INFINITY);
    return f;
}

// Per model, the constants of the bf16 path's per-configuration bounds (see
// the bf16 kernel): cst[2 + o] fixed terms of output o (the |b3| part of the
// fp32 layer-3 bound and the fp64 rounding of the canonical layers 2 and 3),
// cst[4 + o] = sum_v |W3[o][v]| |b2[v]|, cst[6 + o] = max_u sum_v
// |W3[o][v]| |W2[v][u]|, cst[8 + o] = max_v |W3[o][v]|; *mag_thr bounds |thr|
// over the joint space.  Layer 1 is identical on both sides (the same fp32
// chain and bf16 rounding).  Layer 3 runs as four partial fp32 chains of H/8
// terms per output, summed pairwise, plus the cross-half add and b3: at most
// H/8 + 4 roundings.
void bf16_bounds(const mf_problem &p, const std::vector<float> &F, const std::vector<float> &W, int i, float *cst,
                 float *mag_thr)
{
    const int L = p.L, A = p.A, H = p.H1, nin = L + A;
    const float *w = W.data() + (int64_t)i * p.wstride;
    const float *W1 = w, *b1 = W1 + (int64_t)H * nin, *W2 = b1 + H, *b2 = W2 + (int64_t)H * H, *W3 = b2 + H,
                *b3 = W3 + 2 * H;
    // largest |input| of model i: its own options' local columns, and per
    // aggregate slot the sum over models of the largest |column value|
    std::vector<double> zmax(nin, 0.0);
    for (int o = 0; o < p.K[i]; o++)
        for (int k = 0; k < L; k++)
            zmax[k] = std::max(zmax[k], (double)std::fabs(F[(int64_t)(p.opt_off[i] + o) * L + k]));
    for (int k = 0; k < A; k++) {
        double s = 0.0;
        for (int j = 0; j < p.N; j++) {
            double m = 0.0;
            for (int o = 0; o < p.K[j]; o++)
                m = std::max(m, (double)std::fabs(F[(int64_t)(p.opt_off[j] + o) * L + p.agg_cols[k]]));
            s += m;
        }
        zmax[L + k] = s;
    }
    // |h1| (fp32 chain, then bf16 rounding), |h2| bounds
    std::vector<double> M1(H), M2(H);
    for (int u = 0; u < H; u++) {
        double m = std::fabs((double)b1[u]);
        for (int k = 0; k < nin; k++) m += std::fabs((double)W1[(int64_t)u * nin + k]) * zmax[k];
        M1[u] = m * (1.0 + gam(nin, kU32)) * (1.0 + 0x1p-8);
    }
    for (int v = 0; v < H; v++) {
        double m = std::fabs((double)b2[v]);
        for (int u = 0; u < H; u++) m += std::fabs((double)W2[(int64_t)v * H + u]) * M1[u];
        M2[v] = m * (1.0 + 1e-12);
    }
    const double g3 = gam(H / 8 + 4, kU32), g64 = gam(H + 1, kU64);
    for (int o = 0; o < 2; o++) {
        double cb = 0.0, e64 = 0.0, m3 = std::fabs((double)b3[o]);
        for (int v = 0; v < H; v++) {
            const double a3 = std::fabs((double)W3[o * H + v]);
            cb += a3 * std::fabs((double)b2[v]);
            e64 += a3 * g64 * M2[v];          // canonical layer 2 (fp64 chain)
            m3 += a3 * M2[v];
        }
        e64 += g64 * m3;                      // canonical layer 3 (fp64 chain)
        double rmax = 0.0;
        for (int u = 0; u < H; u++) {
            double r = 0.0;
            for (int v = 0; v < H; v++)
                r += std::fabs((double)W3[o * H + v]) * std::fabs((double)W2[(int64_t)v * H + u]);
            rmax = std::max(rmax, r);
        }
        cst[2 + o] = f32_up_host((g3 * std::fabs((double)b3[o]) + e64) * 1.01 + 1e-30);
        cst[4 + o] = f32_up_host(cb * (1.0 + 1e-6));
        cst[6 + o] = f32_up_host(rmax * (1.0 + 1e-6));
        double w3max = 0.0;
        for (int v = 0; v < H; v++) w3max = std::max(w3max, std::fabs((double)W3[o * H + v]));
        cst[8 + o] = f32_up_host(w3max);
        if (o == 1) *mag_thr = f32_up_host(m3 * 1.01);
    }
}

uint32_t magic_for(int K) { return K <= 1 ? 0u : (uint32_t)((0x100000000ull / (uint64_t)K) + 1ull); }

// Length of the fast candidate list: twice the top-k (so that the k-th
// canonical value usually clears the list's last upper bound), within the
// kernel's limit.
int choose_kp(int top_k, int max_kp)
{
    int kp = 16;
    while (kp < 2 * top_k && kp < max_kp) kp *= 2;
    return kp;
}

void stride_digits(const mf_problem &p, uint64_t stride, uint32_t *out)
{
    const uint64_t s = stride % p.space;
    uint64_t x = s;
    for (int i = p.N - 1; i >= 0; i--) {
        out[i] = (uint32_t)(x % (uint64_t)p.K[i]);
        x /= (uint64_t)p.K[i];
    }
    for (int i = p.N; i < kMaxN; i++) out[i] = 0;
}

// Workspace layout for one search launch set over n configurations.
struct WsLayout {
    size_t res, work, workJ, collect, lists, counts, cand, entJ, entF, parts, seg, segJ, rec, wtop, total;
    uint32_t work_cap, collect_cap, seg_cap;
    int kp, grid, waves, n_parts, eval_top;
    bool small;   // fp32 path over at most kSmallRange configurations: fast kernel + finish kernel
};

WsLayout ws_layout(const mf_problem &p, uint64_t n, int top_k, uint32_t worklist_cap)
{
    WsLayout w{};
    if (p.bf_ok) {
        w.kp = choose_kp(top_k, 128);
        w.waves = kBf16Waves;
        const uint64_t per_wg = (uint64_t)kBf16Waves * kBf16Tiles * 32;
        const uint64_t g = (n + per_wg - 1) / per_wg;
        w.grid = (int)std::max<uint64_t>(1, std::min<uint64_t>(g, (uint64_t)p.num_cus));
    } else {
        w.kp = choose_kp(top_k, 64);
        w.waves = fast_waves_for(p.N, p.lay, w.kp, p.act);
        const uint64_t tiles = (n + 31) / 32;
        const uint64_t g = (tiles + w.waves - 1) / w.waves;
        w.grid = (int)std::max<uint64_t>(1, std::min<uint64_t>(g, (uint64_t)p.num_cus));
    }
    // certification list: 1/64 of the range, at least 2^20 entries (never
    // more than the range), at most 2^26
    const uint64_t want = std::min<uint64_t>(std::max<uint64_t>(n / 64, (uint64_t)kDefaultWorklist), 1ull << 26);
    uint64_t cap = std::max<uint64_t>(std::min<uint64_t>(want, n), 1024);
    // the caller may bound the list (a full list splits the range)
    if (worklist_cap >= 1) cap = std::min<uint64_t>(cap, (uint64_t)worklist_cap);
    w.work_cap = (uint32_t)cap;
    w.collect_cap = (uint32_t)std::max<uint64_t>(std::min<uint64_t>((uint64_t)kDefaultWorklist, n), 1024);
    size_t o = 0;
    w.res = o; o = align256(o + sizeof(DevResult));
    w.work = o; o = align256(o + (size_t)w.work_cap * 8);
    w.workJ = o; o = align256(o + (size_t)w.work_cap * 4);
    w.collect = o; o = align256(o + (size_t)w.collect_cap * 4);
    w.lists = o; o = align256(o + (size_t)w.grid * w.kp * 8);
    w.counts = o; o = align256(o + (size_t)w.grid * 16);
    w.cand = o; o = align256(o + (size_t)w.kp * 8);
    const size_t n_ent = (size_t)w.kp + w.work_cap + w.collect_cap;
    w.entJ = o; o = align256(o + n_ent * 8);
    w.entF = o; o = align256(o + n_ent * 4);
    // the exact selection runs in two levels over long ranges
    w.n_parts = n > kSelSingleMax ? kSelParts : 1;
    w.parts = o; o = align256(o + (w.n_parts > 1 ? (size_t)w.n_parts * sizeof(SelPart) : 0));
    // small ranges: a certification segment per workgroup (its entries and
    // upper bounds), the record and the best top_k canonical keys of each
    // workgroup.  Each workgroup evaluates canonically its first eval_top list
    // entries and its segment.  eval_top: at least 4 and k/2 + 1
    // (the workgroups scan runs of consecutive configurations, so one of them
    // may hold several of the best), and enough that the evaluated entries of
    // all workgroups cover twice the top-k.  Too few evaluated entries only
    // cost the fallback pass, never exactness.
    w.small = !p.bf_ok && n <= kSmallRange && w.grid < 512;
    w.seg_cap = w.small ? (uint32_t)(((uint64_t)w.work_cap + w.grid - 1) / w.grid) : 0;
    w.eval_top = std::min(w.kp, std::max(std::max(4, top_k / 2 + 1), (2 * top_k + w.grid - 1) / w.grid + 2));
    const size_t n_seg = (size_t)w.seg_cap * (w.small ? w.grid : 0);
    w.seg = o; o = align256(o + n_seg * 8);
    w.segJ = o; o = align256(o + n_seg * 4);
    w.rec = o; o = align256(o + (w.small ? (size_t)w.grid * 64 : 0));
    w.wtop = o; o = align256(o + (w.small ? (size_t)w.grid * top_k * sizeof(K128) : 0));
    w.total = o;
    return w;
}

constexpr uint64_t kMaxLaunch = 1ull << 32;   // offsets within one launch set fit in 32 bits

mf_status hip_status(hipError_t e) { return e == hipSuccess ? MF_OK : MF_EDEVICE; }

// Waits until the finish kernel has published sequence number `seq` in the
// host copy of the result.  The stream is queried every 64 polls: if it has
// finished without the number appearing, or reports an error, the wait ends
// with MF_EDEVICE instead of spinning on.
mf_status wait_done(const DevResult *h, unsigned long long seq, hipStream_t s)
{
    const volatile unsigned long long *flag = &h->done_seq;
    for (unsigned it = 1;; it++) {
        if (*flag == seq) break;
        if ((it & 63u) == 0) {
            const hipError_t q = hipStreamQuery(s);
            if (q == hipSuccess) {
                if (*flag == seq) break;
                return MF_EDEVICE;
            }
            if (q != hipErrorNotReady) return MF_EDEVICE;
        }
        __builtin_ia32_pause();
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    return MF_OK;
}

#define MF_HIP(x)                                         \
    do {                                                  \
        hipError_t e_ = (x);                              \
        if (e_ != hipSuccess) return MF_EDEVICE;          \
    } while (0)

void merge_into(mf_result &acc, const mf_result &part, int k)
{
    acc.n_eval += part.n_eval;
    acc.n_vram += part.n_vram;
    acc.n_feas += part.n_feas;
    acc.n_flagged += part.n_flagged;
    acc.n_topk_collect += part.n_topk_collect;
    acc.n_splits += part.n_splits;
    acc.main_kernel_ms += part.main_kernel_ms;
    std::vector<std::pair<double, uint64_t>> v;
    for (int q = 0; q < acc.n_top; q++) v.push_back({acc.top_J[q], acc.top_idx[q]});
    for (int q = 0; q < part.n_top; q++) v.push_back({part.top_J[q], part.top_idx[q]});
    std::sort(v.begin(), v.end(), [](const auto &x, const auto &y) {
        return x.first > y.first || (x.first == y.first && x.second < y.second);
    });
    acc.n_top = (int32_t)std::min<size_t>(v.size(), (size_t)k);
    for (int q = 0; q < MF_MAX_TOPK; q++) {
        acc.top_idx[q] = q < acc.n_top ? v[q].second : UINT64_MAX;
        acc.top_J[q] = q < acc.n_top ? v[q].first : -INFINITY;
    }
}

void empty_result(mf_result &r)
{
    std::memset(&r, 0, sizeof(r));
    for (int q = 0; q < MF_MAX_TOPK; q++) {
        r.top_idx[q] = UINT64_MAX;
        r.top_J[q] = -INFINITY;
    }
}

ObjArgs obj_args(const mf_problem *p, const mf_objective &o)
{
    ObjArgs a{};
    a.kind = o.kind;
    a.alpha = o.alpha;
    a.beta = o.beta;
    a.delta = o.delta;
    for (int i = 0; i < kMaxN; i++) {
        a.tau[i] = i < p->N ? o.tau[i] : 0.f;
        a.prev[i] = i < p->N ? o.prev_variant[i] : -1;
    }
    a.vrow = p->d_vrow;
    return a;
}

// Launch the fast kernel of the problem's path (fp32 or bf16) over the range,
// list or collect pass described by fa.
hipError_t launch_fast_path(const mf_problem *p, const FastArgs &fa, int grid, int kp, int mode, hipStream_t s)
{
    if (!p->bf_ok) return launch_fast_impl(fa, p->fc, grid, kp, mode, s);
    Bf16Args ba{};
    ba.models = p->d_bmodels;
    ba.g_image = p->d_bg;
    ba.phat = p->d_phat;
    ba.lay = p->blay;
    ba.lo = fa.lo;
    ba.n = fa.n;
    ba.idx_list = fa.idx_list;
    ba.sla = fa.sla;
    ba.omega = fa.omega;
    ba.res = fa.res;
    ba.work = fa.work;
    ba.work_J = fa.work_J;
    ba.work_cap = fa.work_cap;
    ba.collect = fa.collect;
    ba.collect_cap = fa.collect_cap;
    ba.theta = fa.theta;
    ba.wg_lists = fa.wg_lists;
    ba.wg_counts = fa.wg_counts;
    ba.mask = fa.mask;
    ba.pred = fa.pred;
    ba.obj = fa.obj;
    return launch_bf16_impl(ba, p->fc, p->bcst, grid, kp, mode, s);
}

enum RangeOutcome { kRangeOk, kRangeSplit };

// One launch set over [lo, lo + n), n <= 2^32.
mf_status run_range(mf_problem *p, const mf_search_args *args, uint64_t lo, uint64_t n, char *ws, hipStream_t s,
                    const EventLease &ev, mf_result &out, RangeOutcome &outcome)
{
    const WsLayout w = ws_layout(*p, n, args->top_k, args->worklist_cap);
    DevResult *R = reinterpret_cast<DevResult *>(ws + w.res);
    unsigned long long *work = reinterpret_cast<unsigned long long *>(ws + w.work);
    float *workJ = reinterpret_cast<float *>(ws + w.workJ);
    uint32_t *collect = reinterpret_cast<uint32_t *>(ws + w.collect);
    unsigned long long *lists = reinterpret_cast<unsigned long long *>(ws + w.lists);
    unsigned long long *counts = reinterpret_cast<unsigned long long *>(ws + w.counts);
    unsigned long long *cand = reinterpret_cast<unsigned long long *>(ws + w.cand);
    double *entJ = reinterpret_cast<double *>(ws + w.entJ);
    uint32_t *entF = reinterpret_cast<uint32_t *>(ws + w.entF);
    const bool dump = (args->flags & MF_DUMP) != 0;
    const uint64_t dump_off = lo - args->lo;

    FastArgs fa{};
    fa.image = p->d_image;
    fa.image_f4 = p->lay.total_floats / 4;
    fa.lay = p->lay;
    fa.lo = lo;
    fa.n = n;
    fa.total_waves = w.grid * w.waves;
    fa.waves = w.waves;
    stride_digits(*p, (uint64_t)fa.total_waves * 32u, fa.stride_digits);
    fa.sla = args->d_sla;
    fa.omega = args->d_omega;
    fa.res = R;
    fa.work = work;
    fa.work_J = workJ;
    fa.work_cap = w.work_cap;
    fa.collect = collect;
    fa.collect_cap = w.collect_cap;
    fa.wg_lists = lists;
    fa.wg_counts = counts;
    fa.mask = dump ? args->d_mask + dump_off : nullptr;
    fa.pred = dump ? args->d_pred + dump_off * (uint64_t)p->N * 2u : nullptr;
    fa.obj = obj_args(p, args->objective);

    CanonArgs ca{};
    ca.n_models = p->N; ca.L = p->L; ca.A = p->A; ca.H1 = p->H1; ca.H2 = p->H2; ca.bf16 = p->bf16; ca.act = p->act;
    for (int i = 0; i < p->N; i++) { ca.K[i] = p->K[i]; ca.opt_off[i] = p->opt_off[i]; }
    ca.agg_cols = p->d_agg_cols; ca.vram_slot = p->vram_slot; ca.vram_cap = p->vram_cap;
    ca.features = p->d_features; ca.weights = p->d_canon; ca.wstride = p->wstride;
    ca.sla = args->d_sla; ca.omega = args->d_omega;
    ca.lo = lo;
    ca.cand_keys = cand; ca.n_cand_keys = w.kp;
    ca.work = work; ca.work_J = workJ; ca.work_cap = w.work_cap;
    ca.collect = collect; ca.collect_cap = w.collect_cap;
    ca.res = R; ca.top_k = args->top_k; ca.collect_mode = 0;
    ca.ent_J = entJ; ca.ent_flags = entF;
    ca.mask = fa.mask;
    ca.obj = fa.obj;

    SelectArgs sa{};
    sa.top_k = args->top_k; sa.kp = w.kp; sa.cand_keys = cand; sa.work = work; sa.collect = collect;
    sa.work_cap = w.work_cap; sa.collect_cap = w.collect_cap; sa.ent_J = entJ; sa.ent_flags = entF;
    sa.lo = lo; sa.collect_mode = 0; sa.res = R;
    sa.parts = reinterpret_cast<SelPart *>(ws + w.parts);
    sa.n_parts = w.n_parts;

    hipEvent_t ev0 = ev.start(), ev1 = ev.stop();
#define MF_HIP2(x)                                  \
    do {                                            \
        if ((x) != hipSuccess) return MF_EDEVICE;   \
    } while (0)

    DevResult h{};
    float ms = 0.f;
    // the small path's fast kernel keeps its certification tail's buffers
    // after the workgroup lists in LDS
    const size_t ep_bytes = fast_small_epilogue_bytes(p->N);
    const size_t small_lds = fast_dyn_lds(p->lay, w.waves, w.kp, ep_bytes);
    if (w.small && small_lds <= (size_t)kFastLdsMax) {
        // two launches and no memset: the fast kernel leaves per-workgroup
        // lists, counts and certification segments; one workgroup completes
        // the search and writes every field of the result block; the fast
        // kernel's time comes from the workgroups' wall-clock stamps
        fa.small = 1;
        fa.ep_bytes = (int)ep_bytes;
        fa.canon = p->d_canon;
        fa.seg_cap = w.seg_cap;
        fa.seg = reinterpret_cast<unsigned long long *>(ws + w.seg);
        fa.seg_J = reinterpret_cast<float *>(ws + w.segJ);
        fa.wg_rec = reinterpret_cast<unsigned long long *>(ws + w.rec);
        fa.eval_top = w.eval_top;
        fa.wg_k = args->top_k;
        fa.wg_top = reinterpret_cast<K128 *>(ws + w.wtop);
        fa.wstride = p->wstride;
        fa.features = p->d_features;
        fa.agg_cols = p->d_agg_cols;
        fa.n_local = p->L;
        fa.vram_slot = p->vram_slot;
        MF_HIP2(launch_fast_path(p, fa, w.grid, w.kp, kModeSearch, s));
        FinishArgs fin{};
        fin.res = R;
        fin.res_host = ev.host_result();
        fin.seq = p->call_seq.fetch_add(1) + 1;
        if (fin.res_host) fin.res_host->done_seq = 0;
        fin.omega = args->d_omega;
        fin.top_k = args->top_k;
        fin.n_wg = w.grid;
        fin.seg_cap = w.seg_cap;
        fin.work_cap = w.work_cap;
        fin.wg_counts = counts;
        fin.wg_rec = fa.wg_rec;
        fin.wg_top = fa.wg_top;
        MF_HIP2(launch_finish_small(fin, p->fc, s));
        if (fin.res_host) {
            // the finish kernel writes the result into pinned host memory,
            // the sequence number last
            const mf_status ws = wait_done(fin.res_host, fin.seq, s);
            if (ws != MF_OK) return ws;
            std::memcpy(&h, fin.res_host, sizeof(DevResult));
        } else {
            MF_HIP2(hipMemcpyAsync(&h, R, sizeof(DevResult), hipMemcpyDeviceToHost, s));
            MF_HIP2(hipStreamSynchronize(s));
        }
        if (!(h.status & kStatWorkOverflow)) ms = (float)((double)h.fast_ticks / p->wall_khz);
        if (!(h.status & (kStatWorkOverflow | kStatSelfCheck | kStatVerified))) {
            // the fallback reads the certification list in one piece
            GatherArgs ga{};
            ga.n_wg = w.grid;
            ga.seg_cap = w.seg_cap;
            ga.wg_rec = fa.wg_rec;
            ga.seg = fa.seg;
            ga.seg_J = fa.seg_J;
            ga.work_out = work;
            ga.work_J_out = workJ;
            MF_HIP2(launch_gather_small(ga, s));
        }
        fa.small = 0;
        fa.ep_bytes = 0;
    } else {
        MF_HIP2(hipMemsetAsync(R, 0, sizeof(DevResult), s));
        if (ev0) MF_HIP2(hipEventRecord(ev0, s));
        MF_HIP2(launch_fast_path(p, fa, w.grid, w.kp, kModeSearch, s));
        if (ev1) MF_HIP2(hipEventRecord(ev1, s));
        MF_HIP2(launch_merge_lists(lists, w.grid, w.kp, cand, counts, &R->n_vram, s));
        ca.phase = 0;
        MF_HIP2(launch_canonical(ca, w.kp, true, s));
        MF_HIP2(launch_kth_candidate(cand, entJ, entF, w.kp, args->top_k, R, s));
        ca.phase = 1;
        MF_HIP2(launch_canonical(ca, (int)std::min<uint64_t>(w.work_cap, 1u << 20), true, s));
        MF_HIP2(launch_select(sa, s));
        MF_HIP2(hipMemcpyAsync(&h, R, sizeof(DevResult), hipMemcpyDeviceToHost, s));
        MF_HIP2(hipStreamSynchronize(s));
        if (ev0) MF_HIP2(hipEventElapsedTime(&ms, ev0, ev1));
    }

    if (h.status & kStatWorkOverflow) {
        outcome = kRangeSplit;
        return MF_OK;
    }
    if (h.status & kStatSelfCheck) return MF_EINTERNAL;
    uint64_t n_collect = 0;
    if (!(h.status & kStatVerified)) {
        // top-k fallback: gather every sure-feasible configuration whose fast
        // J could reach the k-th canonical value, then select canonically
        fa.theta = h.theta;
        fa.mask = nullptr;
        fa.pred = nullptr;
        MF_HIP2(hipMemsetAsync(&R->n_collect, 0, sizeof(unsigned long long), s));
        if (ev0) MF_HIP2(hipEventRecord(ev0, s));
        MF_HIP2(launch_fast_path(p, fa, w.grid, w.kp, kModeCollect, s));
        if (ev1) MF_HIP2(hipEventRecord(ev1, s));
        ca.collect_mode = 1;
        ca.phase = 1;
        ca.mask = nullptr;
        MF_HIP2(launch_canonical(ca, (int)std::min<uint64_t>((uint64_t)w.work_cap + w.collect_cap, 1u << 20), true, s));
        sa.collect_mode = 1;
        MF_HIP2(launch_select(sa, s));
        DevResult h2{};
        MF_HIP2(hipMemcpyAsync(&h2, R, sizeof(DevResult), hipMemcpyDeviceToHost, s));
        MF_HIP2(hipStreamSynchronize(s));
        float ms2 = 0.f;
        if (ev0) MF_HIP2(hipEventElapsedTime(&ms2, ev0, ev1));
        ms += ms2;
        if (h2.status & kStatCollectOverflow) {
            outcome = kRangeSplit;
            return MF_OK;
        }
        n_collect = h2.n_collect;
        h.n_top = h2.n_top;
        std::memcpy(h.top_idx, h2.top_idx, sizeof(h.top_idx));
        std::memcpy(h.top_J, h2.top_J, sizeof(h.top_J));
    }
#undef MF_HIP2
    empty_result(out);
    out.n_eval = n;
    out.n_vram = h.n_vram;
    out.n_feas = h.n_feas_sure + h.n_feas_cert;
    out.n_flagged = h.n_work;
    out.n_topk_collect = n_collect;
    out.n_top = h.n_top;
    for (int q = 0; q < MF_MAX_TOPK; q++) {
        out.top_idx[q] = q < h.n_top ? h.top_idx[q] : UINT64_MAX;
        out.top_J[q] = q < h.n_top ? h.top_J[q] : -INFINITY;
    }
    out.main_kernel_ms = ms;
    outcome = kRangeOk;
    return MF_OK;
}

mf_status search_range(mf_problem *p, const mf_search_args *args, uint64_t lo, uint64_t n, char *ws, hipStream_t s,
                       const EventLease &ev, mf_result &acc, int depth)
{
    if (n == 0) return MF_OK;
    if (n > kMaxLaunch) {
        const uint64_t h = n / 2;
        mf_status st = search_range(p, args, lo, h, ws, s, ev, acc, depth);
        if (st != MF_OK) return st;
        return search_range(p, args, lo + h, n - h, ws, s, ev, acc, depth);
    }
    mf_result part;
    RangeOutcome oc;
    mf_status st = run_range(p, args, lo, n, ws, s, ev, part, oc);
    if (st != MF_OK) return st;
    if (oc == kRangeSplit) {
        if (n < 2 || depth > 40) return MF_ENOMEM;
        const uint64_t h = n / 2;
        acc.n_splits += 1;
        st = search_range(p, args, lo, h, ws, s, ev, acc, depth + 1);
        if (st != MF_OK) return st;
        return search_range(p, args, lo + h, n - h, ws, s, ev, acc, depth + 1);
    }
    merge_into(acc, part, args->top_k);
    return MF_OK;
}

// ---- fixed observed state (MF_FIXED_STATE)

constexpr uint64_t kFixedChunk = 1ull << 36;   // configurations per scan launch set
constexpr uint32_t kFixedInnerMin = 256;       // inner configurations per block (unless the space is smaller)

struct FixedWs {
    size_t res, rows, pens, prow, lists, counts, total;
    int grid;
};

// Inner models: the shortest suffix whose configurations number at least
// kFixedInnerMin (all models if none does).
void fixed_split(const mf_problem &p, int &n_outer, uint32_t &inner)
{
    uint64_t m = 1;
    int j = p.N;
    while (j > 0 && m < kFixedInnerMin) {
        j--;
        m *= (uint64_t)p.K[j];
    }
    n_outer = j;
    inner = (uint32_t)m;
}

uint64_t fixed_blocks(const mf_problem &p, uint64_t lo, uint64_t n, uint64_t &block0)
{
    int n_outer;
    uint32_t M;
    fixed_split(p, n_outer, M);
    block0 = lo / M;
    const uint64_t hi = lo + n;
    const uint64_t block_end = hi / M + (hi % M != 0 ? 1 : 0);
    return block_end - block0;
}

// One wave per block at least; at most the workgroups the CUs hold at once
// (every wave gets the same number of blocks, so one resident round).
// Workgroups of the scan: at most wgs_per_cu per CU.  Every wave takes the
// same number of consecutive blocks where a grid of wgs_per_cu or
// wgs_per_cu - 1 workgroups per CU allows it (measured on the MI355X: an even
// split beats one more workgroup per CU with a ragged one, e.g. the 24^6
// scan on 3 per CU, the 16^8 one on 4); otherwise the largest grid.
int fixed_grid(const mf_problem &p, uint64_t n_blocks, int wgs_per_cu)
{
    const uint64_t g = (n_blocks + kFixedWaves - 1) / kFixedWaves;
    for (int w = wgs_per_cu; w >= 1 && w >= wgs_per_cu - 1; w--) {
        const uint64_t waves = (uint64_t)p.num_cus * w * kFixedWaves;
        if (waves <= n_blocks && n_blocks % waves == 0) return (int)((uint64_t)p.num_cus * w);
    }
    return (int)std::max<uint64_t>(1, std::min<uint64_t>(g, (uint64_t)p.num_cus * wgs_per_cu));
}

FixedWs fixed_ws_layout(const mf_problem &p, int grid, int top_k)
{
    FixedWs w{};
    w.grid = grid;
    size_t o = 0;
    w.res = o; o = align256(o + sizeof(DevResult));
    w.rows = o; o = align256(o + (size_t)p.sumK * sizeof(FixedRow));
    w.pens = o; o = align256(o + (size_t)p.sumK * sizeof(FixedPen));
    w.prow = o; o = align256(o + (size_t)p.sumK * 8);
    w.lists = o; o = align256(o + (size_t)grid * top_k * sizeof(K128));
    w.counts = o; o = align256(o + (size_t)grid * 16);
    w.total = o;
    return w;
}

size_t fixed_ws_bytes(const mf_problem &p, int top_k)
{
    return fixed_ws_layout(p, p.num_cus * kFixedMaxWgsPerCu, top_k).total;
}

// The search with the aggregate input held at args->state: one table of
// canonical per-row terms, then scans of the joint space in chunks.
// Shape, block split and table pointers of a fixed-state (or static) scan.
FixedArgs fixed_base(const mf_problem *p, const mf_objective &objective, int top_k)
{
    FixedArgs a{};
    a.n_models = p->N; a.L = p->L; a.A = p->A; a.H1 = p->H1; a.H2 = p->H2; a.bf16 = p->bf16; a.sumK = p->sumK;
    a.act = p->act;
    for (int i = 0; i < p->N; i++) {
        a.K[i] = p->K[i];
        a.opt_off[i] = p->opt_off[i];
        a.magic[i] = magic_for(p->K[i]);
    }
    fixed_split(*p, a.n_outer, a.inner);
    for (int t = 0; t < p->N - a.n_outer; t++) {
        a.in_K[t] = p->K[a.n_outer + t];
        a.in_off[t] = p->opt_off[a.n_outer + t];
        a.in_magic[t] = magic_for(p->K[a.n_outer + t]);
    }
    // lane-constant last digit: two inner models, the last with a power of
    // two options dividing 64, and the block whole pairs of 64-tiles
    a.lc_shift = -1;
    if (p->N - a.n_outer == 2 && a.inner % 128 == 0) {
        const int kb = a.in_K[1];
        for (int sh = 0; sh <= 6; sh++)
            if (kb == (1 << sh)) a.lc_shift = sh;
    }
    a.row_model = p->d_row_model;
    a.features = p->d_features;
    a.weights = p->d_canon;
    a.wstride = p->wstride;
    a.vram_col = p->agg_cols[p->vram_slot];
    a.vram_cap = p->vram_cap;
    a.top_k = top_k;
    a.obj = obj_args(p, objective);
    return a;
}

mf_status search_fixed(mf_problem *p, const mf_search_args *args, char *ws, hipStream_t s, const EventLease &ev,
                       mf_result &acc)
{
    if (args->hi == args->lo) return MF_OK;
    const FixedWs w = fixed_ws_layout(*p, p->num_cus * kFixedMaxWgsPerCu, args->top_k);
    FixedArgs a = fixed_base(p, args->objective, args->top_k);
    for (int k = 0; k < p->A; k++) a.state[k] = args->state[k];
    a.sla = args->d_sla;
    a.omega = args->d_omega;
    a.rows = reinterpret_cast<FixedRow *>(ws + w.rows);
    a.pens = reinterpret_cast<FixedPen *>(ws + w.pens);
    a.pred_rows = reinterpret_cast<float2 *>(ws + w.prow);
    a.wg_lists = reinterpret_cast<K128 *>(ws + w.lists);
    a.wg_counts = reinterpret_cast<unsigned long long *>(ws + w.counts);
    a.res = reinterpret_cast<DevResult *>(ws + w.res);
    const bool dump = (args->flags & MF_DUMP) != 0;

    hipEvent_t ev0 = ev.start(), ev1 = ev.stop();
    mf_status st = MF_OK;
    for (uint64_t lo = args->lo; lo < args->hi;) {
        const uint64_t n = std::min<uint64_t>(args->hi - lo, kFixedChunk);
        a.lo = lo;
        a.n = n;
        a.n_blocks = fixed_blocks(*p, lo, n, a.block0);
        a.part_block_lo = lo % a.inner ? lo / a.inner : ~0ull;
        a.part_block_hi = (lo + n) % a.inner ? (lo + n) / a.inner : ~0ull;
        a.mask = dump ? args->d_mask + (lo - args->lo) : nullptr;
        a.pred = dump ? args->d_pred + (lo - args->lo) * (uint64_t)p->N * 2u : nullptr;
        // the scan kernel depends on these fields: its occupancy is queried
        // with them set (blocks per wave at one workgroup per CU, a bound)
        const uint64_t waves1 = (uint64_t)p->num_cus * kFixedWaves;
        a.blocks_per_wave = (a.n_blocks + waves1 - 1) / waves1;
        const int wgs_per_cu = fixed_wgs_per_cu(a);
        const int grid = fixed_grid(*p, a.n_blocks, wgs_per_cu);
        const uint64_t waves = (uint64_t)grid * kFixedWaves;
        a.blocks_per_wave = (a.n_blocks + waves - 1) / waves;
        DevResult h{};
        float ms = 0.f;
        if (hipMemsetAsync(a.res, 0, sizeof(DevResult), s) != hipSuccess ||
            launch_fixed(a, grid, lo == args->lo, s, ev0, ev1) != hipSuccess ||
            hipMemcpyAsync(&h, a.res, sizeof(DevResult), hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess ||
            (ev0 && hipEventElapsedTime(&ms, ev0, ev1) != hipSuccess)) {
            st = MF_EDEVICE;
            break;
        }
        if (!(h.status & kStatVerified)) { st = MF_EINTERNAL; break; }
        mf_result part;
        empty_result(part);
        part.n_eval = n;
        part.n_vram = h.n_vram;
        part.n_feas = h.n_feas_sure;
        part.n_top = h.n_top;
        for (int q = 0; q < h.n_top; q++) {
            part.top_idx[q] = h.top_idx[q];
            part.top_J[q] = h.top_J[q];
        }
        part.main_kernel_ms = ms;
        merge_into(acc, part, args->top_k);
        lo += n;
    }
    return st;
}

// ---- static (multi-step) search

struct StaticWs {
    size_t res, rows, pens, prow, lists, counts, total;
};

StaticWs static_ws_layout(const mf_problem &p, int n_steps, int top_k)
{
    StaticWs w{};
    const size_t tr = (size_t)n_steps * p.sumK;
    size_t o = 0;
    w.res = o; o = align256(o + sizeof(DevResult));
    w.rows = o; o = align256(o + tr * sizeof(FixedRow));
    w.pens = o; o = align256(o + tr * sizeof(FixedPen));
    w.prow = o; o = align256(o + (size_t)p.sumK * 8);
    w.lists = o; o = align256(o + (size_t)p.num_cus * kFixedMaxWgsPerCu * top_k * sizeof(K128));
    w.counts = o; o = align256(o + (size_t)p.num_cus * kFixedMaxWgsPerCu * 16);
    w.total = o;
    return w;
}

// static LDS of the static scan kernel besides the dynamic part
constexpr size_t kStaticLdsFixed = 4 * kMaxN * 2 + 4 * kFixedWaves * kMaxN + (8 + 4) * kFixedWaves * MF_MAX_STEPS;

mf_status check_objective(const mf_problem *p, const mf_objective &o)
{
    if (o.kind != MF_OBJ_LINEAR && o.kind != MF_OBJ_EQ3) return MF_EINVAL;
    if (o.kind == MF_OBJ_EQ3) {
        if (!p->has_var) return MF_EINVAL;
        if (!std::isfinite(o.alpha) || !std::isfinite(o.beta) || !std::isfinite(o.delta) || o.beta < 0.f)
            return MF_EINVAL;
        for (int i = 0; i < p->N; i++) {
            if (std::isnan(o.tau[i]) || o.tau[i] == INFINITY) return MF_EINVAL;
            if (o.prev_variant[i] < -1 || o.prev_variant[i] >= p->n_var[i]) return MF_EINVAL;
        }
    }
    return MF_OK;
}

mf_status check_static_args(const mf_problem *p, const mf_static_args *a, bool search)
{
    if (!p || !a) return MF_EINVAL;
    if (a->n_steps < 1 || a->n_steps > MF_MAX_STEPS) return MF_EINVAL;
    if (!a->d_sla || !a->d_omega || !a->h_state) return MF_EINVAL;
    for (int64_t t = 0; t < (int64_t)a->n_steps * p->A; t++)
        if (!std::isfinite(a->h_state[t])) return MF_EINVAL;
    mf_status st = check_objective(p, a->objective);
    if (st != MF_OK) return st;
    if (search) {
        if (a->lo > a->hi) return MF_EINVAL;
        if (a->hi > p->space) return MF_EOVERFLOW;
        if (a->top_k < 1 || a->top_k > MF_MAX_TOPK) return MF_EINVAL;
        if (a->d_mask && a->hi - a->lo > (1ull << 31)) return MF_EINVAL;
    }
    if (static_lds_bytes(a->n_steps, p->sumK, p->N, a->objective.kind != MF_OBJ_LINEAR) + kStaticLdsFixed > 163840)
        return MF_EUNSUPPORTED;
    return MF_OK;
}

// Per-step tables: step t's observed state, bounds and previous deployment
// (the objective's at step 0, none afterwards: the configuration is its own).
mf_status static_setup(mf_problem *p, const mf_static_args *args, char *ws, int top_k, hipStream_t s, StaticArgs &sa)
{
    const StaticWs w = static_ws_layout(*p, args->n_steps, top_k);
    FixedArgs a = fixed_base(p, args->objective, top_k);
    a.rows = nullptr;
    a.pred_rows = reinterpret_cast<float2 *>(ws + w.prow);
    a.wg_lists = reinterpret_cast<K128 *>(ws + w.lists);
    a.wg_counts = reinterpret_cast<unsigned long long *>(ws + w.counts);
    a.res = reinterpret_cast<DevResult *>(ws + w.res);
    sa = StaticArgs{};
    sa.n_steps = args->n_steps;
    sa.omega_steps = args->d_omega;
    sa.rows_steps = reinterpret_cast<FixedRow *>(ws + w.rows);
    sa.pens_steps = reinterpret_cast<FixedPen *>(ws + w.pens);
    for (int t = 0; t < args->n_steps; t++) {
        FixedArgs ft = a;
        for (int k = 0; k < p->A; k++) ft.state[k] = args->h_state[(size_t)t * p->A + k];
        ft.sla = args->d_sla + (size_t)t * p->N;
        ft.omega = args->d_omega + (size_t)t * p->N;
        ft.rows = sa.rows_steps + (size_t)t * p->sumK;
        ft.pens = sa.pens_steps + (size_t)t * p->sumK;
        if (t > 0)
            for (int i = 0; i < kMaxN; i++) ft.obj.prev[i] = -1;
        if (launch_fixed_table(ft, s) != hipSuccess) return MF_EDEVICE;
    }
    a.sla = args->d_sla;
    a.omega = args->d_omega;
    sa.f = a;
    return MF_OK;
}

mf_status search_static(mf_problem *p, const mf_static_args *args, char *ws, hipStream_t s, mf_result &acc)
{
    if (args->hi == args->lo) return MF_OK;
    StaticArgs sa;
    mf_status st = static_setup(p, args, ws, args->top_k, s, sa);
    if (st != MF_OK) return st;
    const int wgs_per_cu = static_wgs_per_cu(sa);
    const EventLease ev(p, true);
    hipEvent_t ev0 = ev.start(), ev1 = ev.stop();
    for (uint64_t lo = args->lo; lo < args->hi;) {
        const uint64_t n = std::min<uint64_t>(args->hi - lo, kFixedChunk);
        FixedArgs &a = sa.f;
        a.lo = lo;
        a.n = n;
        a.n_blocks = fixed_blocks(*p, lo, n, a.block0);
        const int grid = fixed_grid(*p, a.n_blocks, wgs_per_cu);
        const uint64_t waves = (uint64_t)grid * kFixedWaves;
        a.blocks_per_wave = (a.n_blocks + waves - 1) / waves;
        a.mask = args->d_mask ? args->d_mask + (lo - args->lo) : nullptr;
        DevResult h{};
        float ms = 0.f;
        if (hipMemsetAsync(a.res, 0, sizeof(DevResult), s) != hipSuccess ||
            launch_static(sa, grid, s, ev0, ev1) != hipSuccess ||
            hipMemcpyAsync(&h, a.res, sizeof(DevResult), hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess ||
            (ev0 && hipEventElapsedTime(&ms, ev0, ev1) != hipSuccess)) {
            st = MF_EDEVICE;
            break;
        }
        if (!(h.status & kStatVerified)) { st = MF_EINTERNAL; break; }
        mf_result part;
        empty_result(part);
        part.n_eval = n;
        part.n_vram = h.n_vram;
        part.n_feas = h.n_feas_sure;
        part.n_top = h.n_top;
        for (int q = 0; q < h.n_top; q++) {
            part.top_idx[q] = h.top_idx[q];
            part.top_J[q] = h.top_J[q];
        }
        part.main_kernel_ms = ms;
        merge_into(acc, part, args->top_k);
        lo += n;
    }
    return st;
}

// ---- problem tables

// Shape of a description: option counts, first row of each model, |Lambda|.
struct Shape {
    std::vector<int32_t> K, opt_off;
    int sumK = 0;
    uint64_t space = 0;
    int64_t wstride = 0;
};

mf_status check_desc(const mf_desc *desc, Shape &sh)
{
    if (!desc) return MF_EINVAL;
    const int N = desc->n_models, L = desc->n_local, A = desc->n_agg, H1 = desc->hidden1, H2 = desc->hidden2;
    if (N < 1 || N > MF_MAX_MODELS || L < 1 || A < 1 || A > MF_MAX_AGG || L + A > 64 || H1 < 1 || H1 > 256 || H2 < 1 ||
        H2 > 256 || !desc->h_n_options || !desc->h_agg_cols)
        return MF_EINVAL;
    // the enum field is read through its integer representation: a C caller
    // may store any int there, which a C++ enum load may not see
    int dtype;
    static_assert(sizeof dtype == sizeof desc->dtype, "mf_dtype is int-sized");
    std::memcpy(&dtype, &desc->dtype, sizeof dtype);
    if (dtype != MF_F32 && dtype != MF_BF16) return MF_EINVAL;
    if (desc->output_act != MF_ACT_IDENTITY && desc->output_act != MF_ACT_SIGMOID) return MF_EINVAL;
    if (desc->vram_slot < 0 || desc->vram_slot >= A || !std::isfinite(desc->vram_cap)) return MF_EINVAL;
    sh.K.assign(desc->h_n_options, desc->h_n_options + N);
    sh.opt_off.clear();
    uint64_t space = 1;
    int sumK = 0;
    for (int i = 0; i < N; i++) {
        const int k = sh.K[i];
        if (k < 1 || k > 255) return MF_EINVAL;
        if (space > UINT64_MAX / (uint64_t)k) return MF_EOVERFLOW;
        space *= (uint64_t)k;
        sh.opt_off.push_back(sumK);
        sumK += k;
    }
    for (int k = 0; k < A; k++)
        if (desc->h_agg_cols[k] < 0 || desc->h_agg_cols[k] >= L) return MF_EINVAL;
    sh.sumK = sumK;
    sh.space = space;
    sh.wstride = (int64_t)H1 * (L + A) + H1 + (int64_t)H2 * H1 + H2 + 2 * H2 + 2;
    return MF_OK;
}

// Where each table sits in the caller's device buffer (byte offsets, 256-byte
// aligned).  A function of the description alone, so that the buffer can be
// sized before creation.
struct TableLayout {
    bool fast_ok = false, bf_ok = false;
    FastLayout lay{};
    Bf16Layout blay{};
    size_t o_pre = 0;   // [sumK][H1] doubles: canonical layer-1 chain over each option's local features
    size_t o_img = 0, o_can = 0, o_fea = 0, o_agg = 0, o_rm = 0, o_z = 0, o_c = 0, o_w64 = 0, o_bm = 0, o_bg = 0,
           o_ph = 0, o_vr = 0, total = 0;
};

TableLayout table_layout(const mf_desc &d, const Shape &sh)
{
    TableLayout t;
    const int N = d.n_models, L = d.n_local, A = d.n_agg, H1 = d.hidden1, H2 = d.hidden2, sumK = sh.sumK;
    const bool bf16 = d.dtype == MF_BF16;
    const int H = H1;
    // fp32 fast path: H1 == H2 in {32, 64}, A in {2,4,6,8}, the image within LDS
    t.fast_ok = !bf16 && H1 == H2 && fast_kernel_supported(N, A, H1, 64);
    if (t.fast_ok) {
        FastLayout &ly = t.lay;
        ly.H = H; ly.A = A; ly.AP = 8; ly.MB = H / 32; ly.S1 = A / 2; ly.PST = H + 4;
        int o = 0;
        ly.off_w1a = o; o += N * ly.MB * 64 * (A <= 4 ? 2 : 4);
        ly.off_b2 = o; o += N * H;
        ly.off_w2 = o; o += N * H * H;
        ly.off_w3 = o; o += N * 2 * H;
        ly.off_b3 = o; o += N * 4;
        ly.off_p = o; o += sumK * ly.PST;
        ly.off_g = o; o += sumK * ly.AP;
        ly.off_c = o; o += 8;
        ly.total_floats = (o + 3) & ~3;
        if (fast_dyn_lds(ly, kSearchWaves, 64, 0) > (size_t)kFastLdsMax) t.fast_ok = false;
        // the canonical first layer of every model goes into the image when
        // the image, 16 waves' lists and the small-range tail still fit
        ly.off_c1 = -1;
        ly.off_feat = -1;
        ly.c1_stride = (int)((sh.wstride + 3) & ~(int64_t)3);
        const int with_c1 = (ly.total_floats + N * ly.c1_stride + sumK * L + 3) & ~3;
        if ((size_t)with_c1 * 4 + kFastPar * 4 + (size_t)kSearchWavesWide * 64 * 8 + fast_small_epilogue_bytes(N) <=
            (size_t)kFastLdsMax) {
            ly.off_c1 = ly.total_floats;
            ly.off_feat = ly.off_c1 + N * ly.c1_stride;
            ly.total_floats = with_c1;
        }
    }
    // bf16 fast path: H1 == H2 in {64, 128, 256}, A in {2,4,6,8}
    t.bf_ok = bf16 && H1 == H2 && bf16_kernel_supported(N, A, H1);
    if (t.bf_ok) {
        t.blay = bf16_layout(H, A, sumK);
        if (bf16_lds_bytes(t.blay, 128) > 163840) t.bf_ok = false;
    }
    const size_t n_img = t.fast_ok ? (size_t)t.lay.total_floats : 0;
    const size_t n_w = (size_t)N * sh.wstride;
    const size_t n_bimg = t.bf_ok ? (size_t)N * t.blay.model_floats : 0;
    const size_t n_bg = t.bf_ok ? (size_t)sumK * 8 + t.blay.gv_floats : 0;
    const size_t n_phat = t.bf_ok ? (size_t)sumK * t.blay.PST : 0;
    const size_t n_vrow = d.variants ? (size_t)sumK * 8 : 0;
    size_t off = 0;
    t.o_img = off; off = align256(off + n_img * 4);
    t.o_can = off; off = align256(off + n_w * 4);
    t.o_fea = off; off = align256(off + (size_t)sumK * L * 4);
    t.o_agg = off; off = align256(off + (size_t)A * 4);
    t.o_rm = off; off = align256(off + (size_t)sumK * 4);
    t.o_z = off; off = align256(off + 64 * 4);
    t.o_c = off; off = align256(off + (size_t)A * 4);
    t.o_w64 = off; off = align256(off + n_w * 8);
    t.o_pre = off; off = align256(off + (size_t)sumK * d.hidden1 * 8);
    t.o_bm = off; off = align256(off + n_bimg * 4);
    t.o_bg = off; off = align256(off + n_bg * 4);
    t.o_ph = off; off = align256(off + n_phat * 4);
    t.o_vr = off; off = align256(off + n_vrow * 4);
    t.total = off;
    return t;
}

}  // namespace

extern "C" {


const char *mf_status_string(mf_status s)
{
    // A C caller may pass any int; in C++ an enum object holding a value
    // outside the enumerators' range is undefined, so the argument is read
    // through its integer representation.
    int v;
    static_assert(sizeof v == sizeof s, "mf_status is int-sized");
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
        case MF_OK: return "MF_OK";
        case MF_EINVAL: return "MF_EINVAL: invalid argument";
        case MF_ENOMEM: return "MF_ENOMEM: workspace too small or allocation failed";
        case MF_EDEVICE: return "MF_EDEVICE: HIP runtime call or kernel launch failed";
        case MF_EUNSUPPORTED: return "MF_EUNSUPPORTED: shape not supported by the kernels";
        case MF_EOVERFLOW: return "MF_EOVERFLOW: joint space or range does not fit";
        case MF_EINTERNAL: return "MF_EINTERNAL: fast-path self-check failed";
        case MF_ESCRATCH: return "MF_ESCRATCH: the search needs more workspace than mf_search_noalloc's scratch holds";
    }
    return "unknown mf_status";
}

mf_status mf_problem_bytes(const mf_desc *desc, size_t *bytes)
{
    if (!bytes) return MF_EINVAL;
    Shape sh;
    const mf_status st = check_desc(desc, sh);
    if (st != MF_OK) return st;
    *bytes = table_layout(*desc, sh).total;
    return MF_OK;
}

mf_status mf_problem_create(const mf_desc *desc, const float *d_features, const float *d_weights, void *d_tables,
                            size_t table_bytes, void *stream, mf_problem **out)
{
    if (!desc || !d_features || !d_weights || !d_tables || !out) return MF_EINVAL;
    *out = nullptr;
    Shape sh;
    const mf_status st0 = check_desc(desc, sh);
    if (st0 != MF_OK) return st0;
    const TableLayout tl = table_layout(*desc, sh);
    if (table_bytes < tl.total) return MF_ENOMEM;
    if (((uintptr_t)d_tables & 255u) != 0) return MF_EINVAL;
    const int N = desc->n_models, L = desc->n_local, A = desc->n_agg, H1 = desc->hidden1, H2 = desc->hidden2;
    mf_problem *p = new (std::nothrow) mf_problem();
    if (!p) return MF_ENOMEM;
    p->N = N; p->L = L; p->A = A; p->H1 = H1; p->H2 = H2;
    p->bf16 = desc->dtype == MF_BF16;
    p->act = desc->output_act;
    p->vram_slot = desc->vram_slot;
    p->vram_cap = desc->vram_cap;
    p->K = sh.K;
    p->opt_off = sh.opt_off;
    p->agg_cols.assign(desc->h_agg_cols, desc->h_agg_cols + A);
    p->space = sh.space;
    p->sumK = sh.sumK;
    p->wstride = sh.wstride;
    const int sumK = sh.sumK, nin = L + A;

    // the caller's inputs, read in the order of `stream`
    hipStream_t s = (hipStream_t)stream;
    std::vector<float> F((size_t)sumK * L), W((size_t)N * p->wstride);
    if (hipMemcpyAsync(F.data(), d_features, F.size() * 4, hipMemcpyDefault, s) != hipSuccess ||
        hipMemcpyAsync(W.data(), d_weights, W.size() * 4, hipMemcpyDefault, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) {
        delete p;
        return MF_EINVAL;
    }
    if (!all_finite(F) || !all_finite(W)) { delete p; return MF_EINVAL; }

    // every table is written into one host image of the caller's buffer,
    // uploaded with one copy (zero where nothing is written)
    std::vector<unsigned char> himg(tl.total, 0);
    auto at_f = [&](size_t off) { return reinterpret_cast<float *>(himg.data() + off); };

    if (desc->variants) {
        const mf_variants *mv = desc->variants;
        if (!mv->h_variant || !mv->h_n_variants || !mv->h_fmin || !mv->h_fmax || !mv->h_quality ||
            !mv->h_reload_cost) { delete p; return MF_EINVAL; }
        p->n_var.assign(mv->h_n_variants, mv->h_n_variants + N);
        float *vrow = at_f(tl.o_vr);
        for (int i = 0; i < N; i++) {
            const int nv = p->n_var[i];
            const float c = mv->h_reload_cost[i];
            if (nv < 1 || nv > MF_MAX_VARIANTS || !std::isfinite(c) || c < 0.f) { delete p; return MF_EINVAL; }
            for (int v = 0; v < nv; v++) {
                const float lo = mv->h_fmin[i * MF_MAX_VARIANTS + v], hi = mv->h_fmax[i * MF_MAX_VARIANTS + v];
                const float q = mv->h_quality[i * MF_MAX_VARIANTS + v];
                if (!std::isfinite(lo) || !std::isfinite(hi) || !std::isfinite(q) || !(lo < hi) ||
                    !std::isfinite((double)hi - (double)lo) || !std::isfinite(1.0 / ((double)hi - (double)lo))) {
                    delete p;
                    return MF_EINVAL;
                }
            }
            for (int o = 0; o < p->K[i]; o++) {
                const int r = p->opt_off[i] + o, v = mv->h_variant[r];
                if (v < 0 || v >= nv) { delete p; return MF_EINVAL; }
                const float lo = mv->h_fmin[i * MF_MAX_VARIANTS + v], hi = mv->h_fmax[i * MF_MAX_VARIANTS + v];
                float *e = vrow + (size_t)r * 8;
                e[0] = lo;
                e[1] = hi;
                e[2] = (float)(1.0 / ((double)hi - (double)lo));
                e[3] = mv->h_quality[i * MF_MAX_VARIANTS + v];
                std::memcpy(&e[4], &v, 4);
                e[5] = c;
            }
        }
        p->has_var = true;
    }
    if (p->bf16) {
        for (int i = 0; i < N; i++) {
            const float *w = W.data() + (int64_t)i * p->wstride;
            const int64_t n1 = (int64_t)H1 * nin, n2 = (int64_t)H2 * H1;
            for (int64_t t = 0; t < n1; t++)
                if (!bf16_exact(w[t])) { delete p; return MF_EINVAL; }
            for (int64_t t = 0; t < n2; t++)
                if (!bf16_exact(w[n1 + H1 + t])) { delete p; return MF_EINVAL; }
            for (int64_t t = 0; t < 2 * H2; t++)
                if (!bf16_exact(w[n1 + H1 + n2 + H2 + t])) { delete p; return MF_EINVAL; }
        }
    }
    int wall_rate = 0;
    if (hipGetDevice(&p->device) != hipSuccess ||
        hipDeviceGetAttribute(&p->num_cus, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess ||
        hipDeviceGetAttribute(&wall_rate, hipDeviceAttributeWallClockRate, p->device) != hipSuccess ||
        scratch_ptr(p->device, &p->d_scratch) != hipSuccess) {
        delete p;
        return MF_EDEVICE;
    }
    p->wall_khz = wall_rate > 0 ? (double)wall_rate : 1e5;

    // aggregate centre per slot: the mean of the slot over the joint space
    // (sum over models of the mean option value), rounded to the 2^-14 grid
    p->centre.assign(A, 0.f);
    for (int k = 0; k < A; k++) {
        double m = 0.0;
        for (int i = 0; i < N; i++) {
            double s1 = 0.0;
            for (int o = 0; o < p->K[i]; o++) s1 += F[(int64_t)(p->opt_off[i] + o) * L + p->agg_cols[k]];
            m += s1 / p->K[i];
        }
        p->centre[k] = (float)(std::nearbyint(m * 16384.0) / 16384.0);
    }

    // ---- fast path (fp32, H1 == H2 in {32, 64}, A in {2,4,6,8})
    p->fast_ok = tl.fast_ok;
    p->lay = tl.lay;
    const int H = H1;
    const FastLayout &ly = p->lay;
    if (p->fast_ok) {
        std::vector<double> amax_all, amaxc_all;
        agg_ranges(*p, F, amax_all, amaxc_all);
        const std::vector<int> ex = agg_exponents(amaxc_all);
        for (int i = 0; i < N && p->fast_ok; i++)
            if (!model_bounds(*p, F, W, i, ex, &p->fc.bound_lat[i], &p->fc.bound_thr[i], &p->fc.mag_thr[i],
                              &p->fast_e1[i], &p->fast_e2[i]))
                p->fast_ok = false;   // no binary16 scaling fits this model's ranges
    }
    if (p->fast_ok) {
        float *img = at_f(tl.o_img);
        std::vector<double> amax_all, amaxc_all;
        agg_ranges(*p, F, amax_all, amaxc_all);
        const std::vector<int> ex = agg_exponents(amaxc_all);
        // internal aggregate slot order: the VRAM slot first
        std::vector<int> perm;
        perm.push_back(p->vram_slot);
        for (int k = 0; k < A; k++)
            if (k != p->vram_slot) perm.push_back(k);
        for (int i = 0; i < N; i++) {
            const float *w = W.data() + (int64_t)i * p->wstride;
            const float *W1 = w, *b1 = W1 + (int64_t)H * nin, *W2 = b1 + H, *b2 = W2 + (int64_t)H * H,
                        *W3 = b2 + H, *b3 = W3 + 2 * H;
            // power-of-two scales (exact): 2^e1 on layer 1, 2^e2 on W2, so
            // the layer-2 accumulator holds 2^(e1+e2) z2 and W3 takes it back
            const int e1 = p->fast_e1[i], e2 = p->fast_e2[i];
            const double s1 = std::ldexp(1.0, e1), s2 = std::ldexp(1.0, e2), S = s1 * s2;
            // layer 1's aggregate columns: per (block, lane) w1 of the lane
            // half's internal slots 2j + l/32 (j < ns: 4 slots, or 2 when
            // A <= 4), then their w2
            const int ns = A <= 4 ? 2 : 4;
            uint16_t *w1p = reinterpret_cast<uint16_t *>(img + ly.off_w1a + i * (ly.MB * 64 * ns));
            for (int mb = 0; mb < ly.MB; mb++)
                for (int l = 0; l < 64; l++)
                    for (int j = 0; j < ns; j++) {
                        const int k = 2 * j + l / 32;
                        double w1 = 0.0, w2 = 0.0, ew;
                        if (k < A)
                            split_w_f16(s1 * std::ldexp((double)W1[(int64_t)(32 * mb + l % 32) * nin + L + perm[k]],
                                                        -ex[perm[k]]),
                                        &w1, &w2, &ew);
                        w1p[(mb * 64 + l) * 2 * ns + j] = f16_bits(w1);
                        w1p[(mb * 64 + l) * 2 * ns + ns + j] = f16_bits(w2);
                    }
            for (int h = 0; h < H; h++) img[ly.off_b2 + i * H + h] = (float)(S * b2[h]);
            uint16_t *w2p = reinterpret_cast<uint16_t *>(img + ly.off_w2 + i * H * H);
            for (int mb2 = 0; mb2 < ly.MB; mb2++)
                for (int mb1 = 0; mb1 < ly.MB; mb1++)
                    for (int kh = 0; kh < 2; kh++)
                        for (int l = 0; l < 64; l++)
                            for (int j = 0; j < 8; j++) {
                                const double w = s2 * W2[(int64_t)(32 * mb2 + l % 32) * H + 32 * mb1 + 16 * kh +
                                                         8 * (j / 4) + 4 * (l / 32) + j % 4];
                                double w1, w2, ew;
                                split_w_f16(w, &w1, &w2, &ew);
                                const int64_t at = ((((int64_t)(mb2 * ly.MB + mb1) * 2 + kh) * 2) * 64 + l) * 8 + j;
                                w2p[at] = f16_bits(w1);
                                w2p[at + 64 * 8] = f16_bits(w2);
                            }
            for (int o2 = 0; o2 < 2; o2++)
                for (int mb = 0; mb < ly.MB; mb++)
                    for (int q = 0; q < 4; q++)
                        for (int hf = 0; hf < 2; hf++)
                            for (int j = 0; j < 4; j++)
                                img[ly.off_w3 + i * 2 * H + (((o2 * ly.MB + mb) * 4 + q) * 2 + hf) * 4 + j] =
                                    (float)(W3[o2 * H + 32 * mb + 8 * q + 4 * hf + j] / S);
            img[ly.off_b3 + 4 * i + 0] = b3[0];
            img[ly.off_b3 + 4 * i + 1] = b3[1];
        }
        // aggregate rows as [half][s]: internal slot 2s + half
        for (int r = 0; r < sumK; r++)
            for (int hf = 0; hf < 2; hf++)
                for (int st = 0; st < 4; st++) {
                    const int k = 2 * st + hf;
                    img[ly.off_g + r * ly.AP + hf * 4 + st] = k < A ? F[(int64_t)r * L + p->agg_cols[perm[k]]] : 0.f;
                }
        for (int hf = 0; hf < 2; hf++)
            for (int st = 0; st < 4; st++) {
                const int k = 2 * st + hf;
                img[ly.off_c + hf * 4 + st] = k < A ? p->centre[perm[k]] : 0.f;
                p->fc.agg_scale[hf][st] = k < A ? (float)std::ldexp(1.0, ex[perm[k]]) : 1.f;
            }
        if (ly.off_feat >= 0) std::memcpy(img + ly.off_feat, F.data(), F.size() * 4);
        if (p->act == MF_ACT_SIGMOID)
            for (int i = 0; i < N; i++) {
                // the sigmoid is 1/4-Lipschitz, and its fp32 evaluation is within
                // 2^-20; the latency bound stays on the pre-activation scale (its
                // decision compares the pre-activation with logit thresholds)
                p->fc.bound_thr[i] = p->fc.bound_thr[i] * 0.25 + 0x1p-20;
                p->fc.mag_thr[i] = 1.0;
            }
    }
    {
        FastConst &fc = p->fc;
        fc.n_models = N;
        fc.act = p->act;
        for (int i = 0; i < N; i++) {
            fc.K[i] = p->K[i];
            fc.opt_off[i] = p->opt_off[i];
            fc.magic[i] = magic_for(p->K[i]);
        }
        fc.vram_cap = p->vram_cap;
    }

    // ---- bf16 fast path (H1 == H2 in {64, 128, 256}, A in {2,4,6,8})
    p->bf_ok = tl.bf_ok;
    p->blay = tl.blay;
    const Bf16Layout &bl = p->blay;
    if (p->bf_ok) {
        float *bimg = at_f(tl.o_bm);
        for (int i = 0; i < N; i++) {
            const float *w = W.data() + (int64_t)i * p->wstride;
            const float *W1 = w, *b1 = W1 + (int64_t)H * nin, *W2 = b1 + H, *b2 = W2 + (int64_t)H * H,
                        *W3 = b2 + H, *b3 = W3 + 2 * H;
            float *blk = bimg + (size_t)i * bl.model_floats;
            uint16_t *w2a = reinterpret_cast<uint16_t *>(blk + bl.off_w2a);
            for (int mb2 = 0; mb2 < bl.MB; mb2++)
                for (int ks = 0; ks < bl.KS; ks++)
                    for (int l = 0; l < 64; l++)
                        for (int j = 0; j < 8; j++) {
                            const int v = 32 * mb2 + l % 32;
                            const int u = 32 * (ks / 2) + 16 * (ks % 2) + 8 * (j / 4) + 4 * (l / 32) + j % 4;
                            uint32_t bits;
                            std::memcpy(&bits, &W2[(int64_t)v * H + u], 4);
                            w2a[(((size_t)mb2 * bl.KS + ks) * 64 + l) * 8 + j] = (uint16_t)(bits >> 16);
                        }
            for (int mb = 0; mb < bl.MB; mb++)
                for (int st = 0; st < bl.S1; st++)
                    for (int l = 0; l < 64; l++)
                        blk[bl.off_w1a + (mb * bl.S1 + st) * 64 + l] =
                            W1[(int64_t)(32 * mb + l % 32) * nin + L + 2 * st + l / 32];
            for (int h = 0; h < H; h++) blk[bl.off_b2 + h] = b2[h];
            for (int o2 = 0; o2 < 2; o2++)
                for (int mb = 0; mb < bl.MB; mb++)
                    for (int q = 0; q < 4; q++)
                        for (int hf = 0; hf < 2; hf++)
                            for (int j = 0; j < 4; j++)
                                blk[bl.off_w3 + (((o2 * bl.MB + mb) * 4 + q) * 2 + hf) * 4 + j] =
                                    W3[o2 * H + 32 * mb + 8 * q + 4 * hf + j];
            float cst[12] = {};
            bf16_bounds(*p, F, W, i, cst, &p->bcst.mag_thr[i]);
            if (p->act == MF_ACT_SIGMOID) p->bcst.mag_thr[i] = 1.0f;
            cst[0] = b3[0];
            cst[1] = b3[1];
            for (int t = 0; t < 12; t++) blk[bl.off_cst + t] = cst[t];
        }
        float *bg = at_f(tl.o_bg);
        for (int r = 0; r < sumK; r++) {
            for (int hf = 0; hf < 2; hf++)
                for (int st = 0; st < 4; st++) {
                    const int k = 2 * st + hf;
                    bg[(size_t)r * 8 + hf * 4 + st] = k < A ? F[(int64_t)r * L + p->agg_cols[k]] : 0.f;
                }
            bg[(size_t)sumK * 8 + r] = F[(int64_t)r * L + p->agg_cols[p->vram_slot]];
        }
        p->bcst.g2 = f32_up_host(gam(2.0 * bl.KS, kU32));
        p->bcst.g3 = f32_up_host(gam(H / 8 + 4, kU32));
        p->bcst.gN = f32_up_host(gam(N, kU32));
        p->bcst.act = p->act;
    }

    // ---- canonical image: per model W1T[nin][H1] b1 W2T[H1][H2] b2 W3[2][H2] b3
    float *canon = at_f(tl.o_can);
    for (int i = 0; i < N; i++) {
        const float *w = W.data() + (int64_t)i * p->wstride;
        float *c = canon + (int64_t)i * p->wstride;
        const float *W1 = w, *b1 = W1 + (int64_t)H1 * nin, *W2 = b1 + H1, *rest = W2 + (int64_t)H2 * H1;
        float *cW1T = c, *cb1 = c + (int64_t)nin * H1, *cW2T = cb1 + H1, *crest = cW2T + (int64_t)H1 * H2;
        for (int h = 0; h < H1; h++)
            for (int k = 0; k < nin; k++) cW1T[(int64_t)k * H1 + h] = W1[(int64_t)h * nin + k];
        std::memcpy(cb1, b1, (size_t)H1 * 4);
        for (int v = 0; v < H2; v++)
            for (int h = 0; h < H1; h++) cW2T[(int64_t)h * H2 + v] = W2[(int64_t)v * H1 + h];
        std::memcpy(crest, rest, (size_t)(H2 + 2 * H2 + 2) * 4);
    }
    // the fast image's copy of each model's canonical block (small-range
    // certification reads it from LDS)
    if (p->fast_ok && ly.off_c1 >= 0)
        for (int i = 0; i < N; i++)
            std::memcpy(at_f(tl.o_img) + ly.off_c1 + i * ly.c1_stride, canon + (int64_t)i * p->wstride,
                        (size_t)p->wstride * 4);
    std::memcpy(himg.data() + tl.o_fea, F.data(), F.size() * 4);
    std::memcpy(himg.data() + tl.o_agg, p->agg_cols.data(), (size_t)A * 4);
    int32_t *row_model = reinterpret_cast<int32_t *>(himg.data() + tl.o_rm);
    for (int i = 0; i < N; i++)
        for (int o = 0; o < p->K[i]; o++) row_model[p->opt_off[i] + o] = i;
    std::memcpy(himg.data() + tl.o_c, p->centre.data(), (size_t)A * 4);
    double *w64 = reinterpret_cast<double *>(himg.data() + tl.o_w64);
    for (size_t t = 0; t < W.size(); t++) w64[t] = (double)W[t];
    // the first L steps of each hidden unit's canonical layer-1 chain (Eq. 6:
    // the option's local features come first in the input), per option row:
    // fp64 fused multiply-adds, or fp32 ones for bf16 weights; both are
    // correctly rounded here as on the device, so the GA fitness continues
    // these values with the aggregate inputs bit for bit
    {
        double *pre = reinterpret_cast<double *>(himg.data() + tl.o_pre);
        const int nin = L + A;
        for (int i = 0; i < N; i++) {
            const float *W1 = W.data() + (int64_t)i * p->wstride, *b1 = W1 + (int64_t)p->H1 * nin;
            for (int o = 0; o < p->K[i]; o++) {
                const int row = p->opt_off[i] + o;
                const float *x = F.data() + (int64_t)row * L;
                for (int u = 0; u < p->H1; u++) {
                    double a;
                    if (p->bf16) {
                        float af = b1[u];
                        for (int k = 0; k < L; k++) af = std::fmaf(W1[(int64_t)u * nin + k], x[k], af);
                        a = (double)af;
                    } else {
                        a = (double)b1[u];
                        for (int k = 0; k < L; k++) a = std::fma((double)W1[(int64_t)u * nin + k], (double)x[k], a);
                    }
                    pre[(int64_t)row * p->H1 + u] = a;
                }
            }
        }
    }
    // ---- the caller's buffer
    char *base = (char *)d_tables;
    p->d_tables = d_tables;
    p->d_image = reinterpret_cast<float4 *>(base + tl.o_img);
    p->d_canon = reinterpret_cast<float *>(base + tl.o_can);
    p->d_features = reinterpret_cast<float *>(base + tl.o_fea);
    p->d_agg_cols = reinterpret_cast<int32_t *>(base + tl.o_agg);
    p->d_row_model = reinterpret_cast<int32_t *>(base + tl.o_rm);
    p->d_zeros = reinterpret_cast<float *>(base + tl.o_z);
    p->d_centre = reinterpret_cast<float *>(base + tl.o_c);
    p->d_w64 = reinterpret_cast<double *>(base + tl.o_w64);
    p->d_pre = reinterpret_cast<double *>(base + tl.o_pre);
    p->d_bmodels = reinterpret_cast<float4 *>(base + tl.o_bm);
    p->d_bg = reinterpret_cast<float4 *>(base + tl.o_bg);
    p->d_phat = reinterpret_cast<float *>(base + tl.o_ph);
    p->d_vrow = reinterpret_cast<float4 *>(base + tl.o_vr);
    bool ok = hipMemcpyAsync(d_tables, himg.data(), tl.total, hipMemcpyHostToDevice, s) == hipSuccess;
    if (ok && p->bf_ok)
        ok = launch_precompute_phat(p->d_features, p->d_canon, sumK, L, A, H, p->wstride, p->d_row_model, p->d_phat,
                                    bl.PST, s) == hipSuccess;
    if (ok && p->fast_ok)
    {
        Pow2Scales sc{};
        for (int i = 0; i < N; i++) sc.e[i] = p->fast_e1[i];
        ok = launch_precompute_p(p->d_features, p->d_canon, p->d_centre, sumK, L, A, H, p->wstride, p->d_row_model,
                                 reinterpret_cast<float *>(p->d_image) + ly.off_p, ly.PST, sc, s) == hipSuccess;
    }
    ok = ok && hipStreamSynchronize(s) == hipSuccess;
    // one pair of timing events up front (searches on several streams at
    // once take more from the pool)
    EventPair ev{};
    ok = ok && create_event_pair(ev);
    if (!ok) {
        delete p;
        return MF_EDEVICE;
    }
    p->ev_free.push_back(ev);
    p->ev_all.push_back(ev);
    *out = p;
    return MF_OK;
}

void mf_problem_destroy(mf_problem *p)
{
    if (!p) return;
    for (const EventPair &e : p->ev_all) {
        (void)hipEventDestroy(e.a);
        (void)hipEventDestroy(e.b);
        if (e.h_res) (void)hipHostFree(e.h_res);
    }
    delete p;
}

mf_status mf_space_size(const mf_problem *p, uint64_t *out)
{
    if (!p || !out) return MF_EINVAL;
    *out = p->space;
    return MF_OK;
}

mf_status mf_decode(const mf_problem *p, uint64_t idx, int32_t *h_digits)
{
    if (!p || !h_digits || idx >= p->space) return MF_EINVAL;
    for (int i = p->N - 1; i >= 0; i--) {
        h_digits[i] = (int32_t)(idx % (uint64_t)p->K[i]);
        idx /= (uint64_t)p->K[i];
    }
    return MF_OK;
}

static mf_status check_search_args(const mf_problem *p, const mf_search_args *a)
{
    if (!p || !a) return MF_EINVAL;
    if (a->lo > a->hi) return MF_EINVAL;
    if (a->hi > p->space) return MF_EOVERFLOW;
    if (a->top_k < 1 || a->top_k > MF_MAX_TOPK) return MF_EINVAL;
    if (!a->d_sla || !a->d_omega) return MF_EINVAL;
    if (a->flags & ~(MF_DUMP | MF_FIXED_STATE)) return MF_EINVAL;
    if ((a->flags & MF_DUMP) && (!a->d_mask || !a->d_pred || a->hi - a->lo > (1ull << 31))) return MF_EINVAL;
    if (a->flags & MF_FIXED_STATE) {
        for (int k = 0; k < p->A; k++)
            if (!std::isfinite(a->state[k])) return MF_EINVAL;
    } else if (!p->fast_ok && !p->bf_ok) {
        return MF_EUNSUPPORTED;
    }
    return check_objective(p, a->objective);
}

// Bytes of workspace a validated search needs.
static size_t search_ws_bytes(const mf_problem *p, const mf_search_args *args)
{
    if (args->flags & MF_FIXED_STATE) return fixed_ws_bytes(*p, args->top_k);
    const uint64_t n = std::min<uint64_t>(args->hi - args->lo, kMaxLaunch);
    return ws_layout(*p, n, args->top_k, args->worklist_cap).total;
}

// A validated search on a workspace of at least search_ws_bytes.
static mf_status search_impl(mf_problem *p, const mf_search_args *args, char *ws, hipStream_t s,
                             bool may_create_events, mf_result *h_out)
{
    const EventLease ev(p, may_create_events);
    mf_result acc;
    empty_result(acc);
    const mf_status st = (args->flags & MF_FIXED_STATE)
                             ? search_fixed(p, args, ws, s, ev, acc)
                             : search_range(p, args, args->lo, args->hi - args->lo, ws, s, ev, acc, 0);
    if (st != MF_OK) return st;
    *h_out = acc;
    return MF_OK;
}

mf_status mf_workspace_size(const mf_problem *p, const mf_search_args *args, size_t *bytes)
{
    if (!bytes) return MF_EINVAL;
    mf_status st = check_search_args(p, args);
    if (st != MF_OK) return st;
    *bytes = search_ws_bytes(p, args);
    return MF_OK;
}

mf_status mf_search(mf_problem *p, const mf_search_args *args, void *d_ws, size_t ws_bytes, void *stream,
                    mf_result *h_out)
{
    if (!h_out || !d_ws) return MF_EINVAL;
    mf_status st = check_search_args(p, args);
    if (st != MF_OK) return st;
    if (ws_bytes < search_ws_bytes(p, args)) return MF_ENOMEM;
    if (((uintptr_t)d_ws & 255u) != 0) return MF_EINVAL;
    return search_impl(p, args, (char *)d_ws, (hipStream_t)stream, true, h_out);
}

mf_status mf_search_noalloc(mf_problem *p, const mf_search_args *args, void *stream, mf_result *h_out)
{
    if (!h_out) return MF_EINVAL;
    mf_status st = check_search_args(p, args);
    if (st != MF_OK) return st;
    if (search_ws_bytes(p, args) > (size_t)MF_NOALLOC_SCRATCH_BYTES) return MF_ESCRATCH;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return MF_EDEVICE;
    if (dev != p->device) return MF_EINVAL;
    // the problem's pre-created timing events only (none free: untimed)
    return search_impl(p, args, (char *)p->d_scratch, (hipStream_t)stream, false, h_out);
}

mf_status mf_static_workspace_size(const mf_problem *p, const mf_static_args *args, size_t *bytes)
{
    if (!bytes) return MF_EINVAL;
    mf_status st = check_static_args(p, args, false);
    if (st != MF_OK) return st;
    *bytes = static_ws_layout(*p, args->n_steps, MF_MAX_TOPK).total;
    return MF_OK;
}

mf_status mf_search_static(mf_problem *p, const mf_static_args *args, void *d_ws, size_t ws_bytes, void *stream,
                           mf_result *h_out)
{
    if (!h_out || !d_ws) return MF_EINVAL;
    mf_status st = check_static_args(p, args, true);
    if (st != MF_OK) return st;
    if (ws_bytes < static_ws_layout(*p, args->n_steps, MF_MAX_TOPK).total) return MF_ENOMEM;
    if (((uintptr_t)d_ws & 255u) != 0) return MF_EINVAL;
    mf_result acc;
    empty_result(acc);
    st = search_static(p, args, (char *)d_ws, (hipStream_t)stream, acc);
    if (st != MF_OK) return st;
    *h_out = acc;
    return MF_OK;
}

mf_status mf_eval_static(mf_problem *p, const mf_static_args *args, const uint64_t *d_idx, int64_t n, double *d_J,
                         double *d_S, uint32_t *d_flags, void *d_ws, size_t ws_bytes, void *stream)
{
    if (!d_ws || n < 0 || (n > 0 && !d_idx)) return MF_EINVAL;
    mf_status st = check_static_args(p, args, false);
    if (st != MF_OK) return st;
    if (ws_bytes < static_ws_layout(*p, args->n_steps, MF_MAX_TOPK).total) return MF_ENOMEM;
    if (((uintptr_t)d_ws & 255u) != 0) return MF_EINVAL;
    if (n == 0) return MF_OK;
    hipStream_t s = (hipStream_t)stream;
    StaticArgs sa;
    st = static_setup(p, args, (char *)d_ws, 1, s, sa);
    if (st != MF_OK) return st;
    sa.idx = d_idx;
    sa.n_list = n;
    sa.out_J = d_J;
    sa.out_S = d_S;
    sa.out_flags = d_flags;
    if (launch_static_eval(sa, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return MF_EDEVICE;
    return MF_OK;
}

mf_status mf_eval_fast(mf_problem *p, const uint64_t *d_idx, int64_t n, float *d_pred, void *stream)
{
    if (!p || n < 0 || (n > 0 && (!d_idx || !d_pred))) return MF_EINVAL;
    if (!p->fast_ok && !p->bf_ok) return MF_EUNSUPPORTED;
    if (n == 0) return MF_OK;
    if (p->bf_ok) {
        FastArgs fa{};
        fa.lo = 0;
        fa.n = (uint64_t)n;
        fa.idx_list = d_idx;
        fa.sla = p->d_zeros;
        fa.omega = p->d_zeros;
        fa.pred = d_pred;
        const uint64_t per_wg = (uint64_t)kBf16Waves * kBf16Tiles * 32;
        const int grid = (int)std::max<uint64_t>(1, std::min<uint64_t>(((uint64_t)n + per_wg - 1) / per_wg,
                                                                        (uint64_t)p->num_cus));
        return hip_status(launch_fast_path(p, fa, grid, 16, kModeList, (hipStream_t)stream));
    }
    FastArgs fa{};
    fa.image = p->d_image;
    fa.image_f4 = p->lay.total_floats / 4;
    fa.lay = p->lay;
    fa.lo = 0;
    fa.n = (uint64_t)n;
    fa.idx_list = d_idx;
    const uint64_t tiles = ((uint64_t)n + 31) / 32;
    fa.waves = fast_waves_for(p->N, p->lay, 16, p->act);
    const int grid = (int)std::max<uint64_t>(1, std::min<uint64_t>((tiles + fa.waves - 1) / fa.waves,
                                                                    (uint64_t)p->num_cus));
    fa.total_waves = grid * fa.waves;
    fa.sla = p->d_zeros;
    fa.omega = p->d_zeros;
    fa.pred = d_pred;
    return hip_status(launch_fast_impl(fa, p->fc, grid, 16, kModeList, (hipStream_t)stream));
}

mf_status mf_eval_canonical(mf_problem *p, const uint64_t *d_idx, int64_t n, const float *d_sla,
                            const float *d_omega, double *d_pred, double *d_J, uint32_t *d_flags, void *stream)
{
    if (!p || n < 0 || (n > 0 && (!d_idx || !d_sla || !d_omega))) return MF_EINVAL;
    if (n == 0) return MF_OK;
    CanonArgs ca{};
    ca.n_models = p->N; ca.L = p->L; ca.A = p->A; ca.H1 = p->H1; ca.H2 = p->H2; ca.bf16 = p->bf16; ca.act = p->act;
    for (int i = 0; i < p->N; i++) { ca.K[i] = p->K[i]; ca.opt_off[i] = p->opt_off[i]; }
    ca.agg_cols = p->d_agg_cols; ca.vram_slot = p->vram_slot; ca.vram_cap = p->vram_cap;
    ca.features = p->d_features; ca.weights = p->d_canon; ca.wstride = p->wstride;
    ca.sla = d_sla; ca.omega = d_omega;
    ca.idx64 = d_idx;
    ca.n_list = n;
    ca.ent_J = d_J;
    ca.ent_flags = d_flags;
    ca.pred = d_pred;
    return hip_status(launch_canonical(ca, (int)std::min<int64_t>(n, 1 << 20), false, (hipStream_t)stream));
}

static mf_status check_ga_args(const mf_problem *p, const mf_ga_args *a)
{
    if (!p || !a) return MF_EINVAL;
    if (a->n_scen < 1 || a->pop < 4 || a->pop > 4096 || (a->pop & 1) || a->gens < 0 || a->tourn_k < 1 ||
        a->tourn_k > 8 || !a->d_sla || !a->d_omega)
        return MF_EINVAL;
    for (float q : {a->p_cx, a->p_swap, a->p_mut})
        if (!std::isfinite(q)) return MF_EINVAL;
    if (a->flags & ~MF_FIXED_STATE) return MF_EINVAL;
    if (a->flags & MF_FIXED_STATE)
        for (int k = 0; k < p->A; k++)
            if (!std::isfinite(a->state[k])) return MF_EINVAL;
    mf_status st = check_objective(p, a->objective);
    if (st != MF_OK) return st;
    if (p->space > (1ull << 32)) return MF_EUNSUPPORTED;
    return MF_OK;
}

struct GaWs {
    size_t cnt, off, nfl, fl, popA, popB, fit, bJ, bI, memo, tag, nfwd, total;
    bool use_memo;
};

// The GAConst of a run without its device pointers' workspace parts (the
// shape fields the kernels' choices depend on).
static GAConst ga_shape(const mf_problem *p)
{
    GAConst c{};
    c.N = p->N; c.L = p->L; c.A = p->A; c.H1 = p->H1; c.H2 = p->H2; c.bf16 = p->bf16; c.act = p->act;
    c.pre = p->d_pre;
    c.sumK = p->sumK;
    return c;
}

static GaWs ga_ws(const mf_problem *p, const mf_ga_args *a)
{
    GaWs w{};
    const uint64_t n_blk = (p->space + 255) / 256;
    const size_t sp = (size_t)a->n_scen * a->pop;
    size_t o = 0;
    w.cnt = o; o = align256(o + n_blk * 4);
    w.off = o; o = align256(o + n_blk * 8);
    w.nfl = o; o = align256(o + 8);
    w.fl = o; o = align256(o + p->space * 4);
    w.popA = o; o = align256(o + sp * 8);
    w.popB = o; o = align256(o + sp * 8);
    w.fit = o; o = align256(o + sp * 8);
    w.bJ = o; o = align256(o + (size_t)a->n_scen * 8);
    w.bI = o; o = align256(o + (size_t)a->n_scen * 8);
    // the run's memo of canonical predictions per joint index (large
    // populations over spaces small enough to tabulate)
    const uint64_t memo_bytes = p->space * (uint64_t)p->N * 16u + p->space * 4u;
    w.use_memo = ga_memo_supported(ga_shape(p), a->n_scen, a->pop) && memo_bytes <= kGaMemoMaxBytes;
    w.memo = o; o = align256(o + (w.use_memo ? p->space * (size_t)p->N * 16 : 0));
    w.tag = o; o = align256(o + (w.use_memo ? p->space * 4 : 0));
    w.nfwd = o; o = align256(o + 8);
    w.total = o;
    return w;
}

mf_status mf_ga_workspace_size(const mf_problem *p, const mf_ga_args *args, size_t *bytes)
{
    if (!bytes) return MF_EINVAL;
    mf_status st = check_ga_args(p, args);
    if (st != MF_OK) return st;
    *bytes = ga_ws(p, args).total;
    return MF_OK;
}

mf_status mf_ga_run(mf_problem *p, const mf_ga_args *args, void *d_ws, size_t ws_bytes, void *stream,
                    uint64_t *h_best_idx, double *h_best_J, uint64_t *d_final_pop)
{
    if (!h_best_idx || !h_best_J || !d_ws) return MF_EINVAL;
    mf_status st = check_ga_args(p, args);
    if (st != MF_OK) return st;
    const GaWs w = ga_ws(p, args);
    if (ws_bytes < w.total) return MF_ENOMEM;
    if (((uintptr_t)d_ws & 255u) != 0) return MF_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)d_ws;
    uint32_t *cnt = reinterpret_cast<uint32_t *>(ws + w.cnt);
    uint64_t *blk_off = reinterpret_cast<uint64_t *>(ws + w.off);
    unsigned long long *n_fl = reinterpret_cast<unsigned long long *>(ws + w.nfl);
    uint32_t *fl = reinterpret_cast<uint32_t *>(ws + w.fl);
    uint64_t *pa = reinterpret_cast<uint64_t *>(ws + w.popA), *pb = reinterpret_cast<uint64_t *>(ws + w.popB);
    double *fit = reinterpret_cast<double *>(ws + w.fit);
    double *bJ = reinterpret_cast<double *>(ws + w.bJ);
    uint64_t *bI = reinterpret_cast<uint64_t *>(ws + w.bI);

    GAConst c{};
    c.N = p->N; c.L = p->L; c.A = p->A; c.H1 = p->H1; c.H2 = p->H2; c.bf16 = p->bf16; c.act = p->act;
    for (int i = 0; i < p->N; i++) { c.K[i] = p->K[i]; c.opt_off[i] = p->opt_off[i]; }
    c.vram_col = p->agg_cols[p->vram_slot];
    c.vram_slot = p->vram_slot;
    c.vram_cap = p->vram_cap;
    c.space = p->space;
    c.features = p->d_features;
    c.agg_cols = p->d_agg_cols;
    c.w64 = p->d_w64;
    c.pre = p->d_pre;
    c.sumK = p->sumK;
    c.canon = p->d_canon;
    c.wstride = p->wstride;
    c.fixed = (args->flags & MF_FIXED_STATE) ? 1 : 0;
    for (int k = 0; k < p->A; k++) c.state[k] = c.fixed ? args->state[k] : 0.f;
    c.obj = obj_args(p, args->objective);
    c.memo = w.use_memo ? reinterpret_cast<double *>(ws + w.memo) : nullptr;
    c.memo_tag = w.use_memo ? reinterpret_cast<uint32_t *>(ws + w.tag) : nullptr;
    c.n_forwards = reinterpret_cast<unsigned long long *>(ws + w.nfwd);

    const int S = args->n_scen, P = args->pop;
    // an empty feasible list is handled on the device (the best stays unset,
    // the final population reads all ones): no synchronisation mid-run
    MF_HIP(launch_ga_feasible(c, cnt, blk_off, n_fl, fl, s));
    MF_HIP(launch_ga_init(args->seed, S, P, fl, n_fl, pa, bJ, bI, s));
    // generation 0 always runs the surrogates (and fills the memo); without
    // the memo every generation does
    const unsigned long long sp = (unsigned long long)S * (unsigned long long)P;
    MF_HIP(launch_ga_memo_clear(c.memo_tag, c.memo ? p->space : 0, c.n_forwards,
                                c.memo ? sp : sp * (unsigned long long)(args->gens + 1), s));
    for (int g = 0; g <= args->gens; g++) {
        // generation g's entries carry tag g + 1
        MF_HIP(launch_ga_fitness(c, S, P, pa, args->d_sla, args->d_omega, fit, s, (uint32_t)g + 1u));
        MF_HIP(launch_ga_ops(c, args->seed, S, P, g, args->gens, args->tourn_k, args->p_cx, args->p_swap,
                             args->p_mut, fl, n_fl, pa, fit, pb, bJ, bI, d_final_pop, s));
        std::swap(pa, pb);
    }
    MF_HIP(hipMemcpyAsync(h_best_J, bJ, (size_t)S * 8, hipMemcpyDeviceToHost, s));
    MF_HIP(hipMemcpyAsync(h_best_idx, bI, (size_t)S * 8, hipMemcpyDeviceToHost, s));
    if (args->h_forwards)
        MF_HIP(hipMemcpyAsync(args->h_forwards, c.n_forwards, 8, hipMemcpyDeviceToHost, s));
    MF_HIP(hipStreamSynchronize(s));
    return MF_OK;
}

}  // extern "C"
