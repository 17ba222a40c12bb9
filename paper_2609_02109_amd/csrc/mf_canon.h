// Canonical fp64 evaluation shared by the certification kernel and the
// fixed-state search (HIP translation units only).  Results of every search
// are defined by these semantics: each dot product is one fused multiply-add
// chain in ascending input order from the bias; relu(x) = x > 0 ? x : +0; in
// bf16 mode the first hidden layer accumulates in fp32 (one fmaf chain in
// input order from the bias) and is rounded to bfloat16 after the relu.
#pragma once

#include "mf_device.h"

namespace mfi {

constexpr int kCanonMaxH = 256;
constexpr int kCanonMaxIn = 64;

__device__ __forceinline__ double bf16_round_d(double x)
{
    // nearest bfloat16 value (8 significant bits), ties to even; x finite
    if (x == 0.0) return x;
    int e = ilogb(x);
    if (e < -126) e = -126;                 // bf16 subnormal spacing 2^-133
    const double scale = ldexp(1.0, 7 - e); // |x| * scale in [128, 256)
    return rint(x * scale) / scale;
}

// e^x for |x| <= 700, defined by its algorithm so that it is the same
// function wherever it runs: x = k ln 2 + r with k = rint(x / ln 2) and r
// from two fmas (ln 2 split into a 24-bit head and a tail: k ln2_hi is
// exact), e^r by its Taylor series to degree 13 (Horner with fma, |r| <=
// ln 2 / 2: truncation below 4e-18), then times 2^k (exact in this range).
__device__ __forceinline__ double canon_exp(double x)
{
    constexpr double kInvLn2 = 1.4426950408889634;        // 1 / ln 2
    constexpr double kLn2Hi = 0.693147182464599609375;    // ln 2 rounded to 24 significant bits
    constexpr double kLn2Lo = -1.904654299957768e-09;     // ln 2 - kLn2Hi
    const double k = rint(x * kInvLn2);
    double r = fma(-k, kLn2Hi, x);
    r = fma(-k, kLn2Lo, r);
    double inv_fact[14];
    double fact = 1.0;
#pragma unroll
    for (int n = 0; n < 14; n++) {
        if (n > 0) fact *= (double)n;
        inv_fact[n] = 1.0 / fact;
    }
    double p = inv_fact[13];
#pragma unroll
    for (int n = 12; n >= 0; n--) p = fma(p, r, inv_fact[n]);
    return ldexp(p, (int)k);
}

// The surrogate's sigmoid output: 1 / (1 + e^-y), y clamped to [-700, 700].
__device__ __forceinline__ double canon_sigmoid(double y)
{
    const double c = y < -700.0 ? -700.0 : (y > 700.0 ? 700.0 : y);
    return 1.0 / (1.0 + canon_exp(-c));
}

// One model's surrogate (Eq. 6) on the inputs zs [nin] (shared memory), by one
// 64-thread workgroup: lanes take hidden units; h1s, h2s are shared scratch.
// w: the model's canonical image W1^T[nin][H1], b1, W2^T[H1][H2], b2,
// W3[2][H2], b3; sigmoid: both outputs pass canon_sigmoid.  Every lane returns
// (lat, thr).  Contains barriers: call from all lanes.  WAVE: zs, h1s, h2s
// belong to the calling wave alone, whose LDS accesses complete in program
// order, so wave barriers (which only keep the compiler from moving the
// accesses across them) replace the workgroup barriers.
template <bool BF16, bool WAVE = false>
__device__ inline void canon_model(const float *w, int nin, int H1, int H2, const double *zs, double *h1s,
                                   double *h2s, int lane, double &lat, double &thr, int sigmoid)
{
    const float *W1T = w, *b1 = W1T + (int64_t)nin * H1, *W2T = b1 + H1, *b2 = W2T + (int64_t)H1 * H2,
                *W3 = b2 + H2, *b3 = W3 + 2 * H2;
    for (int u = lane; u < H1; u += 64) {
        if (BF16) {
            float c = b1[u];
            #pragma unroll 8
            for (int k = 0; k < nin; k++) c = fmaf(W1T[(int64_t)k * H1 + u], (float)zs[k], c);
            c = c > 0.f ? c : 0.f;
            h1s[u] = bf16_round_d((double)c);
        } else {
            double c = (double)b1[u];
            #pragma unroll 8
            for (int k = 0; k < nin; k++) c = fma((double)W1T[(int64_t)k * H1 + u], zs[k], c);
            h1s[u] = c > 0.0 ? c : 0.0;
        }
    }
    if (WAVE) __builtin_amdgcn_wave_barrier(); else __syncthreads();
    for (int v = lane; v < H2; v += 64) {
        double c = (double)b2[v];
        #pragma unroll 8
        for (int u = 0; u < H1; u++) c = fma((double)W2T[(int64_t)u * H2 + v], h1s[u], c);
        h2s[v] = c > 0.0 ? c : 0.0;
    }
    if (WAVE) __builtin_amdgcn_wave_barrier(); else __syncthreads();
    double y = 0.0;
    if (lane < 2) {
        double c = (double)b3[lane];
        #pragma unroll 8
        for (int v = 0; v < H2; v++) c = fma((double)W3[lane * H2 + v], h2s[v], c);
        y = sigmoid ? canon_sigmoid(c) : c;
    }
    lat = __shfl(y, 0);
    thr = __shfl(y, 1);
}

// The canonical term of model i under the full utility (Section II, Eq. 3)
// for option row `row` and throughput thr: q = Q f with f = (thr - fmin) /
// (fmax - fmin); reload (when the variant changed; *do_P) and soft-SLA
// penalty (when d = tau + delta - f > 0; *do_pen) to subtract after
// J = fma(omega, q, J).  Returns whether the floor f >= tau holds.
__device__ __forceinline__ bool canon_eq3_rows(const float4 r0, const float4 r1, const ObjArgs &o, double thr,
                                               float tau, int prev, double &q, double &P, bool &do_P, double &pen,
                                               bool &do_pen)
{
    const int var = __float_as_int(r1.x);
    const double fmin = (double)r0.x;
    const double rg = (double)r0.y - fmin;
    const double f = (thr - fmin) / rg;
    q = (double)r0.w * f;
    do_P = prev >= 0 && var != prev;
    P = do_P ? (double)o.alpha * (double)r1.y : 0.0;
    const double dd = ((double)tau + (double)o.delta) - f;
    do_pen = dd > 0.0;
    pen = do_pen ? (double)o.beta * (dd * dd) : 0.0;
    return f >= (double)tau;
}

__device__ __forceinline__ bool canon_eq3(const ObjArgs &o, int64_t row, double thr, float tau, int prev, double &q,
                                          double &P, bool &do_P, double &pen, bool &do_pen)
{
    return canon_eq3_rows(o.vrow[2 * row], o.vrow[2 * row + 1], o, thr, tau, prev, q, P, do_P, pen, do_pen);
}

}  // namespace mfi
