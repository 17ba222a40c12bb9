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
