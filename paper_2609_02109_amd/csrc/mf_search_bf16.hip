// bf16 fast path, host side: the per-option layer-1 seed, the LDS budget and
// the dispatch to the kernel instantiations (mf_bf16_kernel.h).
#include "mf_device.h"

namespace mfi {

// Per-option layer-1 seed of the bf16 path: the fp32 fma chain over the L
// local columns from the bias (the first L steps of the canonical chain).
// canon_w holds, per model, W1 transposed ([L + A][H]) followed by b1.
__global__ void precompute_phat_kernel(const float *features, const float *canon_w, int n_rows, int L, int A, int H,
                                       int64_t wstride, const int32_t *row_model, float *phat, int pst)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_rows * H) return;
    const int row = (int)(t / H), h = (int)(t % H);
    const float *W1T = canon_w + (int64_t)row_model[row] * wstride;
    const float *b1 = W1T + (int64_t)(L + A) * H;
    float c = b1[h];
    for (int k = 0; k < L; k++) c = fmaf(W1T[(int64_t)k * H + h], features[(int64_t)row * L + k], c);
    phat[(int64_t)row * pst + h] = c;
}

hipError_t launch_precompute_phat(const float *features, const float *canon_w, int n_rows, int L, int A, int H,
                                  int64_t wstride, const int32_t *row_model, float *phat, int pst, hipStream_t s)
{
    const int64_t total = (int64_t)n_rows * H;
    hipLaunchKernelGGL(precompute_phat_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, features,
                       canon_w, n_rows, L, A, H, wstride, row_model, phat, pst);
    return hipGetLastError();
}

size_t bf16_lds_bytes(const Bf16Layout &lay, int kp)
{
    return (size_t)(lay.model_floats + lay.sumK * 8 + lay.gv_floats + kBf16Par) * 4 + (size_t)kBf16Waves * kp * 8;
}

int bf16_kernel_supported(int n_models, int A, int H)
{
    return n_models >= 1 && n_models <= kMaxN && (A == 2 || A == 4 || A == 6 || A == 8) &&
           (H == 64 || H == 128 || H == 256);
}

hipError_t launch_bf16_impl(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                            hipStream_t s)
{
    if (kp < 1 || kp > 128 || fc.n_models < 1 || fc.n_models > kMaxN) return hipErrorInvalidValue;
    switch (a.lay.H) {
        case 64: return launch_bf16_h64(a, fc, bc, grid, kp, mode, s);
        case 128: return launch_bf16_h128(a, fc, bc, grid, kp, mode, s);
        case 256: return launch_bf16_h256(a, fc, bc, grid, kp, mode, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace mfi
