// The bf16 fast search kernel (template), included by one translation unit
// per hidden width so that its instantiations compile in parallel.
//
// Per model (Eq. 6), for tiles of 32 joint configurations per wave:
//   layer 1   the pre-activation accumulates in fp32 in input order: the
//             per-option part (local columns, an fp32 fma chain precomputed
//             once per option) seeds the accumulator, then
//             v_mfma_f32_32x32x2f32 adds the aggregate slots two at a time,
//             slot 2s before 2s+1 (each step a correctly rounded fused
//             multiply-add), so the result equals the canonical fp32 chain
//             bit for bit and so does its bfloat16 rounding.
//   layer 2   relu -> bf16, packed straight from the accumulator registers
//             into B operands of v_mfma_f32_32x32x16_bf16 (the accumulator
//             row order is absorbed into W2's A-operand layout); fp32
//             accumulation.  W2 (128 KB per model at H=256) is staged in LDS
//             one model at a time: a workgroup runs the model over all of its
//             tiles before staging the next.
//   layer 3   VALU fp32, four partial chains per output.  The only difference
//             from the canonical values is the fp32 accumulation of layers 2
//             and 3, bounded per configuration by
//               gamma_{2 KS} (|W3||b2| + max_u r_u sum_u h1[u]),  r = |W3||W2|
//             + gamma_{H/8+4} (|b3| + max_v |W3[o][v]| sum_v h2[v]).
// Within a tile, the MFMAs of each 32-row block overlap the VALU epilogue of
// the previous block (relu and bf16 packing after layer 1, relu and layer 3
// after layer 2).  Per-tile state (J, its bound, flags) rotates through
// registers so that the runtime tile loop never indexes a private array.
#pragma once

#include "mf_device.h"

namespace mfi {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr uint32_t kFlagFail = 0x80000000u;   // some model surely misses its bound
constexpr uint32_t kFlagVram = 0x40000000u;   // VRAM cap met


// 16 accumulator rows of one 32-row block: [q][j] = p[8 q + j], j < 4
__device__ __forceinline__ floatx16 load16(const float *p)
{
    floatx16 r;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const float4 v = *reinterpret_cast<const float4 *>(p + 8 * q);
        r[4 * q + 0] = v.x;
        r[4 * q + 1] = v.y;
        r[4 * q + 2] = v.z;
        r[4 * q + 3] = v.w;
    }
    return r;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short short2v __attribute__((ext_vector_type(2)));

// relu on two packed bfloat16 values: a packed 16-bit integer max with 0 (a
// set sign bit, -0 included, maps to +0)
__device__ __forceinline__ bf16x2 relu2(bf16x2 v)
{
    short2v t;
    __builtin_memcpy(&t, &v, 4);
    t = __builtin_elementwise_max(t, (short2v){0, 0});
    __builtin_memcpy(&v, &t, 4);
    return v;
}

// Layer-1 epilogue for 16 accumulator rows: round to bfloat16 (nearest even),
// relu on the packed values (rounding to nearest commutes with relu, so this
// is bf16(relu(x))), and the running sum of the activations by bf16 dot
// products with (1, 1); B operands for rows 0-7 and 8-15.
typedef float float2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void layer1_epilogue(const floatx16 &acc, bf16x8 &lo, bf16x8 &hi, float &sh)
{
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    bf16x2 w[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
        // one v_cvt_pk_bf16_f32 (nearest even), then relu on the pair
        w[j] = relu2(__builtin_convertvector((float2v){acc[2 * j], acc[2 * j + 1]}, bf16x2));
        sh = __builtin_amdgcn_fdot2_f32_bf16(w[j], one, sh, false);
    }
    __builtin_memcpy(&lo, w, 16);
    __builtin_memcpy(&hi, w + 4, 16);
}

// Layer-3 weights of one 32-row block for this lane's half: [q] = rows 8 q + j
__device__ __forceinline__ void load_w3(const float *wl, const float *wt, float4 *pwl, float4 *pwt)
{
#pragma unroll
    for (int q = 0; q < 4; q++) {
        pwl[q] = *reinterpret_cast<const float4 *>(wl + 8 * q);
        pwt[q] = *reinterpret_cast<const float4 *>(wt + 8 * q);
    }
}

__device__ __forceinline__ float f4get(const float4 &v, int j)
{
    return j == 0 ? v.x : (j == 1 ? v.y : (j == 2 ? v.z : v.w));
}

// relu of accumulator row r (= 4 q + j) of a layer-2 block and its layer-3
// contribution: partial chain q takes rows 8 q + j; s2 sums the activations
// (for the rounding bound).  r is a compile-time constant after unrolling.
__device__ __forceinline__ void layer3_row(const floatx16 &acc, int r, const float4 *pwl, const float4 *pwt,
                                           float *yl, float *yt, float &s2)
{
    const int q = r >> 2, j = r & 3;
    const float h = relu_f32(acc[r]);
    yl[q] = fmaf(f4get(pwl[q], j), h, yl[q]);
    yt[q] = fmaf(f4get(pwt[q], j), h, yt[q]);
    s2 += h;
}

// FULL: the problem has exactly MAXN models, each with more than one option
// (no per-model range checks, no special case in the decode).
// LIST: evaluate the configurations of args.idx_list (predictions only).
// OBJ: score with the full utility of Eq. 3 (otherwise the linear objective).
template <int MAXN, int A, int H, bool FULL, bool LIST, bool OBJ, bool SIG = false>
__global__ void __launch_bounds__(kBf16Waves * 64, 1)
fast_bf16_kernel(const Bf16Args args, const FastConst fc, const Bf16Const bc, const int mode, const int kp)
{
    constexpr int MB = H / 32, KS = H / 16, S1 = A / 2;
    constexpr Bf16Layout CL = bf16_layout(H, A, 0);
    constexpr int WAVES = kBf16Waves, TW = kBf16Tiles;
    constexpr uint64_t SUP = (uint64_t)WAVES * TW * 32;
    extern __shared__ float4 smem4[];
    float *smem = reinterpret_cast<float *>(smem4);
    const Bf16Layout &Ly = args.lay;
    const int N = FULL ? MAXN : fc.n_models;
    float *G = smem + CL.model_floats;            // [sumK][half][4]: slot 2s+half at [half][s]
    float *Gv = G + Ly.sumK * 8;                   // [sumK] VRAM column
    // [0,16) sla (sigmoid outputs: the pass threshold of the pre-activation) [16,32) |thr| bound
    // [32,48) omega [48,64) rows [64,80) floor tau [80,96) previous variant [96,112) miss threshold
    // of the pre-activation (sigmoid outputs)
    float *par = Gv + Ly.gv_floats;
    int *par_off = reinterpret_cast<int *>(par + 48);
    int *par_prev = reinterpret_cast<int *>(par + 80);
    unsigned long long *lst = reinterpret_cast<unsigned long long *>(par + kBf16Par);

    for (int t = threadIdx.x; t < (Ly.sumK * 8 + Ly.gv_floats) / 4; t += blockDim.x)
        reinterpret_cast<float4 *>(G)[t] = args.g_image[t];
#pragma unroll
    for (int i = 0; i < kMaxN; i++) {
        if (threadIdx.x == (unsigned)i && i < N) {
            par[i] = args.sla[i];
            if constexpr (SIG) {
                // sigmoid outputs: the latency decision compares the
                // pre-activation with logit thresholds (the canonical sigmoid
                // is within 2^-49 relative of the exact one; outputs lie in [0, 1])
                auto logit = [](double p) {
                    return p <= 0.0 ? -INFINITY : (p >= 1.0 ? INFINITY : log(p / (1.0 - p)));
                };
                const double sd = (double)args.sla[i];
                par[i] = (float)(sd >= 1.0 ? INFINITY : logit(sd * (1.0 - 0x1p-49)));
                par[96 + i] = (float)(sd >= 1.0 ? INFINITY : logit(sd * (1.0 + 0x1p-48)));
            }
            par[16 + i] = bc.mag_thr[i];
            par[32 + i] = args.omega[i];
            par_off[i] = fc.opt_off[i];
            if constexpr (OBJ) {
                par[64 + i] = args.obj.tau[i];
                par_prev[i] = args.obj.prev[i];
            }
        }
    }
    __syncthreads();
    constexpr bool eq3 = OBJ;

    const int lane = threadIdx.x & 63, half = lane >> 5, col = lane & 31;
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint64_t n = args.n;
    const uint64_t n_super = (n + SUP - 1) / SUP;
    // rounding of the canonical fp64 objective chain (N <= 16 terms)
    double eJ0 = 0.0;
    for (int i = 0; i < N; i++) eJ0 += fabs((double)par[32 + i]) * (double)par[16 + i];
    eJ0 = eJ0 * 0x1p-48 + 1e-30;

    WaveList<2> wl;
    wl_init(wl);
    uint32_t c_vram = 0, c_feas = 0;

    for (uint64_t st = blockIdx.x; st < n_super; st += gridDim.x) {
        const uint64_t wbase = st * SUP + (uint64_t)wv * (TW * 32);
        uint32_t bd[MAXN];
        {
            uint64_t x = args.lo + wbase;
#pragma unroll
            for (int j = MAXN - 1; j >= 0; j--) {
                if (j < N) {
                    const uint64_t k = (uint64_t)fc.K[j];
                    bd[j] = (uint32_t)(x % k);
                    x /= k;
                } else {
                    bd[j] = 0;
                }
            }
        }
        float Jt[TW], Et[TW];
        uint32_t Ft[TW];
#pragma unroll
        for (int t = 0; t < TW; t++) { Jt[t] = 0.f; Et[t] = 0.f; Ft[t] = 0u; }

        for (int i = 0; i < N; i++) {
            // ---- stage model i: W2 A operands, W1 aggregate columns, b2, W3, constants
            __syncthreads();
            {
                // direct global -> LDS copies, 1 KB per wave instruction (the
                // block is padded to whole 1 KB chunks), all in flight at once
                constexpr int CHUNKS = CL.model_floats / 256;
                const float4 *src = args.models + (size_t)i * (CL.model_floats / 4) + lane;
#pragma unroll
                for (int c0 = 0; c0 < CHUNKS; c0 += WAVES) {
                    const int c = c0 + wv;
                    if (c < CHUNKS)
                        __builtin_amdgcn_global_load_lds((const void *)(src + c * 64),
                                                         (__attribute__((address_space(3))) void *)(smem4 + c * 64),
                                                         16, 0, 0);
                }
                __builtin_amdgcn_s_waitcnt(0);
            }
            __syncthreads();
            const float *cst = smem + CL.off_cst;
            const float b30 = cst[0], b31 = cst[1];
            const float k0l = cst[2], k0t = cst[3], cbl = cst[4], cbt = cst[5], rml = cst[6], rmt = cst[7];
            const float m3l = cst[8], m3t = cst[9];
            const float sla_i = par[i], om_i = par[32 + i];
            const float sla_hi_i = SIG ? par[96 + i] : 0.f;
            const float tau_i = OBJ ? par[64 + i] : 0.f;
            const int prev_i = OBJ ? par_prev[i] : -1;
            const uint32_t row0 = (uint32_t)par_off[i];

            for (int t = 0; t < TW; t++) {
                // The staged weights are re-read from LDS for every tile: an
                // opaque zero offset keeps the compiler from hoisting those
                // reads out of the tile loop (they would not fit in registers).
                int z0 = 0;
                asm volatile("" : "+v"(z0));
                const uint4 *w2a = reinterpret_cast<const uint4 *>(smem + CL.off_w2a + z0) + lane;
                const float *w1a = smem + CL.off_w1a + z0 + lane;
                const float *b2 = smem + CL.off_b2 + 4 * half + z0;
                const float *w3 = smem + CL.off_w3 + 4 * half + z0;
                const uint64_t off = wbase + (uint64_t)t * 32 + (uint64_t)col;
                const bool valid = off < n;
                uint32_t d[MAXN];
                if (LIST) {
                    uint64_t x = valid ? args.idx_list[off] : 0ull;
#pragma unroll
                    for (int j = MAXN - 1; j >= 0; j--) {
                        if (j < N) {
                            const uint64_t k = (uint64_t)fc.K[j];
                            d[j] = (uint32_t)(x % k);
                            x /= k;
                        } else {
                            d[j] = 0;
                        }
                    }
                } else {
                    uint32_t carry = (uint32_t)(t * 32 + col);
#pragma unroll
                    for (int j = MAXN - 1; j >= 0; j--) {
                        if (j < N) {
                            const uint32_t sj = bd[j] + carry;
                            // FULL kernels run only when every option count exceeds 1
                            const uint32_t q = FULL ? __umulhi(sj, fc.magic[j])
                                                    : (fc.magic[j] ? __umulhi(sj, fc.magic[j]) : sj);
                            d[j] = sj - q * (uint32_t)fc.K[j];
                            carry = q;
                        } else {
                            d[j] = 0;
                        }
                    }
                }
                // this model's option row first, so that the loads of its
                // layer-1 seeds are in flight during the aggregate
                uint64_t dig0 = 0, dig1 = 0;
#pragma unroll
                for (int j = 0; j < MAXN; j++) {
                    if (j < N) {
                        if (j < 8) dig0 |= (uint64_t)d[j] << (8 * j);
                        else dig1 |= (uint64_t)d[j] << (8 * (j - 8));
                    }
                }
                const uint64_t sel = (uint64_t)0 - (uint64_t)(i >= 8);
                const uint64_t dw = dig0 ^ ((dig0 ^ dig1) & sel);
                const uint32_t row = row0 + (uint32_t)((dw >> (8 * (i & 7))) & 0xFFu);
                const float *prow = args.phat + (size_t)row * CL.PST + 4 * half;
                // the seeds of blocks mb and mb + 1 are in flight while block
                // mb - 1 runs (H >= 64, so MB >= 2)
                static_assert(MB >= 2, "two seed blocks in flight");
                floatx16 seed0 = load16(prow), seed1 = load16(prow + 32);

                // aggregate (fp32, model order)
                float ah[4] = {0.f, 0.f, 0.f, 0.f};
                float vsum = 0.f;
#pragma unroll
                for (int j = 0; j < MAXN; j++) {
                    if (j < N) {
                        const uint32_t r = (uint32_t)fc.opt_off[j] + d[j];
                        const float4 v = *reinterpret_cast<const float4 *>(G + r * 8 + 4 * half);
                        ah[0] += v.x;
                        ah[1] += v.y;
                        ah[2] += v.z;
                        ah[3] += v.w;
                        vsum += Gv[r];
                    }
                }

                // ---- layer 1: the canonical fp32 chain, seeded with the
                // option's local part; block mb's MFMAs overlap block mb-1's
                // relu / bf16 packing
                bf16x8 hp[KS];
                float sh = 0.f;
                floatx16 prev1 = seed0;
#pragma unroll
                for (int mb = 0; mb < MB; mb++) {
                    floatx16 acc = seed0;
                    seed0 = seed1;
                    if (mb + 2 < MB) seed1 = load16(prow + 32 * (mb + 2));
#pragma unroll
                    for (int s1 = 0; s1 < S1; s1++)
                        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(w1a[(mb * S1 + s1) * 64], ah[s1], acc, 0, 0, 0);
                    if (mb > 0) layer1_epilogue(prev1, hp[2 * mb - 2], hp[2 * mb - 1], sh);
                    prev1 = acc;
                }
                layer1_epilogue(prev1, hp[KS - 2], hp[KS - 1], sh);

                // ---- layer 2 (bf16 MFMA, A fragments prefetched 4 ahead) and
                // layer 3 (four partial chains per output); block mb2's MFMAs
                // overlap block mb2-1's layer-3 work
                constexpr int PF = 4, NF = MB * KS, EPS = 16 / KS;   // epilogue rows per MFMA step
                uint4 af[PF];
#pragma unroll
                for (int f = 0; f < PF; f++) af[f] = w2a[f * 64];
                float yl[4] = {0.f, 0.f, 0.f, 0.f}, yt[4] = {0.f, 0.f, 0.f, 0.f};
                float s2 = 0.f;
                floatx16 prev2 = {};
                float4 pwl[4], pwt[4];
#pragma unroll
                for (int mb2 = 0; mb2 < MB; mb2++) {
                    floatx16 acc2 = load16(b2 + 32 * mb2);
                    if (mb2 > 0) load_w3(w3 + (mb2 - 1) * 32, w3 + (MB + mb2 - 1) * 32, pwl, pwt);
#pragma unroll
                    for (int ks = 0; ks < KS; ks++) {
                        const int f = mb2 * KS + ks;
                        const uint4 a = af[f % PF];
                        if (f + PF < NF) af[f % PF] = w2a[(f + PF) * 64];
                        bf16x8 av;
                        __builtin_memcpy(&av, &a, 16);
                        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, hp[ks], acc2, 0, 0, 0);
                        // the previous block's relu and layer-3 rows, a share per step
                        if (mb2 > 0) {
#pragma unroll
                            for (int e = 0; e < EPS; e++) layer3_row(prev2, ks * EPS + e, pwl, pwt, yl, yt, s2);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    prev2 = acc2;
                }
                load_w3(w3 + (MB - 1) * 32, w3 + (2 * MB - 1) * 32, pwl, pwt);
#pragma unroll
                for (int r = 0; r < 16; r++) layer3_row(prev2, r, pwl, pwt, yl, yt, s2);

                float ylf = (yl[0] + yl[1]) + (yl[2] + yl[3]);
                float ytf = (yt[0] + yt[1]) + (yt[2] + yt[3]);
                ylf += __shfl_xor(ylf, 32);
                ytf += __shfl_xor(ytf, 32);
                s2 += __shfl_xor(s2, 32);
                sh += __shfl_xor(sh, 32);
                const float lat = ylf + b30;
                const float thr = SIG ? sigmoid_f32(ytf + b31) : ytf + b31;
                // per-configuration bounds on |fast - canonical|, inflated
                // for their own fp32 evaluation (sh and s2 are rounded sums);
                // through the sigmoid (1/4-Lipschitz, fp32 evaluation within
                // 2^-20) for the throughput
                const float el = (k0l + bc.g2 * (cbl + rml * sh * 1.001f) + bc.g3 * m3l * s2) * 1.001f + 1e-30f;
                float et = (k0t + bc.g2 * (cbt + rmt * sh * 1.001f) + bc.g3 * m3t * s2) * 1.001f + 1e-30f;
                if constexpr (SIG) et = et * 0.25f + 0x1p-20f;
                const float slack = SIG ? el + fabsf(lat) * 0x1p-20f + 1e-12f : el + (fabsf(lat) + fabsf(sla_i)) * 0x1p-20f;
                bool pass = lat + slack <= sla_i, fail = lat - slack > (SIG ? sla_hi_i : sla_i);
                float jn, en;
                if constexpr (eq3) {
                    const Eq3Term q3 = eq3_term(args.obj.vrow[2 * row], args.obj.vrow[2 * row + 1], thr, et, om_i,
                                                tau_i, prev_i, args.obj.alpha, args.obj.beta, args.obj.delta);
                    pass = pass && q3.pass;
                    fail = fail || q3.fail;
                    jn = Jt[0] + q3.c;
                    // the fp32 sum over models: N u relative to each term's magnitude
                    en = Et[0] + q3.e + q3.mag * (float)N * 0x1p-22f;
                } else {
                    jn = fmaf(om_i, thr, Jt[0]);
                    en = Et[0] + fabsf(om_i) * (et + bc.gN * fabsf(thr));
                }
                uint32_t fl = Ft[0] | (fail ? kFlagFail : 0u) | ((pass || fail) ? 0u : (1u << i));
                if (i == 0 && (double)vsum <= (double)fc.vram_cap) fl |= kFlagVram;
                // rotate the per-tile state: slot 0 becomes the next tile
#pragma unroll
                for (int u = 0; u < TW - 1; u++) { Jt[u] = Jt[u + 1]; Et[u] = Et[u + 1]; Ft[u] = Ft[u + 1]; }
                Jt[TW - 1] = jn;
                Et[TW - 1] = en;
                Ft[TW - 1] = fl;
                if (args.pred && valid && half == 0) {
                    args.pred[(off * (uint64_t)N + (uint64_t)i) * 2u + 0u] = SIG ? sigmoid_f32(lat) : lat;
                    args.pred[(off * (uint64_t)N + (uint64_t)i) * 2u + 1u] = thr;
                }
            }
        }
        if (LIST) continue;

        // ---- per-configuration decisions (the state is back in tile order)
#pragma unroll
        for (int t = 0; t < TW; t++) {
            const uint64_t off = wbase + (uint64_t)t * 32 + (uint64_t)col;
            const bool mine = off < n && half == 0;
            const bool vram_ok = (Ft[t] & kFlagVram) != 0u;
            const bool anyfail = (Ft[t] & kFlagFail) != 0u;
            const uint32_t umask = Ft[t] & 0xFFFFu;
            const bool sla_sure = !anyfail && umask == 0u;
            const bool feas_sure = mine && vram_ok && sla_sure;
            const bool unc = mine && !anyfail && umask != 0u && (vram_ok || args.mask != nullptr);
            const float U = f32_up((double)Jt[t] + (double)Et[t] * (1.0 + 0x1p-10) + eJ0);
            if (mode == kModeSearch) {
                c_vram += (mine && vram_ok) ? 1u : 0u;
                c_feas += feas_sure ? 1u : 0u;
                work_append(unc, (unsigned long long)(uint32_t)off | ((unsigned long long)umask << 32), U, lane,
                            &args.res->n_work, args.work, args.work_J, args.work_cap);
                const unsigned long long key =
                    feas_sure
                        ? (((unsigned long long)ord_f32(U) << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)off))
                        : 0ull;
                wl_offer(wl, key, lane, kp);
                if (args.mask && mine)
                    args.mask[off] = (uint8_t)((vram_ok ? 1u : 0u) | (sla_sure ? 2u : 0u) | (feas_sure ? 4u : 0u) |
                                               (unc ? 8u : 0u));
            } else {
                list_append(feas_sure && (double)U >= args.theta, (uint32_t)off, lane, &args.res->n_collect,
                            args.collect, args.collect_cap);
            }
        }
    }

    if (!LIST && mode == kModeSearch) {
        // counts and list per workgroup (the merge kernel sums and merges them)
        __shared__ unsigned long long s_cnt[2 * WAVES];
        const unsigned long long sv = wave_sum64(c_vram), sf = wave_sum64(c_feas);
        if (lane == 0) {
            s_cnt[wv] = sv;
            s_cnt[WAVES + wv] = sf;
        }
#pragma unroll
        for (int j = 0; j < 2; j++)
            if (j * 64 + lane < kp) lst[wv * kp + j * 64 + lane] = wl.s[j];
        wl_tree_merge<2, WAVES>(wl, lst, kp, wv, lane, kp);
        if (wv == 0) {
#pragma unroll
            for (int j = 0; j < 2; j++)
                if (j * 64 + lane < kp) args.wg_lists[(uint64_t)blockIdx.x * kp + j * 64 + lane] = wl.s[j];
            if (lane < 2) {
                unsigned long long t = 0;
                for (int w = 0; w < WAVES; w++) t += s_cnt[lane * WAVES + w];
                args.wg_counts[2 * (uint64_t)blockIdx.x + lane] = t;
            }
        }
    }
}

template <int MAXN, int A, int H, bool FULL, bool LIST, bool OBJ, bool SIG = false>
hipError_t launch_bf16_t(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                         hipStream_t s)
{
    const size_t lds = bf16_lds_bytes(a.lay, kp);
    auto fn = fast_bf16_kernel<MAXN, A, H, FULL, LIST, OBJ, SIG>;
    hipError_t e = ensure_dyn_lds((const void *)fn, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kBf16Waves * 64), lds, s, a, fc, bc, mode, kp);
    return hipGetLastError();
}

// Instantiations for one hidden width: search/collect kernels for up to 8 and
// up to 16 models (with exact-count variants), list kernels for up to 16;
// under the full utility of Eq. 3 the exact-8 kernel and the generic one.
template <int H>
hipError_t launch_bf16_for_width(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp,
                                 int mode, hipStream_t s)
{
    const int N = fc.n_models, A = a.lay.A;
    bool multi = true;   // every option count exceeds 1
    for (int j = 0; j < N; j++) multi = multi && fc.K[j] > 1;
    const bool obj = a.obj.kind != 0;
#define MF_BF_CASE(AA)                                                                                          \
    if (A == AA && bc.act) {   /* sigmoid outputs: the generic kernel */                                        \
        if (mode == kModeList) return launch_bf16_t<16, AA, H, false, true, false, true>(a, fc, bc, grid, kp, mode, s); \
        if (obj) return launch_bf16_t<16, AA, H, false, false, true, true>(a, fc, bc, grid, kp, mode, s);       \
        return launch_bf16_t<16, AA, H, false, false, false, true>(a, fc, bc, grid, kp, mode, s);               \
    }                                                                                                           \
    if (A == AA) {                                                                                              \
        if (mode == kModeList) return launch_bf16_t<16, AA, H, false, true, false>(a, fc, bc, grid, kp, mode, s); \
        if (obj) {                                                                                              \
            if (N == 8 && multi) return launch_bf16_t<8, AA, H, true, false, true>(a, fc, bc, grid, kp, mode, s);  \
            return launch_bf16_t<16, AA, H, false, false, true>(a, fc, bc, grid, kp, mode, s);                  \
        }                                                                                                       \
        if (N == 8 && multi) return launch_bf16_t<8, AA, H, true, false, false>(a, fc, bc, grid, kp, mode, s);     \
        if (N <= 8) return launch_bf16_t<8, AA, H, false, false, false>(a, fc, bc, grid, kp, mode, s);            \
        if (N == 16 && multi) return launch_bf16_t<16, AA, H, true, false, false>(a, fc, bc, grid, kp, mode, s);  \
        return launch_bf16_t<16, AA, H, false, false, false>(a, fc, bc, grid, kp, mode, s);                      \
    }
    MF_BF_CASE(2) MF_BF_CASE(4) MF_BF_CASE(6) MF_BF_CASE(8)
#undef MF_BF_CASE
    return hipErrorInvalidValue;
}

}  // namespace mfi
