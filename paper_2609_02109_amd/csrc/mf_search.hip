// Fast path of the exhaustive surrogate search (fp32 MFMA), gfx950.
//
// One wave evaluates a tile of 32 consecutive joint indices per step:
//   decode       mixed-radix digits (Eq. 1) by odometer: the wave decodes its
//                first tile once and then adds a fixed stride in mixed radix;
//                each lane adds its column (0..31) with carries
//   aggregate    fp32 sum in model order of every model's option row
//                (the aggregate field of Section III-B), from LDS; slot 0 is
//                the VRAM sum, compared with the cap (Eq. 4)
//   surrogate    per model (Eq. 6): layer 1 = per-option precompute
//                P[row] = b1 + W1_local x (the option's own columns, done once
//                per option) as the accumulator init, plus W1_agg a on MFMA;
//                layer 2 on binary16 matrix cores at fp32-level accuracy: the
//                layer-1 accumulator registers are split into two binary16
//                pieces each (x1 = x truncated, x2 = the rest truncated), W2
//                into two precomputed pieces (w1 + w2), and the three leading
//                cross products x1 w1 + x1 w2 + x2 w1 run on
//                v_mfma_f32_32x32x16_f16 with fp32 accumulation (the dropped
//                term and the pieces' truncation are below 2^-20 relative, and
//                go into the a-priori bound); power-of-two scales folded into
//                the layer-1, b2 and W3 tables keep every piece inside the
//                binary16 range without changing any fp32 rounding; the
//                accumulator row order is absorbed into W2's A-operand layout;
//                layer 3 (2 outputs) on VALU with one cross-half add
//   mask/score   latency bound per model decided with an a-priori error bound:
//                sure pass, sure fail, or "left to canonical re-evaluation";
//                J = fma chain over models of omega_i thr_i
//   top-K'       sure-feasible keys (J, lowest index) kept in a sorted
//                register list per wave (lane l holds slot l), merged per
//                workgroup at the end
// Everything the kernel reads per configuration lives in LDS; the only HBM
// traffic is the image load in the prologue and O(K') results.
#include "mf_canon.h"

namespace mfi {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f16x8 as_f16x8(uint4 v)
{
    f16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

__device__ __forceinline__ uint32_t pk_f16_rtz(float a, float b)
{
    const auto h = __builtin_amdgcn_cvt_pkrtz(a, b);
    uint32_t u;
    __builtin_memcpy(&u, &h, 4);
    return u;
}

// x - x1 for the binary16 value x1 in the low (HI = false) or high half of
// the packed register p: one mixed-precision fma, exact (x1 is x truncated).
// Its result feeds only vector instructions the compiler emits itself (the
// packing below), so the compiler's own wait states cover every matrix-core
// read of the pieces.
template <bool HI>
__device__ __forceinline__ float f16_residual(uint32_t p, float x)
{
    float r;
    if constexpr (HI)
        asm("v_fma_mix_f32 %0, -%1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(p), "v"(x));
    else
        asm("v_fma_mix_f32 %0, -%1, 1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(p), "v"(x));
    return r;
}

// The pair (a, b) as binary16 pieces: *x1 = (a, b) rounded toward zero,
// return (a - a1, b - b1) rounded to nearest.  |x - x1 - x2| <= 2^-21 |x| +
// 2^-24 (binary16 subnormals are kept, by the conversions under the kernel's
// denormal mode and by the matrix cores).
__device__ __forceinline__ uint32_t split_f16_pair(float a, float b, uint32_t *x1)
{
    const uint32_t h = pk_f16_rtz(a, b);
    typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
    const f16x2 l = {(_Float16)f16_residual<false>(h, a), (_Float16)f16_residual<true>(h, b)};
    uint32_t u;
    __builtin_memcpy(&u, &l, 4);
    *x1 = h;
    return u;
}

// Eight fp32 values v[r0 .. r0 + 7] as two binary16 B operands (x1, x2).
__device__ __forceinline__ void split_f16x8(const floatx16 &v, int r0, f16x8 &hi, f16x8 &lo)
{
    uint32_t h[4], l[4];
#pragma unroll
    for (int t = 0; t < 4; t++) l[t] = split_f16_pair(v[r0 + 2 * t], v[r0 + 2 * t + 1], &h[t]);
    __builtin_memcpy(&hi, h, 16);
    __builtin_memcpy(&lo, l, 16);
}

// Bytes of LDS (after the workgroup lists) the certification tail needs: the
// evaluated list keys, a status word, per (entry, model) predictions of one
// chunk of kCertChunk entries, and each chunk entry's option rows.
constexpr int kCertChunk = 64;
size_t fast_small_epilogue_bytes(int n_models)
{
    return 64 * 8 + 16 + (size_t)kCertChunk * n_models * 16 + (size_t)kCertChunk * kMaxN * 4 +
           (size_t)kSearchWavesWide * 64 * 8 + (size_t)kCertChunk * sizeof(K128);
}

// One model's surrogate (Eq. 6) on canonical semantics, by one wave with no
// barriers: one configuration (lane u computes hidden unit u, H <= 64), or,
// when PAIR (H <= 32 and at most 32 inputs), two configurations of the same
// model, one per 32-lane half.  Each unit's chain takes its inputs in
// ascending order.  The inputs of a layer (z, then h1, then h2: input k of a
// half in its lane k) pass through the wave's 64 doubles of LDS, xb, and are
// read back at one address per half (a broadcast read), so that the VALU
// issues the chains themselves.  cb is the model's canonical fp32 block
// (W1T[nin][H], b1[H], W2T[H][H], b2[H], W3[2][H], b3[2]; LDS or global):
// lane u reads column u of a transposed matrix, consecutive lanes consecutive
// words.  fp32 weights are exact in fp64.  A wave's LDS accesses complete in
// program order; wave barriers keep the compiler from moving them across a
// layer's store.  Outputs: (lat, thr) of the configuration of half h in lanes
// 32 h and 32 h + 1 of y.
template <int H, bool PAIR>
__device__ inline double canon_forward_block(const float *cb, int nin, double z, int lane, bool sigmoid, double *xb)
{
    static_assert(!PAIR || H <= 32, "two configurations per wave need H <= 32");
    const int uu = PAIR ? (lane & 31) : lane;
    const int u = uu < H ? uu : H - 1;   // lanes past H repeat the last unit and are ignored
    const int hb = PAIR ? (lane & 32) : 0;
    const float *c1 = cb, *w2t = cb + nin * H + H, *b2 = w2t + H * H, *w3 = b2 + H, *b3 = w3 + 2 * H;
    xb[lane] = z;
    __builtin_amdgcn_wave_barrier();
    double c = (double)c1[nin * H + u];
    int k = 0;
    for (; k + 8 <= nin; k += 8) {
        float wv[8];
        double zk[8];
#pragma unroll
        for (int j = 0; j < 8; j++) {
            wv[j] = c1[(k + j) * H + u];
            zk[j] = xb[hb + k + j];
        }
#pragma unroll
        for (int j = 0; j < 8; j++) c = fma((double)wv[j], zk[j], c);
    }
    for (; k < nin; k++) c = fma((double)c1[k * H + u], xb[hb + k], c);
    __builtin_amdgcn_wave_barrier();
    xb[lane] = c > 0.0 ? c : 0.0;   // h1
    __builtin_amdgcn_wave_barrier();
    c = (double)b2[u];
#pragma unroll
    for (int u0 = 0; u0 < H; u0 += 8) {
        float wv[8];
        double hk[8];
#pragma unroll
        for (int j = 0; j < 8; j++) {
            wv[j] = w2t[(u0 + j) * H + u];
            hk[j] = xb[hb + u0 + j];
        }
#pragma unroll
        for (int j = 0; j < 8; j++) c = fma((double)wv[j], hk[j], c);
    }
    __builtin_amdgcn_wave_barrier();
    xb[lane] = c > 0.0 ? c : 0.0;   // h2
    __builtin_amdgcn_wave_barrier();
    // layer 3: lanes 32 h + o, W3[o][v] contiguous in v
    const int o = lane & 1;
    c = (double)b3[o];
#pragma unroll
    for (int v0 = 0; v0 < H; v0 += 8) {
        float wv[8];
        double hk[8];
#pragma unroll
        for (int j = 0; j < 8; j++) {
            wv[j] = w3[o * H + v0 + j];
            hk[j] = xb[hb + v0 + j];
        }
#pragma unroll
        for (int j = 0; j < 8; j++) c = fma((double)wv[j], hk[j], c);
    }
    return sigmoid ? canon_sigmoid(c) : c;
}

// Small ranges, after the scan: the workgroup evaluates canonically (the
// defining semantics) its first eval_top list entries and the configurations
// of its certification segment, one wave per (entry, model), then each
// entry's constraints and J in model order (Section II, Eq. 3 and 4).  The
// image stays in LDS; the tail's buffers follow the workgroup lists.
// listkey: wave 0 holds the workgroup's sorted list, slot lane.
template <int H, int WAVES, bool OBJ, bool SIG>
__device__ inline void small_certify(const FastArgs &args, const FastConst &fc, float *smem, float *par,
                                     unsigned long long listkey, int kp, unsigned int n_offered, int lane, int wv,
                                     unsigned long long t_start)
{
    const FastLayout &Ly = args.lay;
    const int N = fc.n_models, L = args.n_local, A = Ly.A, nin = L + A, T = args.eval_top;
    const uint64_t g = blockIdx.x;
    const int *pK = reinterpret_cast<const int *>(par + 112), *pOff = reinterpret_cast<const int *>(par + 48);
    const int *pPrev = reinterpret_cast<const int *>(par + 80);
    unsigned long long *ekey = reinterpret_cast<unsigned long long *>(par + kFastPar) +
                               (args.lst_off == 0 ? 0 : WAVES * kp);   // [64]
    unsigned int *estat = reinterpret_cast<unsigned int *>(ekey + 64);                               // status, rest
    double *eout = reinterpret_cast<double *>(ekey + 66);                                            // [chunk][N][2]
    int *erow = reinterpret_cast<int *>(eout + (size_t)kCertChunk * N * 2);                          // [chunk][kMaxN]
    static_assert(WAVES <= kSearchWavesWide, "one 64-double forward buffer per wave");
    double *xb = reinterpret_cast<double *>(erow + kCertChunk * kMaxN) + wv * 64;
    // the chunk's canonical keys (J, joint index; 0 when infeasible)
    K128 *eck = reinterpret_cast<K128 *>(reinterpret_cast<double *>(erow + kCertChunk * kMaxN) + kSearchWavesWide * 64);
    if (wv == 0) {
        ekey[lane] = lane < T ? listkey : 0ull;
        // a bound on the upper bound U of every sure-feasible configuration
        // of the workgroup left unevaluated: list entry T when the list goes
        // past T, its last entry (itself evaluated) when T covers the whole
        // list; 0 when the list ends before (nothing left)
        const unsigned long long rest = readlane64(listkey, T < kp ? T : kp - 1);
        if (lane == 0) {
            estat[0] = 0;
            estat[1] = (uint32_t)(rest >> 32);
            estat[2] = 0;   // segment entries found feasible
        }
    }
    __syncthreads();
    // wave 0: the workgroup's best wg_k canonical keys so far
    K128 tslot = {0ull, 0ull}, tthr = {0ull, 0ull};
    const int n_list = __popcll(__ballot(lane < T && ekey[lane] != 0ull));
    const int n_seg = (int)(n_offered < args.seg_cap ? n_offered : args.seg_cap);
    const int n_ent = n_list + n_seg;
    const int *pCols = reinterpret_cast<const int *>(par + 144);
    const float *feat = Ly.off_feat >= 0 ? smem + Ly.off_feat : args.features;
    const bool pair = H <= 32 && nin <= 32;
    for (int c0 = 0; c0 < n_ent; c0 += kCertChunk) {
        const int nc = n_ent - c0 < kCertChunk ? n_ent - c0 : kCertChunk;
        // each entry's option rows (model order)
        for (int t = threadIdx.x; t < nc; t += WAVES * 64) {
            const int e = c0 + t;
            uint64_t x = args.lo + (e < n_list ? 0xFFFFFFFFu - (uint32_t)(ekey[e] & 0xFFFFFFFFull)
                                               : (uint32_t)args.seg[g * args.seg_cap + (e - n_list)]);
            for (int j = N - 1; j >= 0; j--) {
                const uint64_t kj = (uint64_t)pK[j];
                erow[t * kMaxN + j] = pOff[j] + (int)(x % kj);
                x /= kj;
            }
        }
        __syncthreads();
        // items (entry group, model): one entry per wave, or two (one per
        // half) when the model fits a half
        const int per = pair ? 2 : 1;
        const int n_grp = (nc + per - 1) / per;
        for (int q = wv; q < n_grp * N; q += WAVES) {
            const int p = q / N, i = q % N;
            const int half = pair ? (lane >> 5) : 0, kl = pair ? (lane & 31) : lane;
            const int t_raw = p * per + half;
            const int t = t_raw < nc ? t_raw : nc - 1;   // a spare half repeats the last entry
            const int *rows = erow + t * kMaxN;
            double z = 0.0;
            if (kl < L) {
                z = (double)feat[rows[i] * L + kl];
            } else if (kl < nin) {
                const int col = pCols[kl - L];
                int rj[kMaxN];
#pragma unroll
                for (int j = 0; j < kMaxN; j++) rj[j] = j < N ? rows[j] : 0;
                float sa = 0.f;
#pragma unroll
                for (int j = 0; j < kMaxN; j++)
                    if (j < N) sa = sa + feat[rj[j] * L + col];
                z = (double)sa;
            }
            const float *cb = Ly.off_c1 >= 0 ? smem + Ly.off_c1 + i * Ly.c1_stride
                                             : args.canon + (int64_t)i * args.wstride;
            double y;
            if constexpr (H <= 32) {
                y = pair ? canon_forward_block<H, true>(cb, nin, z, lane, SIG, xb)
                         : canon_forward_block<H, false>(cb, nin, z, lane, SIG, xb);
            } else {
                y = canon_forward_block<H, false>(cb, nin, z, lane, SIG, xb);
            }
            const double lat0 = readlane_f64(y, 0), thr0 = readlane_f64(y, 1);
            const double lat1 = readlane_f64(y, 32), thr1 = readlane_f64(y, 33);
            if (lane == 0) {
                const int tq = p * per;
                eout[2 * (tq * N + i)] = lat0;
                eout[2 * (tq * N + i) + 1] = thr0;
                if (pair && tq + 1 < nc) {
                    eout[2 * ((tq + 1) * N + i)] = lat1;
                    eout[2 * ((tq + 1) * N + i) + 1] = thr1;
                }
            }
        }
        __syncthreads();
        for (int t = threadIdx.x; t < nc; t += WAVES * 64) {
            const int e = c0 + t;
            const uint32_t off = e < n_list ? 0xFFFFFFFFu - (uint32_t)(ekey[e] & 0xFFFFFFFFull)
                                            : (uint32_t)args.seg[g * args.seg_cap + (e - n_list)];
            const int vcol = pCols[args.vram_slot];
            float va = 0.f;
            for (int j = 0; j < N; j++) va = va + feat[erow[t * kMaxN + j] * L + vcol];
            const bool vram_ok = (double)va <= (double)fc.vram_cap;
            bool sla_ok = true;
            double J = 0.0;
            for (int i = 0; i < N; i++) {
                const double lat = eout[2 * (t * N + i)], thr = eout[2 * (t * N + i) + 1];
                if (!(lat <= (double)par[128 + i])) sla_ok = false;
                if constexpr (OBJ) {
                    double qv, P, pen;
                    bool do_P, do_pen;
                    if (!canon_eq3(args.obj, erow[t * kMaxN + i], thr, par[64 + i], pPrev[i], qv, P, do_P, pen,
                                   do_pen))
                        sla_ok = false;
                    J = fma((double)par[32 + i], qv, J);
                    if (do_P) J = J - P;
                    if (do_pen) J = J - pen;
                } else {
                    J = fma((double)par[32 + i], thr, J);
                }
            }
            const bool feas = vram_ok && sla_ok;
            eck[t] = feas ? K128{ord_f64(J), ~(args.lo + (uint64_t)off)} : K128{0ull, 0ull};
            if (e < n_list) {
                // a sure-feasible fast decision must be canonically feasible,
                // and the key's U must bound the canonical J
                const double U = (double)unord_f32((uint32_t)(ekey[e] >> 32));
                if (!feas || !(U - J >= 0.0)) atomicOr(&estat[0], kStatSelfCheck);
            } else {
                if (feas) atomicAdd(&estat[2], 1u);
                if (args.mask)
                    args.mask[off] = (uint8_t)((vram_ok ? 1u : 0u) | (sla_ok ? 2u : 0u) | (feas ? 4u : 0u) | 8u);
            }
        }
        __syncthreads();
        // wave 0 takes the chunk's keys (kCertChunk = 64: one per lane); the
        // next chunk writes eck only after two more barriers
        static_assert(kCertChunk == 64, "one key per lane");
        if (wv == 0) list128_offer_many(tslot, lane < nc ? eck[lane] : K128{0ull, 0ull}, lane, args.wg_k, tthr);
    }
    if (wv == 0 && lane < args.wg_k) args.wg_top[g * (uint64_t)args.wg_k + lane] = tslot;
    if (threadIdx.x == 0) {
        unsigned long long *r = args.wg_rec + 8 * g;
        r[0] = n_offered;
        r[1] = t_start;
        r[2] = (unsigned long long)wall_clock64();
        r[3] = ((unsigned long long)estat[0] << 32) | estat[1];
        r[4] = estat[2];
    }
}

// OBJ: score with the full utility of Eq. 3 (otherwise the linear objective).
// SIG: the surrogates' outputs pass a sigmoid; the latency decision then
// compares the pre-activation with logit thresholds.
template <int MAXN, int A, int H, int WAVES, bool OBJ, bool SIG = false>
__global__ void __launch_bounds__(WAVES * 64, 1)
fast_kernel(const FastArgs args, const FastConst fc, const int mode, const int kp)
{
    constexpr int MB = H / 32;         // 32-row blocks of a hidden layer
    static_assert(A <= 8, "layer 1 takes at most 4 aggregate slots per lane half");
    constexpr bool L1ONE = A <= 4;     // two slots per lane half: one layer-1 instruction per block
    constexpr int AP = 8;              // aggregate row stride in LDS: [half][4]
    extern __shared__ float4 smem4[];
    float *smem = reinterpret_cast<float *>(smem4);
    const FastLayout &Ly = args.lay;
    const int N = fc.n_models;

    for (int t = threadIdx.x; t < args.image_f4; t += blockDim.x) smem4[t] = args.image[t];
    // [0,16) sla_lo  [16,32) sla_hi  [32,48) omega  [48,64) first option row per model (int)
    // [64,80) floor tau  [80,96) previous variant (int)  [96,112) throughput bound
    // [112,128) option count per model (int)  [128,144) latency bound  [144,160) aggregate column (int)
    float *par = smem + Ly.total_floats;
    int *par_off = reinterpret_cast<int *>(par + 48);
    int *par_prev = reinterpret_cast<int *>(par + 80);
    unsigned long long *lst = reinterpret_cast<unsigned long long *>(smem + args.lst_off);
#pragma unroll
    for (int i = 0; i < kMaxN; i++) {
        // compile-time index into the argument block (keeps it out of scratch)
        if (threadIdx.x == (unsigned)i && i < N) {
            const double s = (double)args.sla[i], b = fc.bound_lat[i];
            if constexpr (SIG) {
                // canonical sigmoid within 2^-49 relative of the exact one:
                // pre-activation <= logit(s (1 - 2^-49)) gives a sure pass,
                // > logit(s (1 + 2^-48)) a sure miss (outputs lie in [0, 1])
                auto logit = [](double p) {
                    return p <= 0.0 ? -INFINITY : (p >= 1.0 ? INFINITY : log(p / (1.0 - p)));
                };
                const double lo = s >= 1.0 ? INFINITY : logit(s * (1.0 - 0x1p-49));
                const double hi = s >= 1.0 ? INFINITY : logit(s * (1.0 + 0x1p-48));
                par[i] = isinf(lo) ? (float)lo : (float)(lo - b - ((fabs(lo) + b) * 0x1p-22 + 1e-12));
                par[16 + i] = isinf(hi) ? (float)hi : (float)(hi + b + ((fabs(hi) + b) * 0x1p-22 + 1e-12));
            } else {
                const double slack = (fabs(s) + b) * 0x1p-22 + 1e-30;
                const bool inf = isinf(s);
                par[i] = inf ? (float)s : (float)(s - b - slack);       // lat <= this  => canonical lat <= sla
                par[16 + i] = inf ? (float)s : (float)(s + b + slack);  // lat >  this  => canonical lat >  sla
            }
            par[32 + i] = args.omega[i];
            par_off[i] = fc.opt_off[i];
            reinterpret_cast<int *>(par + 112)[i] = fc.K[i];
            par[128 + i] = args.sla[i];
            if constexpr (OBJ) {
                par[64 + i] = args.obj.tau[i];
                par_prev[i] = args.obj.prev[i];
                par[96 + i] = f32_up(fc.bound_thr[i]);
            }
        }
    }
    if (mode == kModeSearch && args.small && threadIdx.x < (unsigned)Ly.A)
        reinterpret_cast<int *>(par + 144)[threadIdx.x] = args.agg_cols[threadIdx.x];
    constexpr bool eq3 = OBJ;
    // global bound on |fast J - canonical J|: keys and certification entries
    // carry the upper bound U = J + eJ
    const double eJ = bound_eJ(fc, args.omega);
    // small ranges: certification entries counted per workgroup in LDS
    __shared__ unsigned int s_nwork;
    unsigned long long t_start = 0;
    const bool small = mode == kModeSearch && args.small;
    if (threadIdx.x == 0) {
        s_nwork = 0;
        t_start = (unsigned long long)wall_clock64();
    }
    if (mode == kModeSearch && !small && blockIdx.x == 0 && threadIdx.x == 0) args.res->eJ = eJ;
    __syncthreads();

    const int lane = threadIdx.x & 63, half = lane >> 5, col = lane & 31;
    // aggregate centre of the slots this lane feeds to layer 1
    // aggregate centre and power-of-two scale of the slots this lane feeds
    // to layer 1 (read per tile: registers are the kernel's limit)
    const float4 *cen_p = reinterpret_cast<const float4 *>(smem + Ly.off_c + 4 * half);
    const float sx_s[4] = {half ? fc.agg_scale[1][0] : fc.agg_scale[0][0], half ? fc.agg_scale[1][1] : fc.agg_scale[0][1],
                           half ? fc.agg_scale[1][2] : fc.agg_scale[0][2], half ? fc.agg_scale[1][3] : fc.agg_scale[0][3]};
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));   // wave-uniform
    const int gw = blockIdx.x * WAVES + wv;
    const uint64_t n = args.n;
    const uint64_t n_tiles = (n + 31) >> 5;

    uint32_t bd[MAXN];
    if (mode != kModeList) {
        uint64_t x = args.lo + (uint64_t)gw * 32u;
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

    WaveList<1> wl;
    wl_init(wl);
    uint32_t c_vram = 0, c_feas = 0;
    WorkBuf wbuf;   // certification entries (the general search path)
    wbuf.e = 0ull;
    wbuf.j = 0.f;
    wbuf.n = 0;

    for (uint64_t tile = gw; tile < n_tiles; tile += (uint64_t)args.total_waves) {
        const uint64_t off = tile * 32u + (uint64_t)col;
        const bool valid = off < n;
        uint32_t d[MAXN];
        if (mode == kModeList) {
            uint64_t x = args.idx_list[valid ? off : n - 1];
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
            uint32_t carry = (uint32_t)col;
#pragma unroll
            for (int j = MAXN - 1; j >= 0; j--) {
                if (j < N) {
                    const uint32_t t = bd[j] + carry;
                    const uint32_t q = fc.magic[j] ? __umulhi(t, fc.magic[j]) : t;
                    d[j] = t - q * (uint32_t)fc.K[j];
                    carry = q;
                } else {
                    d[j] = 0;
                }
            }
        }

        // aggregate field (model order, fp32).  Lane half h accumulates the
        // slots it feeds to layer 1 as B operand: internal slots 2s + h.
        // Slot 0 (half 0, s 0) is the VRAM sum.
        float ah[4] = {0.f, 0.f, 0.f, 0.f};
        uint64_t dig0 = 0, dig1 = 0;   // digits packed 8 bits each: models 0..7, 8..15
#pragma unroll
        for (int j = 0; j < MAXN; j++) {
            if (j < N) {
                if (j < 8) dig0 |= (uint64_t)d[j] << (8 * j);
                else dig1 |= (uint64_t)d[j] << (8 * (j - 8));
                const uint32_t row = (uint32_t)fc.opt_off[j] + d[j];
                const float4 v = *reinterpret_cast<const float4 *>(smem + Ly.off_g + row * AP + 4 * half);
                ah[0] += v.x;
                ah[1] += v.y;
                ah[2] += v.z;
                ah[3] += v.w;
            }
        }
        const bool vram_ok = ah[0] <= fc.vram_cap;
        // layer 1's B operands, shared by every model of the tile: the lane's
        // slots s (2s + half) as x = 2^ex (a - c) in binary16 pieces x1 + x2.
        // Four slots (A > 4): in k = 8 half + j, j and j + 4 both hold slot
        // j, bx1 its x1, bx2 its x2.  Two slots: one operand, j = 0, 1 and
        // 2, 3 hold x1 of slots 0, 1, j = 4, 5 and 6, 7 their x2.
        f16x8 bx1, bx2;
        {
            const float4 cen = cen_p[0];
            uint32_t q[2], r[2];
            r[0] = split_f16_pair((ah[0] - cen.x) * sx_s[0], (ah[1] - cen.y) * sx_s[1], &q[0]);
            if constexpr (L1ONE) {
                const uint32_t w1[4] = {q[0], q[0], r[0], r[0]};
                __builtin_memcpy(&bx1, w1, 16);
                bx2 = bx1;
            } else {
                r[1] = split_f16_pair((ah[2] - cen.z) * sx_s[2], (ah[3] - cen.w) * sx_s[3], &q[1]);
                const uint32_t w1[4] = {q[0], q[1], q[0], q[1]}, w2[4] = {r[0], r[1], r[0], r[1]};
                __builtin_memcpy(&bx1, w1, 16);
                __builtin_memcpy(&bx2, w2, 16);
            }
        }

        float J = 0.f, EJ = 0.f, MJ = 0.f;   // fast J; under Eq. 3 its bound and magnitude
        bool anyfail = false;
        uint32_t umask = 0;   // models whose service decision is left to the canonical pass
        for (int i = 0; i < N; i++) {
            const uint64_t sel = (uint64_t)0 - (uint64_t)(i >= 8);
            const uint64_t dw = dig0 ^ ((dig0 ^ dig1) & sel);
            const uint32_t row = (uint32_t)par_off[i] + (uint32_t)((dw >> (8 * (i & 7))) & 0xFFu);
            // ---- layer 1: P[row] + W1_agg a
            floatx16 acc1[MB];
            const float *prow = smem + Ly.off_p + row * (uint32_t)Ly.PST + 4 * half;
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const float4 v = *reinterpret_cast<const float4 *>(prow + 32 * mb + 8 * q);
                    acc1[mb][4 * q + 0] = v.x;
                    acc1[mb][4 * q + 1] = v.y;
                    acc1[mb][4 * q + 2] = v.z;
                    acc1[mb][4 * q + 3] = v.w;
                }
            // W1_agg 2^(e1 - ex) in binary16 pieces w1 + w2, row 32 mb + l%32
            // of lane l.  Four slots: 16 bytes per lane and block, w1 (j < 4)
            // then w2 (j >= 4) of the slots 2 (j % 4) + l/32; one A operand
            // for both instructions, w1 x1 + w2 x1, then w1 x2 + w2 x2.  Two
            // slots: 8 bytes, w1 then w2 of slots l/32 and 2 + l/32, read
            // twice into one operand, all four products in one instruction.
            if constexpr (L1ONE) {
                const uint2 *w1a = reinterpret_cast<const uint2 *>(smem + Ly.off_w1a + i * (MB * 64 * 2)) + lane;
#pragma unroll
                for (int mb = 0; mb < MB; mb++) {
                    const uint2 p = w1a[mb * 64];
                    const uint4 a = {p.x, p.y, p.x, p.y};
                    acc1[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_f16x8(a), bx1, acc1[mb], 0, 0, 0);
                }
            } else {
                const uint4 *w1a = reinterpret_cast<const uint4 *>(smem + Ly.off_w1a + i * (MB * 64 * 4)) + lane;
#pragma unroll
                for (int mb = 0; mb < MB; mb++) {
                    const f16x8 a = as_f16x8(w1a[mb * 64]);
                    acc1[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bx1, acc1[mb], 0, 0, 0);
                    acc1[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bx2, acc1[mb], 0, 0, 0);
                }
            }
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int r = 0; r < 16; r++) acc1[mb][r] = relu_f32(acc1[mb][r]);
            // ---- layer 2: b2 + W2 h1.  h1 (the relu'd layer-1 accumulators)
            // becomes binary16 pieces first, K-block by K-block (accumulator
            // registers 8 kh .. 8 kh + 7 of block mb1): x1 = x truncated, x2
            // = (x - x1) rounded to nearest, as many registers as h1 itself
            f16x8 xh[MB][2], xl[MB][2];
#pragma unroll
            for (int mb1 = 0; mb1 < MB; mb1++)
#pragma unroll
                for (int kh = 0; kh < 2; kh++) split_f16x8(acc1[mb1], 8 * kh, xh[mb1][kh], xl[mb1][kh]);
            // W2 as two binary16 pieces (w1 + w2 ~ 2^e2 W2) in the A-operand
            // order of v_mfma_f32_32x32x16_f16: per (mb2, mb1, kh) 1 KB of w1
            // then 1 KB of w2, lane l's 16 bytes holding K-block elements 0..7;
            // the products x1 w1 + x1 w2 + x2 w1 accumulate in fp32.  One
            // output block at a time: block mb2's relu and layer-3 rows (VALU)
            // are independent of block mb2 + 1's matrix instructions.
            const float *b2 = smem + Ly.off_b2 + i * H + 4 * half;
            const uint4 *w2p = reinterpret_cast<const uint4 *>(smem + Ly.off_w2 + i * (H * H)) + lane;
            const float *w3 = smem + Ly.off_w3 + i * (2 * H) + 4 * half;
            float pl = 0.f, pt = 0.f;
#pragma unroll
            for (int mb2 = 0; mb2 < MB; mb2++) {
                floatx16 acc2;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const float4 v = *reinterpret_cast<const float4 *>(b2 + 32 * mb2 + 8 * q);
                    acc2[4 * q + 0] = v.x;
                    acc2[4 * q + 1] = v.y;
                    acc2[4 * q + 2] = v.z;
                    acc2[4 * q + 3] = v.w;
                }
                // the small cross products first, while the accumulator holds
                // only the bias (each matrix instruction's error grows with
                // the accumulator it adds to), then the leading ones, K-block
                // by K-block
                f16x8 wa[MB][2];   // the w1 pieces, kept for the leading products
#pragma unroll
                for (int mb1 = 0; mb1 < MB; mb1++)
#pragma unroll
                    for (int kh = 0; kh < 2; kh++) {
                        wa[mb1][kh] = as_f16x8(w2p[(((mb2 * MB + mb1) * 2 + kh) * 2 + 0) * 64]);
                        const f16x8 wb = as_f16x8(w2p[(((mb2 * MB + mb1) * 2 + kh) * 2 + 1) * 64]);
                        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wb, xh[mb1][kh], acc2, 0, 0, 0);
                        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wa[mb1][kh], xl[mb1][kh], acc2, 0, 0, 0);
                    }
#pragma unroll
                for (int mb1 = 0; mb1 < MB; mb1++)
#pragma unroll
                    for (int kh = 0; kh < 2; kh++)
                        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wa[mb1][kh], xh[mb1][kh], acc2, 0, 0, 0);
                // ---- layer 3 (2 outputs) on VALU, this block's rows
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const float4 wl = *reinterpret_cast<const float4 *>(w3 + ((0 * MB + mb2) * 4 + q) * 8);
                    const float4 wt = *reinterpret_cast<const float4 *>(w3 + ((1 * MB + mb2) * 4 + q) * 8);
                    const float h0 = relu_f32(acc2[4 * q + 0]), h1 = relu_f32(acc2[4 * q + 1]);
                    const float h2 = relu_f32(acc2[4 * q + 2]), h3 = relu_f32(acc2[4 * q + 3]);
                    pl = fmaf(wl.x, h0, pl); pt = fmaf(wt.x, h0, pt);
                    pl = fmaf(wl.y, h1, pl); pt = fmaf(wt.y, h1, pt);
                    pl = fmaf(wl.z, h2, pl); pt = fmaf(wt.z, h2, pt);
                    pl = fmaf(wl.w, h3, pl); pt = fmaf(wt.w, h3, pt);
                }
            }
            pl += __shfl_xor(pl, 32);
            pt += __shfl_xor(pt, 32);
            const float *b3 = smem + Ly.off_b3 + 4 * i;
            const float lat = pl + b3[0];
            const float thr = SIG ? sigmoid_f32(pt + b3[1]) : pt + b3[1];
            bool pass = lat <= par[i], fail = lat > par[16 + i];
            if constexpr (eq3) {
                const Eq3Term t = eq3_term(args.obj.vrow[2 * row], args.obj.vrow[2 * row + 1], thr, par[96 + i],
                                           par[32 + i], par[64 + i], par_prev[i], args.obj.alpha, args.obj.beta,
                                           args.obj.delta);
                fail = fail || t.fail;
                pass = pass && t.pass;
                J += t.c;
                EJ += t.e;
                MJ += t.mag;
            } else {
                J = fmaf(par[32 + i], thr, J);
            }
            anyfail |= fail;
            umask |= (pass || fail) ? 0u : (1u << i);
            if (args.pred && valid && half == 0) {
                args.pred[(off * (uint64_t)N + (uint64_t)i) * 2u + 0u] = SIG ? sigmoid_f32(lat) : lat;
                args.pred[(off * (uint64_t)N + (uint64_t)i) * 2u + 1u] = thr;
            }
        }

        if (mode != kModeList) {
            const bool mine = valid && half == 0;
            const bool anyunc = umask != 0u;
            const bool sla_sure = !anyfail && !anyunc;
            const bool feas_sure = mine && vram_ok && sla_sure;
            // a latency decision the bound cannot settle: re-evaluated
            // canonically when it can change the count (VRAM ok) or, in dump
            // mode, the mask
            const bool unc = mine && !anyfail && anyunc && (vram_ok || args.mask != nullptr);
            // Eq. 3: the sum of per-model bounds, plus the fp32 sum over models
            // (N u relative to the magnitudes)
            const float U = eq3 ? f32_up((double)J + (double)EJ * (1.0 + 0x1p-10) + (double)MJ * N * 0x1p-22 + 1e-30)
                                : f32_up((double)J + eJ);
            if (mode == kModeSearch) {
                c_vram += (mine && vram_ok) ? 1u : 0u;
                c_feas += feas_sure ? 1u : 0u;
                const unsigned long long went = (unsigned long long)(uint32_t)off | ((unsigned long long)umask << 32);
                if (small) {
                    const unsigned long long m = __ballot(unc);
                    if (m) {
                        unsigned int base = 0;
                        if (lane == 0) base = atomicAdd(&s_nwork, (unsigned int)__popcll(m));
                        base = (unsigned int)__builtin_amdgcn_readfirstlane((int)base);
                        const unsigned int slot = base + (unsigned int)__popcll(m & ((1ull << lane) - 1ull));
                        if (unc && slot < args.seg_cap) {
                            const uint64_t at = (uint64_t)blockIdx.x * args.seg_cap + slot;
                            args.seg[at] = went;
                            args.seg_J[at] = U;
                        }
                    }
                } else {
                    wb_append(wbuf, unc, went, U, lane, &args.res->n_work, args.work, args.work_J, args.work_cap);
                }
                const unsigned long long key = feas_sure
                    ? (((unsigned long long)ord_f32(U) << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)off))
                    : 0ull;
                wl_offer_many(wl, key, lane, kp);
                if (args.mask && mine)
                    args.mask[off] = (uint8_t)((vram_ok ? 1u : 0u) | (sla_sure ? 2u : 0u) |
                                               (feas_sure ? 4u : 0u) | (unc ? 8u : 0u));
            } else {
                list_append(feas_sure && (double)U >= args.theta, (uint32_t)off, lane, &args.res->n_collect,
                            args.collect, args.collect_cap);
            }
        }

        if (mode != kModeList) {
            // advance the tile base by the grid stride, in mixed radix
            uint32_t carry = 0;
#pragma unroll
            for (int j = MAXN - 1; j >= 0; j--) {
                if (j < N) {
                    uint32_t t = bd[j] + args.stride_digits[j] + carry;
                    carry = t >= (uint32_t)fc.K[j] ? 1u : 0u;
                    bd[j] = carry ? t - (uint32_t)fc.K[j] : t;
                }
            }
        }
    }

    if (mode == kModeSearch && !small)
        wb_flush(wbuf, lane, &args.res->n_work, args.work, args.work_J, args.work_cap);
    if (mode == kModeSearch) {
        // counts and list per workgroup (the merge kernel sums and merges them)
        __shared__ unsigned long long s_cnt[2 * WAVES];
        const unsigned long long sv = wave_sum64(c_vram), sf = wave_sum64(c_feas);
        if (lane == 0) {
            s_cnt[wv] = sv;
            s_cnt[WAVES + wv] = sf;
        }
        if (args.lst_off == 0) __syncthreads();   // the lists overwrite the weights: every wave's scan is done
        if (lane < kp) lst[wv * kp + lane] = wl.s[0];
        wl_tree_merge<1, WAVES>(wl, lst, kp, wv, lane, kp);
        if (wv == 0) {
            if (lane < kp) args.wg_lists[(uint64_t)blockIdx.x * kp + lane] = wl.s[0];
            if (lane < 2) {
                unsigned long long t = 0;
                for (int w = 0; w < WAVES; w++) t += s_cnt[lane * WAVES + w];
                args.wg_counts[2 * (uint64_t)blockIdx.x + lane] = t;
            }
        }
        if (small) {
            // s_nwork is final: every wave's appends precede the tree merge's barriers
            small_certify<H, WAVES, OBJ, SIG>(args, fc, smem, par, wl.s[0], kp, s_nwork, lane, wv, t_start);
        }
    }
}

// ---------------------------------------------------------------------------
// Merge the per-workgroup lists into one sorted top-kp list (one workgroup).
// ---------------------------------------------------------------------------
constexpr int kMergeWaves = 16;

constexpr int kMergeStageKeys = 4096;   // keys staged in LDS per pass

// Each per-workgroup list is sorted: the lists are staged in LDS a batch at a
// time (every thread loading), wave w merges lists w, w + 16, ... of the
// batch into its own, then wave 0 merges the 16.  The workgroups' counts are
// summed into counts_out[0..1] (VRAM-feasible, surely feasible).
template <int NS>
__global__ void __launch_bounds__(kMergeWaves * 64)
merge_lists_kernel(const unsigned long long *lists, int n_lists, int kp, unsigned long long *out,
                   const unsigned long long *wg_counts, unsigned long long *counts_out)
{
    __shared__ unsigned long long stage[kMergeStageKeys];
    __shared__ unsigned long long lst[kMergeWaves * 64 * NS];
    __shared__ unsigned long long s_cnt[2 * kMergeWaves];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    WaveList<NS> L, L2;   // two independent merge chains per wave
    wl_init(L);
    wl_init(L2);
    const int per_pass = kMergeStageKeys / kp;   // kp <= 128: at least 32 lists
    for (int l0 = 0; l0 < n_lists; l0 += per_pass) {
        const int nl = n_lists - l0 < per_pass ? n_lists - l0 : per_pass;
        __syncthreads();
        for (int t = threadIdx.x; t < nl * kp; t += kMergeWaves * 64) stage[t] = lists[(uint64_t)l0 * kp + t];
        __syncthreads();
        for (int i = wv; i < nl; i += 2 * kMergeWaves) {
            const int i2 = i + kMergeWaves;
            unsigned long long b[NS], b2[NS];
#pragma unroll
            for (int j = 0; j < NS; j++) {
                const bool in = j * 64 + lane < kp;
                b[j] = in ? stage[i * kp + j * 64 + lane] : 0ull;
                b2[j] = in && i2 < nl ? stage[i2 * kp + j * 64 + lane] : 0ull;
            }
            wl_merge_sorted(L, b, lane, kp);
            wl_merge_sorted(L2, b2, lane, kp);
        }
    }
    wl_merge_sorted(L, L2.s, lane, kp);
    unsigned long long cv = 0, cf = 0;
    if (wg_counts)
        for (int i = threadIdx.x; i < n_lists; i += kMergeWaves * 64) {
            cv += wg_counts[2 * (uint64_t)i];
            cf += wg_counts[2 * (uint64_t)i + 1];
        }
    cv = wave_sum64(cv);
    cf = wave_sum64(cf);
    if (lane == 0) {
        s_cnt[wv] = cv;
        s_cnt[kMergeWaves + wv] = cf;
    }
#pragma unroll
    for (int j = 0; j < NS; j++) lst[(wv * NS + j) * 64 + lane] = L.s[j];
    wl_tree_merge<NS, kMergeWaves>(L, lst, NS * 64, wv, lane, kp);
    if (wv == 0) {
#pragma unroll
        for (int j = 0; j < NS; j++)
            if (j * 64 + lane < kp) out[j * 64 + lane] = L.s[j];
        if (wg_counts && lane < 2) {
            unsigned long long t = 0;
            for (int w = 0; w < kMergeWaves; w++) t += s_cnt[lane * kMergeWaves + w];
            counts_out[lane] = t;
        }
    }
}

template <int MAXN, int A, int H, int WAVES>
static hipError_t launch_fast_t(const FastArgs &a, const FastConst &fc, int grid, int kp, int mode,
                                hipStream_t s)
{
    FastArgs b = a;
    b.lst_off = fast_lists_in_image(a.lay, WAVES, kp) ? 0 : a.lay.total_floats + kFastPar;
    const size_t lds = fast_dyn_lds(a.lay, WAVES, kp, (size_t)a.ep_bytes);
    auto fn = a.obj.kind != 0 ? fast_kernel<MAXN, A, H, WAVES, true> : fast_kernel<MAXN, A, H, WAVES, false>;
    if constexpr (MAXN == kMaxN && WAVES == kSearchWaves)   // the sigmoid output runs on the generic kernel
        if (fc.act) fn = a.obj.kind != 0 ? fast_kernel<MAXN, A, H, WAVES, true, true>
                                         : fast_kernel<MAXN, A, H, WAVES, false, true>;
    hipError_t e = ensure_dyn_lds((const void *)fn, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(WAVES * 64), lds, s, b, fc, mode, kp);
    return hipGetLastError();
}

int fast_kernel_supported(int n_models, int A, int H, int kp)
{
    if (n_models < 1 || n_models > 16) return 0;
    if (!(A == 2 || A == 4 || A == 6 || A == 8)) return 0;
    if (!(H == 32 || H == 64)) return 0;
    if (kp < 1 || kp > 64) return 0;
    return 1;
}

// 16 waves per workgroup (4 per SIMD) when the per-wave registers fit 128
// VGPRs (up to 8 models) and the image plus 16 candidate lists fit in LDS.
int fast_waves_for(int n_models, const FastLayout &lay, int kp, int act)
{
    const size_t lds = fast_dyn_lds(lay, kSearchWavesWide, kp, 0);
    return (n_models <= 8 && lds <= (size_t)kFastLdsMax && !act) ? kSearchWavesWide : kSearchWaves;
}

hipError_t launch_fast_impl(const FastArgs &a, const FastConst &fc, int grid, int kp, int mode, hipStream_t s)
{
    const int N = fc.n_models, A = a.lay.A, H = a.lay.H;
    const bool wide = a.waves == kSearchWavesWide;
    if (fc.act) {   // sigmoid outputs: the generic kernel (16 models, base waves)
        if (wide) return hipErrorInvalidValue;
#define MF_FAST_CASE(MN, AA, HH) \
    if (A == AA && H == HH) return launch_fast_t<MN, AA, HH, kSearchWaves>(a, fc, grid, kp, mode, s);
#define MF_FAST_A(MN, HH) MF_FAST_CASE(MN, 2, HH) MF_FAST_CASE(MN, 4, HH) MF_FAST_CASE(MN, 6, HH) MF_FAST_CASE(MN, 8, HH)
        MF_FAST_A(16, 32) MF_FAST_A(16, 64)
#undef MF_FAST_A
#undef MF_FAST_CASE
        return hipErrorInvalidValue;
    }
#define MF_FAST_CASE(MN, AA, HH)                                                                        \
    if (N <= MN && A == AA && H == HH) {                                                                \
        if (wide) return launch_fast_t<MN, AA, HH, kSearchWavesWide>(a, fc, grid, kp, mode, s);         \
        return launch_fast_t<MN, AA, HH, kSearchWaves>(a, fc, grid, kp, mode, s);                       \
    }
#define MF_FAST_A(MN, HH) MF_FAST_CASE(MN, 2, HH) MF_FAST_CASE(MN, 4, HH) MF_FAST_CASE(MN, 6, HH) MF_FAST_CASE(MN, 8, HH)
    MF_FAST_A(8, 32) MF_FAST_A(8, 64)
#undef MF_FAST_CASE
#define MF_FAST_CASE(MN, AA, HH) \
    if (N <= MN && A == AA && H == HH) return launch_fast_t<MN, AA, HH, kSearchWaves>(a, fc, grid, kp, mode, s);
    MF_FAST_A(16, 32) MF_FAST_A(16, 64)
#undef MF_FAST_A
#undef MF_FAST_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_merge_lists(const unsigned long long *lists, int n_lists, int kp, unsigned long long *out,
                              const unsigned long long *wg_counts, unsigned long long *counts_out, hipStream_t s)
{
    if (kp <= 64)
        hipLaunchKernelGGL(merge_lists_kernel<1>, dim3(1), dim3(kMergeWaves * 64), 0, s, lists, n_lists, kp, out,
                           wg_counts, counts_out);
    else
        hipLaunchKernelGGL(merge_lists_kernel<2>, dim3(1), dim3(kMergeWaves * 64), 0, s, lists, n_lists, kp, out,
                           wg_counts, counts_out);
    return hipGetLastError();
}

}  // namespace mfi

namespace mfi {

// Per-option first-layer precompute (the option's own columns, Eq. 6, plus
// the aggregate centre c the fast path subtracts from the aggregate):
// P[row][h] = b1[h] + sum_k W1[h][k] x[row][k] + sum_k W1_agg[h][k] c[k],
// one fp64 fma chain, rounded to fp32.  Reads the canonical image (W1T[k][h]).
__global__ void precompute_p_kernel(const float *features, const float *canon_w, const float *centre, int n_rows,
                                    int L, int A, int H, int64_t wstride, const int32_t *row_model, float *image_p,
                                    int pst, Pow2Scales sc)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_rows * H) return;
    const int row = (int)(t / H), h = (int)(t % H);
    const int nin = L + A;
    const float *w = canon_w + (int64_t)row_model[row] * wstride;
    const float *W1T = w, *b1 = w + (int64_t)nin * H;
    double c = (double)b1[h];
    for (int k = 0; k < L; k++) c = fma((double)W1T[(int64_t)k * H + h], (double)features[(int64_t)row * L + k], c);
    for (int k = 0; k < A; k++) c = fma((double)W1T[(int64_t)(L + k) * H + h], (double)centre[k], c);
    // the fast image's layer-1 scale 2^e (exact: rounding commutes with it)
    image_p[(int64_t)row * pst + h] = (float)ldexp(c, sc.e[row_model[row]]);
}

hipError_t launch_precompute_p(const float *features, const float *weights, const float *centre, int n_rows, int L,
                               int A, int H, int64_t wstride, const int32_t *row_model, float *image_p, int pst,
                               const Pow2Scales &sc, hipStream_t s)
{
    const int64_t total = (int64_t)n_rows * H;
    const int blk = 256;
    const int grid = (int)((total + blk - 1) / blk);
    hipLaunchKernelGGL(precompute_p_kernel, dim3(grid), dim3(blk), 0, s, features, weights, centre, n_rows, L, A, H,
                       wstride, row_model, image_p, pst, sc);
    return hipGetLastError();
}

}  // namespace mfi
