// Exhaustive search with the observed state held fixed (Section III-B: the
// aggregate GPU state the surrogates see is observed by the runtime monitor
// and held fixed during the search, the paper's own semantics).
//
// With the aggregate input fixed, model i's prediction depends on its own
// option only, so the surrogates run once per option row (sum_i K_i canonical
// forwards, `fixed_table_kernel`) and the joint search sums table entries
// under the VRAM cap (`fixed_scan_kernel`): per configuration a decode, N LDS
// reads, an fp32 VRAM sum and the canonical fp64 objective chain.  Every value
// the scan combines is canonical, and it combines them in the canonical order,
// so the search is exact without any certification: top-k are selected on
// 128-bit (J, index) keys, per wave, per workgroup, then over the grid.
#include "mf_canon.h"

namespace mfi {

// ---------------------------------------------------------------------------
// Table: one 64-thread workgroup per option row.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ void __launch_bounds__(64) fixed_table_kernel(const FixedArgs a)
{
    __shared__ double h1s[kCanonMaxH];
    __shared__ double h2s[kCanonMaxH];
    __shared__ double zs[kCanonMaxIn];
    __shared__ float s_tau[kMaxN];
    __shared__ int32_t s_prev[kMaxN];
    const int lane = threadIdx.x;
#pragma unroll
    for (int i = 0; i < kMaxN; i++)   // compile-time index into the argument block
        if (lane == i) {
            s_tau[i] = a.obj.tau[i];
            s_prev[i] = a.obj.prev[i];
        }
    const int nin = a.L + a.A;
    for (int r = blockIdx.x; r < a.sumK; r += gridDim.x) {
        const int i = a.row_model[r];
        const float *x = a.features + (int64_t)r * a.L;
        __syncthreads();
        for (int k = lane; k < nin; k += 64) zs[k] = k < a.L ? (double)x[k] : (double)a.state[k - a.L];
        __syncthreads();
        double lat, thr;
        canon_model<BF16>(a.weights + (int64_t)i * a.wstride, nin, a.H1, a.H2, zs, h1s, h2s, lane, lat, thr);
        if (lane == 0) {
            FixedRow row;
            uint32_t fl = lat <= (double)a.sla[i] ? kRowOk : 0u;
            row.q = thr;
            row.P = 0.0;
            row.pen = 0.0;
            if (a.obj.kind != 0) {
                bool do_P, do_pen;
                if (!canon_eq3(a.obj, r, thr, s_tau[i], s_prev[i], row.q, row.P, do_P, row.pen, do_pen)) fl = 0u;
                fl |= (do_P ? kRowP : 0u) | (do_pen ? kRowPen : 0u);
            }
            row.vram = x[a.vram_col];
            row.flags = fl;
            a.rows[r] = row;
            a.pred_rows[r] = make_float2((float)lat, (float)thr);
        }
    }
}

// ---------------------------------------------------------------------------
// Scan: one configuration per lane, 64 per wave and step.
// ---------------------------------------------------------------------------
template <int MAXN>
__global__ void __launch_bounds__(kFixedWaves * 64) fixed_scan_kernel(const FixedArgs a)
{
    extern __shared__ float4 smem4[];
    FixedRow *rows = reinterpret_cast<FixedRow *>(smem4);
    double *om = reinterpret_cast<double *>(rows + a.sumK);
    K128 *lst = reinterpret_cast<K128 *>(om + kMaxN);
    const int N = a.n_models, k = a.top_k;
    for (int t = threadIdx.x; t < a.sumK; t += blockDim.x) rows[t] = a.rows[t];
#pragma unroll
    for (int i = 0; i < kMaxN; i++)
        if (threadIdx.x == (unsigned)i && i < N) om[i] = (double)a.omega[i];
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int gw = blockIdx.x * kFixedWaves + wv;
    const uint64_t n = a.n;
    const uint64_t n_tiles = (n + 63) >> 6;

    // digits of this wave's first tile; advanced by the grid stride in mixed radix
    uint32_t bd[MAXN];
    {
        uint64_t x = a.lo + (uint64_t)gw * 64u;
#pragma unroll
        for (int j = MAXN - 1; j >= 0; j--) {
            if (j < N) {
                bd[j] = (uint32_t)(x % (uint64_t)a.K[j]);
                x /= (uint64_t)a.K[j];
            } else {
                bd[j] = 0;
            }
        }
    }
    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    uint32_t c_vram = 0, c_feas = 0;

    for (uint64_t tile = gw; tile < n_tiles; tile += (uint64_t)a.total_waves) {
        const uint64_t off = tile * 64u + (uint64_t)lane;
        const bool valid = off < n;
        uint32_t carry = (uint32_t)lane;
        float vram = 0.f;
        bool ok = true;
        double J = 0.0;
        uint32_t rowj[MAXN];
#pragma unroll
        for (int j = MAXN - 1; j >= 0; j--) {
            if (j < N) {
                const uint32_t t = bd[j] + carry;
                const uint32_t q = a.magic[j] ? __umulhi(t, a.magic[j]) : t;
                rowj[j] = (uint32_t)a.opt_off[j] + (t - q * (uint32_t)a.K[j]);
                carry = q;
            } else {
                rowj[j] = 0;
            }
        }
        // VRAM sum and the objective chain, model order
#pragma unroll
        for (int j = 0; j < MAXN; j++) {
            if (j < N) {
                const FixedRow r = rows[rowj[j]];
                vram += r.vram;
                ok = ok && (r.flags & kRowOk);
                J = fma(om[j], r.q, J);
                if (r.flags & kRowP) J = J - r.P;
                if (r.flags & kRowPen) J = J - r.pen;
            }
        }
        const bool vram_ok = (double)vram <= (double)a.vram_cap;
        const bool feas = valid && vram_ok && ok;
        c_vram += (valid && vram_ok) ? 1u : 0u;
        c_feas += feas ? 1u : 0u;
        const K128 key = key_if(feas, K128{ord_f64(J), ~(a.lo + off)});
        list128_offer(slot, key, lane, k, thr);
        if (a.mask && valid) {
            a.mask[off] = (uint8_t)((vram_ok ? 1u : 0u) | (ok ? 2u : 0u) | (feas ? 4u : 0u));
#pragma unroll
            for (int j = 0; j < MAXN; j++)
                if (j < N) {
                    const float2 pr = a.pred_rows[rowj[j]];
                    a.pred[(off * (uint64_t)N + (uint64_t)j) * 2u + 0u] = pr.x;
                    a.pred[(off * (uint64_t)N + (uint64_t)j) * 2u + 1u] = pr.y;
                }
        }
        // advance the base digits by the grid stride
        uint32_t c2 = 0;
#pragma unroll
        for (int j = MAXN - 1; j >= 0; j--) {
            if (j < N) {
                const uint32_t t = bd[j] + a.stride_digits[j] + c2;
                c2 = t >= (uint32_t)a.K[j] ? 1u : 0u;
                bd[j] = c2 ? t - (uint32_t)a.K[j] : t;
            }
        }
    }

    const unsigned long long sv = wave_sum64(c_vram), sf = wave_sum64(c_feas);
    if (lane == 0) {
        if (sv) atomicAdd(&a.res->n_vram, sv);
        if (sf) atomicAdd(&a.res->n_feas_sure, sf);
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
        for (int w = 1; w < kFixedWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        if (lane < k) a.wg_lists[(uint64_t)blockIdx.x * k + lane] = slot;
    }
}

// ---------------------------------------------------------------------------
// Merge: the workgroup lists into the final top-k (one workgroup).
// ---------------------------------------------------------------------------
constexpr int kFixedMergeWaves = 16;

__global__ void __launch_bounds__(kFixedMergeWaves * 64)
fixed_merge_kernel(const K128 *lists, int n_lists, int k, DevResult *R)
{
    __shared__ K128 lst[kFixedMergeWaves * 64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    K128 slot = {0ull, 0ull}, thr = {0ull, 0ull};
    const int64_t n_keys = (int64_t)n_lists * k;
    for (int64_t base = (int64_t)wv * 64; base < n_keys; base += kFixedMergeWaves * 64) {
        const int64_t e = base + lane;
        K128 key = {0ull, 0ull};
        if (e < n_keys) key = lists[e];
        list128_offer(slot, key, lane, k, thr);
    }
    lst[wv * 64 + lane] = key_if(lane < k, slot);
    __syncthreads();
    if (wv == 0) {
        for (int w = 1; w < kFixedMergeWaves; w++) list128_offer(slot, lst[w * 64 + lane], lane, k, thr);
        const int n_top = __popcll(__ballot(lane < k && nz128(slot)));
        if (lane < MF_MAX_TOPK) {
            const bool ok = lane < n_top;
            R->top_idx[lane] = ok ? ~slot.lo : ~0ull;
            R->top_J[lane] = ok ? unord_f64(slot.hi) : -INFINITY;
        }
        if (lane == 0) {
            R->n_top = n_top;
            R->status |= kStatVerified;
        }
    }
}

size_t fixed_lds_bytes(int sumK)
{
    return (size_t)sumK * sizeof(FixedRow) + kMaxN * 8 + (size_t)kFixedWaves * 64 * sizeof(K128);
}

hipError_t launch_fixed(const FixedArgs &a, int grid, bool table, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1)
{
    hipError_t e;
    if (table) {
        if (a.bf16)
            hipLaunchKernelGGL(fixed_table_kernel<true>, dim3(a.sumK), dim3(64), 0, s, a);
        else
            hipLaunchKernelGGL(fixed_table_kernel<false>, dim3(a.sumK), dim3(64), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const size_t lds = fixed_lds_bytes(a.sumK);
    auto fn = a.n_models <= 8 ? fixed_scan_kernel<8> : fixed_scan_kernel<16>;
    e = hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if ((e = hipEventRecord(ev0, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kFixedWaves * 64), lds, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hipEventRecord(ev1, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(fixed_merge_kernel, dim3(1), dim3(kFixedMergeWaves * 64), 0, s, a.wg_lists, grid, a.top_k,
                       a.res);
    return hipGetLastError();
}

}  // namespace mfi
