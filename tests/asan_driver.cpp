// Host-side sanitizer driver for libmf (test infrastructure).
//
// Built by tests/test_sanitizers.py with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code of csrc/mf_api.cpp (device code
// is not instrumented) and linked with the library's other objects.  It calls
// only the C ABI of include/mf.h.
//
//   mf_asan_driver            argument validation and table sizing: no device
//                             call is made
//   mf_asan_driver --device   also creates problems on device 0 and runs every
//                             entry point on small shapes (fp32 and bf16,
//                             linear and Eq. 3, derived and fixed state)
//
// Exit status 0 when every check holds; a sanitizer report aborts the process.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "mf.h"

namespace {

int g_fail = 0;

#define EXPECT(cond)                                                              \
    do {                                                                          \
        if (!(cond)) {                                                            \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            g_fail++;                                                             \
        }                                                                         \
    } while (0)

// splitmix64: seeded values for the synthetic tables
struct Rng {
    uint64_t s;
    uint64_t next()
    {
        uint64_t z = (s += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    // uniform on [a, b), on a 2^-12 grid
    float uni(float a, float b) { return a + (b - a) * (float)(next() >> 52) * 0x1p-12f; }
};

struct Shape {
    std::vector<int32_t> K;
    int L, A, H;
    mf_dtype dt;
};

mf_desc make_desc(const Shape &s, const std::vector<int32_t> &cols)
{
    mf_desc d;
    std::memset(&d, 0, sizeof d);
    d.n_models = (int32_t)s.K.size();
    d.n_local = s.L;
    d.n_agg = s.A;
    d.hidden1 = s.H;
    d.hidden2 = s.H;
    d.h_n_options = s.K.data();
    d.h_agg_cols = cols.data();
    d.vram_slot = 1;
    d.vram_cap = 1e30f;
    d.dtype = s.dt;
    return d;
}

std::vector<int32_t> default_cols(int A, int L)
{
    std::vector<int32_t> c(A);
    for (int a = 0; a < A; a++) c[a] = (3 + a) % L;
    return c;
}

void check_host_only()
{
    for (int s = 0; s <= 8; s++) EXPECT(mf_status_string((mf_status)s) != nullptr);
    EXPECT(mf_status_string((mf_status)99) != nullptr);

    // table sizing over a grid of shapes
    const int Ks[] = {1, 2, 7, 24, 255};
    const int Hs[] = {32, 64, 128, 256};
    size_t nb = 0;
    for (int N = 1; N <= 16; N += 3)
        for (int K : Ks)
            for (int H : Hs)
                for (int dt = 0; dt < 2; dt++) {
                    Shape sh{std::vector<int32_t>(N, K), 8, 4, H, (mf_dtype)dt};
                    auto cols = default_cols(4, 8);
                    mf_desc d = make_desc(sh, cols);
                    mf_status st = mf_problem_bytes(&d, &nb);
                    double space = std::pow((double)K, N);
                    if (space > 1.8e19) {
                        EXPECT(st == MF_EOVERFLOW);
                    } else {
                        EXPECT(st == MF_OK);
                        EXPECT(nb > 0 && nb % 256 == 0);
                    }
                }
    // argument validation before any device call
    Shape sh{{3, 4}, 8, 4, 32, MF_F32};
    auto cols = default_cols(4, 8);
    mf_desc d = make_desc(sh, cols);
    std::vector<float> dummy(64, 0.f);
    mf_problem *p = nullptr;
    auto create = [&](const mf_desc &dd) {
        return mf_problem_create(&dd, dummy.data(), dummy.data(), dummy.data(), 0, nullptr, &p);
    };
    mf_desc b = d;
    b.n_models = 0;
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.n_models = 17;
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.h_n_options = nullptr;
    EXPECT(create(b) == MF_EINVAL);
    std::vector<int32_t> badk{3, 0};
    b = d;
    b.h_n_options = badk.data();
    EXPECT(create(b) == MF_EINVAL);
    std::vector<int32_t> badcols{3, 4, 5, 9};
    b = d;
    b.h_agg_cols = badcols.data();
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.vram_slot = 4;
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.vram_cap = NAN;
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.dtype = (mf_dtype)7;
    EXPECT(create(b) == MF_EINVAL);
    b = d;
    b.hidden1 = 0;
    EXPECT(create(b) == MF_EINVAL);
    EXPECT(create(d) == MF_ENOMEM);   // table buffer below mf_problem_bytes
    EXPECT(mf_problem_create(nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr) == MF_EINVAL);
    EXPECT(mf_problem_bytes(nullptr, &nb) == MF_EINVAL);
    EXPECT(mf_problem_bytes(&d, nullptr) == MF_EINVAL);

    uint64_t u = 0;
    EXPECT(mf_space_size(nullptr, &u) == MF_EINVAL);
    EXPECT(mf_decode(nullptr, 0, nullptr) == MF_EINVAL);
    EXPECT(mf_search(nullptr, nullptr, nullptr, 0, nullptr, nullptr) == MF_EINVAL);
    EXPECT(mf_search_noalloc(nullptr, nullptr, nullptr, nullptr) == MF_EINVAL);
    EXPECT(mf_eval_fast(nullptr, nullptr, 0, nullptr, nullptr) == MF_EINVAL);
    EXPECT(mf_ga_run(nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, nullptr) == MF_EINVAL);
    mf_problem_destroy(nullptr);
}

// ------------------------------------------------------------- device part

#define HIPCHK(x)                                                                        \
    do {                                                                                 \
        hipError_t e_ = (x);                                                             \
        if (e_ != hipSuccess) {                                                          \
            std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            std::exit(3);                                                                \
        }                                                                                \
    } while (0)

template <class T>
T *upload(const std::vector<T> &v)
{
    T *d = nullptr;
    HIPCHK(hipMalloc((void **)&d, std::max<size_t>(1, v.size()) * sizeof(T)));
    if (!v.empty()) HIPCHK(hipMemcpy(d, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice));
    return d;
}

float bf16_trunc(float x)
{
    uint32_t u;
    std::memcpy(&u, &x, 4);
    u &= 0xFFFF0000u;
    std::memcpy(&x, &u, 4);
    return x;
}

struct Instance {
    Shape sh;
    std::vector<int32_t> cols;
    std::vector<float> feat, w;
    std::vector<int32_t> variant, n_var;
    std::vector<float> fmin, fmax, qual, reload;
    float cap;
};

Instance make_instance(const Shape &sh, uint64_t seed)
{
    Instance in{sh, default_cols(sh.A, sh.L), {}, {}, {}, {}, {}, {}, {}, {}, 0.f};
    Rng r{seed};
    int sumK = 0;
    for (int k : sh.K) sumK += k;
    in.feat.resize((size_t)sumK * sh.L);
    for (auto &x : in.feat) x = r.uni(0.f, 1.f);
    const int S = sh.H * (sh.L + sh.A) + sh.H + sh.H * sh.H + sh.H + 2 * sh.H + 2;
    in.w.resize((size_t)sh.K.size() * S);
    for (size_t i = 0; i < in.w.size(); i++) {
        float x = r.uni(-0.35f, 0.35f);
        in.w[i] = sh.dt == MF_BF16 ? bf16_trunc(x) : x;
    }
    // VRAM cap near the middle of the sum of per-model column means
    float mean = 0.f;
    for (size_t m = 0, row = 0; m < sh.K.size(); m++) {
        float s = 0.f;
        for (int k = 0; k < sh.K[m]; k++, row++) s += in.feat[row * sh.L + in.cols[1]];
        mean += s / sh.K[m];
    }
    in.cap = mean;
    in.variant.resize(sumK);
    for (int i = 0; i < sumK; i++) in.variant[i] = i % 2;
    const int N = (int)sh.K.size();
    in.n_var.assign(N, 2);
    in.fmin.assign(N * MF_MAX_VARIANTS, -4.f);
    in.fmax.assign(N * MF_MAX_VARIANTS, 4.f);
    in.qual.assign(N * MF_MAX_VARIANTS, 0.5f);
    in.reload.assign(N, 0.25f);
    return in;
}

void run_device_case(const Shape &sh, bool fast, uint64_t seed)
{
    Instance in = make_instance(sh, seed);
    const int N = (int)sh.K.size();
    mf_variants var{in.variant.data(), in.n_var.data(), in.fmin.data(), in.fmax.data(), in.qual.data(),
                    in.reload.data()};
    mf_desc d = make_desc(sh, in.cols);
    d.vram_cap = in.cap;
    d.variants = &var;
    size_t nb = 0;
    EXPECT(mf_problem_bytes(&d, &nb) == MF_OK);
    float *d_feat = upload(in.feat), *d_w = upload(in.w);
    void *d_tab = nullptr;
    HIPCHK(hipMalloc(&d_tab, nb));
    hipStream_t s;
    HIPCHK(hipStreamCreate(&s));
    mf_problem *p = nullptr;
    EXPECT(mf_problem_create(&d, d_feat, d_w, d_tab, nb, s, &p) == MF_OK);
    if (!p) return;
    HIPCHK(hipFree(d_feat));
    HIPCHK(hipFree(d_w));

    uint64_t space = 0;
    EXPECT(mf_space_size(p, &space) == MF_OK);
    std::vector<int32_t> dig(N);
    EXPECT(mf_decode(p, space - 1, dig.data()) == MF_OK);
    for (int i = 0; i < N; i++) EXPECT(dig[i] == sh.K[i] - 1);
    EXPECT(mf_decode(p, space, dig.data()) == MF_EINVAL);

    std::vector<float> sla(N, 0.8f), om(N, 1.f);
    float *d_sla = upload(sla), *d_om = upload(om);

    for (int obj = 0; obj < 2; obj++)
        for (int fixed = 0; fixed < 2; fixed++) {
            mf_search_args a;
            std::memset(&a, 0, sizeof a);
            a.lo = 0;
            a.hi = space;
            a.top_k = 8;
            a.d_sla = d_sla;
            a.d_omega = d_om;
            if (fixed) {
                a.flags = MF_FIXED_STATE;
                for (int k = 0; k < sh.A; k++) a.state[k] = 0.5f * N;
            }
            if (obj) {
                a.objective.kind = MF_OBJ_EQ3;
                a.objective.alpha = 0.5f;
                a.objective.beta = 0.25f;
                a.objective.delta = 0.1f;
                for (int i = 0; i < N; i++) {
                    a.objective.tau[i] = -INFINITY;
                    a.objective.prev_variant[i] = i % 2 ? 0 : -1;
                }
            }
            size_t wsb = 0;
            const mf_status wst = mf_workspace_size(p, &a, &wsb);
            if (!fixed && !fast) {
                // no fast kernel for this shape: only the fixed-state search runs
                EXPECT(wst == MF_EUNSUPPORTED);
                continue;
            }
            EXPECT(wst == MF_OK);
            void *ws = nullptr;
            HIPCHK(hipMalloc(&ws, std::max<size_t>(wsb, 256)));
            mf_result full{}, lo{}, hi{}, na{};
            EXPECT(mf_search(p, &a, ws, wsb, s, &full) == MF_OK);
            EXPECT(full.n_eval == space && full.n_feas <= full.n_vram && full.n_vram <= space);
            EXPECT(full.n_top == (int)std::min<uint64_t>(8, full.n_feas));
            // two halves: counts add up, the better half-argmax is the argmax
            mf_search_args h = a;
            h.hi = space / 2;
            EXPECT(mf_search(p, &h, ws, wsb, s, &lo) == MF_OK);
            h.lo = space / 2;
            h.hi = space;
            EXPECT(mf_search(p, &h, ws, wsb, s, &hi) == MF_OK);
            EXPECT(lo.n_feas + hi.n_feas == full.n_feas && lo.n_vram + hi.n_vram == full.n_vram);
            if (full.n_top > 0) {
                const bool from_lo = lo.n_top > 0 && (hi.n_top == 0 || lo.top_J[0] >= hi.top_J[0]);
                EXPECT(full.top_idx[0] == (from_lo ? lo.top_idx[0] : hi.top_idx[0]));
            }
            EXPECT(mf_search_noalloc(p, &a, s, &na) == MF_OK);
            EXPECT(na.n_feas == full.n_feas && na.top_idx[0] == full.top_idx[0]);
            // refusals
            mf_search_args bad = a;
            bad.top_k = 0;
            EXPECT(mf_search(p, &bad, ws, wsb, s, &na) == MF_EINVAL);
            bad = a;
            bad.hi = space + 1;
            EXPECT(mf_search(p, &bad, ws, wsb, s, &na) == MF_EOVERFLOW);
            bad = a;
            bad.d_sla = nullptr;
            EXPECT(mf_search(p, &bad, ws, wsb, s, &na) == MF_EINVAL);
            EXPECT(mf_search(p, &a, ws, wsb / 2, s, &na) != MF_OK);
            HIPCHK(hipFree(ws));
        }

    // index lists
    std::vector<uint64_t> idx;
    for (uint64_t t = 0; t < 300; t++) idx.push_back((t * 7919u) % space);
    uint64_t *d_idx = upload(idx);
    float *d_pred = nullptr;
    double *d_pc = nullptr, *d_J = nullptr;
    uint32_t *d_fl = nullptr;
    HIPCHK(hipMalloc((void **)&d_pred, idx.size() * N * 2 * sizeof(float)));
    HIPCHK(hipMalloc((void **)&d_pc, idx.size() * N * 2 * sizeof(double)));
    HIPCHK(hipMalloc((void **)&d_J, idx.size() * sizeof(double)));
    HIPCHK(hipMalloc((void **)&d_fl, idx.size() * sizeof(uint32_t)));
    const mf_status fst = mf_eval_fast(p, d_idx, (int64_t)idx.size(), d_pred, s);
    EXPECT(fst == (fast ? MF_OK : MF_EUNSUPPORTED));
    EXPECT(mf_eval_canonical(p, d_idx, (int64_t)idx.size(), d_sla, d_om, d_pc, d_J, d_fl, s) == MF_OK);
    HIPCHK(hipStreamSynchronize(s));
    if (fast) {
        std::vector<float> pf(idx.size() * N * 2);
        std::vector<double> pc(idx.size() * N * 2);
        HIPCHK(hipMemcpy(pf.data(), d_pred, pf.size() * 4, hipMemcpyDeviceToHost));
        HIPCHK(hipMemcpy(pc.data(), d_pc, pc.size() * 8, hipMemcpyDeviceToHost));
        for (size_t t = 0; t < pf.size(); t++) EXPECT(std::fabs(pf[t] - pc[t]) <= 2e-2 * (1.0 + std::fabs(pc[t])));
    }

    // static search and evaluation over two steps
    {
        const int T = 2;
        std::vector<float> sla2(T * N, 0.8f), om2(T * N, 1.f), st2(T * sh.A, 0.5f * N);
        float *d_sla2 = upload(sla2), *d_om2 = upload(om2);
        mf_static_args sa;
        std::memset(&sa, 0, sizeof sa);
        sa.lo = 0;
        sa.hi = space;
        sa.top_k = 4;
        sa.n_steps = T;
        sa.d_sla = d_sla2;
        sa.d_omega = d_om2;
        sa.h_state = st2.data();
        size_t wsb = 0;
        EXPECT(mf_static_workspace_size(p, &sa, &wsb) == MF_OK);
        void *ws = nullptr;
        HIPCHK(hipMalloc(&ws, std::max<size_t>(wsb, 256)));
        mf_result r{};
        EXPECT(mf_search_static(p, &sa, ws, wsb, s, &r) == MF_OK);
        EXPECT(r.n_feas <= r.n_vram && r.n_vram <= space);
        double *d_S = nullptr;
        HIPCHK(hipMalloc((void **)&d_S, idx.size() * sizeof(double)));
        EXPECT(mf_eval_static(p, &sa, d_idx, (int64_t)idx.size(), nullptr, d_S, nullptr, ws, wsb, s) == MF_OK);
        HIPCHK(hipStreamSynchronize(s));
        HIPCHK(hipFree(d_S));
        HIPCHK(hipFree(ws));
        HIPCHK(hipFree(d_sla2));
        HIPCHK(hipFree(d_om2));
    }

    // GA over three scenarios
    {
        const int S = 3;
        std::vector<float> slaS(S * N, 0.8f), omS(S * N, 1.f);
        float *d_slaS = upload(slaS), *d_omS = upload(omS);
        mf_ga_args g;
        std::memset(&g, 0, sizeof g);
        g.n_scen = S;
        g.pop = 64;
        g.gens = 5;
        g.tourn_k = 3;
        g.p_cx = 0.7f;
        g.p_swap = 0.5f;
        g.p_mut = 0.05f;
        g.seed = seed;
        g.d_sla = d_slaS;
        g.d_omega = d_omS;
        size_t wsb = 0;
        EXPECT(mf_ga_workspace_size(p, &g, &wsb) == MF_OK);
        void *ws = nullptr;
        HIPCHK(hipMalloc(&ws, std::max<size_t>(wsb, 256)));
        std::vector<uint64_t> bi(S);
        std::vector<double> bJ(S);
        EXPECT(mf_ga_run(p, &g, ws, wsb, s, bi.data(), bJ.data(), nullptr) == MF_OK);
        for (int k = 0; k < S; k++) EXPECT(bi[k] == UINT64_MAX || bi[k] < space);
        HIPCHK(hipFree(ws));
        HIPCHK(hipFree(d_slaS));
        HIPCHK(hipFree(d_omS));
    }

    mf_problem_destroy(p);
    HIPCHK(hipStreamSynchronize(s));
    HIPCHK(hipStreamDestroy(s));
    for (void *q : {(void *)d_tab, (void *)d_sla, (void *)d_om, (void *)d_idx, (void *)d_pred, (void *)d_pc,
                    (void *)d_J, (void *)d_fl})
        HIPCHK(hipFree(q));
}

}  // namespace

int main(int argc, char **argv)
{
    check_host_only();
    std::printf("host-only checks: %d failures\n", g_fail);
    if (argc > 1 && std::strcmp(argv[1], "--device") == 0) {
        // the last shape has no fast kernel (hidden width 48)
        const struct {
            Shape sh;
            bool fast;
        } cases[] = {
            {{{12, 12, 9, 9, 9}, 8, 4, 32, MF_F32}, true},
            {{{6, 7, 5}, 16, 6, 64, MF_F32}, true},
            {{{5, 4, 3, 2}, 32, 8, 256, MF_BF16}, true},
            {{{5, 3}, 8, 3, 48, MF_F32}, false},
        };
        uint64_t seed = 1;
        for (const auto &c : cases) {
            std::printf("device case N=%zu H=%d dtype=%d\n", c.sh.K.size(), c.sh.H, (int)c.sh.dt);
            std::fflush(stdout);
            run_device_case(c.sh, c.fast, seed++);
        }
        std::printf("device checks: %d failures\n", g_fail);
    }
    return g_fail ? 1 : 0;
}
