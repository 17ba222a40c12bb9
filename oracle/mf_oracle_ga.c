/*
 * CPU oracle of the genetic-algorithm scheduler (test infrastructure only;
 * see mf_oracle.c for the rules on who may use the oracle).
 *
 * The paper's GA (Section IV-C): a population of candidate joint
 * configurations, tournament selection (k = 3), crossover, mutation and
 * elitism over a number of generations; VRAM-infeasible offspring are repaired
 * by replacement with a randomly sampled feasible individual and candidates
 * that miss a latency bound score J = -inf (Section II, after Eq. 4).  Fitness
 * is the canonical J of each individual (mf_oracle.c).
 *
 * The paper fixes neither the RNG nor the order of the operators; this is the
 * definition used here (the same one the GPU implements on its own):
 *
 *   RNG: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
 *     as easy as 1, 2, 3", SC'11): ten rounds of the 4x64 Philox round with
 *     the Weyl key schedule.  Key = (seed, 0).  Counter = (item, gen, scen,
 *     purpose); every draw is one 64-bit output word.
 *     uniform(r) = (r >> 11) * 2^-53 (compared as double with the float p);
 *     int(r, n)  = ((r >> 32) * n) >> 32.
 *   Feasible list FL: the VRAM-feasible joint indices in ascending order.
 *   Generation 0: slot j takes FL[int(R(j, 0, s, INIT)[0], |FL|)].
 *   For g = 0..gens: evaluate every individual (fitness f = canonical J, -inf
 *     when infeasible); the best ever (J desc, index asc) is updated.  If
 *     g < gens the next population is built:
 *     slot 0 <- the elite: the best of the population (f desc, index asc,
 *       slot asc);
 *     for pair q = 0 .. pop/2-1 (children at slots 1+2q and 2+2q, the second
 *     child of the last pair is dropped):
 *       parents: two tournaments of k draws with replacement; draw m in
 *         0..2k-1 is int(R(q, g+1, s, SEL + m/4)[m%4], pop); parent A wins
 *         among draws 0..k-1, parent B among k..2k-1; the winner is the draw
 *         with the best (f desc, index asc), the earliest draw on equality;
 *       crossover: if uniform(R(q, g+1, s, CX)[0]) < p_cx, gene i is swapped
 *         between the children when uniform(R(q, g+1, s, SWAP + i/4)[i%4]) <
 *         p_swap; otherwise the children copy the parents;
 *       mutation of the child at slot j: gene i is redrawn uniformly over its
 *         K_i options, int(v, K_i), when uniform(u) < p_mut, where u and v are
 *         words 2i and 2i+1 of R(j, g+1, s, MUT + 2i/4) (words in order
 *         across consecutive purposes);
 *       repair of the child at slot j: if its VRAM sum exceeds the cap it is
 *         replaced by FL[int(R(j, g+1, s, REP)[0], |FL|)].
 *   Evaluations per scenario: (gens + 1) * pop.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#include "mf_oracle.h"

enum { P_INIT = 1, P_SEL = 2, P_CX = 8, P_SWAP = 9, P_MUT = 16, P_REP = 32 };

typedef struct {
    int32_t n_scen, pop, gens, tourn_k;
    float p_cx, p_swap, p_mut, pad;
    uint64_t seed;
} orc_ga_params;

/* -------------------------------------------------------------- Philox */

static void mulhilo64(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo)
{
    const unsigned __int128 p = (unsigned __int128)a * b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void orc_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3], k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; r++) {
        if (r) { k0 += W0; k1 += W1; }
        uint64_t h0, l0, h1, l1;
        mulhilo64(M0, x0, &h0, &l0);
        mulhilo64(M1, x2, &h1, &l1);
        const uint64_t y0 = h1 ^ x1 ^ k0, y1 = l1, y2 = h0 ^ x3 ^ k1, y3 = l0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

static uint64_t draw(uint64_t seed, uint64_t item, uint64_t gen, uint64_t scen, uint64_t purpose, int word)
{
    const uint64_t c[4] = {item, gen, scen, purpose}, k[2] = {seed, 0};
    uint64_t o[4];
    orc_philox4x64(c, k, o);
    return o[word];
}

static double uni(uint64_t r) { return (double)(r >> 11) * 0x1p-53; }
static uint64_t below(uint64_t r, uint64_t n) { return ((r >> 32) * n) >> 32; }

/* --------------------------------------------------------- GA operators */

static int better(double fa, uint64_t ia, double fb, uint64_t ib)
{
    return fa > fb || (fa == fb && ia < ib);
}

static float vram_of(const orc_instance *in, const int32_t *d)
{
    float a[ORC_MAX_AGG];
    orc_aggregate(in, d, a);
    return a[in->vram_slot];
}

/* Next population of scenario s after generation g (see the file header). */
int orc_ga_next(const orc_instance *in, const orc_ga_params *gp, int s, int g, const uint64_t *pop_idx,
                const double *fit, const uint32_t *fl, uint64_t n_fl, uint64_t *out_idx)
{
    const int P = gp->pop, N = in->n_models, kt = gp->tourn_k;
    if (P < 2 || (P & 1) || kt < 1 || kt > 8 || n_fl == 0) return -1;
    const uint64_t gen = (uint64_t)g + 1, sc = (uint64_t)s, seed = gp->seed;
    int e = 0;
    for (int j = 1; j < P; j++)
        if (better(fit[j], pop_idx[j], fit[e], pop_idx[e])) e = j;
    out_idx[0] = pop_idx[e];
    for (int q = 0; q < P / 2; q++) {
        int par[2];
        for (int t = 0; t < 2; t++) {
            int best = -1;
            for (int m = t * kt; m < (t + 1) * kt; m++) {
                const int d = (int)below(draw(seed, (uint64_t)q, gen, sc, P_SEL + m / 4, m % 4), (uint64_t)P);
                if (best < 0 || better(fit[d], pop_idx[d], fit[best], pop_idx[best])) best = d;
            }
            par[t] = best;
        }
        int32_t c[2][ORC_MAX_MODELS];
        orc_decode(in, pop_idx[par[0]], c[0]);
        orc_decode(in, pop_idx[par[1]], c[1]);
        if (uni(draw(seed, (uint64_t)q, gen, sc, P_CX, 0)) < (double)gp->p_cx) {
            for (int i = 0; i < N; i++) {
                if (uni(draw(seed, (uint64_t)q, gen, sc, P_SWAP + i / 4, i % 4)) < (double)gp->p_swap) {
                    const int32_t t = c[0][i];
                    c[0][i] = c[1][i];
                    c[1][i] = t;
                }
            }
        }
        for (int t = 0; t < 2; t++) {
            const int j = 1 + 2 * q + t;
            if (j >= P) break;
            for (int i = 0; i < N; i++) {
                const int wu = 2 * i, wv = 2 * i + 1;
                const uint64_t u = draw(seed, (uint64_t)j, gen, sc, P_MUT + wu / 4, wu % 4);
                const uint64_t v = draw(seed, (uint64_t)j, gen, sc, P_MUT + wv / 4, wv % 4);
                if (uni(u) < (double)gp->p_mut) c[t][i] = (int32_t)below(v, (uint64_t)in->n_options[i]);
            }
            if ((double)vram_of(in, c[t]) <= (double)in->vram_cap)
                out_idx[j] = orc_encode(in, c[t]);
            else
                out_idx[j] = fl[below(draw(seed, (uint64_t)j, gen, sc, P_REP, 0), n_fl)];
        }
    }
    return 0;
}

/* The whole GA.  sla, omega: [S][N].  best_idx / best_J: [S].  final_pop:
 * [S][pop] (the last evaluated population) or NULL.  Scenarios run in
 * parallel (they are independent); results do not depend on the threads. */
int orc_ga(const orc_instance *in, const orc_ga_params *gp, const float *sla, const float *omega,
           uint64_t *best_idx, double *best_J, uint64_t *final_pop, int nthreads)
{
    const int S = gp->n_scen, P = gp->pop, N = in->n_models;
    if (S < 1 || P < 2 || (P & 1) || gp->gens < 0 || gp->tourn_k < 1 || gp->tourn_k > 8) return -1;
    const uint64_t space = orc_space_size(in);
    if (space == 0 || space > 0xFFFFFFFFull) return -1;
    uint32_t *fl = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)space);
    double *w64 = orc_weights_f64(in);
    if (!fl || !w64) { free(fl); free(w64); return -1; }
    const uint64_t n_fl = orc_vram_feasible(in, fl, space);
    if (nthreads < 1) nthreads = omp_get_max_threads();
    int rc = 0;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int s = 0; s < S; s++) {
        uint64_t *cur = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)P);
        uint64_t *nxt = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)P);
        double *fit = (double *)malloc(sizeof(double) * (size_t)P);
        double *scr = (double *)malloc(sizeof(double) * orc_scratch_doubles(in));
        double bj = -INFINITY;
        uint64_t bi = UINT64_MAX;
        if (n_fl == 0) {
            for (int j = 0; j < P && final_pop; j++) final_pop[(size_t)s * P + j] = UINT64_MAX;
        } else {
            for (int j = 0; j < P; j++)
                cur[j] = fl[below(draw(gp->seed, (uint64_t)j, 0, (uint64_t)s, P_INIT, 0), n_fl)];
            for (int g = 0; g <= gp->gens; g++) {
                for (int j = 0; j < P; j++) {
                    double lat[ORC_MAX_MODELS], thr[ORC_MAX_MODELS], J;
                    uint32_t f;
                    orc_eval_w(in, w64, cur[j], sla + (size_t)s * N, omega + (size_t)s * N, lat, thr, &J, &f, scr);
                    fit[j] = J;
                    if (J > -INFINITY && better(J, cur[j], bj, bi)) { bj = J; bi = cur[j]; }
                }
                if (g == gp->gens) break;
                if (orc_ga_next(in, gp, s, g, cur, fit, fl, n_fl, nxt) != 0) { rc = -1; break; }
                uint64_t *t = cur; cur = nxt; nxt = t;
            }
            if (final_pop) memcpy(final_pop + (size_t)s * P, cur, sizeof(uint64_t) * (size_t)P);
        }
        best_idx[s] = bi;
        best_J[s] = bj;
        free(cur); free(nxt); free(fit); free(scr);
    }
    free(fl);
    free(w64);
    return rc;
}
