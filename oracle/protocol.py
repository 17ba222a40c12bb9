"""CPU oracle of the scheduling protocol (Section IV-C, Table II) on synthetic
dynamic scenarios.  TEST INFRASTRUCTURE ONLY (see mf_oracle.c for who may use
the oracle).

Every decision and every recorded value comes from the oracle's canonical
evaluation: the per-step exhaustive argmax, the GA replay, the static
composition over steps.  The rules (written out here on their own):

  * scenario s, step t: observed state states[s][t] held fixed for the step's
    surrogates, bounds sla[s][t], weights omega[s][t]; utility of Eq. 3 with
    the scheduler's own previous decision as the previous deployment (the
    objective's prev_variant before step 0);
  * exhaustive: the step's argmax (ties to the lowest index); ga: the GA's
    best with key ga_seed[s][t]; random: the first candidate of
    random[s][t] within the VRAM cap (else the first candidate); a dynamic
    scheduler with no feasible configuration keeps its previous decision
    (index 0 before the first step);
  * static_full: the argmax of S = sum_t J_t over the whole space among the
    configurations feasible at every step (the configuration is its own
    previous deployment after step 0); static_budget_K: the best S among the
    first K offline samples that are feasible at every step (all samples if
    none is), ties to the lowest index;
  * recorded per step: J_t of the decision (its value also where a
    constraint fails) and whether every constraint holds;
  * gap per scenario = 100 (mean_t J_exh - mean_t J) / |mean_t J_exh|;
    Avg./Worst gap over scenarios; SLA % = share of steps with a failure.
"""
from dataclasses import replace

import numpy as np

from . import FLAG_FEAS, FLAG_SLA, FLAG_VRAM, Problem, static_eval, static_search

NO_INDEX = 2 ** 64 - 1


def _variants(inst, objective, idx):
    d = Problem(inst).decode(int(idx))
    off = np.concatenate([[0], np.cumsum(inst.n_options)[:-1]]).astype(np.int64)
    return np.array([objective.variant[off[i] + d[i]] for i in range(inst.n_models)], np.int32)


def _record(inst, ob_t, st, sla, om, idx):
    r = Problem(inst, ob_t, state=st).eval_list(np.array([idx], np.uint64), sla, om, raw=True)
    f = int(r["flags"][0])
    return float(r["J"][0]), (f & FLAG_VRAM) != 0 and (f & FLAG_SLA) != 0


def run_dynamic(inst, objective, kind, states, slas, omegas, draws, s, params):
    T = len(states)
    dec, J, ok = [], [], []
    prev = np.array(objective.prev_variant, np.int32)
    last = 0
    for t in range(T):
        ob_t = replace(objective, prev_variant=prev)
        prob = Problem(inst, ob_t, state=states[t])
        if kind == "exhaustive":
            r = prob.search(slas[t], omegas[t], k=1)
            if len(r["top_idx"]) > 0:
                last = int(r["top_idx"][0])
        elif kind == "ga":
            r = prob.ga(slas[t][None, :], omegas[t][None, :], pop=params.ga_pop, gens=params.ga_gens,
                        tourn_k=params.ga_tourn, p_cx=params.ga_p_cx, p_swap=params.ga_p_swap,
                        p_mut=params.ga_p_mut, seed=int(draws.ga_seed[s, t]))
            if int(r["best_idx"][0]) != NO_INDEX:
                last = int(r["best_idx"][0])
        else:
            cand = np.asarray(draws.random[s, t], np.uint64)
            fl = prob.eval_list(cand, slas[t], omegas[t], raw=True)["flags"]
            within = [c for c, f in zip(cand, fl) if int(f) & FLAG_VRAM]
            last = int(within[0]) if within else int(cand[0])
        j, o = _record(inst, ob_t, states[t], slas[t], omegas[t], last)
        dec.append(last)
        J.append(j)
        ok.append(o)
        prev = _variants(inst, objective, last)
    return np.array(dec, np.uint64), np.array(J), np.array(ok)


def run_static(inst, objective, kind, states, slas, omegas, draws, s):
    T = len(states)
    if kind == "static_full":
        r = static_search(inst, objective, states, slas, omegas, k=1)
        pick = int(r["top_idx"][0]) if len(r["top_idx"]) else 0
    else:
        K = int(kind.split("_")[-1])
        cand = np.asarray(draws.budget[s, :K], np.uint64)
        Jc, Fc, Sc = static_eval(inst, objective, states, slas, omegas, cand)
        every = ((Fc[:, 0] & FLAG_VRAM) != 0) & np.all((Fc & FLAG_SLA) != 0, axis=1)
        best = None
        for q in range(K):
            if every.any() and not every[q]:
                continue
            key = (-Sc[q], int(cand[q]))
            if best is None or key < best:
                best = key
        pick = best[1]
    Jp, Fp, _ = static_eval(inst, objective, states, slas, omegas, np.array([pick], np.uint64))
    ok = ((Fp[0] & FLAG_VRAM) != 0) & ((Fp[0] & FLAG_SLA) != 0)
    return np.full(T, pick, np.uint64), Jp[0], ok


def run(inst, objective, scenarios, draws, params, names):
    out = {}
    S = scenarios.states.shape[0]
    for name in names:
        rows = []
        for s in range(S):
            a = (scenarios.states[s], scenarios.sla[s], scenarios.omega[s], draws, s)
            if name.startswith("static"):
                rows.append(run_static(inst, objective, name, *a))
            else:
                rows.append(run_dynamic(inst, objective, name, *a, params))
        out[name] = dict(idx=np.stack([r[0] for r in rows]), J=np.stack([r[1] for r in rows]),
                         ok=np.stack([r[2] for r in rows]))
    return out


def table(run_results):
    """Mean J, Avg./Worst gap (%) and SLA (%) per scheduler over a list of runs."""
    res = {}
    names = list(run_results[0].keys())
    for name in names:
        J = np.concatenate([r[name]["J"] for r in run_results])
        E = np.concatenate([r["exhaustive"]["J"] for r in run_results])
        ok = np.concatenate([r[name]["ok"] for r in run_results])
        e_mean = E.mean(axis=1)
        gaps = 100.0 * (e_mean - J.mean(axis=1)) / np.abs(e_mean)
        res[name] = dict(mean_J=float(J.mean()), avg_gap=float(gaps.mean()), worst_gap=float(gaps.max()),
                         sla_pct=float(100.0 * np.count_nonzero(~ok) / ok.size))
    return res
