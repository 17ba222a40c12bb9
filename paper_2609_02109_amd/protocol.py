"""The scheduling protocol of Section IV-C (Table II) on synthetic dynamic
scenarios, driven through the C ABI.

Each scenario is a sequence of decision steps; at step t the runtime observes
an aggregate state, and the weights may raise one model's priority.  The
surrogates see the observed state (held fixed within a step, Section III-B)
and every decision is scored with the full utility of Eq. 3, whose reload
term depends on the scheduler's own previous decision.  Schedulers:

  exhaustive          per step, the argmax over the whole space (mf_search)
  ga                  per step, the GA of Section IV-C (mf_ga_run)
  random              per step, the first of the step's uniform candidates
                      that meets the VRAM cap (its floors may fail)
  static_full         one configuration for every step, the argmax of the
                      step-order sum of utilities over the whole space,
                      feasible at every step (mf_search_static)
  static_budget_K     the same choice among K offline samples
                      (mf_eval_static on the samples)

A dynamic scheduler that finds no feasible configuration keeps its previous
decision (index 0 before the first).  Each step records the decision's
utility J_t (its Eq. 3 value also when a floor fails) and whether it breaks a
constraint (the VRAM cap or a service constraint).  Metrics per scheduler:
mean J over all steps; the gap to exhaustive, 100 (mean_t J_exh - mean_t J) /
|mean_t J_exh| per scenario, averaged (Avg. Gap) and maximised (Worst Gap)
over scenarios; the share of steps that break a constraint (SLA %).

The random choices (samples, candidates, GA keys) are inputs, drawn by
`synth.protocol_draws`.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, replace

import numpy as np

from . import mf as _mf

NONE = np.uint64(2 ** 64 - 1)


@dataclass
class ProtocolParams:
    budgets: tuple = (5000, 500)
    ga_pop: int = 100            # the GA of Section IV-C: 100 candidates, 30 generations,
    ga_gens: int = 30            # crossover 0.7, mutation 0.1, tournament 3, elitism
    ga_p_cx: float = 0.7
    ga_p_swap: float = 0.5
    ga_p_mut: float = 0.1
    ga_tourn: int = 3


def scheduler_names(params: ProtocolParams):
    return (["exhaustive", "static_full", "ga"] + [f"static_budget_{k}" for k in params.budgets] + ["random"])


class Protocol:
    """Runs the schedulers of one instance over dynamic scenarios."""

    def __init__(self, inst, objective, params: ProtocolParams | None = None):
        self.inst = inst
        self.ob = objective
        self.params = params or ProtocolParams()
        self.p = _mf.Problem(inst, variants=objective)
        self.off = inst.option_offsets

    def variants_of(self, idx) -> np.ndarray:
        d = self.p.decode(int(idx))
        return self.ob.variant[self.off + d].astype(np.int32)

    def step_value(self, idx, st, sla, om, ob):
        """Utility of one decision at one step, and whether it meets every
        constraint."""
        e = self.p.eval_static(np.array([idx], np.uint64), st[None, :], sla[None, :], om[None, :], objective=ob)
        return float(e["J"][0, 0]), bool((e["flags"][0, 0] & 3) == 3)

    def dynamic(self, kind, st, sla, om, draws, s):
        P = self.params
        T = len(st)
        J = np.zeros(T)
        ok = np.zeros(T, bool)
        idx = np.zeros(T, np.uint64)
        ms = np.zeros(T)
        prev = self.ob.prev_variant.astype(np.int32)
        cur = np.uint64(0)
        for t in range(T):
            ob_t = replace(self.ob, prev_variant=prev)
            t0 = time.perf_counter()
            if kind == "exhaustive":
                r = self.p.search(sla[t], om[t], k=1, objective=ob_t, state=st[t])
                if len(r["top_idx"]):
                    cur = r["top_idx"][0]
            elif kind == "ga":
                r = self.p.ga(sla[t][None, :], om[t][None, :], pop=P.ga_pop, gens=P.ga_gens, tourn_k=P.ga_tourn,
                              p_cx=P.ga_p_cx, p_swap=P.ga_p_swap, p_mut=P.ga_p_mut, seed=int(draws.ga_seed[s, t]),
                              objective=ob_t, state=st[t])
                if r["best_idx"][0] != NONE:
                    cur = r["best_idx"][0]
            else:
                cand = draws.random[s, t]
                e = self.p.eval_static(cand, st[t][None, :], sla[t][None, :], om[t][None, :], objective=ob_t)
                fits = np.flatnonzero(e["flags"][:, 0] & 1)
                cur = cand[fits[0]] if len(fits) else cand[0]
            ms[t] = (time.perf_counter() - t0) * 1e3   # the decision's wall time (blocking calls)
            idx[t] = cur
            J[t], ok[t] = self.step_value(cur, st[t], sla[t], om[t], ob_t)
            prev = self.variants_of(cur)
        return idx, J, ok, ms

    def static(self, kind, st, sla, om, draws, s):
        T = len(st)
        t0 = time.perf_counter()
        if kind == "static_full":
            r = self.p.search_static(st, sla, om, k=1, objective=self.ob)
            cur = r["top_idx"][0] if len(r["top_idx"]) else np.uint64(0)
        else:
            K = int(kind.rsplit("_", 1)[1])
            cand = draws.budget[s, :K]
            e = self.p.eval_static(cand, st, sla, om, objective=self.ob)
            good = ((e["flags"][:, 0] & 1) != 0) & np.all((e["flags"] & 2) != 0, axis=1)
            pool = np.flatnonzero(good) if good.any() else np.arange(len(cand))
            order = np.lexsort((cand[pool], -e["S"][pool]))
            cur = cand[pool[order[0]]]
        ms = np.full(T, (time.perf_counter() - t0) * 1e3 / T)
        e = self.p.eval_static(np.array([cur], np.uint64), st, sla, om, objective=self.ob)
        return np.full(T, cur, np.uint64), e["J"][0].copy(), (e["flags"][0] & 3) == 3, ms

    def run(self, scenarios, draws):
        """Every scheduler on every scenario: per scheduler, decisions [S][T],
        utilities [S][T], constraint flags [S][T] and decision wall times
        [S][T] in ms (a static choice's time spread over its steps)."""
        out = {}
        S, T = scenarios.states.shape[:2]
        for name in scheduler_names(self.params):
            idx = np.zeros((S, T), np.uint64)
            J = np.zeros((S, T))
            ok = np.zeros((S, T), bool)
            ms = np.zeros((S, T))
            for s in range(S):
                args = (scenarios.states[s], scenarios.sla[s], scenarios.omega[s], draws, s)
                f = self.static if name.startswith("static") else self.dynamic
                idx[s], J[s], ok[s], ms[s] = f(name, *args)
            out[name] = dict(idx=idx, J=J, ok=ok, ms=ms)
        return out


def metrics(runs):
    """Table II's columns from one or more run() results (seeds): mean J,
    Avg./Worst gap (%) to exhaustive per scenario, SLA violations (%)."""
    if isinstance(runs, dict):
        runs = [runs]
    table = {}
    for name in runs[0]:
        Js = np.concatenate([r[name]["J"] for r in runs])
        ex = np.concatenate([r["exhaustive"]["J"] for r in runs]).mean(axis=1)
        ok = np.concatenate([r[name]["ok"] for r in runs])
        gap = 100.0 * (ex - Js.mean(axis=1)) / np.abs(ex)
        table[name] = dict(mean_J=float(Js.mean()), avg_gap=float(gap.mean()), worst_gap=float(gap.max()),
                           sla_pct=float(100.0 * (1.0 - ok.mean())))
    return table
