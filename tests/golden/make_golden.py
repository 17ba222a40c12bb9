"""Write stored expected results for the parity tests.

Calls only the CPU oracle (oracle/) on instances from the seeded generator.
Each record carries a fingerprint of the instance arrays so that a test can
tell a stale file from a changed generator.

    python tests/golden/make_golden.py [--only NAME ...] [--threads T]

Floating-point values are stored as float.hex() strings (exact).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2609_02109_amd import synth  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def fingerprint(inst) -> str:
    h = hashlib.sha256()
    for a in (inst.n_options, inst.features, inst.agg_cols, inst.weights, inst.sla, inst.omega):
        h.update(np.ascontiguousarray(a).tobytes())
    h.update(np.float32(inst.vram_cap).tobytes())
    return h.hexdigest()[:16]


def search_record(name, inst, k, threads):
    p = oracle.Problem(inst)
    t0 = time.time()
    r = p.search(inst.sla, inst.omega, k=k, threads=threads)
    dt = time.time() - t0
    return dict(name=name, seed=inst.seed, fingerprint=fingerprint(inst), k=k,
                space_size=p.space_size, n_eval=r["n_eval"], n_vram=r["n_vram"],
                n_feas=r["n_feas"], n_near=r["n_near"],
                top_idx=[int(x) for x in r["top_idx"]],
                top_J=[float(x).hex() for x in r["top_J"]],
                oracle_seconds=round(dt, 3), oracle_threads=threads)


def chunk_starts(space, size, count, seed):
    """Chunk starts over [0, space): the head, one chunk across the midpoint
    of the space, the tail, and seeded uniform starts (not tile aligned)."""
    rng = np.random.default_rng(seed)
    starts = [0, space // 2 - size // 2, space - size]
    starts += [int(x) for x in rng.integers(0, space - size + 1, size=count - len(starts), dtype=np.uint64)]
    return sorted(starts)


def chunks_record(name, inst, k, threads, size, count, seed):
    """Full oracle results on `count` chunks of `size` consecutive joint
    configurations each: counts, the top-k, and a SHA-256 over the chunk's
    flag bytes (bit0 VRAM ok, bit1 every bound met, bit2 feasible)."""
    p = oracle.Problem(inst)
    space = p.space_size
    recs, t0 = [], time.time()
    for lo in chunk_starts(space, size, count, seed):
        r = p.search(inst.sla, inst.omega, k=k, lo=lo, hi=lo + size, threads=threads, dump=True)
        flags = (r["flags"] & 7).astype(np.uint8)
        recs.append(dict(lo=lo, hi=lo + size, n_vram=r["n_vram"], n_feas=r["n_feas"],
                         top_idx=[int(x) for x in r["top_idx"]], top_J=[float(x).hex() for x in r["top_J"]],
                         flags_sha256=hashlib.sha256(flags.tobytes()).hexdigest()))
        print(f"  {name} [{lo}, {lo + size}) n_feas={r['n_feas']} ({time.time() - t0:.0f}s)", flush=True)
    return dict(name=name, seed=inst.seed, fingerprint=fingerprint(inst), k=k, space_size=space,
                chunk_size=size, chunk_seed=seed, chunks=recs, oracle_seconds=round(time.time() - t0, 1),
                oracle_threads=threads)


CASES = {
    **{f"cfg0_s{s}": (lambda s=s: synth.cfg0(s), 1) for s in (0, 1, 2)},
    **{f"cfg1_s{s}": (lambda s=s: synth.cfg1(s), 16) for s in (0, 1, 2)},
    "cfg2_s0": (lambda: synth.cfg2(0), 16),
}

# the N=8 bf16 workload: too large for a full oracle run (about 5e15 fp64
# flops), so 64 chunks of 2^18 consecutive configurations are compared in full
CHUNK_CASES = {
    "cfg4_s0_chunks": (lambda: synth.cfg4(0), 64, 1 << 18, 64, 20261202),
}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", nargs="*")
    ap.add_argument("--threads", type=int, default=0)
    args = ap.parse_args()
    if not os.path.exists(oracle.LIB):
        oracle.build()
    for name, (make, k) in CASES.items():
        if args.only and name not in args.only:
            continue
        rec = search_record(name, make(), k, args.threads)
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(rec, f, indent=1)
        print(name, rec["n_vram"], rec["n_feas"], rec["top_idx"][:3], f"{rec['oracle_seconds']}s",
              flush=True)
    for name, (make, k, size, count, seed) in CHUNK_CASES.items():
        if args.only and name not in args.only:
            continue
        rec = chunks_record(name, make(), k, args.threads, size, count, seed)
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(rec, f, indent=1)
        print(name, len(rec["chunks"]), f"{rec['oracle_seconds']}s", flush=True)


if __name__ == "__main__":
    main()
