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


CASES = {
    **{f"cfg0_s{s}": (lambda s=s: synth.cfg0(s), 1) for s in (0, 1, 2)},
    **{f"cfg1_s{s}": (lambda s=s: synth.cfg1(s), 16) for s in (0, 1, 2)},
    "cfg2_s0": (lambda: synth.cfg2(0), 16),
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


if __name__ == "__main__":
    main()
