"""Retention policies on the synthetic decode streams -- TEST INFRASTRUCTURE.

Prints, per budget and policy, the output deviation from dense attention and
the recall of the planted milestone tokens (oracle.baselines.evaluate), as
one JSON line each. It calls only oracle/ and the input generator.

    python3 -m oracle.compare_policies [--steps 2048] [--units 2]
"""
from __future__ import annotations

import argparse
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import synth  # noqa: E402
from oracle import baselines as bl  # noqa: E402


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="llama8b-b1-L1024")
    ap.add_argument("--steps", type=int, default=2048)
    ap.add_argument("--units", type=int, default=2, help="KV heads of sequence 0 evaluated")
    ap.add_argument("--budgets", default="256,512,1024")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args()
    w = synth.get_workload(args.workload)
    ps = w.page_size
    for L in (int(x) for x in args.budgets.split(",")):
        pols = {
            "sink": lambda K, V, L=L: bl.Sink(K, V, L),
            "h2o": lambda K, V, L=L: bl.H2O(K, V, L),
            "quest": lambda K, V, L=L: bl.Quest(K, V, L, ps),
            "raas-token": lambda K, V, L=L: bl.TokenRaaS(K, V, L, r=w.r),
            "raas-page": lambda K, V, L=L: bl.PageRaaS(K, V, L, ps, r=w.r),
        }
        acc = {}
        for kvh in range(args.units):
            res = bl.evaluate(w, args.seed, 0, kvh, args.steps, pols)
            for name, m in res.items():
                a = acc.setdefault(name, {k: 0.0 for k in m})
                for k, val in m.items():
                    a[k] = max(a[k], val) if k == "max_attended" else a[k] + val / args.units
        for name, m in acc.items():
            print(json.dumps({"workload": w.name, "prefill_len": w.prefill_len, "steps": args.steps,
                              "units": args.units, "budget": L, "policy": name,
                              **{k: round(v, 5) for k, v in m.items()}}), flush=True)


if __name__ == "__main__":
    main()
