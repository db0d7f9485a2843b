"""Write tests/golden/tiny_oracle.json from the CPU oracle alone.

The paper prints no worked numeric example, so this fixture is a regression
record of the oracle on the seeded tiny workload (1 layer, 2 MHA heads, D=128,
T=512, fp32, w=8, budget 128): per-head statistics, a sample of scores and the
selected positions.  Any later change to the oracle's arithmetic that moves
these values must say, in its commit message, which passage of the paper
justifies it.  Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402


def main():
    oracle.build(force=False)
    wl = W.tiny()
    S, st = oracle.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w)
    idx, counts, offsets = oracle.select(S, wl.L, wl.Hkv, wl.cu_seqlens, wl.w, wl.budget)
    sample = list(range(0, S.shape[-1], 37))
    out = {
        "workload": "tiny seed 0 (1 layer, 2 MHA heads, D=128, T=512, fp32, w=8, budget 128)",
        "stat_names": ["lambda", "r_C", "r_E", "D_E", "dE_min", "dE_max", "sdiv_min", "sdiv_max",
                       "imp_mean", "sbar_mean", "mu_norm2", "scale"],
        "heads": [
            {
                "stats": st[0, h, 0].tolist(),
                "score_positions": sample,
                "scores": S[0, h, sample].tolist(),
                "selected": idx[offsets[0, h, 0]:offsets[0, h, 0] + counts[0, h, 0]].tolist(),
            }
            for h in range(wl.Hkv)
        ],
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_oracle.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
