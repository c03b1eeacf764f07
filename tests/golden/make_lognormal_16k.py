"""Write lognormal_16k_solutions.txt: the oracle's budget solves of the
gradient-like workload (d = 16384 fp32, exp(Normal(0,1)) with random signs,
seed 0; s = 32; budgets 1.5, 2.5, 3.5 bits per entry), with the library's
default search (one multiplier per pass, aimed queries) and codebook recovery
by the argmin traceback, without refinement (R = 0) and with five rounds
(R = 5).  Calls only oracle/ (and the seeded input generator).  About ten
minutes on eight cores:

    python tests/golden/make_lognormal_16k.py
"""
import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import pipeline  # noqa: E402
from paper_2608_18147_amd import inputs  # noqa: E402

S = 32
BUDGETS = (1.5, 2.5, 3.5)
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lognormal_16k_solutions.txt")


def hx(v):
    return float(v).hex()


def main():
    x = inputs.make("lognormal_16k", 0)
    H = pipeline.prepare(x)
    lines = ["# oracle budget solves of lognormal_16k (seed 0), s = 32; written by",
             "# make_lognormal_16k.py; floats as C99 hex; traj rows: lambda H(I,B) vNMSE t",
             f"p = {H.p}"]
    for b in BUDGETS:
        sr = pipeline.search(H, S, b, width=1)
        chain, _ = pipeline._recover(H, sr["t"], sr["lam"], "backpointers", S)
        lam = sr["lam_final"]
        tag = f"b{b}"
        lines.append(f"{tag}.solves = {sr['solves']}")
        lines.append(f"{tag}.passes = {sr['passes']}")
        lines.append(f"{tag}.status = {sr['status']}")
        lines.append(f"{tag}.lambda_B = {hx(sr['lam'])}")
        lines.append(f"{tag}.lambda = {hx(lam)}")
        lines.append(f"{tag}.traj = " + " ".join(hx(v) for v in sr["traj"].ravel()))
        for R in (0, 5):
            ch = chain
            rounds = 0
            if R > 0 and math.isfinite(lam) and len(chain) >= 3:
                ch, rounds, _ = pipeline.refine(H, chain, lam * H.s2tot, b, True, R)
            m = pipeline.chain_metrics(H, ch, lam)
            k = f"{tag}.R{R}"
            lines.append(f"{k}.rank = " + " ".join(str(int(a)) for a in ch))
            lines.append(f"{k}.rounds = {rounds}")
            for name in ("mse", "vnmse", "entropy", "entropy_surrogate", "objective",
                         "rate_total"):
                lines.append(f"{k}.{name} = {hx(m[name])}")
        print(tag, "solves", sr["solves"], "t", len(chain), flush=True)
    with open(OUT, "w") as fh:
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
