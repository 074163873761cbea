"""Find the logit scale beta of the skewed-routing workload (id 3).

The router logits of that workload get a per-expert bias beta*log(p_e), with
p_e proportional to rank_e**-1.2 and the non-resident experts ranked first.
beta is chosen by bisection so that 70% of the top-1 routes (seed 42) land on
non-resident experts.  Calls only the CPU oracle; prints the value stored as
ZIPF_BETA_W3 in paper_2606_19025_amd/inputs.py.
"""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

from oracle import moe_oracle as O  # noqa: E402
from paper_2606_19025_amd import inputs as I  # noqa: E402


def top1_ghost_fraction(beta):
    inp = I.make_layer_inputs(3, zipf_beta=beta, with_experts=False)
    r = O.route(inp["x"], inp["w_router"], 2, inp["resident"], bias=inp["router_bias"])
    return float((r["local"][:, 0] < 0).mean())


def main(target=0.70):
    lo, hi = 0.0, 4.0
    for _ in range(14):  # beta on a 2**-12 grid
        mid = (lo + hi) / 2
        if top1_ghost_fraction(mid) < target:
            lo = mid
        else:
            hi = mid
    beta = hi
    print(f"beta={beta!r} top1_ghost_fraction={top1_ghost_fraction(beta):.4f}")


if __name__ == "__main__":
    main()
