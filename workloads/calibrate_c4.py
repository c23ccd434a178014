"""Pick the C4 logit correlation c so greedy verification emits 3.80 tokens/step.

The paper's greedy EAGLE+FP8 configuration reaches a mean generated length
(MGL, tokens emitted per verify step) of 3.80 (Table 1).  This script bisects
the correlation c of the synthetic C4 logits (workloads.gen.accept_logits)
until the CPU oracle's greedy verification emits a mean of 3.80 tokens per
step (a_b + 1 averaged over the batch) and prints the value to store as
workloads.configs.C4_CORRELATION.  It calls only the oracle.

    python -m workloads.calibrate_c4
"""

from __future__ import annotations

import sys

import numpy as np

from workloads import gen
from workloads.configs import CONFIGS

TARGET_MGL = 3.80


def greedy_mgl(c: float) -> float:
    from oracle import accept as oa      # the oracle is the only judge of acceptance
    cfg = CONFIGS["C4"]
    zt, zd = gen.accept_logits(cfg["B"], cfg["k"], cfg["V"], cfg["seed"], c,
                               scale=cfg["logit_std"], rank=cfg["rank"])
    x = gen.draft_tokens_greedy(zd)
    _, num = oa.accept_greedy(zt, x)
    return float(np.mean(num + 1))


def main() -> int:
    lo, hi = 0.0, 1.0
    for _ in range(14):
        mid = 0.5 * (lo + hi)
        m = greedy_mgl(mid)
        print(f"c={mid:.6f} MGL={m:.4f}", flush=True)
        if m < TARGET_MGL:
            lo = mid
        else:
            hi = mid
    c = round(0.5 * (lo + hi), 4)
    print(f"C4_CORRELATION = {c}  (greedy MGL {greedy_mgl(c):.4f})")
    return 0


if __name__ == "__main__":
    sys.exit(main())
