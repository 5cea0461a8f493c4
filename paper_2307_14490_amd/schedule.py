"""Learning-rate schedules for the training step (host side: the step takes
its learning rate per call).

LWSGD (Table 2): SGD with a linear warm-up and a linear decay of the learning
rate, given by four numbers -- warm-up steps, the value reached at the end of
the warm-up, decay steps, and the value reached at the end of the decay,
which is then held.  The paper does not say where the warm-up starts or how
steps are counted; here steps count from 0, the warm-up rises linearly from 0
so that step warmup - 1 uses `peak`, and the decay falls linearly so that
step warmup + decay - 1 uses `final`.
"""
from __future__ import annotations

# Table 2: (5K, 0.01, 100K, 0.001) for the TPU runs.
PAPER_LWSGD = (5_000, 0.01, 100_000, 0.001)


def lwsgd(step: int, warmup: int = PAPER_LWSGD[0], peak: float = PAPER_LWSGD[1],
          decay: int = PAPER_LWSGD[2], final: float = PAPER_LWSGD[3]) -> float:
    """Learning rate of step `step` (0-based) under LWSGD."""
    if step < 0:
        raise ValueError("step must be >= 0")
    if warmup < 0 or decay < 0:
        raise ValueError("warmup and decay must be >= 0")
    if step < warmup:
        return peak * (step + 1) / warmup
    done = step - warmup + 1  # decay steps taken, counting this one
    if done < decay:
        return peak + (final - peak) * done / decay
    return final
