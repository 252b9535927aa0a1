"""Controller and pruning parameters of one run (values only).

The paper names these symbols but gives no values: the gain and target of
the temperature law (Section 3.3), the clip bounds T_min/T_max, the
estimator error bound epsilon_H (Section 3.3), and the guards H_min and
B_min (Section 3.3, "Conservative pruning under uncertainty bounds";
Section 5, "Robust control with uncertainty floors").  The defaults below are
readings of those passages, chosen here.  Both the HIP library configuration and the oracle
are driven from one `Params` object in tests and benchmarks.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np

from .workloads import Workload


@dataclass(frozen=True)
class Params:
    scale: float          # softmax scale of scoring and attention, 1/sqrt(d)
    eta: float            # signed gain of the temperature law (negative = stabilising)
    h_target: float       # H*
    t_min: float
    t_max: float
    eps_h: float          # bound on the entropy estimator error
    h_min: float          # entropy floor used for pruning decisions
    kappa_min: float      # smallest kept fraction of blocks
    b_min: int            # smallest number of kept blocks
    log_v: float          # log |V| rounded to float32
    t0: float = 1.0       # initial temperature
    estimator: int = 0    # entropy the controller acts on: 0 exact, 1 top-k, 2 tail-corrected
    est_k: int = 256      # k of the top-k and tail-corrected estimators
    t_cal: float = 1.0    # calibration temperature wrapping the logits (1 = none)
    rho_t: float = math.inf   # bound on |ln T_{t+1} - ln T_t| before clipping (inf = none)
    dkappa: float = 1.0   # largest decrease of the kept fraction per step (1 = none)
    h_bias: float = 0.0   # offset added to the entropy the controller acts on (stress tests)
    scoring: int = 0      # block scores: 0 mean-key reading, 1 exact token-level weights
    keep_first: int = 0   # leading blocks always kept
    keep_last: int = 0    # trailing blocks always kept

    def __post_init__(self):
        # Every float is held at float32 precision: the library receives
        # float32 values, and the oracle must see the same numbers.
        for f in dataclasses.fields(self):
            v = getattr(self, f.name)
            if isinstance(v, float):
                object.__setattr__(self, f.name, float(np.float32(v)))

    def replace(self, **kw) -> "Params":
        return dataclasses.replace(self, **kw)


def default_params(w: Workload) -> Params:
    return Params(
        scale=float(np.float32(1.0 / math.sqrt(w.head_dim))),
        eta=-0.05,
        h_target=float(np.float32(w.h_target)),
        t_min=0.05,
        t_max=5.0,
        eps_h=0.0,
        h_min=float(np.float32(w.h_target)),
        kappa_min=0.05,
        b_min=4,
        log_v=float(np.float32(math.log(w.vocab))),
    )
