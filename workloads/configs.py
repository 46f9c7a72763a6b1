"""The five synthetic workloads of the partial-straggler gradient-coding hot path.

Each workload fixes the cyclic assignment (N = m chunks and workers, s
stragglers, load delta = s + 1), the gradient length d, how the chunk
gradients arise (a regression problem over n samples per chunk, or i.i.d.
N(0, 1) chunk gradients given directly), the straggler-pattern model and the
communication factors ell that are exercised.  The straggler models follow the
simulation model of the paper's numerical section (random failed workers,
i.i.d. exponential per-chunk times, N(0, 1) entries of R) at the sizes below.

This module holds sizes and distribution parameters only; it computes nothing
of the gradient-coding method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    N: int                      # chunks
    m: int                      # workers
    s: int                      # stragglers tolerated by the cyclic code
    d: int                      # gradient length
    P: int                      # straggler patterns
    ells: Tuple[int, ...]       # communication factors exercised
    n: Optional[int] = None     # samples per chunk (None: chunk gradients given)
    loss: Optional[str] = None  # "linear" | "logistic" | None
    x_std: float = 1.0          # std of the entries of X
    w_std: float = 0.0          # std of the entries of the evaluation point w
    noise_std: float = 0.1      # label noise (linear model)
    g_dtype: str = "f32"        # storage type of given chunk gradients
    pattern: str = "uniform"    # straggler model, see workloads.gen.psi
    forced_zero: int = 0        # workers forced to psi = 0 per pattern
    ls_forced_zero: int = 0     # extra forced zeros of the least-squares run
    ls_ells: Tuple[int, ...] = field(default_factory=tuple)
    assignment: str = "cyclic"  # "cyclic" | "regular_graph" (random nu-regular graph, nu = s + 1)
    deadline: float = 0.0       # fixed deadline of the "fail_exp_deadline" pattern model

    @property
    def delta(self) -> int:
        return self.s + 1

    @property
    def gamma(self) -> int:
        return self.s + 1


# Tiny exact GC: linear regression at w = 0, psi_j uniform on {0..3}.
TINY = Workload(name="tiny_m6_d64", N=6, m=6, s=2, d=64, P=100, ells=(1, 2, 3),
                n=32, loss="linear", x_std=1.0, w_std=0.0, pattern="uniform")

# m = 20, linear regression, Exp(1) chunk times, deadline = median completion.
SMALL = Workload(name="linreg_m20_d4096", N=20, m=20, s=3, d=4096, P=1000,
                 ells=(1, 2), n=256, loss="linear", x_std=1.0, w_std=0.1,
                 pattern="exp_median")

# Headline: m = 50 logistic regression, 20% full stragglers, the rest uniform
# partial progress.
HEADLINE = Workload(name="logreg_m50_d16384", N=50, m=50, s=4, d=16384,
                    P=10000, ells=(1, 2), n=512, loss="logistic",
                    x_std=16384 ** -0.5, w_std=0.1,
                    pattern="uniform", forced_zero=10)

# Bandwidth-bound: given N(0,1) fp32 chunk gradients, shifted-exponential chunk
# times, fixed deadline.
BANDWIDTH = Workload(name="given_m100_d1M", N=100, m=100, s=9, d=1 << 20,
                     P=10000, ells=(1, 2, 8), g_dtype="f32",
                     pattern="shifted_exp_fixed")

# Large: given bf16 chunk gradients, heterogeneous worker speeds; exact run
# plus a least-squares run with 50% forced stragglers.
LARGE = Workload(name="given_m200_d16M_bf16", N=200, m=200, s=19, d=1 << 24,
                 P=100000, ells=(1, 2), g_dtype="bf16", pattern="hetero_median",
                 ls_forced_zero=100, ls_ells=(1, 2, 4))

# Regular-graph assignment of the paper's approximate-GC experiments: a random
# 8-regular graph on m = 200 vertices as the support, ordered by Algorithm 2;
# nu - 1 = 7 failed workers, Exp(1) chunk times, deadline T.
GRAPH = Workload(name="graph_m200_nu8", N=200, m=200, s=7, d=4096, P=2000, ells=(1, 2, 3),
                 g_dtype="f32", pattern="fail_exp_deadline", forced_zero=7,
                 assignment="regular_graph", deadline=6.0)

ALL = (TINY, SMALL, HEADLINE, BANDWIDTH, LARGE)
EXTRA = (GRAPH,)
BY_NAME = {w.name: w for w in ALL + EXTRA}
