"""Workload definitions: the five seeded synthetic MAP-Elites configurations.

This module holds sizes, hyper-parameters and seeds only -- none of the
method's arithmetic.  Both the HIP library binding and the CPU oracle's test
wrapper build their own config structs from these plain dicts.

Shapes follow the paper where it gives them: genotype dimension 100 for
Rastrigin/Sphere and their (theta_0, theta_1) descriptor (Appendix B.2), a
100x100 grid (Section 5.1), Iso+LineDD sigmas, two hidden tanh layers of 64
(Section 5.1), 8 actions and a 4-D descriptor in [0,1]^4 as for the
uni-directional Ant (Appendix B.2, task table).  The rest (projection
descriptor, CVT sizes, synthetic dynamics, episode lengths) is synthetic and
stands in for workloads the paper ran on a physics simulator.
"""
from __future__ import annotations

import copy

RASTRIGIN, SPHERE, RASTRIGIN_PROJ, MLP_SYNTH = 0, 1, 2, 3
GRID, CVT = 0, 1

_BASE = dict(
    task=RASTRIGIN, tess=GRID, n=100, batch=128, D=2, grid=(100, 100), C=10000,
    lo=(-5.12, -5.12), hi=(5.12, 5.12), iso_sigma=0.005, line_sigma=0.05,
    init_lo=-0.1, init_hi=0.1, obs=27, hid=64, act=8, T=250, seed=0, generations=100,
    cvt_samples=0, cvt_iters=0, death_mode=0, death_below=0.0, init_mode=0,
)

WORKLOADS = {
    # Rastrigin n=100, 100x100 grid, N_B=128, 100 generations.
    "rastrigin_grid_b128": dict(_BASE),
    # Sphere n=100, 100x100 grid, N_B=16384, 500 generations.
    "sphere_grid_b16384": dict(_BASE, task=SPHERE, batch=16384, generations=500),
    # Rastrigin n=1000 with the two-half projection descriptor, CVT of 10^4
    # centroids uniform in [0,1]^2, N_B=65536, 200 generations.
    "rastrigin_proj_cvt_b65536": dict(
        _BASE, task=RASTRIGIN_PROJ, tess=CVT, n=1000, batch=65536, grid=(0, 0),
        C=10000, generations=200),
    # The same shape with a spread first batch: each individual adds one
    # level per genotype half, uniform over the descriptor box, so the first
    # batch fills nearly all 10^4 cells and parents are distinct rows.
    "rastrigin_proj_cvt_b65536_spread": dict(
        _BASE, task=RASTRIGIN_PROJ, tess=CVT, n=1000, batch=65536, grid=(0, 0),
        C=10000, generations=200, init_mode=1),
    # Policy 27->64->64->8, T=250, CVT 1024 in [0,1]^4, N_B=8192, 100 generations.
    "mlp64_cvt_b8192": dict(
        _BASE, task=MLP_SYNTH, tess=CVT, n=0, batch=8192, D=4, grid=(0, 0, 0, 0), C=1024,
        lo=(0.0, 0.0, 0.0, 0.0), hi=(1.0, 1.0, 1.0, 1.0), hid=64, T=250, generations=100),
    # Policy 27->128->128->8, T=1000, CVT 10^4 in [0,1]^4, N_B=65536, 50 generations.
    "mlp128_cvt_b65536": dict(
        _BASE, task=MLP_SYNTH, tess=CVT, n=0, batch=65536, D=4, grid=(0, 0, 0, 0), C=10000,
        lo=(0.0, 0.0, 0.0, 0.0), hi=(1.0, 1.0, 1.0, 1.0), hid=128, T=1000, generations=50),
}

# Order of the configurations as listed for the benchmark.
ORDER = ["rastrigin_grid_b128", "sphere_grid_b16384", "rastrigin_proj_cvt_b65536",
         "mlp64_cvt_b8192", "mlp128_cvt_b65536"]


def workload(name: str, **overrides) -> dict:
    """A copy of a named workload with some fields replaced (e.g. a smaller batch)."""
    w = copy.deepcopy(WORKLOADS[name])
    w.update(overrides)
    return w


def genotype_len(w: dict) -> int:
    if w["task"] == MLP_SYNTH:
        o, h, a = w["obs"], w["hid"], w["act"]
        return h * o + h + h * h + h + a * h + a
    return int(w["n"])
