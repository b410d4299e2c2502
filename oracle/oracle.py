"""ctypes wrapper of the CPU oracle (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
import this module.  It takes plain workload dicts and never imports the HIP
library's package.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

MAP_RSINPI, MAP_EXP, MAP_TANH, MAP_SIGMOID = 1, 2, 3, 4


class OrConfig(C.Structure):
    _fields_ = [
        ("task", C.c_int32), ("tess", C.c_int32), ("n", C.c_int32), ("batch", C.c_int32),
        ("D", C.c_int32), ("grid", C.c_int32 * 4), ("C", C.c_int32),
        ("lo", C.c_float * 4), ("hi", C.c_float * 4),
        ("iso_sigma", C.c_float), ("line_sigma", C.c_float),
        ("init_lo", C.c_float), ("init_hi", C.c_float),
        ("obs", C.c_int32), ("hid", C.c_int32), ("act", C.c_int32), ("T", C.c_int32),
        ("cvt_samples", C.c_int32), ("cvt_iters", C.c_int32),
        ("death_mode", C.c_int32), ("death_below", C.c_float), ("init_mode", C.c_int32),
        ("seed", C.c_uint64),
    ]


_lib = None


def lib(path: str | None = None):
    """The oracle library (built on first use).  With `path`, a separately
    built copy of it (e.g. the single-threaded build), loaded afresh."""
    global _lib
    if path is not None or _lib is None:
        if path is None and not os.path.exists(LIB_PATH):
            from oracle import build as _b
            _b.build()
        L = C.CDLL(path or LIB_PATH)
        P = C.c_void_p
        f32p, u32p, i32p, u8p = (C.POINTER(C.c_float), C.POINTER(C.c_uint32),
                                 C.POINTER(C.c_int32), C.POINTER(C.c_uint8))
        sig = {
            "or_philox": (None, [u32p, u32p, u32p]),
            "or_u24": (C.c_float, [C.c_uint32]),
            "or_u24p": (C.c_float, [C.c_uint32]),
            "or_normal": (C.c_float, [C.c_uint32]),
            "or_normal_quantile": (C.c_double, [C.c_double]),
            "or_normal_table": (None, [f32p]),
            "or_rsinpi": (C.c_float, [C.c_float]),
            "or_rsin_coef": (None, [C.POINTER(C.c_float)]),
            "or_expf": (C.c_float, [C.c_float]),
            "or_tanhf": (C.c_float, [C.c_float]),
            "or_sigmoidf": (C.c_float, [C.c_float]),
            "or_r64_sum": (C.c_float, [f32p, C.c_int32, C.c_int32]),
            "or_eval_testfn": (None, [C.c_int32, f32p, C.c_int32, f32p, f32p, f32p, f32p]),
            "or_grid_cell": (C.c_int32, [f32p, C.c_int32, i32p, f32p, f32p]),
            "or_cvt_cell": (C.c_int32, [f32p, C.c_int32, f32p, f32p, f32p, C.c_int32]),
            "or_mlp_rollout": (None, [f32p, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                      f32p, f32p, f32p, C.c_int32, C.c_float, f32p, f32p]),
            "or_key": (C.c_uint64, [C.c_float, C.c_int32, C.c_int32]),
            "or_map_f32": (None, [C.c_int32, f32p, f32p, C.c_int64]),
            "or_philox_many": (None, [u32p, u32p, u32p, C.c_int64]),
            "or_normal_many": (None, [u32p, f32p, C.c_int64]),
            "or_genotype_len": (C.c_int32, [C.POINTER(OrConfig)]),
            "or_env_len": (C.c_int32, [C.POINTER(OrConfig)]),
            "or_new": (P, [C.POINTER(OrConfig), C.c_int32]),
            "or_free": (None, [P]),
            "or_setup": (None, [P]),
            "or_init": (C.c_int32, [P]),
            "or_generation": (C.c_int32, [P, C.c_uint32]),
            "or_offspring": (C.c_int32, [P, C.c_uint32, C.c_int32, f32p, f32p, f32p, i32p]),
            "or_offspring_many": (C.c_int32, [P, C.c_uint32, i32p, C.c_int32, f32p, f32p,
                                              i32p]),
            "or_set_threads": (C.c_int32, [C.c_int32]),
            "or_insert_driven": (C.c_int32, [P, f32p, f32p, f32p, C.c_int32, i32p, u8p]),
            "or_stats": (None, [P, C.c_double, C.POINTER(C.c_double)]),
            "or_archive_geno": (f32p, [P]), "or_archive_fit": (f32p, [P]),
            "or_archive_desc": (f32p, [P]), "or_archive_occ": (u8p, [P]),
            "or_centroids": (f32p, [P]), "or_env": (f32p, [P]),
            "or_off_parents": (i32p, [P]), "or_off_fit": (f32p, [P]),
            "or_off_desc": (f32p, [P]), "or_off_cell": (i32p, [P]),
            "or_off_won": (u8p, [P]), "or_off_geno": (f32p, [P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        if path is not None:
            return L
        _lib = L
    return _lib


def set_threads(n: int = 0) -> int:
    """Threads of the oracle's per-offspring loops (0: keep); returns the count."""
    return int(lib().or_set_threads(n))


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def make_config(w: dict) -> OrConfig:
    c = OrConfig()
    c.task, c.tess, c.n, c.batch, c.D = w["task"], w["tess"], w["n"], w["batch"], w["D"]
    for k in range(4):
        c.grid[k] = w["grid"][k] if k < len(w["grid"]) else 0
        c.lo[k] = w["lo"][k] if k < len(w["lo"]) else 0.0
        c.hi[k] = w["hi"][k] if k < len(w["hi"]) else 1.0
    c.C = w["C"]
    c.iso_sigma, c.line_sigma = w["iso_sigma"], w["line_sigma"]
    c.init_lo, c.init_hi = w["init_lo"], w["init_hi"]
    c.obs, c.hid, c.act, c.T = w["obs"], w["hid"], w["act"], w["T"]
    c.cvt_samples, c.cvt_iters = w.get("cvt_samples", 0), w.get("cvt_iters", 0)
    c.death_mode, c.death_below = w.get("death_mode", 0), w.get("death_below", 0.0)
    c.init_mode = w.get("init_mode", 0)
    c.seed = w["seed"]
    return c


# ---------------------------------------------------------------- primitives
def philox(ctr, key) -> np.ndarray:
    ctr = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32).reshape(-1, 4))
    key = np.ascontiguousarray(np.asarray(key, dtype=np.uint32).reshape(2))
    out = np.zeros_like(ctr)
    lib().or_philox_many(_ptr(ctr, C.c_uint32), _ptr(key, C.c_uint32), _ptr(out, C.c_uint32),
                         ctr.shape[0])
    return out


def normal(x) -> np.ndarray:
    """One standard normal per Philox word (the inverse-CDF sampler)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.uint32).ravel())
    out = np.zeros(x.size, dtype=np.float32)
    lib().or_normal_many(_ptr(x, C.c_uint32), _ptr(out, C.c_float), x.size)
    return out


def normal_quantile(p: float) -> float:
    """Phi^-1(1 - p/2) in fp64, the sampler's table source."""
    return float(lib().or_normal_quantile(float(p)))


NORMAL_ROWS = 385


def normal_table() -> np.ndarray:
    out = np.zeros((NORMAL_ROWS, 4), dtype=np.float32)
    lib().or_normal_table(_ptr(out, C.c_float))
    return out


def map_f32(fn: int, x) -> np.ndarray:
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32).ravel())
    out = np.zeros_like(x)
    lib().or_map_f32(fn, _ptr(x, C.c_float), _ptr(out, C.c_float), x.size)
    return out


def rsin_coef() -> np.ndarray:
    out = np.zeros(6, np.float32)
    lib().or_rsin_coef(_ptr(out, C.c_float))
    return out


def u24(x: int) -> float:
    return lib().or_u24(x)


def u24p(x: int) -> float:
    return lib().or_u24p(x)


def r64_sum(t, a: int = 0, b: int | None = None) -> np.float32:
    t = np.ascontiguousarray(np.asarray(t, dtype=np.float32))
    b = t.size if b is None else b
    return np.float32(lib().or_r64_sum(_ptr(t, C.c_float), a, b))


def eval_testfn(task: int, x, lo=(-5.12, -5.12), hi=(5.12, 5.12)):
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    lo_a = np.asarray(list(lo) + [0] * (4 - len(lo)), dtype=np.float32)
    hi_a = np.asarray(list(hi) + [1] * (4 - len(hi)), dtype=np.float32)
    fit = np.zeros(1, np.float32)
    desc = np.zeros(2, np.float32)
    lib().or_eval_testfn(task, _ptr(x, C.c_float), x.size, _ptr(lo_a, C.c_float),
                         _ptr(hi_a, C.c_float), _ptr(fit, C.c_float), _ptr(desc, C.c_float))
    return fit[0], desc


def grid_cell(d, grid, lo, hi) -> int:
    D = len(grid)
    d = np.asarray(d, dtype=np.float32)
    g = np.asarray(grid, dtype=np.int32)
    lo_a = np.asarray(lo, dtype=np.float32)
    hi_a = np.asarray(hi, dtype=np.float32)
    return lib().or_grid_cell(_ptr(d, C.c_float), D, _ptr(g, C.c_int32), _ptr(lo_a, C.c_float),
                              _ptr(hi_a, C.c_float))


def cvt_cell(d, lo, hi, cent) -> int:
    d = np.asarray(d, dtype=np.float32)
    cent = np.ascontiguousarray(np.asarray(cent, dtype=np.float32))
    lo_a = np.asarray(lo, dtype=np.float32)
    hi_a = np.asarray(hi, dtype=np.float32)
    return lib().or_cvt_cell(_ptr(d, C.c_float), d.size, _ptr(lo_a, C.c_float),
                             _ptr(hi_a, C.c_float), _ptr(cent, C.c_float), cent.shape[0])


def mlp_rollout(w, obs, hid, act, T, A, B, s0, death_mode=0, death_below=0.0):
    w = np.ascontiguousarray(np.asarray(w, dtype=np.float32))
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float32))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float32))
    s0 = np.ascontiguousarray(np.asarray(s0, dtype=np.float32))
    fit = np.zeros(1, np.float32)
    desc = np.zeros(4, np.float32)
    lib().or_mlp_rollout(_ptr(w, C.c_float), obs, hid, act, T, _ptr(A, C.c_float),
                         _ptr(B, C.c_float), _ptr(s0, C.c_float), death_mode, death_below,
                         _ptr(fit, C.c_float), _ptr(desc, C.c_float))
    return fit[0], desc


def key(f: float, j: int, batch: int) -> int:
    return int(lib().or_key(f, j, batch))


# ---------------------------------------------------------------- the run
class Oracle:
    """One oracle archive with its configuration (Algorithm 1 state).  `path`
    selects a separately built copy of the oracle library."""

    def __init__(self, w: dict, path: str | None = None):
        self.w = dict(w)
        self.cfg = make_config(w)
        self._L = L = lib(path) if path is not None else lib()
        self.n = L.or_genotype_len(C.byref(self.cfg))
        self.env_len = L.or_env_len(C.byref(self.cfg))
        self._s = L.or_new(C.byref(self.cfg), 0)
        self.C, self.D, self.batch = w["C"], w["D"], w["batch"]

    def __del__(self):
        s = getattr(self, "_s", None)
        if s:
            self._L.or_free(s)
            self._s = None

    # -- steps
    def setup(self):
        self._L.or_setup(self._s)

    def init(self):
        return self._L.or_init(self._s)

    def generation(self, g: int):
        rc = self._L.or_generation(self._s, g)
        if rc != 0:
            raise RuntimeError("oracle generation failed (empty archive)")

    def offspring(self, g: int, j: int):
        geno = np.zeros(self.n, np.float32)
        fit = np.zeros(1, np.float32)
        desc = np.zeros(4, np.float32)
        par = np.zeros(2, np.int32)
        rc = self._L.or_offspring(self._s, g, j, _ptr(geno, C.c_float), _ptr(fit, C.c_float),
                                _ptr(desc, C.c_float), _ptr(par, C.c_int32))
        if rc != 0:
            raise RuntimeError("oracle offspring failed (empty archive)")
        return geno, fit[0], desc[: self.D].copy(), par

    def offspring_many(self, g: int, js):
        """Objectives, descriptors and parents of offspring js of generation g
        from the archive as it stands (parallel over js; nothing inserted)."""
        js = np.ascontiguousarray(np.asarray(js, dtype=np.int32).ravel())
        fit = np.zeros(js.size, np.float32)
        desc = np.zeros((js.size, self.D), np.float32)
        par = np.zeros((js.size, 2), np.int32)
        rc = self._L.or_offspring_many(self._s, g, _ptr(js, C.c_int32), js.size,
                                       _ptr(fit, C.c_float), _ptr(desc, C.c_float),
                                       _ptr(par, C.c_int32))
        if rc != 0:
            raise RuntimeError("oracle offspring failed (empty archive)")
        return fit, desc, par

    def insert_driven(self, fit, desc, geno=None):
        fit = np.ascontiguousarray(np.asarray(fit, dtype=np.float32))
        desc = np.ascontiguousarray(np.asarray(desc, dtype=np.float32).reshape(fit.size, self.D))
        nb = fit.size
        cell = np.zeros(nb, np.int32)
        won = np.zeros(nb, np.uint8)
        gp = None
        if geno is not None:
            geno = np.ascontiguousarray(np.asarray(geno, dtype=np.float32).reshape(nb, self.n))
            gp = _ptr(geno, C.c_float)
        self._L.or_insert_driven(self._s, _ptr(fit, C.c_float), _ptr(desc, C.c_float), gp, nb,
                               _ptr(cell, C.c_int32), _ptr(won, C.c_uint8))
        return cell, won

    def stats(self, offset: float = 0.0):
        out = (C.c_double * 3)()
        self._L.or_stats(self._s, offset, out)
        return dict(qd_score=out[0], coverage=int(out[1]), best=out[2])

    # -- views (copies)
    def _arr(self, fn, ctype, count, shape):
        p = getattr(self._L, fn)(self._s)
        return np.ctypeslib.as_array(C.cast(p, C.POINTER(ctype)), shape=(count,)).reshape(
            shape).copy()

    def archive(self):
        C_, D, n = self.C, self.D, self.n
        return dict(
            geno=self._arr("or_archive_geno", C.c_float, C_ * n, (C_, n)),
            fit=self._arr("or_archive_fit", C.c_float, C_, (C_,)),
            desc=self._arr("or_archive_desc", C.c_float, C_ * D, (C_, D)),
            occ=self._arr("or_archive_occ", C.c_uint8, C_, (C_,)),
        )

    def set_archive(self, geno, fit, desc, occ):
        C_, D, n = self.C, self.D, self.n
        for fn, arr, ctype, cnt in (("or_archive_geno", geno, C.c_float, C_ * n),
                                    ("or_archive_fit", fit, C.c_float, C_),
                                    ("or_archive_desc", desc, C.c_float, C_ * D),
                                    ("or_archive_occ", occ, C.c_uint8, C_)):
            p = getattr(self._L, fn)(self._s)
            dst = np.ctypeslib.as_array(C.cast(p, C.POINTER(ctype)), shape=(cnt,))
            dst[:] = np.asarray(arr).reshape(-1)

    def centroids(self):
        return self._arr("or_centroids", C.c_float, self.C * self.D, (self.C, self.D))

    def env(self):
        return self._arr("or_env", C.c_float, max(self.env_len, 1), (max(self.env_len, 1),))[
            : self.env_len]

    def last_batch(self):
        nb, D = self.batch, self.D
        return dict(
            parents=self._arr("or_off_parents", C.c_int32, nb * 2, (nb, 2)),
            fit=self._arr("or_off_fit", C.c_float, nb, (nb,)),
            desc=self._arr("or_off_desc", C.c_float, nb * D, (nb, D)),
            cell=self._arr("or_off_cell", C.c_int32, nb, (nb,)),
            won=self._arr("or_off_won", C.c_uint8, nb, (nb,)),
        )

    def last_offspring(self):
        nb, n = self.batch, self.n
        return self._arr("or_off_geno", C.c_float, nb * n, (nb, n))
