"""Python binding of libqd.so (the C ABI of include/qd.h).

Argument marshalling only: the binding allocates the one workspace tensor with
torch (device memory), passes torch's current HIP stream, and calls the
library.  Every step of a generation runs in the library's HIP kernels.  There
is no fallback: without the built library or a GPU the calls raise.
"""
from __future__ import annotations

import ctypes as C
import os

from . import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqd.so")

ABI_VERSION = 6
CAND_SLOTS = 16
NORMAL_ROWS = 385
QD_OK, QD_ERR_INVALID_ARG, QD_ERR_WORKSPACE_TOO_SMALL, QD_ERR_EMPTY_ARCHIVE, \
    QD_ERR_UNSUPPORTED, QD_ERR_HIP = range(6)

(BUF_ARCHIVE_KEY, BUF_ARCHIVE_FIT, BUF_ARCHIVE_DESC, BUF_ARCHIVE_SLOT, BUF_ARCHIVE_GENO,
 BUF_CENTROIDS, BUF_BUCKET_START, BUF_BUCKET_ITEMS, BUF_CAND_COUNT, BUF_CAND_PTS,
 BUF_LLOYD_ACC, BUF_ENV, BUF_OCC_LIST, BUF_COUNTERS, BUF_OFF_PARENTS, BUF_OFF_FIT, BUF_OFF_DESC,
 BUF_OFF_CELL, BUF_OFF_WON, BUF_OFF_KEY, BUF_OFF_BANK, BUF_OFF_GENO, BUF_STATS,
 BUF_NORMAL_TAB, NUM_BUFFERS) = range(25)

(K_VARY_EVAL, K_ROLLOUT, K_INSERT, K_REGEN, K_SETUP, NUM_KERNELS) = range(6)
KERNEL_NAMES = ["vary_eval", "rollout", "insert", "regen", "setup"]

# Offspring per wave of the test-function generation kernel (the library's
# choice by batch size; the same constants as in csrc/qd_kernels.hpp).  It
# names the kernel instance a profile refers to; results do not depend on it.
OFFSPRING_PER_WAVE, ONE_OFFSPRING_BATCH, TWO_OFFSPRING_BATCH = 4, 2048, 8192


def offspring_per_wave(nb: int) -> int:
    if nb <= ONE_OFFSPRING_BATCH:
        return 1
    return 2 if nb <= TWO_OFFSPRING_BATCH else OFFSPRING_PER_WAVE

# Every symbol include/qd.h declares.
EXPORTS = ["qd_layout_query", "qd_archive_init", "qd_generation", "qd_generations",
           "qd_archive_stats", "qd_archive_stats_noalloc",
           "qd_archive_layout", "qd_normal_table", "qd_sample_normals", "qd_set_kernel_timing",
           "qd_kernel_times",
           "qd_check_fast_arith", "qd_archive_destroy", "qd_status_str"]


class QdConfig(C.Structure):
    _fields_ = [
        ("abi_version", C.c_uint32), ("task", C.c_int32), ("tess", C.c_int32),
        ("genotype_dim", C.c_int32), ("batch_size", C.c_int32), ("desc_dim", C.c_int32),
        ("grid_shape", C.c_int32 * 4), ("num_cells", C.c_int32),
        ("desc_lo", C.c_float * 4), ("desc_hi", C.c_float * 4),
        ("iso_sigma", C.c_float), ("line_sigma", C.c_float),
        ("init_lo", C.c_float), ("init_hi", C.c_float),
        ("mlp_obs", C.c_int32), ("mlp_hidden", C.c_int32), ("mlp_act", C.c_int32),
        ("episode_len", C.c_int32), ("keep_offspring", C.c_int32),
        ("cvt_samples", C.c_int32), ("cvt_iters", C.c_int32),
        ("death_mode", C.c_int32), ("death_below", C.c_float), ("init_mode", C.c_int32),
        ("seed", C.c_uint64),
    ]


class QdLayout(C.Structure):
    _fields_ = [
        ("workspace_bytes", C.c_uint64), ("offset", C.c_uint64 * NUM_BUFFERS),
        ("bytes", C.c_uint64 * NUM_BUFFERS), ("genotype_dim", C.c_int32),
        ("row_stride", C.c_int32), ("bucket_res", C.c_int32), ("num_buckets", C.c_int32),
        ("cand_res", C.c_int32), ("cand_buckets", C.c_int32),
    ]


class QdStats(C.Structure):
    _fields_ = [
        ("qd_score", C.c_double), ("coverage", C.c_double), ("best_fitness", C.c_float),
        ("num_occupied", C.c_int32), ("flags", C.c_uint32), ("reserved", C.c_int32),
    ]


class QdError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_str(status)} (status {status})")


_lib = None


def lib():
    """The loaded libqd.so; raises if it was never built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = C.CDLL(LIB_PATH)
        P, S = C.c_void_p, C.c_int
        L.qd_layout_query.argtypes = [C.POINTER(QdConfig), C.POINTER(QdLayout)]
        L.qd_archive_init.argtypes = [C.POINTER(QdConfig), P, C.c_uint64, P, C.POINTER(P)]
        L.qd_generation.argtypes = [P, C.c_uint32, P]
        L.qd_generations.argtypes = [P, C.c_uint32, C.c_uint32, P]
        L.qd_archive_stats.argtypes = [P, C.c_double, P, C.POINTER(QdStats)]
        L.qd_archive_stats_noalloc.argtypes = [P, C.c_double, P, C.POINTER(QdStats)]
        L.qd_archive_layout.argtypes = [P, C.POINTER(QdLayout)]
        L.qd_sample_normals.argtypes = [P, P, P, C.c_uint64, P]
        L.qd_normal_table.argtypes = [C.POINTER(C.c_float)]
        L.qd_set_kernel_timing.argtypes = [P, C.c_uint32]
        L.qd_kernel_times.argtypes = [P, C.POINTER(C.c_double), C.POINTER(C.c_int32)]
        L.qd_check_fast_arith.argtypes = [P, P, C.POINTER(C.c_uint64)]
        L.qd_archive_destroy.argtypes = [P]
        L.qd_status_str.argtypes = [S]
        L.qd_status_str.restype = C.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = S
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().qd_status_str(status).decode()


def _check(status: int, what: str):
    if status != QD_OK:
        raise QdError(status, what)


def make_config(w: dict, keep_offspring: bool = False) -> QdConfig:
    """qd_config from a workload dict (see workloads.py)."""
    c = QdConfig()
    c.abi_version = ABI_VERSION
    c.task, c.tess = w["task"], w["tess"]
    c.genotype_dim = 0 if w["task"] == W.MLP_SYNTH else w["n"]
    c.batch_size, c.desc_dim, c.num_cells = w["batch"], w["D"], w["C"]
    for k in range(4):
        c.grid_shape[k] = w["grid"][k] if k < len(w["grid"]) else 0
        c.desc_lo[k] = w["lo"][k] if k < len(w["lo"]) else 0.0
        c.desc_hi[k] = w["hi"][k] if k < len(w["hi"]) else 1.0
    c.iso_sigma, c.line_sigma = w["iso_sigma"], w["line_sigma"]
    c.init_lo, c.init_hi = w["init_lo"], w["init_hi"]
    c.mlp_obs, c.mlp_hidden, c.mlp_act, c.episode_len = w["obs"], w["hid"], w["act"], w["T"]
    c.keep_offspring = 1 if keep_offspring else 0
    c.cvt_samples, c.cvt_iters = w.get("cvt_samples", 0), w.get("cvt_iters", 0)
    c.death_mode, c.death_below = w.get("death_mode", 0), w.get("death_below", 0.0)
    c.init_mode = w.get("init_mode", 0)
    c.seed = w["seed"]
    return c


def layout_query(cfg: QdConfig) -> QdLayout:
    out = QdLayout()
    _check(lib().qd_layout_query(C.byref(cfg), C.byref(out)), "qd_layout_query")
    return out


def normal_table():
    """The Gaussian sampler's table as the library builds it (host only):
    numpy float32 [NORMAL_ROWS, 4]."""
    import numpy as np
    out = np.zeros((NORMAL_ROWS, 4), dtype=np.float32)
    _check(lib().qd_normal_table(out.ctypes.data_as(C.POINTER(C.c_float))), "qd_normal_table")
    return out


def check_fast_arith(device: str = "cuda:0") -> list:
    """Mismatch counts of the short division sequences against IEEE
    arithmetic: [tanh (all 2^32 inputs), sigmoid (|x| <= 1)], run on `device`
    and its current stream."""
    import torch
    with torch.cuda.device(torch.device(device)):
        scratch = torch.zeros(2, dtype=torch.int64, device=device)
        out = (C.c_uint64 * 2)()
        _check(lib().qd_check_fast_arith(C.c_void_p(scratch.data_ptr()),
                                         C.c_void_p(_stream_handle(None)), out),
               "qd_check_fast_arith")
    return [int(v) for v in out]


def _stream_handle(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class Archive:
    """An archive in one workspace tensor, created by qd_archive_init."""

    def __init__(self, w: dict, keep_offspring: bool = False, device: str = "cuda:0",
                 stream=None):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("libqd needs a GPU (torch.cuda.is_available() is False)")
        self.w = dict(w)
        self.device = torch.device(device)
        self.cfg = make_config(w, keep_offspring)
        self.layout = layout_query(self.cfg)
        self.n = self.layout.genotype_dim
        self.stride = self.layout.row_stride
        self.C, self.D, self.batch = w["C"], w["D"], w["batch"]
        with torch.cuda.device(self.device):
            self.ws = torch.empty(self.layout.workspace_bytes, dtype=torch.uint8,
                                  device=self.device)
            self.stream = stream if stream is not None else torch.cuda.current_stream()
            h = C.c_void_p()
            _check(lib().qd_archive_init(C.byref(self.cfg), C.c_void_p(self.ws.data_ptr()),
                                         self.layout.workspace_bytes,
                                         C.c_void_p(_stream_handle(self.stream)), C.byref(h)),
                   "qd_archive_init")
        self._h = h
        self._destroy = lib().qd_archive_destroy

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            try:
                self.stream.synchronize()
            except Exception:
                pass
            self._destroy(h)   # bound at creation: module globals may be gone at exit
            self._h = None

    # -- the path
    def generation(self, g: int):
        _check(lib().qd_generation(self._h, g, C.c_void_p(_stream_handle(self.stream))),
               "qd_generation")

    def generations(self, first: int, count: int):
        """Generations first .. first + count - 1, enqueued by one library call."""
        _check(lib().qd_generations(self._h, first, count,
                                    C.c_void_p(_stream_handle(self.stream))), "qd_generations")

    def sample_normals(self, words) -> "np.ndarray":
        """The archive's Gaussian sampler applied to each 32-bit word (array-like
        of uint32); runs on the archive's device and stream, returns numpy f32."""
        import numpy as np
        import torch
        w = np.ascontiguousarray(np.asarray(words, dtype=np.uint32).ravel())
        with torch.cuda.stream(self.stream):
            d_w = torch.from_numpy(w.view(np.int32)).to(self.ws.device)
            d_z = torch.empty(w.size, dtype=torch.float32, device=self.ws.device)
            _check(lib().qd_sample_normals(self._h, C.c_void_p(d_w.data_ptr()),
                                           C.c_void_p(d_z.data_ptr()), w.size,
                                           C.c_void_p(_stream_handle(self.stream))),
                   "qd_sample_normals")
        self.stream.synchronize()
        return d_z.cpu().numpy()

    def stats(self, offset: float = 0.0, noalloc: bool = False) -> dict:
        """QD-score, coverage, best objective and flags (qd_archive_stats, or
        with noalloc=True qd_archive_stats_noalloc)."""
        out = QdStats()
        fn = lib().qd_archive_stats_noalloc if noalloc else lib().qd_archive_stats
        _check(fn(self._h, offset, C.c_void_p(_stream_handle(self.stream)), C.byref(out)),
               "qd_archive_stats_noalloc" if noalloc else "qd_archive_stats")
        return dict(qd_score=out.qd_score, coverage=out.coverage, best=out.best_fitness,
                    num_occupied=out.num_occupied, flags=out.flags)

    def set_kernel_timing(self, kernels=()):
        """Time the launches of the named kernels (KERNEL_NAMES); () turns it off."""
        mask = 0
        for k in kernels:
            mask |= 1 << KERNEL_NAMES.index(k)
        _check(lib().qd_set_kernel_timing(self._h, mask), "qd_set_kernel_timing")

    def kernel_times(self) -> dict:
        ms = (C.c_double * NUM_KERNELS)()
        cnt = (C.c_int32 * NUM_KERNELS)()
        _check(lib().qd_kernel_times(self._h, ms, cnt), "qd_kernel_times")
        return {KERNEL_NAMES[k]: (ms[k], cnt[k]) for k in range(NUM_KERNELS)}

    # -- typed views onto the workspace (torch tensors sharing its memory)
    def view(self, buf: int, dtype, shape):
        import torch
        off, nbytes = self.layout.offset[buf], self.layout.bytes[buf]
        if nbytes == 0:
            return None
        item = torch.empty((), dtype=dtype).element_size()
        count = 1
        for s in shape:
            count *= s
        assert count * item <= nbytes, (buf, shape, nbytes)
        return self.ws[off: off + count * item].view(dtype).view(*shape)

    def views(self) -> dict:
        import torch
        C_, D, nb, st = self.C, self.D, self.batch, self.stride
        return dict(
            key=self.view(BUF_ARCHIVE_KEY, torch.int64, (C_,)),
            fit=self.view(BUF_ARCHIVE_FIT, torch.float32, (C_,)),
            desc=self.view(BUF_ARCHIVE_DESC, torch.float32, (C_, D)),
            slot=self.view(BUF_ARCHIVE_SLOT, torch.int32, (C_,)),
            geno=self.view(BUF_ARCHIVE_GENO, torch.float32, (2, C_, st)),
            centroids=self.view(BUF_CENTROIDS, torch.float32, (C_, D)),
            cand_count=self.view(BUF_CAND_COUNT, torch.int32, (self.layout.cand_buckets,)),
            cand_pts=self.view(BUF_CAND_PTS, torch.float32,
                               (self.layout.cand_buckets, CAND_SLOTS, 4)),
            env=self.view(BUF_ENV, torch.float32, (self.layout.bytes[BUF_ENV] // 4,)),
            occ_list=self.view(BUF_OCC_LIST, torch.int32, (C_,)),
            counters=self.view(BUF_COUNTERS, torch.int32, (64,)),
            parents=self.view(BUF_OFF_PARENTS, torch.int32, (nb, 2)),
            off_fit=self.view(BUF_OFF_FIT, torch.float32, (nb,)),
            off_desc=self.view(BUF_OFF_DESC, torch.float32, (nb, D)),
            off_cell=self.view(BUF_OFF_CELL, torch.int32, (nb,)),
            off_won=self.view(BUF_OFF_WON, torch.uint8, (nb,)),
            off_key=self.view(BUF_OFF_KEY, torch.int64, (nb,)),
            off_bank=self.view(BUF_OFF_BANK, torch.uint8, (nb,)),
            off_geno=self.view(BUF_OFF_GENO, torch.float32, (nb, st)),
            normal_tab=self.view(BUF_NORMAL_TAB, torch.float32, (NORMAL_ROWS, 4)),
        )

    def snapshot(self) -> dict:
        """Host copies of the archive (elite genotypes gathered from their banks)."""
        import torch
        self.stream.synchronize()
        v = self.views()
        key = v["key"].cpu().numpy().view("uint64")
        occ = (key != 0).astype("uint8")
        slot = v["slot"].cpu().long()
        rows = v["geno"][slot.to(self.device), torch.arange(self.C, device=self.device)]
        return dict(
            key=key, occ=occ, fit=v["fit"].cpu().numpy(), desc=v["desc"].cpu().numpy(),
            geno=rows[:, : self.n].cpu().numpy(), slot=slot.numpy(),
            n_occ=int(v["counters"][0].item()), occ_list=v["occ_list"].cpu().numpy(),
        )

    def last_batch(self) -> dict:
        self.stream.synchronize()
        v = self.views()
        out = dict(parents=v["parents"].cpu().numpy(), fit=v["off_fit"].cpu().numpy(),
                   desc=v["off_desc"].cpu().numpy(), cell=v["off_cell"].cpu().numpy(),
                   won=v["off_won"].cpu().numpy())
        if v["off_geno"] is not None:
            out["geno"] = v["off_geno"][:, : self.n].cpu().numpy()
        return out
