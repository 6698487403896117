"""ctypes binding of libaspis (include/aspis.h).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the path runs in the library (host C++ for the
assignment and clique steps, gfx950 kernels for everything that touches the
gradients).  If the library is not built this module raises on import of
the library -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaspis.so")

OK, ERR_INVALID_ARG, ERR_OVERFLOW, ERR_BUFFER_SMALL, ERR_DEVICE, ERR_NO_FILES = range(6)
REDUCE = {"median": 0, "mean": 1, "paper": 2}
ATTACK = {"weak": 0, "optimal": 1}
FLAG_TWO_PASS = 1
FLAG_TIMING = 2
FLAG_FULL_KEYS = 4
FLAG_HALF_KEYS = 8
FLAG_PROBE_PREFIX = 16

EXPORTED = (
    "aspis_num_files", "aspis_assign", "aspis_detect", "aspis_clique",
    "aspis_aggregate_workspace", "aspis_aggregate", "aspis_detect_aggregate",
    "aspis_detect_aggregate_wm", "aspis_detect_aggregate_noalloc", "aspis_worker_rows",
    "aspis_plan",
    "aspis_read_probe_sink_words", "aspis_read_probe", "aspis_simulate", "aspis_detox",
    "aspis_last_error",
)


class AspisError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"aspis status {status}: {message}")
        self.status = status


class DetectOut(ctypes.Structure):
    _fields_ = [("pair_diff", ctypes.c_void_p), ("vote", ctypes.c_void_p),
                ("has_majority", ctypes.c_void_p), ("disagree", ctypes.c_void_p)]


class CliqueResult(ctypes.Structure):
    _fields_ = [("success", ctypes.c_int32), ("omega", ctypes.c_int32),
                ("n_maximum", ctypes.c_int32), ("n_words", ctypes.c_int32),
                ("n_maximal", ctypes.c_int64), ("honest", ctypes.c_uint64 * 2),
                ("detected", ctypes.c_uint64 * 2), ("first", ctypes.c_uint64 * 2)]

    def as_dict(self, K: int) -> dict:
        def members(words):
            return frozenset(u for u in range(K) if (words[u // 64] >> (u % 64)) & 1)
        return {"success": bool(self.success), "omega": self.omega,
                "n_maximum": self.n_maximum, "n_maximal": self.n_maximal,
                "honest": members(self.honest) if self.success else frozenset(),
                "detected": members(self.detected) if self.success else frozenset(),
                "first": members(self.first)}


class SimResult(ctypes.Structure):
    _fields_ = [("files", ctypes.c_int64), ("distorted", ctypes.c_int64),
                ("dropped", ctypes.c_int64), ("success", ctypes.c_int32),
                ("omega", ctypes.c_int32), ("n_maximum", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("n_maximal", ctypes.c_int64),
                ("epsilon", ctypes.c_double), ("epsilon_baseline", ctypes.c_double),
                ("ms_files", ctypes.c_double), ("ms_clique", ctypes.c_double)]

    def as_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "reserved"}
        d["success"] = bool(d["success"])
        return d


class RunStats(ctypes.Structure):
    _fields_ = [("fused", ctypes.c_int32), ("speculation_hit", ctypes.c_int32),
                ("probe_coords", ctypes.c_int64), ("ms_probe", ctypes.c_float),
                ("ms_main", ctypes.c_float), ("ms_fallback", ctypes.c_float),
                ("ms_total", ctypes.c_float), ("tile_cols", ctypes.c_int32),
                ("half_keys", ctypes.c_int32), ("tie_rows", ctypes.c_int32),
                ("probe_blocks", ctypes.c_int32), ("repair_groups", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


KERNEL = {0: "none", 1: "fused_ws", 2: "fused", 3: "median_ws", 4: "median_tile",
          5: "median_radix"}


class KernelPlan(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("tile_cols", ctypes.c_int32),
                ("sweeps", ctypes.c_int32), ("half_keys", ctypes.c_int32),
                ("stream_threads", ctypes.c_int32), ("row_table", ctypes.c_int32),
                ("block", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int64)]

    def as_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "reserved"}
        d["kernel"] = KERNEL.get(self.kernel, str(self.kernel))
        return d


_lib = None


def lib():
    """Load libaspis.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python -c 'import __graft_entry__ as g; "
                          f"g.build()'` (or python paper_2108_02416_amd/build.py) first")
    # torch bundles a HIP runtime whose soname equals the system one; it must
    # be mapped first so that torch and this library share one runtime.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    L.aspis_num_files.argtypes = [i32, i32]
    L.aspis_num_files.restype = i64
    L.aspis_assign.argtypes = [i32, i32, P, i64]
    L.aspis_assign.restype = ctypes.c_int
    L.aspis_detect.argtypes = [P, i32, i32, i64, P, ctypes.POINTER(DetectOut), P]
    L.aspis_detect.restype = ctypes.c_int
    L.aspis_clique.argtypes = [P, i32, i32, ctypes.POINTER(CliqueResult)]
    L.aspis_clique.restype = ctypes.c_int
    L.aspis_aggregate_workspace.argtypes = [i32, i32, i64]
    L.aspis_aggregate_workspace.restype = ctypes.c_size_t
    L.aspis_aggregate.argtypes = [P, i32, i32, i64, P, ctypes.POINTER(DetectOut),
                                  ctypes.POINTER(CliqueResult), ctypes.c_int, P, P,
                                  ctypes.POINTER(i64), P, ctypes.c_size_t, P]
    L.aspis_aggregate.restype = ctypes.c_int
    L.aspis_detect_aggregate.argtypes = [P, i32, i32, i32, i64, P, ctypes.POINTER(DetectOut),
                                         ctypes.c_int, P, P, ctypes.POINTER(CliqueResult),
                                         ctypes.POINTER(i64), P, ctypes.c_size_t, u32,
                                         ctypes.POINTER(RunStats), P]
    L.aspis_detect_aggregate.restype = ctypes.c_int
    L.aspis_detect_aggregate_wm.argtypes = L.aspis_detect_aggregate.argtypes
    L.aspis_detect_aggregate_wm.restype = ctypes.c_int
    L.aspis_detect_aggregate_noalloc.argtypes = [P, i32, i32, i32, i64, P,
                                                 ctypes.POINTER(DetectOut), ctypes.c_int, P, P,
                                                 ctypes.POINTER(CliqueResult),
                                                 ctypes.POINTER(i64), u32,
                                                 ctypes.POINTER(RunStats), P]
    L.aspis_detect_aggregate_noalloc.restype = ctypes.c_int
    L.aspis_worker_rows.argtypes = [i32, i32, P, i64]
    L.aspis_worker_rows.restype = ctypes.c_int
    L.aspis_plan.argtypes = [i32, i32, i64, i32, u32, ctypes.POINTER(KernelPlan),
                             ctypes.POINTER(KernelPlan)]
    L.aspis_plan.restype = ctypes.c_int
    L.aspis_read_probe_sink_words.argtypes = []
    L.aspis_read_probe_sink_words.restype = ctypes.c_size_t
    L.aspis_read_probe.argtypes = [P, ctypes.c_size_t, P, P]
    L.aspis_read_probe.restype = ctypes.c_int
    L.aspis_simulate.argtypes = [i32, i32, i32, ctypes.c_int, P, P, ctypes.POINTER(SimResult), P]
    L.aspis_simulate.restype = ctypes.c_int
    L.aspis_detox.argtypes = [i32, i32, i32, ctypes.c_int, ctypes.POINTER(i64),
                              ctypes.POINTER(ctypes.c_double)]
    L.aspis_detox.restype = ctypes.c_int
    L.aspis_last_error.argtypes = []
    L.aspis_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int):
    if status != OK:
        raise AspisError(status, lib().aspis_last_error().decode())


# ---------------------------------------------------------------- host steps

def num_files(K: int, r: int) -> int:
    return int(lib().aspis_num_files(K, r))


def assign(K: int, r: int) -> np.ndarray:
    f = num_files(K, r)
    if f <= 0:
        raise AspisError(ERR_INVALID_ARG, f"invalid (K={K}, r={r})")
    out = np.zeros((f, r), dtype=np.int32)
    _check(lib().aspis_assign(K, r, out.ctypes.data, f))
    return out


def worker_rows(K: int, r: int) -> np.ndarray:
    """Row of replica (i, s) in the worker-major upload [K][l][d]:
    int32 [f, r] (aspis_worker_rows)."""
    f = num_files(K, r)
    if f <= 0:
        raise AspisError(ERR_INVALID_ARG, f"invalid (K={K}, r={r})")
    out = np.zeros((f, r), dtype=np.int32)
    _check(lib().aspis_worker_rows(K, r, out.ctypes.data, f * r))
    return out


def plan(K: int, r: int, d: int, layout: str = "file", flags: int = 0) -> tuple[dict, dict]:
    """The kernels the device entry points take for this shape (aspis_plan):
    (single pass, median), each a dict of the kernel's tile parameters;
    flags may hold FLAG_FULL_KEYS."""
    sp, med = KernelPlan(), KernelPlan()
    _check(lib().aspis_plan(K, r, d, 1 if layout == "worker" else 0, flags, ctypes.byref(sp),
                            ctypes.byref(med)))
    return sp.as_dict(), med.as_dict()


def clique(disagree_rows: np.ndarray, K: int, q: int) -> CliqueResult:
    rows = np.ascontiguousarray(disagree_rows, dtype=np.uint64).reshape(K, -1)
    res = CliqueResult()
    _check(lib().aspis_clique(rows.ctypes.data, K, q, ctypes.byref(res)))
    return res


def simulate(K: int, r: int, q: int, attack: str = "optimal", adversaries=None,
             disagree_set=None, want_rows: bool = False) -> dict:
    """Distortion-fraction simulation of one attack on symbolic replicas
    (aspis_simulate); returns the result fields, plus the disagreement rows
    when want_rows."""
    def ids(x):
        if x is None:
            return None, None
        a = np.ascontiguousarray(np.asarray(x, dtype=np.int32).reshape(-1))
        if a.size != q:
            raise AspisError(ERR_INVALID_ARG, f"need {q} worker ids, got {a.size}")
        return a, a.ctypes.data
    a_arr, a_ptr = ids(adversaries)
    d_arr, d_ptr = ids(disagree_set)
    res = SimResult()
    rows = np.zeros((K, (K + 63) // 64), dtype=np.uint64) if want_rows else None
    _check(lib().aspis_simulate(K, r, q, ATTACK[attack], a_ptr, d_ptr, ctypes.byref(res),
                                rows.ctypes.data if rows is not None else None))
    out = res.as_dict()
    if want_rows:
        out["disagree_rows"] = rows
    return out


def detox(K: int, r: int, q: int, attack: str = "optimal") -> tuple[int, float]:
    """DETOX group-majority distortion (aspis_detox): (groups, epsilon)."""
    groups = ctypes.c_int64(0)
    eps = ctypes.c_double(0.0)
    _check(lib().aspis_detox(K, r, q, ATTACK[attack], ctypes.byref(groups), ctypes.byref(eps)))
    return int(groups.value), float(eps.value)


# -------------------------------------------------------------- device steps

def _torch():
    import torch
    return torch


def _stream_ptr():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check_grads(grads, K: int, r: int):
    torch = _torch()
    f = num_files(K, r)
    if not (grads.is_cuda and grads.dtype == torch.float32 and grads.dim() == 3
            and grads.is_contiguous() and grads.shape[0] == f and grads.shape[1] == r):
        raise AspisError(ERR_INVALID_ARG,
                         f"grads must be a contiguous cuda float32 [{f}, {r}, d] tensor")
    return f, grads.shape[2]


def _check_buffer(name: str, t, dtype, n: int, device):
    """A caller-supplied buffer must be a contiguous tensor of `dtype` with at
    least n elements on the replicas' device: the kernels write n elements."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise AspisError(ERR_INVALID_ARG, f"{name} must be a torch tensor")
    if t.dtype != dtype or not t.is_contiguous() or t.device != device or t.numel() < n:
        raise AspisError(ERR_INVALID_ARG,
                         f"{name} must be a contiguous {dtype} tensor on {device} with at "
                         f"least {n} elements (got {t.dtype}, {tuple(t.shape)}, {t.device}, "
                         f"contiguous={t.is_contiguous()})")


def _check_outputs(device, f: int, K: int, d: int, bufs=None, out=None, sel_out=None, ws=None):
    torch = _torch()
    if bufs is not None:
        _check_buffer("bufs.pair_diff", bufs.pair_diff, torch.int32, f, device)
        _check_buffer("bufs.vote", bufs.vote, torch.int8, f, device)
        _check_buffer("bufs.has_majority", bufs.has_majority, torch.uint8, f, device)
        _check_buffer("bufs.disagree", bufs.disagree, torch.int64, K, device)
    if out is not None:
        _check_buffer("out", out, torch.float32, d, device)
    if sel_out is not None:
        _check_buffer("sel_out", sel_out, torch.int32, f, device)
    if ws is not None:
        _check_buffer("ws", ws, torch.uint8, 1, device)


@dataclass
class DetectBuffers:
    pair_diff: object
    vote: object
    has_majority: object
    disagree: object

    @classmethod
    def empty(cls, f: int, K: int, device):
        torch = _torch()
        return cls(torch.empty(f, dtype=torch.int32, device=device),
                   torch.empty(f, dtype=torch.int8, device=device),
                   torch.empty(f, dtype=torch.uint8, device=device),
                   torch.empty(K, dtype=torch.int64, device=device))

    def c(self) -> DetectOut:
        return DetectOut(self.pair_diff.data_ptr(), self.vote.data_ptr(),
                         self.has_majority.data_ptr(), self.disagree.data_ptr())


_subsets_cache: dict = {}


def subsets_device(K: int, r: int, device):
    key = (K, r, str(device))
    if key not in _subsets_cache:
        torch = _torch()
        _subsets_cache[key] = torch.from_numpy(assign(K, r)).to(device)
    return _subsets_cache[key]


def workspace(K: int, r: int, d: int, device):
    torch = _torch()
    n = int(lib().aspis_aggregate_workspace(K, r, d))
    if n == 0:
        raise AspisError(ERR_INVALID_ARG, "invalid shape for workspace")
    return torch.empty(n + 256, dtype=torch.uint8, device=device)


def _aligned_ptr(ws) -> tuple[int, int]:
    p = ws.data_ptr()
    off = (-p) % 256
    return p + off, ws.numel() - off


def detect(grads, K: int, r: int, bufs: DetectBuffers | None = None) -> DetectBuffers:
    f, d = _check_grads(grads, K, r)
    bufs = bufs or DetectBuffers.empty(f, K, grads.device)
    _check_outputs(grads.device, f, K, d, bufs=bufs)
    sub = subsets_device(K, r, grads.device)
    out = bufs.c()
    _check(lib().aspis_detect(grads.data_ptr(), K, r, d, sub.data_ptr(), ctypes.byref(out),
                              _stream_ptr()))
    return bufs


def aggregate(grads, K: int, r: int, bufs: DetectBuffers, res: CliqueResult,
              mode: str = "median", out=None, sel_out=None, ws=None):
    torch = _torch()
    f, d = _check_grads(grads, K, r)
    out = out if out is not None else torch.empty(d, dtype=torch.float32, device=grads.device)
    ws = ws if ws is not None else workspace(K, r, d, grads.device)
    _check_outputs(grads.device, f, K, d, bufs=bufs, out=out, sel_out=sel_out, ws=ws)
    wp, wn = _aligned_ptr(ws)
    n_sel = ctypes.c_int64(0)
    det = bufs.c()
    st = lib().aspis_aggregate(grads.data_ptr(), K, r, d,
                               subsets_device(K, r, grads.device).data_ptr(), ctypes.byref(det),
                               ctypes.byref(res), REDUCE[mode], out.data_ptr(),
                               sel_out.data_ptr() if sel_out is not None else None,
                               ctypes.byref(n_sel), wp, wn, _stream_ptr())
    _check(st)
    return out, int(n_sel.value)


def _check_grads_wm(grads, K: int, r: int):
    torch = _torch()
    f = num_files(K, r)
    l_files = f * r // K
    if not (grads.is_cuda and grads.dtype == torch.float32 and grads.dim() == 3
            and grads.is_contiguous() and grads.shape[0] == K and grads.shape[1] == l_files):
        raise AspisError(ERR_INVALID_ARG,
                         f"grads must be a contiguous cuda float32 [{K}, {l_files}, d] tensor")
    return f, grads.shape[2]


def detect_aggregate(grads, K: int, r: int, q: int, mode: str = "median", flags: int = 0,
                     bufs: DetectBuffers | None = None, out=None, sel_out=None, ws=None,
                     want_sel: bool = True, layout: str = "file") -> dict:
    """The whole step (Algorithm 3 then Algorithm 1) in one library call.
    layout "file": grads is [f][r][d]; "worker": grads is the workers'
    upload [K][l][d] (aspis_detect_aggregate_wm)."""
    torch = _torch()
    if layout not in ("file", "worker"):
        raise AspisError(ERR_INVALID_ARG, f"unknown layout {layout!r}")
    f, d = (_check_grads if layout == "file" else _check_grads_wm)(grads, K, r)
    bufs = bufs or DetectBuffers.empty(f, K, grads.device)
    out = out if out is not None else torch.empty(d, dtype=torch.float32, device=grads.device)
    if sel_out is None and want_sel:
        sel_out = torch.empty(f, dtype=torch.int32, device=grads.device)
    ws = ws if ws is not None else workspace(K, r, d, grads.device)
    _check_outputs(grads.device, f, K, d, bufs=bufs, out=out, sel_out=sel_out, ws=ws)
    wp, wn = _aligned_ptr(ws)
    res = CliqueResult()
    stats = RunStats()
    n_sel = ctypes.c_int64(0)
    det = bufs.c()
    entry = lib().aspis_detect_aggregate if layout == "file" else lib().aspis_detect_aggregate_wm
    st = entry(
        grads.data_ptr(), K, r, q, d, subsets_device(K, r, grads.device).data_ptr(),
        ctypes.byref(det), REDUCE[mode], out.data_ptr(),
        sel_out.data_ptr() if sel_out is not None else None, ctypes.byref(res),
        ctypes.byref(n_sel), wp, wn, flags, ctypes.byref(stats), _stream_ptr())
    _check(st)
    return {"out": out, "sel": sel_out, "bufs": bufs, "clique": res,
            "n_selected": int(n_sel.value), "stats": stats.as_dict()}


def detect_aggregate_noalloc(grads, K: int, r: int, q: int, bufs: DetectBuffers, out,
                             sel_out=None, mode: str = "median", flags: int = 0) -> dict:
    """aspis_detect_aggregate_noalloc: the whole step with the library's
    static device scratch instead of a workspace; the caller passes every
    output buffer (nothing is allocated here either)."""
    f, d = _check_grads(grads, K, r)
    _check_outputs(grads.device, f, K, d, bufs=bufs, out=out, sel_out=sel_out)
    res = CliqueResult()
    stats = RunStats()
    n_sel = ctypes.c_int64(0)
    det = bufs.c()
    st = lib().aspis_detect_aggregate_noalloc(
        grads.data_ptr(), K, r, q, d, subsets_device(K, r, grads.device).data_ptr(),
        ctypes.byref(det), REDUCE[mode], out.data_ptr(),
        sel_out.data_ptr() if sel_out is not None else None, ctypes.byref(res),
        ctypes.byref(n_sel), flags, ctypes.byref(stats), _stream_ptr())
    _check(st)
    return {"out": out, "sel": sel_out, "bufs": bufs, "clique": res,
            "n_selected": int(n_sel.value), "stats": stats.as_dict()}


def read_probe(buf, sink=None) -> float:
    """Stream buf once; returns nothing useful on the host (see bench.py)."""
    torch = _torch()
    words = int(lib().aspis_read_probe_sink_words())
    if sink is None:
        sink = torch.empty(words, dtype=torch.int32, device=buf.device)
    nbytes = buf.numel() * buf.element_size()
    nbytes -= nbytes % 16
    _check(lib().aspis_read_probe(buf.data_ptr(), nbytes, sink.data_ptr(), _stream_ptr()))
    return sink
