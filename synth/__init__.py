"""Seeded synthetic workloads for the detect-and-aggregate step.

This is the single input generator that both the oracle and the HIP path
consume.  It holds none of the method's arithmetic: the file->worker table is
passed in by the caller, and this module only decides which replica carries
which value (the attack simulation of Section 4.1 / 4.2 of the paper) and
writes the numbers (``synth.hip``: a host fill for the oracle and a GPU fill
that writes the same bytes straight into device memory).

Workloads (shapes of the paper's CIFAR-10 / ResNet-18 experiments; r = 3
except workload 6):

  1  K=7,  q=2, d=100,000     weak attack, workers {0,1}, reversed gradient
  2  K=15, q=3, d=1,000,000   weak attack, 3 seeded-random workers, ALIE
  3  K=15, q=4, d=11,200,000  optimal attack (Theorem 1), exhaustive choice
                              of the adversary set, ALIE          (headline)
  4  K=21, q=5, d=5,000,000   weak attack, 5 seeded-random workers: 3 ALIE
                              colluders + 2 independent N(0,1) noise senders
  5  K=25, q=6, d=2,000,000   optimal attack, greedy choice, Student-t(3)
                              honest gradients, reversed gradient
  6  K=11, r=5, q=4, d=6,500,000  optimal attack, exhaustive choice, ALIE:
                              the redundancy r = 5 at 462 files
"""
from __future__ import annotations

import ctypes
import itertools
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "libsynth.so")
_lib = None

ROLE_HONEST, ROLE_REVERSED, ROLE_ALIE, ROLE_NOISE = 0, 1, 2, 3
DIST_NORMAL, DIST_STUDENT3, DIST_TIED = 0, 1, 2
SEED = 428          # the paper's primary seed (its repeat seed is 50)
SEED_REPEAT = 50


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    # torch bundles a HIP runtime whose soname equals the system one; it must
    # be mapped first so that torch and the GPU fill share one runtime.
    import torch  # noqa: F401
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    lib.synth_fill.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64,
                               ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                               ctypes.c_double, P, ctypes.c_int32]
    lib.synth_fill.restype = ctypes.c_int
    lib.synth_u32.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64]
    lib.synth_u32.restype = ctypes.c_uint32
    lib.synth_honest_value.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_uint32,
                                       ctypes.c_uint64]
    lib.synth_honest_value.restype = ctypes.c_float
    lib.synth_fill_device.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64,
                                      ctypes.c_int32, ctypes.c_uint64, ctypes.c_double,
                                      ctypes.c_int32, P, P, P]
    lib.synth_fill_device.restype = ctypes.c_int
    lib.synth_fnv1a.argtypes = [P, ctypes.c_int64]
    lib.synth_fnv1a.restype = ctypes.c_uint64
    lib.synth_normal.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                 ctypes.c_uint32, ctypes.c_uint64]
    lib.synth_normal.restype = ctypes.c_double
    lib.synth_log.argtypes = [ctypes.c_double]
    lib.synth_log.restype = ctypes.c_double
    _lib = lib
    return lib


@dataclass(frozen=True)
class Workload:
    index: int
    K: int
    r: int
    q: int
    d: int
    dist: int
    attack: str        # "weak" | "optimal"
    distortion: str    # "reversed" | "alie" | "alie+noise"
    choice: str        # "fixed" | "random" | "exhaustive" | "greedy"
    alie_z: float = 1.0

    @property
    def name(self) -> str:
        return (f"aspis-K{self.K}-r{self.r}-q{self.q}-d{self.d}-"
                f"{self.attack}-{self.distortion}")

    @property
    def f(self) -> int:
        from math import comb
        return comb(self.K, self.r)

    def replica_bytes(self) -> int:
        return self.f * self.r * self.d * 4


WORKLOADS = {
    1: Workload(1, 7, 3, 2, 100_000, DIST_NORMAL, "weak", "reversed", "fixed"),
    2: Workload(2, 15, 3, 3, 1_000_000, DIST_NORMAL, "weak", "alie", "random"),
    3: Workload(3, 15, 3, 4, 11_200_000, DIST_NORMAL, "optimal", "alie", "exhaustive"),
    4: Workload(4, 21, 3, 5, 5_000_000, DIST_NORMAL, "weak", "alie+noise", "random"),
    5: Workload(5, 25, 3, 6, 2_000_000, DIST_STUDENT3, "optimal", "reversed", "greedy"),
    # r = 5: five replicas a file, 462 files (the headline's file count), 60 GB
    6: Workload(6, 11, 5, 4, 6_500_000, DIST_NORMAL, "optimal", "alie", "exhaustive"),
}


def u32(seed: int, stream: int, index: int) -> int:
    return int(_load().synth_u32(seed, stream, index))


def seeded_permutation(n: int, seed: int, stream: int = 7) -> list[int]:
    """Fisher-Yates shuffle of range(n) driven by Philox draws."""
    perm = list(range(n))
    for i in range(n - 1, 0, -1):
        j = u32(seed, stream, i) % (i + 1)
        perm[i], perm[j] = perm[j], perm[i]
    return perm


def _majority_files(subsets: np.ndarray, A) -> int:
    r = subsets.shape[1]
    need = (r + 1) // 2
    inA = np.isin(subsets, list(A))
    return int((inA.sum(axis=1) >= need).sum())


def choose_adversaries(wl: Workload, subsets: np.ndarray, seed: int) -> list[int]:
    """The attacker's choice of the q Byzantine workers."""
    K, q = wl.K, wl.q
    if wl.choice == "fixed":
        return list(range(q))
    if wl.choice == "random":
        return sorted(seeded_permutation(K, seed)[:q])
    if wl.choice == "exhaustive":
        best, best_set = -1, None
        for A in itertools.combinations(range(K), q):
            c = _majority_files(subsets, A)
            if c > best:
                best, best_set = c, list(A)
        return best_set
    if wl.choice == "greedy":
        A: list[int] = []
        for _ in range(q):
            best, best_u = -1, None
            for u in range(K):
                if u in A:
                    continue
                c = _majority_files(subsets, A + [u])
                if c > best:
                    best, best_u = c, u
            A.append(best_u)
        return sorted(A)
    raise ValueError(wl.choice)


def make_roles(wl: Workload, subsets: np.ndarray, seed: int = SEED,
               adversaries=None, disagree_set=None):
    """Per-replica role table for the workload's attack.

    weak    (Section 4.1): every adversary distorts every file it holds.
    optimal (Section 4.2, Theorem 1): all adversaries disagree with one fixed
            set D of q honest workers; an adversary distorts file F exactly
            when the adversaries hold a majority of F and every honest
            member of F is in D.
    Returns (role uint8 [f, r], worker int32 [f, r], A list, D list).
    """
    subsets = np.ascontiguousarray(subsets, dtype=np.int32)
    f, r = subsets.shape
    need = (r + 1) // 2
    A = list(adversaries) if adversaries is not None else choose_adversaries(wl, subsets, seed)
    Aset = set(A)
    honest = [u for u in range(wl.K) if u not in Aset]
    D = list(disagree_set) if disagree_set is not None else honest[: wl.q]
    Dset = set(D)
    # role of each adversary
    kind = {}
    if wl.distortion == "reversed":
        kind = {u: ROLE_REVERSED for u in A}
    elif wl.distortion == "alie":
        kind = {u: ROLE_ALIE for u in A}
    elif wl.distortion == "alie+noise":
        order = [u for u in seeded_permutation(wl.K, seed, stream=11) if u in Aset]
        n_alie = (len(A) + 1) // 2
        kind = {u: (ROLE_ALIE if j < n_alie else ROLE_NOISE) for j, u in enumerate(order)}
    else:
        raise ValueError(wl.distortion)
    role = np.zeros((f, r), dtype=np.uint8)
    for i in range(f):
        members = [int(u) for u in subsets[i]]
        advs = [u for u in members if u in Aset]
        if wl.attack == "weak":
            distort = True
        else:
            others = [u for u in members if u not in Aset]
            distort = len(advs) >= need and all(u in Dset for u in others)
        if not distort:
            continue
        for s, u in enumerate(members):
            if u in Aset:
                role[i, s] = kind[u]
    return role, subsets.copy(), A, D


def fill(role: np.ndarray, worker: np.ndarray, k0: int, nk: int, dist: int,
         seed: int = SEED, alie_z: float = 1.0, out: np.ndarray | None = None,
         nthreads: int | None = None) -> np.ndarray:
    """Coordinates [k0, k0+nk) of every replica as float32 [f, r, nk]."""
    role = np.ascontiguousarray(role, dtype=np.uint8)
    worker = np.ascontiguousarray(worker, dtype=np.int32)
    f, r = role.shape
    if out is None:
        out = np.empty((f, r, nk), dtype=np.float32)
    if out.dtype != np.float32 or not out.flags.c_contiguous or out.size != f * r * nk:
        raise ValueError("out must be contiguous float32 [f, r, nk]")
    if nthreads is None:
        nthreads = min(16, os.cpu_count() or 1)
    rc = _load().synth_fill(role.ctypes.data, worker.ctypes.data, f, r, k0, nk, dist,
                            seed, alie_z, out.ctypes.data, nthreads)
    if rc != 0:
        raise RuntimeError(f"synth_fill failed ({rc})")
    return out


def fill_device(role: np.ndarray, worker: np.ndarray, out, dist: int, seed: int = SEED,
                alie_z: float = 1.0):
    """Write every replica of all d coordinates into the device tensor
    ``out`` (contiguous float32 [f, r, d]) -- the same bytes as ``fill``."""
    import torch
    role = np.ascontiguousarray(role, dtype=np.uint8)
    worker = np.ascontiguousarray(worker, dtype=np.int32)
    f, r = role.shape
    if not (out.is_cuda and out.dtype == torch.float32 and out.is_contiguous()
            and out.dim() == 3 and tuple(out.shape[:2]) == (f, r)):
        raise ValueError("out must be a contiguous cuda float32 [f, r, d] tensor")
    d = out.shape[2]
    dev = out.device
    role_d = torch.from_numpy(role).to(dev)
    worker_d = torch.from_numpy(worker).to(dev)
    need_alie = int((role == ROLE_ALIE).any())
    alie = torch.empty(d if need_alie else 1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    rc = _load().synth_fill_device(role_d.data_ptr(), worker_d.data_ptr(), f, r, d, dist, seed,
                                   alie_z, need_alie, alie.data_ptr(), out.data_ptr(), stream)
    if rc != 0:
        raise RuntimeError(f"synth_fill_device failed ({rc})")
    torch.cuda.current_stream().synchronize()
    del alie, role_d, worker_d
    return out


def generate(wl: Workload, subsets: np.ndarray, d: int | None = None, seed: int = SEED,
             **role_kw) -> tuple[np.ndarray, dict]:
    """A whole small input [f, r, d] and its attack description."""
    d = wl.d if d is None else d
    role, worker, A, D = make_roles(wl, subsets, seed, **role_kw)
    g = fill(role, worker, 0, d, wl.dist, seed, wl.alie_z)
    return g, {"role": role, "worker": worker, "A": A, "D": D}


def normal(seed: int, stream: int, sub: int, file: int, k: int) -> float:
    """The generator's standard normal deviate of one counter."""
    return float(_load().synth_normal(seed, stream, sub, file, k))


def log(x: float) -> float:
    """The generator's own natural logarithm (x > 0, normal)."""
    return float(_load().synth_log(x))


def fnv1a(buf: np.ndarray) -> int:
    buf = np.ascontiguousarray(buf)
    return int(_load().synth_fnv1a(buf.ctypes.data, buf.nbytes))
