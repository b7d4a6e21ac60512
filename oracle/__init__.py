"""OptCC oracle: plain, slow, obviously correct CPU reference.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke entry point and the
benchmark's CPU-baseline leg may import this package.  The product library
never imports, links or executes anything here, and this package imports
nothing from the product.

Parts (paper: "Don't Let a Few Network Failures Slow the Entire AllReduce"):

* ``Schedule`` / ``run`` / ``run_parallel`` / ``run_sampled``: the schedule built from the rules
  of Sec. 4.1-4.2, App. C (bubble filling) and App. D (several stragglers),
  executed serially step by step in plain C (``optcc_oracle.c``).
* ``brute_sum``: the definition of the result (Sec. 3, problem setting): the
  elementwise sum over ranks, in fp64 (int64 for int32, wrapped mod 2**32).
* ``provenance`` / ``provenance_steps``: the correctness conditions of Sec. 3 checked symbolically
  with contributor sets: a REDUCE never counts a rank twice, and at the end
  every rank holds the contribution of every rank exactly once.
* ``model``: the closed-form times and lower bounds, in exact rationals.
* ``timeline``: the plan's flows timed in the paper's network model, in
  exact rationals, and a validator of any timeline.
* ``closed_form``: every coordinate's final value written directly from the
  readings, without the step list, to check the step execution against.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "optcc_oracle.c")
_LIB = os.path.join(_HERE, "liboptcc_oracle.so")

DTYPES = {"f32": 0, "bf16": 1, "i32": 2, "f16": 3}
NP_DTYPES = {"f32": np.float32, "bf16": np.uint16, "i32": np.int32, "f16": np.uint16}
KINDS = {0: "ring", 1: "single_ge2", 2: "single_lt2", 3: "multi", 4: "servers"}
COPY, REDUCE = 0, 1
NUM_SLOTS = 6           # one GPU per server
NUM_SERVER_SLOTS = 12   # several GPUs per server

_lib = None


def build_lib() -> str:
    """Compile the oracle with plain gcc: no fast-math, no contraction."""
    cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-shared", "-fPIC", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build_lib()
        L = ctypes.CDLL(_LIB)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.orc_build.argtypes = [i32, vp, i64, i32, i32, i32, ctypes.POINTER(vp)]
        L.orc_build.restype = i32
        L.orc_build_servers.argtypes = [i32, i32, vp, i64, i32, i32, i32, ctypes.POINTER(vp)]
        L.orc_build_servers.restype = i32
        L.orc_free.argtypes = [vp]
        L.orc_info.argtypes = [vp, vp, vp, vp, vp]
        L.orc_segments.argtypes = [vp, vp, vp, vp]
        L.orc_steps.argtypes = [vp, vp, vp, vp]
        L.orc_run.argtypes = [vp, i32, vp, i32, i32]
        L.orc_run.restype = i32
        L.orc_run_parallel.argtypes = [vp, i32, vp, i32, i32, i32]
        L.orc_run_parallel.restype = i32
        L.orc_run_sampled.argtypes = [vp, i32, vp, vp, i64, i32, i32]
        L.orc_run_sampled.restype = i32
        L.orc_last_error.restype = ctypes.c_char_p
        L.orc_bf16_round_array.argtypes = [vp, vp, i64]
        L.orc_f16_round_array.argtypes = [vp, vp, i64]
        L.orc_f16_widen_array.argtypes = [vp, vp, i64]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"oracle status {status}: {msg}")
        self.status = status


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class Schedule:
    """The oracle's own schedule for (p, bandwidths, N, k); optionally only
    the steps of segments [seg_lo, seg_hi).  ``Schedule.servers`` builds the
    several-GPUs-per-server schedule (App. E)."""

    def __init__(self, p, bandwidths, n, k, seg_lo=0, seg_hi=0, _servers=None):
        L = lib()
        bw = np.ascontiguousarray(np.asarray(bandwidths, dtype=np.float64))
        h = ctypes.c_void_p()
        if _servers is None:
            if bw.shape != (p,):
                raise ValueError("need one bandwidth per rank")
            rc = L.orc_build(int(p), _ptr(bw), int(n), int(k), int(seg_lo), int(seg_hi),
                             ctypes.byref(h))
        else:
            q, g = _servers
            if bw.shape != (q,):
                raise ValueError("need one bandwidth per server")
            rc = L.orc_build_servers(int(q), int(g), _ptr(bw), int(n), int(k), int(seg_lo),
                                     int(seg_hi), ctypes.byref(h))
            p = q * g
        if rc != 0:
            raise OracleError(rc, L.orc_last_error().decode())
        self._h = h
        self._L = L  # the library that owns the handle frees it
        info = np.zeros(12, np.int64)
        ring = np.zeros(max(p, 1), np.int32)
        strag = np.zeros(max(p, 1), np.int32)
        ell = np.zeros(p, np.float64)
        L.orc_info(h, _ptr(info), _ptr(ring), _ptr(strag), _ptr(ell))
        self.p, self.k, self.m = int(info[0]), int(info[1]), int(info[2])
        self.kind = KINDS[int(info[3])]
        self.pp, self.n = int(info[4]), int(info[5])
        self.nsteps, self.npool = int(info[6]), int(info[7])
        self.g, self.q, self.nseg = int(info[8]), int(info[9]), int(info[10])
        self.num_slots = NUM_SERVER_SLOTS if self.g > 1 else NUM_SLOTS
        self.ring = ring[: self.pp].copy()
        self.stragglers = strag[: self.m].copy()
        self.ell = ell
        off = np.zeros(self.nseg, np.int64)
        ln = np.zeros(self.nseg, np.int64)
        p2p = np.zeros(self.nseg, np.int64)
        L.orc_segments(h, _ptr(off), _ptr(ln), _ptr(p2p))
        self.seg_off, self.seg_len, self.p2p_len = off, ln, p2p

    @classmethod
    def servers(cls, q, g, server_bandwidths, n, k, seg_lo=0, seg_hi=0):
        """q servers of g GPUs (ranks server-major), one bandwidth per server."""
        return cls(q * g, server_bandwidths, n, k, seg_lo, seg_hi, _servers=(q, g))

    def __del__(self):
        h = getattr(self, "_h", None)
        L = getattr(self, "_L", None)
        if h is not None and L is not None:
            L.orc_free(h)
            self._h = None

    def steps(self):
        """All steps in serial order as a list of dicts."""
        ints = np.zeros((max(self.nsteps, 1), 6), np.int32)
        offs = np.zeros((max(self.nsteps, 1), 3), np.int64)
        pool = np.zeros(max(self.npool, 1), np.int32)
        self._L.orc_steps(self._h, _ptr(ints), _ptr(offs), _ptr(pool))
        out = []
        for i in range(self.nsteps):
            slot, seg, sec, op, dst, nsrc = (int(v) for v in ints[i])
            at, off, ln = (int(v) for v in offs[i])
            out.append(dict(slot=slot, seg=seg, sec=sec, op=op, dst=dst,
                            srcs=[int(v) for v in pool[at:at + nsrc]], off=off, len=ln))
        return out

    def flows(self):
        """Point-to-point flows (Sec. 4.1: a flow moves one section between two
        ranks): one per (step, source)."""
        return [(st["slot"], src, st["dst"], st["off"], st["len"], st["op"])
                for st in self.steps() for src in st["srcs"]]


def run(sched: Schedule, dtype: str, bufs: np.ndarray, slot_lo=0, slot_hi=NUM_SERVER_SLOTS):
    """Execute the schedule in place on a C-contiguous [p, N] host array."""
    if not (bufs.flags.c_contiguous and bufs.shape == (sched.p, sched.n)
            and bufs.dtype == NP_DTYPES[dtype]):
        raise ValueError("bufs must be a C-contiguous [p, N] array of the dtype")
    ptrs = (ctypes.c_void_p * sched.p)(*[bufs[r].ctypes.data for r in range(sched.p)])
    rc = sched._L.orc_run(sched._h, DTYPES[dtype], ptrs, int(slot_lo), int(slot_hi))
    if rc != 0:
        raise OracleError(rc, sched._L.orc_last_error().decode())
    return bufs


def run_parallel(sched: Schedule, dtype: str, bufs: np.ndarray, threads: int,
                 slot_lo=0, slot_hi=NUM_SERVER_SLOTS):
    """``run`` on `threads` host threads (OpenMP over segments): the same
    bits as the serial execution, used to time the oracle on all cores."""
    if not (bufs.flags.c_contiguous and bufs.shape == (sched.p, sched.n)
            and bufs.dtype == NP_DTYPES[dtype]):
        raise ValueError("bufs must be a C-contiguous [p, N] array of the dtype")
    ptrs = (ctypes.c_void_p * sched.p)(*[bufs[r].ctypes.data for r in range(sched.p)])
    rc = sched._L.orc_run_parallel(sched._h, DTYPES[dtype], ptrs, int(slot_lo), int(slot_hi),
                                   int(threads))
    if rc != 0:
        raise OracleError(rc, sched._L.orc_last_error().decode())
    return bufs


def run_sampled(sched: Schedule, dtype: str, cols: np.ndarray, coords: np.ndarray,
                slot_lo=0, slot_hi=NUM_SERVER_SLOTS):
    """Execute the schedule at sorted coordinates only; cols is [p, S] and is
    updated in place."""
    coords = np.ascontiguousarray(coords, dtype=np.int64)
    if not (cols.flags.c_contiguous and cols.shape == (sched.p, coords.size)
            and cols.dtype == NP_DTYPES[dtype]):
        raise ValueError("cols must be a C-contiguous [p, S] array of the dtype")
    ptrs = (ctypes.c_void_p * sched.p)(*[cols[r].ctypes.data for r in range(sched.p)])
    rc = sched._L.orc_run_sampled(sched._h, DTYPES[dtype], ptrs, _ptr(coords), coords.size,
                               int(slot_lo), int(slot_hi))
    if rc != 0:
        raise OracleError(rc, sched._L.orc_last_error().decode())
    return cols


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even, through the oracle's C rule."""
    flat = np.ascontiguousarray(x, dtype=np.float32).ravel()
    out = np.empty(flat.size, np.uint16)
    lib().orc_bf16_round_array(_ptr(flat), _ptr(out), flat.size)
    return out.reshape(np.shape(x))


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> IEEE binary16 bits, round to nearest even, through the oracle's C rule."""
    flat = np.ascontiguousarray(x, dtype=np.float32).ravel()
    out = np.empty(flat.size, np.uint16)
    lib().orc_f16_round_array(_ptr(flat), _ptr(out), flat.size)
    return out.reshape(np.shape(x))


def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    """binary16 bits -> values, through the oracle's exact C widening."""
    flat = np.ascontiguousarray(bits, dtype=np.uint16).ravel()
    out = np.empty(flat.size, np.float32)
    lib().orc_f16_widen_array(_ptr(flat), _ptr(out), flat.size)
    return out.reshape(np.shape(bits)).astype(np.float64)


def values_f64(dtype: str, bufs: np.ndarray) -> np.ndarray:
    """The values a buffer of `dtype` holds, in fp64."""
    if dtype == "f32":
        return bufs.astype(np.float64)
    if dtype == "bf16":
        return bf16_to_f64(bufs)
    if dtype == "f16":
        return f16_to_f64(bufs)
    raise ValueError("integers are compared exactly")


def brute_sum(dtype: str, bufs: np.ndarray) -> np.ndarray:
    """The definition of the result: sum over ranks of every coordinate.
    fp64 for floating point; int32 wraps modulo 2**32 like two's complement."""
    if dtype in ("f32", "bf16", "f16"):
        return values_f64(dtype, bufs).sum(axis=0)
    s = bufs.astype(np.int64).sum(axis=0)
    return ((s + 2**31) % 2**32 - 2**31).astype(np.int32)


def abs_sum(dtype: str, bufs: np.ndarray) -> np.ndarray:
    if dtype == "i32":
        raise ValueError("no tolerance for integers: they are exact")
    return np.abs(values_f64(dtype, bufs)).sum(axis=0)


def tolerance(dtype: str, p: int, bufs: np.ndarray) -> np.ndarray:
    """Elementwise bound |y - sum| <= p u sum|x_i| with u = 2**-24 (fp32),
    2**-11 (fp16) or 2**-8 (bf16); it covers recursive summation with one
    rounding per add (no overflow)."""
    u = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}[dtype]
    return p * u * abs_sum(dtype, bufs)


def provenance(sched: Schedule, n_small: int | None = None):
    """Symbolic execution of a schedule with contributor sets; see
    ``provenance_steps``."""
    n = sched.n if n_small is None else n_small
    return provenance_steps(sched.p, n, sched.steps())


def provenance_steps(p: int, n: int, steps):
    """Symbolic execution with contributor sets (bitmasks over ranks) of a
    step list in serial order (dicts with op, dst, srcs, off, len).

    Returns (ok, message).  Checks, for every coordinate below n: a REDUCE
    adds sets that are disjoint from the destination's and from each other
    (nothing is counted twice), and at the end every rank holds all p
    contributions (Sec. 3: every rank ends with the sum of all inputs)."""
    full = (1 << p) - 1
    held = [[1 << r for _ in range(n)] for r in range(p)]
    for st in steps:
        for c in range(st["off"], min(st["off"] + st["len"], n)):
            if st["op"] == COPY:
                held[st["dst"]][c] = held[st["srcs"][0]][c]
            else:
                acc = held[st["dst"]][c]
                for s in st["srcs"]:
                    if acc & held[s][c]:
                        return False, f"double count at rank {st['dst']} coord {c}"
                    acc |= held[s][c]
                held[st["dst"]][c] = acc
    for r in range(p):
        for c in range(n):
            if held[r][c] != full:
                return False, f"rank {r} coord {c} misses contributions"
    return True, "ok"
