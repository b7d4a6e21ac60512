"""ctypes binding of liboptcc.so: the same entry points as include/optcc.h.

Argument marshalling only.  Every step of the schedule runs in the library's
HIP kernels; there is no Python or CPU fallback, and importing this module
fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liboptcc.so")

OPTCC_OK, OPTCC_EINVAL, OPTCC_ENOMEM, OPTCC_EUNSUPPORTED, OPTCC_EDEVICE = 0, -1, -2, -3, -4
OPTCC_NUM_SLOTS = 6
OPTCC_NUM_SERVER_SLOTS = 12
OPTCC_MAX_GPUS_PER_SERVER = 64
OPTCC_QUANTUM = 64
OPTCC_MAX_EMULATE_RANKS = 256
DTYPES = {"f32": 0, "bf16": 1, "i32": 2, "f16": 3}
KINDS = {0: "ring", 1: "single_ge2", 2: "single_lt2", 3: "multi", 4: "servers"}

EXPORTED = ("optcc_plan", "optcc_plan_servers", "optcc_plan_free", "optcc_allreduce_emulate",
            "optcc_allreduce_emulate_slots", "optcc_allreduce_emulate_noalloc",
            "optcc_model_time", "optcc_lower_bound",
            "optcc_lower_bound_servers", "optcc_last_error", "optcc_plan_info",
            "optcc_plan_segments", "optcc_plan_num_flows", "optcc_plan_get_flows",
            "optcc_plan_traffic", "optcc_plan_timeline", "optcc_narrow_f32")


class PlanInfo(ctypes.Structure):
    _fields_ = [("p", ctypes.c_int32), ("k", ctypes.c_int32), ("m", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("healthy", ctypes.c_int32),
                ("quantum", ctypes.c_int32), ("n", ctypes.c_int64),
                ("num_steps", ctypes.c_int64), ("num_flows", ctypes.c_int64),
                ("g", ctypes.c_int32), ("q", ctypes.c_int32),
                ("num_segments", ctypes.c_int32), ("num_slots", ctypes.c_int32)]


FLOW_DTYPE = np.dtype([("slot", np.int32), ("segment", np.int32), ("section", np.int32),
                       ("op", np.int32), ("src", np.int32), ("dst", np.int32),
                       ("stage", np.int32), ("hop", np.int32),
                       ("step", np.int64), ("offset", np.int64), ("length", np.int64)])
# the paper's stages (optcc_flow_t.stage)
STAGE_NAMES = {1: "S1", 2: "S2", 3: "S3", 4: "S4", 5: "N1", 6: "N2", 7: "N3", 8: "N4"}


class OptccError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"optcc status {status}: {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2606_01680_amd.build`")
    # One HIP runtime per process: torch ships its own libamdhip64 with the
    # same soname as the system one the library is linked against, and the
    # first one loaded serves everybody.  Load torch first, so that the
    # library runs on the runtime that owns torch's device memory and streams.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - plain C-ABI use without torch
        pass
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
    L.optcc_plan.argtypes = [i32, vp, i64, i32, ctypes.POINTER(vp)]
    L.optcc_plan.restype = i32
    L.optcc_plan_servers.argtypes = [i32, i32, vp, i64, i32, ctypes.POINTER(vp)]
    L.optcc_plan_servers.restype = i32
    L.optcc_lower_bound_servers.argtypes = [i32, i32, vp, i64]
    L.optcc_lower_bound_servers.restype = dbl
    L.optcc_plan_free.argtypes = [vp]
    L.optcc_plan_free.restype = None
    L.optcc_allreduce_emulate.argtypes = [vp, i32, i64, i32, vp, vp]
    L.optcc_allreduce_emulate.restype = i32
    L.optcc_allreduce_emulate_slots.argtypes = [vp, i32, i64, i32, vp, i32, i32, i32, vp]
    L.optcc_allreduce_emulate_slots.restype = i32
    L.optcc_allreduce_emulate_noalloc.argtypes = [vp, i32, i64, i32, vp, vp]
    L.optcc_allreduce_emulate_noalloc.restype = i32
    L.optcc_model_time.argtypes = [vp, vp]
    L.optcc_model_time.restype = dbl
    L.optcc_lower_bound.argtypes = [i32, vp, i64]
    L.optcc_lower_bound.restype = dbl
    L.optcc_last_error.argtypes = []
    L.optcc_last_error.restype = ctypes.c_char_p
    L.optcc_plan_info.argtypes = [vp, ctypes.POINTER(PlanInfo), vp, vp, vp]
    L.optcc_plan_info.restype = i32
    L.optcc_plan_segments.argtypes = [vp, vp, vp, vp]
    L.optcc_plan_segments.restype = i32
    L.optcc_plan_num_flows.argtypes = [vp]
    L.optcc_plan_num_flows.restype = i64
    L.optcc_plan_get_flows.argtypes = [vp, vp, i64]
    L.optcc_plan_get_flows.restype = i64
    L.optcc_plan_traffic.argtypes = [vp, i32, i32, i32, i32, ctypes.POINTER(i64),
                                     ctypes.POINTER(i64)]
    L.optcc_plan_traffic.restype = i32
    L.optcc_plan_timeline.argtypes = [vp, vp, vp, i64, ctypes.POINTER(dbl)]
    L.optcc_plan_timeline.restype = i32
    L.optcc_narrow_f32.argtypes = [vp, vp, i64, i32, vp]
    L.optcc_narrow_f32.restype = i32
    # the HIP runtime the library is linked against (found through its handle)
    L.hipStreamIsCapturing.argtypes = [vp, ctypes.POINTER(i32)]
    L.hipStreamIsCapturing.restype = i32
    return L


_lib = _load()


def lib():
    return _lib


def optcc_last_error() -> str:
    return _lib.optcc_last_error().decode()


def _check(rc):
    if rc < 0:
        raise OptccError(rc, optcc_last_error())
    return rc


def _f64(a, p):
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    if arr.shape != (p,):
        raise ValueError("need one bandwidth per rank")
    return arr


class Plan:
    """Owner of an optcc_plan_t (freed with the object)."""

    def __init__(self, handle):
        self._h = handle
        info = PlanInfo()
        _check(_lib.optcc_plan_info(self._h, ctypes.byref(info), None, None, None))
        self.p, self.k, self.m = info.p, info.k, info.m
        self.kind = KINDS[info.kind]
        self.healthy, self.n = info.healthy, info.n
        self.num_steps, self.num_flows = info.num_steps, info.num_flows
        self.g, self.q = info.g, info.q
        self.num_segments, self.num_slots = info.num_segments, info.num_slots
        ring = np.zeros(max(self.healthy, 1), np.int32)
        strag = np.zeros(max(self.m, 1), np.int32)
        ell = np.zeros(self.p, np.float64)
        _check(_lib.optcc_plan_info(self._h, ctypes.byref(info), ring.ctypes.data,
                                    strag.ctypes.data, ell.ctypes.data))
        self.ring = ring[: self.healthy].copy()
        self.stragglers = strag[: self.m].copy()
        self.slowdowns = ell

    @property
    def handle(self):
        return self._h

    def segments(self):
        off = np.zeros(self.num_segments, np.int64)
        ln = np.zeros(self.num_segments, np.int64)
        p2p = np.zeros(self.num_segments, np.int64)
        _check(_lib.optcc_plan_segments(self._h, off.ctypes.data, ln.ctypes.data, p2p.ctypes.data))
        return off, ln, p2p

    def flows(self) -> np.ndarray:
        n = _check(_lib.optcc_plan_num_flows(self._h))
        out = np.zeros(max(n, 1), FLOW_DTYPE)
        got = _check(_lib.optcc_plan_get_flows(self._h, out.ctypes.data, n))
        assert got == n
        return out[:n]

    def traffic(self, dtype: str, slot_begin=0, slot_end=None, launches=1):
        slot_end = self.num_slots if slot_end is None else slot_end
        r, w = ctypes.c_int64(), ctypes.c_int64()
        _check(_lib.optcc_plan_traffic(self._h, DTYPES[dtype], slot_begin, slot_end, launches,
                                       ctypes.byref(r), ctypes.byref(w)))
        return r.value, w.value

    def timeline(self, with_flows=True):
        """(makespan, start[], finish[]) of the evaluated schedule."""
        n = self.num_flows if with_flows else 0
        st = np.zeros(max(n, 1), np.float64)
        fi = np.zeros(max(n, 1), np.float64)
        mk = ctypes.c_double()
        _check(_lib.optcc_plan_timeline(self._h, st.ctypes.data, fi.ctypes.data, n,
                                        ctypes.byref(mk)))
        return mk.value, st[:n], fi[:n]

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:  # _lib is gone at interpreter exit
            _lib.optcc_plan_free(h)
            self._h = None


def optcc_plan(p: int, link_bandwidths, N: int, n_chunks: int) -> Plan:
    bw = _f64(link_bandwidths, p)
    h = ctypes.c_void_p()
    _check(_lib.optcc_plan(int(p), bw.ctypes.data, int(N), int(n_chunks), ctypes.byref(h)))
    return Plan(h)


def optcc_plan_servers(q: int, g: int, server_bandwidths, N: int, n_chunks: int) -> Plan:
    """q servers of g GPUs each (ranks server-major), one bandwidth per server."""
    bw = _f64(server_bandwidths, q)
    h = ctypes.c_void_p()
    _check(_lib.optcc_plan_servers(int(q), int(g), bw.ctypes.data, int(N), int(n_chunks),
                                   ctypes.byref(h)))
    return Plan(h)


# Plans whose emulation calls were captured into a HIP graph.  A graph keeps
# the addresses of the plan's device tables, so such a plan is kept alive
# (never freed by garbage collection) until release_captured_plans() is
# called, which the caller does once every graph that captured it has been
# destroyed.
_captured_plans: dict = {}


def release_captured_plans() -> None:
    """Drop the references kept for plans used under graph capture.  Call
    it only after destroying every HIP graph that captured one of them."""
    _captured_plans.clear()


def optcc_plan_free(plan: Plan) -> None:
    if id(plan) in _captured_plans:
        raise RuntimeError("this plan was used inside a HIP graph capture: destroy the graphs "
                           "that captured it and call release_captured_plans() first")
    h = plan._h
    plan._h = None
    if h is not None:
        _lib.optcc_plan_free(h)


ESIZE = {"f32": 4, "bf16": 2, "i32": 4, "f16": 2}


def _ptr_array(bufs, p, n=None, dtype=None):
    """bufs: a [p, N] device tensor or a sequence of p device tensors (or raw
    device addresses).  Tensors must hold N elements per rank of the element
    size of `dtype`: the library reads and writes N elements at each address
    and cannot see allocation sizes."""
    try:
        import torch
    except ImportError:  # pragma: no cover
        torch = None

    if dtype is not None and dtype not in ESIZE:
        raise ValueError(f"unknown dtype {dtype!r}")

    def check(t, what):
        if dtype is not None and t.element_size() != ESIZE[dtype]:
            raise ValueError(f"{what} has {t.element_size()}-byte elements, dtype {dtype!r} "
                             f"needs {ESIZE[dtype]}")
        if n is not None and t.shape[-1] != n:
            raise ValueError(f"{what} holds {t.shape[-1]} elements per rank, N is {n}")

    if torch is not None and isinstance(bufs, torch.Tensor):
        if bufs.dim() != 2 or bufs.shape[0] != p or not bufs.is_contiguous():
            raise ValueError("bufs must be a contiguous [p, N] tensor")
        if not bufs.is_cuda:
            raise ValueError("bufs must live on the GPU")
        check(bufs, "bufs")
        base, stride = bufs.data_ptr(), bufs.stride(0) * bufs.element_size()
        ptrs = [base + r * stride for r in range(p)]
    else:
        if len(bufs) != p:
            raise ValueError("need p buffers")
        ptrs = []
        for r, b in enumerate(bufs):
            if torch is not None and isinstance(b, torch.Tensor):
                if not b.is_cuda or not b.is_contiguous() or b.dim() != 1:
                    raise ValueError("every buffer must be a contiguous 1-D GPU tensor")
                check(b, f"bufs[{r}]")
                ptrs.append(b.data_ptr())
            else:
                ptrs.append(int(b))
    return (ctypes.c_void_p * p)(*ptrs)


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def _keep_if_captured(plan: Plan, stream: int) -> None:
    """Keep `plan` alive if the call just made on `stream` was captured."""
    status = ctypes.c_int(0)
    if _lib.hipStreamIsCapturing(ctypes.c_void_p(stream), ctypes.byref(status)) == 0 \
            and status.value != 0:
        _captured_plans[id(plan)] = plan


def optcc_allreduce_emulate(bufs, p: int, N: int, dtype: str, plan: Plan, stream=None) -> None:
    """Run the whole schedule in place (one fused launch) on `stream`
    (default: torch's current stream).  A call captured into a HIP graph
    keeps `plan` alive (see release_captured_plans)."""
    arr = _ptr_array(bufs, p, int(N), dtype)
    st = _stream(stream)
    _check(_lib.optcc_allreduce_emulate(arr, int(p), int(N), DTYPES[dtype], plan.handle,
                                        ctypes.c_void_p(st)))
    _keep_if_captured(plan, st)


def optcc_allreduce_emulate_noalloc(bufs, p: int, N: int, dtype: str, plan: Plan,
                                    stream=None) -> None:
    """optcc_allreduce_emulate without any device allocation: the plan's
    tables are staged in the library's static per-GPU array on `stream`
    (calls on one GPU that overlap in time race)."""
    arr = _ptr_array(bufs, p, int(N), dtype)
    st = _stream(stream)
    _check(_lib.optcc_allreduce_emulate_noalloc(arr, int(p), int(N), DTYPES[dtype], plan.handle,
                                                ctypes.c_void_p(st)))
    _keep_if_captured(plan, st)


def optcc_allreduce_emulate_slots(bufs, p: int, N: int, dtype: str, plan: Plan, slot_begin: int,
                                  slot_end: int, launches: int = 1, stream=None) -> None:
    arr = _ptr_array(bufs, p, int(N), dtype)
    st = _stream(stream)
    _check(_lib.optcc_allreduce_emulate_slots(arr, int(p), int(N), DTYPES[dtype], plan.handle,
                                              int(slot_begin), int(slot_end), int(launches),
                                              ctypes.c_void_p(st)))
    _keep_if_captured(plan, st)


def optcc_model_time(plan: Plan, link_bandwidths=None) -> float:
    """link_bandwidths: one per rank, or one per server for a server plan."""
    nb = plan.q if plan.kind == "servers" else plan.p
    bw = None if link_bandwidths is None else _f64(link_bandwidths, nb)
    t = _lib.optcc_model_time(plan.handle, None if bw is None else bw.ctypes.data)
    if math.isnan(t):
        raise OptccError(OPTCC_EINVAL, optcc_last_error())
    return t


def optcc_lower_bound(p: int, link_bandwidths, N: int) -> float:
    bw = np.ascontiguousarray(np.asarray(link_bandwidths, dtype=np.float64))
    if bw.shape != (p,):
        raise ValueError("need one bandwidth per rank")
    t = _lib.optcc_lower_bound(int(p), bw.ctypes.data, int(N))
    if math.isnan(t):
        raise OptccError(OPTCC_EINVAL, optcc_last_error())
    return t


def optcc_lower_bound_servers(q: int, g: int, server_bandwidths, N: int) -> float:
    bw = _f64(server_bandwidths, q)
    t = _lib.optcc_lower_bound_servers(int(q), int(g), bw.ctypes.data, int(N))
    if math.isnan(t):
        raise OptccError(OPTCC_EINVAL, optcc_last_error())
    return t


def optcc_plan_timeline(plan: Plan):
    return plan.timeline()


def optcc_narrow_f32(src, dst, dtype: str, stream=None) -> None:
    """Round the fp32 device tensor `src` into the 16-bit device tensor `dst`
    (same length) with the executor's per-step rounding rule for `dtype`
    ("bf16" or "f16")."""
    if dtype not in ("bf16", "f16"):
        raise ValueError("dtype must be 'bf16' or 'f16'")
    if src.element_size() != 4 or dst.element_size() != 2:
        raise ValueError("src must hold 4-byte and dst 2-byte elements")
    if not (src.is_cuda and dst.is_cuda and src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("src and dst must be contiguous GPU tensors")
    if src.numel() != dst.numel():
        raise ValueError("src and dst must have the same length")
    _check(_lib.optcc_narrow_f32(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                                 int(src.numel()), DTYPES[dtype],
                                 ctypes.c_void_p(_stream(stream))))
