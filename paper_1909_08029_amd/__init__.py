"""Python binding of librip (P-Reduce with fused local update on one MI355X).

Argument marshalling only: every step of the hot path runs in librip's HIP
kernels; torch supplies device memory (``data_ptr``) and streams.  The names
follow the C ABI in include/rip.h, which documents each call.  Importing this
module loads ``librip.so`` and raises if it is missing -- there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import functools
import os
from typing import List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librip.so")

RIP_OK = 0
RIP_E_INVAL = -1
RIP_E_ALIGN = -2
RIP_E_OVERLAP = -3
RIP_E_UNSUPPORTED = -4
RIP_E_HIP = -5
RIP_E_NOMEM = -6

RIP_FP32 = 0
RIP_BF16 = 1
RIP_MAX_REPLICAS = 256

SCHED_TABLE = 0
SCHED_STATIC = 1
SCHED_RANDOM_GB = 2
SCHED_GD = 3
SCHED_SCRIPTED = 4
SCHED_RULE = 5
SCHED_INTER_INTRA = 6
SCHED_ADPSGD = 7

_i32p = ctypes.POINTER(ctypes.c_int32)


class RipError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"librip error {code}: {message}")
        self.code = code


class SchedCfg(ctypes.Structure):
    _fields_ = [
        ("n_workers", ctypes.c_int32), ("mode", ctypes.c_int32), ("seed", ctypes.c_uint64),
        ("group_size", ctypes.c_int32), ("period", ctypes.c_int32),
        ("kmin", ctypes.c_int32), ("kmax", ctypes.c_int32), ("c_thres", ctypes.c_int32),
        ("n_nodes", ctypes.c_int32),
        ("row_offsets", _i32p), ("group_offsets", _i32p), ("members", _i32p),
        ("n_groups", ctypes.c_int32),
    ]


class WorkerState(ctypes.Structure):
    _fields_ = [("requests", ctypes.c_int64), ("syncs", ctypes.c_int64),
                ("skips", ctypes.c_int64), ("waiting", ctypes.c_int32),
                ("gb_depth", ctypes.c_int32)]


class Sgd(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("nesterov", ctypes.c_int32)]


@functools.lru_cache(maxsize=64)
def _sgd(lr: float, momentum: float, weight_decay: float, nesterov: bool) -> Sgd:
    """The optimizer struct for these values, built once (the library only
    reads it), so a loop of steps does not rebuild it every call."""
    return Sgd(lr, momentum, weight_decay, int(bool(nesterov)))


def _load():
    # torch ships its own HIP runtime.  Importing it first makes librip bind
    # to that same runtime (the soname matches); loading librip first would
    # pull in a second HIP runtime from /opt/rocm and the two do not mix.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp = ctypes.c_void_p
    sigs = {
        "rip_last_error": (ctypes.c_char_p, []),
        "rip_abi_version": (ctypes.c_int32, []),
        "rip_last_launch_count": (ctypes.c_int32, []),
        "rip_sched_create": (ctypes.c_int32, [ctypes.POINTER(SchedCfg), ctypes.POINTER(vp)]),
        "rip_sched_destroy": (None, [vp]),
        "rip_schedule_groups": (ctypes.c_int32, [vp, ctypes.c_int64, ctypes.c_char_p, _i32p,
                                                 _i32p, _i32p, _i32p, _i32p]),
        "rip_sched_worker": (ctypes.c_int32, [vp, ctypes.c_int32, ctypes.POINTER(WorkerState)]),
        "rip_replicas_create": (ctypes.c_int32, [
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
            ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp)]),
        "rip_replicas_create_noalloc": (ctypes.c_int32, [
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
            ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp)]),
        "rip_replicas_destroy": (None, [vp]),
        "rip_local_step": (ctypes.c_int32, [vp, _i32p, ctypes.c_int32, ctypes.POINTER(Sgd), vp]),
        "rip_preduce": (ctypes.c_int32, [vp, _i32p, _i32p, ctypes.c_int32, _i32p,
                                         ctypes.c_int32, ctypes.POINTER(Sgd), vp]),
        "rip_step": (ctypes.c_int32, [vp, vp, ctypes.c_int64, ctypes.c_char_p,
                                      ctypes.POINTER(Sgd), vp, _i32p, _i32p, _i32p, _i32p,
                                      _i32p]),
        "rip_set_max_blocks": (ctypes.c_int32, [ctypes.c_int32]),
        "rip_set_blocks_per_cu": (ctypes.c_int32, [ctypes.c_int32]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def _check(rc: int):
    if rc != RIP_OK:
        raise RipError(rc, lib.rip_last_error().decode())


def _i32_array(values: Sequence[int]):
    arr = (ctypes.c_int32 * max(1, len(values)))(*values)
    return arr


def _csr(groups: Sequence[Sequence[int]]):
    offsets, members = [0], []
    for g in groups:
        members.extend(int(m) for m in g)
        offsets.append(len(members))
    return _i32_array(offsets), _i32_array(members)


# ---------------------------------------------------------------------------
# scheduler
# ---------------------------------------------------------------------------
class Scheduler:
    """Owns a ``rip_sched`` handle (see rip_sched_create in include/rip.h)."""

    def __init__(self, n_workers: int, mode: int, seed: int = 0, group_size: int = 0,
                 period: int = 4, kmin: int = 2, kmax: int = 2, c_thres: int = 0,
                 n_nodes: int = 0, table: Optional[Sequence[Sequence[Sequence[int]]]] = None,
                 script: Optional[Sequence[Sequence[int]]] = None):
        self.n = n_workers
        cfg = SchedCfg(n_workers=n_workers, mode=mode, seed=seed & (2 ** 64 - 1),
                       group_size=group_size, period=period, kmin=kmin, kmax=kmax,
                       c_thres=c_thres, n_nodes=n_nodes)
        keep = []
        if table is not None:
            rows = [0]
            flat = []
            for row in table:
                flat.extend(row)
                rows.append(len(flat))
            ro = _i32_array(rows)
            go, mem = _csr(flat)
            cfg.row_offsets, cfg.group_offsets, cfg.members = (
                ctypes.cast(ro, _i32p), ctypes.cast(go, _i32p), ctypes.cast(mem, _i32p))
            cfg.period, cfg.n_groups = len(table), len(flat)
            keep += [ro, go, mem]
        if script is not None:
            go, mem = _csr(script)
            cfg.group_offsets, cfg.members = ctypes.cast(go, _i32p), ctypes.cast(mem, _i32p)
            cfg.n_groups = len(script)
            keep += [go, mem]
        h = ctypes.c_void_p()
        _check(lib.rip_sched_create(ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h
        self._destroy = lib.rip_sched_destroy  # still reachable at interpreter exit
        n = n_workers
        self._act = (ctypes.c_int32 * n)()
        self._off = (ctypes.c_int32 * (n + 1))()
        self._mem = (ctypes.c_int32 * n)()
        self._na = ctypes.c_int32()
        self._ng = ctypes.c_int32()

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    __del__ = close

    def worker(self, i: int) -> WorkerState:
        ws = WorkerState()
        _check(lib.rip_sched_worker(self._h, i, ctypes.byref(ws)))
        return ws


def rip_schedule_groups(sched: Scheduler, step: int, eligible: Optional[Sequence[bool]] = None
                        ) -> Tuple[List[int], List[Tuple[int, ...]]]:
    """One step of group generation.  Returns (active ids, groups)."""
    el = None if eligible is None else bytes(1 if e else 0 for e in eligible)
    if el is not None and len(el) != sched.n:
        raise ValueError("eligible must have one entry per worker")
    _check(lib.rip_schedule_groups(sched._h, step, el, sched._act, ctypes.byref(sched._na),
                                   sched._off, sched._mem, ctypes.byref(sched._ng)))
    active = list(sched._act[:sched._na.value])
    off = sched._off[:sched._ng.value + 1]
    groups = [tuple(sched._mem[off[g]:off[g + 1]]) for g in range(sched._ng.value)]
    return active, groups


# ---------------------------------------------------------------------------
# replicas and the fused step
# ---------------------------------------------------------------------------
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return RIP_FP32
    if t.dtype == torch.bfloat16:
        return RIP_BF16
    raise TypeError(f"unsupported storage dtype {t.dtype}")


class Replicas:
    """Registers N replicas x S segments of device buffers (torch tensors,
    contiguous, on the current device).  ``param[r][s]`` is segment s of
    replica r; ``grad`` and ``mom`` have the same layout or are None.  The
    tensors must outlive the handle and any work enqueued with it.
    ``noalloc=True`` registers through rip_replicas_create_noalloc (the
    device's one fixed table array; see include/rip.h)."""

    def __init__(self, param, grad=None, mom=None, noalloc=False):
        n = len(param)
        S = len(param[0])
        dtype = _dtype_code(param[0][0])
        numel = [param[0][s].numel() for s in range(S)]
        for kind in (param, grad, mom):
            if kind is None:
                continue
            if len(kind) != n or any(len(row) != S for row in kind):
                raise ValueError("every tensor list must be N x S")
            for row in kind:
                for s, t in enumerate(row):
                    if t.numel() != numel[s] or not t.is_contiguous() or not t.is_cuda:
                        raise ValueError("segments must be contiguous CUDA tensors of equal sizes")
                    if _dtype_code(t) != dtype:
                        raise ValueError("all buffers must share one storage dtype")

        def ptrs(kind):
            if kind is None:
                return None
            return (ctypes.c_void_p * (n * S))(*[kind[r][s].data_ptr()
                                                 for r in range(n) for s in range(S)])

        self._keep = [ptrs(param), ptrs(grad), ptrs(mom)]
        self.n, self.S, self.dtype, self.numel = n, S, dtype, numel
        self.tensors = (param, grad, mom)
        h = ctypes.c_void_p()
        create = lib.rip_replicas_create_noalloc if noalloc else lib.rip_replicas_create
        _check(create(n, S, dtype, (ctypes.c_int64 * S)(*numel), self._keep[0], self._keep[1],
                      self._keep[2], ctypes.byref(h)))
        self._h = h
        self._destroy = lib.rip_replicas_destroy  # still reachable at interpreter exit

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    __del__ = close


def _stream_ptr(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def rip_local_step(rep: Replicas, active: Sequence[int], lr: float, momentum: float = 0.0,
                   stream=None, weight_decay: float = 0.0, nesterov: bool = False) -> None:
    """Step 2 of Fig. 4 for the listed workers (see include/rip.h)."""
    act = _i32_array(list(active))
    sgd = _sgd(lr, momentum, weight_decay, bool(nesterov))
    _check(lib.rip_local_step(rep._h, act, len(active), ctypes.byref(sgd),
                              _stream_ptr(stream)))


def rip_preduce(rep: Replicas, groups: Sequence[Sequence[int]], active: Sequence[int] = (),
                lr: Optional[float] = None, momentum: float = 0.0, stream=None,
                weight_decay: float = 0.0, nesterov: bool = False) -> None:
    """Fused local update of ``active`` and P-Reduce of the disjoint ``groups``
    in one launch (see include/rip.h).  ``lr=None`` is pure P-Reduce."""
    off, mem = _csr(groups)
    act = _i32_array(list(active))
    sgd = None if lr is None else ctypes.byref(
        _sgd(lr, momentum, weight_decay, bool(nesterov)))
    _check(lib.rip_preduce(rep._h, off, mem, len(groups), act, len(active), sgd,
                           _stream_ptr(stream)))


def rip_step(sched: Scheduler, rep: Replicas, step: int, lr: float, momentum: float = 0.0,
             eligible: Optional[Sequence[bool]] = None, stream=None, weight_decay: float = 0.0,
             nesterov: bool = False) -> Tuple[List[int], List[Tuple[int, ...]]]:
    """Group generation for ``step`` and the fused launch in one call (see
    include/rip.h).  Returns (active ids, groups) as rip_schedule_groups."""
    el = None if eligible is None else bytes(1 if e else 0 for e in eligible)
    if el is not None and len(el) != sched.n:
        raise ValueError("eligible must have one entry per worker")
    sgd = _sgd(lr, momentum, weight_decay, bool(nesterov))
    _check(lib.rip_step(sched._h, rep._h, step, el, ctypes.byref(sgd), _stream_ptr(stream),
                        sched._act, ctypes.byref(sched._na), sched._off, sched._mem,
                        ctypes.byref(sched._ng)))
    active = list(sched._act[:sched._na.value])
    off = sched._off[:sched._ng.value + 1]
    groups = [tuple(sched._mem[off[g]:off[g + 1]]) for g in range(sched._ng.value)]
    return active, groups


def rip_set_max_blocks(n: int) -> None:
    _check(lib.rip_set_max_blocks(n))


def rip_set_blocks_per_cu(n: int) -> None:
    _check(lib.rip_set_blocks_per_cu(n))


def abi_version() -> int:
    return lib.rip_abi_version()


def rip_last_launch_count() -> int:
    """Kernel launches the calling thread's last step call enqueued (0-2)."""
    return lib.rip_last_launch_count()
