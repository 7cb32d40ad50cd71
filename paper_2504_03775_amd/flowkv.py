"""ctypes binding to ``libflowkv.so`` (the C ABI in ``include/flowkv.h``).

Argument marshalling only: every step -- allocation, alignment, the copy,
decode attention, the scheduler's evaluation and routing -- runs in the
native library.  PyTorch supplies device memory and streams.  The functions
carry the C names; ``Allocator``, ``Scheduler`` and ``KVPool`` are thin
owners of a handle or of a pool descriptor.

If the library is missing this module raises on import: there is no other
code path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflowkv.so")

OK, EINVAL, ENOSPC, ERANGE, EDUP, ECAP, EHIP, ENOMEM = 0, -1, -2, -3, -4, -5, -6, -7
POLICY_SEGMENT, POLICY_FIFO_SORTED, POLICY_FIFO_SHUFFLED = 0, 1, 2
LAYOUT_LAYER_MAJOR, LAYOUT_BLOCK_MAJOR = 0, 1
MAX_LAYERS = 128
INLINE_RUNS = 64  # plan records flowkv_transfer_inline carries in the kernel arguments
INLINE_RUNS_BLOCK_MAJOR = 300  # ... between two block-major pools, in the planner's form
INLINE_LAYERS = 32  # pools of at most this many layers ...
INLINE_RUNS_LAYER_MAJOR = 264  # ... carry this many planner-form records when one is layer-major

SEGMENT_DTYPE = np.dtype([("src_block", "<i4"), ("dst_block", "<i4"),
                          ("n_blocks", "<i4"), ("first", "<i4")])


class FlowKVError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = _lib.flowkv_last_error().decode() or _lib.flowkv_strerror(code).decode()
        super().__init__(f"{where}: {_lib.flowkv_strerror(code).decode()} ({code}): {msg}")


class flowkv_segment(ctypes.Structure):
    _fields_ = [("src_block", ctypes.c_int32), ("dst_block", ctypes.c_int32),
                ("n_blocks", ctypes.c_int32), ("first", ctypes.c_int32)]


class flowkv_alloc_stats(ctypes.Structure):
    _fields_ = [("free_blocks", ctypes.c_int64), ("free_segments", ctypes.c_int64),
                ("largest_free", ctypes.c_int64)]


class flowkv_pool(ctypes.Structure):
    _fields_ = [("layout", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("num_blocks", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("chunk_bytes", ctypes.c_int64), ("layer_base", ctypes.POINTER(ctypes.c_void_p))]


class flowkv_launch_config(ctypes.Structure):
    _fields_ = [("threads", ctypes.c_int32), ("unroll", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("cache", ctypes.c_int32), ("order", ctypes.c_int32)]


class flowkv_sched_params(ctypes.Structure):
    _fields_ = [("window", ctypes.c_int32), ("scale_after", ctypes.c_int32),
                ("scale", ctypes.c_double * 12), ("w_prefill", ctypes.c_double * 8),
                ("w_decode", ctypes.c_double * 8), ("eps_p_low", ctypes.c_double),
                ("eps_d_low", ctypes.c_double), ("eps_p_high", ctypes.c_double),
                ("eps_d_high", ctypes.c_double), ("idle_threshold", ctypes.c_double),
                ("eps_p_min", ctypes.c_double), ("eps_d_min", ctypes.c_double)]


class flowkv_sched_result(ctypes.Structure):
    _fields_ = [("scenario", ctypes.c_int32), ("n_idle", ctypes.c_int32),
                ("switch_to", ctypes.c_int32), ("scale_prefill", ctypes.c_int32),
                ("scale_decode", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("c_prefill", ctypes.c_double), ("c_decode", ctypes.c_double)]


_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)
_F64P = ctypes.POINTER(ctypes.c_double)
_SEGP = ctypes.POINTER(flowkv_segment)
_POOLP = ctypes.POINTER(flowkv_pool)

# name -> (restype, argtypes); the exported symbol set of include/flowkv.h
SIGNATURES = {
    "flowkv_allocator_create": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64,
                                               ctypes.POINTER(ctypes.c_void_p)]),
    "flowkv_allocator_destroy": (None, [ctypes.c_void_p]),
    "flowkv_alloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]),
    "flowkv_free": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]),
    "flowkv_mark_used": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]),
    "flowkv_allocator_stats": (ctypes.c_int, [ctypes.c_void_p,
                                              ctypes.POINTER(flowkv_alloc_stats)]),
    "flowkv_plan": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_int64, _I64P]),
    "flowkv_plan_batch": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64, _I64P]),
    "flowkv_transfer": (ctypes.c_int, [_POOLP, _POOLP, ctypes.c_void_p, ctypes.c_int64,
                                       ctypes.c_int64, ctypes.c_void_p]),
    "flowkv_transfer_ex": (ctypes.c_int, [_POOLP, _POOLP, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.POINTER(flowkv_launch_config),
                                          ctypes.c_void_p]),
    "flowkv_transfer_inline": (ctypes.c_int, [_POOLP, _POOLP, ctypes.c_void_p, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.POINTER(flowkv_launch_config),
                                              ctypes.c_void_p]),
    "flowkv_inline_capacity": (ctypes.c_int, [_POOLP, _POOLP, _I64P]),
    "flowkv_transfer_request": (ctypes.c_int, [_POOLP, _POOLP, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_int32,
                                               ctypes.POINTER(flowkv_launch_config), _I64P,
                                               ctypes.c_void_p]),
    "flowkv_transfer_layers": (ctypes.c_int, [_POOLP, _POOLP, ctypes.c_void_p, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.POINTER(flowkv_launch_config),
                                              ctypes.c_void_p]),
    "flowkv_decode_attention_split": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32,
                                                     ctypes.POINTER(ctypes.c_int32)]),
    "flowkv_decode_attention_workspace": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32,
                                                         ctypes.c_int32, ctypes.c_int32,
                                                         ctypes.c_int32, _I64P]),
    "flowkv_decode_attention": (ctypes.c_int, [_POOLP, ctypes.c_int32, ctypes.c_void_p,
                                               ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                               ctypes.c_float,
                                               ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_int64, ctypes.c_void_p]),
    "flowkv_decode_attention_noalloc": (ctypes.c_int, [_POOLP, ctypes.c_int32, ctypes.c_void_p,
                                                       ctypes.c_int32, ctypes.c_int32,
                                                       ctypes.c_int32, ctypes.c_int32,
                                                       ctypes.c_void_p, ctypes.c_int32,
                                                       ctypes.c_void_p, ctypes.c_void_p,
                                                       ctypes.c_int32,
                                                       ctypes.c_float, ctypes.c_int32,
                                                       ctypes.c_void_p, ctypes.c_void_p]),
    "flowkv_sched_create": (ctypes.c_int, [ctypes.POINTER(flowkv_sched_params), ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]),
    "flowkv_sched_destroy": (None, [ctypes.c_void_p]),
    "flowkv_sched_set_role": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]),
    "flowkv_sched_observe": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "flowkv_sched_evaluate": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(flowkv_sched_result),
                                             ctypes.c_void_p, ctypes.c_void_p]),
    "flowkv_sched_route": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, _I32P, _I32P]),
    "flowkv_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "flowkv_last_error": (ctypes.c_char_p, []),
}


def _hip_runtimes_loaded():
    try:
        maps = open("/proc/self/maps").read()
    except OSError:
        return []
    return sorted({ln.split()[-1] for ln in maps.splitlines() if "libamdhip64" in ln})


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2504_03775_amd.build.build() "
                          "(or __graft_entry__.build()) first")
    # The library must share PyTorch's HIP runtime: device pointers and stream
    # handles come from torch.  Importing torch first loads its runtime, whose
    # soname (libamdhip64.so.7) then satisfies the library's dependency; loading
    # the library first would pull in a second runtime next to torch's.
    import torch  # noqa: F401

    lib = ctypes.CDLL(LIB_PATH)
    rts = _hip_runtimes_loaded()
    if len(rts) > 1:
        raise ImportError(f"two HIP runtimes loaded in one process: {rts}")
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib():
    return _lib


def _check(rc: int, where: str):
    if rc != OK:
        raise FlowKVError(rc, where)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: np.ndarray) -> int:
    """The array's address, for a c_void_p argument (a typed ctypes pointer
    costs several microseconds per call to build, and the array interface
    dictionary of a structured array as much)."""
    return a.ctypes.data


def _host_segments(segs) -> np.ndarray:
    """A host plan as a contiguous SEGMENT_DTYPE array: one already, or an
    integer (k, 4) array of (src_block, dst_block, n_blocks, first) rows."""
    a = np.asarray(segs)
    if a.dtype == SEGMENT_DTYPE:
        return np.ascontiguousarray(a).reshape(-1)
    if a.dtype.kind in "iu" and a.ndim == 2 and a.shape[1] == 4:
        return np.ascontiguousarray(a, dtype=np.int32).view(SEGMENT_DTYPE).reshape(-1)
    raise ValueError(f"a plan is a SEGMENT_DTYPE array or an integer (k, 4) array, "
                     f"not {a.dtype} {a.shape}")


def _device_segments(segs_dev, n_segs: int, pool: "KVPool") -> int:
    """Address of a device plan: a contiguous int32 tensor of at least n_segs
    rows of 4 on the pools' device (0 when n_segs is 0)."""
    if n_segs <= 0:
        return 0
    import torch

    if segs_dev.dtype != torch.int32 or not segs_dev.is_contiguous() \
            or segs_dev.device != pool.device or segs_dev.numel() < 4 * n_segs:
        raise ValueError(f"device plan: need a contiguous int32 tensor of >= {n_segs} x 4 "
                         f"on {pool.device}, got {segs_dev.dtype} {tuple(segs_dev.shape)} "
                         f"on {segs_dev.device}")
    return segs_dev.data_ptr()


# ---- allocator ---------------------------------------------------------------

def flowkv_allocator_create(num_blocks: int, policy: int = POLICY_SEGMENT, seed: int = 0):
    h = ctypes.c_void_p()
    _check(_lib.flowkv_allocator_create(num_blocks, policy, seed & (2**64 - 1), ctypes.byref(h)),
           "flowkv_allocator_create")
    return h


def flowkv_allocator_destroy(h) -> None:
    _lib.flowkv_allocator_destroy(h)


def flowkv_alloc(h, n_blocks: int) -> np.ndarray:
    out = np.empty(max(n_blocks, 0), dtype=np.int32)
    _check(_lib.flowkv_alloc(h, n_blocks, _ptr(out)), "flowkv_alloc")
    return out


def flowkv_free(h, ids) -> None:
    ids = _i32(ids)
    _check(_lib.flowkv_free(h, _ptr(ids), ids.size), "flowkv_free")


def flowkv_mark_used(h, ids) -> None:
    ids = _i32(ids)
    _check(_lib.flowkv_mark_used(h, _ptr(ids), ids.size), "flowkv_mark_used")


def flowkv_allocator_stats(h) -> dict:
    st = flowkv_alloc_stats()
    _check(_lib.flowkv_allocator_stats(h, ctypes.byref(st)), "flowkv_allocator_stats")
    return {"free_blocks": st.free_blocks, "free_segments": st.free_segments,
            "largest_free": st.largest_free}


class Allocator:
    """Owner of one allocator handle."""

    def __init__(self, num_blocks: int, policy: int = POLICY_SEGMENT, seed: int = 0):
        self.num_blocks = num_blocks
        self.policy = policy
        self._h = flowkv_allocator_create(num_blocks, policy, seed)
        self._destroy = _lib.flowkv_allocator_destroy  # kept: module globals may be gone at exit

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h:
            self._destroy(h)

    def alloc(self, n: int) -> np.ndarray:
        return flowkv_alloc(self._h, n)

    def free(self, ids) -> None:
        flowkv_free(self._h, ids)

    def mark_used(self, ids) -> None:
        flowkv_mark_used(self._h, ids)

    def stats(self) -> dict:
        return flowkv_allocator_stats(self._h)


# ---- load-aware scheduler ------------------------------------------------------

ROLE_PREFILL, ROLE_DECODE, ROLE_OFFLINE = 0, 1, 2
SCENARIO_NORMAL, SCENARIO_IMBALANCED, SCENARIO_EXTREME, SCENARIO_LOW_LOAD = 0, 1, 2, 3
SCHED_INDICATORS = 12


def sched_params(window: int, scale, w_prefill, w_decode, eps_p_low: float, eps_d_low: float,
                 eps_p_high: float, eps_d_high: float, idle_threshold: float,
                 scale_after: int, eps_p_min: float = 0.0,
                 eps_d_min: float = 0.0) -> flowkv_sched_params:
    p = flowkv_sched_params()
    p.window, p.scale_after = window, scale_after
    p.scale[:] = [float(x) for x in scale]
    p.w_prefill[:] = [float(x) for x in w_prefill]
    p.w_decode[:] = [float(x) for x in w_decode]
    p.eps_p_low, p.eps_d_low = eps_p_low, eps_d_low
    p.eps_p_high, p.eps_d_high = eps_p_high, eps_d_high
    p.idle_threshold = idle_threshold
    p.eps_p_min, p.eps_d_min = eps_p_min, eps_d_min
    return p


class Scheduler:
    """Owner of one flowkv_sched handle (Algorithm 1 of the paper)."""

    def __init__(self, params: flowkv_sched_params, roles):
        r = _i32(roles)
        self.n = int(r.size)
        h = ctypes.c_void_p()
        _check(_lib.flowkv_sched_create(ctypes.byref(params), self.n, _ptr(r), ctypes.byref(h)),
               "flowkv_sched_create")
        self._h = h.value
        self._destroy = _lib.flowkv_sched_destroy  # kept: module globals may be gone at exit
        self._idle = np.empty(self.n, dtype=np.int32)
        self._scores = np.empty((self.n, 2), dtype=np.float64)

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h:
            self._destroy(h)

    def set_role(self, node: int, role: int) -> None:
        _check(_lib.flowkv_sched_set_role(self._h, node, role), "flowkv_sched_set_role")

    def observe(self, status) -> None:
        st = np.ascontiguousarray(np.asarray(status, dtype=np.float64))
        if st.shape != (self.n, SCHED_INDICATORS):
            raise ValueError(f"status must be ({self.n}, {SCHED_INDICATORS})")
        _check(_lib.flowkv_sched_observe(self._h, _ptr(st)),
               "flowkv_sched_observe")

    def evaluate(self):
        """Returns (result struct, idle node array, (n, 2) array of C_i^p, C_i^d)."""
        r = flowkv_sched_result()
        _check(_lib.flowkv_sched_evaluate(self._h, ctypes.byref(r), _ptr(self._idle),
                                          _ptr(self._scores)),
               "flowkv_sched_evaluate")
        return r, self._idle[: r.n_idle].copy(), self._scores.copy()

    def route(self, prompt_tokens: int, prefix_hit, queued_tokens, prefill_rate, kv_bytes: int,
              xfer_sec_per_byte, xfer_latency, free_bytes):
        """(prefill node, decode node) for one request; -1 where none qualifies."""
        n = self.n
        hit = np.ascontiguousarray(np.asarray(prefix_hit, dtype=np.int64))
        q = np.ascontiguousarray(np.asarray(queued_tokens, dtype=np.int64))
        rate = np.ascontiguousarray(np.asarray(prefill_rate, dtype=np.float64))
        spb = np.ascontiguousarray(np.asarray(xfer_sec_per_byte, dtype=np.float64))
        lat = np.ascontiguousarray(np.asarray(xfer_latency, dtype=np.float64))
        free = np.ascontiguousarray(np.asarray(free_bytes, dtype=np.int64))
        if hit.shape != (n,) or q.shape != (n,) or rate.shape != (n,) or free.shape != (n,) \
                or spb.shape != (n, n) or lat.shape != (n, n):
            raise ValueError("routing arrays do not match the node count")
        pn, dn = ctypes.c_int32(), ctypes.c_int32()
        _check(_lib.flowkv_sched_route(self._h, prompt_tokens, _ptr(hit), _ptr(q),
                                       _ptr(rate), kv_bytes,
                                       _ptr(spb), _ptr(lat),
                                       _ptr(free), ctypes.byref(pn), ctypes.byref(dn)),
               "flowkv_sched_route")
        return pn.value, dn.value


# ---- planner -----------------------------------------------------------------

def flowkv_plan(src_ids, dst_ids, src_pool_blocks: int, dst_pool_blocks: int) -> np.ndarray:
    """Aligned runs of one request as a SEGMENT_DTYPE array."""
    s, d = _i32(src_ids), _i32(dst_ids)
    if s.size != d.size:
        raise ValueError("sender and receiver lists differ in length")
    out = np.empty(max(s.size, 1), dtype=SEGMENT_DTYPE)
    n = ctypes.c_int64()
    _check(_lib.flowkv_plan(_ptr(s), _ptr(d), s.size, src_pool_blocks, dst_pool_blocks,
                            _ptr(out), out.size, ctypes.byref(n)), "flowkv_plan")
    return out[: n.value]


def flowkv_plan_batch(offsets, src_ids, dst_ids, src_pool_blocks: int,
                      dst_pool_blocks: int) -> np.ndarray:
    """Aligned runs of a batch (request r = offsets[r] .. offsets[r+1])."""
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
    s, d = _i32(src_ids), _i32(dst_ids)
    if s.size != d.size:
        raise ValueError("sender and receiver lists differ in length")
    # the planner reads the lists up to offsets[-1]: it must be their length
    if off.ndim != 1 or off.size < 1 or int(off[-1]) != s.size:
        raise ValueError(f"offsets must be 1-D, n_req + 1 entries ending at the lists' length "
                         f"{s.size}, got shape {off.shape}"
                         + (f" ending at {int(off[-1])}" if off.ndim == 1 and off.size else ""))
    out = np.empty(max(s.size, 1), dtype=SEGMENT_DTYPE)
    n = ctypes.c_int64()
    _check(_lib.flowkv_plan_batch(off.size - 1, _ptr(off), _ptr(s), _ptr(d),
                                  src_pool_blocks, dst_pool_blocks, _ptr(out),
                                  out.size, ctypes.byref(n)), "flowkv_plan_batch")
    return out[: n.value]


def plan_total_blocks(segs: np.ndarray) -> int:
    if segs.size == 0:
        return 0
    return int(segs["first"][-1]) + int(segs["n_blocks"][-1])


# ---- pools and transfer ------------------------------------------------------

class KVPool:
    """Device pool descriptor over caller-owned torch tensors.

    Block-major: one contiguous tensor shaped (B, L, 2, block_size, kv_heads,
    head_dim).  Layer-major: a list of L contiguous tensors, each shaped
    (2, B, block_size, kv_heads, head_dim).
    """

    def __init__(self, layout: int, tensors):
        import torch  # device memory only

        if layout == LAYOUT_BLOCK_MAJOR:
            t = tensors[0] if isinstance(tensors, (list, tuple)) else tensors
            if t.dim() != 6:
                raise ValueError("block-major pool tensor must be (B, L, 2, bs, Hkv, Dh)")
            B, L, two, bs, hkv, dh = t.shape
            self.tensors = [t]
        elif layout == LAYOUT_LAYER_MAJOR:
            ts = list(tensors)
            if not ts or any(x.dim() != 5 for x in ts):
                raise ValueError("layer-major pool needs L tensors shaped (2, B, bs, Hkv, Dh)")
            two, B, bs, hkv, dh = ts[0].shape
            L = len(ts)
            if any(tuple(x.shape) != tuple(ts[0].shape) or x.dtype != ts[0].dtype for x in ts):
                raise ValueError("layer tensors differ in shape or dtype")
            self.tensors = ts
        else:
            raise ValueError(f"unknown layout {layout}")
        if two != 2:
            raise ValueError("the K/V axis must have size 2")
        for x in self.tensors:
            if not x.is_contiguous() or x.device.type != "cuda":
                raise ValueError("pool tensors must be contiguous device tensors")
        self.layout, self.num_layers, self.num_blocks = layout, L, B
        self.block_size, self.kv_heads, self.head_dim = bs, hkv, dh
        self.elem_bytes = self.tensors[0].element_size()
        self.chunk_bytes = bs * hkv * dh * self.elem_bytes
        self.block_bytes = 2 * L * self.chunk_bytes
        self.device = self.tensors[0].device
        self._bases = (ctypes.c_void_p * len(self.tensors))(*[x.data_ptr() for x in self.tensors])
        self.desc = flowkv_pool(layout, L, B, 0, self.chunk_bytes,
                                ctypes.cast(self._bases, ctypes.POINTER(ctypes.c_void_p)))


def _stream_handle(stream) -> Optional[int]:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _pools(src: KVPool, dst: KVPool):
    """The two descriptors, by reference, for a copy between pools of one
    element type: the library compares byte geometry only, so bf16 into fp16
    (same sizes, other encoding) is refused here."""
    if src.tensors[0].dtype != dst.tensors[0].dtype:
        raise ValueError(f"pools of different element types: {src.tensors[0].dtype} and "
                         f"{dst.tensors[0].dtype}")
    return ctypes.byref(src.desc), ctypes.byref(dst.desc)


def flowkv_transfer(src: KVPool, dst: KVPool, segs_dev, n_segs: int, total_blocks: int,
                    stream=None) -> None:
    """Enqueue the one-launch copy; segs_dev is a device int32 (k, 4) tensor
    on the pools' device."""
    _check(_lib.flowkv_transfer(*_pools(src, dst),
                                ctypes.c_void_p(_device_segments(segs_dev, n_segs, src)),
                                n_segs, total_blocks, ctypes.c_void_p(_stream_handle(stream))),
           "flowkv_transfer")


def flowkv_transfer_ex(src: KVPool, dst: KVPool, segs_dev, n_segs: int, total_blocks: int,
                       threads: int = 0, unroll: int = 0, grid: int = 0, cache: int = 0,
                       order: int = 0, stream=None) -> None:
    cfg = flowkv_launch_config(threads, unroll, grid, cache, order)
    _check(_lib.flowkv_transfer_ex(*_pools(src, dst),
                                   ctypes.c_void_p(_device_segments(segs_dev, n_segs, src)),
                                   n_segs, total_blocks, ctypes.byref(cfg),
                                   ctypes.c_void_p(_stream_handle(stream))),
           "flowkv_transfer_ex")


def inline_capacity(src: KVPool, dst: KVPool) -> int:
    """Most plan records (as flowkv_plan writes them) that flowkv_transfer_inline
    carries in the kernel arguments between these two pools."""
    n = ctypes.c_int64()
    _check(_lib.flowkv_inline_capacity(ctypes.byref(src.desc), ctypes.byref(dst.desc),
                                       ctypes.byref(n)), "flowkv_inline_capacity")
    return n.value


def flowkv_transfer_inline(src: KVPool, dst: KVPool, segs: np.ndarray, total_blocks: int,
                           threads: int = 0, unroll: int = 0, grid: int = 0, cache: int = 0,
                           order: int = 0, stream=None) -> None:
    """Enqueue the one-launch copy with a host plan (SEGMENT_DTYPE array, or
    int (k, 4) rows) carried in the kernel arguments: at most INLINE_RUNS
    records; in the planner's form, INLINE_RUNS_BLOCK_MAJOR between
    block-major pools, or INLINE_RUNS_LAYER_MAJOR when a pool is layer-major
    and neither has more than INLINE_LAYERS layers (``inline_capacity``)."""
    segs = _host_segments(segs)
    cfg = flowkv_launch_config(threads, unroll, grid, cache, order)
    _check(_lib.flowkv_transfer_inline(*_pools(src, dst),
                                       _ptr(segs), len(segs), total_blocks,
                                       ctypes.byref(cfg), ctypes.c_void_p(_stream_handle(stream))),
           "flowkv_transfer_inline")


def flowkv_transfer_request(src: KVPool, dst: KVPool, src_ids, dst_ids, threads: int = 0,
                            unroll: int = 0, grid: int = 0, cache: int = 0, order: int = 0,
                            stream=None) -> int:
    """Plan one request and enqueue its copy with the plan in the kernel
    arguments, in one library call; returns the plan's run count.  Raises
    FlowKVError(ECAP) when the plan does not fit there (``inline_capacity``)."""
    s, d = _i32(src_ids), _i32(dst_ids)
    if s.size != d.size:
        raise ValueError("sender and receiver lists differ in length")
    cfg = flowkv_launch_config(threads, unroll, grid, cache, order)
    n = ctypes.c_int64()
    _check(_lib.flowkv_transfer_request(*_pools(src, dst),
                                        _ptr(s), _ptr(d), s.size, ctypes.byref(cfg),
                                        ctypes.byref(n), ctypes.c_void_p(_stream_handle(stream))),
           "flowkv_transfer_request")
    return n.value


def flowkv_transfer_layers(src: KVPool, dst: KVPool, segs_dev, n_segs: int, total_blocks: int,
                           layer_begin: int, layer_count: int, threads: int = 0, unroll: int = 0,
                           grid: int = 0, cache: int = 0, order: int = 0, stream=None) -> None:
    """Enqueue the copy of layers [layer_begin, layer_begin + layer_count) only."""
    cfg = flowkv_launch_config(threads, unroll, grid, cache, order)
    _check(_lib.flowkv_transfer_layers(*_pools(src, dst),
                                       ctypes.c_void_p(_device_segments(segs_dev, n_segs, src)),
                                       n_segs, total_blocks, layer_begin, layer_count,
                                       ctypes.byref(cfg), ctypes.c_void_p(_stream_handle(stream))),
           "flowkv_transfer_layers")


def flowkv_decode_attention_split(n_req: int, max_seq_len: int) -> int:
    """The split length flowkv_decode_attention uses when split_tokens is 0."""
    s = ctypes.c_int32()
    _check(_lib.flowkv_decode_attention_split(n_req, max_seq_len, ctypes.byref(s)),
           "flowkv_decode_attention_split")
    return s.value


def flowkv_decode_attention_workspace(n_req: int, q_heads: int, head_dim: int,
                                      max_seq_len: int, split_tokens: int = 0) -> int:
    b = ctypes.c_int64()
    _check(_lib.flowkv_decode_attention_workspace(n_req, q_heads, head_dim, max_seq_len,
                                                  split_tokens, ctypes.byref(b)),
           "flowkv_decode_attention_workspace")
    return b.value


ATTN_SCRATCH_BYTES = 16 << 20  # scratch of flowkv_decode_attention_noalloc, per GPU
ATTN_INLINE_LENS = 512  # most host lengths a call carries in the kernel arguments


def _host_lens(seq_lens_host, n):
    """The host copy of the lengths as a contiguous int32 array (kept alive by
    the caller for the duration of the call), or None."""
    if seq_lens_host is None:
        return None
    h = np.ascontiguousarray(seq_lens_host, dtype=np.int32)
    if h.shape != (n,):
        raise ValueError("seq_lens_host: need one length per request")
    return h


def _check_attention_tensors(pool: KVPool, q, block_tables, seq_lens, out):
    import torch

    n, hq, dh = q.shape
    # the kernels read K and V as bfloat16; the C ABI sees only byte sizes,
    # so a pool of another 2-byte type is refused here
    if any(t.dtype != torch.bfloat16 for t in pool.tensors):
        raise ValueError(f"attention reads bfloat16 K/V: the pool holds {pool.tensors[0].dtype}")
    for t, dt in ((q, torch.bfloat16), (block_tables, torch.int32), (seq_lens, torch.int32),
                  (out, torch.float32)):
        if t.dtype != dt or not t.is_contiguous() or t.device != pool.device:
            raise ValueError("attention tensors: wrong dtype, layout or device")
    if tuple(out.shape) != (n, hq, dh) or block_tables.shape[0] != n or seq_lens.shape[0] != n:
        raise ValueError("attention tensors: shapes disagree")
    return n, hq, dh


def flowkv_decode_attention_noalloc(pool: KVPool, layer: int, q, block_tables, seq_lens,
                                    max_seq_len: int, scale: float, out,
                                    split_tokens: int = 0, stream=None,
                                    seq_lens_host=None) -> None:
    """flowkv_decode_attention without a workspace argument: the partial
    results go to the library's fixed per-GPU scratch (ATTN_SCRATCH_BYTES);
    calls that overlap on one GPU race."""
    n, hq, dh = _check_attention_tensors(pool, q, block_tables, seq_lens, out)
    hl = _host_lens(seq_lens_host, n)
    _check(_lib.flowkv_decode_attention_noalloc(
        ctypes.byref(pool.desc), layer, ctypes.c_void_p(q.data_ptr()), n, hq, pool.kv_heads, dh,
        ctypes.c_void_p(block_tables.data_ptr()), block_tables.shape[1],
        ctypes.c_void_p(seq_lens.data_ptr()), _ptr(hl) if hl is not None else None,
        max_seq_len, scale, split_tokens,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(_stream_handle(stream))),
        "flowkv_decode_attention_noalloc")


def flowkv_decode_attention(pool: KVPool, layer: int, q, block_tables, seq_lens,
                            max_seq_len: int, scale: float, out, workspace,
                            split_tokens: int = 0, stream=None, seq_lens_host=None) -> None:
    """Decode attention of layer `layer` over `pool` (torch device tensors:
    q (n, Hq, Dh) bf16, block_tables (n, max_blocks) int32, seq_lens (n,)
    int32, out (n, Hq, Dh) float32, workspace uint8).  seq_lens_host, an
    optional host copy of the lengths (int32-convertible, one per request),
    lets the call carry them in the kernel arguments (ATTN_INLINE_LENS)."""
    n, hq, dh = _check_attention_tensors(pool, q, block_tables, seq_lens, out)
    if not workspace.is_contiguous() or workspace.device != pool.device:
        raise ValueError("attention workspace: not a contiguous tensor on the pool's device")
    hl = _host_lens(seq_lens_host, n)
    _check(_lib.flowkv_decode_attention(
        ctypes.byref(pool.desc), layer, ctypes.c_void_p(q.data_ptr()), n, hq, pool.kv_heads, dh,
        ctypes.c_void_p(block_tables.data_ptr()), block_tables.shape[1],
        ctypes.c_void_p(seq_lens.data_ptr()), _ptr(hl) if hl is not None else None,
        max_seq_len, scale, split_tokens,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(workspace.data_ptr()),
        workspace.numel() * workspace.element_size(), ctypes.c_void_p(_stream_handle(stream))),
        "flowkv_decode_attention")


def segments_to_device(segs: np.ndarray, device, stream=None):
    """Stage a plan in pinned memory and copy it to the device on `stream`.

    Returns the device tensor (int32, (k, 4)); it must outlive the transfer
    that reads it (torch's caching allocator keeps it while referenced)."""
    import torch

    host = torch.from_numpy(_host_segments(segs).view(np.int32).reshape(-1, 4))
    pinned = host.pin_memory()
    if stream is None:
        return pinned.to(device, non_blocking=True)
    with torch.cuda.stream(stream):
        return pinned.to(device, non_blocking=True)


class PlanStager:
    """Ring of pinned host and device buffers for plans.

    ``stage(segs, stream)`` copies a plan to the device.  While ``stream``
    still runs earlier work, the copy goes on a side stream and ``stream``
    waits for it, so the upload overlaps that work; on an idle stream it goes
    on ``stream`` itself, which saves the cross-stream wait (about 35 us on
    an MI355X).  ``release(stream)`` marks the slot busy until ``stream``
    passes the kernel that reads it.  A slot is reused only after that (the
    host waits), so at most ``slots`` plans are in flight."""

    def __init__(self, device, capacity: int = 4096, slots: int = 4):
        import torch

        self.device = torch.device(device)
        self.slots = slots
        self.capacity = 0
        self.copy_stream = torch.cuda.Stream(self.device)
        self.copied = [torch.cuda.Event() for _ in range(slots)]
        self.done = [torch.cuda.Event() for _ in range(slots)]
        self.used = [False] * slots
        self.i = -1
        self._grow(capacity)

    def _grow(self, capacity: int):
        import torch

        torch.cuda.synchronize(self.device)
        self.capacity = capacity
        self.host = [torch.empty((capacity, 4), dtype=torch.int32, pin_memory=True)
                     for _ in range(self.slots)]
        self.dev = [torch.empty((capacity, 4), dtype=torch.int32, device=self.device)
                    for _ in range(self.slots)]
        self.used = [False] * self.slots

    def stage(self, segs: np.ndarray, stream=None):
        import torch

        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        k = len(segs)
        if k > self.capacity:
            self._grow(max(k, 2 * self.capacity))
        self.i = (self.i + 1) % self.slots
        j = self.i
        if self.used[j]:
            self.done[j].synchronize()
        if k:
            self.host[j].numpy()[:k] = _host_segments(segs).view(np.int32).reshape(-1, 4)
            if stream.query():
                with torch.cuda.stream(stream):
                    self.dev[j][:k].copy_(self.host[j][:k], non_blocking=True)
            else:
                with torch.cuda.stream(self.copy_stream):
                    self.dev[j][:k].copy_(self.host[j][:k], non_blocking=True)
                    self.copied[j].record(self.copy_stream)
                stream.wait_event(self.copied[j])
        self.used[j] = True
        return self.dev[j][:k]

    def release(self, stream=None):
        import torch

        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        self.done[self.i].record(stream)


def strerror(code: int) -> str:
    return _lib.flowkv_strerror(code).decode()
