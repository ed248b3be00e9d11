"""Thin ctypes binding of libpfxattn.so (include/pfx_attn.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  PyTorch supplies device memory and the current stream.  If the
library has not been built the import fails loudly; there is no fallback.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpfxattn.so")

PFX_OK = 0
PFX_EINVAL = -1
PFX_ERANGE = -2
PFX_ENOMEM = -3
PFX_EUNSUPPORTED = -4
PFX_EHIP = -5
PFX_PAGE_SIZE = 16
PFX_MODE_EXTEND = 1
PFX_MODE_DECODE = 2
PFX_MODE_MIXED = 3
PFX_DECODE_MFMA = 0
PFX_DECODE_VALU = 1
PFX_NOALLOC_MAX_WORKSPACE = 128 << 20

_ERR_NAMES = {PFX_EINVAL: "PFX_EINVAL", PFX_ERANGE: "PFX_ERANGE", PFX_ENOMEM: "PFX_ENOMEM",
              PFX_EUNSUPPORTED: "PFX_EUNSUPPORTED", PFX_EHIP: "PFX_EHIP"}

EXPORTED = [
    "pfx_version", "pfx_last_error",
    "pfx_alloc_create", "pfx_alloc_pages", "pfx_free_pages", "pfx_alloc_num_free", "pfx_alloc_destroy",
    "pfx_plan_create", "pfx_plan_workspace_bytes", "pfx_plan_get_stats", "pfx_plan_export",
    "pfx_plan_upload", "pfx_plan_destroy",
    "pfx_append_kv", "pfx_attention", "pfx_step", "pfx_merge_states",
    "pfx_page_copy_workspace_bytes", "pfx_page_copy", "pfx_sync_check", "pfx_attention_noalloc",
]


class PfxError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{_ERR_NAMES.get(code, code)}: {message}")
        self.code = code


class pfx_pool(C.Structure):
    _fields_ = [("num_pages", C.c_int32), ("page_size", C.c_int32), ("num_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("k_pages", C.c_void_p), ("v_pages", C.c_void_p)]


class pfx_prefix_table(C.Structure):
    _fields_ = [("num_agents", C.c_int32), ("page_indptr", C.POINTER(C.c_int32)),
                ("page_ids", C.POINTER(C.c_int32)), ("prefix_len", C.POINTER(C.c_int32))]


class pfx_batch(C.Structure):
    _fields_ = [("num_reqs", C.c_int32), ("agent", C.POINTER(C.c_int32)),
                ("suffix_indptr", C.POINTER(C.c_int32)), ("suffix_page_ids", C.POINTER(C.c_int32)),
                ("suffix_len", C.POINTER(C.c_int32)), ("q_indptr", C.POINTER(C.c_int32))]


class pfx_plan_opts(C.Structure):
    _fields_ = [("decode_workers", C.c_int32), ("piece_steps", C.c_int32), ("decode_engine", C.c_int32),
                ("reserved", C.c_int32 * 5)]


class pfx_plan_stats(C.Structure):
    _fields_ = [("num_requests", C.c_int32), ("num_tokens", C.c_int32), ("num_items", C.c_int32),
                ("num_prefix_items", C.c_int32), ("num_suffix_items", C.c_int32),
                ("num_extend_items", C.c_int32), ("num_partial_rows", C.c_int32),
                ("pages_needed", C.c_int32), ("num_decode_steps", C.c_int32), ("num_decode_pieces", C.c_int32),
                ("num_wide_blocks", C.c_int32), ("reserved", C.c_int32), ("workspace_bytes", C.c_int64)]


# Shapes of the arrays pfx_plan_export returns (int32 columns per record).
EXPORT_WIDTH = {0: 32, 1: 1, 2: 1, 3: 272, 6: 1, 7: 2, 8: 1}


def _load(path: str = LIB_PATH):
    # torch bundles its own HIP runtime with the same soname as the system
    # one.  Loading torch first makes this library bind to that same runtime,
    # so one process never holds two HIP runtimes (the second would find no
    # device).
    import torch  # noqa: F401

    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2608_25523_amd.build` "
                          "(there is no CPU fallback)")
    lib = C.CDLL(path)
    P = C.c_void_p
    i32, i64, sz = C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "pfx_version": ([], C.c_int),
        "pfx_last_error": ([], C.c_char_p),
        "pfx_alloc_create": ([i32, C.POINTER(P)], C.c_int),
        "pfx_alloc_pages": ([P, i32, P], C.c_int),
        "pfx_free_pages": ([P, P, i32], C.c_int),
        "pfx_alloc_num_free": ([P, C.POINTER(i32)], C.c_int),
        "pfx_alloc_destroy": ([P], None),
        "pfx_plan_create": ([C.POINTER(pfx_pool), C.POINTER(pfx_prefix_table), C.POINTER(pfx_batch), i32, i32,
                             C.POINTER(pfx_plan_opts), C.POINTER(P)], C.c_int),
        "pfx_plan_workspace_bytes": ([P, C.POINTER(sz)], C.c_int),
        "pfx_plan_get_stats": ([P, C.POINTER(pfx_plan_stats)], C.c_int),
        "pfx_plan_export": ([P, i32, P, i64, C.POINTER(i64)], C.c_int),
        "pfx_plan_upload": ([P, P, sz, P], C.c_int),
        "pfx_plan_destroy": ([P], None),
        "pfx_append_kv": ([C.POINTER(pfx_pool), P, P, P, P], C.c_int),
        "pfx_attention": ([C.POINTER(pfx_pool), P, P, P, P, C.c_float, P], C.c_int),
        "pfx_step": ([C.POINTER(pfx_pool), P, P, P, P, P, P, C.c_float, P], C.c_int),
        "pfx_merge_states": ([P, P, i32, i32, i32, P, P, P], C.c_int),
        "pfx_page_copy_workspace_bytes": ([i32], sz),
        "pfx_page_copy": ([C.POINTER(pfx_pool), C.POINTER(pfx_pool), P, P, i32, P, sz, P], C.c_int),
        "pfx_sync_check": ([P], C.c_int),
        "pfx_attention_noalloc": ([C.POINTER(pfx_pool), P, P, P, P, P, P, C.c_float, P], C.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


def _check(rc: int):
    if rc != PFX_OK:
        raise PfxError(rc, LIB.pfx_last_error().decode())


def _i32(a):
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(C.POINTER(C.c_int32))


def _ptr(t) -> int | None:
    """Device (or pinned host) address of a torch tensor, or None."""
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream=None):
    if stream is not None:
        return C.c_void_p(stream)
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def pfx_version() -> int:
    return LIB.pfx_version()


def pfx_last_error() -> str:
    return LIB.pfx_last_error().decode()


def make_pool(num_pages: int, num_kv_heads: int, head_dim: int, k_pages=None, v_pages=None) -> pfx_pool:
    """Pool descriptor over two tensors of shape [num_pages][Hkv][16][d] (bf16)."""
    return pfx_pool(num_pages, PFX_PAGE_SIZE, num_kv_heads, head_dim, _ptr(k_pages), _ptr(v_pages))


# --------------------------------------------------------------------------- allocator

class Allocator:
    def __init__(self, num_pages: int):
        h = C.c_void_p()
        _check(LIB.pfx_alloc_create(num_pages, C.byref(h)))
        self.h = h

    def alloc(self, n: int) -> np.ndarray:
        out = np.zeros(max(n, 0), np.int32)
        _check(LIB.pfx_alloc_pages(self.h, n, out.ctypes.data_as(C.c_void_p)))
        return out

    def free(self, ids):
        arr, _ = _i32(ids)
        _check(LIB.pfx_free_pages(self.h, arr.ctypes.data_as(C.c_void_p), len(arr)))

    def num_free(self) -> int:
        n = C.c_int32()
        _check(LIB.pfx_alloc_num_free(self.h, C.byref(n)))
        return n.value

    def __del__(self):
        if getattr(self, "h", None) and LIB is not None:
            LIB.pfx_alloc_destroy(self.h)
            self.h = None


# --------------------------------------------------------------------------- plan

class Plan:
    """Owns a pfx_plan handle and (after upload) its device workspace."""

    def __init__(self, handle):
        self.h = handle
        self.workspace = None

    def stats(self) -> pfx_plan_stats:
        s = pfx_plan_stats()
        _check(LIB.pfx_plan_get_stats(self.h, C.byref(s)))
        return s

    def workspace_bytes(self) -> int:
        n = C.c_size_t()
        _check(LIB.pfx_plan_workspace_bytes(self.h, C.byref(n)))
        return n.value

    def export(self, which: int) -> np.ndarray:
        cnt = C.c_int64()
        _check(LIB.pfx_plan_export(self.h, which, None, 0, C.byref(cnt)))
        out = np.zeros(cnt.value, np.int32)
        _check(LIB.pfx_plan_export(self.h, which, out.ctypes.data_as(C.c_void_p), cnt.value, C.byref(cnt)))
        w = EXPORT_WIDTH[which]
        return out.reshape(-1, w) if w > 1 else out

    def upload(self, workspace=None, stream=None, device="cuda"):
        """Copy the plan into a device workspace (a uint8 tensor; allocated by
        torch here if not given -- the library itself never allocates)."""
        import torch
        nbytes = self.workspace_bytes()
        if workspace is None:
            workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = workspace.data_ptr()
        pad = (-base) % 256
        _check(LIB.pfx_plan_upload(self.h, C.c_void_p(base + pad), workspace.numel() - pad, _stream(stream)))
        self.workspace = workspace
        return self

    def __del__(self):
        if getattr(self, "h", None) and LIB is not None:
            LIB.pfx_plan_destroy(self.h)
            self.h = None


def pfx_plan_create(pool: pfx_pool, prefix_page_indptr, prefix_page_ids, prefix_len, agent, suffix_indptr,
                    suffix_page_ids, suffix_len, q_indptr, num_q_heads: int, mode: int,
                    decode_workers: int = 0, piece_steps: int = 0, decode_engine: int = 0) -> Plan:
    keep = []

    def arr(x):
        a, p = _i32(x)
        keep.append(a)
        return p

    num_agents = len(prefix_len)
    pt = pfx_prefix_table(num_agents, arr(prefix_page_indptr), arr(prefix_page_ids), arr(prefix_len))
    num_reqs = len(agent)
    b = pfx_batch(num_reqs, arr(agent), arr(suffix_indptr), arr(suffix_page_ids), arr(suffix_len), arr(q_indptr))
    opts = pfx_plan_opts(decode_workers, piece_steps, decode_engine)
    h = C.c_void_p()
    _check(LIB.pfx_plan_create(C.byref(pool), C.byref(pt), C.byref(b), num_q_heads, mode, C.byref(opts),
                               C.byref(h)))
    return Plan(h)


def plan_from_batch(pool: pfx_pool, batch, mode: int = PFX_MODE_MIXED, **kw) -> Plan:
    """Convenience: plan for a ``workloads.Batch``."""
    pind, pids, plen = batch.prefix_csr()
    sind, sids = batch.suffix_csr()
    return pfx_plan_create(pool, pind, pids, plen, batch.agent, sind, sids, batch.suffix_len, batch.q_indptr(),
                           batch.num_q_heads, mode, **kw)


# --------------------------------------------------------------------------- device calls

def pfx_append_kv(pool: pfx_pool, plan: Plan, k_new, v_new, stream=None):
    _check(LIB.pfx_append_kv(C.byref(pool), plan.h, _ptr(k_new), _ptr(v_new), _stream(stream)))


def pfx_attention(pool: pfx_pool, plan: Plan, q, o, lse=None, sm_scale: float = 0.0, stream=None):
    _check(LIB.pfx_attention(C.byref(pool), plan.h, _ptr(q), _ptr(o), _ptr(lse), C.c_float(sm_scale),
                             _stream(stream)))


def pfx_step(pool: pfx_pool, plan: Plan, k_new, v_new, q, o, lse=None, sm_scale: float = 0.0, stream=None):
    _check(LIB.pfx_step(C.byref(pool), plan.h, _ptr(k_new), _ptr(v_new), _ptr(q), _ptr(o), _ptr(lse),
                        C.c_float(sm_scale), _stream(stream)))


def pfx_attention_noalloc(pool: pfx_pool, plan: Plan, q, o, lse=None, k_new=None, v_new=None,
                          sm_scale: float = 0.0, stream=None):
    _check(LIB.pfx_attention_noalloc(C.byref(pool), plan.h, _ptr(k_new), _ptr(v_new), _ptr(q), _ptr(o), _ptr(lse),
                                     C.c_float(sm_scale), _stream(stream)))


def pfx_merge_states(o_parts, lse_parts, o, lse=None, stream=None):
    num_parts, rows, d = o_parts.shape
    _check(LIB.pfx_merge_states(_ptr(o_parts), _ptr(lse_parts), num_parts, rows, d, _ptr(o), _ptr(lse),
                                _stream(stream)))


def pfx_page_copy_workspace_bytes(n: int) -> int:
    return LIB.pfx_page_copy_workspace_bytes(n)


def pfx_page_copy(dst: pfx_pool, src: pfx_pool, dst_pages, src_pages, workspace, stream=None):
    d, dp = _i32(dst_pages)
    s, sp = _i32(src_pages)
    if len(d) != len(s):
        raise ValueError("dst_pages and src_pages differ in length")
    base = workspace.data_ptr()
    pad = (-base) % 256
    _check(LIB.pfx_page_copy(C.byref(dst), C.byref(src), d.ctypes.data_as(C.c_void_p),
                             s.ctypes.data_as(C.c_void_p), len(d), C.c_void_p(base + pad),
                             workspace.numel() * workspace.element_size() - pad, _stream(stream)))


def pfx_sync_check(stream=None):
    _check(LIB.pfx_sync_check(_stream(stream)))
