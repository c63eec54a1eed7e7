"""ctypes binding of libpearl_attn.so (the C ABI in include/pearl_attn.h).

Argument marshalling only: every step of the computation runs in the library's HIP kernels.
Tensors are torch tensors on the current HIP device; the torch current stream is passed as the
launch stream.  If the library is missing or fails to load, every call raises -- there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpearl_attn.so")

PEARL_OK = 0
_lib = None


class PearlError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        super().__init__("%s failed: %s: %s" % (func, _status_name(status), detail))
        self.status = status


class KvShape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


class SeqDesc(ctypes.Structure):
    _fields_ = [("block_table", ctypes.c_void_p), ("bt_stride", ctypes.c_int32),
                ("ctx_lens", ctypes.c_void_p), ("cu_q_lens", ctypes.c_void_p),
                ("batch", ctypes.c_int32), ("total_q", ctypes.c_int32),
                ("max_q_len", ctypes.c_int32), ("max_kv_len", ctypes.c_int32)]


EXPORTED = ("pearl_abi_version", "pearl_status_str", "pearl_last_error", "pearl_kv_append",
            "pearl_attn_workspace_bytes", "pearl_attn_prefill_append", "pearl_attn_decode",
            "pearl_attn_mixed", "pearl_kv_pack", "pearl_kv_unpack", "pearl_set_kernel_events",
            "pearl_hbm_copy", "pearl_hbm_read", "pearl_hbm_read_nt", "pearl_hbm_fill", "pearl_attn_decode_static",
            "pearl_attn_decode_static_max_bytes", "pearl_attn_decode_append")


def load(path: str = LIB_PATH):
    """Load (once) and type the library.  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("HIP library %s is not built (run __graft_entry__.build() or "
                           "python -m paper_2609_35158_amd.build)" % path)
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.pearl_abi_version.restype = ctypes.c_int
    lib.pearl_abi_version.argtypes = []
    lib.pearl_status_str.restype = ctypes.c_char_p
    lib.pearl_status_str.argtypes = [ctypes.c_int]
    lib.pearl_last_error.restype = ctypes.c_char_p
    lib.pearl_last_error.argtypes = []
    lib.pearl_kv_append.restype = ctypes.c_int
    lib.pearl_kv_append.argtypes = [P(KvShape), P(SeqDesc), ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    for name in ("pearl_kv_pack", "pearl_kv_unpack"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [P(KvShape), P(SeqDesc), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                      ctypes.c_void_p]
    lib.pearl_attn_workspace_bytes.restype = ctypes.c_size_t
    lib.pearl_attn_workspace_bytes.argtypes = [P(KvShape), P(SeqDesc)]
    for name in ("pearl_attn_prefill_append", "pearl_attn_decode", "pearl_attn_mixed"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [P(KvShape), P(SeqDesc), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                      ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                      ctypes.c_size_t, ctypes.c_void_p]
    lib.pearl_attn_decode_append.restype = ctypes.c_int
    lib.pearl_attn_decode_append.argtypes = [P(KvShape), P(SeqDesc), ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                             ctypes.c_void_p]
    lib.pearl_attn_decode_static.restype = ctypes.c_int
    lib.pearl_attn_decode_static.argtypes = [P(KvShape), P(SeqDesc), ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p]
    lib.pearl_attn_decode_static_max_bytes.restype = ctypes.c_size_t
    lib.pearl_attn_decode_static_max_bytes.argtypes = []
    lib.pearl_set_kernel_events.restype = None
    lib.pearl_set_kernel_events.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    # measurement tooling (include/pearl_bench.h)
    lib.pearl_hbm_copy.restype = ctypes.c_int
    lib.pearl_hbm_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    for name in ("pearl_hbm_read", "pearl_hbm_read_nt"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    lib.pearl_hbm_fill.restype = ctypes.c_int
    lib.pearl_hbm_fill.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint32, ctypes.c_void_p]
    _lib = lib
    return lib


def set_kernel_events(before: Optional[int], after: Optional[int]) -> None:
    """Record raw hipEvent_t handles around the next calls' main kernel (None, None clears)."""
    load().pearl_set_kernel_events(before, after)


def _status_name(st: int) -> str:
    try:
        return load().pearl_status_str(st).decode()
    except Exception:
        return str(st)


def last_error() -> str:
    return load().pearl_last_error().decode()


def abi_version() -> int:
    return int(load().pearl_abi_version())


def _check(st: int, func: str) -> None:
    if st != PEARL_OK:
        raise PearlError(st, func, last_error())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype: torch.dtype) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be on the GPU" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def make_shape(num_q_heads: int, k_pool: torch.Tensor) -> KvShape:
    if k_pool.dim() != 4:
        raise ValueError("pools must be [num_pages][num_kv_heads][page_size][head_dim]")
    n, hkv, ps, d = k_pool.shape
    return KvShape(int(num_q_heads), int(hkv), int(d), int(ps), int(n))


def make_desc(block_table: torch.Tensor, ctx_lens: torch.Tensor, cu_q_lens: Optional[torch.Tensor],
              total_q: int, max_q_len: int, max_kv_len: int) -> SeqDesc:
    _need(block_table, "block_table", torch.int32)
    _need(ctx_lens, "ctx_lens", torch.int32)
    if block_table.dim() != 2:
        raise ValueError("block_table must be [batch][bt_stride]")
    batch = int(ctx_lens.shape[0])
    if block_table.shape[0] != batch:
        raise ValueError("block_table rows (%d) != batch (%d)" % (block_table.shape[0], batch))
    if cu_q_lens is not None:
        _need(cu_q_lens, "cu_q_lens", torch.int32)
        if cu_q_lens.shape[0] != batch + 1:
            raise ValueError("cu_q_lens must have batch+1 entries")
    return SeqDesc(block_table.data_ptr(), int(block_table.shape[1]), ctx_lens.data_ptr(),
                   _ptr(cu_q_lens), batch, int(total_q), int(max_q_len), int(max_kv_len))


def workspace_bytes(num_q_heads: int, k_pool: torch.Tensor, desc: SeqDesc) -> int:
    shape = make_shape(num_q_heads, k_pool)
    n = load().pearl_attn_workspace_bytes(ctypes.byref(shape), ctypes.byref(desc))
    if n == 0:
        raise PearlError(1, "pearl_attn_workspace_bytes", last_error())
    return int(n)


def kv_append(k_new: torch.Tensor, v_new: torch.Tensor, k_pool: torch.Tensor, v_pool: torch.Tensor,
              block_table: torch.Tensor, ctx_lens: torch.Tensor, cu_q_lens: Optional[torch.Tensor],
              max_q_len: int, max_kv_len: int) -> None:
    """Scatter new K/V rows [total_q][H_kv][d] into the pools (pearl_kv_append)."""
    for t, n in ((k_new, "k_new"), (v_new, "v_new"), (k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t, n, torch.bfloat16)
    desc = make_desc(block_table, ctx_lens, cu_q_lens, int(k_new.shape[0]), max_q_len, max_kv_len)
    shape = make_shape(k_pool.shape[1], k_pool)   # H_q is not used by the append
    st = load().pearl_kv_append(ctypes.byref(shape), ctypes.byref(desc), k_new.data_ptr(),
                                v_new.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), _stream())
    _check(st, "pearl_kv_append")


def kv_pack(k_pool: torch.Tensor, v_pool: torch.Tensor, block_table: torch.Tensor, ctx_lens: torch.Tensor,
            cu_q_lens: Optional[torch.Tensor], total: int, max_q_len: int, max_kv_len: int,
            out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Gather token ranges [ctx_lens[b], ctx_lens[b] + n_b) of every sequence out of the pools into
    a transfer buffer bf16 [2][total][H_kv][d] (pearl_kv_pack)."""
    for t, n in ((k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t, n, torch.bfloat16)
    H_kv, d = int(k_pool.shape[1]), int(k_pool.shape[3])
    if out is None:
        out = torch.empty((2, total, H_kv, d), dtype=torch.bfloat16, device=k_pool.device)
    _need(out, "out", torch.bfloat16)
    if tuple(out.shape) != (2, total, H_kv, d):
        raise ValueError("out must have shape (2, %d, %d, %d)" % (total, H_kv, d))
    desc = make_desc(block_table, ctx_lens, cu_q_lens, total, max_q_len, max_kv_len)
    shape = make_shape(H_kv, k_pool)
    st = load().pearl_kv_pack(ctypes.byref(shape), ctypes.byref(desc), k_pool.data_ptr(), v_pool.data_ptr(),
                              out.data_ptr(), _stream())
    _check(st, "pearl_kv_pack")
    return out


def kv_unpack(buf: torch.Tensor, k_pool: torch.Tensor, v_pool: torch.Tensor, block_table: torch.Tensor,
              ctx_lens: torch.Tensor, cu_q_lens: Optional[torch.Tensor], max_q_len: int,
              max_kv_len: int) -> None:
    """Scatter a transfer buffer bf16 [2][total][H_kv][d] into the pools at positions
    ctx_lens[b] + t through this pool's block table (pearl_kv_unpack)."""
    for t, n in ((buf, "buf"), (k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t, n, torch.bfloat16)
    if buf.dim() != 4 or buf.shape[0] != 2:
        raise ValueError("buf must have shape (2, total, H_kv, d)")
    desc = make_desc(block_table, ctx_lens, cu_q_lens, int(buf.shape[1]), max_q_len, max_kv_len)
    shape = make_shape(k_pool.shape[1], k_pool)
    st = load().pearl_kv_unpack(ctypes.byref(shape), ctypes.byref(desc), buf.data_ptr(), k_pool.data_ptr(),
                                v_pool.data_ptr(), _stream())
    _check(st, "pearl_kv_unpack")


def _attention(fname: str, q: torch.Tensor, k_pool: torch.Tensor, v_pool: torch.Tensor,
               block_table: torch.Tensor, ctx_lens: torch.Tensor, cu_q_lens: Optional[torch.Tensor],
               max_q_len: int, max_kv_len: int, scale: Optional[float], return_lse: bool,
               out: Optional[torch.Tensor], lse: Optional[torch.Tensor],
               workspace: Optional[torch.Tensor]):
    _need(q, "q", torch.bfloat16)
    _need(k_pool, "k_pool", torch.bfloat16)
    _need(v_pool, "v_pool", torch.bfloat16)
    if q.dim() != 3:
        raise ValueError("q must be [total_q][num_q_heads][head_dim]")
    total_q, H_q, d = q.shape
    desc = make_desc(block_table, ctx_lens, cu_q_lens, total_q, max_q_len, max_kv_len)
    shape = make_shape(H_q, k_pool)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", torch.bfloat16)
    if return_lse and lse is None:
        lse = torch.empty((total_q, H_q), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, "lse", torch.float32)
    if workspace is None:
        nbytes = load().pearl_attn_workspace_bytes(ctypes.byref(shape), ctypes.byref(desc))
        if nbytes == 0:
            raise PearlError(1, "pearl_attn_workspace_bytes", last_error())
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    else:
        _need(workspace, "workspace", torch.uint8)   # the library checks its size
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    st = getattr(load(), fname)(ctypes.byref(shape), ctypes.byref(desc), q.data_ptr(),
                                k_pool.data_ptr(), v_pool.data_ptr(), float(scale), out.data_ptr(),
                                _ptr(lse), workspace.data_ptr(), workspace.numel(), _stream())
    _check(st, fname)
    return (out, lse) if (return_lse or lse is not None) else out


def prefill_append(q, k_pool, v_pool, block_table, ctx_lens, cu_q_lens, max_q_len, max_kv_len,
                   scale=None, return_lse=False, out=None, lse=None, workspace=None):
    """Causal prefill-append attention of each sequence's new tokens (pearl_attn_prefill_append)."""
    return _attention("pearl_attn_prefill_append", q, k_pool, v_pool, block_table, ctx_lens, cu_q_lens,
                      max_q_len, max_kv_len, scale, return_lse, out, lse, workspace)


def decode(q, k_pool, v_pool, block_table, ctx_lens, max_kv_len, scale=None, return_lse=False,
           out=None, lse=None, workspace=None):
    """Single-token decode for every sequence (pearl_attn_decode); q is [batch][H_q][d]."""
    return _attention("pearl_attn_decode", q, k_pool, v_pool, block_table, ctx_lens, None,
                      1, max_kv_len, scale, return_lse, out, lse, workspace)


def decode_append(q, k_new, v_new, k_pool, v_pool, block_table, ctx_lens, max_kv_len, scale=None,
                  return_lse=False, out=None, lse=None, workspace=None):
    """One decode step with its append (pearl_attn_decode_append): k_new / v_new [batch][H_kv][d]
    are written at position ctx_lens[b] of every sequence, which then attends over ctx_lens[b] + 1
    keys; q is [batch][H_q][d]."""
    for t, n in ((q, "q"), (k_new, "k_new"), (v_new, "v_new"), (k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t, n, torch.bfloat16)
    if q.dim() != 3:
        raise ValueError("q must be [batch][num_q_heads][head_dim]")
    batch, H_q, d = q.shape
    if tuple(k_new.shape) != (batch, k_pool.shape[1], d) or tuple(v_new.shape) != tuple(k_new.shape):
        raise ValueError("k_new and v_new must be [batch][num_kv_heads][head_dim]")
    desc = make_desc(block_table, ctx_lens, None, batch, 1, max_kv_len)
    shape = make_shape(H_q, k_pool)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", torch.bfloat16)
    if return_lse and lse is None:
        lse = torch.empty((batch, H_q), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, "lse", torch.float32)
    if workspace is None:
        nbytes = load().pearl_attn_workspace_bytes(ctypes.byref(shape), ctypes.byref(desc))
        if nbytes == 0:
            raise PearlError(1, "pearl_attn_workspace_bytes", last_error())
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    else:
        _need(workspace, "workspace", torch.uint8)
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    st = load().pearl_attn_decode_append(ctypes.byref(shape), ctypes.byref(desc), q.data_ptr(), k_new.data_ptr(),
                                         v_new.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), float(scale),
                                         out.data_ptr(), _ptr(lse), workspace.data_ptr(), workspace.numel(),
                                         _stream())
    _check(st, "pearl_attn_decode_append")
    return (out, lse) if (return_lse or lse is not None) else out


def decode_static(q, k_pool, v_pool, block_table, ctx_lens, max_kv_len, scale=None, return_lse=False,
                  out=None, lse=None):
    """Single-token decode with the library's static per-GPU workspace (pearl_attn_decode_static):
    no device memory is allocated by the call (out and lse are allocated here only when not
    given)."""
    for t, n in ((q, "q"), (k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t, n, torch.bfloat16)
    if q.dim() != 3:
        raise ValueError("q must be [batch][num_q_heads][head_dim]")
    batch, H_q, d = q.shape
    desc = make_desc(block_table, ctx_lens, None, batch, 1, max_kv_len)
    shape = make_shape(H_q, k_pool)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", torch.bfloat16)
    if return_lse and lse is None:
        lse = torch.empty((batch, H_q), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, "lse", torch.float32)
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    st = load().pearl_attn_decode_static(ctypes.byref(shape), ctypes.byref(desc), q.data_ptr(), k_pool.data_ptr(),
                                         v_pool.data_ptr(), float(scale), out.data_ptr(), _ptr(lse), _stream())
    _check(st, "pearl_attn_decode_static")
    return (out, lse) if (return_lse or lse is not None) else out


def decode_static_max_bytes() -> int:
    return int(load().pearl_attn_decode_static_max_bytes())


def mixed(q, k_pool, v_pool, block_table, ctx_lens, cu_q_lens, max_q_len, max_kv_len, scale=None,
          return_lse=False, out=None, lse=None, workspace=None):
    """Colocated prefill chunks and decodes in one attention launch (pearl_attn_mixed)."""
    return _attention("pearl_attn_mixed", q, k_pool, v_pool, block_table, ctx_lens, cu_q_lens,
                      max_q_len, max_kv_len, scale, return_lse, out, lse, workspace)


# ------------------------------------------------------------------------------------------------
# measurement tooling (include/pearl_bench.h): bandwidth probes and the cache flush
# ------------------------------------------------------------------------------------------------

def hbm_copy(src: torch.Tensor, dst: torch.Tensor) -> None:
    """dst <- src, byte for byte (both contiguous GPU tensors of the same byte size)."""
    if not (src.is_cuda and dst.is_cuda and src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("hbm_copy needs contiguous GPU tensors")
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("hbm_copy: byte sizes differ")
    _check(load().pearl_hbm_copy(src.data_ptr(), dst.data_ptr(), n, _stream()), "pearl_hbm_copy")


def hbm_read(src: torch.Tensor, sink: torch.Tensor, nontemporal: bool = False) -> None:
    """Stream-read src; `sink` is a 16-byte (or larger) GPU tensor the kernel may overwrite.  Over
    >= 1 GiB the plain read is the cache flush (it leaves no dirty lines behind); nontemporal=True
    is pearl_hbm_read_nt, the faster read mode, which is no flush."""
    if not (src.is_cuda and src.is_contiguous() and sink.is_cuda and sink.numel() * sink.element_size() >= 16):
        raise ValueError("hbm_read needs a contiguous GPU source and a 16-byte GPU sink")
    name = "pearl_hbm_read_nt" if nontemporal else "pearl_hbm_read"
    _check(getattr(load(), name)(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(), _stream()),
           name)


def hbm_fill(dst: torch.Tensor, pattern: int = 0) -> None:
    """Write a 32-bit pattern over dst."""
    if not (dst.is_cuda and dst.is_contiguous()):
        raise ValueError("hbm_fill needs a contiguous GPU tensor")
    _check(load().pearl_hbm_fill(dst.data_ptr(), dst.numel() * dst.element_size(), pattern & 0xFFFFFFFF,
                                 _stream()), "pearl_hbm_fill")
