"""Thin Python binding of libkvpattn (ctypes).  Argument marshalling only: every step of the attention
path runs in the HIP library; there is no fallback.  Device arrays are torch tensors on the GPU (torch
provides device memory and streams), host metadata arrays are numpy int32.

The names follow the C-ABI in include/kvpattn.h.
"""
from __future__ import annotations

import ctypes as C
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvpattn.so")

KVP_OK, KVP_EINVAL, KVP_ERANGE, KVP_EGROUP, KVP_ESHARED, KVP_EWORKSPACE, KVP_EUNSUPPORTED, KVP_EHIP, KVP_ENOMEM = \
    0, -1, -2, -3, -4, -5, -6, -7, -8
KVP_BF16, KVP_F32, KVP_FP8_E4M3 = 0, 1, 2
PAGE = 16

# Every symbol the header declares (kept in sync by a CPU test that parses include/kvpattn.h).
EXPORTS = ["kv_pool_create", "kv_pool_destroy", "kv_pool_reset", "kv_pool_layer_ptr", "kv_pool_info",
           "kv_pool_dtype", "kv_pool_set_scales", "kv_pool_device_error", "kv_append", "kv_gather",
           "paged_decode_workspace_size", "paged_decode_attn", "paged_decode_attn_noalloc",
           "prefix_chunk_prefill_workspace_size", "prefix_chunk_prefill_attn", "mixed_step_workspace_size",
           "mixed_step_attn", "kv_pool_page_bytes", "kv_offload",
           "kv_restore", "kvp_block_hashes", "kvp_group_shared_pages", "kvp_prefix_table_create",
           "kvp_prefix_table_destroy", "kvp_prefix_table_clear", "kvp_prefix_table_insert", "kvp_prefix_table_erase",
           "kvp_prefix_lookup", "kvp_prefix_table_error", "kvp_check_tables",
           "kvp_plan_decode", "kvp_strerror", "kvp_last_error", "kvp_version"]


class KvpError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {detail} (code {code})")
        self.code = code


class GroupPrefix(C.Structure):
    _fields_ = [("group_id", C.POINTER(C.c_int32)), ("shared_pages", C.POINTER(C.c_int32)),
                ("num_groups", C.c_int32)]


_lib = None


def lib() -> C.CDLL:
    """Load the built library.  Raises if it has not been built: there is no CPU fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_11152_amd.build`")
        L = C.CDLL(LIB_PATH)
        p, i, vp, sz = C.c_void_p, C.c_int, C.c_void_p, C.c_size_t
        i32p = C.POINTER(C.c_int32)
        gpp = C.POINTER(GroupPrefix)
        L.kv_pool_create.argtypes = [C.POINTER(p), i, i, i, i, i, i]
        L.kv_pool_destroy.argtypes = [p]
        L.kv_pool_reset.argtypes = [p, vp]
        L.kv_pool_layer_ptr.argtypes = [p, i, C.POINTER(vp), C.POINTER(sz)]
        L.kv_pool_info.argtypes = [p, C.POINTER(i), C.POINTER(i), C.POINTER(i), C.POINTER(i)]
        L.kv_pool_device_error.argtypes = [p, C.POINTER(i)]
        L.kv_pool_dtype.argtypes = [p, C.POINTER(i)]
        L.kv_pool_set_scales.argtypes = [p, i, C.c_float, C.c_float]
        L.kv_append.argtypes = [p, i, vp, vp, vp, i, i32p, i32p, i, gpp, vp]
        L.kv_gather.argtypes = [p, i, vp, i, i32p, i, vp, vp, vp]
        L.paged_decode_workspace_size.argtypes = [p, i32p, i, gpp, i, C.POINTER(sz)]
        L.paged_decode_attn.argtypes = [vp, p, i, vp, i, i32p, i, gpp, i, C.c_float, vp, i, vp, sz, vp]
        L.paged_decode_attn_noalloc.argtypes = [vp, p, i, vp, i, i32p, i, gpp, i, C.c_float, vp, i, vp]
        L.prefix_chunk_prefill_workspace_size.argtypes = [p, i32p, i32p, i, i, C.POINTER(sz)]
        L.prefix_chunk_prefill_attn.argtypes = [vp, p, i, vp, i, i32p, i32p, i, i, C.c_float, vp, i, vp, sz, vp]
        L.mixed_step_workspace_size.argtypes = [p, i32p, i, gpp, i32p, i32p, i, i, C.POINTER(sz)]
        L.mixed_step_attn.argtypes = [p, i, i, C.c_float, i, vp, vp, i, i32p, i, gpp, vp, vp, vp, i, i32p, i32p, i,
                                      vp, vp, sz, vp]
        L.kv_pool_page_bytes.argtypes = [p, C.POINTER(sz)]
        L.kv_offload.argtypes = [p, i, i32p, i, vp, vp]
        L.kv_restore.argtypes = [p, i, vp, i32p, i, vp, i, i, i32p, i32p, vp]
        L.kvp_block_hashes.argtypes = [vp, i32p, i, C.c_uint64, vp, vp]
        L.kvp_group_shared_pages.argtypes = [vp, i32p, i, i32p, i, vp, vp]
        L.kvp_prefix_table_create.argtypes = [C.POINTER(p), i]
        L.kvp_prefix_table_destroy.argtypes = [p]
        L.kvp_prefix_table_clear.argtypes = [p, vp]
        L.kvp_prefix_table_insert.argtypes = [p, vp, vp, C.c_int64, vp]
        L.kvp_prefix_table_erase.argtypes = [p, vp, vp, C.c_int64, vp]
        L.kvp_prefix_lookup.argtypes = [p, vp, i32p, i, vp, vp, vp]
        L.kvp_prefix_table_error.argtypes = [p, C.POINTER(i)]
        L.kvp_check_tables.argtypes = [i32p, i, i32p, i, i, gpp]
        L.kvp_plan_decode.argtypes = [i32p, i, gpp, i, i, i32p, i, C.POINTER(i), C.POINTER(i), C.POINTER(i)]
        L.kvp_strerror.argtypes = [i]
        L.kvp_strerror.restype = C.c_char_p
        L.kvp_last_error.restype = C.c_char_p
        L.kvp_version.restype = C.c_char_p
        for name in EXPORTS:
            if name not in ("kvp_strerror", "kvp_last_error", "kvp_version"):
                getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != KVP_OK:
        raise KvpError(rc, where, lib().kvp_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


class _GP:
    """Keeps the numpy arrays of a group-prefix hint alive while the C struct points into them."""

    def __init__(self, group_id, shared_pages):
        self.gid = _i32(group_id)
        self.sp = _i32(shared_pages)
        self.s = GroupPrefix(_ptr(self.gid), _ptr(self.sp) if self.sp.size else None, len(self.sp))

    def ref(self):
        return C.byref(self.s)


def group_prefix(group_id, shared_pages):
    return _GP(group_id, shared_pages)


def _gp_ref(gp):
    if gp is None:
        return None
    if isinstance(gp, tuple):
        gp = _GP(*gp)
    return gp.ref()


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def _torch_stream(stream):
    """The torch stream the library's kernels will run on (the current one when `stream` is None)."""
    import torch
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, int):
        return torch.cuda.ExternalStream(stream)
    return stream


def _alloc_on(stream, shape, dtype, device):
    """A buffer the kernels enqueued on `stream` write or read: allocated in that stream's context, so the
    caching allocator does not hand its memory to another stream's allocation while the work is pending."""
    import torch
    with torch.cuda.stream(_torch_stream(stream)):
        return torch.empty(shape, dtype=dtype, device=device)


def _check_q_heads(q, pool: "Pool"):
    """The kernels take head_dim from the pool and the GQA ratio from Hq / num_kv_heads."""
    _, Hq, d = q.shape
    if d != pool.head_dim:
        raise ValueError(f"q has head_dim {d}, the pool {pool.head_dim}")
    if Hq % pool.num_kv_heads:
        raise ValueError(f"q has {Hq} heads, not a multiple of the pool's {pool.num_kv_heads} KV heads")


def _dptr(t) -> C.c_void_p:
    return C.c_void_p(t.data_ptr() if t is not None else 0)


def _dev(t, name: str, dtypes, ndim: int | None = None, rows: int | None = None, tail=None):
    """The library receives device tensors as bare pointers laid out as the header states (dense, row
    major).  Check here what those pointers are assumed to hold, before anything is launched: on the GPU,
    dense, of the expected dtype and rank, with at least `rows` rows and trailing dimensions `tail`."""
    if t is None:
        raise ValueError(f"{name} is None")
    if not getattr(t, "is_cuda", False):
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}; expected one of {', '.join(str(d) for d in dtypes)}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} has {t.dim()} dimensions, expected {ndim}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if rows is not None and t.shape[0] < rows:
        raise ValueError(f"{name} has {t.shape[0]} rows, {rows} needed")
    if tail is not None and tuple(t.shape[1:]) != tuple(tail):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected (*, {', '.join(map(str, tail))})")
    return t


def _bf16():
    import torch
    return (torch.bfloat16,)


def _i32t():
    import torch
    return (torch.int32,)


def _outt():
    import torch
    return (torch.float32, torch.bfloat16)


class Pool:
    """A paged KV pool owned by the library (kv_pool_create / kv_pool_destroy)."""

    def __init__(self, num_layers: int, num_pages: int, num_kv_heads: int, head_dim: int, page_size: int = PAGE,
                 dtype: int = KVP_BF16):
        h = C.c_void_p()
        _check(lib().kv_pool_create(C.byref(h), num_layers, num_pages, page_size, num_kv_heads, head_dim, dtype),
               "kv_pool_create")
        self.handle = h
        self.num_layers, self.num_pages, self.num_kv_heads, self.head_dim = num_layers, num_pages, num_kv_heads, head_dim
        self.dtype = dtype

    def set_scales(self, layer: int, k_scale: float, v_scale: float):
        _check(lib().kv_pool_set_scales(self.handle, layer, float(k_scale), float(v_scale)), "kv_pool_set_scales")

    def kv_dtype(self) -> int:
        d = C.c_int()
        _check(lib().kv_pool_dtype(self.handle, C.byref(d)), "kv_pool_dtype")
        return d.value

    def layer_bytes(self, layer: int = 0):
        """A zero-copy uint8 device view of one pool layer's raw bytes."""
        import torch
        ptr, nbytes = self.layer_ptr(layer)

        class _View:
            __cuda_array_interface__ = {"shape": (nbytes,), "typestr": "|u1", "data": (ptr, False),
                                        "version": 3, "strides": None}
        return torch.as_tensor(_View(), device="cuda")

    def close(self):
        if self.handle:
            lib().kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset(self, stream=None):
        _check(lib().kv_pool_reset(self.handle, _stream(stream)), "kv_pool_reset")

    def layer_ptr(self, layer: int = 0):
        p, n = C.c_void_p(), C.c_size_t()
        _check(lib().kv_pool_layer_ptr(self.handle, layer, C.byref(p), C.byref(n)), "kv_pool_layer_ptr")
        return p.value, n.value

    def layer_raw(self, layer: int = 0):
        """A zero-copy int16 device view of one pool layer's raw bf16 bits (layout in include/kvpattn.h)."""
        import torch
        ptr, nbytes = self.layer_ptr(layer)

        class _View:
            __cuda_array_interface__ = {"shape": (nbytes // 2,), "typestr": "<i2", "data": (ptr, False),
                                        "version": 3, "strides": None}
        return torch.as_tensor(_View(), device="cuda")

    def device_error(self) -> int:
        c = C.c_int()
        _check(lib().kv_pool_device_error(self.handle, C.byref(c)), "kv_pool_device_error")
        return c.value


def kv_pool_create(num_layers, num_pages, num_kv_heads, head_dim, page_size=PAGE, dtype=KVP_BF16) -> Pool:
    return Pool(num_layers, num_pages, num_kv_heads, head_dim, page_size, dtype)


def kv_pool_destroy(pool: Pool):
    pool.close()


def kv_pool_reset(pool: Pool, stream=None):
    pool.reset(stream)


def kv_pool_device_error(pool: Pool) -> int:
    return pool.device_error()


def kv_append(pool: Pool, layer, k, v, block_tables, start_pos, cu_new, group_prefix=None, stream=None):
    """k, v: device bf16 [T, Hkv, d]; block_tables: device int32 [B, maxp]; start_pos, cu_new: host."""
    sp, cu = _i32(start_pos), _i32(cu_new)
    if len(cu) != len(sp) + 1:
        raise ValueError(f"cu_new has {len(cu)} entries, {len(sp) + 1} needed")
    _dev(block_tables, "block_tables", _i32t(), 2, rows=len(sp))
    if len(sp) and int(cu[-1]) > 0:
        tail = (pool.num_kv_heads, pool.head_dim)
        _dev(k, "k", _bf16(), 3, rows=int(cu[-1]), tail=tail)
        _dev(v, "v", _bf16(), 3, rows=int(cu[-1]), tail=tail)
    _check(lib().kv_append(pool.handle, layer, _dptr(k), _dptr(v), _dptr(block_tables), block_tables.shape[1],
                           _ptr(sp), _ptr(cu), len(sp), _gp_ref(group_prefix), _stream(stream)), "kv_append")


def kv_gather(pool: Pool, layer, block_tables, lens, stream=None):
    import torch
    ln = _i32(lens)
    _dev(block_tables, "block_tables", _i32t(), 2, rows=len(ln))
    T = int(ln.sum())
    shape = (T, pool.num_kv_heads, pool.head_dim)
    k = _alloc_on(stream, shape, torch.bfloat16, "cuda")
    v = _alloc_on(stream, shape, torch.bfloat16, "cuda")
    _check(lib().kv_gather(pool.handle, layer, _dptr(block_tables), block_tables.shape[1], _ptr(ln), len(ln),
                           _dptr(k), _dptr(v), _stream(stream)), "kv_gather")
    return k, v


def paged_decode_workspace_size(pool: Pool, seq_lens, num_q_heads, group_prefix=None) -> int:
    sl = _i32(seq_lens)
    n = C.c_size_t()
    _check(lib().paged_decode_workspace_size(pool.handle, _ptr(sl), len(sl), _gp_ref(group_prefix), num_q_heads,
                                             C.byref(n)), "paged_decode_workspace_size")
    return n.value


def paged_decode_attn(q, pool: Pool, layer, block_tables, seq_lens, group_prefix=None, scale=None, out=None,
                      out_dtype=None, ws=None, stream=None):
    """q: device bf16 [B, Hq, d]; block_tables: device int32 [B, maxp]; seq_lens: host int32 [B]."""
    import torch
    sl = _i32(seq_lens)
    _dev(q, "q", _bf16(), 3)
    B, Hq, d = q.shape
    _check_q_heads(q, pool)
    if B != len(sl):
        raise ValueError(f"q holds {B} sequences, seq_lens {len(sl)}")
    _dev(block_tables, "block_tables", _i32t(), 2, rows=B)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = _alloc_on(stream, (B, Hq, d), out_dtype or torch.float32, q.device)
    _dev(out, "out", _outt(), 3, rows=B, tail=(Hq, d))
    od = KVP_F32 if out.dtype == torch.float32 else KVP_BF16
    gpr = group_prefix if not isinstance(group_prefix, tuple) else _GP(*group_prefix)
    if ws is None:
        ws = _alloc_on(stream, max(1, paged_decode_workspace_size(pool, sl, Hq, gpr)), torch.uint8, q.device)
    _dev(ws, "ws", (ws.dtype,))
    _check(lib().paged_decode_attn(_dptr(q), pool.handle, layer, _dptr(block_tables), block_tables.shape[1],
                                   _ptr(sl), len(sl), _gp_ref(gpr), Hq, float(scale), _dptr(out), od, _dptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)), "paged_decode_attn")
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20  # KVP_NOALLOC_SCRATCH_BYTES


def paged_decode_attn_noalloc(q, pool: Pool, layer, block_tables, seq_lens, out, group_prefix=None, scale=None,
                              stream=None):
    """paged_decode_attn through the allocation-free entry point: the caller passes `out`; the library
    keeps the work list and partials in its own per-GPU scratch (calls that overlap on one GPU race)."""
    import torch
    sl = _i32(seq_lens)
    _dev(q, "q", _bf16(), 3)
    B, Hq, d = q.shape
    _check_q_heads(q, pool)
    if B != len(sl):
        raise ValueError(f"q holds {B} sequences, seq_lens {len(sl)}")
    _dev(block_tables, "block_tables", _i32t(), 2, rows=B)
    _dev(out, "out", _outt(), 3, rows=B, tail=(Hq, d))
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    od = KVP_F32 if out.dtype == torch.float32 else KVP_BF16
    gpr = group_prefix if not isinstance(group_prefix, tuple) else _GP(*group_prefix)
    _check(lib().paged_decode_attn_noalloc(_dptr(q), pool.handle, layer, _dptr(block_tables), block_tables.shape[1],
                                           _ptr(sl), len(sl), _gp_ref(gpr), Hq, float(scale), _dptr(out), od,
                                           _stream(stream)), "paged_decode_attn_noalloc")
    return out


def prefix_chunk_prefill_workspace_size(pool: Pool, ctx_lens, cu_q, num_q_heads) -> int:
    cl, cq = _i32(ctx_lens), _i32(cu_q)
    n = C.c_size_t()
    _check(lib().prefix_chunk_prefill_workspace_size(pool.handle, _ptr(cl), _ptr(cq), len(cl), num_q_heads,
                                                     C.byref(n)), "prefix_chunk_prefill_workspace_size")
    return n.value


def prefix_chunk_prefill_attn(q, pool: Pool, layer, block_tables, ctx_lens, cu_q, scale=None, out=None,
                              out_dtype=None, ws=None, stream=None):
    """q: device bf16 [sum C, Hq, d]; block_tables: device int32 [B, maxp]; ctx_lens, cu_q: host."""
    import torch
    cl, cq = _i32(ctx_lens), _i32(cu_q)
    if len(cq) != len(cl) + 1:
        raise ValueError(f"cu_q has {len(cq)} entries, {len(cl) + 1} needed")
    _dev(q, "q", _bf16(), 3)
    T, Hq, d = q.shape
    _check_q_heads(q, pool)
    if len(cl) and T != int(cq[-1]):
        raise ValueError(f"q holds {T} rows, cu_q ends at {int(cq[-1])}")
    _dev(block_tables, "block_tables", _i32t(), 2, rows=len(cl))
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = _alloc_on(stream, (T, Hq, d), out_dtype or torch.float32, q.device)
    _dev(out, "out", _outt(), 3, rows=T, tail=(Hq, d))
    od = KVP_F32 if out.dtype == torch.float32 else KVP_BF16
    if ws is None:
        ws = _alloc_on(stream, max(1, prefix_chunk_prefill_workspace_size(pool, cl, cq, Hq)), torch.uint8, q.device)
    _dev(ws, "ws", (ws.dtype,))
    _check(lib().prefix_chunk_prefill_attn(_dptr(q), pool.handle, layer, _dptr(block_tables), block_tables.shape[1],
                                           _ptr(cl), _ptr(cq), len(cl), Hq, float(scale), _dptr(out), od, _dptr(ws),
                                           ws.numel() * ws.element_size(), _stream(stream)), "prefix_chunk_prefill_attn")
    return out


def mixed_step_workspace_size(pool: Pool, seq_lens, ctx_lens, cu_q, num_q_heads, group_prefix=None) -> int:
    sl, cl, cq = _i32(seq_lens), _i32(ctx_lens), _i32(cu_q)
    n = C.c_size_t()
    _check(lib().mixed_step_workspace_size(pool.handle, _ptr(sl), len(sl), _gp_ref(group_prefix), _ptr(cl), _ptr(cq),
                                           len(cl), num_q_heads, C.byref(n)), "mixed_step_workspace_size")
    return n.value


def mixed_step_attn(pool: Pool, layer, q_dec, block_tables_dec, seq_lens, q_pf, block_tables_pf, ctx_lens, cu_q,
                    group_prefix=None, scale=None, out_dec=None, out_pf=None, out_dtype=None, ws=None, stream=None):
    """paged_decode_attn and prefix_chunk_prefill_attn of one step in one launch.  Either part may be
    empty (q_dec with 0 rows / q_pf with 0 rows).  Returns (out_dec, out_pf)."""
    import torch
    sl, cl, cq = _i32(seq_lens), _i32(ctx_lens), _i32(cu_q)
    if len(cq) != len(cl) + 1:
        raise ValueError(f"cu_q has {len(cq)} entries, {len(cl) + 1} needed")
    _dev(q_dec, "q_dec", _bf16(), 3)
    _dev(q_pf, "q_pf", _bf16(), 3)
    B, Hq, d = q_dec.shape
    T = q_pf.shape[0]
    _check_q_heads(q_dec, pool)
    _check_q_heads(q_pf, pool)
    if tuple(q_pf.shape[1:]) != (Hq, d):
        raise ValueError(f"q_pf rows are {tuple(q_pf.shape[1:])}, q_dec rows {(Hq, d)}")
    if B != len(sl):
        raise ValueError(f"q_dec holds {B} sequences, seq_lens {len(sl)}")
    if len(cl) and T != int(cq[-1]):
        raise ValueError(f"q_pf holds {T} rows, cu_q ends at {int(cq[-1])}")
    _dev(block_tables_dec, "block_tables_dec", _i32t(), 2, rows=B)
    _dev(block_tables_pf, "block_tables_pf", _i32t(), 2, rows=len(cl))
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out_dec is None:
        out_dec = _alloc_on(stream, (B, Hq, d), out_dtype or (out_pf.dtype if out_pf is not None else torch.float32),
                            q_dec.device)
    if out_pf is None:
        out_pf = _alloc_on(stream, (T, Hq, d), out_dec.dtype, q_pf.device)
    _dev(out_dec, "out_dec", _outt(), 3, rows=B, tail=(Hq, d))
    _dev(out_pf, "out_pf", _outt(), 3, rows=T, tail=(Hq, d))
    if out_dec.dtype != out_pf.dtype:
        raise ValueError(f"out_dec is {out_dec.dtype}, out_pf {out_pf.dtype}: one output dtype per call")
    od = KVP_F32 if out_dec.dtype == torch.float32 else KVP_BF16
    gpr = group_prefix if not isinstance(group_prefix, tuple) else _GP(*group_prefix)
    if ws is None:
        ws = _alloc_on(stream, max(1, mixed_step_workspace_size(pool, sl, cl, cq, Hq, gpr)), torch.uint8, q_dec.device)
    _dev(ws, "ws", (ws.dtype,))
    _check(lib().mixed_step_attn(pool.handle, layer, Hq, float(scale), od, _dptr(q_dec), _dptr(block_tables_dec),
                                 block_tables_dec.shape[1], _ptr(sl), len(sl), _gp_ref(gpr), _dptr(out_dec),
                                 _dptr(q_pf), _dptr(block_tables_pf), block_tables_pf.shape[1], _ptr(cl), _ptr(cq),
                                 len(cl), _dptr(out_pf), _dptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "mixed_step_attn")
    return out_dec, out_pf


def kv_pool_page_bytes(pool: Pool) -> int:
    n = C.c_size_t()
    _check(lib().kv_pool_page_bytes(pool.handle, C.byref(n)), "kv_pool_page_bytes")
    return n.value


def _check_host_size(pool: Pool, host, n: int, what: str):
    """The library trusts the host tier's extent (like any caller pointer): check it here."""
    if host is not None and host.numel() * host.element_size() < n * kv_pool_page_bytes(pool):
        raise ValueError(f"{what} holds {host.numel() * host.element_size()} bytes, "
                         f"{n} pages need {n * kv_pool_page_bytes(pool)}")


def kv_offload(pool: Pool, layer, page_ids, host_dst, stream=None):
    """Copy pool pages to the host tier.  host_dst: pinned host tensor of len(page_ids) * page_bytes bytes."""
    ids = _i32(page_ids)
    _check_host_size(pool, host_dst, len(ids), "host_dst")
    _check(lib().kv_offload(pool.handle, layer, _ptr(ids), len(ids), _dptr(host_dst), _stream(stream)), "kv_offload")


def kv_restore(pool: Pool, layer, host_src, page_ids, block_tables=None, rows=None, lpages=None, stream=None):
    """Copy host-tier pages into pool pages page_ids; optionally patch block_tables[rows, lpages] = page_ids."""
    ids = _i32(page_ids)
    _check_host_size(pool, host_src, len(ids), "host_src")
    if block_tables is not None:
        r, lp = _i32(rows), _i32(lpages)
        if len(r) != len(ids) or len(lp) != len(ids):
            raise ValueError("rows and lpages need one entry per page id")
        nr, mp = block_tables.shape
        rp, lpp = _ptr(r), _ptr(lp)
    else:
        nr, mp, rp, lpp = 0, 0, None, None
    _check(lib().kv_restore(pool.handle, layer, _dptr(host_src), _ptr(ids), len(ids), _dptr(block_tables), nr, mp,
                            rp, lpp, _stream(stream)), "kv_restore")


def block_hash_offsets(cu_tokens) -> np.ndarray:
    """Start of each sequence's block hashes, plus the total, for host cu_tokens (full pages only)."""
    cu = _i32(cu_tokens)
    return np.concatenate([[0], np.cumsum(np.diff(cu) // PAGE)]).astype(np.int64)


def kvp_block_hashes(tokens, cu_tokens, seed: int = 0, out=None, stream=None):
    """Block hashes of every full page: tokens device int32; returns device int64 [pages] (uint64 bits)."""
    import torch
    cu = _i32(cu_tokens)
    total = int(block_hash_offsets(cu)[-1])
    if len(cu) and tokens.numel() < int(cu[-1]):
        raise ValueError(f"tokens holds {tokens.numel()} ids, cu_tokens ends at {int(cu[-1])}")
    if out is None:
        out = _alloc_on(stream, max(1, total), torch.int64, "cuda")
    elif out.numel() < total:
        raise ValueError(f"out holds {out.numel()} hashes, {total} needed")
    _check(lib().kvp_block_hashes(_dptr(tokens), _ptr(cu), len(cu) - 1, C.c_uint64(seed & (2**64 - 1)), _dptr(out),
                                  _stream(stream)), "kvp_block_hashes")
    return out[:total]


def kvp_group_shared_pages(hashes, cu_tokens, group_id, num_groups: int, stream=None) -> np.ndarray:
    """Shared whole pages of each rollout group, derived on the device; returned on the host."""
    import torch
    cu, gid = _i32(cu_tokens), _i32(group_id)
    out = _alloc_on(stream, max(1, num_groups), torch.int32, "cuda")
    _check(lib().kvp_group_shared_pages(_dptr(hashes), _ptr(cu), len(cu) - 1, _ptr(gid), num_groups, _dptr(out),
                                        _stream(stream)), "kvp_group_shared_pages")
    _torch_stream(stream).synchronize()  # the copy below runs on torch's current stream
    return out[:num_groups].cpu().numpy()


class PrefixTable:
    """Device hash table from block hash to pool page (kvp_prefix_table_*)."""

    def __init__(self, capacity_log2: int = 20):
        h = C.c_void_p()
        _check(lib().kvp_prefix_table_create(C.byref(h), capacity_log2), "kvp_prefix_table_create")
        self.handle = h

    def close(self):
        if self.handle:
            lib().kvp_prefix_table_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def clear(self, stream=None):
        _check(lib().kvp_prefix_table_clear(self.handle, _stream(stream)), "kvp_prefix_table_clear")

    def insert(self, hashes, page_ids, stream=None):
        if page_ids.numel() < hashes.numel():
            raise ValueError("one page id per hash")
        _check(lib().kvp_prefix_table_insert(self.handle, _dptr(hashes), _dptr(page_ids), hashes.numel(),
                                             _stream(stream)), "kvp_prefix_table_insert")

    def erase(self, hashes, page_ids, stream=None):
        if page_ids.numel() < hashes.numel():
            raise ValueError("one page id per hash")
        _check(lib().kvp_prefix_table_erase(self.handle, _dptr(hashes), _dptr(page_ids), hashes.numel(),
                                            _stream(stream)), "kvp_prefix_table_erase")

    def lookup(self, hashes, cu_tokens, stream=None):
        """(matched_pages device int32 [num_seqs], page_ids device int32 [pages])."""
        import torch
        cu = _i32(cu_tokens)
        total = int(block_hash_offsets(cu)[-1])
        if hashes.numel() < total:
            raise ValueError(f"hashes holds {hashes.numel()} entries, cu_tokens needs {total}")
        matched = _alloc_on(stream, max(1, len(cu) - 1), torch.int32, "cuda")
        pages = _alloc_on(stream, max(1, total), torch.int32, "cuda")
        _check(lib().kvp_prefix_lookup(self.handle, _dptr(hashes), _ptr(cu), len(cu) - 1, _dptr(matched),
                                       _dptr(pages), _stream(stream)), "kvp_prefix_lookup")
        return matched[: len(cu) - 1], pages[:total]

    def error(self) -> int:
        c = C.c_int()
        _check(lib().kvp_prefix_table_error(self.handle, C.byref(c)), "kvp_prefix_table_error")
        return c.value


def kvp_check_tables(block_tables_host, lens, num_pages, group_prefix=None) -> int:
    """Host validation of a host copy of the block tables; returns the kvp_status code."""
    bt = _i32(block_tables_host)
    ln = _i32(lens)
    return lib().kvp_check_tables(_ptr(bt), bt.shape[1], _ptr(ln), len(ln), num_pages, _gp_ref(group_prefix))


def kvp_plan_decode(seq_lens, num_q_heads, num_kv_heads, group_prefix=None):
    """The decode work plan (host only): returns (items [n, 8] int32, n_partials, pages_per_split)."""
    sl = _i32(seq_lens)
    n, parts, ch = C.c_int(), C.c_int(), C.c_int()
    _check(lib().kvp_plan_decode(_ptr(sl), len(sl), _gp_ref(group_prefix), num_q_heads, num_kv_heads, None, 0,
                                 C.byref(n), C.byref(parts), C.byref(ch)), "kvp_plan_decode")
    items = np.zeros((max(1, n.value), 8), dtype=np.int32)
    _check(lib().kvp_plan_decode(_ptr(sl), len(sl), _gp_ref(group_prefix), num_q_heads, num_kv_heads,
                                 _ptr(items), n.value, C.byref(n), C.byref(parts), C.byref(ch)), "kvp_plan_decode")
    return items[: n.value], parts.value, ch.value


def kvp_strerror(code: int) -> str:
    return lib().kvp_strerror(code).decode()


def kvp_version() -> str:
    return lib().kvp_version().decode()
