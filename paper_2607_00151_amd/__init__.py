"""MI355X-native segment re-prefill: Python binding of the C ABI in include/sa.h.

The binding only marshals arguments: torch tensors supply device pointers and
the current HIP stream, host length arrays are converted to int32, and every
computation happens in the HIP kernels of ``libsa.so``.  If the library is not
built, importing works but every call raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "Layout", "Context", "SaError", "library_path", "load_library",
    "sa_kv_append", "sa_kv_assemble", "sa_kv_assemble_append", "sa_kv_splice_alias",
    "sa_segment_prefill_attn", "sa_segment_prefill_attn_append", "sa_set_exact_scale", "sa_set_fused_append",
    "sa_set_kernel_events", "sa_set_block_clock", "sa_set_xcd_weights", "sa_sync_check", "sa_reserve",
    "sa_segment_prefill_attn_noalloc", "sa_attn_plan_stats", "EXPORTED_SYMBOLS",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libsa.so")
_lib = None

EXPORTED_SYMBOLS = ("sa_create", "sa_destroy", "sa_status_string", "sa_last_error",
                    "sa_sync_check", "sa_kv_append", "sa_kv_assemble", "sa_kv_assemble_append",
                    "sa_kv_splice_alias", "sa_segment_prefill_attn", "sa_segment_prefill_attn_append",
                    "sa_set_exact_scale", "sa_set_fused_append", "sa_set_kernel_events",
                    "sa_set_block_clock", "sa_set_xcd_weights", "sa_reserve",
                    "sa_segment_prefill_attn_noalloc", "sa_attn_plan_stats")

STATUS = {0: "SA_OK", 1: "SA_ERR_NULL", 2: "SA_ERR_SHAPE", 3: "SA_ERR_UNSUPPORTED",
          4: "SA_ERR_ALIGN", 5: "SA_ERR_RANGE", 6: "SA_ERR_NO_PAGES", 7: "SA_ERR_HIP",
          8: "SA_ERR_DEVICE", 9: "SA_ERR_OVERLAP"}


class SaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class Layout(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_layers", ctypes.c_int32), ("num_slots", ctypes.c_int64)]


class _Pages(ctypes.Structure):
    _fields_ = [("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p)]


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libsa.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run paper_2607_00151_amd.build.build()")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    LP = ctypes.POINTER(Layout)
    lib.sa_create.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_void_p)]
    lib.sa_destroy.argtypes = [P]
    lib.sa_destroy.restype = None
    lib.sa_status_string.argtypes = [ctypes.c_int]
    lib.sa_status_string.restype = ctypes.c_char_p
    lib.sa_last_error.argtypes = []
    lib.sa_last_error.restype = ctypes.c_char_p
    lib.sa_sync_check.argtypes = [P, P]
    lib.sa_kv_append.argtypes = [P, LP, I32, P, P, P, P, I32, P, P, _Pages, P]
    lib.sa_kv_assemble.argtypes = [P, LP, P, P, P, P, I32, P, P, P, P, _Pages, P, I32, P, P, I32,
                                   P, P]
    lib.sa_kv_assemble_append.argtypes = [P, LP, P, P, P, P, I32, P, P, P, P, _Pages, P, I32, P, P, I32,
                                          P, I32, P, P, P, P]
    lib.sa_kv_splice_alias.argtypes = [P, LP, I32, P, P, P, P, _Pages, P, I32, P, P, I32, P, P]
    lib.sa_segment_prefill_attn.argtypes = [P, LP, I32, P, P, P, I32, P, P, _Pages, ctypes.c_float,
                                            P, P, P]
    lib.sa_segment_prefill_attn_append.argtypes = [P, LP, I32, P, P, P, P, P, I32, P, P, _Pages,
                                                   ctypes.c_float, P, P, P]
    lib.sa_set_exact_scale.argtypes = [P, I32]
    lib.sa_set_fused_append.argtypes = [P, I32]
    lib.sa_set_kernel_events.argtypes = [P, I32, P, P]
    lib.sa_set_block_clock.argtypes = [P, P, I64, ctypes.POINTER(ctypes.c_int64)]
    lib.sa_set_xcd_weights.argtypes = [P, P]
    lib.sa_reserve.argtypes = [P, I64, I64]
    lib.sa_segment_prefill_attn_noalloc.argtypes = lib.sa_segment_prefill_attn.argtypes
    lib.sa_attn_plan_stats.argtypes = [LP, I32, P, P, I32, P]
    for name in ("sa_create", "sa_sync_check", "sa_kv_append", "sa_kv_assemble", "sa_kv_assemble_append",
                 "sa_kv_splice_alias", "sa_segment_prefill_attn", "sa_segment_prefill_attn_append",
                 "sa_set_exact_scale", "sa_set_fused_append", "sa_set_kernel_events", "sa_set_block_clock",
                 "sa_set_xcd_weights",
                 "sa_reserve", "sa_segment_prefill_attn_noalloc", "sa_attn_plan_stats"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        msg = load_library().sa_last_error().decode(errors="replace")
        raise SaError(status, msg)


def _ptr(t):
    """Address of a host numpy array, or None."""
    if t is None:
        return None
    return t.ctypes.data


def _dev(t, what: str, kind: str, min_numel: int = 0, nullable: bool = False):
    """Device address of a caller tensor after checking what the C ABI will assume
    of it: a contiguous CUDA tensor whose element type matches `kind` ("i32": int32
    table entries, "b16": 2-byte bf16 bit patterns, "f32": float32) and that holds at
    least min_numel elements.  Raises ValueError otherwise; None passes only when
    nullable."""
    if t is None:
        if nullable:
            return None
        raise ValueError(f"{what}: a device tensor is required")
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what}: expected a torch tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{what}: tensor is not on a GPU")
    if not t.is_contiguous():
        raise ValueError(f"{what}: tensor is not contiguous")
    ok = {"i32": t.dtype == torch.int32,
          "b16": t.element_size() == 2 and t.dtype != torch.bool,
          "f32": t.dtype == torch.float32}[kind]
    if not ok:
        want = {"i32": "torch.int32", "b16": "a 2-byte dtype (bf16 bits)", "f32": "torch.float32"}[kind]
        raise ValueError(f"{what}: dtype {t.dtype}, expected {want}")
    if t.numel() < min_numel:
        raise ValueError(f"{what}: {t.numel()} elements, at least {min_numel} needed")
    return t.data_ptr() or None


def _pool_numel(layout) -> int:
    return (int(layout.num_layers) * int(layout.num_slots) * int(layout.num_kv_heads)
            * int(layout.page_size) * int(layout.head_dim))


def _host_i32(x):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int64))
    if a.size and (a.min() < -2**31 or a.max() >= 2**31):
        raise OverflowError("value does not fit int32")
    return np.ascontiguousarray(a, dtype=np.int32)


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream
    return int(stream)


def _pages(indptr, indices, batch: int, what: str = "page table"):
    return _Pages(_dev(indptr, f"{what} indptr", "i32", batch + 1),
                  _dev(indices, f"{what} indices", "i32", 0))


class Context:
    """Owns an sa_ctx (plan buffers, staging, split scratch) on one device."""

    def __init__(self, device: int = 0):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.sa_create(int(device), ctypes.byref(h)))
        self._h = h
        self.device = device

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load_library().sa_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def _ctx_handle(ctx):
    if ctx is None:
        return None
    return ctx.handle if isinstance(ctx, Context) else ctx


def sa_reserve(ctx, plan_bytes: int, split_bytes: int = 0):
    """Size ctx's plan buffers (each call kind's, and the pinned staging) to plan_bytes and
    its split-KV partials to split_bytes, so later calls that fit allocate nothing."""
    _check(load_library().sa_reserve(_ctx_handle(ctx), int(plan_bytes), int(split_bytes)))


def sa_attn_plan_stats(layout: Layout, q_len, kv_len, num_cu: int = 256) -> dict:
    """Shape of the attention launch these lengths make (host only, no GPU): workgroups,
    split parts, 64-key tiles and the makespan in tiles over 2 x num_cu slots."""
    q_len, kv_len = _host_i32(q_len), _host_i32(kv_len)
    if q_len.shape != kv_len.shape:
        raise ValueError("q_len and kv_len differ in length")
    out = np.zeros(4, dtype=np.int64)
    _check(load_library().sa_attn_plan_stats(ctypes.byref(layout), int(len(q_len)), _ptr(q_len), _ptr(kv_len),
                                             int(num_cu), out.ctypes.data))
    return {"items": int(out[0]), "parts": int(out[1]), "tiles": int(out[2]), "makespan_tiles": int(out[3])}


def sa_sync_check(ctx, stream=None):
    _check(load_library().sa_sync_check(_ctx_handle(ctx), _stream(stream)))


def sa_kv_append(ctx, layout: Layout, layer: int, k_pool, v_pool, k_new, v_new, start, new_len,
                 pages_indptr, pages_indices, stream=None):
    start, new_len = _host_i32(start), _host_i32(new_len)
    if start.shape != new_len.shape:
        raise ValueError("start and new_len differ in length")
    B = len(new_len)
    rows = int(new_len.astype(np.int64).sum()) * int(layout.num_kv_heads) * int(layout.head_dim)
    _check(load_library().sa_kv_append(
        _ctx_handle(ctx), ctypes.byref(layout), int(layer),
        _dev(k_pool, "k_pool", "b16", _pool_numel(layout)), _dev(v_pool, "v_pool", "b16", _pool_numel(layout)),
        _dev(k_new, "k_new", "b16", rows, nullable=rows == 0), _dev(v_new, "v_new", "b16", rows, nullable=rows == 0),
        int(B), _ptr(start), _ptr(new_len), _pages(pages_indptr, pages_indices, B), _stream(stream)))


def _splice_host(layout, src_len, keep_indptr, keep_spans, reserve):
    src_len, reserve = _host_i32(src_len), _host_i32(reserve)
    keep_indptr = _host_i32(keep_indptr)
    keep_spans = _host_i32(np.asarray(keep_spans).reshape(-1))
    B = len(src_len)
    if len(reserve) != B or len(keep_indptr) != B + 1:
        raise ValueError("per-sequence arrays disagree on the batch size")
    return src_len, keep_indptr, keep_spans, reserve, B


def _splice_dev(layout, B, k_src, v_src, k_dst, v_dst, src_indptr, src_indices, fresh, dst_indptr,
                dst_indices, fresh_nullable=False):
    n = _pool_numel(layout)
    return (_dev(k_src, "k_src", "b16", n), _dev(v_src, "v_src", "b16", n),
            _dev(k_dst, "k_dst", "b16", n), _dev(v_dst, "v_dst", "b16", n),
            _Pages(_dev(src_indptr, "src indptr", "i32", B + 1),
                   _dev(src_indices, "src indices", "i32", 0, nullable=True)),
            _dev(fresh, "fresh", "i32", 0, nullable=fresh_nullable),
            0 if fresh is None else int(fresh.numel()),
            _dev(dst_indptr, "dst indptr", "i32", B + 1),
            _dev(dst_indices, "dst indices", "i32", 0, nullable=True),
            0 if dst_indices is None else int(dst_indices.numel()))


def sa_kv_assemble(ctx, layout: Layout, k_src, v_src, k_dst, v_dst, src_len, keep_indptr,
                   keep_spans, reserve, src_indptr, src_indices, fresh, dst_indptr, dst_indices,
                   stream=None):
    """Returns the kept token count of every sequence (numpy int32)."""
    src_len, keep_indptr, keep_spans, reserve, B = _splice_host(layout, src_len, keep_indptr, keep_spans,
                                                                reserve)
    ks, vs, kd, vd, src, fr, nfr, dip, dix, cap = _splice_dev(layout, B, k_src, v_src, k_dst, v_dst,
                                                              src_indptr, src_indices, fresh, dst_indptr,
                                                              dst_indices)
    dst_len = np.zeros(B, dtype=np.int32)
    _check(load_library().sa_kv_assemble(
        _ctx_handle(ctx), ctypes.byref(layout), ks, vs, kd, vd, B, _ptr(src_len), _ptr(keep_indptr),
        _ptr(keep_spans) if keep_spans.size else None, _ptr(reserve), src, fr, nfr, dip, dix, cap,
        _ptr(dst_len), _stream(stream)))
    return dst_len


def sa_kv_assemble_append(ctx, layout: Layout, k_src, v_src, k_dst, v_dst, src_len, keep_indptr,
                          keep_spans, reserve, src_indptr, src_indices, fresh, dst_indptr, dst_indices,
                          layer, k_new, v_new, new_len, stream=None):
    """Splice and the segment's append in one launch.  Returns the kept token
    count of every sequence (numpy int32); the new rows follow it."""
    src_len, keep_indptr, keep_spans, reserve, B = _splice_host(layout, src_len, keep_indptr, keep_spans,
                                                                reserve)
    new_len = _host_i32(new_len)
    if len(new_len) != B:
        raise ValueError("per-sequence arrays disagree on the batch size")
    ks, vs, kd, vd, src, fr, nfr, dip, dix, cap = _splice_dev(layout, B, k_src, v_src, k_dst, v_dst,
                                                              src_indptr, src_indices, fresh, dst_indptr,
                                                              dst_indices)
    rows = int(new_len.astype(np.int64).sum()) * int(layout.num_kv_heads) * int(layout.head_dim)
    dst_len = np.zeros(B, dtype=np.int32)
    _check(load_library().sa_kv_assemble_append(
        _ctx_handle(ctx), ctypes.byref(layout), ks, vs, kd, vd, B, _ptr(src_len), _ptr(keep_indptr),
        _ptr(keep_spans) if keep_spans.size else None, _ptr(reserve), src, fr, nfr, dip, dix, cap,
        _ptr(dst_len), int(layer), _dev(k_new, "k_new", "b16", rows, nullable=rows == 0),
        _dev(v_new, "v_new", "b16", rows, nullable=rows == 0), _ptr(new_len), _stream(stream)))
    return dst_len


def sa_kv_splice_alias(ctx, layout: Layout, src_len, keep_indptr, keep_spans, reserve, src_indptr,
                       src_indices, fresh, dst_indptr, dst_indices, stream=None):
    """Zero-copy splice: the destination table shares the surviving source slots.
    Returns the kept token count of every sequence (numpy int32)."""
    src_len, keep_indptr, keep_spans, reserve, B = _splice_host(layout, src_len, keep_indptr, keep_spans,
                                                                reserve)
    dst_len = np.zeros(B, dtype=np.int32)
    _check(load_library().sa_kv_splice_alias(
        _ctx_handle(ctx), ctypes.byref(layout), B, _ptr(src_len), _ptr(keep_indptr),
        _ptr(keep_spans) if keep_spans.size else None, _ptr(reserve),
        _Pages(_dev(src_indptr, "src indptr", "i32", B + 1),
               _dev(src_indices, "src indices", "i32", 0, nullable=True)),
        _dev(fresh, "fresh", "i32", 0, nullable=True), 0 if fresh is None else int(fresh.numel()),
        _dev(dst_indptr, "dst indptr", "i32", B + 1), _dev(dst_indices, "dst indices", "i32", 0, nullable=True),
        0 if dst_indices is None else int(dst_indices.numel()), _ptr(dst_len), _stream(stream)))
    return dst_len


def _attn_dev(layout, q_len, q, o, lse):
    T = int(q_len.astype(np.int64).sum())
    n = T * int(layout.num_q_heads) * int(layout.head_dim)
    return (_dev(q, "q", "b16", n, nullable=T == 0), _dev(o, "o", "b16", n, nullable=T == 0),
            _dev(lse, "lse", "f32", T * int(layout.num_q_heads), nullable=True), T)


def sa_segment_prefill_attn(ctx, layout: Layout, layer: int, q, k_pool, v_pool, q_len, kv_len,
                            pages_indptr, pages_indices, softmax_scale: float, o, lse=None,
                            stream=None):
    q_len, kv_len = _host_i32(q_len), _host_i32(kv_len)
    if q_len.shape != kv_len.shape:
        raise ValueError("q_len and kv_len differ in length")
    qp, op, lp, _ = _attn_dev(layout, q_len, q, o, lse)
    n = _pool_numel(layout)
    _check(load_library().sa_segment_prefill_attn(
        _ctx_handle(ctx), ctypes.byref(layout), int(layer), qp, _dev(k_pool, "k_pool", "b16", n),
        _dev(v_pool, "v_pool", "b16", n), int(len(q_len)), _ptr(q_len), _ptr(kv_len),
        _pages(pages_indptr, pages_indices, len(q_len)), float(softmax_scale), op, lp, _stream(stream)))


def sa_segment_prefill_attn_noalloc(ctx, layout: Layout, layer: int, q, k_pool, v_pool, q_len, kv_len,
                                    pages_indptr, pages_indices, softmax_scale: float, o, lse=None, stream=None):
    """sa_segment_prefill_attn without any device allocation: plan and split partials in the
    library's fixed per-GPU scratch array (calls on one GPU must not overlap in time)."""
    q_len, kv_len = _host_i32(q_len), _host_i32(kv_len)
    if q_len.shape != kv_len.shape:
        raise ValueError("q_len and kv_len differ in length")
    qp, op, lp, _ = _attn_dev(layout, q_len, q, o, lse)
    n = _pool_numel(layout)
    _check(load_library().sa_segment_prefill_attn_noalloc(
        _ctx_handle(ctx), ctypes.byref(layout), int(layer), qp, _dev(k_pool, "k_pool", "b16", n),
        _dev(v_pool, "v_pool", "b16", n), int(len(q_len)), _ptr(q_len), _ptr(kv_len),
        _pages(pages_indptr, pages_indices, len(q_len)), float(softmax_scale), op, lp, _stream(stream)))


def sa_set_exact_scale(ctx, enable: bool = True):
    """Later attention calls on ctx apply the softmax scale to each score in fp32
    (enable, the default) or fold it into the bf16 query rows."""
    _check(load_library().sa_set_exact_scale(_ctx_handle(ctx), int(bool(enable))))


def sa_set_fused_append(ctx, enable: bool = True):
    """Later sa_segment_prefill_attn_append calls on ctx write the segment's rows
    inside the attention launch (enable) or with an append launch before it (the
    default)."""
    _check(load_library().sa_set_fused_append(_ctx_handle(ctx), int(bool(enable))))


def sa_set_block_clock(ctx, buf=None) -> int:
    """Later launches of the default attention kernel on ctx write, per workgroup,
    four int64 words into buf (a device int64 tensor of 4 x max workgroups):
    start and end clock, sequence, q_len.  Returns the clock's rate in kHz.
    None clears."""
    khz = ctypes.c_int64(0)
    if buf is not None and (not hasattr(buf, "element_size") or buf.element_size() != 8 or not buf.is_cuda
                            or not buf.is_contiguous()):
        raise ValueError("sa_set_block_clock needs a contiguous device tensor of 8-byte elements")
    n = 0 if buf is None else buf.numel() // 4
    _check(load_library().sa_set_block_clock(_ctx_handle(ctx), None if buf is None else buf.data_ptr(), n,
                                             ctypes.byref(khz)))
    return int(khz.value)


def sa_set_xcd_weights(ctx, speeds=None):
    """Relative speeds of the 8 XCDs for the attention planner (None: equal)."""
    if speeds is None:
        _check(load_library().sa_set_xcd_weights(_ctx_handle(ctx), None))
        return
    w = np.ascontiguousarray(speeds, dtype=np.float32)
    if w.shape != (8,):
        raise ValueError("sa_set_xcd_weights needs 8 speeds")
    _check(load_library().sa_set_xcd_weights(_ctx_handle(ctx), w.ctypes.data))


TIMED_ATTN, TIMED_PAGES = 0, 1


def sa_set_kernel_events(ctx, which: int, start_event=None, stop_event=None):
    """Later kernels of kind `which` (TIMED_ATTN, TIMED_PAGES) on ctx are launched
    bound to these two hipEvent_t handles (ints), which then time the kernel
    itself; None, None clears."""
    _check(load_library().sa_set_kernel_events(_ctx_handle(ctx), int(which), start_event or None,
                                               stop_event or None))


def sa_segment_prefill_attn_append(ctx, layout: Layout, layer: int, q, k_pool, v_pool, k_new, v_new, q_len,
                                   kv_len, pages_indptr, pages_indices, softmax_scale: float, o, lse=None,
                                   stream=None):
    """Writes each sequence's q_len new K/V rows at positions kv_len - q_len .. kv_len - 1,
    then runs sa_segment_prefill_attn over the result."""
    q_len, kv_len = _host_i32(q_len), _host_i32(kv_len)
    if q_len.shape != kv_len.shape:
        raise ValueError("q_len and kv_len differ in length")
    qp, op, lp, T = _attn_dev(layout, q_len, q, o, lse)
    rows = T * int(layout.num_kv_heads) * int(layout.head_dim)
    n = _pool_numel(layout)
    _check(load_library().sa_segment_prefill_attn_append(
        _ctx_handle(ctx), ctypes.byref(layout), int(layer), qp, _dev(k_pool, "k_pool", "b16", n),
        _dev(v_pool, "v_pool", "b16", n), _dev(k_new, "k_new", "b16", rows, nullable=T == 0),
        _dev(v_new, "v_new", "b16", rows, nullable=T == 0), int(len(q_len)), _ptr(q_len), _ptr(kv_len),
        _pages(pages_indptr, pages_indices, len(q_len)), float(softmax_scale), op, lp, _stream(stream)))
