"""Tile-major GEMM for AMD MI355X (gfx950): Python binding over libtl's C ABI.

Every step of the path runs in libtl's HIP kernels; this module only marshals
arguments (torch tensors -> device pointers, the current torch stream -> a
hipStream_t) and turns status codes into exceptions.  The entry points carry
the C names and argument order of ``include/tl.h``:

    tl_tile_bytes(rows, cols, elem_bytes, G, block_rows) -> int
    tl_repack(src, dst, rows, cols, elem_bytes, G, block_rows, stream=None)
    tl_unpack(src_tm, dst, rows, cols, elem_bytes, G, block_rows, stream=None)
    tl_gemm(A, W, C, M, N, K, layout, fetch_mode, stream=None)
    tl_gemm_noalloc(A, W, C, M, N, K, layout, fetch_mode, stream=None)
    tl_gemm_plan(M, N, K, layout, fetch_mode) -> dict
    tl_gemm_grouped / tl_gemm_grouped_swiglu (..., layout, fetch_mode, stream=None)
    tl_read_amp(M, N, K, tile_m, tile_n, tile_k, layout, G) -> dict
    tl_fetch_counter_read(stream=None) -> int
    tl_release()
    tl_strerror(status) -> str

Pointer arguments accept a torch CUDA tensor or a raw integer address.
``layout`` is a :class:`LayoutDesc` (or a dict of its fields).  A few helpers
(``repack``, ``gemm``, ``layout``) build outputs and descriptors for callers
that just hold tensors.

If libtl.so has not been built the first call raises ``ImportError``; there is
no fallback path of any kind.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtl.so")

TL_OK, TL_EINVAL, TL_EUNSUPPORTED, TL_EHIP, TL_ENOMEM, TL_ESCRATCH = 0, -1, -2, -3, -4, -5
TL_NOALLOC_SCRATCH_BYTES = 64 << 20
TL_LAYOUT_NK_ROW, TL_LAYOUT_KN_ROW, TL_LAYOUT_TILE = 0, 1, 2
TL_OUT_F32, TL_OUT_BF16 = 0, 1
TL_FETCH_NATIVE, TL_FETCH_BLOCK, TL_FETCH_COUNT = 0, 1, 0x100

EXPORTED = ("tl_tile_bytes", "tl_repack", "tl_unpack", "tl_gemm", "tl_gemm_noalloc", "tl_gemm_w8", "tl_gemm_plan", "tl_gemm_grouped", "tl_gemm_grouped_swiglu", "tl_read_amp",
            "tl_view_offsets", "tl_view_load", "tl_prefetch_degree", "tl_gemm_lgms", "tl_lgms_occupancy",
            "tl_stream_read", "tl_fetch_counter_read", "tl_release", "tl_strerror")
TL_VIEW_MAX_RANK = 5


class View(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32),
                ("box", ctypes.c_int32 * 5),
                ("strides", ctypes.c_int64 * 5),
                ("coords", ctypes.c_int64 * 5)]


def view(strides, coords, box) -> View:
    """tl_view of rank len(box); dimension 0 is the contiguous one."""
    v = View()
    v.rank = len(box)
    assert len(strides) == len(coords) == v.rank <= 5
    for d in range(v.rank):
        v.box[d], v.strides[d], v.coords[d] = int(box[d]), int(strides[d]), int(coords[d])
    return v


class LayoutDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32),
                ("elem_bytes", ctypes.c_int32),
                ("G", ctypes.c_int64),
                ("block_rows", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32),
                ("tile_m", ctypes.c_int32),
                ("tile_n", ctypes.c_int32),
                ("tile_k", ctypes.c_int32),
                ("split_k", ctypes.c_int32)]


class Amp(ctypes.Structure):
    _fields_ = [("compute_tiles", ctypes.c_int64),
                ("requests", ctypes.c_int64),
                ("fetched_bytes", ctypes.c_int64),
                ("useful_bytes", ctypes.c_int64),
                ("unique_blocks", ctypes.c_int64),
                ("min_blocks_per_tile", ctypes.c_int64),
                ("max_blocks_per_tile", ctypes.c_int64),
                ("amp", ctypes.c_double)]


class Plan(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32),
                ("tile_m", ctypes.c_int32),
                ("tile_n", ctypes.c_int32),
                ("tile_k", ctypes.c_int32),
                ("split_k", ctypes.c_int32),
                ("waves", ctypes.c_int32),
                ("workgroups", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64)]


def _struct_dict(s):
    return {name: getattr(s, name) for name, _ in s._fields_}


class TLError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {tl_strerror(status)} ({status})")


_lib = None


def load_library():
    """Load libtl.so (after torch, so both share torch's HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libtl.so is not built ({LIB_PATH}); run python -m paper_2607_04031_amd.build")
    import torch  # noqa: F401  (binds libtl to torch's libamdhip64)
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, p = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    lib.tl_tile_bytes.restype = ctypes.c_int
    lib.tl_tile_bytes.argtypes = [i64, i64, i32, i64, i32, ctypes.POINTER(i64)]
    lib.tl_repack.restype = ctypes.c_int
    lib.tl_repack.argtypes = [p, p, i64, i64, i32, i64, i32, p]
    lib.tl_unpack.restype = ctypes.c_int
    lib.tl_unpack.argtypes = [p, p, i64, i64, i32, i64, i32, p]
    lib.tl_gemm.restype = ctypes.c_int
    lib.tl_gemm.argtypes = [p, p, p, i64, i64, i64, ctypes.POINTER(LayoutDesc), i32, p]
    lib.tl_gemm_noalloc.restype = ctypes.c_int
    lib.tl_gemm_noalloc.argtypes = [p, p, p, i64, i64, i64, ctypes.POINTER(LayoutDesc), i32, p]
    lib.tl_gemm_w8.restype = ctypes.c_int
    lib.tl_gemm_w8.argtypes = [p, p, p, p, i64, i64, i64, ctypes.POINTER(LayoutDesc), i32, p]
    lib.tl_gemm_plan.restype = ctypes.c_int
    lib.tl_gemm_plan.argtypes = [i64, i64, i64, ctypes.POINTER(LayoutDesc), i32, ctypes.POINTER(Plan)]
    lib.tl_gemm_grouped.restype = ctypes.c_int
    lib.tl_gemm_grouped.argtypes = [p, i64, p, p, i32, i64, i64, p, i64, p, i64, i64,
                                    ctypes.POINTER(LayoutDesc), i32, p]
    lib.tl_gemm_grouped_swiglu.restype = ctypes.c_int
    lib.tl_gemm_grouped_swiglu.argtypes = [p, i64, p, p, i32, i64, i64, p, i64, p, i64, i64,
                                           ctypes.POINTER(LayoutDesc), i32, p]
    lib.tl_prefetch_degree.restype = ctypes.c_int
    lib.tl_prefetch_degree.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double, i64, ctypes.c_double,
                                       ctypes.POINTER(i64)]
    lib.tl_gemm_lgms.restype = ctypes.c_int
    lib.tl_gemm_lgms.argtypes = [p, p, p, i64, i64, i64, ctypes.POINTER(LayoutDesc), i64, i32, p]
    lib.tl_lgms_occupancy.restype = ctypes.c_int
    lib.tl_lgms_occupancy.argtypes = [i32, ctypes.POINTER(i32)]
    lib.tl_view_offsets.restype = ctypes.c_int
    lib.tl_view_offsets.argtypes = [ctypes.POINTER(View), i64, i64, i32, i64, i32, p, i64, ctypes.POINTER(i64)]
    lib.tl_view_load.restype = ctypes.c_int
    lib.tl_view_load.argtypes = [p, ctypes.POINTER(View), i64, i64, i32, i64, i32, p, p]
    lib.tl_read_amp.restype = ctypes.c_int
    lib.tl_read_amp.argtypes = [i64, i64, i64, i32, i32, i32, ctypes.POINTER(LayoutDesc), i64,
                                ctypes.POINTER(Amp)]
    lib.tl_stream_read.restype = ctypes.c_int
    lib.tl_stream_read.argtypes = [p, i64, p, p]
    lib.tl_fetch_counter_read.restype = ctypes.c_int
    lib.tl_fetch_counter_read.argtypes = [p, ctypes.POINTER(i64)]
    lib.tl_release.restype = ctypes.c_int
    lib.tl_release.argtypes = []
    lib.tl_strerror.restype = ctypes.c_char_p
    lib.tl_strerror.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        if not x.is_cuda:
            raise ValueError("libtl needs device tensors")
        if not x.is_contiguous():
            raise ValueError("libtl needs contiguous tensors")
        return x.data_ptr()
    raise TypeError(f"cannot pass {type(x)!r} as a device pointer")


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _desc(layout) -> LayoutDesc:
    if isinstance(layout, LayoutDesc):
        return layout
    d = LayoutDesc()
    d.kind, d.elem_bytes, d.G, d.block_rows = TL_LAYOUT_TILE, 2, 4096, 32
    for k, v in dict(layout).items():
        setattr(d, k, v)
    return d


def _check(rc: int, where: str):
    if rc != TL_OK:
        raise TLError(rc, where)


# ---------------------------------------------------------------------------
# C ABI, same names and argument order
# ---------------------------------------------------------------------------

def tl_tile_bytes(rows, cols, elem_bytes, G, block_rows) -> int:
    out = ctypes.c_int64()
    _check(load_library().tl_tile_bytes(rows, cols, elem_bytes, G, block_rows, ctypes.byref(out)), "tl_tile_bytes")
    return out.value


def tl_repack(src, dst, rows, cols, elem_bytes, G, block_rows, stream=None):
    _check(load_library().tl_repack(_ptr(src), _ptr(dst), rows, cols, elem_bytes, G, block_rows,
                                    _stream(stream)), "tl_repack")


def tl_unpack(src_tm, dst, rows, cols, elem_bytes, G, block_rows, stream=None):
    _check(load_library().tl_unpack(_ptr(src_tm), _ptr(dst), rows, cols, elem_bytes, G, block_rows,
                                    _stream(stream)), "tl_unpack")


def tl_gemm(A, W, C, M, N, K, layout, fetch_mode=TL_FETCH_BLOCK, stream=None):
    d = _desc(layout)
    _check(load_library().tl_gemm(_ptr(A), _ptr(W), _ptr(C), M, N, K, ctypes.byref(d), fetch_mode,
                                  _stream(stream)), "tl_gemm")


def tl_gemm_noalloc(A, W, C, M, N, K, layout, fetch_mode=TL_FETCH_BLOCK, stream=None):
    d = _desc(layout)
    _check(load_library().tl_gemm_noalloc(_ptr(A), _ptr(W), _ptr(C), M, N, K, ctypes.byref(d), fetch_mode,
                                          _stream(stream)), "tl_gemm_noalloc")


def tl_gemm_w8(A, W_fp8, scales, C, M, N, K, layout, fetch_mode=TL_FETCH_BLOCK, stream=None):
    """scales may be None (all 1)."""
    d = _desc(layout)
    _check(load_library().tl_gemm_w8(_ptr(A), _ptr(W_fp8), _ptr(scales), _ptr(C), M, N, K, ctypes.byref(d),
                                     fetch_mode, _stream(stream)), "tl_gemm_w8")


def tl_gemm_plan(M, N, K, layout, fetch_mode=TL_FETCH_BLOCK) -> dict:
    d = _desc(layout)
    out = Plan()
    _check(load_library().tl_gemm_plan(M, N, K, ctypes.byref(d), fetch_mode, ctypes.byref(out)),
           "tl_gemm_plan")
    return _struct_dict(out)


def tl_gemm_grouped(A, a_rows, token_ids, group_offsets, num_groups, total_rows, max_group_rows, W,
                    group_stride, C, N, K, layout, fetch_mode=TL_FETCH_BLOCK, stream=None):
    """token_ids may be None (row r of C reads row r of A)."""
    d = _desc(layout)
    _check(load_library().tl_gemm_grouped(_ptr(A), a_rows, _ptr(token_ids), _ptr(group_offsets), num_groups,
                                          total_rows, max_group_rows, _ptr(W), group_stride, _ptr(C), N, K,
                                          ctypes.byref(d), fetch_mode, _stream(stream)), "tl_gemm_grouped")


def tl_gemm_grouped_swiglu(A, a_rows, token_ids, group_offsets, num_groups, total_rows, max_group_rows, W_gate_up,
                           group_stride, H, I, K, layout, fetch_mode=TL_FETCH_BLOCK, stream=None):
    """H [total_rows, I] = silu(A W_gate^T) * (A W_up^T) per group; W_gate_up stacks [2I, K] per group."""
    d = _desc(layout)
    _check(load_library().tl_gemm_grouped_swiglu(_ptr(A), a_rows, _ptr(token_ids), _ptr(group_offsets), num_groups,
                                                 total_rows, max_group_rows, _ptr(W_gate_up), group_stride, _ptr(H),
                                                 I, K, ctypes.byref(d), fetch_mode, _stream(stream)),
           "tl_gemm_grouped_swiglu")


def tl_prefetch_degree(bandwidth, latency, bytes_per_iteration, k_iterations, collision_factor=1.0) -> int:
    d = ctypes.c_int64(0)
    _check(load_library().tl_prefetch_degree(float(bandwidth), float(latency), float(bytes_per_iteration),
                                             int(k_iterations), float(collision_factor), ctypes.byref(d)),
           "tl_prefetch_degree")
    return d.value


def tl_gemm_lgms(A, W, C, M, N, K, layout, latency_ns, steps_in_flight, stream=None):
    d = _desc(layout)
    _check(load_library().tl_gemm_lgms(_ptr(A), _ptr(W), _ptr(C), M, N, K, ctypes.byref(d), int(latency_ns),
                                       int(steps_in_flight), _stream(stream)), "tl_gemm_lgms")


def tl_lgms_occupancy(steps_in_flight) -> int:
    n = ctypes.c_int32(0)
    _check(load_library().tl_lgms_occupancy(int(steps_in_flight), ctypes.byref(n)), "tl_lgms_occupancy")
    return n.value


def tl_view_offsets(v: View, K, N, elem_bytes, G, block_rows):
    """numpy int64 byte offsets of the box's elements (view order)."""
    import numpy as np
    lib = load_library()
    n = ctypes.c_int64(0)
    _check(lib.tl_view_offsets(ctypes.byref(v), K, N, elem_bytes, G, block_rows, None, 0, ctypes.byref(n)),
           "tl_view_offsets")
    out = np.empty(n.value, dtype=np.int64)
    _check(lib.tl_view_offsets(ctypes.byref(v), K, N, elem_bytes, G, block_rows, out.ctypes.data, n.value,
                               ctypes.byref(n)), "tl_view_offsets")
    return out


def tl_view_load(src_tm, v: View, K, N, elem_bytes, G, block_rows, dst, stream=None):
    _check(load_library().tl_view_load(_ptr(src_tm), ctypes.byref(v), K, N, elem_bytes, G, block_rows, _ptr(dst),
                                       _stream(stream)), "tl_view_load")


def tl_read_amp(M, N, K, tile_m, tile_n, tile_k, layout, G) -> dict:
    d = _desc(layout)
    out = Amp()
    _check(load_library().tl_read_amp(M, N, K, tile_m, tile_n, tile_k, ctypes.byref(d), G,
                                      ctypes.byref(out)), "tl_read_amp")
    return _struct_dict(out)


def tl_stream_read(src, nbytes, checksum, stream=None):
    """checksum: a device uint32/int32 tensor of one element; the XOR of src's 32-bit words is XORed into it."""
    _check(load_library().tl_stream_read(_ptr(src), nbytes, _ptr(checksum), _stream(stream)), "tl_stream_read")


def tl_fetch_counter_read(stream=None) -> int:
    v = ctypes.c_int64(0)
    _check(load_library().tl_fetch_counter_read(_stream(stream), ctypes.byref(v)),
           "tl_fetch_counter_read")
    return v.value


def tl_release():
    _check(load_library().tl_release(), "tl_release")


def tl_strerror(status: int) -> str:
    return load_library().tl_strerror(status).decode()


# ---------------------------------------------------------------------------
# Tensor helpers (allocation + the calls above)
# ---------------------------------------------------------------------------

def layout(kind=TL_LAYOUT_TILE, G=4096, block_rows=32, out_dtype=TL_OUT_F32, elem_bytes=2,
           tile_m=0, tile_n=0, tile_k=0, split_k=0) -> LayoutDesc:
    return _desc(dict(kind=kind, G=G, block_rows=block_rows, out_dtype=out_dtype,
                      elem_bytes=elem_bytes, tile_m=tile_m, tile_n=tile_n, tile_k=tile_k,
                      split_k=split_k))


def padded_shape(rows, cols, elem_bytes, G=4096, block_rows=32):
    """(rows, cols) rounded up to whole memory tiles: the shape of a tensor
    that holds the tile-major copy (tl_tile_bytes bytes)."""
    bc = G // (elem_bytes * block_rows)
    return (-(-rows // block_rows) * block_rows, -(-cols // bc) * bc)


def repack(w, G=4096, block_rows=32, out=None, stream=None):
    """Tile-major copy of a 2-D device tensor, same dtype, shape rounded up
    to whole memory tiles (the input's shape when the tile divides it)."""
    import torch
    rows, cols = w.shape
    if out is None:
        out = torch.empty(padded_shape(rows, cols, w.element_size(), G, block_rows), dtype=w.dtype, device=w.device)
    tl_repack(w, out, rows, cols, w.element_size(), G, block_rows, stream)
    return out


def unpack(w_tm, G=4096, block_rows=32, rows=None, cols=None, out=None, stream=None):
    """Row-major [rows, cols] (default: w_tm's shape) from a tile-major copy."""
    import torch
    rows = w_tm.shape[0] if rows is None else rows
    cols = w_tm.shape[1] if cols is None else cols
    out = torch.empty((rows, cols), dtype=w_tm.dtype, device=w_tm.device) if out is None else out
    tl_unpack(w_tm, out, rows, cols, w_tm.element_size(), G, block_rows, stream)
    return out


def gemm(A, W, N, desc: LayoutDesc, fetch_mode=TL_FETCH_BLOCK, out=None, stream=None):
    """C = A @ W^T for bf16 A [M, K] and a bf16 weight of logical shape [N, K]."""
    import torch
    M, K = A.shape
    dt = torch.bfloat16 if desc.out_dtype == TL_OUT_BF16 else torch.float32
    C = torch.empty((M, N), dtype=dt, device=A.device) if out is None else out
    tl_gemm(A, W, C, M, N, K, desc, fetch_mode, stream)
    return C
