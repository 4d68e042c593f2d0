"""CPU oracle for the tile-major GEMM path -- TEST INFRASTRUCTURE ONLY.

Only tests/, ``__graft_entry__.smoke()`` and bench.py's ``cpu_baseline`` leg
may import this package.  The product library (``paper_2607_04031_amd``) never
imports it, and it imports nothing from the product library.

The arithmetic lives in ``tl_oracle.c`` (plain C, fp64, '/' and '%' only);
this module is argument marshalling over ctypes plus numpy buffers.

What each function follows (TileLens, arxiv 2607.04031):
  tm_offset      Eq. 1 and Eq. 2, Section 3.2; Section 3.3 (a dimension that
                 is not a multiple of the memory tile is padded to whole tiles)
  packed_bytes   Section 3.3: bytes of the padded tile-major copy
  repack/unpack  Section 3.2 (the permutation Eq. 2 defines, padding zero);
                 Section 5.1 (weights are written in this order once, at
                 load time)
  gemm_f64       Section 2.3 (C = A W^T over the K dimension), fp64
  grouped_gemm_f64  the expert GEMMs of a mixture-of-experts layer (Sections
                 2.3 and 6.2): per group, gather its rows of A and apply
                 gemm_f64 with that group's weight
  view_offsets   Section 4.3: tile-major byte offsets of the elements of a
                 box of a multi-dimensional view (linear index -> (i, j) ->
                 Eq. 2), in the order a TMA load visits them
  silu / swiglu_f64 / grouped_swiglu_f64  the gated expert activation of
                 fused_moe (Sections 2.3 and 6.2): silu(x W_gate^T) * (x W_up^T)
                 with gate and up stacked in one [2I, K] weight, per group
  fp8_e4m3 / gemm_w8_f64  the FP8 weights the paper's 64 x 64 memory tile
                 holds (Section 3.1): OCP E4M3 decoded by its definition, and
                 the GEMM over them with per-output-channel scales, fp64
  round_bf16     round-to-nearest-even to 8 significant bits
  read_amp       Sections 1, 2.5 and 6.5 (requests per compute tile at
                 granularity G; weights only, Section 5.1)
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

NK_ROW, KN_ROW, TILE = 0, 1, 2


class Amp(ctypes.Structure):
    _fields_ = [("compute_tiles", ctypes.c_int64),
                ("requests", ctypes.c_int64),
                ("fetched_bytes", ctypes.c_int64),
                ("useful_bytes", ctypes.c_int64),
                ("unique_blocks", ctypes.c_int64),
                ("min_blocks_per_tile", ctypes.c_int64),
                ("max_blocks_per_tile", ctypes.c_int64),
                ("amp", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, p = ctypes.c_int64, ctypes.c_void_p
    lib.orc_tm_offset.restype = i64
    lib.orc_tm_offset.argtypes = [i64] * 6
    lib.orc_packed_bytes.restype = i64
    lib.orc_packed_bytes.argtypes = [i64] * 5
    lib.orc_elem_offset.restype = i64
    lib.orc_elem_offset.argtypes = [ctypes.c_int] + [i64] * 7
    lib.orc_repack.restype = None
    lib.orc_repack.argtypes = [p, p] + [i64] * 5
    lib.orc_unpack.restype = None
    lib.orc_unpack.argtypes = [p, p] + [i64] * 5
    lib.orc_gemm_f64.restype = None
    lib.orc_gemm_f64.argtypes = [p, p, p, i64, i64, i64]
    lib.orc_gemm_f64_points.restype = None
    lib.orc_gemm_f64_points.argtypes = [p, p, p, p, p, i64, i64]
    lib.orc_round_bf16.restype = ctypes.c_uint16
    lib.orc_round_bf16.argtypes = [ctypes.c_double]
    lib.orc_round_bf16_array.restype = None
    lib.orc_round_bf16_array.argtypes = [p, p, i64]
    lib.orc_fp8_e4m3.restype = ctypes.c_double
    lib.orc_fp8_e4m3.argtypes = [ctypes.c_uint8]
    lib.orc_gemm_w8_f64.restype = None
    lib.orc_gemm_w8_f64.argtypes = [p, p, p, p, i64, i64, i64]
    lib.orc_silu.restype = ctypes.c_double
    lib.orc_silu.argtypes = [ctypes.c_double]
    lib.orc_swiglu_f64.restype = None
    lib.orc_swiglu_f64.argtypes = [p, p, p, i64, i64, i64]
    lib.orc_view_offsets.restype = i64
    lib.orc_view_offsets.argtypes = [ctypes.c_int, p, p, p, i64, i64, i64, i64, p]
    lib.orc_read_amp.restype = ctypes.c_int
    lib.orc_read_amp.argtypes = [i64] * 6 + [ctypes.c_int] + [i64] * 4 + [
        ctypes.c_int, ctypes.POINTER(Amp)]
    _lib = lib
    return lib


def set_threads(n: int) -> None:
    """OpenMP threads of the oracle's parallel loops (for timing only: every
    output element is summed by one thread in a fixed order, so results do
    not depend on it)."""
    _load().omp_set_num_threads(ctypes.c_int(int(n)))


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def tm_offset(r: int, c: int, cols: int, s: int, G: int, block_rows: int) -> int:
    """Eq. 2 byte offset of stored element (r, c); c is the contiguous index."""
    return _load().orc_tm_offset(r, c, cols, s, G, block_rows)


def elem_offset(kind: int, n: int, k: int, N: int, K: int, s: int,
                layout_G: int = 4096, block_rows: int = 32) -> int:
    return _load().orc_elem_offset(kind, n, k, N, K, s, layout_G, block_rows)


def _as_bytes(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x).view(np.uint8).reshape(-1)


def packed_bytes(rows: int, cols: int, s: int, G: int, block_rows: int) -> int:
    """Bytes of the tile-major copy: whole memory tiles (Section 3.3)."""
    return _load().orc_packed_bytes(rows, cols, s, G, block_rows)


def padded_shape(rows: int, cols: int, s: int, G: int, block_rows: int):
    """(rows, cols) rounded up to whole memory tiles of block_rows x G / (s * block_rows)."""
    a = G // (s * block_rows)
    return (-(-rows // block_rows) * block_rows, -(-cols // a) * a)


def repack(src: np.ndarray, G: int, block_rows: int) -> np.ndarray:
    """Row-major [rows, cols] -> tile-major copy, same dtype, shape rounded up
    to whole memory tiles (= the input's shape when the tile divides it);
    padding elements are zero."""
    rows, cols = src.shape
    s = src.dtype.itemsize
    out = np.empty(padded_shape(rows, cols, s, G, block_rows), dtype=src.dtype)
    assert out.nbytes == packed_bytes(rows, cols, s, G, block_rows)
    _load().orc_repack(_ptr(_as_bytes(src)), _ptr(out), rows, cols, s, G, block_rows)
    return out


def unpack(src_tm: np.ndarray, G: int, block_rows: int, rows: int = None, cols: int = None) -> np.ndarray:
    """Tile-major copy -> row-major [rows, cols] (default: src_tm's shape)."""
    rows = src_tm.shape[0] if rows is None else rows
    cols = src_tm.shape[1] if cols is None else cols
    s = src_tm.dtype.itemsize
    assert src_tm.nbytes >= packed_bytes(rows, cols, s, G, block_rows)
    out = np.empty((rows, cols), dtype=src_tm.dtype)
    _load().orc_unpack(_ptr(_as_bytes(src_tm)), _ptr(out), rows, cols, s, G, block_rows)
    return out


def view_offsets(strides, coords, box, K: int, s: int, G: int, block_rows: int) -> np.ndarray:
    """int64 byte offsets, dimension 0 fastest, of every element of the box."""
    rank = len(box)
    assert len(strides) == len(coords) == rank <= 8
    st = np.ascontiguousarray(strides, dtype=np.int64)
    co = np.ascontiguousarray(coords, dtype=np.int64)
    bx = np.ascontiguousarray(box, dtype=np.int64)
    out = np.empty(int(np.prod(bx)), dtype=np.int64)
    _load().orc_view_offsets(rank, _ptr(st), _ptr(co), _ptr(bx), K, s, G, block_rows, _ptr(out))
    return out


def view_gather(src_tm: np.ndarray, strides, coords, box, K: int, s: int, G: int, block_rows: int) -> np.ndarray:
    """Bytes of the box's elements from a tile-major buffer, in view order (uint8 [elements * s])."""
    offs = view_offsets(strides, coords, box, K, s, G, block_rows)
    raw = _as_bytes(src_tm).reshape(-1)
    return raw[(offs[:, None] + np.arange(s)[None, :]).reshape(-1)]


def gemm_f64(A_bf16: np.ndarray, W_bf16: np.ndarray) -> np.ndarray:
    """A: uint16 bf16 bits [M,K]; W: uint16 bf16 bits [N,K] ROW-MAJOR -> fp64 [M,N]."""
    A = np.ascontiguousarray(A_bf16, dtype=np.uint16)
    W = np.ascontiguousarray(W_bf16, dtype=np.uint16)
    M, K = A.shape
    N, K2 = W.shape
    assert K == K2
    Y = np.empty((M, N), dtype=np.float64)
    _load().orc_gemm_f64(_ptr(A), _ptr(W), _ptr(Y), M, N, K)
    return Y


def grouped_gemm_f64(A_bf16: np.ndarray, token_ids, offsets, W_list) -> np.ndarray:
    """Rows [offsets[e], offsets[e+1]) of the result are A[token_ids[r]] @ W_list[e]^T
    (token_ids None: A[r]); fp64 [offsets[-1], N].  Empty groups contribute nothing."""
    offsets = [int(x) for x in offsets]
    assert len(offsets) == len(W_list) + 1 and offsets[0] == 0
    N = W_list[0].shape[0]
    Y = np.zeros((offsets[-1], N), dtype=np.float64)
    for e, W in enumerate(W_list):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 <= r0:
            continue
        rows = np.arange(r0, r1) if token_ids is None else np.asarray(token_ids[r0:r1], dtype=np.int64)
        Y[r0:r1] = gemm_f64(A_bf16[rows], W)
    return Y


def silu(x: float) -> float:
    return _load().orc_silu(float(x))


def swiglu_f64(A_bf16: np.ndarray, W_bf16: np.ndarray) -> np.ndarray:
    """A: uint16 bf16 bits [M,K]; W: [2I,K] (gate rows then up rows) -> fp64 [M,I]."""
    A = np.ascontiguousarray(A_bf16, dtype=np.uint16)
    W = np.ascontiguousarray(W_bf16, dtype=np.uint16)
    M, K = A.shape
    I2, K2 = W.shape
    assert K == K2 and I2 % 2 == 0
    H = np.empty((M, I2 // 2), dtype=np.float64)
    _load().orc_swiglu_f64(_ptr(A), _ptr(W), _ptr(H), M, I2 // 2, K)
    return H


def grouped_swiglu_f64(A_bf16: np.ndarray, token_ids, offsets, W_list) -> np.ndarray:
    """Rows [offsets[e], offsets[e+1]) are swiglu_f64(A[token_ids[r]], W_list[e]) (token_ids None: A[r])."""
    offsets = [int(x) for x in offsets]
    assert len(offsets) == len(W_list) + 1 and offsets[0] == 0
    I = W_list[0].shape[0] // 2
    H = np.zeros((offsets[-1], I), dtype=np.float64)
    for e, W in enumerate(W_list):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 <= r0:
            continue
        rows = np.arange(r0, r1) if token_ids is None else np.asarray(token_ids[r0:r1], dtype=np.int64)
        H[r0:r1] = swiglu_f64(A_bf16[rows], W)
    return H


def fp8_e4m3(v: int) -> float:
    return _load().orc_fp8_e4m3(int(v))


def gemm_w8_f64(A_bf16: np.ndarray, W_fp8: np.ndarray, scales=None) -> np.ndarray:
    """A: uint16 bf16 bits [M,K]; W_fp8: uint8 E4M3 bytes [N,K] row-major; scales: [N] or None -> fp64 [M,N]."""
    A = np.ascontiguousarray(A_bf16, dtype=np.uint16)
    W = np.ascontiguousarray(W_fp8, dtype=np.uint8)
    M, K = A.shape
    N, K2 = W.shape
    assert K == K2
    sc = None if scales is None else np.ascontiguousarray(scales, dtype=np.float64)
    Y = np.empty((M, N), dtype=np.float64)
    _load().orc_gemm_w8_f64(_ptr(A), _ptr(W), None if sc is None else _ptr(sc), _ptr(Y), M, N, K)
    return Y


def gemm_f64_points(A_bf16: np.ndarray, W_bf16: np.ndarray, ms, ns) -> np.ndarray:
    A = np.ascontiguousarray(A_bf16, dtype=np.uint16)
    W = np.ascontiguousarray(W_bf16, dtype=np.uint16)
    ms = np.ascontiguousarray(ms, dtype=np.int64)
    ns = np.ascontiguousarray(ns, dtype=np.int64)
    assert ms.shape == ns.shape
    y = np.empty(ms.shape, dtype=np.float64)
    _load().orc_gemm_f64_points(_ptr(A), _ptr(W), _ptr(ms), _ptr(ns), _ptr(y),
                                ms.size, A.shape[1])
    return y


def round_bf16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().orc_round_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


def read_amp(M: int, N: int, K: int, tm: int, tn: int, tk: int, kind: int,
             G: int, s: int = 2, layout_G: int = 4096, block_rows: int = 32,
             brute_m: bool = False) -> dict:
    """Brute-force read amplification (see tl_oracle.c for the model)."""
    out = Amp()
    rc = _load().orc_read_amp(M, N, K, tm, tn, tk, kind, s, layout_G, block_rows, G,
                              1 if brute_m else 0, ctypes.byref(out))
    if rc != 0:
        raise ValueError("orc_read_amp: bad arguments")
    return out.as_dict()
