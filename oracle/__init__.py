"""fp64 CPU oracle for paged GQA decode attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product (``paper_2509_04827_amd``)
never imports, links or calls it; the two share no code.

The arithmetic lives in ``vdo_oracle.c`` (plain C, fp64, OpenMP over
(request, query head)); this module only compiles it with gcc and marshals
numpy arrays through ctypes.  bf16 tensors are passed as their raw uint16 bit
patterns, so the oracle reads exactly the bytes the GPU reads.

What it computes is the plain definition of softmax attention of one query
token per request over that request's paged KV cache (the attention work the
paper attributes to N_kv in the decode latency model, Sec. 5.4, Eq. pred-itl;
paging as in PagedAttention, Sec. 2.1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vdo_oracle.c")
_LIB = os.path.join(_HERE, "libvdo_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, strict IEEE: no -ffast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
             "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
             "-o", tmp, _SRC, "-lm"],
            check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.vdo_decode_attn_f64.argtypes = [P, P, P, P, P, P, I, I, I, I, I, ctypes.c_float, I, I]
        lib.vdo_decode_attn_f64.restype = I
        lib.vdo_decode_attn_rows_f64.argtypes = [P, P, P, P, P, P, P, I, P, I, I, I, I, I,
                                                 ctypes.c_float, I, I]
        lib.vdo_decode_attn_rows_f64.restype = I
        lib.vdo_gather.argtypes = [P, P, P, P, P, P, I, I, I, I, I]
        lib.vdo_gather.restype = I
        lib.vdo_kv_append.argtypes = [P, P, P, P, P, P, I, I, I, I, I]
        lib.vdo_kv_append.restype = I
        lib.vdo_gemm_f64.argtypes = [P, P, P, I, I, I, I]
        lib.vdo_gemm_f64.restype = I
        lib.vdo_softmax_f64.argtypes = [P, I, P]
        lib.vdo_softmax_f64.restype = None
        lib.vdo_max_threads.argtypes = []
        lib.vdo_max_threads.restype = I
        _lib = lib
    return _lib


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 inputs are passed as uint16 bit patterns, got %s" % a.dtype)
    return a


def _i32(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.int32:
        raise TypeError("expected int32, got %s" % a.dtype)
    return a


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def max_threads() -> int:
    return _load().vdo_max_threads()


def decode_attn(q, k_pages, v_pages, page_table, seq_lens, scale: float,
                nthreads: int = 0) -> np.ndarray:
    """out float64 [B][Hq][D] of paged GQA decode attention.

    q uint16 [B][Hq][D]; k_pages/v_pages uint16 [num_pages][S][Hkv][D];
    page_table int32 [B][max_pages_per_seq]; seq_lens int32 [B].
    """
    q, k_pages, v_pages = _u16(q), _u16(k_pages), _u16(v_pages)
    page_table, seq_lens = _i32(page_table), _i32(seq_lens)
    B, Hq, D = q.shape
    _, S, Hkv, D2 = k_pages.shape
    assert D2 == D and v_pages.shape == k_pages.shape and seq_lens.shape == (B,)
    assert page_table.ndim == 2 and page_table.shape[0] == B
    out = np.zeros((B, Hq, D), dtype=np.float64)
    rc = _load().vdo_decode_attn_f64(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(page_table),
                                     _ptr(seq_lens), _ptr(out), B, Hq, Hkv, D, S,
                                     float(scale), page_table.shape[1], int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle vdo_decode_attn_f64 failed with code %d" % rc)
    return out


def decode_attn_rows(q, k_pages, v_pages, page_table, seq_lens, scale: float,
                     sel_b, sel_h, nthreads: int = 0) -> np.ndarray:
    """out float64 [n_sel][D] for the selected (request, query head) pairs."""
    q, k_pages, v_pages = _u16(q), _u16(k_pages), _u16(v_pages)
    page_table, seq_lens = _i32(page_table), _i32(seq_lens)
    sel_b = np.ascontiguousarray(sel_b, dtype=np.int32)
    sel_h = np.ascontiguousarray(sel_h, dtype=np.int32)
    assert sel_b.shape == sel_h.shape and sel_b.ndim == 1
    B, Hq, D = q.shape
    _, S, Hkv, _ = k_pages.shape
    out = np.zeros((sel_b.shape[0], D), dtype=np.float64)
    rc = _load().vdo_decode_attn_rows_f64(_ptr(q), _ptr(k_pages), _ptr(v_pages),
                                          _ptr(page_table), _ptr(seq_lens), _ptr(sel_b),
                                          _ptr(sel_h), sel_b.shape[0], _ptr(out), B, Hq, Hkv,
                                          D, S, float(scale), page_table.shape[1],
                                          int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle vdo_decode_attn_rows_f64 failed with code %d" % rc)
    return out


def gather(k_pages, v_pages, page_table, seq_lens):
    """(k_rows, v_rows) uint16 [sum L_b][Hkv][D] in logical token order."""
    k_pages, v_pages = _u16(k_pages), _u16(v_pages)
    page_table, seq_lens = _i32(page_table), _i32(seq_lens)
    _, S, Hkv, D = k_pages.shape
    n = int(np.clip(seq_lens, 0, None).sum())
    k_out = np.zeros((n, Hkv, D), dtype=np.uint16)
    v_out = np.zeros((n, Hkv, D), dtype=np.uint16)
    rc = _load().vdo_gather(_ptr(k_pages), _ptr(v_pages), _ptr(page_table), _ptr(seq_lens),
                            _ptr(k_out), _ptr(v_out), seq_lens.shape[0], Hkv, D, S,
                            page_table.shape[1])
    if rc != 0:
        raise RuntimeError("oracle vdo_gather failed with code %d" % rc)
    return k_out, v_out


def kv_append(k_new, v_new, k_pages, v_pages, page_table, positions) -> None:
    """In place: write k_new[b] / v_new[b] (uint16 [B][Hkv][D]) at token
    positions[b] of request b's pages; negative or out-of-table positions skip."""
    k_new, v_new = _u16(k_new), _u16(v_new)
    page_table, positions = _i32(page_table), _i32(positions)
    assert k_pages.flags.c_contiguous and v_pages.flags.c_contiguous
    assert k_pages.dtype == np.uint16 and v_pages.dtype == np.uint16
    _, S, Hkv, D = k_pages.shape
    rc = _load().vdo_kv_append(_ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages),
                               _ptr(page_table), _ptr(positions), positions.shape[0], Hkv, D, S,
                               page_table.shape[1])
    if rc != 0:
        raise RuntimeError("oracle vdo_kv_append failed with code %d" % rc)


def gemm(x, w, nthreads: int = 0) -> np.ndarray:
    """y float64 [M][N] = x [M][K] . w [N][K]^T for bf16 bit patterns (uint16)."""
    x, w = _u16(x), _u16(w)
    M, K = x.shape
    N, K2 = w.shape
    assert K2 == K
    y = np.zeros((M, N), dtype=np.float64)
    rc = _load().vdo_gemm_f64(_ptr(x), _ptr(w), _ptr(y), M, N, K, int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle vdo_gemm_f64 failed with code %d" % rc)
    return y


def softmax(s) -> np.ndarray:
    s = np.ascontiguousarray(s, dtype=np.float64)
    w = np.zeros_like(s)
    _load().vdo_softmax_f64(_ptr(s), s.shape[0], _ptr(w))
    return w
