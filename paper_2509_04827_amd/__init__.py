"""Python binding of libvdecode (paged GQA decode attention on MI355X).

Argument marshalling only: every step of the decode-attention path runs in the
HIP kernels of ``libvdecode.so``, reached through its C ABI
(``include/vdecode.h``) with ctypes.  torch is used for device memory and
streams.  There is no fallback: if the library is not built, every call
raises.

The functions carry the C names; tensors stand in for pointers (contiguous,
on the device; dtypes checked) and the sizes are read from their shapes.
step_info(workspace) reads back the step record (vd_step_info) an attention
call leaves at the head of its workspace.

    q          bf16  [num_seqs, n_q_heads, head_dim]           (cuda)
    k_pages    bf16  [num_pages, page_size, n_kv_heads, head_dim]
    v_pages    bf16  same shape as k_pages
    page_table int32 [num_seqs, max_pages_per_seq]
    seq_lens   int32 [num_seqs]
    out        bf16 or float32 [num_seqs, n_q_heads, head_dim]  (float32 sets VD_FLAG_OUT_F32)
    workspace  uint8 [>= vd_decode_workspace_size(...)]
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvdecode.so")

VD_SUCCESS = 0
VD_ERROR_INVALID_VALUE = 1
VD_ERROR_NOT_SUPPORTED = 2
VD_ERROR_WORKSPACE_TOO_SMALL = 3
VD_ERROR_LAUNCH = 4
VD_ERROR_SCRATCH_LIMIT = 5
VD_NOALLOC_SCRATCH_BYTES = 64 << 20
VD_FLAG_OUT_F32 = 1 << 0
VD_FLAG_SELF_PLAN = 1 << 1
VD_FLAG_SCORE_MFMA = 1 << 2   # matrix-core score for G <= 8 (measurement of the score paths)
VD_FLAG_RANGE_SHIFT = 8

EXPORTS = ("vd_status_string", "vd_decode_workspace_size", "vd_decode_attn", "vd_decode_attn_noalloc", "vd_decode_plan",
           "vd_decode_partial", "vd_decode_combine", "vd_decode_gather", "vd_kv_append", "vd_gemm_workspace_size", "vd_gemm_bf16",
           "vd_stream_read")


def VD_FLAG_RANGE_TILES(n: int) -> int:
    return (int(n) & 0xFF) << VD_FLAG_RANGE_SHIFT


VD_GEMM_FLAG_TILE_SHIFT = 8
VD_GEMM_FLAG_SLICES_SHIFT = 12


def VD_GEMM_FLAG_TILE(c: int) -> int:
    """vd_gemm_bf16: force tile configuration c (0..7)."""
    return ((int(c) + 1) & 0xF) << VD_GEMM_FLAG_TILE_SHIFT


def VD_GEMM_FLAG_SLICES_LOG2(l: int) -> int:
    """vd_gemm_bf16: force 2^l K slices (l <= 4)."""
    return ((int(l) + 1) & 0xF) << VD_GEMM_FLAG_SLICES_SHIFT


class VdError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s returned %d (%s)" % (where, status, vd_status_string(status)))
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libvdecode.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libvdecode.so is not built: run python -m paper_2509_04827_amd.build "
                               "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P, I, U, Z, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint, ctypes.c_size_t, ctypes.c_float
        L.vd_status_string.argtypes = [I]
        L.vd_status_string.restype = ctypes.c_char_p
        L.vd_decode_workspace_size.argtypes = [I, I, I, I, I, I, U]
        L.vd_decode_workspace_size.restype = Z
        attn = [P, P, P, P, P, P, I, I, I, I, I, F, I, P, Z, U, P]
        L.vd_decode_attn.argtypes = attn
        L.vd_decode_partial.argtypes = attn
        L.vd_decode_attn_noalloc.argtypes = [P, P, P, P, P, P, I, I, I, I, I, F, I, U, P]
        L.vd_decode_plan.argtypes = [P, I, I, I, I, I, I, P, Z, U, P]
        L.vd_decode_combine.argtypes = [P, I, I, I, I, I, I, P, Z, U, P]
        L.vd_decode_gather.argtypes = [P, P, P, P, P, P, I, I, I, I, I, P, Z, P]
        L.vd_kv_append.argtypes = [P, P, P, P, P, P, I, I, I, I, I, P]
        L.vd_gemm_workspace_size.argtypes = [I, I, I, U]
        L.vd_gemm_workspace_size.restype = Z
        L.vd_gemm_bf16.argtypes = [P, P, P, I, I, I, P, Z, U, P]
        L.vd_stream_read.argtypes = [P, Z, P, I, P]
        for n in ("vd_decode_attn", "vd_decode_attn_noalloc", "vd_decode_partial", "vd_decode_plan", "vd_decode_combine",
                  "vd_decode_gather", "vd_kv_append", "vd_gemm_bf16", "vd_stream_read"):
            getattr(L, n).restype = I
        # every export has a prototype: pointers travel as plain ints, which
        # ctypes would otherwise pass as 32-bit C ints
        missing = [n for n in EXPORTS if getattr(L, n).argtypes is None]
        if missing:
            raise RuntimeError("no ctypes prototype for %s" % ", ".join(missing))
        _lib = L
    return _lib


def vd_status_string(status: int) -> str:
    return lib().vd_status_string(int(status)).decode()


def vd_decode_workspace_size(num_seqs: int, n_q_heads: int, n_kv_heads: int, head_dim: int = 128,
                             page_size: int = 16, max_pages_per_seq: int = 1,
                             flags: int = 0) -> int:
    return int(lib().vd_decode_workspace_size(num_seqs, n_q_heads, n_kv_heads, head_dim,
                                              page_size, max_pages_per_seq, flags))


def alloc_workspace(num_seqs, n_q_heads, n_kv_heads, max_pages_per_seq, flags=0,
                    head_dim=128, page_size=16, device="cuda") -> torch.Tensor:
    n = vd_decode_workspace_size(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                                 max_pages_per_seq, flags)
    if n == 0:
        raise VdError(VD_ERROR_INVALID_VALUE, "vd_decode_workspace_size")
    return torch.empty(n, dtype=torch.uint8, device=device)


def _ptr(t):
    """Device address of a tensor the kernels read or write as a dense array
    (an int, which ctypes passes as void *)."""
    if t is None:
        return None
    if t.is_cuda and t.is_contiguous():
        return t.data_ptr()
    if not t.is_contiguous():
        raise ValueError("libvdecode needs contiguous tensors (got strides %s)" % (t.stride(),))
    raise ValueError("libvdecode needs device tensors (got one on %s)" % t.device)


def _dtype(t, allowed, what):
    if t.dtype not in allowed:
        raise ValueError("%s must be %s (got %s)" % (what, " or ".join(map(str, allowed)), t.dtype))


_BF16, _I32, _F32 = torch.bfloat16, torch.int32, torch.float32


def _attn_dtypes(q, k_pages, v_pages, page_table, seq_lens, out):
    # one comparison chain on the common path; the per-tensor checks name the culprit
    if (q.dtype is _BF16 and k_pages.dtype is _BF16 and v_pages.dtype is _BF16
            and page_table.dtype is _I32 and seq_lens.dtype is _I32
            and (out.dtype is _BF16 or out.dtype is _F32)):
        return
    for t, n in ((q, "q"), (k_pages, "k_pages"), (v_pages, "v_pages")):
        _dtype(t, (_BF16,), n)
    _dtype(page_table, (_I32,), "page_table")
    _dtype(seq_lens, (_I32,), "seq_lens")
    _dtype(out, (_BF16, _F32), "out")


def step_info(workspace) -> dict:
    """The step record (vd_step_info) an attention call left at the head of
    `workspace`, read back to the host (synchronises with the device): the
    plan's sizes, the first workgroup's time in microseconds and the mean
    shader clock over it in MHz (real-time counter at 100 MHz)."""
    raw = workspace[:48].cpu().numpy()
    n = raw[:16].view("<i4")
    t0, c0, t1, c1 = (int(x) for x in raw[16:48].view("<u8"))
    dt = max(t1 - t0, 1)
    return {"n_ranges": int(n[0]), "n_tiles": int(n[1]), "n_empty": int(n[2]),
            "first_group_us": dt * 0.01, "sclk_mhz": (c1 - c0) * 100.0 / dt}


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(stream, t=None):
    """hipStream_t of `stream`: torch's current stream (on t's device) when
    None, a torch.cuda.Stream, or a raw handle (int) taken from one.  The
    current stream's handle is read without building a Stream object when
    torch offers that (a few microseconds less per call)."""
    if stream is None:
        dev = -1 if t is None else t.get_device()
        if _raw_stream is not None and dev >= 0:
            return _raw_stream(dev)
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st, where):
    if st != VD_SUCCESS:
        raise VdError(st, where)


def _shape(t, shape, what):
    """Raise ValueError unless tensor t has exactly `shape` (None matches any
    extent).  A mismatched tensor would otherwise be read or written out of
    bounds on the device."""
    if t.dim() != len(shape) or any(s is not None and t.shape[i] != s for i, s in enumerate(shape)):
        want = "[%s]" % ", ".join("*" if s is None else str(s) for s in shape)
        raise ValueError("%s has shape %s, expected %s" % (what, list(t.shape), want))


def _nbytes(t):
    return t.numel() * t.element_size()


def _kv_sizes(k_pages, v_pages):
    _shape(k_pages, (None, None, None, None), "k_pages")
    _shape(v_pages, tuple(k_pages.shape), "v_pages")
    _, S, Hkv, D = k_pages.shape
    return S, Hkv, D


def _attn_sizes(q, k_pages, v_pages, page_table, seq_lens, out):
    """Sizes of an attention call, read from q, k_pages and page_table; every
    other tensor must agree with them."""
    _shape(q, (None, None, None), "q")
    B, Hq, D = q.shape
    S, Hkv, Dk = _kv_sizes(k_pages, v_pages)
    if Dk != D:
        raise ValueError("k_pages head_dim %d differs from q's %d" % (Dk, D))
    _shape(page_table, (B, None), "page_table")
    _shape(seq_lens, (B,), "seq_lens")
    _shape(out, (B, Hq, D), "out")
    return B, Hq, Hkv, D, S, page_table.shape[1]


def _out_flags(out, flags):
    return flags | (VD_FLAG_OUT_F32 if out.dtype is _F32 else 0)


def vd_decode_attn(q, k_pages, v_pages, page_table, seq_lens, out, scale: float, workspace,
                   flags: int = 0, stream=None) -> None:
    _attn_dtypes(q, k_pages, v_pages, page_table, seq_lens, out)
    B, Hq, Hkv, D, S, maxp = _attn_sizes(q, k_pages, v_pages, page_table, seq_lens, out)
    _check(lib().vd_decode_attn(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(page_table),
                                _ptr(seq_lens), _ptr(out), B, Hq, Hkv, D, S, float(scale), maxp,
                                _ptr(workspace), _nbytes(workspace), _out_flags(out, flags),
                                _stream(stream, out)), "vd_decode_attn")


def vd_decode_attn_noalloc(q, k_pages, v_pages, page_table, seq_lens, out, scale: float,
                           flags: int = 0, stream=None) -> None:
    """vd_decode_attn with the library's fixed scratch as its workspace: the
    call allocates nothing.  Calls that overlap on one device share that
    scratch and race."""
    _attn_dtypes(q, k_pages, v_pages, page_table, seq_lens, out)
    B, Hq, Hkv, D, S, maxp = _attn_sizes(q, k_pages, v_pages, page_table, seq_lens, out)
    _check(lib().vd_decode_attn_noalloc(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(page_table),
                                        _ptr(seq_lens), _ptr(out), B, Hq, Hkv, D, S, float(scale),
                                        maxp, _out_flags(out, flags), _stream(stream, out)),
           "vd_decode_attn_noalloc")


def vd_decode_plan(seq_lens, n_q_heads: int, n_kv_heads: int, max_pages_per_seq: int, workspace,
                   flags: int = 0, head_dim: int = 128, page_size: int = 16, stream=None) -> None:
    _shape(seq_lens, (None,), "seq_lens")
    _check(lib().vd_decode_plan(_ptr(seq_lens), seq_lens.shape[0], n_q_heads, n_kv_heads,
                                head_dim, page_size, max_pages_per_seq, _ptr(workspace),
                                _nbytes(workspace), flags, _stream(stream, seq_lens)), "vd_decode_plan")


def vd_decode_partial(q, k_pages, v_pages, page_table, seq_lens, out, scale: float, workspace,
                      flags: int = 0, stream=None) -> None:
    _attn_dtypes(q, k_pages, v_pages, page_table, seq_lens, out)
    B, Hq, Hkv, D, S, maxp = _attn_sizes(q, k_pages, v_pages, page_table, seq_lens, out)
    _check(lib().vd_decode_partial(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(page_table),
                                   _ptr(seq_lens), _ptr(out), B, Hq, Hkv, D, S, float(scale),
                                   maxp, _ptr(workspace), _nbytes(workspace),
                                   _out_flags(out, flags), _stream(stream, out)), "vd_decode_partial")


def vd_decode_combine(out, n_kv_heads: int, max_pages_per_seq: int, workspace, flags: int = 0,
                      page_size: int = 16, stream=None) -> None:
    _dtype(out, (_BF16, _F32), "out")
    _shape(out, (None, None, None), "out")
    B, Hq, D = out.shape
    _check(lib().vd_decode_combine(_ptr(out), B, Hq, n_kv_heads, D, page_size, max_pages_per_seq,
                                   _ptr(workspace), _nbytes(workspace), _out_flags(out, flags),
                                   _stream(stream, out)), "vd_decode_combine")


def vd_decode_gather(k_pages, v_pages, page_table, seq_lens, k_out, v_out, workspace,
                     stream=None) -> None:
    for t, n in ((k_pages, "k_pages"), (v_pages, "v_pages"), (k_out, "k_out"), (v_out, "v_out")):
        _dtype(t, (_BF16,), n)
    _dtype(page_table, (_I32,), "page_table")
    _dtype(seq_lens, (_I32,), "seq_lens")
    S, Hkv, D = _kv_sizes(k_pages, v_pages)
    _shape(seq_lens, (None,), "seq_lens")
    B = seq_lens.shape[0]
    _shape(page_table, (B, None), "page_table")
    # the output holds every gathered row: sum of the lengths as the kernels
    # clamp them (a device read, so this call synchronises; it is a check)
    maxp = page_table.shape[1]
    rows = int(seq_lens.clamp(0, maxp * S).sum().item()) if B else 0
    _shape(k_out, (None, Hkv, D), "k_out")
    _shape(v_out, tuple(k_out.shape), "v_out")
    if k_out.shape[0] < rows:
        raise ValueError("k_out / v_out hold %d rows, the lengths need %d" % (k_out.shape[0], rows))
    _check(lib().vd_decode_gather(_ptr(k_pages), _ptr(v_pages), _ptr(page_table), _ptr(seq_lens),
                                  _ptr(k_out), _ptr(v_out), B, Hkv, D, S,
                                  maxp, _ptr(workspace), _nbytes(workspace),
                                  _stream(stream, k_pages)), "vd_decode_gather")


def vd_kv_append(k_new, v_new, k_pages, v_pages, page_table, positions, stream=None) -> None:
    """Write k_new[b] / v_new[b] at token positions[b] of request b's pages."""
    for t, n in ((k_new, "k_new"), (v_new, "v_new"), (k_pages, "k_pages"), (v_pages, "v_pages")):
        _dtype(t, (_BF16,), n)
    _dtype(page_table, (_I32,), "page_table")
    _dtype(positions, (_I32,), "positions")
    S, Hkv, D = _kv_sizes(k_pages, v_pages)
    _shape(positions, (None,), "positions")
    B = positions.shape[0]
    _shape(k_new, (B, Hkv, D), "k_new")
    _shape(v_new, (B, Hkv, D), "v_new")
    _shape(page_table, (B, None), "page_table")
    _check(lib().vd_kv_append(_ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages),
                              _ptr(page_table), _ptr(positions), B, Hkv, D, S,
                              page_table.shape[1], _stream(stream, k_pages)), "vd_kv_append")


def vd_gemm_workspace_size(M: int, N: int, K: int, flags: int = 0) -> int:
    return int(lib().vd_gemm_workspace_size(M, N, K, flags))


def vd_gemm_bf16(x, w, y, workspace=None, flags: int = 0, stream=None) -> None:
    """y [M][N] = x [M][K] . w [N][K]^T (y fp32 sets VD_FLAG_OUT_F32)."""
    _dtype(x, (_BF16,), "x")
    _dtype(w, (_BF16,), "w")
    _dtype(y, (_BF16, _F32), "y")
    _shape(x, (None, None), "x")
    M, K = x.shape
    _shape(w, (None, K), "w")
    N = w.shape[0]
    _shape(y, (M, N), "y")
    _check(lib().vd_gemm_bf16(_ptr(x), _ptr(w), _ptr(y), M, N, K, _ptr(workspace),
                              0 if workspace is None else _nbytes(workspace),
                              _out_flags(y, flags), _stream(stream, y)), "vd_gemm_bf16")


def vd_stream_read(buf, sink, blocks: int = 16384, stream=None) -> None:
    """Read all of `buf` (a measurement of the HBM read rate; see the header)."""
    _check(lib().vd_stream_read(_ptr(buf), _nbytes(buf), _ptr(sink), int(blocks),
                                _stream(stream, buf)), "vd_stream_read")
