"""C-ABI library on the CPU: it loads, exports what include/vdecode.h declares,
sizes workspaces sensibly and rejects bad arguments before touching the GPU.
No call here reaches a kernel launch (every argument set is invalid)."""
import ctypes
import os
import re

import pytest

import paper_2509_04827_amd as vd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "vdecode.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vd_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = vd.lib()
    names = declared_functions()
    assert names, "no declarations parsed"
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(vd.EXPORTS)


def test_status_strings():
    assert vd.vd_status_string(0) == "VD_SUCCESS"
    assert vd.vd_status_string(3) == "VD_ERROR_WORKSPACE_TOO_SMALL"
    assert vd.vd_status_string(99) == "VD_UNKNOWN_STATUS"


def test_workspace_size_rules():
    ws = vd.vd_decode_workspace_size
    base = ws(256, 32, 8, 128, 16, 1024)
    assert base > 0
    assert ws(256, 32, 8, 128, 16, 1024) == base          # deterministic
    assert ws(256, 64, 8, 128, 16, 1024) > base            # more heads per group
    assert ws(0, 32, 8, 128, 16, 1) > 0                    # empty batch is valid
    assert ws(256, 32, 8, 64, 16, 1024) == 0               # head_dim unsupported
    assert ws(256, 32, 8, 128, 32, 1024) == 0              # page_size unsupported
    assert ws(256, 24, 8, 128, 16, 1024) == 0              # G = 3 unsupported
    assert ws(256, 30, 8, 128, 16, 1024) == 0              # Hq % Hkv != 0
    assert ws(8193, 32, 8, 128, 16, 16) == 0               # too many requests
    assert ws(4, 32, 8, 128, 16, 63, 1 << 5) == 0          # unknown flag bit
    # planning in the attention kernel needs no other workspace
    assert ws(4, 32, 8, 128, 16, 63, vd.VD_FLAG_SELF_PLAN) == ws(4, 32, 8, 128, 16, 63)
    assert ws(4, 32, 8, 128, 16, 63, vd.VD_FLAG_SELF_PLAN | vd.VD_FLAG_OUT_F32) == ws(4, 32, 8, 128, 16, 63)
    # the score path does not change the workspace, for any G
    for hq in (8, 32, 64, 128):
        assert ws(4, hq, 8, 128, 16, 63, vd.VD_FLAG_SCORE_MFMA) == ws(4, hq, 8, 128, 16, 63) > 0
    # one tile per range: up to one partial per (page, KV head) plus one per segment
    small = ws(4, 32, 8, 128, 16, 63, vd.VD_FLAG_RANGE_TILES(1))
    assert small >= (4 * 63 * 8 + 4 * 8) * 4 * 128 * 4
    assert ws(4, 32, 8, 128, 16, 63, vd.VD_FLAG_RANGE_TILES(200)) < small


P = ctypes.c_void_p
FAKE = P(0x10000)      # aligned, never dereferenced: validation fails first
MIS = P(0x10002)       # misaligned


def call_attn(fn, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, pt=FAKE, sl=FAKE, out=FAKE, B=4, Hq=32, Hkv=8, D=128, S=16,
             scale=0.088, maxp=63, ws=FAKE, wsb=0, flags=0, stream=None)
    a.update(kw)
    return fn(a["q"], a["k"], a["v"], a["pt"], a["sl"], a["out"], a["B"], a["Hq"], a["Hkv"],
              a["D"], a["S"], a["scale"], a["maxp"], a["ws"], a["wsb"], a["flags"], a["stream"])


@pytest.mark.parametrize("entry", ["vd_decode_attn", "vd_decode_partial"])
def test_argument_errors(entry):
    fn = getattr(vd.lib(), entry)
    need = vd.vd_decode_workspace_size(4, 32, 8, 128, 16, 63)
    ok = dict(wsb=need)
    assert call_attn(fn, q=None, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, out=None, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, ws=None, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, q=MIS, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, k=MIS, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, pt=P(0x10001), **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, B=-1, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, Hq=30, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, maxp=0, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, scale=float("nan"), **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, scale=float("inf"), **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, flags=1 << 7, **ok) == vd.VD_ERROR_INVALID_VALUE
    assert call_attn(fn, D=64, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    assert call_attn(fn, S=32, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    assert call_attn(fn, Hq=24, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    assert call_attn(fn, Hq=256, Hkv=8, **ok) == vd.VD_ERROR_NOT_SUPPORTED   # G = 32
    assert call_attn(fn, B=9000, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    # output rows (request, query head) and partial slots must fit 32 bits
    assert call_attn(fn, B=8192, Hq=262144, Hkv=16384, maxp=1, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    assert call_attn(fn, B=8192, Hq=16384, Hkv=8192, maxp=31, **ok) == vd.VD_ERROR_NOT_SUPPORTED
    assert call_attn(fn, wsb=need - 1) == vd.VD_ERROR_WORKSPACE_TOO_SMALL
    assert call_attn(fn, wsb=0) == vd.VD_ERROR_WORKSPACE_TOO_SMALL
    forced = vd.VD_FLAG_RANGE_TILES(1)
    need1 = vd.vd_decode_workspace_size(4, 32, 8, 128, 16, 63, forced)
    assert call_attn(fn, wsb=need1 - 1, flags=forced) == vd.VD_ERROR_WORKSPACE_TOO_SMALL


def test_plan_combine_gather_argument_errors():
    L = vd.lib()
    need = vd.vd_decode_workspace_size(4, 32, 8, 128, 16, 63)
    assert L.vd_decode_plan(None, 4, 32, 8, 128, 16, 63, FAKE, need, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_decode_plan(FAKE, 4, 32, 8, 128, 16, 63, FAKE, need - 1, 0, None) == \
        vd.VD_ERROR_WORKSPACE_TOO_SMALL
    assert L.vd_decode_plan(FAKE, 4, 32, 8, 128, 8, 63, FAKE, need, 0, None) == vd.VD_ERROR_NOT_SUPPORTED
    assert L.vd_decode_combine(None, 4, 32, 8, 128, 16, 63, FAKE, need, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_decode_combine(MIS, 4, 32, 8, 128, 16, 63, FAKE, need, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_decode_combine(FAKE, 4, 32, 8, 128, 16, 63, FAKE, 0, 0, None) == \
        vd.VD_ERROR_WORKSPACE_TOO_SMALL
    gneed = vd.vd_decode_workspace_size(4, 8, 8, 128, 16, 63)
    assert L.vd_decode_gather(FAKE, FAKE, FAKE, FAKE, None, FAKE, 4, 8, 128, 16, 63, FAKE, gneed,
                              None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_decode_gather(FAKE, FAKE, FAKE, FAKE, FAKE, MIS, 4, 8, 128, 16, 63, FAKE, gneed,
                              None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_decode_gather(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 128, 16, 63, FAKE,
                              gneed - 1, None) == vd.VD_ERROR_WORKSPACE_TOO_SMALL
    assert L.vd_decode_gather(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 96, 16, 63, FAKE, gneed,
                              None) == vd.VD_ERROR_NOT_SUPPORTED


def test_noalloc_argument_errors():
    """vd_decode_attn_noalloc checks its arguments as vd_decode_attn does
    (minus the workspace) before it looks at the device."""
    fn = vd.lib().vd_decode_attn_noalloc

    def call(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, pt=FAKE, sl=FAKE, out=FAKE, B=4, Hq=32, Hkv=8, D=128,
                 S=16, scale=0.088, maxp=63, flags=0, stream=None)
        a.update(kw)
        return fn(a["q"], a["k"], a["v"], a["pt"], a["sl"], a["out"], a["B"], a["Hq"], a["Hkv"],
                  a["D"], a["S"], a["scale"], a["maxp"], a["flags"], a["stream"])

    assert call(q=None) == vd.VD_ERROR_INVALID_VALUE
    assert call(out=MIS) == vd.VD_ERROR_INVALID_VALUE
    assert call(scale=float("nan")) == vd.VD_ERROR_INVALID_VALUE
    assert call(flags=1 << 7) == vd.VD_ERROR_INVALID_VALUE
    assert call(D=64) == vd.VD_ERROR_NOT_SUPPORTED
    assert call(B=9000) == vd.VD_ERROR_NOT_SUPPORTED
    assert call(B=0) == vd.VD_SUCCESS              # nothing to do, nothing enqueued
    assert vd.vd_status_string(vd.VD_ERROR_SCRATCH_LIMIT) == "VD_ERROR_SCRATCH_LIMIT"
    hdr = open(os.path.join(ROOT, "include", "vdecode.h")).read()
    assert vd.VD_NOALLOC_SCRATCH_BYTES == int(re.search(r"VD_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", hdr).group(1)) << \
        int(re.search(r"VD_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", hdr).group(2))


def test_append_and_stream_argument_errors():
    L = vd.lib()
    assert L.vd_kv_append(None, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 128, 16, 63, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_kv_append(FAKE, FAKE, MIS, FAKE, FAKE, FAKE, 4, 8, 128, 16, 63, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_kv_append(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 16, 63, None) == vd.VD_ERROR_NOT_SUPPORTED
    assert L.vd_kv_append(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, -1, 8, 128, 16, 63, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_stream_read(None, 1024, FAKE, 8, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_stream_read(FAKE, 1000, FAKE, 8, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_stream_read(FAKE, 1024, FAKE, 0, None) == vd.VD_ERROR_INVALID_VALUE


def test_gemm_argument_errors():
    L = vd.lib()
    ws = vd.vd_gemm_workspace_size
    # the workspace holds S fp32 partials of M x N when K is split S ways
    for M, N, K in ((64, 4096, 4096), (1, 28672, 4096), (1024, 4096, 4096), (300, 4096, 14336)):
        n = ws(M, N, K)
        assert n % (M * N * 4) == 0 and n // (M * N * 4) in (0, 2, 4, 8)
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_SLICES_LOG2(0)) == 0
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_SLICES_LOG2(3)) == 8 * 64 * 4096 * 4
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_TILE(5) | vd.VD_GEMM_FLAG_SLICES_LOG2(4)) == 16 * 64 * 4096 * 4
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_TILE(11)) == 0   # no such tile
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_TILE(7) | vd.VD_GEMM_FLAG_SLICES_LOG2(0)) == 0
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_TILE(9) | vd.VD_GEMM_FLAG_SLICES_LOG2(1)) == 2 * 64 * 4096 * 4
    assert ws(4, 192, 512, vd.VD_GEMM_FLAG_TILE(6)) == 0       # 128-column LDS-fed tile, N % 128
    assert ws(4, 384, 512, vd.VD_GEMM_FLAG_TILE(8)) == 0       # 256-column tile, N % 256
    assert ws(4, 384, 512, vd.VD_GEMM_FLAG_TILE(9)) == 0
    assert ws(4, 384, 512, vd.VD_GEMM_FLAG_TILE(10)) == 0
    assert ws(64, 4096, 4096, vd.VD_GEMM_FLAG_SLICES_LOG2(5)) == 0   # 32 slices
    assert ws(4, 4096, 512, vd.VD_GEMM_FLAG_SLICES_LOG2(3)) == 0     # 64-column slices: not whole 128-column stages
    assert ws(4, 192, 512, vd.VD_GEMM_FLAG_TILE(4)) == 0       # 128-column tile, N % 128
    assert ws(8, 4128, 4096) == 0       # N % 64
    assert ws(8, 4096, 4000) == 0       # K % 512
    assert ws(0, 4096, 4096) == 0       # M = 0
    assert L.vd_gemm_bf16(None, FAKE, FAKE, 4, 64, 512, FAKE, 1 << 20, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_gemm_bf16(FAKE, MIS, FAKE, 4, 64, 512, FAKE, 1 << 20, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_gemm_bf16(FAKE, FAKE, FAKE, 0, 64, 512, FAKE, 1 << 20, 0, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_gemm_bf16(FAKE, FAKE, FAKE, 4, 64, 512, FAKE, 1 << 20, 1 << 4, None) == vd.VD_ERROR_INVALID_VALUE
    assert L.vd_gemm_bf16(FAKE, FAKE, FAKE, 99, 64, 500, FAKE, 1 << 20, 0, None) == vd.VD_ERROR_NOT_SUPPORTED
    assert L.vd_gemm_bf16(FAKE, FAKE, FAKE, 4, 64, 512, FAKE, 1 << 20, vd.VD_GEMM_FLAG_TILE(4), None) == \
        vd.VD_ERROR_NOT_SUPPORTED


def test_product_does_not_reference_oracle():
    """The product package neither imports nor links the oracle."""
    pkg = os.path.join(ROOT, "paper_2509_04827_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "vdo_" not in text, f
    with open(os.path.join(pkg, "libvdecode.so"), "rb") as fh:
        blob = fh.read()
    assert b"vdo_" not in blob and b"libvdo_oracle" not in blob


def test_binding_constants_match_header():
    """The binding's status codes and flags are the header's."""
    hdr = open(os.path.join(ROOT, "include", "vdecode.h")).read()
    for name, val in re.findall(r"#define (VD_FLAG_\w+) \(1u << (\d+)\)", hdr):
        assert getattr(vd, name) == 1 << int(val), name
    for name, val in re.findall(r"(VD_(?:SUCCESS|ERROR_\w+)) = (\d+)", hdr):
        assert getattr(vd, name) == int(val), name
    assert vd.VD_FLAG_RANGE_SHIFT == int(re.search(r"#define VD_FLAG_RANGE_SHIFT (\d+)u", hdr).group(1))



def test_binding_rejects_host_and_strided_tensors_before_any_call():
    """The binding's marshalling: host tensors, strided views and wrong dtypes
    raise ValueError naming the problem; nothing reaches the library."""
    import torch
    t = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensors"):
        vd._ptr(t)
    with pytest.raises(ValueError, match="contiguous"):
        vd._ptr(t.t())
    assert vd._ptr(None) is None
    bf, i32, f32 = torch.bfloat16, torch.int32, torch.float32
    ok = [torch.zeros(1, dtype=d) for d in (bf, bf, bf, i32, i32, bf)]
    vd._attn_dtypes(*ok)
    vd._attn_dtypes(*ok[:5], torch.zeros(1, dtype=f32))
    for i, name in enumerate(("q", "k_pages", "v_pages", "page_table", "seq_lens", "out")):
        bad = list(ok)
        bad[i] = torch.zeros(1, dtype=torch.float16)
        with pytest.raises(ValueError, match=name):
            vd._attn_dtypes(*bad)
    assert vd._stream(12345) == 12345          # raw hipStream_t handles pass through


def test_binding_prototypes_match_the_header():
    """Every export has a ctypes prototype with as many arguments as its C
    declaration (pointers are passed as ints, which need the prototype to
    travel as 64-bit pointers)."""
    src = open(os.path.join(ROOT, "include", "vdecode.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    decl = dict(re.findall(r"\b(vd_[a-z_0-9]+)\s*\(([^)]*)\)\s*;", src))
    L = vd.lib()
    assert set(decl) == set(vd.EXPORTS)
    for name, params in decl.items():
        n = 0 if params.strip() in ("", "void") else params.count(",") + 1
        assert getattr(L, name).argtypes is not None, name
        assert len(getattr(L, name).argtypes) == n, (name, len(getattr(L, name).argtypes), n)


def test_empty_batch_is_a_no_op():
    """num_seqs = 0 with valid arguments returns VD_SUCCESS from every
    per-request entry point without launching anything (so no device is
    needed here); its arguments are still checked."""
    L = vd.lib()
    big = 1 << 30
    ws = vd.vd_decode_workspace_size(0, 32, 8, 128, 16, 4, 0)
    assert ws > 0
    attn = (FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 32, 8, 128, 16, 0.125, 4, FAKE, big, 0, None)
    assert L.vd_decode_attn(*attn) == vd.VD_SUCCESS
    assert L.vd_decode_partial(*attn) == vd.VD_SUCCESS
    assert L.vd_decode_plan(FAKE, 0, 32, 8, 128, 16, 4, FAKE, big, 0, None) == vd.VD_SUCCESS
    assert L.vd_decode_combine(FAKE, 0, 32, 8, 128, 16, 4, FAKE, big, 0, None) == vd.VD_SUCCESS
    assert L.vd_decode_gather(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 8, 128, 16, 4, FAKE, big,
                              None) == vd.VD_SUCCESS
    assert L.vd_kv_append(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 8, 128, 16, 4, None) == vd.VD_SUCCESS
    # still validated: a NULL output or a short workspace is an error
    bad = list(attn)
    bad[5] = None
    assert L.vd_decode_attn(*bad) == vd.VD_ERROR_INVALID_VALUE
    bad = list(attn)
    bad[14] = 16
    assert L.vd_decode_attn(*bad) == vd.VD_ERROR_WORKSPACE_TOO_SMALL


def test_binding_rejects_mismatched_shapes_before_any_call():
    """Sizes come from q, k_pages and page_table (attention), positions
    (append) and x / w (GEMM); every other tensor must agree with them, or the
    binding raises ValueError naming it before anything reaches the library
    (a mismatched tensor would be read or written out of bounds)."""
    import torch
    bf, i32, f32 = torch.bfloat16, torch.int32, torch.float32
    B, Hq, Hkv, D, S, maxp, P = 3, 8, 2, 128, 16, 4, 12

    def attn_args(**kw):
        a = dict(q=torch.zeros(B, Hq, D, dtype=bf), k=torch.zeros(P, S, Hkv, D, dtype=bf),
                 v=torch.zeros(P, S, Hkv, D, dtype=bf), pt=torch.zeros(B, maxp, dtype=i32),
                 sl=torch.zeros(B, dtype=i32), out=torch.zeros(B, Hq, D, dtype=f32))
        a.update(kw)
        return a

    bad = {
        "out": dict(out=torch.zeros(B, Hq, D + 1, dtype=f32)),
        "v_pages": dict(v=torch.zeros(P - 1, S, Hkv, D, dtype=bf)),
        "seq_lens": dict(sl=torch.zeros(B + 1, dtype=i32)),
        "page_table": dict(pt=torch.zeros(B - 1, maxp, dtype=i32)),
        "q": dict(q=torch.zeros(B, Hq * D, dtype=bf)),
        "head_dim": dict(k=torch.zeros(P, S, Hkv, 64, dtype=bf), v=torch.zeros(P, S, Hkv, 64, dtype=bf)),
    }
    for entry in (vd.vd_decode_attn, vd.vd_decode_partial):
        for what, kw in bad.items():
            a = attn_args(**kw)
            with pytest.raises(ValueError, match=what):
                entry(a["q"], a["k"], a["v"], a["pt"], a["sl"], a["out"], 0.125, torch.zeros(16, dtype=torch.uint8))
    # the well-shaped call gets past the shape checks and stops at the host tensors
    a = attn_args()
    with pytest.raises(ValueError, match="device tensors"):
        vd.vd_decode_attn(a["q"], a["k"], a["v"], a["pt"], a["sl"], a["out"], 0.125,
                          torch.zeros(16, dtype=torch.uint8))
    with pytest.raises(ValueError, match="out"):
        vd.vd_decode_combine(torch.zeros(B, Hq * D, dtype=f32), Hkv, maxp, torch.zeros(16, dtype=torch.uint8))

    k, v = torch.zeros(P, S, Hkv, D, dtype=bf), torch.zeros(P, S, Hkv, D, dtype=bf)
    pt, sl = torch.zeros(B, maxp, dtype=i32), torch.full((B,), 20, dtype=i32)
    ws = torch.zeros(16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="k_out"):      # 60 rows needed
        vd.vd_decode_gather(k, v, pt, sl, torch.zeros(59, Hkv, D, dtype=bf),
                            torch.zeros(59, Hkv, D, dtype=bf), ws)
    with pytest.raises(ValueError, match="v_out"):
        vd.vd_decode_gather(k, v, pt, sl, torch.zeros(60, Hkv, D, dtype=bf),
                            torch.zeros(60, Hkv + 1, D, dtype=bf), ws)
    with pytest.raises(ValueError, match="page_table"):
        vd.vd_decode_gather(k, v, pt[:2].contiguous(), sl, torch.zeros(60, Hkv, D, dtype=bf),
                            torch.zeros(60, Hkv, D, dtype=bf), ws)

    kn, vn, pos = torch.zeros(B, Hkv, D, dtype=bf), torch.zeros(B, Hkv, D, dtype=bf), torch.zeros(B, dtype=i32)
    with pytest.raises(ValueError, match="k_new"):
        vd.vd_kv_append(kn[:2].contiguous(), vn, k, v, pt, pos)
    with pytest.raises(ValueError, match="v_new"):
        vd.vd_kv_append(kn, torch.zeros(B, Hkv, D + 8, dtype=bf), k, v, pt, pos)
    with pytest.raises(ValueError, match="page_table"):
        vd.vd_kv_append(kn, vn, k, v, torch.zeros(B + 1, maxp, dtype=i32), pos)
    with pytest.raises(ValueError, match="v_pages"):
        vd.vd_kv_append(kn, vn, k, torch.zeros(P, S, Hkv, 64, dtype=bf), pt, pos)

    x, w = torch.zeros(4, 512, dtype=bf), torch.zeros(64, 512, dtype=bf)
    with pytest.raises(ValueError, match="w has shape"):
        vd.vd_gemm_bf16(x, torch.zeros(64, 1024, dtype=bf), torch.zeros(4, 64, dtype=f32))
    with pytest.raises(ValueError, match="y has shape"):
        vd.vd_gemm_bf16(x, w, torch.zeros(4, 128, dtype=f32))
    with pytest.raises(ValueError, match="y has shape"):
        vd.vd_gemm_bf16(x, w, torch.zeros(5, 64, dtype=f32))
    with pytest.raises(ValueError, match="x must be"):
        vd.vd_gemm_bf16(x.float(), w, torch.zeros(4, 64, dtype=f32))


def test_binding_passes_workspace_bytes_not_elements():
    """A workspace of any dtype is passed with its size in bytes."""
    import torch
    assert vd._nbytes(torch.zeros(10, dtype=torch.float32)) == 40
    assert vd._nbytes(torch.zeros(10, dtype=torch.uint8)) == 10
