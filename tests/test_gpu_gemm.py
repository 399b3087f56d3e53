"""GPU parity of the decode-step projection GEMM (vd_gemm_bf16) against the
fp64 oracle, through the C ABI.

Tolerance (fp32 output): the products of bf16 values are exact in fp32 and the
kernel sums them in fp32 in blocks (MFMA steps, K stages, K slices), so an output
of K terms carries rounding of order eps32 * sqrt(K) * rms(terms) with
eps32 = 2^-24; the gate is |err| <= 2^-17 * sqrt(K) * (|y| / sqrt(K) + 1)
per element, i.e. about 8e-6 relative to the output scale sqrt(K) of unit
normal inputs, ~100x the expected rounding.  bf16 output adds half an ulp.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2509_04827_amd as vd
from workloads import bits

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# Automatic plans over the decode range: the narrow 16-64-row tiles with 1-4
# K slices, the 64x128 and 128x128 tiles with and without slices, the larger
# LDS-fed tiles, rows that are not whole tiles, and the batch-size steps of
# the paper's tile quantisation (255/256/257, 512/513) up to 1024 rows.
SHAPES = [(1, 4096, 4096), (7, 6144, 4096), (9, 4096, 4096), (16, 512, 512),
          (33, 1024, 14336), (48, 4096, 14336), (64, 28672, 4096), (64, 64, 512), (17, 128, 1024),
          (3, 4096, 14336), (4, 2048, 2048),
          (96, 4096, 4096), (128, 6144, 4096), (192, 2048, 14336), (255, 4096, 4096),
          (256, 4096, 4096), (257, 4096, 4096), (512, 2048, 2048), (513, 2048, 4096),
          (1024, 1024, 2048), (1024, 4096, 1024),
          # shapes whose automatic plan takes each of the larger LDS-fed tiles
          # (256x128, 192x256, 256x256, 320x256)
          (257, 16384, 512), (257, 28672, 512), (1024, 12288, 512), (513, 28672, 512)]

# Every tile configuration with 1, 2, 8 and 16 K slices at two row counts
# (37: several narrow row tiles; 300: a partial last tile of every size).
FORCED = [(M, c, l) for M in (37, 300) for c in range(11) for l in (0, 1, 3, 4)]

# The LDS-fed tiles on many column tiles (2560 / BN of them, not a multiple of
# the 8 XCDs, so both parts of the workgroup order are used) and a last row
# tile that holds one row.
WIDE = [(M, c, l) for M in (257, 513) for c in (6, 7, 8, 9, 10) for l in (0, 1)]

# The 64-column-stage tiles on K slices of one and two stages (K = 512 in 8
# or 4 slices): the shortest pipelines, where the ring's loads past the end
# and the first stage's wait meet.
SHORT_K = [(M, c, l) for M in (37, 300) for c in (4, 5, 6, 7, 8, 9, 10) for l in (2, 3)]


def inputs(M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((M, K), generator=g).to(torch.bfloat16)
    w = torch.randn((N, K), generator=g).to(torch.bfloat16)
    return x, w


def run(x, w, dtype, flags=0):
    M, K = x.shape
    N = w.shape[0]
    y = torch.full((M, N), float("nan"), dtype=dtype, device=DEV)
    n = vd.vd_gemm_workspace_size(M, N, K, flags)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device=DEV)
    vd.vd_gemm_bf16(x.to(DEV), w.to(DEV), y, ws, flags=flags)
    torch.cuda.synchronize()
    return y.cpu()


def check(x, w, ref, flags=0, bf16=True):
    K = x.shape[1]
    got = run(x, w, torch.float32, flags).double().numpy()
    assert np.isfinite(got).all()
    bound = 2.0 ** -17 * np.sqrt(K) * (np.abs(ref) / np.sqrt(K) + 1.0)
    err = np.abs(got - ref)
    print("  fp32 max err/bound %.3e rel-L2 %.3e" % ((err / bound).max(),
          np.linalg.norm(got - ref) / np.linalg.norm(ref)), flush=True)
    assert (err <= bound).all()
    if bf16:
        g16 = run(x, w, torch.bfloat16, flags).float().double().numpy()
        ulp = np.ldexp(1.0, (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7).astype(int))
        assert (np.abs(g16 - ref) <= 0.5 * ulp + bound).all()


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_parity(M, N, K):
    print("case: gemm M %d N %d K %d workspace %d B" % (M, N, K, vd.vd_gemm_workspace_size(M, N, K)),
          flush=True)
    x, w = inputs(M, N, K, M * 131 + N + K)
    check(x, w, oracle.gemm(bits(x), bits(w)))


@pytest.mark.parametrize("M,cfg,slices_log2", FORCED)
def test_gemm_forced_tiles(M, cfg, slices_log2):
    """Each tile configuration and slice count, forced, against the oracle."""
    N, K = 256, 8192
    flags = vd.VD_GEMM_FLAG_TILE(cfg) | vd.VD_GEMM_FLAG_SLICES_LOG2(slices_log2)
    print("case: gemm forced tile %d, %d slices, M %d N %d K %d" % (cfg, 1 << slices_log2, M, N, K),
          flush=True)
    x, w = inputs(M, N, K, 7 * M + cfg)
    check(x, w, oracle.gemm(bits(x), bits(w)), flags, bf16=slices_log2 == 1)


@pytest.mark.parametrize("M,cfg,slices_log2", WIDE)
def test_gemm_forced_wide(M, cfg, slices_log2):
    N, K = 2560, 1024
    flags = vd.VD_GEMM_FLAG_TILE(cfg) | vd.VD_GEMM_FLAG_SLICES_LOG2(slices_log2)
    print("case: gemm forced tile %d, %d slices, M %d N %d K %d" % (cfg, 1 << slices_log2, M, N, K),
          flush=True)
    x, w = inputs(M, N, K, 3 * M + cfg)
    check(x, w, oracle.gemm(bits(x), bits(w)), flags, bf16=slices_log2 == 0)


@pytest.mark.parametrize("M,cfg,slices_log2", SHORT_K)
def test_gemm_forced_short_slices(M, cfg, slices_log2):
    N, K = 512, 512
    flags = vd.VD_GEMM_FLAG_TILE(cfg) | vd.VD_GEMM_FLAG_SLICES_LOG2(slices_log2)
    print("case: gemm forced tile %d, %d slices, M %d N %d K %d" % (cfg, 1 << slices_log2, M, N, K),
          flush=True)
    x, w = inputs(M, N, K, 5 * M + cfg)
    check(x, w, oracle.gemm(bits(x), bits(w)), flags, bf16=False)


def test_gemm_deterministic():
    x, w = inputs(40, 4096, 4096, 5)
    a = run(x, w, torch.float32)
    b = run(x, w, torch.float32)
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_gemm_argument_errors_on_device():
    x, w = inputs(4, 64, 512, 6)
    y = torch.empty((4, 64), dtype=torch.float32, device=DEV)
    with pytest.raises(vd.VdError) as e:
        vd.vd_gemm_bf16(x.to(DEV)[:, :500].contiguous(), w.to(DEV)[:, :500].contiguous(), y)
    assert e.value.status == vd.VD_ERROR_NOT_SUPPORTED
    # a 128-column tile on 64 columns; slices of 64 columns (not whole
    # 128-column stages of the narrow tile)
    for flags in (vd.VD_GEMM_FLAG_TILE(4), vd.VD_GEMM_FLAG_SLICES_LOG2(3)):
        with pytest.raises(vd.VdError) as e:
            vd.vd_gemm_bf16(x.to(DEV), w.to(DEV), y, flags=flags)
        assert e.value.status == vd.VD_ERROR_NOT_SUPPORTED


def test_gemm_sliced_equals_unsliced_bits():
    """K slices change the order of the sum, not its terms: every slice count
    agrees with the unsliced result within fp32 rounding, and each is the same
    bit pattern on every call."""
    x, w = inputs(64, 1024, 8192, 11)
    base = run(x, w, torch.float32, vd.VD_GEMM_FLAG_TILE(3) | vd.VD_GEMM_FLAG_SLICES_LOG2(0))
    for l in (1, 2, 3, 4):
        f = vd.VD_GEMM_FLAG_TILE(3) | vd.VD_GEMM_FLAG_SLICES_LOG2(l)
        a, b = run(x, w, torch.float32, f), run(x, w, torch.float32, f)
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
        assert ((a - base).abs() <= 2.0 ** -17 * np.sqrt(8192) * (base.abs() / np.sqrt(8192) + 1)).all()
