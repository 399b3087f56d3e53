"""GPU parity of the decode-step projection GEMM (vd_gemm_bf16) against the
fp64 oracle, through the C ABI.

Tolerance (fp32 output): the products of bf16 values are exact in fp32 and the
kernel sums them in fp32 in blocks (MFMA, four waves, K slices), so an output
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

# 8-wave workgroups: (1, 4096, 4096), (3, 4096, 14336) and, with K split over
# two workgroups, (4, 2048, 2048); the others take four waves
SHAPES = [(1, 4096, 4096), (7, 6144, 4096), (9, 4096, 4096), (16, 512, 512),
          (33, 1024, 14336), (48, 4096, 14336), (64, 28672, 4096), (64, 64, 512), (17, 128, 1024),
          (3, 4096, 14336), (4, 2048, 2048)]


def inputs(M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((M, K), generator=g).to(torch.bfloat16)
    w = torch.randn((N, K), generator=g).to(torch.bfloat16)
    return x, w


def run(x, w, dtype):
    M, K = x.shape
    N = w.shape[0]
    y = torch.full((M, N), float("nan"), dtype=dtype, device=DEV)
    n = vd.vd_gemm_workspace_size(M, N, K)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device=DEV)
    vd.vd_gemm_bf16(x.to(DEV), w.to(DEV), y, ws)
    torch.cuda.synchronize()
    return y.cpu()


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_parity(M, N, K):
    print("case: gemm M %d N %d K %d" % (M, N, K), flush=True)
    x, w = inputs(M, N, K, M * 131 + N + K)
    ref = oracle.gemm(bits(x), bits(w))
    got = run(x, w, torch.float32).double().numpy()
    assert np.isfinite(got).all()
    bound = 2.0 ** -17 * np.sqrt(K) * (np.abs(ref) / np.sqrt(K) + 1.0)
    err = np.abs(got - ref)
    print("  fp32 max err/bound %.3e rel-L2 %.3e" % ((err / bound).max(),
          np.linalg.norm(got - ref) / np.linalg.norm(ref)), flush=True)
    assert (err <= bound).all()
    g16 = run(x, w, torch.bfloat16).float().double().numpy()
    ulp = np.ldexp(1.0, (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7).astype(int))
    assert (np.abs(g16 - ref) <= 0.5 * ulp + bound).all()


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
