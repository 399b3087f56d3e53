"""The GPU tests' precision canary (fp32-out max-abs and rel-L2 <= 1e-4) must
tell the kernel's softmax weights apart from a cheaper variant that passes the
contract gates.  The kernel feeds the weights P to the PV matrix product as a
bf16 high part plus a bf16 low part (about 16 significant bits); rounding P to
bf16 only keeps 8.  This CPU emulation of that arithmetic, on N(0,1) bf16
inputs at the workloads' lengths, checks that the hi + lo form stays well
inside the canary and the bf16-only form fails it while meeting the contract
(max-abs 1e-2, rel-L2 5e-3).  fp64 reference from the definition."""
import numpy as np
import torch

from parity_gates import CANARY_MAX_ABS, CANARY_REL_L2, GATE_MAX_ABS, GATE_REL_L2


def bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy()


def test_canary_separates_weight_precisions():
    rng = np.random.default_rng(0)
    scale = np.float32(1.0 / np.sqrt(128.0))
    log2e = np.float32(1.4426950408889634)
    refs, hi_only, hi_lo = [], [], []
    for L in (37, 128, 500, 1000, 3000):
        for _ in range(8):
            q = bf16(rng.standard_normal(128))
            K = bf16(rng.standard_normal((L, 128)))
            V = bf16(rng.standard_normal((L, 128)))
            s = (K.astype(np.float64) @ q) * np.float64(scale)
            w = np.exp(s - s.max())
            refs.append((w @ V) / w.sum())
            # the kernel's form: fp32 scores in log2 units, exp2, P = hi + lo
            s2 = (K @ q) * (scale * log2e)
            p = np.exp2(s2 - s2.max()).astype(np.float32)
            hi = bf16(p)
            lo = bf16(p - hi)
            for P, dst in ((hi, hi_only), (hi + lo, hi_lo)):
                dst.append((P.astype(np.float64) @ V) / P.astype(np.float64).sum())
    R = np.array(refs)

    def errs(O):
        O = np.array(O)
        return np.abs(O - R).max(), np.linalg.norm(O - R) / np.linalg.norm(R)

    a_hl, r_hl = errs(hi_lo)
    a_hi, r_hi = errs(hi_only)
    assert a_hl <= CANARY_MAX_ABS / 10 and r_hl <= CANARY_REL_L2 / 10
    assert a_hi > CANARY_MAX_ABS and r_hi > CANARY_REL_L2
    assert a_hi <= GATE_MAX_ABS and r_hi <= GATE_REL_L2
