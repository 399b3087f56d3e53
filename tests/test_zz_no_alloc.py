"""The no-allocation entry point (vd_decode_attn_noalloc, the library's fixed
scratch as workspace) against vd_decode_attn, through the C ABI: two calls in
a row, the second with a smaller input, each bit-identical to vd_decode_attn
(same plan, same kernels) and within the parity gates of the fp64 oracle;
sizes beyond the scratch are refused with nothing enqueued."""
import numpy as np
import pytest
import torch

import oracle
import paper_2509_04827_amd as vd
from parity_gates import GATE_MAX_ABS, GATE_REL_L2
from workloads import bits, make_case

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def _dev(c):
    return {k: (c[k].to(DEV) if isinstance(c.get(k), torch.Tensor) else c[k]) for k in c}


def _oracle(c):
    return oracle.decode_attn(bits(c["q"]), bits(c["k_pages"]), bits(c["v_pages"]),
                              c["page_table"].numpy(), c["seq_lens"].numpy(), c["scale"])


def _run(d, dtype, noalloc, flags=0):
    out = torch.full(d["q"].shape, float("nan"), dtype=dtype, device=DEV)
    args = (d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out, d["scale"])
    if noalloc:
        vd.vd_decode_attn_noalloc(*args, flags=flags)
    else:
        ws = vd.alloc_workspace(d["num_seqs"], d["n_q_heads"], d["n_kv_heads"],
                                d["max_pages_per_seq"], flags)
        vd.vd_decode_attn(*args, ws, flags=flags)
    torch.cuda.synchronize()
    return out


def test_noalloc_equals_attn_two_calls_second_smaller():
    torch.cuda.set_device(DEV)
    for name in ("llama8b_b64", "tiny_b4"):      # 64 requests / 139k tokens, then 4 / 1.7k
        say("case: noalloc %s seed 0" % name)
        c = make_case(name, seed=0, fill="nan")
        d = _dev(c)
        ref = _oracle(c)
        for dtype in (torch.float32, torch.bfloat16):
            got = _run(d, dtype, True)
            base = _run(d, dtype, False)
            view = torch.int32 if dtype is torch.float32 else torch.int16
            assert torch.equal(got.view(view), base.view(view)), "%s %s" % (name, dtype)
            g = got.double().cpu().numpy()
            err = np.abs(g - ref).max()
            rel = np.linalg.norm(g - ref) / np.linalg.norm(ref)
            say("  %s: max-abs %.3e rel-L2 %.3e, equal to vd_decode_attn" % (dtype, err, rel))
            if dtype is torch.float32:
                assert err <= GATE_MAX_ABS and rel <= GATE_REL_L2


def test_noalloc_forced_ranges_and_empty_requests():
    """Many partials (one tile per range) and requests without tokens: the
    combine reads what this call's attention kernel left in the scratch."""
    torch.cuda.set_device(DEV)
    from workloads import Workload
    w = Workload("custom", 9, 32, 8, 128, 16, "fixed", (1, 15, 16, 17, 0, 33, 640, 1000, 3))
    c = make_case(w, seed=4, fill="nan")
    d = _dev(c)
    flags = vd.VD_FLAG_RANGE_TILES(1)
    say("case: noalloc forced one-tile ranges, lengths %s" % c["seq_lens"].tolist())
    got = _run(d, torch.float32, True, flags)
    base = _run(d, torch.float32, False, flags)
    assert torch.equal(got.view(torch.int32), base.view(torch.int32))
    g = got.double().cpu().numpy()
    ref = _oracle(c)
    assert np.abs(g - ref).max() <= GATE_MAX_ABS


def test_noalloc_short_plan():
    """A step of short requests takes the short plan (no combine kernel;
    the attention kernel writes the empty rows): equal to vd_decode_attn."""
    torch.cuda.set_device(DEV)
    from workloads import Workload
    lens = (0, 12, 64, 3, 0, 40, 16, 1)
    w = Workload("custom", len(lens), 32, 8, 128, 16, "fixed", lens)
    c = make_case(w, seed=5, fill="nan")
    d = _dev(c)
    say("case: noalloc short plan, lengths %s" % (lens,))
    got = _run(d, torch.float32, True)
    base = _run(d, torch.float32, False)
    assert torch.equal(got.view(torch.int32), base.view(torch.int32))
    assert torch.equal(got[0], torch.zeros_like(got[0])) and torch.equal(got[4], torch.zeros_like(got[4]))
    g = got.double().cpu().numpy()
    assert np.abs(g - _oracle(c)).max() <= GATE_MAX_ABS


def test_noalloc_refuses_sizes_beyond_the_scratch():
    torch.cuda.set_device(DEV)
    B, Hq, Hkv = 4000, 32, 8       # ~66 MB of partial slots at one page per request
    say("case: noalloc %d requests (beyond the scratch)" % B)
    q = torch.zeros((B, Hq, 128), dtype=torch.bfloat16, device=DEV)
    kp = torch.zeros((1, 16, Hkv, 128), dtype=torch.bfloat16, device=DEV)
    pt = torch.zeros((B, 1), dtype=torch.int32, device=DEV)
    sl = torch.ones(B, dtype=torch.int32, device=DEV)
    out = torch.full((B, Hq, 128), 7.0, dtype=torch.float32, device=DEV)
    with pytest.raises(vd.VdError) as e:
        vd.vd_decode_attn_noalloc(q, kp, kp, pt, sl, out, 0.088)
    assert e.value.status == vd.VD_ERROR_SCRATCH_LIMIT
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())            # nothing ran
    # a smaller batch of the same shape still runs afterwards
    q2, pt2, sl2, out2 = q[:64].contiguous(), pt[:64].contiguous(), sl[:64].contiguous(), out[:64].contiguous()
    vd.vd_decode_attn_noalloc(q2, kp, kp, pt2, sl2, out2, 0.088)
    torch.cuda.synchronize()
    assert bool((out2 == 0).all())             # q = k = v = 0, one token: out = v = 0
