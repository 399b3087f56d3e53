"""The two score paths of the attention kernel, through the C ABI.

For G <= 8 the default path computes the scores Q.K^T on the vector ALU:
bf16 pair dot products summed in fp32 across the 16 lanes that hold a
token's dimensions (DPP row exchanges).  VD_FLAG_SCORE_MFMA computes them on
the matrix cores instead (the only path for G = 16).  Loads, softmax, P.V and
the combine are shared.  The default path is what every other parity test
runs; here the matrix-core path is held to the same bar against the fp64
oracle (gates and precision canary, bf16 within an ulp), the closed forms stay
exact (one token, one-hot scores), the output does not depend on page
placement or on what fills the pages past a request's end, and the whole step
equals the staged calls (planner kernel or self-planned) bit for bit.  The two
paths agree with each other to fp32 rounding.
"""
import numpy as np
import pytest
import torch

import oracle_pins as pins
import paper_2509_04827_amd as vd
import test_gpu_parity as P
from workloads import ORDER, make_case

pytestmark = pytest.mark.gpu

DEV = P.DEV
M = vd.VD_FLAG_SCORE_MFMA


@pytest.mark.parametrize("name", ORDER)
def test_workload_parity_mfma(name):
    P.say("case: workload %s seed 0, matrix-core score" % name)
    c = make_case(name, seed=0, fill="nan")
    d = P.dev_case(c)
    ref = P.ref_of(c)
    P.check_f32(P.run_gpu(d, torch.float32, flags=M), ref, name + " mfma", canary=True)
    P.check_bf16(P.run_gpu(d, torch.bfloat16, flags=M), ref, name + " mfma")


def test_valu_and_mfma_scores_agree():
    """Both score paths sum the same exact bf16 products in fp32, in different
    orders: their outputs agree to fp32 rounding."""
    c = make_case("chat_b256", seed=1, fill="nan")
    d = P.dev_case(c)
    a = P.run_gpu(d, torch.float32, flags=M).cpu().double()
    b = P.run_gpu(d, torch.float32).cpu().double()
    rel = ((a - b).norm() / a.norm()).item()
    P.say("case: chat_b256 seed 1, valu vs mfma rel-L2 %.3e max-abs %.3e"
          % (rel, (a - b).abs().max().item()))
    assert rel <= 1e-6 and (a - b).abs().max().item() <= 1e-5


@pytest.mark.parametrize("G,hkv", [(1, 4), (2, 4), (4, 2), (8, 2), (8, 8), (4, 16), (1, 16), (16, 2)])
@pytest.mark.parametrize("path", ["default", "mfma"])
def test_gqa_ratios_both_paths(G, hkv, path):
    """Every G on both paths (the DPP reduction scatters one to three head
    bits over the lanes and sums the rest; G = 16 is the matrix cores' on
    both), with empty, one-token and page-boundary lengths and a long
    request."""
    flags = M if path == "mfma" else 0
    P.say("case: %s score G=%d Hkv=%d" % (path, G, hkv))
    c = P.custom([1, 20, 0, 300, 2222, 64, 15, 16, 17, 4097], hq=G * hkv, hkv=hkv, seed=113 + G)
    d = P.dev_case(c)
    ref = P.ref_of(c)
    got = P.run_gpu(d, flags=flags)
    assert torch.equal(got[2], torch.zeros_like(got[2]))
    P.check_f32(got, ref, "%s G=%d" % (path, G), canary=True)
    P.check_bf16(P.run_gpu(d, torch.bfloat16, flags=flags), ref, "%s G=%d" % (path, G))
    if G == 16:   # one path for G = 16: the flag changes nothing
        other = P.run_gpu(d, flags=flags ^ M)
        assert torch.equal(got.view(torch.int32).cpu(), other.view(torch.int32).cpu())


def test_single_token_is_v_row_mfma():
    P.say("case: mfma score, L=1 x 37 requests")
    c = P.custom([1] * 37, hq=32, hkv=8, seed=3)
    d = P.dev_case(c)
    pt = c["page_table"].numpy()
    expect = np.repeat(P.bits(c["v_pages"])[pt[:, 0], 0], 4, axis=1)
    assert np.array_equal(P.bits(P.run_gpu(d, torch.bfloat16, flags=M).cpu()), expect)


@pytest.mark.parametrize("split", [0, 3])
def test_one_hot_is_v_row_mfma(split):
    """Scores that single out one token per (request, head): the output is
    that token's V row exactly on the matrix-core path too."""
    lengths = [1, 40, 300, 17, 2000, 5000, 16, 33]
    hot = [0, 39, 150, 16, 1999, 2500, 0, 32]
    P.say("case: mfma score one-hot split=%d" % split)
    c = pins.onehot_case(lengths, 32, 8, 11, hot)
    q = torch.from_numpy(c["q"].view(np.int16)).view(torch.bfloat16)
    k = torch.from_numpy(c["k"].view(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(c["v"].view(np.int16)).view(torch.bfloat16)
    d = dict(q=q.to(DEV), k_pages=k.to(DEV), v_pages=v.to(DEV),
             page_table=torch.from_numpy(c["pt"]).to(DEV), seq_lens=torch.from_numpy(c["L"]).to(DEV),
             scale=c["scale"], num_seqs=len(lengths), n_q_heads=32, n_kv_heads=8,
             max_pages_per_seq=c["pt"].shape[1])
    flags = M | (vd.VD_FLAG_RANGE_TILES(split) if split else 0)
    got = P.run_gpu(d, torch.float32, flags=flags).cpu().numpy()
    for b, t in enumerate(hot):
        vrow = c["v"][c["pt"][b, t // 16], t % 16]
        expect = (np.repeat(vrow, 4, axis=0).astype(np.uint32) << 16).view(np.float32)
        assert np.array_equal(got[b], expect), b


def test_fill_and_placement_invariance_mfma():
    """NaN or zero past each request's end, pages permuted: the same bits."""
    P.say("case: mfma score, NaN vs zero fill, page permutation, determinism")
    lengths = [5, 17, 31, 250, 1111, 4097, 1]
    a = P.custom(lengths, seed=7, fill="nan", shuffle=False)
    z = P.custom(lengths, seed=7, fill="zero", shuffle=False)
    perm = torch.randperm(a["num_pages"], generator=torch.Generator().manual_seed(9))
    b = dict(a)
    b["k_pages"] = torch.empty_like(a["k_pages"])
    b["v_pages"] = torch.empty_like(a["v_pages"])
    b["k_pages"][perm] = a["k_pages"]
    b["v_pages"][perm] = a["v_pages"]
    b["page_table"] = perm.to(torch.int32)[a["page_table"].long()]
    x1 = P.run_gpu(P.dev_case(a), flags=M).cpu()
    x2 = P.run_gpu(P.dev_case(a), flags=M).cpu()
    y = P.run_gpu(P.dev_case(z), flags=M).cpu()
    w = P.run_gpu(P.dev_case(b), flags=M).cpu()
    assert torch.isfinite(x1).all()
    for other in (x2, y, w):
        assert torch.equal(x1.view(torch.int32), other.view(torch.int32))
    P.check_f32(x1, P.ref_of(a), "mfma fill/placement", canary=True)


@pytest.mark.parametrize("case", ["short_mixed", "split_many", "mixed_forced7", "many_pieces"])
def test_whole_equals_staged_mfma(case):
    """With the matrix-core score: vd_decode_attn against the planner kernel
    plus the planned vd_decode_partial plus vd_decode_combine, and against
    the self-planned vd_decode_partial plus vd_decode_combine: bit for bit;
    and against the oracle."""
    flags = M
    hq, hkv = 32, 8
    if case == "short_mixed":
        lengths = [0, 5, 0, 64, 0, 17, 1, 33]
    elif case == "split_many":
        lengths = [16384, 3, 0, 9000]
    elif case == "mixed_forced7":
        lengths = [0, 5, 300, 0, 2049, 1, 16, 17, 7000, 0]
        flags |= vd.VD_FLAG_RANGE_TILES(7)
    else:                     # more pieces per wave than LDS result entries
        rng = np.random.default_rng(58)
        lengths = [int(x) for x in rng.choice([1, 3, 16, 17, 40, 100], 3000)]
        hq, hkv = 16, 2
    P.say("case: mfma score, whole vs staged %s (%d requests)" % (case, len(lengths)))
    c = P.custom(lengths, hq=hq, hkv=hkv, seed=122)
    d = P.dev_case(c)
    B, maxp = c["num_seqs"], c["max_pages_per_seq"]
    for dt in (torch.float32, torch.bfloat16):
        whole = P.run_gpu(d, dt, flags=flags)
        ws = vd.alloc_workspace(B, hq, hkv, maxp, flags)
        staged = torch.full(d["q"].shape, float("nan"), dtype=dt, device=DEV)
        vd.vd_decode_plan(d["seq_lens"], hq, hkv, maxp, ws, flags=flags)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             staged, d["scale"], ws, flags=flags)
        vd.vd_decode_combine(staged, hkv, maxp, ws, flags=flags)
        selfp = torch.full(d["q"].shape, float("nan"), dtype=dt, device=DEV)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             selfp, d["scale"], ws, flags=flags | vd.VD_FLAG_SELF_PLAN)
        vd.vd_decode_combine(selfp, hkv, maxp, ws, flags=flags)
        torch.cuda.synchronize()
        iv = torch.int32 if dt == torch.float32 else torch.int16
        assert torch.equal(whole.view(iv).cpu(), staged.view(iv).cpu()), case
        assert torch.equal(whole.view(iv).cpu(), selfp.view(iv).cpu()), case
        if dt == torch.float32:
            P.check_f32(whole, P.ref_of(c), "mfma " + case, canary=True)
