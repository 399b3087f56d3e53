"""GPU parity of libvdecode against the fp64 oracle, called through the C ABI.

Gates (fp32 output): max-abs <= 1e-2 and rel-L2 <= 5e-3 over the whole output
of a workload.  bf16 output adds its own rounding (half an ulp, up to 0.0156
for |out| in [4, 8)), so its gate is rel-L2 <= 5e-3 and, per element,
|err| <= max(1e-2, one bf16 ulp of the oracle value).  Copy-through gather,
L = 1, one-hot, page permutation, NaN fill and determinism are bit-exact.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import oracle_pins as pins
import paper_2509_04827_amd as vd
from parity_gates import CANARY_MAX_ABS, CANARY_REL_L2, GATE_MAX_ABS, GATE_REL_L2
from workloads import ORDER, SHARDS, Workload, bits, make_case

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def dev_case(c):
    return {k: (c[k].to(DEV) if isinstance(c.get(k), torch.Tensor) else c[k]) for k in c}


def host(c):
    return (bits(c["q"]), bits(c["k_pages"]), bits(c["v_pages"]), c["page_table"].numpy(),
            c["seq_lens"].numpy())


def run_gpu(d, out_dtype=torch.float32, flags=0, ws=None):
    out = torch.full(d["q"].shape, float("nan"), dtype=out_dtype, device=DEV)
    if ws is None:
        ws = vd.alloc_workspace(d["num_seqs"], d["n_q_heads"], d["n_kv_heads"],
                                d["max_pages_per_seq"], flags)
    vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out,
                      d["scale"], ws, flags=flags)
    torch.cuda.synchronize()
    return out


def ref_of(c):
    return oracle.decode_attn(*host(c), c["scale"])


def bf16_ulp(x):
    a = np.abs(x).astype(np.float32)
    e = np.floor(np.log2(np.maximum(a, np.float32(2.0 ** -126))))
    return np.ldexp(1.0, (e - 7).astype(np.int64))


def check_f32(got, ref, what, canary=False):
    got = got.double().cpu().numpy() if isinstance(got, torch.Tensor) else got
    assert np.isfinite(got).all(), "%s: non-finite output" % what
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    say("%s: fp32 out max-abs %.3e rel-L2 %.3e" % (what, err.max(), rel))
    assert err.max() <= GATE_MAX_ABS and rel <= GATE_REL_L2, what
    if canary:
        assert err.max() <= CANARY_MAX_ABS and rel <= CANARY_REL_L2, \
            "%s: precision canary (max-abs %.3e rel-L2 %.3e)" % (what, err.max(), rel)
    return err.max(), rel


def check_bf16(got, ref, what):
    got = got.float().cpu().double().numpy()
    assert np.isfinite(got).all()
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    bound = np.maximum(1e-2, bf16_ulp(ref))
    say("%s: bf16 out max-abs %.3e rel-L2 %.3e worst err/bound %.3f"
        % (what, err.max(), rel, (err / bound).max()))
    assert rel <= 5e-3 and (err <= bound).all(), what


def custom(lengths, hq=32, hkv=8, seed=0, fill="nan", shuffle=True, pt_stride=None):
    w = Workload("custom", len(lengths), hq, hkv, 128, 16, "fixed", tuple(lengths))
    return make_case(w, seed=seed, fill=fill, shuffle=shuffle, pt_stride=pt_stride)


# ------------------------------------------------------------------ workloads
@pytest.mark.parametrize("name", ORDER + SHARDS)
def test_workload_parity(name):
    say("case: workload %s seed 0" % name)
    c = make_case(name, seed=0, fill="nan")
    say("  N_req %d N_kv %d pages %d" % (c["num_seqs"], c["n_kv"], c["num_pages"]))
    d = dev_case(c)
    got32 = run_gpu(d, torch.float32)
    got16 = run_gpu(d, torch.bfloat16)
    ref = ref_of(c)
    check_f32(got32, ref, name, canary=True)
    check_bf16(got16, ref, name)


# ------------------------------------------------------------------ bit-exact gather
@pytest.mark.parametrize("name", ["tiny_b4", "llama8b_b64", "long_b16", "edges"])
def test_gather_copy_through_bit_exact(name):
    say("case: gather %s" % name)
    if name == "edges":
        c = custom([1, 15, 16, 17, 0, 33, 64, 1000, 3], hkv=8)
    else:
        c = make_case(name, seed=0, fill="nan")
    d = dev_case(c)
    n = c["n_kv"]
    ko = torch.empty((max(n, 1), c["n_kv_heads"], 128), dtype=torch.bfloat16, device=DEV)
    vo = torch.empty_like(ko)
    ws = vd.alloc_workspace(c["num_seqs"], c["n_kv_heads"], c["n_kv_heads"], c["max_pages_per_seq"])
    vd.vd_decode_gather(d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], ko, vo, ws)
    torch.cuda.synchronize()
    kr, vr = oracle.gather(bits(c["k_pages"]), bits(c["v_pages"]), c["page_table"].numpy(),
                           c["seq_lens"].numpy())
    assert np.array_equal(bits(ko[:n].cpu()), kr)
    assert np.array_equal(bits(vo[:n].cpu()), vr)


# ------------------------------------------------------------------ closed forms, exact
def test_single_token_is_v_row():
    say("case: L=1 x 37 requests")
    c = custom([1] * 37, hq=32, hkv=8, seed=3)
    d = dev_case(c)
    pt = c["page_table"].numpy()
    vrows = bits(c["v_pages"])[pt[:, 0], 0]                    # [B][Hkv][D]
    expect = np.repeat(vrows, 4, axis=1)                       # [B][Hq][D]
    got16 = bits(run_gpu(d, torch.bfloat16).cpu())
    assert np.array_equal(got16, expect)
    got32 = run_gpu(d, torch.float32).cpu().numpy()
    assert np.array_equal(got32, (expect.astype(np.uint32) << 16).view(np.float32))


@pytest.mark.parametrize("split", [0, 1, 3])
def test_one_hot_is_v_row(split):
    lengths = [1, 40, 300, 17, 2000, 5000, 16, 33]
    hot = [0, 39, 150, 16, 1999, 2500, 0, 32]
    say("case: one-hot split=%d" % split)
    c = pins.onehot_case(lengths, 32, 8, 11, hot)
    q = torch.from_numpy(c["q"].view(np.int16)).view(torch.bfloat16)
    k = torch.from_numpy(c["k"].view(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(c["v"].view(np.int16)).view(torch.bfloat16)
    d = dict(q=q.to(DEV), k_pages=k.to(DEV), v_pages=v.to(DEV),
             page_table=torch.from_numpy(c["pt"]).to(DEV), seq_lens=torch.from_numpy(c["L"]).to(DEV),
             scale=c["scale"], num_seqs=len(lengths), n_q_heads=32, n_kv_heads=8,
             max_pages_per_seq=c["pt"].shape[1])
    flags = vd.VD_FLAG_RANGE_TILES(split) if split else 0
    got = run_gpu(d, torch.float32, flags=flags).cpu().numpy()
    for b, t in enumerate(hot):
        vrow = c["v"][c["pt"][b, t // 16], t % 16]             # [Hkv][D]
        expect = (np.repeat(vrow, 4, axis=0).astype(np.uint32) << 16).view(np.float32)
        assert np.array_equal(got[b], expect), b


def test_constant_v():
    say("case: constant V")
    c = custom([1, 15, 16, 17, 100, 3000], hq=32, hkv=8, seed=4)
    vb = c["v_pages"].view(torch.int16)
    const = torch.randn(8, 128).to(torch.bfloat16).view(torch.int16)
    pt = c["page_table"].numpy()
    for b, n in enumerate(c["seq_lens"].tolist()):
        for t in range(n):
            vb[pt[b, t // 16], t % 16] = const
    got = run_gpu(dev_case(c), torch.float32).cpu().double()
    expect = const.view(torch.bfloat16).double().repeat_interleave(4, dim=0)
    rel = ((got - expect).abs() / expect.abs().clamp_min(1e-30)).max().item()
    say("  constant V max rel %.3e" % rel)
    assert rel <= 1e-5


# ------------------------------------------------------------------ invariances
def test_page_permutation_bit_exact():
    say("case: page permutation")
    lengths = [37, 128, 500, 1000, 4000, 1]
    a = custom(lengths, seed=6, shuffle=False)
    perm = torch.randperm(a["num_pages"], generator=torch.Generator().manual_seed(9))
    b = dict(a)
    b["k_pages"] = torch.empty_like(a["k_pages"])
    b["v_pages"] = torch.empty_like(a["v_pages"])
    b["k_pages"][perm] = a["k_pages"]
    b["v_pages"][perm] = a["v_pages"]
    b["page_table"] = perm.to(torch.int32)[a["page_table"].long()]
    for dt in (torch.float32, torch.bfloat16):
        x = run_gpu(dev_case(a), dt).cpu()
        y = run_gpu(dev_case(b), dt).cpu()
        assert torch.equal(x.view(torch.int16) if dt == torch.bfloat16 else x.view(torch.int32),
                           y.view(torch.int16) if dt == torch.bfloat16 else y.view(torch.int32))


def test_nan_fill_and_determinism():
    say("case: NaN vs zero fill, determinism")
    lengths = [5, 17, 31, 250, 1111, 4097]
    a = custom(lengths, seed=7, fill="nan")
    z = custom(lengths, seed=7, fill="zero")
    x1 = run_gpu(dev_case(a)).cpu()
    x2 = run_gpu(dev_case(a)).cpu()
    y = run_gpu(dev_case(z)).cpu()
    assert torch.isfinite(x1).all()
    assert torch.equal(x1.view(torch.int32), x2.view(torch.int32))
    assert torch.equal(x1.view(torch.int32), y.view(torch.int32))


def test_split_invariance():
    say("case: forced range lengths")
    c = make_case("tiny_b4", seed=0)
    extra = custom([3000, 77, 1, 4096, 700], seed=8)
    for cc in (c, extra):
        d = dev_case(cc)
        base = run_gpu(d).cpu().double()
        ref = ref_of(cc)
        check_f32(base, ref, "split auto")
        for s in (1, 2, 7, 64, 255):
            got = run_gpu(d, flags=vd.VD_FLAG_RANGE_TILES(s)).cpu().double()
            rel = ((got - base).norm() / base.norm()).item()
            say("  split %d rel diff %.3e" % (s, rel))
            assert rel <= 1e-5
            check_f32(got, ref, "split %d" % s)


@pytest.mark.parametrize("lengths", [[16384], [60000, 3], [131072]])
def test_few_long_requests(lengths):
    """Few long requests: every CU takes a slice of them, so each (request,
    head group) is split into many pieces that the combine must merge."""
    say("case: long requests %s" % lengths)
    c = custom(lengths, seed=20 + len(lengths))
    d = dev_case(c)
    ref = ref_of(c)
    check_f32(run_gpu(d), ref, "long %s" % lengths, canary=True)
    check_bf16(run_gpu(d, torch.bfloat16), ref, "long %s" % lengths)


def test_pt_stride():
    say("case: wide page-table rows")
    c = custom([100, 7, 900], seed=10, pt_stride=200)
    check_f32(run_gpu(dev_case(c)), ref_of(c), "pt stride 200")


def test_length_clamped_to_table():
    """A length past the page table's capacity (max_pages_per_seq * 16) is
    clamped to it: the result equals that of the capacity itself, bit for
    bit, in the whole step, the staged calls and the gather."""
    say("case: lengths clamped to the table")
    c = custom([40, 160, 7], seed=24, pt_stride=10)       # 10 pages = 160 tokens
    d = dev_case(c)
    ref = run_gpu(d)
    check_f32(ref, ref_of(c), "at capacity")
    d2 = dict(d)
    d2["seq_lens"] = torch.tensor([40, 1000, 7], dtype=torch.int32, device=DEV)
    assert torch.equal(run_gpu(d2).view(torch.int32).cpu(), ref.view(torch.int32).cpu())
    ws = vd.alloc_workspace(3, 32, 8, 10)
    staged = torch.empty_like(ref)
    vd.vd_decode_plan(d2["seq_lens"], 32, 8, 10, ws)
    vd.vd_decode_partial(d2["q"], d2["k_pages"], d2["v_pages"], d2["page_table"], d2["seq_lens"],
                         staged, d2["scale"], ws)
    vd.vd_decode_combine(staged, 8, 10, ws)
    torch.cuda.synchronize()
    assert torch.equal(staged.view(torch.int32).cpu(), ref.view(torch.int32).cpu())
    n = 40 + 160 + 7
    ko = torch.empty((n, 8, 128), dtype=torch.bfloat16, device=DEV)
    vo = torch.empty_like(ko)
    gws = vd.alloc_workspace(3, 8, 8, 10)
    vd.vd_decode_gather(d2["k_pages"], d2["v_pages"], d2["page_table"], d2["seq_lens"], ko, vo, gws)
    torch.cuda.synchronize()
    kr, vr = oracle.gather(bits(c["k_pages"]), bits(c["v_pages"]), c["page_table"].numpy(),
                           c["seq_lens"].numpy())
    assert np.array_equal(bits(ko.cpu()), kr) and np.array_equal(bits(vo.cpu()), vr)


# ------------------------------------------------------------------ shapes and edges
def test_page_boundary_lengths():
    lengths = [1, 15, 16, 17, 31, 32, 33, 255, 256, 257, 1023, 1024, 1025]
    say("case: page-boundary lengths %s" % lengths)
    c = custom(lengths, seed=12)
    d = dev_case(c)
    ref = ref_of(c)
    check_f32(run_gpu(d), ref, "boundaries")
    check_bf16(run_gpu(d, torch.bfloat16), ref, "boundaries")


@pytest.mark.parametrize("G,hkv", [(1, 4), (2, 4), (4, 2), (8, 2), (16, 1), (8, 8)])
def test_gqa_ratios(G, hkv):
    say("case: G=%d Hkv=%d" % (G, hkv))
    c = custom([1, 20, 300, 2222, 64], hq=G * hkv, hkv=hkv, seed=13 + G)
    d = dev_case(c)
    ref = ref_of(c)
    check_f32(run_gpu(d), ref, "G=%d" % G)
    check_bf16(run_gpu(d, torch.bfloat16), ref, "G=%d" % G)


def test_max_requests():
    """8192 requests (the supported maximum): every planner thread owns eight
    requests, every thread of a self-planning attention workgroup 64; mixed
    tiny, empty and one long request.  Staged and whole step agree bit for
    bit."""
    rng = np.random.default_rng(40)
    lengths = [int(x) for x in rng.choice([0, 1, 2, 7, 16, 17, 40], 8192)]
    lengths[4097] = 5000
    say("case: 8192 requests, N_kv %d" % sum(lengths))
    c = custom(lengths, hq=8, hkv=2, seed=41)
    d = dev_case(c)
    ref = ref_of(c)
    whole = run_gpu(d)
    check_f32(whole, ref, "8192 requests")
    maxp = c["max_pages_per_seq"]
    ws = vd.alloc_workspace(8192, 8, 2, maxp)
    staged = torch.full(d["q"].shape, float("nan"), dtype=torch.float32, device=DEV)
    vd.vd_decode_plan(d["seq_lens"], 8, 2, maxp, ws)
    vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                         staged, d["scale"], ws)
    vd.vd_decode_combine(staged, 2, maxp, ws)
    torch.cuda.synchronize()
    assert torch.equal(whole.view(torch.int32).cpu(), staged.view(torch.int32).cpu())


@pytest.mark.parametrize("G,hkv", [(16, 1), (16, 2), (8, 2)])
def test_many_pieces_per_wave(G, hkv):
    """Thousands of short requests: a wave finishes more pieces than it can
    hold results for in LDS (64 / G), so results are written out mid-stream
    as well as at the end."""
    rng = np.random.default_rng(50 + G + hkv)
    lengths = [int(x) for x in rng.choice([1, 3, 16, 17, 40, 100], 3000)]
    say("case: 3000 short requests, G=%d Hkv=%d, N_kv %d" % (G, hkv, sum(lengths)))
    c = custom(lengths, hq=G * hkv, hkv=hkv, seed=51 + G)
    d = dev_case(c)
    ref = ref_of(c)
    check_f32(run_gpu(d), ref, "many pieces G=%d" % G)
    check_bf16(run_gpu(d, torch.bfloat16), ref, "many pieces G=%d" % G)


def test_sixteen_kv_heads():
    say("case: 32:16 heads and 16:16 heads")
    for hq, hkv in ((32, 16), (16, 16)):
        c = custom([1, 100, 2049, 33], hq=hq, hkv=hkv, seed=42 + hq)
        check_f32(run_gpu(dev_case(c)), ref_of(c), "Hq %d Hkv %d" % (hq, hkv))


def test_empty_requests():
    say("case: empty requests")
    c = custom([0, 5, 0, 300, 0], seed=14)
    got = run_gpu(dev_case(c)).cpu()
    assert torch.equal(got[0], torch.zeros_like(got[0])) and torch.equal(got[2], torch.zeros_like(got[2]))
    assert torch.equal(got[4], torch.zeros_like(got[4]))
    check_f32(got, ref_of(c), "empty")
    z = custom([0, 0, 0], seed=15)
    got = run_gpu(dev_case(z)).cpu()
    assert torch.equal(got, torch.zeros_like(got))


@pytest.mark.parametrize("case", ["mixed_le64", "ragged_le16", "one_page_each", "all_empty_short",
                                  "at_limit"])
def test_short_plan_steps(case):
    """Tiny steps (every request at most 4 pages, at most a quarter as many
    (page, head group) tiles as resident workgroups) take the short plan:
    ranges start at segment starts, every piece is a whole segment, the whole
    step runs no combine kernel and the attention kernel writes the empty
    requests' zeros.  Against the oracle, empty rows exactly zero over
    NaN-filled output, and bit for bit equal to the staged calls (planner
    kernel, attention, combine) on the same plan."""
    rng = np.random.default_rng(77)
    if case == "mixed_le64":
        lengths = [0, 5, 0, 64, 0, 17, 1, 33]
    elif case == "ragged_le16":
        lengths = [int(x) for x in rng.integers(0, 17, 30)]
        lengths[7] = 0
    elif case == "one_page_each":
        lengths = [16] * 32
    elif case == "all_empty_short":
        lengths = [0] * 30
    else:                             # 8 x 2 x 4 tiles: exactly R / 4 at 256 workgroups
        lengths = [64, 49, 50, 63, 64, 1, 60, 64]
    say("case: short plan %s (%d requests, longest %d)" % (case, len(lengths), max(lengths)))
    c = custom(lengths, seed=78)
    d = dev_case(c)
    ref = ref_of(c)
    for dtype in (torch.float32, torch.bfloat16):
        whole = run_gpu(d, dtype)
        empty = [b for b, x in enumerate(lengths) if x == 0]
        if empty:
            assert torch.equal(whole[empty], torch.zeros_like(whole[empty]))
        if dtype is torch.float32:
            check_f32(whole, ref, "short " + case, canary=True)
        else:
            check_bf16(whole, ref, "short " + case)
        maxp = d["page_table"].shape[1]
        ws = vd.alloc_workspace(len(lengths), 32, 8, maxp)
        staged = torch.full(d["q"].shape, float("nan"), dtype=dtype, device=DEV)
        vd.vd_decode_plan(d["seq_lens"], 32, 8, maxp, ws)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], staged,
                             d["scale"], ws)
        vd.vd_decode_combine(staged, 8, maxp, ws)
        torch.cuda.synchronize()
        view = torch.int32 if dtype is torch.float32 else torch.int16
        assert torch.equal(staged.view(view), whole.view(view))
        info = vd.step_info(ws)
        assert info["n_ranges"] <= 256 and info["n_empty"] == len(empty)


def test_large_scores():
    """Scores around 5.8e3: only a max-subtracted softmax survives."""
    say("case: large scores")
    c = custom([40, 3, 777, 5000], seed=16, fill="zero")
    c["k_pages"].view(torch.int16)[:, :, :, 7] = pins.bf16_bits(256.0)
    c["q"].view(torch.int16)[:, :, 7] = pins.bf16_bits(256.0)
    check_f32(run_gpu(dev_case(c)), ref_of(c), "large scores")


def test_staged_plan_once_two_layers():
    say("case: plan once, two attention layers")
    c = custom([33, 900, 5000, 1], seed=17)
    c2 = custom([33, 900, 5000, 1], seed=18, fill="zero")
    d, d2 = dev_case(c), dev_case(c2)
    ws = vd.alloc_workspace(4, 32, 8, c["max_pages_per_seq"])
    vd.vd_decode_plan(d["seq_lens"], 32, 8, c["max_pages_per_seq"], ws)
    outs = []
    for dd in (d, d2):
        out = torch.empty(dd["q"].shape, dtype=torch.float32, device=DEV)
        # same lengths and placement; different values (another layer)
        vd.vd_decode_partial(dd["q"], dd["k_pages"], dd["v_pages"], d["page_table"],
                             d["seq_lens"], out, dd["scale"], ws)
        vd.vd_decode_combine(out, 8, c["max_pages_per_seq"], ws)
        outs.append(out)
    torch.cuda.synchronize()
    c2["page_table"] = c["page_table"]
    check_f32(outs[0], ref_of(c), "layer 0")
    check_f32(outs[1], ref_of(c2), "layer 1")
    fused = run_gpu(d)
    assert torch.equal(outs[0].view(torch.int32).cpu(), fused.view(torch.int32).cpu())


@pytest.mark.parametrize("case", ["tiny_b4", "long_b16", "mixed", "mixed_forced7", "split_many"])
def test_staged_equals_whole_step(case):
    """The whole step plans inside the attention kernel; the staged API runs
    the planner kernel first.  Both cut the same ranges, so their outputs
    agree bit for bit, in both output types."""
    say("case: staged vs whole step, %s" % case)
    flags = 0
    if case in ("tiny_b4", "long_b16"):
        c = make_case(case, seed=0, fill="nan")
    elif case == "split_many":
        c = custom([16384, 3, 0, 9000], seed=21)
    else:
        c = custom([0, 5, 300, 0, 2049, 1, 16, 17, 7000, 0], seed=22)
        flags = vd.VD_FLAG_RANGE_TILES(7) if case == "mixed_forced7" else 0
    d = dev_case(c)
    B, Hq, Hkv, maxp = c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"]
    for dt in (torch.float32, torch.bfloat16):
        whole = run_gpu(d, dt, flags=flags)
        ws = vd.alloc_workspace(B, Hq, Hkv, maxp, flags)
        staged = torch.full(d["q"].shape, float("nan"), dtype=dt, device=DEV)
        vd.vd_decode_plan(d["seq_lens"], Hq, Hkv, maxp, ws, flags=flags)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             staged, d["scale"], ws, flags=flags)
        vd.vd_decode_combine(staged, Hkv, maxp, ws, flags=flags)
        # the self-planned kernel through the staged calls, on a workspace
        # that still holds the planner's tables
        selfp = torch.full(d["q"].shape, float("nan"), dtype=dt, device=DEV)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             selfp, d["scale"], ws, flags=flags | vd.VD_FLAG_SELF_PLAN)
        vd.vd_decode_combine(selfp, Hkv, maxp, ws, flags=flags)
        torch.cuda.synchronize()
        iv = torch.int32 if dt == torch.float32 else torch.int16
        assert torch.equal(whole.view(iv).cpu(), staged.view(iv).cpu()), case
        assert torch.equal(whole.view(iv).cpu(), selfp.view(iv).cpu()), case
    check_f32(run_gpu(d, flags=flags), ref_of(c), case)


def _step_record(ws):
    raw = ws[:48].cpu().numpy()
    n = raw[:16].view(np.int32)
    t0, c0, t1, c1 = (int(x) for x in raw[16:48].view(np.uint64))
    return n, t0, c0, t1, c1


def test_step_record():
    """The step record at the head of the workspace (vd_step_info): the
    plan's tile and empty-request counts, and real-time / shader-clock
    stamps of the first workgroup that fit inside the launch and give a
    plausible clock."""
    say("case: step record")
    lens = [37, 700, 4100, 0, 260]
    c = custom(lens, seed=23)
    d = dev_case(c)
    tiles = sum((x + 15) // 16 for x in lens) * 2          # 8 KV heads in groups of 4
    for staged in (False, True):
        ws = vd.alloc_workspace(5, 32, 8, c["max_pages_per_seq"])
        ws.zero_()
        out = torch.empty(d["q"].shape, dtype=torch.float32, device=DEV)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        flags = 0
        if staged:
            vd.vd_decode_plan(d["seq_lens"], 32, 8, c["max_pages_per_seq"], ws)
        else:
            flags = vd.VD_FLAG_SELF_PLAN
        e0.record()
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             out, d["scale"], ws, flags=flags)
        e1.record()
        vd.vd_decode_combine(out, 8, c["max_pages_per_seq"], ws)
        torch.cuda.synchronize()
        n, t0, c0, t1, c1 = _step_record(ws)
        us_event = e0.elapsed_time(e1) * 1e3
        us_first = (t1 - t0) * 0.01
        mhz = (c1 - c0) * 100.0 / max(t1 - t0, 1)
        say("  staged %s: ranges %d tiles %d empty %d, first group %.1f us (launch %.1f us), "
            "shader clock %.0f MHz" % (staged, n[0], n[1], n[2], us_first, us_event, mhz))
        assert n[1] == tiles and n[2] == 1 and 1 <= n[0] <= tiles
        assert t1 > t0 and c1 > c0
        assert us_first <= 1.5 * us_event + 20.0
        assert 10.0 <= mhz <= 3500.0   # the clock may still be ramping up from idle
        check_f32(out, ref_of(c), "step record run")


def test_largest_surface_point_sampled():
    """The largest point of the latency surface: 512 requests of 16384 tokens
    (8.4 M tokens, 34 GB of K/V), drawn on the device.  32 sampled (request,
    query head) rows against the oracle's row function, which reads only
    those requests' pages (copied to the host as a compact pool with its own
    page table)."""
    from workloads import make_device_case
    B, L = 512, 16384
    say("case: largest surface point, %d requests x %d tokens (sampled)" % (B, L))
    d = make_device_case(B, L, 32, 8, seed=31, device=DEV)
    out = torch.full(d["q"].shape, float("nan"), dtype=torch.float32, device=DEV)
    ws = vd.alloc_workspace(B, 32, 8, d["max_pages_per_seq"])
    vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out,
                      d["scale"], ws)
    torch.cuda.synchronize()
    reqs = [0, 37, 101, 255, 256, 390, 477, 511]
    heads = [0, 5, 18, 31]
    pt = d["page_table"][reqs]                                   # [8][P], device
    P = pt.shape[1]
    kc = bits(d["k_pages"][pt.reshape(-1).long()].cpu())         # compact pools
    vc = bits(d["v_pages"][pt.reshape(-1).long()].cpu())
    ptc = np.arange(len(reqs) * P, dtype=np.int32).reshape(len(reqs), P)
    sel_b = np.repeat(np.arange(len(reqs)), len(heads)).astype(np.int32)
    sel_h = np.tile(heads, len(reqs)).astype(np.int32)
    ref = oracle.decode_attn_rows(bits(d["q"][reqs].cpu()), kc, vc, ptc,
                                  np.full(len(reqs), L, dtype=np.int32), d["scale"], sel_b, sel_h)
    got = out[reqs][:, heads].reshape(-1, 128).double().cpu().numpy()
    check_f32(got, ref, "largest surface point, sampled rows", canary=True)
    del d, out, ws
    torch.cuda.empty_cache()


def test_step_record_clock_after_settle():
    """After the power manager has brought the shader clock up (tens of ms of
    steady work), the stamped clock is a real shader clock: within 1000-2600
    MHz (MI355X peaks at 2400 MHz; its manager moves it between ~1.4 and
    2.4 GHz under load).  A stamp that read the wrong counter (e.g. the
    100 MHz real-time counter twice) would fail.  The first workgroup lives
    for most of the launch: all workgroups are resident from the start and
    take equal shares of the tiles."""
    say("case: step record after clock settle")
    c = custom([2048] * 64, seed=24, fill="zero")
    d = dev_case(c)
    ws = vd.alloc_workspace(64, 32, 8, c["max_pages_per_seq"])
    out = torch.empty(d["q"].shape, dtype=torch.bfloat16, device=DEV)

    def launch():
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             out, d["scale"], ws, flags=vd.VD_FLAG_SELF_PLAN)

    import time
    t_end = time.time() + 0.1
    while time.time() < t_end:
        for _ in range(20):
            launch()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(20):
        launch()
    e1.record()
    torch.cuda.synchronize()
    us_kernel = e0.elapsed_time(e1) * 1e3 / 20
    n, t0, c0, t1, c1 = _step_record(ws)     # the last launch's record
    us_first = (t1 - t0) * 0.01
    mhz = (c1 - c0) * 100.0 / max(t1 - t0, 1)
    say("  first group %.1f us of %.1f us per launch, shader clock %.0f MHz" % (us_first, us_kernel, mhz))
    assert 1000.0 <= mhz <= 2600.0
    assert 0.6 * us_kernel <= us_first <= 1.05 * us_kernel


@pytest.mark.parametrize("trial", range(8))
def test_staged_equals_whole_random(trial):
    """Seeded random shapes, with request counts past one per planning thread
    (up to 3000) and every KV-head group width: the self-planned kernel and
    the planner kernel cut the same ranges, so the whole step, the staged
    calls and the self-planned staged calls agree bit for bit."""
    rng = np.random.default_rng(3000 + trial)
    hkv = int(rng.choice([1, 2, 4, 8, 16]))
    G = int(rng.choice([1, 4, 16])) if hkv < 16 else int(rng.choice([1, 4]))
    B = (7, 64, 300, 1100, 3000, 1, 300, 1100)[trial]
    pool = np.array([0, 1, 15, 16, 17, 33, 100, 257, 700])
    lengths = [int(x) for x in rng.choice(pool, B)]
    lengths[int(rng.integers(0, B))] = int(rng.integers(1000, 6000))
    flags = vd.VD_FLAG_RANGE_TILES(int(rng.integers(1, 256))) if rng.random() < 0.3 else 0
    say("case: staged vs whole, trial %d B %d G %d Hkv %d flags %#x" % (trial, B, G, hkv, flags))
    c = custom(lengths, hq=G * hkv, hkv=hkv, seed=3100 + trial, fill="zero")
    d = dev_case(c)
    Hq, maxp = G * hkv, c["max_pages_per_seq"]
    whole = run_gpu(d, flags=flags)
    outs = []
    for self_plan in (False, True):
        ws = vd.alloc_workspace(B, Hq, hkv, maxp, flags)
        o = torch.full(d["q"].shape, float("nan"), dtype=torch.float32, device=DEV)
        if not self_plan:
            vd.vd_decode_plan(d["seq_lens"], Hq, hkv, maxp, ws, flags=flags)
        vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                             o, d["scale"], ws,
                             flags=flags | (vd.VD_FLAG_SELF_PLAN if self_plan else 0))
        vd.vd_decode_combine(o, hkv, maxp, ws, flags=flags)
        outs.append(o)
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int32).cpu(), whole.view(torch.int32).cpu())
    assert torch.isfinite(whole).all()


def test_hip_graph_replay_staged_layers():
    """A decode iteration of a two-layer model in the staged form, captured
    into one HIP graph: one plan, then attention and combine per layer (each
    layer its own Q and KV pools, one workspace).  Every replay, with eager
    work and a synchronisation between replays, equals the eager calls bit
    for bit, and the per-layer outputs match the oracle."""
    say("case: HIP graph capture and replay of plan + 2 x (partial, combine)")
    layers = [custom([37, 700, 4100, 1, 0, 260], seed=21 + i) for i in range(2)]
    ds = [dev_case(c) for c in layers]
    maxp = layers[0]["max_pages_per_seq"]
    assert all(c["max_pages_per_seq"] == maxp for c in layers)
    assert all(torch.equal(c["seq_lens"], layers[0]["seq_lens"]) for c in layers)
    B = layers[0]["num_seqs"]
    ws = vd.alloc_workspace(B, 32, 8, maxp)

    def iteration(outs):
        vd.vd_decode_plan(ds[0]["seq_lens"], 32, 8, maxp, ws)
        for d, o in zip(ds, outs):
            vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"],
                                 o, d["scale"], ws)
            vd.vd_decode_combine(o, 8, maxp, ws)

    eager = [torch.empty(d["q"].shape, dtype=torch.float32, device=DEV) for d in ds]
    iteration(eager)
    outs = [torch.empty_like(e) for e in eager]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        iteration(outs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        iteration(outs)
    for i in range(3):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o.view(torch.int32), e.view(torch.int32)), "replay %d" % i
        iteration(eager)   # eager work between replays
        torch.cuda.synchronize()
    for o, c in zip(outs, layers):
        check_f32(o, ref_of(c), "staged graph layer")


def test_concurrent_streams_distinct_workspaces():
    """Two steps of different shapes enqueued on two streams at once, each
    with its own workspace (default stream priorities): both results equal
    the same steps run one after the other, bit for bit."""
    say("case: two streams, two workspaces")
    cases = [custom([3000, 17, 900, 0, 64], seed=25),
             custom([5, 12000, 1, 300], hq=64, hkv=8, seed=26)]
    ds = [dev_case(c) for c in cases]
    wss = [vd.alloc_workspace(c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"])
           for c in cases]
    serial = [run_gpu(d) for d in ds]
    outs = [torch.full(d["q"].shape, float("nan"), dtype=torch.float32, device=DEV) for d in ds]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for _ in range(3):
        for d, o, ws, st in zip(ds, outs, wss, streams):
            with torch.cuda.stream(st):
                vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"],
                                  d["seq_lens"], o, d["scale"], ws)
    torch.cuda.synchronize()
    for o, e, c in zip(outs, serial, cases):
        assert torch.equal(o.view(torch.int32), e.view(torch.int32))
        check_f32(o, ref_of(c), "concurrent")


def test_workspace_reuse_across_steps():
    """One workspace serves steps of different length mixes in a row: what a
    longer step left in it (ranges, boundary records, partials) never leaks
    into a later, smaller one."""
    say("case: workspace reuse across steps")
    mixes = [[9000, 4000, 2500, 777], [0, 33, 0, 5], [0, 0, 0, 0], [16, 16, 16, 16], [12000, 1, 0, 40]]
    maxp = (12000 + 15) // 16
    ws = vd.alloc_workspace(4, 32, 8, maxp)
    for i, lens in enumerate(mixes):
        c = custom(lens, seed=40 + i, pt_stride=maxp)
        d = dev_case(c)
        got = run_gpu(d, ws=ws)
        fresh = run_gpu(d)
        assert torch.equal(got.view(torch.int32).cpu(), fresh.view(torch.int32).cpu()), lens
        check_f32(got, ref_of(c), "reuse step %d" % i)


def test_hip_graph_replay():
    """A whole step (attention and combine kernels) captured into a HIP
    graph: every replay, with eager work and a synchronisation between
    replays, equals the eager result bit for bit, and a replay after new Q
    values are written in place gives the new eager result."""
    say("case: HIP graph capture and replay of vd_decode_attn")
    c = custom([37, 700, 4100, 1, 260], seed=19)
    d = dev_case(c)
    maxp = c["max_pages_per_seq"]
    ws = vd.alloc_workspace(5, 32, 8, maxp)

    def step(out):
        vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out,
                          d["scale"], ws)

    eager = torch.empty(d["q"].shape, dtype=torch.float32, device=DEV)
    step(eager)
    out = torch.empty_like(eager)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(out)
    for i in range(4):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), eager.view(torch.int32)), "replay %d" % i
    check_f32(out, ref_of(c), "graph replay")
    gen = torch.Generator(device="cpu").manual_seed(20)
    d["q"].copy_(torch.randn(d["q"].shape, generator=gen).to(torch.bfloat16))
    step(eager)
    out.fill_(float("nan"))
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), eager.view(torch.int32)), "replay with new Q"


# ------------------------------------------------------------------ randomized sweep
@pytest.mark.parametrize("trial", range(12))
def test_random_shapes(trial):
    """Seeded random shapes: request count, GQA ratio, KV heads, a length mix
    with empty, one-token, page-boundary and long requests, table stride and
    range size."""
    rng = np.random.default_rng(1000 + trial)
    hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 8, 16]))
    B = int(rng.integers(1, 40))
    pool = [0, 1, 15, 16, 17, 31, 33, 255, 256, 257] + list(rng.integers(1, 3000, 8))
    lengths = [int(rng.choice(pool)) for _ in range(B)]
    if rng.random() < 0.3:
        lengths[int(rng.integers(0, B))] = int(rng.integers(8000, 40000))
    maxp = max(1, max((x + 15) // 16 for x in lengths))
    stride = maxp + int(rng.integers(0, 5))
    flags = vd.VD_FLAG_RANGE_TILES(int(rng.integers(1, 256))) if rng.random() < 0.4 else 0
    say("case: random trial %d B %d G %d Hkv %d flags %#x lengths %s"
        % (trial, B, G, hkv, flags, lengths))
    c = custom(lengths, hq=G * hkv, hkv=hkv, seed=2000 + trial, pt_stride=stride)
    d = dev_case(c)
    ref = ref_of(c)
    check_f32(run_gpu(d, flags=flags), ref, "random %d" % trial, canary=True)
    check_bf16(run_gpu(d, torch.bfloat16, flags=flags), ref, "random %d" % trial)


@pytest.mark.parametrize("trial", range(40))
def test_random_sweep(trial):
    """A wider seeded sweep: up to 400 requests, KV heads 1-16, every GQA
    ratio, four length laws (short, lognormal, page boundaries, uniform) with
    empty requests and an occasional 10k-60k-token request, table strides
    past the longest request, and forced range lengths.  fp32 output against
    the oracle; the staged calls (planner kernel) equal the whole step bit
    for bit."""
    rng = np.random.default_rng(9000 + trial)
    hkv = int(rng.choice([1, 2, 4, 8, 16]))
    G = int(rng.choice([1, 2, 4, 8, 16]))
    G = min(G, max(1, 128 // hkv))
    B = int(np.exp(rng.uniform(0, np.log(400))))
    law = trial % 4
    if law == 0:
        lengths = rng.integers(0, 40, B)
    elif law == 1:
        lengths = np.clip(np.round(np.exp(rng.normal(np.log(300), 1.0, B))), 0, 20000)
    elif law == 2:
        lengths = rng.choice([0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 255, 256, 257, 1024], B)
    else:
        lengths = rng.integers(1, 3000, B)
    lengths = [int(x) for x in lengths]
    if rng.random() < 0.2:
        lengths[int(rng.integers(0, B))] = int(rng.integers(10000, 60000))
    stride = max(1, max((x + 15) // 16 for x in lengths)) + int(rng.integers(0, 4))
    flags = vd.VD_FLAG_RANGE_TILES(int(rng.integers(1, 256))) if rng.random() < 0.3 else 0
    what = "sweep %d B %d G %d Hkv %d flags %#x N_kv %d" % (trial, B, G, hkv, flags, sum(lengths))
    say("case: " + what)
    c = custom(lengths, hq=G * hkv, hkv=hkv, seed=9500 + trial, pt_stride=stride)
    d = dev_case(c)
    ref = ref_of(c)
    whole = run_gpu(d, torch.float32, flags=flags)
    check_f32(whole, ref, what, canary=True)
    if trial % 4 == 0:
        check_bf16(run_gpu(d, torch.bfloat16, flags=flags), ref, what)
    maxp = d["page_table"].shape[1]
    ws = vd.alloc_workspace(B, G * hkv, hkv, maxp, flags)
    staged = torch.full(d["q"].shape, float("nan"), dtype=torch.float32, device=DEV)
    vd.vd_decode_plan(d["seq_lens"], G * hkv, hkv, maxp, ws, flags=flags)
    vd.vd_decode_partial(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], staged,
                         d["scale"], ws, flags=flags)
    vd.vd_decode_combine(staged, hkv, maxp, ws, flags=flags)
    torch.cuda.synchronize()
    assert torch.equal(staged.view(torch.int32).cpu(), whole.view(torch.int32).cpu()), what


# ------------------------------------------------------------------ KV append
def test_kv_append_bit_exact():
    say("case: KV append")
    c = custom([16, 1, 33, 0, 5, 100, 257, 15], seed=30, pt_stride=20)
    B = c["num_seqs"]
    positions = torch.tensor([15, 1, 33, -1, 4, 100, 320, 319], dtype=torch.int32)
    g = torch.Generator().manual_seed(31)
    k_new = torch.randn((B, 8, 128), generator=g).to(torch.bfloat16)
    v_new = torch.randn((B, 8, 128), generator=g).to(torch.bfloat16)
    d = dev_case(c)
    vd.vd_kv_append(k_new.to(DEV), v_new.to(DEV), d["k_pages"], d["v_pages"], d["page_table"],
                    positions.to(DEV))
    torch.cuda.synchronize()
    hk, hv = bits(c["k_pages"]).copy(), bits(c["v_pages"]).copy()
    oracle.kv_append(bits(k_new), bits(v_new), hk, hv, c["page_table"].numpy(), positions.numpy())
    assert np.array_equal(bits(d["k_pages"].cpu()), hk)
    assert np.array_equal(bits(d["v_pages"].cpu()), hv)


def test_decode_step_append_then_attend():
    """One decode iteration: append each request's newest K/V at position L_b,
    then attend over L_b + 1 tokens."""
    say("case: append then attend")
    lens = [15, 16, 1, 300, 4095, 17]
    c = custom([x + 1 for x in lens], seed=32)        # pages for the new token exist
    B = len(lens)
    pos = torch.tensor(lens, dtype=torch.int32)
    g = torch.Generator().manual_seed(33)
    k_new = torch.randn((B, 8, 128), generator=g).to(torch.bfloat16)
    v_new = torch.randn((B, 8, 128), generator=g).to(torch.bfloat16)
    d = dev_case(c)
    vd.vd_kv_append(k_new.to(DEV), v_new.to(DEV), d["k_pages"], d["v_pages"], d["page_table"],
                    pos.to(DEV))
    got = run_gpu(d)
    hk, hv = bits(c["k_pages"]).copy(), bits(c["v_pages"]).copy()
    oracle.kv_append(bits(k_new), bits(v_new), hk, hv, c["page_table"].numpy(), pos.numpy())
    ref = oracle.decode_attn(bits(c["q"]), hk, hv, c["page_table"].numpy(),
                             c["seq_lens"].numpy(), c["scale"])
    check_f32(got, ref, "append then attend")


def test_device_errors_leave_stream_clean():
    say("case: error codes on device")
    c = custom([10], seed=19)
    d = dev_case(c)
    out = torch.empty(d["q"].shape, dtype=torch.float32, device=DEV)
    small = torch.empty(16, dtype=torch.uint8, device=DEV)
    with pytest.raises(vd.VdError) as e:
        vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out,
                          d["scale"], small)
    assert e.value.status == vd.VD_ERROR_WORKSPACE_TOO_SMALL
    with pytest.raises(vd.VdError) as e:
        vd.vd_decode_attn(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["seq_lens"], out,
                          math.nan, small)
    assert e.value.status == vd.VD_ERROR_INVALID_VALUE
    check_f32(run_gpu(d), ref_of(c), "after errors")
