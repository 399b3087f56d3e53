"""Pins for the fp64 oracle, written independently of it.

Each pin states what the mathematics or the definition of the decode step
fixes (softmax attention of one query per request over its paged KV cache;
EcoPred's N_kv term, Sec. 5.4, Eq. pred-itl; paging, Sec. 2.1), without reusing
the oracle's code.  The pins take the oracle module as an argument so that the
mutation tests can run them against deliberately broken builds.

Every function raises AssertionError on a violated pin.
"""
from __future__ import annotations

import math
import struct

import numpy as np
import torch

from workloads import Workload, bits, make_case

SCALE = float(np.float32(1.0 / math.sqrt(128)))


def case(lengths, hq=8, hkv=2, d=128, s=16, seed=0, shuffle=True, pt_stride=None,
         fill="nan"):
    w = Workload("pin", len(lengths), hq, hkv, d, s, "fixed", tuple(lengths))
    c = make_case(w, seed=seed, fill=fill, shuffle=shuffle, pt_stride=pt_stride, threads=1)
    return dict(q=bits(c["q"]).copy(), k=bits(c["k_pages"]).copy(), v=bits(c["v_pages"]).copy(),
                pt=c["page_table"].numpy().copy(), L=c["seq_lens"].numpy().copy(),
                scale=c["scale"], S=s)


def run(orc, c, **kw):
    return orc.decode_attn(c["q"], c["k"], c["v"], c["pt"], c["L"], c["scale"], **kw)


def bf16_bits(x: float) -> int:
    """bits of an exactly representable bf16 value"""
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    assert u & 0xFFFF == 0, x
    return u >> 16


def f_of(h) -> float:
    return struct.unpack("<f", struct.pack("<I", int(h) << 16))[0]


# ---------------------------------------------------------------- brute force
def brute_force(c) -> np.ndarray:
    """Second formula, pure Python: contiguous gather, exactly rounded dot
    products (math.fsum) and softmax written as 1 / sum_u exp(s_u - s_t)."""
    q, k, v, pt, L, S = c["q"], c["k"], c["v"], c["pt"], c["L"], c["S"]
    B, Hq, D = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, D))
    for b in range(B):
        n = int(L[b])
        if n == 0:
            continue
        Kc = [[[f_of(x) for x in k[pt[b, t // S], t % S, g]] for t in range(n)] for g in range(Hkv)]
        Vc = [[[f_of(x) for x in v[pt[b, t // S], t % S, g]] for t in range(n)] for g in range(Hkv)]
        for h in range(Hq):
            g = h // G
            qh = [f_of(x) for x in q[b, h]]
            s = [c["scale"] * math.fsum(a * kk for a, kk in zip(qh, Kc[g][t])) for t in range(n)]
            w = [1.0 / math.fsum(math.exp(su - st) for su in s) for st in s]
            for d in range(D):
                out[b, h, d] = math.fsum(w[t] * Vc[g][t][d] for t in range(n))
    return out


def pin_brute_force(orc):
    for lengths, hq, hkv in [([5, 1, 40], 8, 2), ([17, 33], 4, 4), ([64], 8, 1), ([0, 16, 3], 8, 8)]:
        c = case(lengths, hq=hq, hkv=hkv, seed=len(lengths) + hq)
        got = run(orc, c)
        ref = brute_force(c)
        err = np.abs(got - ref).max()
        assert err <= 1e-12, ("brute force", lengths, hq, hkv, err)


# ---------------------------------------------------------------- L = 1
def pin_single_token(orc):
    """One cached token: its weight is exp(0) / exp(0) = 1, so out is its V row."""
    c = case([1, 1, 1], hq=8, hkv=2, seed=3)
    got = run(orc, c)
    for b in range(3):
        for h in range(8):
            vrow = np.array([f_of(x) for x in c["v"][c["pt"][b, 0], 0, h // 4]])
            assert np.array_equal(got[b, h], vrow), ("L=1", b, h)


# ---------------------------------------------------------------- constant V
def pin_constant_v(orc):
    """Every V row of a KV head equal to c_g: out is c_g whatever the scores."""
    c = case([1, 15, 16, 17, 100], hq=8, hkv=2, seed=4)
    rng = np.random.default_rng(1)
    const = (rng.standard_normal((2, 128)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    for b, n in enumerate(c["L"]):
        for t in range(int(n)):
            c["v"][c["pt"][b, t // 16], t % 16] = const
    got = run(orc, c)
    for h in range(8):
        expect = np.array([f_of(x) for x in const[h // 4]])
        assert np.abs(got[:, h] - expect).max() <= 1e-12, ("constant V", h)


# ---------------------------------------------------------------- shift invariance
def pin_shift_invariance(orc):
    """softmax(s + c) = softmax(s): k_t[d0] = 1 for every t shifts all scores
    of head h by scale * q[h][d0]; outputs with q[h][d0] in {0, 8, 256^2...}
    must agree.  The large shift (q = k = 256 on d0, scores ~ 5.8e3) also
    demands the max subtraction."""
    for d0val, kval in [(8.0, 1.0), (256.0, 256.0)]:
        c = case([40, 3, 77], hq=8, hkv=2, seed=5)
        for b, n in enumerate(c["L"]):
            for t in range(int(n)):
                c["k"][c["pt"][b, t // 16], t % 16, :, 7] = bf16_bits(kval)
        c0 = {**c, "q": c["q"].copy()}
        c1 = {**c, "q": c["q"].copy()}
        c0["q"][:, :, 7] = bf16_bits(0.0)
        c1["q"][:, :, 7] = bf16_bits(d0val)
        a, b_ = run(orc, c0), run(orc, c1)
        assert np.isfinite(b_).all(), "shift: non-finite output"
        assert np.abs(a - b_).max() <= 1e-12, ("shift", d0val, np.abs(a - b_).max())
    s = np.random.default_rng(2).standard_normal(50) * 4
    w0, w1 = orc.softmax(s), orc.softmax(s + 1234.5)
    assert np.abs(w0 - w1).max() <= 1e-13 and abs(w0.sum() - 1) <= 1e-13


# ---------------------------------------------------------------- page permutation
def pin_page_permutation(orc):
    """Moving physical pages and rewriting the page table to match leaves the
    output bit-identical; widening the page-table rows changes nothing."""
    c = case([37, 128, 500, 5], hq=8, hkv=2, seed=6, shuffle=False)
    base = run(orc, c)
    perm = np.random.default_rng(3).permutation(c["k"].shape[0]).astype(np.int32)
    k2 = np.empty_like(c["k"])
    v2 = np.empty_like(c["v"])
    k2[perm] = c["k"]
    v2[perm] = c["v"]
    c2 = {**c, "k": k2, "v": v2, "pt": perm[c["pt"]]}
    assert np.array_equal(run(orc, c2), base), "page permutation"
    wide = np.full((4, c["pt"].shape[1] + 9), c["pt"].max(), dtype=np.int32)
    wide[:, :c["pt"].shape[1]] = c["pt"]
    c3 = {**c, "pt": wide}
    assert np.array_equal(run(orc, c3), base), "page-table stride"


# ---------------------------------------------------------------- closed forms
def pin_closed_forms(orc):
    """q = 0: all weights equal, out = mean of V rows.  L = 2: out =
    sigmoid(s1 - s2) v1 + sigmoid(s2 - s1) v2."""
    c = case([1, 7, 33, 250], hq=4, hkv=2, seed=7)
    c["q"][:] = 0
    got = run(orc, c)
    for b, n in enumerate(c["L"]):
        for g in range(2):
            rows = np.array([[f_of(x) for x in c["v"][c["pt"][b, t // 16], t % 16, g]]
                             for t in range(int(n))])
            mean = np.array([math.fsum(rows[:, d]) / n for d in range(128)])
            for h in (2 * g, 2 * g + 1):
                assert np.abs(got[b, h] - mean).max() <= 1e-12, ("q=0 mean", b, h)

    c = case([2, 2], hq=4, hkv=1, seed=8)
    got = run(orc, c)
    for b in range(2):
        pg = c["pt"][b, 0]
        k1 = [f_of(x) for x in c["k"][pg, 0, 0]]
        k2 = [f_of(x) for x in c["k"][pg, 1, 0]]
        v1 = np.array([f_of(x) for x in c["v"][pg, 0, 0]])
        v2 = np.array([f_of(x) for x in c["v"][pg, 1, 0]])
        for h in range(4):
            qh = [f_of(x) for x in c["q"][b, h]]
            s1 = c["scale"] * math.fsum(a * x for a, x in zip(qh, k1))
            s2 = c["scale"] * math.fsum(a * x for a, x in zip(qh, k2))
            sig = 1.0 / (1.0 + math.exp(s2 - s1))
            expect = sig * v1 + (1.0 - sig) * v2
            assert np.abs(got[b, h] - expect).max() <= 1e-12, ("L=2 sigmoid", b, h)


# ---------------------------------------------------------------- GQA vs MHA
def pin_gqa_equals_duplicated_mha(orc):
    """Query head h reads KV head floor(h / G): copying each KV head G times
    (Hkv' = Hq) and running plain multi-head attention gives the same bits."""
    for hq, hkv in [(8, 2), (8, 1), (16, 2)]:
        c = case([19, 64, 3], hq=hq, hkv=hkv, seed=9 + hq + hkv)
        G = hq // hkv
        c2 = {**c, "k": np.repeat(c["k"], G, axis=2).copy(), "v": np.repeat(c["v"], G, axis=2).copy()}
        assert np.array_equal(run(orc, c), run(orc, c2)), ("GQA vs MHA", hq, hkv)


# ---------------------------------------------------------------- one-hot
def onehot_case(lengths, hq, hkv, seed, hot):
    """q = 64 e0; k_t[0] = 0 except k_{t*}[0] = 32 at logical token hot[b]:
    s_{t*} = scale * 2048 ~ 181, every other score exactly 0."""
    c = case(lengths, hq=hq, hkv=hkv, seed=seed)
    c["q"][:] = 0
    c["q"][:, :, 0] = bf16_bits(64.0)
    for b, n in enumerate(c["L"]):
        for t in range(int(n)):
            c["k"][c["pt"][b, t // 16], t % 16, :, 0] = bf16_bits(32.0 if t == hot[b] else 0.0)
    return c


def pin_one_hot(orc):
    """exp(-181) ~ 3e-79: the output is the hot token's V row to within
    round-off of that weight."""
    lengths, hot = [1, 40, 300, 17], [0, 39, 150, 16]
    c = onehot_case(lengths, 8, 2, 11, hot)
    got = run(orc, c)
    for b in range(4):
        t = hot[b]
        for h in range(8):
            vrow = np.array([f_of(x) for x in c["v"][c["pt"][b, t // 16], t % 16, h // 4]])
            assert np.allclose(got[b, h], vrow, rtol=1e-15, atol=1e-70), ("one-hot", b, h)


# ---------------------------------------------------------------- library SDPA
def pin_torch_sdpa(orc):
    """float64 scaled_dot_product_attention of a library on the contiguous
    gather, K/V repeated per group, agrees to 1e-10."""
    c = case([37, 128, 200, 1], hq=8, hkv=2, seed=12)
    got = run(orc, c)
    q = torch.from_numpy(c["q"].astype(np.uint32) << 16).view(torch.float32).double()
    for b, n in enumerate(c["L"]):
        n = int(n)
        idx = [(c["pt"][b, t // 16], t % 16) for t in range(n)]
        kk = np.stack([c["k"][p, s] for p, s in idx]).astype(np.uint32) << 16
        vv = np.stack([c["v"][p, s] for p, s in idx]).astype(np.uint32) << 16
        kt = torch.from_numpy(kk).view(torch.float32).double().permute(1, 0, 2)  # [Hkv][n][D]
        vt = torch.from_numpy(vv).view(torch.float32).double().permute(1, 0, 2)
        kt = kt.repeat_interleave(4, dim=0).contiguous()
        vt = vt.repeat_interleave(4, dim=0).contiguous()
        ref = torch.nn.functional.scaled_dot_product_attention(
            q[b][:, None, :], kt, vt, scale=c["scale"])[:, 0, :].numpy()
        assert np.abs(ref - got[b]).max() <= 1e-10, ("torch sdpa", b)


# ---------------------------------------------------------------- edges
def pin_edges(orc):
    """Empty request -> zeros; NaN-filled unused slots and spare page never
    reach the output; page-boundary lengths match brute force."""
    c = case([0, 3, 0], hq=4, hkv=2, seed=13)
    got = run(orc, c)
    assert np.array_equal(got[0], np.zeros_like(got[0])) and np.array_equal(got[2], np.zeros_like(got[2]))
    assert np.isfinite(got).all()
    c = case([1, 15, 16, 17, 31, 32, 33], hq=2, hkv=1, seed=14)
    got = run(orc, c)
    assert np.isfinite(got).all()
    assert np.abs(got - brute_force(c)).max() <= 1e-12, "page-boundary lengths"


def pin_gather(orc):
    """The oracle's gather equals a direct indexing of the page pools."""
    c = case([37, 1, 16, 50], hq=4, hkv=2, seed=15)
    ko, vo = orc.gather(c["k"], c["v"], c["pt"], c["L"])
    rows = [(c["pt"][b, t // 16], t % 16) for b, n in enumerate(c["L"]) for t in range(int(n))]
    assert np.array_equal(ko, np.stack([c["k"][p, s] for p, s in rows]))
    assert np.array_equal(vo, np.stack([c["v"][p, s] for p, s in rows]))


# ---------------------------------------------------------------- KV append
def pin_kv_append(orc):
    """After appending token pos of request b, the request's row pos is the
    new row (direct indexing of the pools) and no other byte changed;
    negative and out-of-table positions write nothing."""
    c = case([16, 1, 33, 0, 5], hq=4, hkv=2, seed=16, pt_stride=4)
    rng = np.random.default_rng(5)
    k_new = rng.integers(0, 1 << 16, (5, 2, 128), dtype=np.uint16)
    v_new = rng.integers(0, 1 << 16, (5, 2, 128), dtype=np.uint16)
    # request 1: position 64 is past its 4-entry table row (a missing bound
    # would read row 2's first entry, still inside the table); request 3: -1
    pos = np.array([15, 64, 33, -1, 4], dtype=np.int32)
    k, v = c["k"].copy(), c["v"].copy()
    orc.kv_append(k_new, v_new, k, v, c["pt"], pos)
    ek, ev = c["k"].copy(), c["v"].copy()
    for b, p in enumerate(pos):
        if 0 <= p < c["pt"].shape[1] * 16:
            ek[c["pt"][b, p // 16], p % 16] = k_new[b]
            ev[c["pt"][b, p // 16], p % 16] = v_new[b]
    assert np.array_equal(k, ek) and np.array_equal(v, ev), "kv append"
    L = np.array([16, 1, 34, 0, 5], dtype=np.int32)
    ko, vo = orc.gather(k, v, c["pt"], L)
    assert np.array_equal(ko[15], k_new[0]) and np.array_equal(vo[15], v_new[0])
    assert np.array_equal(ko[16 + 1 + 33], k_new[2]) and np.array_equal(vo[16 + 1 + 34 + 4], v_new[4])


# ---------------------------------------------------------------- GEMM
def pin_gemm(orc):
    """Brute force with exactly rounded sums; an identity weight returns x;
    float64 matmul of a library agrees."""
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((3, 40)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    w = (rng.standard_normal((5, 40)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y = orc.gemm(x, w)
    for m in range(3):
        for n in range(5):
            ref = math.fsum(f_of(a) * f_of(b) for a, b in zip(x[m], w[n]))
            assert abs(y[m, n] - ref) <= 1e-12, ("gemm brute force", m, n)
    eye = np.zeros((40, 40), dtype=np.uint16)
    eye[np.arange(40), np.arange(40)] = bf16_bits(1.0)
    xf = np.array([[f_of(a) for a in row] for row in x])
    assert np.array_equal(orc.gemm(x, eye), xf), "gemm identity"
    xl = (rng.standard_normal((7, 300)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    wl = (rng.standard_normal((33, 300)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    tx = torch.from_numpy(xl.astype(np.uint32) << 16).view(torch.float32).double()
    tw = torch.from_numpy(wl.astype(np.uint32) << 16).view(torch.float32).double()
    assert np.abs(orc.gemm(xl, wl) - (tx @ tw.T).numpy()).max() <= 1e-10, "gemm vs library"


ALL_PINS = [pin_brute_force, pin_single_token, pin_constant_v, pin_shift_invariance,
            pin_page_permutation, pin_closed_forms, pin_gqa_equals_duplicated_mha,
            pin_one_hot, pin_torch_sdpa, pin_edges, pin_gather, pin_kv_append, pin_gemm]
