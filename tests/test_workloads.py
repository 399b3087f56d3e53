"""The seeded input generator (CPU): same seed, same bytes on any thread count;
the placement, page-table and fill rules of the recipe hold."""
import numpy as np
import torch

from workloads import BF16_NAN_BITS, ORDER, SHARDS, WORKLOADS, bits, kv_bytes, make_case


def _same(a, b):
    """Byte equality (bf16 tensors hold NaN fill, so compare bit patterns)."""
    def raw(t):
        return t.view(torch.int16) if t.dtype == torch.bfloat16 else t
    return all(torch.equal(raw(a[k]), raw(b[k])) if isinstance(a[k], torch.Tensor) else a[k] == b[k]
               for k in ("q", "k_pages", "v_pages", "page_table", "seq_lens", "scale", "n_kv"))


def test_same_seed_same_bytes_any_thread_count():
    a = make_case("tiny_b4", seed=3, threads=1)
    b = make_case("tiny_b4", seed=3, threads=8)
    assert _same(a, b)
    c = make_case("tiny_b4", seed=4)
    assert not torch.equal(a["q"].view(torch.int16), c["q"].view(torch.int16))
    assert not torch.equal(a["k_pages"].view(torch.int16), c["k_pages"].view(torch.int16))
    # a pool larger than one generator chunk (4 Mi elements): chunks are
    # seeded independently, so the split over threads cannot change bytes
    lens = [3000] * 12
    d = make_case("tiny_b4", seed=5, lengths=lens, threads=1)
    e = make_case("tiny_b4", seed=5, lengths=lens, threads=6)
    assert d["k_pages"].numel() > (1 << 22)
    assert _same(d, e)


def test_lengths_follow_the_workload_laws():
    assert make_case("tiny_b4")["seq_lens"].tolist() == [37, 128, 500, 1000]
    for name in ("llama8b_b64", "gqa8_b128"):
        w = WORKLOADS[name]
        from workloads import draw_lengths
        L = draw_lengths(w, np.random.SeedSequence(0).spawn(5)[0])
        lo, hi = w.params
        assert L.shape == (w.num_seqs,) and L.min() >= lo and L.max() <= hi
    from workloads import draw_lengths
    L = draw_lengths(WORKLOADS["long_b16"], np.random.SeedSequence(0).spawn(5)[0])
    assert L[0] == 131072 and L.min() >= 1 and L.max() <= 131072
    L = draw_lengths(WORKLOADS["chat_b256"], np.random.SeedSequence(0).spawn(5)[0])
    assert L.min() >= 16 and L.max() <= 16384 and 800 < np.median(L) < 1600


def test_placement_page_table_and_fill():
    c = make_case("tiny_b4", seed=0, lengths=[37, 16, 1, 0, 33], fill="nan")
    L = c["seq_lens"].numpy()
    P = (L + 15) // 16
    pt = c["page_table"].numpy()
    spare = c["num_pages"] - 1
    used = np.concatenate([pt[b, :P[b]] for b in range(len(L))])
    # a permutation of [0, sum P) dealt in order, plus one spare page
    assert sorted(used.tolist()) == list(range(int(P.sum())))
    for b in range(len(L)):
        assert (pt[b, P[b]:] == spare).all()
    kb, vb = bits(c["k_pages"]), bits(c["v_pages"])
    assert (kb[spare] == BF16_NAN_BITS).all() and (vb[spare] == BF16_NAN_BITS).all()
    for b in range(len(L)):
        if P[b] == 0:
            continue
        last, valid = pt[b, P[b] - 1], L[b] - 16 * (P[b] - 1)
        assert (kb[last, valid:] == BF16_NAN_BITS).all() and (vb[last, valid:] == BF16_NAN_BITS).all()
        assert not (kb[last, :valid] == BF16_NAN_BITS).any()
    z = make_case("tiny_b4", seed=0, lengths=[37, 16, 1, 0, 33], fill="zero")
    assert (bits(z["k_pages"])[spare] == 0).all()
    assert torch.equal(z["q"], c["q"])


def test_identity_placement_and_sizes():
    c = make_case("tiny_b4", seed=0, shuffle=False)
    pt = c["page_table"].numpy()
    P = (c["seq_lens"].numpy() + 15) // 16
    flat = np.concatenate([pt[b, :P[b]] for b in range(4)])
    assert flat.tolist() == list(range(int(P.sum())))
    assert kv_bytes(c) == 1665 * 8 * 128 * 2 * 2
    assert c["scale"] == float(np.float32(1 / np.sqrt(128)))
    assert set(ORDER) | set(SHARDS) == set(WORKLOADS) and not set(ORDER) & set(SHARDS)


def test_tensor_parallel_shards_keep_the_requests():
    """A shard is one GPU's share of gqa8_b128 with KV heads split over GPUs:
    the same request lengths and page placement, Hkv / TP KV heads and the
    query heads that read them (the group size G stays 8)."""
    full = make_case("gqa8_b128", seed=0, fill="zero")
    for name, tp in (("gqa8_b128_tp2", 2), ("gqa8_b128_tp8", 8)):
        c = make_case(name, seed=0, fill="zero")
        assert torch.equal(c["seq_lens"], full["seq_lens"]) and torch.equal(c["page_table"], full["page_table"])
        assert c["n_kv_heads"] * tp == full["n_kv_heads"] and c["n_q_heads"] * tp == full["n_q_heads"]
        assert kv_bytes(c) * tp == kv_bytes(full)
