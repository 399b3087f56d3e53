"""Seeded synthetic decode-attention workloads (inputs only, no attention math).

This module is shared by the tests, the benchmark and the smoke check, on both
sides of a parity comparison.  It draws request lengths, the physical page
placement and the Q/K/V values; it computes nothing of the attention itself.

Shapes follow the decode step the paper profiles: N_req running requests, each
holding N_kv cached tokens in a paged KV cache (Sec. 5.4, Eq. pred-itl; paging
as in PagedAttention, Sec. 2.1).  The paper's length distributions come from
ShareGPT/LMSYS chat traces, which are not used here; the lognormal and
log-uniform length laws below stand in for them.

Recipe (every workload, seed s):
  * streams: numpy SeedSequence(s).spawn(5) -> lengths, placement, Q, K, V;
    large value streams are cut into 4 Mi-element chunks, chunk i drawn from
    torch.Generator seeded by that stream's i-th spawned child, so generation
    runs in parallel and is identical on any machine;
  * lengths: per workload law (below), int32;
  * placement: P_b = ceil(L_b / S) logical pages per request; a random
    permutation of [0, sum P_b) is dealt to the requests in order (identity if
    shuffle=False); physical page sum P_b is a spare page; unused page-table
    entries point at the spare page;
  * values: fp32 N(0, 1), rounded to bf16 with round-to-nearest-even;
    Q [B][Hq][D], K and V pools [num_pages][S][Hkv][D];
  * fill: slots past L_b in a request's last page and the spare page are set
    to bf16 NaN ("nan", parity runs) or 0 ("zero", timing runs), so a kernel
    that reads outside the valid tokens cannot go unnoticed.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np
import torch

BF16_NAN_BITS = 0x7FC0
_CHUNK = 1 << 22


@dataclass(frozen=True)
class Workload:
    name: str
    num_seqs: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    page_size: int
    law: str                      # "fixed" | "uniform" | "lognormal" | "loguniform"
    params: tuple = field(default=())
    shuffle: bool = True
    description: str = ""


WORKLOADS = {
    "tiny_b4": Workload(
        "tiny_b4", 4, 32, 8, 128, 16, "fixed", (37, 128, 500, 1000),
        description="4 requests, 32:8 heads, lengths {37,128,500,1000}"),
    "llama8b_b64": Workload(
        "llama8b_b64", 64, 32, 8, 128, 16, "uniform", (512, 4096),
        description="Llama-3-8B-shaped step: 64 requests, 32:8 heads, L ~ U[512,4096]"),
    "chat_b256": Workload(
        "chat_b256", 256, 32, 8, 128, 16, "lognormal", (1200.0, 0.8, 16, 16384),
        description="chat-like batch: 256 requests, 32:8 heads, "
                    "L ~ lognormal(median 1200, sigma 0.8) clipped to [16,16384]"),
    "gqa8_b128": Workload(
        "gqa8_b128", 128, 64, 8, 128, 16, "uniform", (2048, 8192),
        description="70B-shaped step on one GPU: 128 requests, 64:8 heads, L ~ U[2048,8192]"),
    "long_b16": Workload(
        "long_b16", 16, 32, 8, 128, 16, "loguniform", (1, 131072, 131072),
        description="long ragged: 16 requests, 32:8 heads, L_0 = 131072, "
                    "others log-uniform in [1,131072]"),
    # one GPU's share of gqa8_b128 under tensor parallelism over KV heads:
    # the same requests and lengths, Hkv / TP KV heads and their query heads
    "gqa8_b128_tp2": Workload(
        "gqa8_b128_tp2", 128, 32, 4, 128, 16, "uniform", (2048, 8192),
        description="gqa8_b128 at TP = 2 (one GPU's share): 128 requests, 32:4 heads, L ~ U[2048,8192]"),
    "gqa8_b128_tp8": Workload(
        "gqa8_b128_tp8", 128, 8, 1, 128, 16, "uniform", (2048, 8192),
        description="gqa8_b128 at TP = 8 (one GPU's share): 128 requests, 8:1 heads, L ~ U[2048,8192]"),
}
ORDER = ["tiny_b4", "llama8b_b64", "chat_b256", "gqa8_b128", "long_b16"]
SHARDS = ["gqa8_b128_tp2", "gqa8_b128_tp8"]


def _seed_of(ss: np.random.SeedSequence) -> int:
    return int(ss.generate_state(1, np.uint64)[0] & 0x7FFFFFFFFFFFFFFF)


def _gen(ss: np.random.SeedSequence) -> torch.Generator:
    return torch.Generator().manual_seed(_seed_of(ss))


def draw_lengths(w: Workload, ss: np.random.SeedSequence) -> np.ndarray:
    g = _gen(ss)
    B = w.num_seqs
    if w.law == "fixed":
        L = np.asarray(w.params, dtype=np.int64)
        assert L.shape == (B,)
    elif w.law == "uniform":
        lo, hi = w.params
        L = torch.randint(lo, hi + 1, (B,), generator=g).numpy().astype(np.int64)
    elif w.law == "lognormal":
        median, sigma, lo, hi = w.params
        z = torch.randn(B, generator=g, dtype=torch.float64).numpy()
        L = np.clip(np.round(np.exp(math.log(median) + sigma * z)), lo, hi).astype(np.int64)
    elif w.law == "loguniform":
        lo, hi, first = w.params
        u = torch.rand(B - 1, generator=g, dtype=torch.float64).numpy()
        rest = np.clip(np.round(np.exp(u * math.log(hi))), lo, hi).astype(np.int64)
        L = np.concatenate([[first], rest]).astype(np.int64)
    else:
        raise ValueError(w.law)
    return L.astype(np.int32)


def _randn_bf16(shape, ss: np.random.SeedSequence, threads: int) -> torch.Tensor:
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch.bfloat16)
    nch = max(1, (n + _CHUNK - 1) // _CHUNK)
    kids = ss.spawn(nch)

    def work(i):
        lo = i * _CHUNK
        hi = min(n, lo + _CHUNK)
        if hi > lo:
            out[lo:hi] = torch.randn(hi - lo, generator=_gen(kids[i])).to(torch.bfloat16)

    if nch == 1 or threads <= 1:
        for i in range(nch):
            work(i)
    else:
        prev = torch.get_num_threads()
        torch.set_num_threads(1)
        try:
            with ThreadPoolExecutor(threads) as ex:
                list(ex.map(work, range(nch)))
        finally:
            torch.set_num_threads(prev)
    return out.view(*shape)


def make_case(w, seed: int = 0, fill: str = "nan", lengths=None, shuffle=None,
              pt_stride: int | None = None, threads: int = 16) -> dict:
    """Draw one workload.  Returns CPU tensors and metadata.

    lengths overrides the workload's length law (the other streams are drawn
    as usual); shuffle overrides the page placement; pt_stride (>= max P_b)
    widens the page-table rows.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    root = np.random.SeedSequence(seed)
    ss_len, ss_perm, ss_q, ss_k, ss_v = root.spawn(5)
    B, Hq, Hkv, D, S = w.num_seqs, w.n_q_heads, w.n_kv_heads, w.head_dim, w.page_size

    if lengths is None:
        L = draw_lengths(w, ss_len)
    else:
        L = np.asarray(lengths, dtype=np.int32)
        B = L.shape[0]
    P = (L.astype(np.int64) + S - 1) // S
    total = int(P.sum())
    spare = total
    num_pages = total + 1
    do_shuffle = w.shuffle if shuffle is None else shuffle
    if do_shuffle:
        perm = torch.randperm(total, generator=_gen(ss_perm)).numpy().astype(np.int32)
    else:
        perm = np.arange(total, dtype=np.int32)
    maxp = max(1, int(P.max()) if B > 0 else 1)
    stride = maxp if pt_stride is None else int(pt_stride)
    assert stride >= maxp
    page_table = np.full((B, stride), spare, dtype=np.int32)
    off = 0
    for b in range(B):
        page_table[b, :P[b]] = perm[off:off + P[b]]
        off += int(P[b])

    q = _randn_bf16((B, Hq, D), ss_q, threads)
    k = _randn_bf16((num_pages, S, Hkv, D), ss_k, threads)
    v = _randn_bf16((num_pages, S, Hkv, D), ss_v, threads)

    fill_bits = {"nan": BF16_NAN_BITS, "zero": 0}[fill]
    if fill_bits is not None:
        kb = k.view(torch.int16)
        vb = v.view(torch.int16)
        fv = np.int16(np.uint16(fill_bits).view(np.int16))
        kb[spare] = int(fv)
        vb[spare] = int(fv)
        for b in range(B):
            used = int(L[b]) - S * (int(P[b]) - 1) if P[b] > 0 else S
            if P[b] > 0 and used < S:
                p = int(page_table[b, P[b] - 1])
                kb[p, used:] = int(fv)
                vb[p, used:] = int(fv)

    return dict(
        workload=w, seed=seed, q=q, k_pages=k, v_pages=v,
        page_table=torch.from_numpy(page_table), seq_lens=torch.from_numpy(L.copy()),
        scale=float(np.float32(1.0 / math.sqrt(D))),
        num_seqs=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, page_size=S,
        max_pages_per_seq=stride, num_pages=num_pages, n_kv=int(L.astype(np.int64).sum()),
    )


def bits(t: torch.Tensor) -> np.ndarray:
    """Raw uint16 bit patterns of a bf16 CPU tensor (zero-copy view)."""
    assert t.dtype == torch.bfloat16 and t.device.type == "cpu"
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def kv_bytes(case: dict) -> int:
    """Bytes of K and V a decode step must read: N_kv * Hkv * D * 2 (K,V) * 2 B."""
    return case["n_kv"] * case["n_kv_heads"] * case["head_dim"] * 2 * 2


def make_device_case(num_seqs: int, seq_len: int, n_q_heads: int, n_kv_heads: int, seed: int,
                     device="cuda") -> dict:
    """A large seeded case drawn directly in device memory (for sizes whose
    host copy would be tens of GB): every request holds seq_len tokens,
    pages are a random permutation of the pool, Q/K/V are N(0, 1) rounded to
    bf16 (torch's generator on `device`, seeded).  Tests check it on sampled
    rows, copying only the pages those rows read to the host."""
    gen = torch.Generator(device=device).manual_seed(seed)
    S, D = 16, 128
    P = (seq_len + S - 1) // S
    n_pages = num_seqs * P
    perm = torch.randperm(n_pages, generator=gen, device=device).to(torch.int32)
    pools = []
    for _ in range(2):
        pool = torch.empty((n_pages, S, n_kv_heads, D), dtype=torch.bfloat16, device=device)
        for i in range(0, n_pages, 4096):   # no full-size fp32 temporary
            j = min(n_pages, i + 4096)
            pool[i:j].copy_(torch.randn((j - i, S, n_kv_heads, D), generator=gen, device=device))
        pools.append(pool)
    q = torch.randn((num_seqs, n_q_heads, D), generator=gen, device=device).to(torch.bfloat16)
    return {"q": q, "k_pages": pools[0], "v_pages": pools[1], "page_table": perm.view(num_seqs, P),
            "seq_lens": torch.full((num_seqs,), seq_len, dtype=torch.int32, device=device),
            "num_seqs": num_seqs, "n_q_heads": n_q_heads, "n_kv_heads": n_kv_heads,
            "max_pages_per_seq": P, "scale": float(np.float32(1.0 / np.sqrt(D)))}
