"""Decode-attention benchmark on one MI355X.

One step = one whole decode-attention call (self-planned attention kernel +
combine kernel) over the chat-like batch: 256 requests, 32 query / 8 KV heads, head_dim 128,
lengths lognormal (median 1200, sigma 0.8) clipped to [16, 16384], 16-token
pages in shuffled order, bf16 N(0,1) values, seed 0 (synthetic; stands in for
chat-trace length mixes).  Inputs are resident in HBM before timing starts.
Before the warm-up steps, steps run untimed for --settle seconds: an idle
MI355X drops its shader clock to about 100 MHz and takes milliseconds of
work to return to 2.4 GHz.

Prints one JSON line:
  value         KV bytes per step / step time, GB/s (whole job, all N GPUs)
  ms_per_step   wall time per step from events around the K timed steps
  roofline      the attention kernel: algorithmic bytes per launch / its
                average launch time (HIP events on the launch stream) against
                MI355X's 8 TB/s; traffic from the committed FETCH_SIZE /
                WRITE_SIZE counter summary when it matches this kernel source
  cpu_baseline  the fp64 oracle on the host cores over the same workload
  cold_cache    step times with the caches flushed (a 1 GiB read) before
                each step, one step at a time: p10 / median / p90 of the
                step and of its attention launch, outside the back-to-back
                timing
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
WORKLOAD = "chat_b256"


def kernel_source_hash() -> str:
    """Hash of what the attention kernels are built from: their source and the
    header, with comments and whitespace removed, and the compiler flags of
    that source, so that counters taken on one build are reported only for
    the same code."""
    from paper_2509_04827_amd import build as vbuild
    h = hashlib.sha256()
    for rel in ("paper_2509_04827_amd/csrc/vdecode.hip", "include/vdecode.h"):
        with open(os.path.join(ROOT, rel)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("".join(text.split()).encode())
    h.update(" ".join(vbuild.HIPCC_FLAGS + vbuild.SRC_FLAGS["vdecode.hip"]).encode())
    return h.hexdigest()[:16]


def committed_traffic(workload: str):
    """HBM bytes per attention launch from profiles/, if taken on this source."""
    path = os.path.join(ROOT, "profiles", "attn_kernel_%s_traffic.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t.get("hbm_bytes_per_launch")


def settle_clocks(fn, seconds: float) -> int:
    """Run fn (one step) for `seconds` of wall time before anything is timed.
    Between jobs the GPU sits in a deep-sleep clock state (about 100 MHz
    against its 2.4 GHz) and needs milliseconds of steady work to come back,
    so a few tens of warm-up steps end too early.  Returns the steps run."""
    import torch
    n, t0 = 0, time.time()
    while time.time() - t0 < seconds:
        for _ in range(16):
            fn()
        torch.cuda.synchronize()
        n += 16
    return n


SURFACE_BATCH = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512)
SURFACE_LEN = (16, 64, 256, 1024, 4096, 16384)
SURFACE_GQA8_BATCH = (64, 128, 256)


def latency_surface(outdir: str, iters: int = 10, warmup: int = 3):
    """Step time over (N_req, N_kv): the state the paper's decode-latency
    model consumes (Sec. 5.4, Eq. pred-itl).  Grid: batch x tokens per
    request, equal lengths and a lognormal-ragged mix of the same mean
    (sigma 0.8, clipped to [1, 4 x mean]); plus 64:8 heads at a few batches.
    Values are random bf16 drawn on the GPU (timing only; parity is covered by
    the tests).  Fits T = c*N_req + d*N_kv + e by least squares."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gen = torch.Generator(device=dev).manual_seed(0)
    rng = np.random.default_rng(0)
    Hkv, D, S = 8, 128, 16
    max_tokens = max(SURFACE_BATCH) * max(SURFACE_LEN) * 4 // 3
    max_pages = max_tokens // S + max(SURFACE_BATCH) + 1
    kp = torch.randn((max_pages, S, Hkv, D), generator=gen, device=dev, dtype=torch.float32).to(torch.bfloat16)
    vp = torch.randn((max_pages, S, Hkv, D), generator=gen, device=dev, dtype=torch.float32).to(torch.bfloat16)
    stream = torch.cuda.current_stream()
    rows = []

    def point(B, lens, Hq, law):
        lens = np.asarray(lens, dtype=np.int64)
        P = (lens + S - 1) // S
        if P.sum() > max_pages:
            return
        maxp = int(max(1, P.max()))
        perm = rng.permutation(max_pages)[:int(P.sum())].astype(np.int32)
        pt = np.zeros((B, maxp), dtype=np.int32)
        off = 0
        for b in range(B):
            pt[b, :P[b]] = perm[off:off + P[b]]
            off += int(P[b])
        q = torch.randn((B, Hq, D), generator=gen, device=dev).to(torch.bfloat16)
        out = torch.empty_like(q)
        ptd = torch.from_numpy(pt).to(dev)
        sl = torch.from_numpy(lens.astype(np.int32)).to(dev)
        ws = vd.alloc_workspace(B, Hq, Hkv, maxp)
        scale = float(np.float32(1.0 / np.sqrt(D)))

        def step():
            vd.vd_decode_attn(q, kp, vp, ptd, sl, out, scale, ws, stream=stream)

        settle_clocks(step, 0.02)
        for _ in range(warmup):
            step()
        st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        st.record(stream)
        for _ in range(iters):
            step()
        en.record(stream)
        torch.cuda.synchronize()
        us_step = st.elapsed_time(en) * 1e3 / iters
        # device time per call: `iters` calls captured into one HIP graph and
        # replayed, so the host launches nothing per call and small steps show
        # the device's own time (kernels and the gaps between them), not the
        # binding's call rate; the first replay is a warm-up
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            vd.vd_decode_attn(q, kp, vp, ptd, sl, out, scale, ws)
        stream.wait_stream(side)
        torch.cuda.synchronize()

        def graph_us(call, reps=3):
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for _ in range(iters):
                    call()
            graph.replay()
            torch.cuda.synchronize()
            st.record(stream)
            for _ in range(reps):
                graph.replay()
            en.record(stream)
            torch.cuda.synchronize()
            del graph
            return st.elapsed_time(en) * 1e3 / (reps * iters)

        us_graph = graph_us(lambda: vd.vd_decode_attn(q, kp, vp, ptd, sl, out, scale, ws))
        # the attention kernel alone (the launches vd_decode_attn makes first)
        us_attn = graph_us(lambda: vd.vd_decode_partial(q, kp, vp, ptd, sl, out, scale, ws,
                                                        flags=vd.VD_FLAG_SELF_PLAN))
        n_kv = int(lens.sum())
        kvb = n_kv * Hkv * D * 2 * 2
        rows.append(dict(law=law, n_q_heads=Hq, n_req=B, tokens_per_req=int(round(lens.mean())),
                         n_kv=n_kv, us_step=round(us_step, 2), us_attn=round(us_attn, 2),
                         us_step_graph=round(us_graph, 2),
                         kv_gbs_step=round(kvb / us_step / 1e3, 1),
                         kv_gbs_graph=round(kvb / us_graph / 1e3, 1)))
        print("surface %-8s Hq %2d B %4d L %6d N_kv %8d  step %9.2f us  graph %9.2f us  attn %9.2f us  %7.1f GB/s"
              % (law, Hq, B, lens.mean(), n_kv, us_step, us_graph, us_attn, kvb / us_step / 1e3),
              file=sys.stderr, flush=True)

    for B in SURFACE_BATCH:
        for L in SURFACE_LEN:
            point(B, [L] * B, 32, "equal")
            z = rng.standard_normal(B)
            lens = np.clip(np.round(L * np.exp(0.8 * z - 0.32)), 1, 4 * L)
            point(B, lens, 32, "ragged")
    for B in SURFACE_GQA8_BATCH:
        for L in SURFACE_LEN:
            point(B, [L] * B, 64, "equal")

    os.makedirs(outdir, exist_ok=True)
    keys = list(rows[0].keys())
    with open(os.path.join(outdir, "decode_latency_surface.csv"), "w") as f:
        f.write(",".join(keys) + "\n")
        for r in rows:
            f.write(",".join(str(r[k]) for k in keys) + "\n")
    # Eq. pred-itl: T = c*N_req + d*N_kv + e, fitted on the 32:8 points, for
    # eager steps and for graph replays
    sel = [r for r in rows if r["n_q_heads"] == 32]
    A = np.array([[r["n_req"], r["n_kv"], 1.0] for r in sel], dtype=np.float64)

    def fit_of(key):
        y = np.array([r[key] for r in sel])
        coef, *_ = np.linalg.lstsq(A, y, rcond=None)
        pred = A @ coef
        r2 = 1.0 - ((y - pred) ** 2).sum() / ((y - y.mean()) ** 2).sum()
        mae = float(np.abs(y - pred).mean())
        bw = Hkv * D * 2 * 2 / (coef[1] * 1e-6) / 1e9
        return dict(c_us_per_req=coef[0], d_us_per_kv_token=coef[1], e_us=coef[2], r2=r2,
                    mae_us=mae, implied_kv_gbs=bw, points=len(sel))

    fit = fit_of("us_step")
    fit_graph = fit_of("us_step_graph")
    with open(os.path.join(outdir, "decode_latency_surface_fit.json"), "w") as f:
        json.dump({"eager": fit, "graph": fit_graph}, f, indent=1)
    print(json.dumps({"surface_points": len(rows), "fit": fit, "fit_graph": fit_graph}), flush=True)


def cpu_configs(outdir: str, iters: int = 10):
    """The oracle on the host cores against the GPU, for every seeded
    workload: one wall-clock oracle run with all threads (and one with a
    single thread for the tiny batch), beside the GPU's device time per step
    (10 steps captured into one HIP graph, replayed 3 times after a
    warm-up replay).  Writes oracle_cpu_baseline.{csv,json}."""
    import numpy as np
    import torch

    import oracle
    import paper_2509_04827_amd as vd
    from workloads import WORKLOADS, bits, kv_bytes, make_case

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    rows = []
    for name in ("tiny_b4", "llama8b_b64", "chat_b256", "gqa8_b128", "long_b16"):
        c = make_case(WORKLOADS[name], seed=0, fill="zero")
        q, k, v = c["q"].to(dev), c["k_pages"].to(dev), c["v_pages"].to(dev)
        pt, sl = c["page_table"].to(dev), c["seq_lens"].to(dev)
        out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
        B, Hq, Hkv, maxp = c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"]
        ws = vd.alloc_workspace(B, Hq, Hkv, maxp)

        def step():
            vd.vd_decode_attn(q, k, v, pt, sl, out, c["scale"], ws)

        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(iters):
                step()
        settle_clocks(graph.replay, 0.05)
        graph.replay()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(3):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        us_gpu = e0.elapsed_time(e1) * 1e3 / (3 * iters)
        del graph

        hq, hk, hv = bits(c["q"]), bits(c["k_pages"]), bits(c["v_pages"])
        hpt, hsl = c["page_table"].numpy(), c["seq_lens"].numpy()
        runs = [("all", 0)] + ([("single", 1)] if name == "tiny_b4" else [])
        kvb = kv_bytes(c)
        for tag, nthreads in runs:
            t1 = time.time()
            oracle.decode_attn(hq, hk, hv, hpt, hsl, c["scale"], nthreads=nthreads)
            sec = time.time() - t1
            rows.append(dict(workload=name, n_req=B, n_kv=c["n_kv"], kv_bytes=kvb,
                             cpu_threads=oracle.max_threads() if nthreads == 0 else nthreads,
                             cpu_s=round(sec, 4), cpu_kv_gbs=round(kvb / sec / 1e9, 3),
                             gpu_us=round(us_gpu, 2), gpu_kv_gbs=round(kvb / us_gpu / 1e3, 1),
                             gpu_over_cpu=round(sec * 1e6 / us_gpu, 1)))
            print("cpu-configs %-12s threads %3d  cpu %8.3f s (%6.2f GB/s)  gpu %9.2f us (%7.1f GB/s)"
                  % (name, rows[-1]["cpu_threads"], sec, kvb / sec / 1e9, us_gpu, kvb / us_gpu / 1e3),
                  file=sys.stderr, flush=True)
        del q, k, v, pt, sl, out, ws
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
    except OSError:
        pass
    os.makedirs(outdir, exist_ok=True)
    keys = list(rows[0].keys())
    with open(os.path.join(outdir, "oracle_cpu_baseline.csv"), "w") as f:
        f.write(",".join(keys) + "\n")
        for r in rows:
            f.write(",".join(str(r[k]) for k in keys) + "\n")
    info = {"cpu_model": cpu_model, "nproc": os.cpu_count(), "oracle_threads": oracle.max_threads(),
            "rows": rows}
    with open(os.path.join(outdir, "oracle_cpu_baseline.json"), "w") as f:
        json.dump(info, f, indent=1)
    print(json.dumps({"cpu_configs": len(rows), "cpu_model": cpu_model, "nproc": os.cpu_count()}),
          flush=True)


GEMM_SHAPES = (("qkv", 6144, 4096), ("o_proj", 4096, 4096), ("gate_up", 28672, 4096),
               ("down", 4096, 14336))
GEMM_M = (1, 2, 4, 8, 16, 24, 32, 48, 64, 96, 128, 160, 192, 224, 240, 248, 255, 256, 257, 264,
          272, 288, 320, 384, 448, 512, 513, 640, 768, 1024)
NEXT_PROFILE_M = (1, 16, 64, 256, 257, 1024)


def clock_sweep(outdir: str, bursts: int = 10, steps: int = 60, idle_s: float = 1.5):
    """Attention-kernel time against the shader clock it ran at: the
    frequency-latency relation T ~ f^-beta of Sec. 3.2 (Eq. t-alpha-beta)
    for decode attention on MI355X.  Clocks cannot be set from user space.
    Instead each burst of whole chat_b256 steps starts after the GPU has
    idled, and the power manager moves the shader clock over the burst's
    first tens of steps (between about 1.4 and 2.4 GHz; the memory clock
    stays fixed).  Each step's record (vd_step_info: the shader clock over
    the attention kernel's first workgroup) is copied aside on the stream,
    and events bracket each attention launch.  A burst's first step is left
    out.  Fits ln T = a - beta ln f by least squares, for the event time and
    for the first workgroup's time."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd
    from workloads import make_case

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    c = make_case(WORKLOAD, seed=0, fill="zero")
    q, k, v = c["q"].to(dev), c["k_pages"].to(dev), c["v_pages"].to(dev)
    pt, sl = c["page_table"].to(dev), c["seq_lens"].to(dev)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
    B, Hq, Hkv, maxp = c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"]
    ws = vd.alloc_workspace(B, Hq, Hkv, maxp)
    stream = torch.cuda.current_stream()
    hist = torch.empty((steps, 48), dtype=torch.uint8, device=dev)
    rows = []
    for burst in range(bursts):
        torch.cuda.synchronize()
        time.sleep(idle_s)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        for i, (e0, e1) in enumerate(ev):
            e0.record(stream)
            vd.vd_decode_partial(q, k, v, pt, sl, out, c["scale"], ws,
                                 flags=vd.VD_FLAG_SELF_PLAN, stream=stream)
            e1.record(stream)
            vd.vd_decode_combine(out, Hkv, maxp, ws, stream=stream)
            hist[i].copy_(ws[:48])
        torch.cuda.synchronize()
        h = hist.cpu()
        for i, (e0, e1) in enumerate(ev):
            if i == 0:   # its events also span the GPU's wake-up from idle (up to ms)
                continue
            r = vd.step_info(h[i])
            rows.append({"burst": burst, "step": i, "us_attn": round(e0.elapsed_time(e1) * 1e3, 2),
                         "us_first_group": round(r["first_group_us"], 2),
                         "sclk_mhz": round(r["sclk_mhz"], 1)})
        print("clock sweep: burst %d, shader clock %.0f-%.0f MHz" % (
            burst, min(x["sclk_mhz"] for x in rows[1 - steps:]), max(x["sclk_mhz"] for x in rows[1 - steps:])),
            file=sys.stderr, flush=True)
    f = np.array([r["sclk_mhz"] for r in rows])

    def fit(col):
        T = np.array([r[col] for r in rows])
        A = np.vstack([np.ones_like(f), np.log(f)]).T
        (a, b), *_ = np.linalg.lstsq(A, np.log(T), rcond=None)
        resid = np.log(T) - A @ np.array([a, b])
        r2 = 1.0 - resid.var() / np.log(T).var()
        return {"beta": round(float(-b), 4), "r2": round(float(r2), 3),
                "us_at_2400": round(float(np.exp(a + b * np.log(2400.0))), 2)}

    bins = []
    edges = [1300, 1500, 1700, 1900, 2100, 2300, 2500]
    for lo, hi in zip(edges, edges[1:]):
        sel = [r for r in rows if lo <= r["sclk_mhz"] < hi]
        if sel:
            bins.append({"sclk_lo": lo, "sclk_hi": hi, "n": len(sel),
                         "sclk_median": round(float(np.median([r["sclk_mhz"] for r in sel])), 1),
                         "us_attn_median": round(float(np.median([r["us_attn"] for r in sel])), 2),
                         "us_first_group_median": round(float(np.median([r["us_first_group"] for r in sel])), 2)})

    def fit_bins(col):
        # per-bin medians, weighted by the points in each bin: robust to the
        # odd event interval that also holds a host-side delay
        fb = np.array([b["sclk_median"] for b in bins])
        Tb = np.array([b[col] for b in bins])
        wb = np.sqrt(np.array([b["n"] for b in bins], dtype=float))
        A = np.vstack([np.ones_like(fb), np.log(fb)]).T * wb[:, None]
        (a, b), *_ = np.linalg.lstsq(A, np.log(Tb) * wb, rcond=None)
        return round(float(-b), 4)

    res = {"points": len(rows), "sclk_mhz_min": round(float(f.min()), 1),
           "sclk_mhz_max": round(float(f.max()), 1),
           "first_group": fit("us_first_group"), "attn_events": fit("us_attn"),
           "beta_first_group_bins": fit_bins("us_first_group_median"),
           "beta_attn_events_bins": fit_bins("us_attn_median"), "bins": bins}
    os.makedirs(outdir, exist_ok=True)
    with open(os.path.join(outdir, "decode_clock_sweep.csv"), "w") as fh:
        fh.write("burst,step,us_attn,us_first_group,sclk_mhz\n")
        for r in rows:
            fh.write("%d,%d,%.2f,%.2f,%.1f\n" % (r["burst"], r["step"], r["us_attn"],
                                                  r["us_first_group"], r["sclk_mhz"]))
    with open(os.path.join(outdir, "decode_clock_sweep.json"), "w") as fh:
        json.dump(res, fh, indent=1)
    print(json.dumps(res), flush=True)


def gemm_sweep(outdir: str, iters: int = 20, warmup: int = 3):
    """Decode-step projection GEMMs of a Llama-3-8B-shaped layer (hidden 4096,
    KV 8 x 128, MLP 14336) over the decode batch M: this library's tiled
    kernel against torch.matmul (hipBLASLt), to locate the batch steps the
    paper traces to tile quantisation (Sec. 3.3).  Primary timing is with
    cold weights: each call reads the next of a ring of weight copies that
    together exceed 1 GiB, so neither L2 nor the 256 MB Infinity Cache holds
    them (in a decode step each layer's weights are read once); warm timing
    (one copy, re-read) beside it."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gen = torch.Generator(device=dev).manual_seed(0)
    stream = torch.cuda.current_stream()
    rows = []

    def timed(fn):
        settle_clocks(lambda: fn(0), 0.02)
        for i in range(warmup):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(iters):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / iters

    for name, N, K in GEMM_SHAPES:
        ring_n = max(2, -(-(1 << 30) // (N * K * 2)))
        ring = [torch.randn((N, K), generator=gen, device=dev).to(torch.bfloat16) for _ in range(ring_n)]
        for M in GEMM_M:
            x = torch.randn((M, K), generator=gen, device=dev).to(torch.bfloat16)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            ws = torch.empty(max(16, vd.vd_gemm_workspace_size(M, N, K)), dtype=torch.uint8, device=dev)
            us_lib = timed(lambda i: torch.matmul(x, ring[i % ring_n].t(), out=y))
            us_own = timed(lambda i: vd.vd_gemm_bf16(x, ring[i % ring_n], y, ws, stream=stream))
            us_lib_warm = timed(lambda i: torch.matmul(x, ring[0].t(), out=y))
            us_own_warm = timed(lambda i: vd.vd_gemm_bf16(x, ring[0], y, ws, stream=stream))
            nbytes = (N * K + M * K + M * N) * 2
            flops = 2.0 * M * N * K
            floor_us = max(nbytes / (PEAK_HBM_GBS * 1e3), flops / 2.5e9)
            rows.append(dict(shape=name, M=M, N=N, K=K, us_hipblaslt=round(us_lib, 2),
                             us_own=round(us_own, 2), roofline_us=round(floor_us, 2),
                             gbs_hipblaslt=round(nbytes / us_lib / 1e3, 1),
                             gbs_own=round(nbytes / us_own / 1e3, 1),
                             tflops_own=round(flops / us_own / 1e6, 1),
                             us_hipblaslt_warm=round(us_lib_warm, 2), us_own_warm=round(us_own_warm, 2),
                             workspace_bytes=vd.vd_gemm_workspace_size(M, N, K)))
            print("gemm %-8s M %5d N %6d K %6d  cold: hipBLASLt %8.2f own %8.2f us  warm: %8.2f %8.2f  roofline %6.2f us"
                  % (name, M, N, K, us_lib, us_own, us_lib_warm, us_own_warm, floor_us),
                  file=sys.stderr, flush=True)
            del x, y, ws
        del ring
        torch.cuda.empty_cache()
    os.makedirs(outdir, exist_ok=True)
    keys = list(rows[0].keys())
    with open(os.path.join(outdir, "decode_gemm_sweep.csv"), "w") as f:
        f.write(",".join(keys) + "\n")
        for r in rows:
            f.write(",".join("" if r[k] is None else str(r[k]) for k in keys) + "\n")
    print(json.dumps({"gemm_points": len(rows)}), flush=True)


LAYER_BATCH = (1, 4, 16, 32, 64, 128, 192, 256, 384, 512)
LAYER_LEN = (16, 64, 256, 1024, 4096)
LAYER_RING = 4
# the dense batch grid: both sides of the projection GEMMs' row-tile steps
# (128 -> 160, 256 -> 257, 512 -> 513) at six lengths, layer time only
LAYER_DENSE_BATCH = (1, 32, 64, 96, 128, 144, 160, 192, 224, 240, 248, 255, 256, 257, 264, 272,
                     288, 320, 384, 448, 480, 496, 504, 511, 512, 513, 520, 528, 544, 576, 640)
LAYER_DENSE_LEN = (64, 128, 256, 512, 1024, 2048)


def layer_surface(outdir: str, reps: int = 5, batches=LAYER_BATCH, lengths=LAYER_LEN,
                  components: bool = True, name: str = "decode_layer_surface"):
    """Time of one decode layer step built from this library's kernels over
    (N_req, tokens per request): the decode iteration the paper's latency
    model predicts (Sec. 5.4, Eq. pred-itl), whose N_req term the projection
    GEMMs carry and whose N_kv term attention carries.  A Llama-3-8B-shaped
    layer (hidden 4096, 32 query / 8 KV heads of 128, MLP 14336): qkv GEMM,
    KV append of the new token, decode attention (plan, attention, combine),
    o_proj, gate_up and down GEMMs.  Norms, rotary embedding and the SiLU
    product are elementwise work outside this library and are left out; each
    kernel reads inputs of the right shape, so the timing does not depend on
    the values.  A ring of four layers, each with its own weights (1.7 GB in
    all) and its own pages of the KV cache, keeps every step's weights out of
    the caches, as in a real model whose layers each read theirs once per
    iteration.  Each point: the four layers captured into one HIP graph
    (kernel launches only), replayed `reps` times after a warm-up replay and
    20 ms of untimed replays; per-component graphs of the same four layers
    give the split (`components`).  Fits T = c*N_req + d*N_kv + e, the same
    form per GEMM tile region, and the boosted model."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd
    from paper_2509_04827_amd import latency_model as lm

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gen = torch.Generator(device=dev).manual_seed(0)
    rng = np.random.default_rng(0)
    H, Hq, Hkv, D, S, FF = 4096, 32, 8, 128, 16, 14336
    shapes = {"qkv": (6144, H), "o_proj": (H, H), "gate_up": (2 * FF, H), "down": (H, FF)}

    def rnd(*shape):
        return torch.randn(shape, generator=gen, device=dev).to(torch.bfloat16)

    weights = [{k: rnd(n, kk) for k, (n, kk) in shapes.items()} for _ in range(LAYER_RING)]
    max_tok = max(b * l for b in batches for l in lengths)
    pages_per_layer = max_tok // S + max(batches)
    npages = pages_per_layer * LAYER_RING
    kpool = torch.empty((npages, S, Hkv, D), dtype=torch.bfloat16, device=dev)
    vpool = torch.empty_like(kpool)
    for pool in (kpool, vpool):   # filled in slices: no full-size fp32 temporary
        for i in range(0, npages, 8192):
            pool[i:i + 8192].copy_(torch.randn(pool[i:i + 8192].shape, generator=gen, device=dev))
    stream = torch.cuda.current_stream()
    scale = float(np.float32(1.0 / np.sqrt(D)))
    rows = []

    for B in batches:
        x = rnd(B, H)
        y_qkv = torch.empty((B, 6144), dtype=torch.bfloat16, device=dev)
        q = rnd(B, Hq, D)
        knew, vnew = rnd(B, Hkv, D), rnd(B, Hkv, D)
        attn_out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=dev)
        y_o = torch.empty((B, H), dtype=torch.bfloat16, device=dev)
        y_gu = torch.empty((B, 2 * FF), dtype=torch.bfloat16, device=dev)
        act = rnd(B, FF)
        y_down = torch.empty((B, H), dtype=torch.bfloat16, device=dev)
        gws = {k: torch.empty(max(16, vd.vd_gemm_workspace_size(B, n, kk)), dtype=torch.uint8, device=dev)
               for k, (n, kk) in shapes.items()}
        for L in lengths:
            if B * L > max_tok:
                continue
            P = (L + S - 1) // S
            pts, sl = [], torch.full((B,), L, dtype=torch.int32, device=dev)
            pos = torch.full((B,), L - 1, dtype=torch.int32, device=dev)
            for layer in range(LAYER_RING):
                perm = rng.permutation(pages_per_layer)[:B * P] + layer * pages_per_layer
                pts.append(torch.from_numpy(perm.reshape(B, P).astype(np.int32)).to(dev))
            aws = vd.alloc_workspace(B, Hq, Hkv, P)
            # no explicit stream: each call goes to the current stream, the
            # capture stream while a graph is being recorded
            comps = {
                "qkv": lambda w, pt: vd.vd_gemm_bf16(x, w["qkv"], y_qkv, gws["qkv"]),
                "append": lambda w, pt: vd.vd_kv_append(knew, vnew, kpool, vpool, pt, pos),
                "attn": lambda w, pt: vd.vd_decode_attn(q, kpool, vpool, pt, sl, attn_out, scale, aws),
                "o_proj": lambda w, pt: vd.vd_gemm_bf16(attn_out.view(B, H), w["o_proj"], y_o, gws["o_proj"]),
                "gate_up": lambda w, pt: vd.vd_gemm_bf16(y_o, w["gate_up"], y_gu, gws["gate_up"]),
                "down": lambda w, pt: vd.vd_gemm_bf16(act, w["down"], y_down, gws["down"]),
            }

            def graph_us(names):
                def body():
                    for layer in range(LAYER_RING):
                        for n in names:
                            comps[n](weights[layer], pts[layer])
                side = torch.cuda.Stream()   # one eager pass first: lazy set-up stays out of the capture
                side.wait_stream(stream)
                with torch.cuda.stream(side):
                    body()
                stream.wait_stream(side)
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    body()
                settle_clocks(g.replay, 0.02)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(reps):
                    g.replay()
                e1.record(stream)
                torch.cuda.synchronize()
                del g
                return e0.elapsed_time(e1) * 1e3 / (reps * LAYER_RING)

            row = dict(n_req=B, tokens_per_req=L, n_kv=B * L)
            row["us_layer"] = round(graph_us(list(comps)), 2)
            if components:
                for n in comps:
                    row["us_" + n] = round(graph_us([n]), 2)
            rows.append(row)
            print("layer B %4d L %5d N_kv %8d  layer %8.2f us  %s"
                  % (B, L, B * L, row["us_layer"], " ".join("%s %.1f" % (k[3:], v) for k, v in row.items()
                                                            if k.startswith("us_") and k != "us_layer")),
                  file=sys.stderr, flush=True)
            del aws, pts
    os.makedirs(outdir, exist_ok=True)
    keys = list(rows[0].keys())
    with open(os.path.join(outdir, name + ".csv"), "w") as f:
        f.write(",".join(keys) + "\n")
        for r in rows:
            f.write(",".join(str(r[k]) for k in keys) + "\n")
    n_req = np.array([r["n_req"] for r in rows], float)
    n_kv = np.array([r["n_kv"] for r in rows], float)
    t = np.array([r["us_layer"] for r in rows], float)
    fit = lm.fit_linear(n_req, n_kv, t)
    bounds = lm.tile_bounds(n_req)   # the coarse grid stops at 512: one edge, at 256
    tf = lm.fit_per_tile(n_req, n_kv, t, bounds)
    res = {"points": len(rows), "c_us_per_req": fit.c, "d_us_per_kv_token": fit.d, "e_us": fit.e,
           "r2": fit.r2, "mae_us": fit.mae,
           "per_tile": [{"n_req_max": b, "c": f.c, "d": f.d, "e": f.e, "r2": f.r2, "mae_us": f.mae}
                        for b, f in zip(list(bounds) + [None], tf.fits)],
           "holdout": lm.holdout_mae(n_req, n_kv, t, tile_bounds=bounds)}
    with open(os.path.join(outdir, name + "_fit.json"), "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res), flush=True)


def score_ab(outdir: str, workloads, rounds: int = 7, iters: int = 50, flushed: int = 30):
    """The two score paths of the attention kernel against each other: the
    vector-ALU score (the default for G <= 8: bf16 pair dot products summed
    across lanes by DPP) and the matrix-core one (VD_FLAG_SCORE_MFMA).  Per workload (seed
    0, the bench's inputs), in one process on the same inputs and clocks:
    `rounds` rounds that alternate which path goes first, each timing
    `iters` back-to-back attention launches (the self-planned kernel alone,
    events around the burst) and `iters` whole steps per path; then
    `flushed` single launches per path, interleaved, each after a 1 GiB read
    that flushes the caches.  Medians over rounds / launches.  Writes
    DIR/attn_score_ab.{csv,json}."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd
    from workloads import kv_bytes, make_case

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    paths = (("mfma", vd.VD_FLAG_SCORE_MFMA), ("valu", 0))
    fbuf = torch.zeros(1 << 30, dtype=torch.uint8, device=dev)
    fsink = torch.zeros(4, dtype=torch.int32, device=dev)
    rows = []
    for name in workloads:
        c = make_case(name, seed=0, fill="zero")
        q, k, v = c["q"].to(dev), c["k_pages"].to(dev), c["v_pages"].to(dev)
        pt, sl = c["page_table"].to(dev), c["seq_lens"].to(dev)
        B, Hq, Hkv, maxp = c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"]
        out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
        ws = vd.alloc_workspace(B, Hq, Hkv, maxp)
        nbytes = kv_bytes(c)
        print("score-ab: %s N_req %d N_kv %d" % (name, B, c["n_kv"]), file=sys.stderr, flush=True)

        def attn(f):
            vd.vd_decode_partial(q, k, v, pt, sl, out, c["scale"], ws,
                                 flags=vd.VD_FLAG_SELF_PLAN | f, stream=stream)

        def whole(f):
            vd.vd_decode_attn(q, k, v, pt, sl, out, c["scale"], ws, flags=f, stream=stream)

        def burst(fn, f):
            for _ in range(3):
                fn(f)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(iters):
                fn(f)
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3 / iters

        settle_clocks(lambda: whole(0), 0.3)
        t = {p: {"attn": [], "step": [], "flushed": []} for p, _ in paths}
        for r in range(rounds):
            for p, f in (paths if r % 2 == 0 else paths[::-1]):
                t[p]["attn"].append(burst(attn, f))
                t[p]["step"].append(burst(whole, f))
        for i in range(flushed):
            for p, f in (paths if i % 2 == 0 else paths[::-1]):
                vd.vd_stream_read(fbuf, fsink, stream=stream)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                attn(f)
                e1.record(stream)
                torch.cuda.synchronize()
                t[p]["flushed"].append(e0.elapsed_time(e1) * 1e3)
        row = {"workload": name, "G": Hq // Hkv, "n_req": B, "n_kv": c["n_kv"], "kv_bytes": nbytes,
               "rounds": rounds, "iters": iters, "flushed": flushed}
        for p, _ in paths:
            for kind in ("attn", "step", "flushed"):
                row["%s_%s_us" % (p, kind)] = round(float(np.median(t[p][kind])), 2)
            row["%s_attn_gbs" % p] = round(nbytes / (row["%s_attn_us" % p] * 1e-6) / 1e9, 1)
        for kind in ("attn", "step", "flushed"):
            row["valu_over_mfma_%s" % kind] = round(row["valu_%s_us" % kind] / row["mfma_%s_us" % kind], 4)
        print(json.dumps(row), flush=True)
        rows.append(row)
        del q, k, v, out, ws
        torch.cuda.empty_cache()
    os.makedirs(outdir, exist_ok=True)
    keys = list(rows[0].keys())
    with open(os.path.join(outdir, "attn_score_ab.csv"), "w") as f:
        f.write(",".join(keys) + "\n")
        for r in rows:
            f.write(",".join(str(r[x]) for x in keys) + "\n")
    with open(os.path.join(outdir, "attn_score_ab.json"), "w") as f:
        json.dump(rows, f, indent=1)


def next_profile(outdir: str, iters: int = 20, warmup: int = 3, only=None, hipblaslt: bool = False):
    """A short, profiler-friendly run of the other kernels: vd_gemm_bf16 on
    the four Llama-3-8B-shaped projections at M = 1, 16, 64, 256, 257 and
    1024 (cold weights: a ring of copies over 1 GiB), then
    vd_kv_append on the chat batch's sizes (256 requests, 8 KV heads).  Each
    case is a burst of `iters` calls after `warmup` calls, with a 5 ms pause
    before it, so a kernel trace splits into one burst per case in the order
    of next_profile.csv, and starts with one vd_stream_read of 4 KiB (a
    marker dispatch, so counter runs without timestamps split by case too).
    Optionally ends with --copy-calibration copies.

    `only` = (shape, M) runs that one GEMM case and no KV append; with
    `hipblaslt` the case calls torch.matmul instead of vd_gemm_bf16 (the
    same operands), to set the two kernels' counters side by side."""
    import numpy as np
    import torch

    import paper_2509_04827_amd as vd

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gen = torch.Generator(device=dev).manual_seed(0)
    stream = torch.cuda.current_stream()
    rows = []
    marker = torch.zeros(4096, dtype=torch.uint8, device=dev)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)

    def burst(fn):
        vd.vd_stream_read(marker, sink, blocks=1, stream=stream)
        settle_clocks(fn, 0.02)
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        time.sleep(0.005)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        time.sleep(0.005)
        return e0.elapsed_time(e1) * 1e3 / iters

    for name, N, K in GEMM_SHAPES:
        if only is not None and name != only[0]:
            continue
        # a ring of weight copies over 1 GiB: every call reads weights that
        # no cache holds, as a decode step does
        ring_n = max(2, -(-(1 << 30) // (N * K * 2)))
        ring = [torch.randn((N, K), generator=gen, device=dev).to(torch.bfloat16) for _ in range(ring_n)]
        for M in (NEXT_PROFILE_M if only is None else (only[1],)):
            x = torch.randn((M, K), generator=gen, device=dev).to(torch.bfloat16)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            ws = torch.empty(max(16, vd.vd_gemm_workspace_size(M, N, K)), dtype=torch.uint8, device=dev)
            cnt = [0]

            def call():
                if hipblaslt:
                    torch.matmul(x, ring[cnt[0] % ring_n].t(), out=y)
                else:
                    vd.vd_gemm_bf16(x, ring[cnt[0] % ring_n], y, ws, stream=stream)
                cnt[0] += 1
            us = burst(call)
            rows.append(dict(case="gemm_%s_M%d%s" % (name, M, "_hipblaslt" if hipblaslt else ""),
                             calls=iters, us_events=round(us, 2),
                             algorithmic_bytes=(N * K + M * K + M * N) * 2))
        del ring
        torch.cuda.empty_cache()
    if only is None:
        B, Hkv, S, maxp = 256, 8, 16, 4
        pages = torch.randperm(B * maxp, generator=torch.Generator().manual_seed(1)).to(torch.int32)
        pt = pages.view(B, maxp).to(dev)
        kp = torch.zeros((B * maxp, S, Hkv, 128), dtype=torch.bfloat16, device=dev)
        vp = torch.zeros_like(kp)
        kn = torch.randn((B, Hkv, 128), generator=gen, device=dev).to(torch.bfloat16)
        vn = torch.randn((B, Hkv, 128), generator=gen, device=dev).to(torch.bfloat16)
        pos = torch.arange(B, dtype=torch.int32, device=dev) % (maxp * S)
        us = burst(lambda: vd.vd_kv_append(kn, vn, kp, vp, pt, pos, stream=stream))
        rows.append(dict(case="kv_append_B256", calls=iters, us_events=round(us, 2),
                         algorithmic_bytes=2 * 2 * B * Hkv * 128 * 2 + B * 8))
    os.makedirs(outdir, exist_ok=True)
    with open(os.path.join(outdir, "next_profile.csv"), "w") as f:
        f.write("case,calls,us_events,algorithmic_bytes\n")
        for r in rows:
            f.write("%s,%d,%.2f,%d\n" % (r["case"], r["calls"], r["us_events"], r["algorithmic_bytes"]))
    print(json.dumps({"next_profile_cases": len(rows)}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle", type=float, default=0.3, metavar="SECONDS",
                    help="untimed steps for this long before the warm-up steps, so that the "
                         "GPU has left its idle clock state")
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the flushed-cache step timings")
    ap.add_argument("--flushed", type=int, default=50, metavar="N",
                    help="flushed-cache steps timed one at a time (default 50)")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the HBM read-ceiling run")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the oracle over the whole step for this much wall time "
                         "(at least 3 runs)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="after timing, copy a BYTES-sized buffer 3 times (a plain copy "
                         "kernel of known size, to scale HBM counters by)")
    ap.add_argument("--gemm-sweep", metavar="DIR", default=None,
                    help="instead of the bench line, time the decode-step projection GEMMs "
                         "over the batch size and write DIR/decode_gemm_sweep.csv")
    ap.add_argument("--clock-sweep", metavar="DIR", default=None,
                    help="instead of the bench line, time the attention kernel against the "
                         "shader clock it ran at and write DIR/decode_clock_sweep.{csv,json}")
    ap.add_argument("--clock-bursts", type=int, default=10, metavar="N",
                    help="with --clock-sweep: bursts of steps, each after an idle pause")
    ap.add_argument("--next-profile", metavar="DIR", default=None,
                    help="short run of the GEMM (4 shapes x M 1/16/64/256/257/1024) and KV-append kernels "
                         "for a kernel trace; writes next_profile.csv to DIR")
    ap.add_argument("--gemm-case", metavar="SHAPE:M", default=None,
                    help="with --next-profile: only this GEMM case (e.g. gate_up:1024), no KV append")
    ap.add_argument("--hipblaslt", action="store_true",
                    help="with --gemm-case: run the case through torch.matmul (hipBLASLt) instead")
    ap.add_argument("--cpu-configs", metavar="DIR", default=None,
                    help="time the oracle on the host cores and the GPU on every seeded workload; "
                         "write oracle_cpu_baseline.{csv,json} to DIR")
    ap.add_argument("--layer-dense", metavar="DIR", default=None,
                    help="instead of the bench line, time the decode layer step over a dense batch grid "
                         "around the GEMM tile steps and write DIR/decode_layer_dense.csv")
    ap.add_argument("--layer-surface", metavar="DIR", default=None,
                    help="instead of the bench line, time a decode layer step (qkv GEMM, KV append, "
                         "attention, o_proj / gate_up / down GEMMs) over (batch, tokens per request) "
                         "and write DIR/decode_layer_surface.csv")
    ap.add_argument("--score-ab", metavar="DIR", default=None,
                    help="instead of the bench line, time the matrix-core and vector-ALU score "
                         "paths against each other, interleaved, and write DIR/attn_score_ab.csv")
    ap.add_argument("--ab-workloads", default="tiny_b4,llama8b_b64,chat_b256,gqa8_b128,long_b16",
                    help="comma-separated workloads for --score-ab")
    ap.add_argument("--score", choices=("default", "mfma"), default="default",
                    help="score path of the bench line's attention kernel (mfma: "
                         "VD_FLAG_SCORE_MFMA, for profiling that path)")
    ap.add_argument("--surface", metavar="DIR", default=None,
                    help="instead of the bench line, measure the latency surface over "
                         "(batch, tokens per request) and write DIR/decode_latency_surface.{csv,md}")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the decode-attention path has no "
              "multi-GPU mode (sequences shard across GPUs with no exchange). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2509_04827_amd as vd
    from workloads import WORKLOADS, bits, kv_bytes, make_case

    if args.surface:
        latency_surface(args.surface)
        return
    if args.score_ab:
        score_ab(args.score_ab, [x for x in args.ab_workloads.split(",") if x])
        return
    if args.layer_surface:
        layer_surface(args.layer_surface)
        return
    if args.layer_dense:
        layer_surface(args.layer_dense, batches=LAYER_DENSE_BATCH, lengths=LAYER_DENSE_LEN,
                      components=False, name="decode_layer_dense")
        return
    if args.gemm_sweep:
        gemm_sweep(args.gemm_sweep)
        return
    if args.clock_sweep:
        clock_sweep(args.clock_sweep, bursts=args.clock_bursts)
        return
    if args.cpu_configs:
        cpu_configs(args.cpu_configs)
        return
    if args.next_profile:
        only = None
        if args.gemm_case:
            shape, m = args.gemm_case.split(":")
            if shape not in [g[0] for g in GEMM_SHAPES] or int(m) < 1:
                raise SystemExit("--gemm-case: SHAPE:M with SHAPE one of %s" % [g[0] for g in GEMM_SHAPES])
            only = (shape, int(m))
        elif args.hipblaslt:
            raise SystemExit("--hipblaslt needs --gemm-case")
        next_profile(args.next_profile, only=only, hipblaslt=args.hipblaslt)
        if args.copy_calibration:
            n = args.copy_calibration // 4
            src = torch.ones(n, dtype=torch.int32, device="cuda:0")
            dst = torch.empty_like(src)
            for _ in range(3):
                dst.copy_(src)
            torch.cuda.synchronize()
        return

    w = WORKLOADS[args.workload]
    t0 = time.time()
    c = make_case(w, seed=0, fill="zero")
    print("bench: %s generated in %.1fs: N_req %d N_kv %d pages %d"
          % (w.name, time.time() - t0, c["num_seqs"], c["n_kv"], c["num_pages"]),
          file=sys.stderr, flush=True)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    q = c["q"].to(dev)
    k = c["k_pages"].to(dev)
    v = c["v_pages"].to(dev)
    pt = c["page_table"].to(dev)
    sl = c["seq_lens"].to(dev)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
    B, Hq, Hkv, maxp = c["num_seqs"], c["n_q_heads"], c["n_kv_heads"], c["max_pages_per_seq"]
    ws = vd.alloc_workspace(B, Hq, Hkv, maxp)
    stream = torch.cuda.current_stream()
    SF = vd.VD_FLAG_SCORE_MFMA if args.score == "mfma" else 0
    torch.cuda.synchronize()

    def step(ev0=None, ev1=None):
        # one call, two kernels (self-planned attention, combine); with
        # events, the same two stages called one by one around the attention
        # launch
        if ev0 is None:
            vd.vd_decode_attn(q, k, v, pt, sl, out, c["scale"], ws, flags=SF, stream=stream)
            return
        ev0.record(stream)
        vd.vd_decode_partial(q, k, v, pt, sl, out, c["scale"], ws,
                             flags=vd.VD_FLAG_SELF_PLAN | SF, stream=stream)
        ev1.record(stream)
        vd.vd_decode_combine(out, Hkv, maxp, ws, stream=stream)

    settle_steps = settle_clocks(step, args.settle)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # The timed region: K back-to-back steps and nothing else on the stream.
    K = args.steps
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(K):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / K
    # the last timed step's record: the shader clock its attention kernel ran at
    rec = vd.step_info(ws)

    # The attention kernel's average launch duration: K launches of the
    # step's attention kernel (vd_decode_partial with VD_FLAG_SELF_PLAN, the
    # kernel vd_decode_attn runs) back to back, events around the K.  Events
    # around each launch would also count its dispatch and end-of-kernel
    # write-back, a few microseconds each.
    def attn_only():
        vd.vd_decode_partial(q, k, v, pt, sl, out, c["scale"], ws,
                             flags=vd.VD_FLAG_SELF_PLAN | SF, stream=stream)

    for _ in range(args.warmup):
        attn_only()
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a0.record(stream)
    for _ in range(K):
        attn_only()
    a1.record(stream)
    torch.cuda.synchronize()
    attn_avg_ms = a0.elapsed_time(a1) / K

    # Flushed caches (the measurement protocol's primary timing): before each
    # step, a read of a 1 GiB buffer (vd_stream_read) evicts the 256 MB
    # Infinity Cache and the L2s without leaving dirty lines behind; then the
    # step alone between events, one step at a time (a host synchronisation
    # between steps).  The same with a 1 GiB write as the flush is kept for
    # comparison: the write's dirty lines are written back while the step
    # runs, which slows it.  Untimed: the flushes.
    cold = None
    if not args.no_cold:
        fbuf = torch.zeros(1 << 30, dtype=torch.uint8, device=dev)
        fsink = torch.zeros(4, dtype=torch.int32, device=dev)

        def read_flush():
            vd.vd_stream_read(fbuf, fsink, stream=stream)

        def write_flush():
            fbuf.zero_()

        def flushed(flush, attn_only_events, n):
            out = []
            for _ in range(n):
                flush()
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                if attn_only_events:
                    step(e[0], e[1])
                else:
                    e[0].record(stream)
                    step()
                    e[1].record(stream)
                torch.cuda.synchronize()
                out.append(e[0].elapsed_time(e[1]) * 1e3)
            return np.percentile(out, [10, 50, 90])

        n = args.flushed
        sp = flushed(read_flush, False, n)
        ap_ = flushed(read_flush, True, n)
        wp = flushed(write_flush, False, max(10, n // 5))
        del fbuf, fsink
        cold = {"flush": "read of 1 GiB before each step", "steps": n,
                "us_per_step_p10": round(float(sp[0]), 2), "us_per_step_median": round(float(sp[1]), 2),
                "us_per_step_p90": round(float(sp[2]), 2),
                "attn_us_p10": round(float(ap_[0]), 2), "attn_us_median": round(float(ap_[1]), 2),
                "attn_us_p90": round(float(ap_[2]), 2),
                "kv_gbs_median": round(kv_bytes(c) / (sp[1] * 1e-6) / 1e9, 2),
                "write_flush_us_per_step_median": round(float(wp[1]), 2)}

    # HBM read ceiling on this device: vd_stream_read over 4 GiB.
    ceiling = None
    if not args.no_ceiling:
        buf = torch.zeros(1 << 32, dtype=torch.uint8, device=dev)
        sink = torch.zeros(4, dtype=torch.int32, device=dev)
        for _ in range(2):
            vd.vd_stream_read(buf, sink, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(5):
            vd.vd_stream_read(buf, sink, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ceiling = round((1 << 32) * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
        del buf, sink

    if args.copy_calibration:
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    kvb = kv_bytes(c)
    P = (c["seq_lens"].numpy().astype(np.int64) + 15) // 16
    algo_bytes = (kvb + q.numel() * 2 + out.numel() * 2 + int(P.sum()) * 4 + B * 4)
    achieved = algo_bytes / (attn_avg_ms * 1e-3) / 1e9
    value = kvb / (ms_step * 1e-3) / 1e9
    traffic = committed_traffic(w.name) if args.score == "default" else None

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        hq, hk, hv = bits(c["q"]), bits(c["k_pages"]), bits(c["v_pages"])
        hpt, hsl = c["page_table"].numpy(), c["seq_lens"].numpy()
        times = []
        t_end = time.time() + args.cpu_seconds
        while True:
            t1 = time.time()
            oracle.decode_attn(hq, hk, hv, hpt, hsl, c["scale"])
            times.append(time.time() - t1)
            if (time.time() >= t_end and len(times) >= 3) or len(times) >= 200:
                break
        sec = float(np.median(times))
        cpu_model = None
        try:
            with open("/proc/cpuinfo") as f:
                cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
        except OSError:
            pass
        cpu = {"value": round(kvb / sec / 1e9, 3), "unit": "GB/s", "cores": oracle.max_threads(),
               "kind": "oracle", "cpu_model": cpu_model, "nproc": os.cpu_count(),
               "sample": "the whole %s step (all %d requests, %d KV tokens), fp64, %d run(s), "
                         "median %.2f s" % (w.name, B, c["n_kv"], len(times), sec)}

    line = {
        "metric": "decode-attention achieved HBM GB/s (% of peak) and us/step vs batch x KV tokens",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "settle": {"seconds": args.settle, "steps": settle_steps},
        "ms_per_step": round(ms_step, 5),
        "us_per_step": round(ms_step * 1e3, 2),
        "pct_of_peak": round(100.0 * value / PEAK_HBM_GBS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "num_seqs": B,
                   "n_q_heads": Hq, "n_kv_heads": Hkv, "head_dim": 128, "page_size": 16,
                   "n_kv_tokens": c["n_kv"], "kv_bytes": kvb, "seed": 0,
                   "score": "mfma" if args.score == "mfma" or Hq // Hkv > 8 else "valu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "kernel": "attn_kernel",
                     "algorithmic_bytes": algo_bytes, "avg_launch_us": round(attn_avg_ms * 1e3, 2),
                     "stream_read_ceiling_gbs": ceiling,
                     "frac_of_stream_ceiling": round(achieved / ceiling, 4) if ceiling else None},
        "cold_cache": cold,
        "cpu_baseline": cpu,
        "sclk_mhz": round(rec["sclk_mhz"], 1),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
