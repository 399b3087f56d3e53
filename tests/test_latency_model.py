"""Decode latency model (Eq. pred-itl fit and boosted trees) on synthetic data,
and on the latency surface measured on the GPU (profiles/)."""
import numpy as np

from paper_2509_04827_amd import latency_model as lm


def grid():
    n_req = np.repeat([1, 2, 4, 8, 16, 32, 64, 128, 256, 512], 6).astype(float)
    n_kv = n_req * np.tile([16, 64, 256, 1024, 4096, 16384], 10)
    return n_req, n_kv


def test_linear_fit_recovers_coefficients():
    n_req, n_kv = grid()
    t = 0.02 * n_req + 6.25e-4 * n_kv + 21.5
    f = lm.fit_linear(n_req, n_kv, t)
    assert abs(f.c - 0.02) < 1e-9 and abs(f.d - 6.25e-4) < 1e-12 and abs(f.e - 21.5) < 1e-7
    assert f.r2 > 1 - 1e-12 and f.mae < 1e-7
    # 4096 B of KV per token at 6.25e-4 us per token is 6.5536 TB/s
    assert abs(f.kv_bandwidth_gbs() - 6553.6) < 1e-6


def test_boosted_beats_constant_on_dense_data():
    rng = np.random.default_rng(0)
    n_req = rng.integers(1, 512, 4000).astype(float)
    n_kv = n_req * rng.integers(16, 4096, 4000)
    t = 0.02 * n_req + 6.25e-4 * n_kv + 21.5 + rng.normal(0, 1, 4000)
    m = lm.fit_boosted(n_req[:3000], n_kv[:3000], t[:3000])
    pred = m.predict(np.stack([n_req[3000:], n_kv[3000:]], 1))
    mae = np.abs(pred - t[3000:]).mean()
    assert mae < 0.1 * np.abs(t[3000:] - np.median(t[:3000])).mean()


def test_holdout_reports_both():
    n_req, n_kv = grid()
    t = 0.02 * n_req + 6.25e-4 * n_kv + 21.5
    r = lm.holdout_mae(n_req, n_kv, t)
    assert r["linear_mae_us"] < 1e-6 and r["n_test"] + r["n_train"] == 60


def test_boosted_interpolates_a_sparse_surface():
    """About a hundred points spanning three orders of magnitude, as the
    measured surface: trees with single-sample leaves (XGBoost's default
    minimum child weight) interpolate held-out points within a few percent;
    leaves of twenty samples would not split this grid at all."""
    n_req, n_kv = grid()
    t = 0.02 * n_req + 6.25e-4 * n_kv + 21.5
    rng = np.random.default_rng(1)
    idx = rng.permutation(t.size)
    te, tr = idx[:15], idx[15:]
    m = lm.fit_boosted(n_req[tr], n_kv[tr], t[tr])
    pred = m.predict(np.stack([n_req[te], n_kv[te]], 1))
    assert np.median(np.abs(pred - t[te]) / t[te]) < 0.1


def test_clock_scaled_fit():
    """beta recovered from T ~ f^-beta, and per-clock coefficients scaled by
    (f0 / f)^beta (the same model at its own clock returns itself)."""
    f = np.linspace(1400, 2400, 40)
    t = 250.0 * (2400.0 / f) ** 0.095
    beta = lm.fit_beta(f, t)
    assert abs(beta - 0.095) < 1e-9
    n_req, n_kv = grid()
    base = lm.fit_linear(n_req, n_kv, 0.02 * n_req + 6.25e-4 * n_kv + 21.5)
    m = lm.ClockScaledFit(base, 2400.0, beta)
    assert np.allclose(m.predict(n_req, n_kv, 2400.0), base.predict(n_req, n_kv))
    slow = m.at(1200.0)
    assert abs(slow.d / base.d - 2.0 ** 0.095) < 1e-12 and abs(slow.e / base.e - 2.0 ** 0.095) < 1e-12


def test_committed_surface_loads_and_fits():
    """The measured surface under profiles/ parses with both time columns
    (device time from graph replays, and Python-launched steps), and the
    decode model fits it: R^2 near 1 and a per-token cost d that implies a
    KV read rate below the 8 TB/s of HBM and above half of it."""
    import os
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "profiles", "decode_latency_surface.csv")
    for column in ("us_step_graph", "us_step"):
        n_req, n_kv, t = lm.load_surface(path, column=column)
        assert len(t) >= 100 and (t > 0).all()
        f = lm.fit_linear(n_req, n_kv, t)
        assert f.r2 > 0.999
        assert 4000 < f.kv_bandwidth_gbs() < 8000
        assert 0 < f.e < 50


def test_committed_layer_surface_charges_requests_to_the_gemms():
    """The measured decode layer step (qkv / o_proj / gate_up / down GEMMs,
    KV append, attention) under profiles/: Eq. pred-itl fits it, and the
    N_req term is material there, carried by the GEMMs (the attention-only
    surface has c near zero), while the N_kv term stays attention's K/V
    read rate."""
    import csv
    import os
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "profiles", "decode_layer_surface.csv")
    n_req, n_kv, t = lm.load_surface(path, n_q_heads=None, column="us_layer")
    assert len(t) >= 40 and (t > 0).all()
    f = lm.fit_linear(n_req, n_kv, t)
    assert f.r2 > 0.99
    # c * N_req at 256 requests is at least a fifth of the step at that
    # batch and its median length
    sel = n_req == 256
    assert f.c > 0 and f.c * 256 > 0.2 * np.median(t[sel])
    assert 4000 < f.kv_bandwidth_gbs() < 8000
    # the split: the GEMMs carry c, attention carries d
    rows = list(csv.DictReader(open(path)))
    gemm = np.array([sum(float(r[k]) for k in ("us_qkv", "us_o_proj", "us_gate_up", "us_down")) for r in rows])
    attn = np.array([float(r["us_attn"]) for r in rows])
    fg = lm.fit_linear(n_req, n_kv, gemm)
    fa = lm.fit_linear(n_req, n_kv, attn)
    assert fg.c > 0.8 * f.c and abs(fa.c) < 0.05 * f.c
    assert fa.d > 0.9 * f.d and abs(fg.d) < 0.1 * f.d
    # the layer is the sum of its parts, within what replaying the graphs
    # one component at a time adds in gaps
    parts = gemm + attn + np.array([float(r["us_append"]) for r in rows])
    assert np.all(np.abs(parts - t) < 0.15 * t + 10)


def test_per_tile_fit_follows_a_staircase():
    """Eq. pred-itl within each tile (Sec. 5.4): a surface with steps at the
    tile boundaries is exact per band, and one plane over all bands is not."""
    import pytest
    n_req = np.repeat([1, 32, 64, 128, 192, 255, 256, 257, 300, 384, 448, 512, 513, 576, 640], 3).astype(float)
    n_kv = n_req * np.tile([64, 256, 1024], 15)
    t = 0.4 * n_req + 6e-4 * n_kv + 100 + 20 * (n_req > 256) + 30 * (n_req > 512)
    tf = lm.fit_per_tile(n_req, n_kv, t, (256, 512))
    assert np.abs(tf.predict(n_req, n_kv) - t).max() < 1e-6
    assert list(tf.band([1, 256, 257, 512, 513, 10 ** 6])) == [0, 0, 1, 1, 2, 2]
    assert lm.fit_linear(n_req, n_kv, t).mae > 5
    with pytest.raises(ValueError):
        lm.fit_per_tile(n_req[n_req <= 300], n_kv[n_req <= 300], t[n_req <= 300], (256, 512))
    # band edges follow the grid: none past 512 keeps only the edge at 256,
    # and a held-out split that empties a band reports no per-band figure
    sel = n_req <= 300
    assert lm.tile_bounds(n_req[sel]) == (256,) and lm.tile_bounds(n_req) == (256, 512)
    few = n_req <= 257
    h = lm.holdout_mae(n_req[few], n_kv[few], t[few], test_fraction=0.5, seed=3, tile_bounds=(256,))
    assert h["tile_linear_mae_us"] is None and h["linear_mae_us"] >= 0   # 3 points above 256, halved


def test_committed_dense_surface_shows_the_tile_steps():
    """The decode layer step measured on a dense batch grid (profiles/): it
    jumps where the projection GEMMs need another row tile (Sec. 3.3,
    256 -> 257 and 512 -> 513) at every length, by about the same time
    (the GEMMs do not depend on the context), and Eq. pred-itl fitted per
    band between those boundaries predicts held-out points with well under
    half the error of one plane over all of them."""
    import csv
    import os
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "profiles", "decode_layer_dense.csv")
    rows = list(csv.DictReader(open(path)))
    assert len(rows) >= 80
    for L in {r["tokens_per_req"] for r in rows}:
        v = {int(r["n_req"]): float(r["us_layer"]) for r in rows if r["tokens_per_req"] == L}
        assert v[257] - v[256] > 20 and v[513] - v[512] > 20          # us
        assert v[256] <= 1.02 * v[255] and v[512] <= 1.02 * v[511]   # no step before the boundary
    n_req, n_kv, t = lm.load_surface(path, n_q_heads=None, column="us_layer")
    tf = lm.fit_per_tile(n_req, n_kv, t, (256, 512))
    assert min(f.r2 for f in tf.fits) > 0.97
    ho = [lm.holdout_mae(n_req, n_kv, t, seed=s, tile_bounds=(256, 512)) for s in range(5)]
    tile = np.mean([h["tile_linear_mae_us"] for h in ho])
    lin = np.mean([h["linear_mae_us"] for h in ho])
    assert tile < 0.5 * lin
