"""Decode-attention latency model over (N_req, N_kv), fitted to measurements.

The paper's iteration-level controller needs the decode iteration time as a
function of the system state: EcoPred models it as T_D ~ c_f * N_req +
d_f * N_kv + e_f within a GEMM tile (Sec. 5.4, Eq. pred-itl), with N_kv
driving the attention layer and its KV-cache reads, and fits a boosted-tree
regressor on (f, N_req, N_kv) for accuracy (Sec. 5.4; decode model settings in
the appendix on its XGBoost configuration: absolute-error objective, 1000
rounds, learning rate 0.1, depth 6, early stopping after 200 rounds).

Here the same two models are fitted to the step times this library's
kernels measure on MI355X at its fixed clock: the decode-attention surface
written by ``bench.py --surface``, and the decode layer step (projection
GEMMs, KV append, attention) written by ``bench.py --layer-surface``, where
the N_req term is carried by the GEMMs as the paper's model charges it.  CPU only; it consumes the
measurements and launches nothing.  XGBoost is not available in this
environment, so the boosted model is scikit-learn's histogram gradient
boosting with the same objective, rate, depth, round budget and patience
(it has no row/column subsampling).  Its leaves may hold a single sample, as
XGBoost's default minimum child weight of one allows; scikit-learn's own
default of twenty samples per leaf leaves almost no splits on a surface of
about a hundred points.
"""
from __future__ import annotations

import csv
from dataclasses import dataclass

import numpy as np


@dataclass
class LinearFit:
    """T = c * n_req + d * n_kv + e (microseconds)."""
    c: float
    d: float
    e: float
    r2: float
    mae: float

    def predict(self, n_req, n_kv):
        return self.c * np.asarray(n_req, float) + self.d * np.asarray(n_kv, float) + self.e

    def kv_bandwidth_gbs(self, kv_bytes_per_token: int = 4096) -> float:
        """Bandwidth implied by the marginal cost of one KV token."""
        return kv_bytes_per_token / (self.d * 1e-6) / 1e9


@dataclass
class ClockScaledFit:
    """Per-clock coefficients of Eq. pred-itl from one measured clock: the
    paper fits c_f, d_f, e_f per GPU frequency f (Sec. 5.4); with the
    frequency relation T ~ f^-beta (Sec. 3.2, Eq. t-alpha-beta) measured for
    this kernel, T_f = T_f0 * (f0 / f)^beta scales all three alike."""
    base: LinearFit
    f0_mhz: float
    beta: float

    def at(self, f_mhz: float) -> LinearFit:
        k = (self.f0_mhz / float(f_mhz)) ** self.beta
        b = self.base
        return LinearFit(b.c * k, b.d * k, b.e * k, b.r2, b.mae * k)

    def predict(self, n_req, n_kv, f_mhz):
        return self.at(f_mhz).predict(n_req, n_kv)


def fit_beta(f_mhz, t) -> float:
    """beta of T ~ f^-beta by least squares on ln T = a - beta ln f."""
    f, t = np.asarray(f_mhz, float), np.asarray(t, float)
    A = np.stack([np.ones_like(f), np.log(f)], axis=1)
    (_, b), *_ = np.linalg.lstsq(A, np.log(t), rcond=None)
    return float(-b)


def load_surface(path: str, n_q_heads: int | None = 32, column: str = "us_step_graph"):
    """Rows of a latency-surface CSV as (n_req, n_kv, step time) arrays;
    `column` picks the device time per step (us_step_graph, steps replayed
    from a HIP graph: what an engine that captures its decode iteration
    sees) or the step time when each step is launched from Python
    (us_step, which at small steps is the binding's call rate)."""
    with open(path) as f:
        rows = [r for r in csv.DictReader(f)
                if n_q_heads is None or int(r["n_q_heads"]) == n_q_heads]
    n_req = np.array([int(r["n_req"]) for r in rows], float)
    n_kv = np.array([int(r["n_kv"]) for r in rows], float)
    t = np.array([float(r[column]) for r in rows], float)
    return n_req, n_kv, t


def fit_linear(n_req, n_kv, t) -> LinearFit:
    n_req, n_kv, t = (np.asarray(x, float) for x in (n_req, n_kv, t))
    A = np.stack([n_req, n_kv, np.ones_like(t)], axis=1)
    coef, *_ = np.linalg.lstsq(A, t, rcond=None)
    pred = A @ coef
    ss = ((t - t.mean()) ** 2).sum()
    r2 = 1.0 - ((t - pred) ** 2).sum() / ss if ss > 0 else 1.0
    return LinearFit(float(coef[0]), float(coef[1]), float(coef[2]), float(r2),
                     float(np.abs(t - pred).mean()))


@dataclass
class TileFit:
    """Eq. pred-itl within each GEMM tile (Sec. 5.4): one (c, d, e) per band
    of N_req between the batch sizes where the projection GEMMs need another
    row tile (Sec. 3.3).  Band i holds bounds[i-1] < N_req <= bounds[i]; the
    last band is open above."""
    bounds: tuple
    fits: list

    def band(self, n_req):
        return np.searchsorted(np.asarray(self.bounds, float), np.asarray(n_req, float), side="left")

    def predict(self, n_req, n_kv):
        n_req, n_kv = np.asarray(n_req, float), np.asarray(n_kv, float)
        b = self.band(n_req)
        out = np.empty(n_req.shape, float)
        for i, f in enumerate(self.fits):
            sel = b == i
            out[sel] = f.predict(n_req[sel], n_kv[sel])
        return out


def tile_bounds(n_req, candidates=(256, 512), min_points: int = 3) -> tuple:
    """The band edges among `candidates` that a surface reaches past: an
    edge is kept when at least `min_points` points lie above it."""
    n_req = np.asarray(n_req, float)
    return tuple(b for b in candidates if (n_req > b).sum() >= min_points)


def fit_per_tile(n_req, n_kv, t, bounds=(256, 512)) -> TileFit:
    """Eq. pred-itl fitted separately in each band of N_req (see TileFit);
    every band needs points of its own."""
    n_req, n_kv, t = (np.asarray(x, float) for x in (n_req, n_kv, t))
    b = np.searchsorted(np.asarray(bounds, float), n_req, side="left")
    fits = []
    for i in range(len(bounds) + 1):
        sel = b == i
        if sel.sum() < 3:
            raise ValueError("band %d of N_req has %d points; the fit needs 3" % (i, int(sel.sum())))
        fits.append(fit_linear(n_req[sel], n_kv[sel], t[sel]))
    return TileFit(tuple(bounds), fits)


def fit_boosted(n_req, n_kv, t, random_state: int = 42):
    """Boosted trees on (n_req, n_kv) with the decode settings of the paper."""
    from sklearn.ensemble import HistGradientBoostingRegressor

    X = np.stack([np.asarray(n_req, float), np.asarray(n_kv, float)], axis=1)
    model = HistGradientBoostingRegressor(
        loss="absolute_error", learning_rate=0.1, max_iter=1000, max_depth=6,
        early_stopping=True, n_iter_no_change=200, validation_fraction=0.2,
        min_samples_leaf=1, random_state=random_state)
    model.fit(X, np.asarray(t, float))
    return model


def holdout_mae(n_req, n_kv, t, test_fraction: float = 0.25, seed: int = 0, tile_bounds=None):
    """MAE of the models on a random held-out share of the points: the
    linear form over all points, the boosted trees and, with `tile_bounds`,
    the linear form per tile band."""
    n_req, n_kv, t = (np.asarray(x, float) for x in (n_req, n_kv, t))
    rng = np.random.default_rng(seed)
    idx = rng.permutation(t.shape[0])
    k = max(1, int(round(test_fraction * t.shape[0])))
    te, tr = idx[:k], idx[k:]
    lin = fit_linear(n_req[tr], n_kv[tr], t[tr])
    gb = fit_boosted(n_req[tr], n_kv[tr], t[tr])
    lin_mae = float(np.abs(lin.predict(n_req[te], n_kv[te]) - t[te]).mean())
    gb_mae = float(np.abs(gb.predict(np.stack([n_req[te], n_kv[te]], 1)) - t[te]).mean())
    out = {"linear_mae_us": lin_mae, "boosted_mae_us": gb_mae, "n_train": int(tr.size),
           "n_test": int(te.size)}
    if tile_bounds is not None:
        try:
            tf = fit_per_tile(n_req[tr], n_kv[tr], t[tr], tile_bounds)
            out["tile_linear_mae_us"] = float(np.abs(tf.predict(n_req[te], n_kv[te]) - t[te]).mean())
        except ValueError:   # the split left a band with too few training points
            out["tile_linear_mae_us"] = None
    return out
