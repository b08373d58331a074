"""Pins for the CPU oracle: checks against what the paper and mathematics fix,
never against the oracle itself or the device path.

Every pin takes an ``oracle.Oracle`` and raises AssertionError on failure, so
the same pins run on the real oracle (must pass) and on deliberately broken
copies of it (each must be caught by at least one pin; test_oracle_mutants).

What pins what:
  silu_closed_forms      Eq. 2: SiLU(0)=0, SiLU(z)-SiLU(-z)=z, the minimum
                         obeys SiLU(z*) = 1+z* (stationarity), sigmoid(1),
                         asymptotes (+z, and -0 below about -88)
  dense_vs_library       Eq. 1 against numpy float64 matmuls (non-square
                         shapes, so a transposed operand fails)
  t0_is_dense            t = 0 keeps every neuron: bit-identical to dense
  high_t_is_zero         t above every |v|: y is exactly +0 (or residual)
  single_active          one kept neuron j: y = h_j W_down[j, :] exactly
  tie_is_kept            |v_j| == t keeps j (Eq. 4 uses >=)
  masked_matrix_form     Appendix D: per-neuron "expert" sum equals the
                         masked matrix product (mask*v*u) W_down
  hand_example           tests/golden/hand_example.json, derived by hand
  residual_is_added      y(residual) = residual + y(no residual)
  threshold_rank         Eq. 3: order statistic of rank ceil(k n) vs numpy
                         sort, and #{a<t} <= r-1 < k n <= r <= #{a<=t}
  calib_acts_vs_library  |SiLU(X W_gate)| against numpy matmul
  calib_analytic         t close to the analytic quantile of |SiLU(sigma Z)|
  rmsnorm_closed_forms   constant rows, the (3,4) row, scale invariance
  stack_vs_library       x_{l+1} = x_l + MLP_l(RMSNorm(x_l)) over 3 layers
                         against numpy float64 matmuls, dense and sparse
                         (per-layer thresholds), with the kept counts
  stack_infinite_t_is_identity
                         every neuron masked: each x_l equals x_0 exactly
  sparse_input_gemv      Appendix B's CATS on a layer input: masked product
                         vs numpy, t = 0 plain product, t above all |x| is
                         zero, one kept channel exact, ties kept
  topk_thresholds        per-token cutoffs: each row's own order statistic
                         vs a numpy sort, exact kept counts, k = 0 and 1
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _tol(O, f32: float, f64: float) -> float:
    return f32 if O.precision == "f32" else f64


def _rng_mlp(seed: int, B: int, d: int, m: int, wstd: float = 0.3):
    r = np.random.default_rng(seed)
    x = r.standard_normal((B, d)).astype(np.float32)
    wg = (r.standard_normal((d, m)) * wstd).astype(np.float32)
    wu = (r.standard_normal((d, m)) * wstd).astype(np.float32)
    wd = (r.standard_normal((m, d)) * wstd).astype(np.float32)
    return x, wg, wu, wd


def _np_silu(z):
    return z / (1.0 + np.exp(-z))


def pin_silu_closed_forms(O):
    assert O.silu(0.0) == 0.0
    # SiLU(z) - SiLU(-z) = z (sigmoid(z) + sigmoid(-z) = 1)
    for z in (0.125, 0.5, 1.0, 2.0, 3.5, 7.0):
        lhs = O.silu(z) - O.silu(-z)
        assert abs(lhs - z) <= _tol(O, 4e-7, 1e-15) * max(1.0, z), (z, lhs)
    # sigmoid(1) = 1 / (1 + 1/e)
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    assert abs(O.silu(1.0) - s1) <= _tol(O, 2.5e-7, 2e-16), O.silu(1.0)
    # the minimum z* satisfies SiLU'(z*) = 0, i.e. SiLU(z*) = 1 + z*
    lo, hi = -3.0, 0.0
    gr = (math.sqrt(5.0) - 1.0) / 2.0
    for _ in range(80):  # golden-section search on the oracle's own SiLU
        a = hi - gr * (hi - lo)
        b = lo + gr * (hi - lo)
        if O.silu(a) < O.silu(b):
            hi = b
        else:
            lo = a
    zs = 0.5 * (lo + hi)
    # stationarity 1 + z(1 - sigmoid(z)) = 0 has the closed-form root
    # z* = -1 - W(1/e) (Lambert W), where SiLU(z*) = 1 + z*
    from scipy.special import lambertw

    zstar = -1.0 - float(lambertw(math.exp(-1.0)).real)
    assert abs(zs - zstar) < _tol(O, 2e-3, 1e-6), (zs, zstar)
    assert abs(O.silu(zstar) - (1.0 + zstar)) < _tol(O, 1e-7, 1e-15), (zstar, O.silu(zstar))
    # asymptotes: SiLU(z) -> z for large z, -> -0 for very negative z
    assert abs(O.silu(40.0) - 40.0) <= _tol(O, 0.0, 1e-14)
    assert O.silu(-40.0) < 0.0 and abs(O.silu(-40.0)) < 1e-15
    assert abs(O.silu(-100.0)) < 1e-40 and math.copysign(1.0, O.silu(-100.0)) < 0
    # sign follows z; increasing right of the minimum
    zz = np.linspace(-1.2, 6.0, 50)
    vals = [O.silu(z) for z in zz]
    assert all(np.sign(v) == np.sign(z) for v, z in zip(vals, zz) if z != 0)
    assert all(b >= a for a, b in zip(vals, vals[1:]))


def pin_dense_vs_library(O):
    for seed, (B, d, m) in enumerate([(3, 24, 40), (2, 40, 24), (1, 16, 7)]):
        x, wg, wu, wd = _rng_mlp(100 + seed, B, d, m)
        # dense must ignore t entirely
        got = O.cats_mlp(x, wg, wu, wd, t=1e9, dense=True)
        x64, g64 = x.astype(np.float64), wg.astype(np.float64)
        g = x64 @ g64
        u = x64 @ wu.astype(np.float64)
        v = _np_silu(g)
        y = (v * u) @ wd.astype(np.float64)
        scale = np.abs(y).max()
        err = np.abs(got["y"] - y).max()
        assert err <= _tol(O, 2e-5, 1e-12) * scale, (seed, err, scale)
        assert np.abs(got["v"] - v).max() <= _tol(O, 2e-5, 1e-12) * max(1.0, np.abs(v).max())
        for b in range(B):
            assert got["cnt"][b] == m and list(got["idx"][b]) == list(range(m))
            assert np.abs(got["h"][b] - v[b] * u[b]).max() <= _tol(O, 2e-5, 1e-12) * max(1.0, np.abs(v * u).max())


def pin_t0_is_dense(O):
    x, wg, wu, wd = _rng_mlp(7, 2, 32, 48)
    a = O.cats_mlp(x, wg, wu, wd, t=0.0)
    b = O.cats_mlp(x, wg, wu, wd, t=0.0, dense=True)
    assert np.array_equal(a["y"].view(np.int64), b["y"].view(np.int64))
    assert list(a["cnt"]) == [48, 48]


def pin_high_t_is_zero(O):
    x, wg, wu, wd = _rng_mlp(8, 2, 32, 48)
    v = O.cats_mlp(x, wg, wu, wd, t=0.0)["v"]
    t = float(np.abs(v).max()) * 1.5 + 1.0
    got = O.cats_mlp(x, wg, wu, wd, t=t)
    assert list(got["cnt"]) == [0, 0]
    assert np.all(got["y"] == 0.0) and not np.any(np.signbit(got["y"]))
    res = np.random.default_rng(3).standard_normal((2, 32)).astype(np.float32)
    got = O.cats_mlp(x, wg, wu, wd, t=float("inf"), residual=res)
    assert np.array_equal(got["y"], res.astype(np.float64))


def pin_single_active(O):
    x, wg, wu, wd = _rng_mlp(9, 1, 32, 64)
    g = x.astype(np.float64) @ wg.astype(np.float64)
    av = np.abs(_np_silu(g[0]))
    order = np.argsort(av)
    top, second = av[order[-1]], av[order[-2]]
    assert top - second > 1e-3 * top  # a well separated maximum
    got = O.cats_mlp(x, wg, wu, wd, t=0.5 * (top + second))
    j = int(order[-1])
    assert got["cnt"][0] == 1 and list(got["idx"][0]) == [j]
    h = got["h"][0][0]
    if O.precision == "f32":
        expect = (np.float32(h) * wd[j]).astype(np.float64)
    else:
        expect = h * wd[j].astype(np.float64)
    assert np.array_equal(got["y"][0], expect)


def pin_tie_is_kept(O):
    x, wg, wu, wd = _rng_mlp(10, 1, 32, 64)
    v = O.cats_mlp(x, wg, wu, wd, t=0.0)["v"][0]
    for j in (3, 17, 40):
        t = abs(v[j])  # exactly representable in the oracle's precision
        got = O.cats_mlp(x, wg, wu, wd, t=t)
        assert j in set(got["idx"][0].tolist()), (j, t)
        assert got["cnt"][0] == int(np.sum(np.abs(v) >= t))


def pin_masked_matrix_form(O):
    x, wg, wu, wd = _rng_mlp(11, 3, 8, 16, wstd=0.4)
    x64 = x.astype(np.float64)
    g = x64 @ wg.astype(np.float64)
    u = x64 @ wu.astype(np.float64)
    v = _np_silu(g)
    t = 0.05  # below the |SiLU| bump of 0.2785, so negative activations are kept
    got = O.cats_mlp(x, wg, wu, wd, t=t)
    mask = (np.abs(v) >= t).astype(np.float64)
    assert np.any((mask > 0) & (v < 0)), "the case must keep some negative activations"
    y_matrix = (mask * v * u) @ wd.astype(np.float64)
    for b in range(3):
        y_expert = np.zeros(8)
        for j in range(16):
            if abs(v[b, j]) >= t:
                y_expert += v[b, j] * u[b, j] * wd[j].astype(np.float64)
        assert np.abs(y_expert - y_matrix[b]).max() <= 1e-12 * max(1.0, np.abs(y_matrix[b]).max())
        assert list(got["idx"][b]) == list(np.nonzero(mask[b])[0])
        assert np.abs(got["y"][b] - y_matrix[b]).max() <= _tol(O, 2e-5, 1e-12) * max(1.0, np.abs(y_matrix[b]).max())


def pin_hand_example(O):
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        G = json.load(f)
    x = np.array(G["x"], np.float32)[None, :]
    wg = np.array(G["w_gate"], np.float32)
    wu = np.array(G["w_up"], np.float32)
    wd = np.array(G["w_down"], np.float32)
    for case in G["exact_cases"]:
        got = O.cats_mlp(x, wg, wu, wd, t=case["t"])
        assert list(got["idx"][0]) == case["active"], case
        assert np.array_equal(got["y"][0], np.array(case["y"])), (case, got["y"])
    silu_m1 = -1.0 / (1.0 + math.e)
    wd64 = wd.astype(np.float64)
    for case in G["formula_cases"]:
        got = O.cats_mlp(x, wg, wu, wd, t=case["t"])
        assert list(got["idx"][0]) == case["active"], case
        expect = 40.0 * wd64[0] + 4.0 * silu_m1 * wd64[3] + 21.0 * wd64[4]
        if case["t"] == 0.0:
            silu_m40 = -40.0 / (1.0 + math.exp(40.0))
            expect = expect + 0.0 * wd64[1] + 3.0 * silu_m40 * wd64[2]
        assert np.abs(got["y"][0] - expect).max() <= _tol(O, 1e-5, 1e-12) * np.abs(expect).max(), case


def pin_residual_is_added(O):
    x, wg, wu, wd = _rng_mlp(12, 2, 32, 48)
    res = np.random.default_rng(4).standard_normal((2, 32)).astype(np.float32)
    a = O.cats_mlp(x, wg, wu, wd, t=0.1)
    b = O.cats_mlp(x, wg, wu, wd, t=0.1, residual=res)
    if O.precision == "f32":
        expect = (res + a["y"].astype(np.float32)).astype(np.float64)
    else:
        expect = res.astype(np.float64) + a["y"]
    assert np.array_equal(b["y"], expect)


def _rank(n: int, k: float) -> int:
    if k == 0:
        return 0
    return min(n, max(1, math.ceil(Fraction(repr(k)) * n)))


def pin_threshold_rank(O):
    r = np.random.default_rng(13)
    a = r.standard_normal(1000)
    a[::7] = a[3]  # ties
    a[5] = -a[11]  # ties across sign
    absa = np.sort(np.abs(a))
    n = a.size
    for k in (0.1, 1 / 3, 0.5, 0.7, 0.9, 0.999, 1.0):
        rr = _rank(n, k)
        assert O.cutoff_rank(n, k) == rr, (k, O.cutoff_rank(n, k), rr)
        t = O.threshold(a, k)
        assert t == absa[rr - 1], (k, t, absa[rr - 1])
        below = int(np.sum(absa < t))
        upto = int(np.sum(absa <= t))
        kn = Fraction(repr(k)) * n
        assert below <= rr - 1 < kn <= rr <= upto, (k, below, rr, upto)
    assert O.threshold(a, 0.0) == 0.0
    assert O.threshold(a, 1.0) == absa[-1]
    assert O.cutoff_rank(1000, 0.7) == 700 and O.cutoff_rank(10, 0.05) == 1


def pin_calib_acts_vs_library(O):
    r = np.random.default_rng(14)
    X = r.standard_normal((6, 24)).astype(np.float32)
    wg = (r.standard_normal((24, 40)) * 0.3).astype(np.float32)
    acts = O.calib_acts(X, wg)
    expect = np.abs(_np_silu(X.astype(np.float64) @ wg.astype(np.float64)))
    assert np.abs(acts - expect).max() <= _tol(O, 2e-6, 1e-14) * max(1.0, expect.max())
    pairs = np.array([[0, 0], [5, 39], [2, 17], [3, 3]])
    at = O.calib_acts_at(X, wg, pairs)
    assert np.array_equal(at, acts[pairs[:, 0], pairs[:, 1]])


def _analytic_quantile(sig: np.ndarray, k: float) -> float:
    """t with mean_n P(|SiLU(sig_n Z)| <= t) = k, Z ~ N(0, 1)."""
    from scipy.optimize import brentq
    from scipy.stats import norm

    zmin, smin = -1.2784645427610738, 1.2784645427610738 - 1.0  # |SiLU| bump height 0.2785

    def cdf(t):
        # {s : |SiLU(s)| <= t} = (-inf, a] U [b, c] when t < smin, else (-inf, c]
        c = brentq(lambda s: _np_silu(s) - t, 0.0, 50.0)
        if t >= smin:
            p = norm.cdf(c / sig)
        else:
            b = brentq(lambda s: _np_silu(s) + t, zmin, 0.0)
            a = brentq(lambda s: _np_silu(s) + t, -60.0, zmin)
            p = norm.cdf(a / sig) + norm.cdf(c / sig) - norm.cdf(b / sig)
        return float(np.mean(p))

    return brentq(lambda t: cdf(t) - k, 1e-9, 20.0)


def pin_calib_analytic(O):
    r = np.random.default_rng(15)
    N, d, m = 128, 256, 688
    X = r.standard_normal((N, d)).astype(np.float32)
    wg = (r.standard_normal((d, m)) * 0.02).astype(np.float32)
    acts = O.calib_acts(X, wg)
    sig = 0.02 * np.linalg.norm(X.astype(np.float64), axis=1)
    for k in (0.5, 0.7, 0.9):
        t = O.threshold(acts, k)
        ta = _analytic_quantile(sig, k)
        assert abs(t - ta) <= 0.05 * ta, (k, t, ta)


def pin_rmsnorm_closed_forms(O):
    out = O.rmsnorm(np.full((1, 16), 3.0, np.float32), eps=0.0)
    assert np.abs(out - 1.0).max() <= _tol(O, 1e-7, 1e-15)
    out = O.rmsnorm(np.array([[3.0, 4.0]], np.float32), eps=0.0)
    rms = math.sqrt(12.5)
    assert np.abs(out[0] - np.array([3.0, 4.0]) / rms).max() <= _tol(O, 3e-7, 1e-15)
    out = O.rmsnorm(np.full((1, 8), 2.0, np.float32), eps=12.0)  # 2/sqrt(4+12) = 0.5
    assert np.abs(out - 0.5).max() <= _tol(O, 1e-7, 1e-15)
    x = np.random.default_rng(16).standard_normal((3, 40)).astype(np.float32)
    a = O.rmsnorm(x, eps=0.0)
    b = O.rmsnorm(x * np.float32(8.0), eps=0.0)  # exact power-of-two scaling
    assert np.abs(a - b).max() <= _tol(O, 1e-6, 1e-14)
    assert np.abs(np.mean(a * a, axis=1) - 1.0).max() <= _tol(O, 1e-6, 1e-12)


def _np_stack(x0, layers, ts, eps):
    """The residual stack through numpy float64 matmuls; the stream is
    rounded to float32 between layers, as both sides keep it."""
    x = x0.astype(np.float32)
    out = [x.copy()]
    cnts = []
    for l, (wg, wu, wd) in enumerate(layers):
        x64 = x.astype(np.float64)
        xn = (x64 / np.sqrt(np.mean(x64 * x64, axis=1, keepdims=True) + eps)).astype(np.float32)
        xn = xn.astype(np.float64)
        v = _np_silu(xn @ wg.astype(np.float64))
        u = xn @ wu.astype(np.float64)
        keep = np.ones_like(v, dtype=bool) if ts is None else ~(np.abs(v) < ts[l])
        cnts.append(keep.sum(axis=1))
        x = (x64 + (np.where(keep, v * u, 0.0) @ wd.astype(np.float64))).astype(np.float32)
        out.append(x.copy())
    return np.stack(out), np.array(cnts)


def pin_stack_vs_library(O):
    r = np.random.default_rng(17)
    B, d, m, L = 2, 24, 40, 3
    x0 = (r.standard_normal((B, d)) * 3.0).astype(np.float32)
    layers = [tuple((r.standard_normal(sh) * 0.3).astype(np.float32) for sh in ((d, m), (d, m), (m, d)))
              for _ in range(L)]
    # distinct thresholds per layer, away from every |v| the inputs produce
    ts = [0.4, 0.9, 0.2]
    for thr in (None, ts):
        got, cnt = O.stack(x0, layers, thr, eps=1e-5)
        exp, ecnt = _np_stack(x0, layers, thr, 1e-5)
        assert got.shape == (L + 1, B, d)
        assert np.array_equal(got[0], x0)
        scale = np.abs(exp).max()
        assert np.abs(got.astype(np.float64) - exp).max() <= _tol(O, 2e-5, 2e-6) * scale, thr
        assert np.array_equal(cnt, ecnt), (thr, cnt, ecnt)
    # the sparse and dense stacks differ (the thresholds drop neurons)
    assert not np.array_equal(O.stack(x0, layers, ts)[0][-1], O.stack(x0, layers, None)[0][-1])


def pin_stack_infinite_t_is_identity(O):
    r = np.random.default_rng(18)
    B, d, m, L = 3, 16, 20, 4
    x0 = r.standard_normal((B, d)).astype(np.float32)
    layers = [tuple((r.standard_normal(sh) * 0.3).astype(np.float32) for sh in ((d, m), (d, m), (m, d)))
              for _ in range(L)]
    got, cnt = O.stack(x0, layers, [math.inf] * L)
    for l in range(L + 1):
        assert np.array_equal(got[l], x0)
    assert not cnt.any()


def pin_sparse_input_gemv(O):
    """CATS on a layer's input (Appendix B): against the masked product
    through numpy float64, t = 0 against the plain product, t above every
    |x| gives zero (or the residual), one kept channel gives exactly
    x_i W[i, :], and ties at t are kept."""
    r = np.random.default_rng(19)
    B, d, n = 3, 40, 56
    x = r.standard_normal((B, d)).astype(np.float32)
    w = (r.standard_normal((d, n)) * 0.3).astype(np.float32)
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    for t in (0.0, 0.6, 1.3):
        got = O.sparse_input_gemv(x, w, t)
        keep = ~(np.abs(x64) < t)
        exp = np.where(keep, x64, 0.0) @ w64
        assert np.abs(got["y"] - exp).max() <= _tol(O, 2e-6, 1e-12) * max(1.0, np.abs(exp).max()), t
        for b in range(B):
            assert np.array_equal(got["idx"][b], np.nonzero(keep[b])[0]), (t, b)
    big = O.sparse_input_gemv(x, w, float(np.abs(x).max()) * 2)
    assert not big["y"].any() and not big["cnt"].any()
    res = r.standard_normal((B, n)).astype(np.float32)
    assert np.array_equal(O.sparse_input_gemv(x, w, 1e9, residual=res)["y"], res.astype(np.float64))
    xs = np.zeros((1, d), np.float32)
    xs[0, 7] = 2.5
    one = O.sparse_input_gemv(xs, w, 1.0)
    assert np.array_equal(one["y"][0], (np.float32(2.5) * w[7]).astype(np.float64)) if O.precision == "f32" \
        else np.array_equal(one["y"][0], 2.5 * w64[7])
    tie = O.sparse_input_gemv(xs, w, 2.5)
    assert tie["cnt"][0] == 1


def pin_topk_thresholds(O):
    """Top-k variant: every row's cutoff is its own order statistic of
    |SiLU(x W_gate)| (numpy float64 sort), the rows differ, the kept count
    obeys #{|v| >= t_b} >= m - r + 1 with equality when values are distinct,
    k = 0 gives 0, k = 1 keeps the largest only."""
    r_ = np.random.default_rng(20)
    B, d, m = 4, 24, 37
    x = (r_.standard_normal((B, d)) * np.array([[0.3], [1.0], [2.0], [4.0]])).astype(np.float32)
    wg = (r_.standard_normal((d, m)) * 0.3).astype(np.float32)
    a = np.abs(_np_silu(x.astype(np.float64) @ wg.astype(np.float64)))
    for k in (0.25, 0.5, 0.9, 1.0):
        t = O.topk_thresholds(x, wg, k)
        rr = _rank(m, k)
        for b in range(B):
            exp = np.sort(a[b])[rr - 1]
            assert abs(t[b] - exp) <= _tol(O, 2e-6, 1e-13) * max(1.0, exp), (k, b, t[b], exp)
            ours = O.calib_acts(x[b : b + 1], wg)[0]
            assert int(np.sum(ours >= t[b])) == m - rr + 1, (k, b)
        assert len(set(np.round(t, 9))) > 1, "rows of different scale share a cutoff"
    assert not O.topk_thresholds(x, wg, 0.0).any()
    full = O.topk_mlp(x, wg, wg, wg.T.copy(), 0.5)
    assert np.array_equal(full["cnt"], np.full(B, m - _rank(m, 0.5) + 1))


ALL_PINS = [
    pin_silu_closed_forms,
    pin_dense_vs_library,
    pin_t0_is_dense,
    pin_high_t_is_zero,
    pin_single_active,
    pin_tie_is_kept,
    pin_masked_matrix_form,
    pin_hand_example,
    pin_residual_is_added,
    pin_threshold_rank,
    pin_calib_acts_vs_library,
    pin_calib_analytic,
    pin_rmsnorm_closed_forms,
    pin_stack_vs_library,
    pin_stack_infinite_t_is_identity,
    pin_sparse_input_gemv,
    pin_topk_thresholds,
]
