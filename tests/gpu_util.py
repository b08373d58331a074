"""Shared helpers for the GPU parity tests (device path vs CPU oracle)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

# y agrees when max|y_gpu - y_oracle| <= Y_TOL * ||y_oracle||_inf (bf16 or
# fp32 weights, fp32 accumulation in a different order on each side).
Y_TOL = 2e-2
# Active sets must be identical except for neurons whose oracle |v| lies
# within BAND * t of t (the two sides round the gate dot product differently).
BAND = 1e-3


def say(*a):
    """Name the case on stdout before a GPU step (flushed)."""
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def device_layer(wg, wu, wd) -> P.Layer:
    """Upload math-layout weights and pack them neuron-major on the device."""
    return P.layer_from_math(wg.cuda(), wu.cuda(), wd.cuda())


def host_f32(*ts):
    return [t.float().numpy() for t in ts]


def band_ok(gpu_idx, ora_idx, ora_v_abs, t):
    """Symmetric difference of the two active sets lies inside the band."""
    g, o = set(int(i) for i in gpu_idx), set(int(i) for i in ora_idx)
    diff = sorted(g ^ o)
    bad = [j for j in diff if abs(ora_v_abs[j] - t) > BAND * t]
    return bad, len(diff)


# With the active sets reconciled (see check_forward), y must also agree
# within this much of ||y||_inf: fp32 sums in different orders.
Y_TIGHT = 1e-4


def h_bound(x, w_up, v):
    """Per (row, neuron) bound on |h_gpu - h_oracle| for the matrix-core
    path: x enters as bf16 hi + lo (16 mantissa bits, error below 2^-16 |x|
    per element, doubled for margin) and both sides accumulate d products
    in fp32 in different orders (at most d 2^-24 of the absolute sum):
    |v| (2^-15 + d 2^-24) sum_i |x_i w_up[i, j]|."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    a = x @ np.abs(np.asarray(w_up, dtype=np.float64))
    d = x.shape[1]
    return np.abs(v) * (2.0 ** -15 + d * 2.0 ** -24) * a


def check_forward(y, aux, ref, t, B, label="", h_rtol=1e-4, ref_all=None, w_down=None, h_abs=None):
    """Compare a device forward (y, aux dict) against an oracle result.

    Neurons inside the band may be active on one side only, and one such
    neuron can move y by a few percent of ||y||_inf (its h_j W_down[j] term).
    h_abs (optional, [B, m]) raises the h bar per neuron to a derived error
    bound (see h_bound).  When the oracle's full result (ref_all, every
    neuron kept) and W_down are given, the oracle y is corrected by exactly those neurons' terms, so both
    sides use the same mask, and then both bars (Y_TOL, Y_TIGHT) apply.
    Without that information only Y_TOL is applied.
    """
    y = y.detach().cpu().double().numpy().reshape(B, -1)
    yo = ref["y"]
    scale = float(np.abs(yo).max())
    flips = 0
    y_adj = yo.copy()
    # without the device's active lists the masks cannot be reconciled, so
    # only the spec bar applies
    corrected = aux is not None
    if aux is not None:
        cnt = aux["cnt"].cpu().numpy()
        idx = aux["idx"].cpu().numpy()
        v = aux["v"].cpu().double().numpy()
        h = aux["h"].cpu().double().numpy()
        for b in range(B):
            n = int(cnt[b])
            gi = idx[b, :n]
            assert n == 0 or (np.all(np.diff(gi) > 0) and gi[0] >= 0), f"{label}: row {b} not ascending"
            bad, nd = band_ok(gi, ref["idx"][b], np.abs(ref["v"][b]), t)
            assert not bad, f"{label}: row {b} active-set mismatch outside the band: {bad[:10]}"
            flips += nd
            if nd:
                if ref_all is None or w_down is None:
                    corrected = False
                else:
                    gs, os_ = set(gi.tolist()), set(ref["idx"][b].tolist())
                    for j in gs - os_:
                        y_adj[b] += ref_all["h"][b][j] * w_down[j].astype(np.float64)
                    for j in os_ - gs:
                        y_adj[b] -= ref_all["h"][b][j] * w_down[j].astype(np.float64)
            # v and h on the common active neurons
            common, gpos, opos = np.intersect1d(gi, ref["idx"][b], return_indices=True)
            if common.size:
                vo = ref["v"][b][common]
                assert np.abs(v[b, gpos] - vo).max() <= 1e-4 * max(1.0, np.abs(vo).max()), f"{label}: v"
                ho = ref["h"][b][opos]
                hs = max(float(np.abs(ho).max()), 1e-30)
                tol = h_rtol * hs
                if h_abs is not None:
                    tol = np.maximum(tol, h_abs[b][common])
                assert np.all(np.abs(h[b, gpos] - ho) <= tol), f"{label}: h"
    err = float(np.abs(y - yo).max())
    err_adj = float(np.abs(y - y_adj).max())
    if corrected:
        # same mask on both sides: the spec bar and the tight bar
        assert err_adj <= Y_TOL * max(scale, 1e-30), f"{label}: y err {err_adj} vs scale {scale}"
        assert err_adj <= Y_TIGHT * max(scale, 1e-30), f"{label}: reconciled y err {err_adj} vs scale {scale}"
    else:
        assert err <= Y_TOL * max(scale, 1e-30), f"{label}: y err {err} vs scale {scale} ({flips} band flips)"
    return {"y_err": err, "y_err_reconciled": err_adj, "y_scale": scale, "band_flips": flips}


def quantile_t(v_abs: np.ndarray, k: float) -> float:
    """A threshold at sparsity k of the given |v| values (test helper)."""
    s = np.sort(v_abs.ravel())
    r = max(1, int(np.ceil(k * s.size - 1e-6)))
    return float(np.float32(s[r - 1]))


def cfg(name):
    return W.CONFIGS[name]


def ws_for(layer: P.Layer, B: int = 1, ncal: int = 0):
    return P.workspace(layer.d, layer.m, B, ncal)
