"""CATS CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, sequential C implementation of the CATS gated MLP (Eq. 1-5 and the
"MLP using CATS" kernel algorithm of Section 4.3) and of the cutoff
calibration (Eq. 3), loaded through ctypes.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it; the product library never does, and it shares no code with it.

Two builds of the same source exist: ``f32`` (the paper runs everything in
FP32) accumulates in float, ``f64`` in double.  Both sum every dot product
in ascending index order from +0, without fused multiply-add.  ``f32_omp``
is the f32 build compiled with OpenMP: threads split independent outputs
(neurons, output columns, calibration vectors), never a sum, so it returns
the f32 build's bits on all the host's cores (a CPU baseline, not a
reference).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "cats_oracle.c")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def lib_path(precision: str = "f32") -> str:
    return os.path.join(_HERE, f"liboracle_{precision}.so")


def compile_oracle(out_path: str, source: str = SOURCE, precision: str = "f32") -> str:
    """Compile the oracle source to a shared library with gcc."""
    flags = list(CFLAGS)
    if precision == "f64":
        flags.append("-DORACLE_F64")
    elif precision == "f32_omp":
        flags.append("-fopenmp")
    elif precision != "f32":
        raise ValueError(f"unknown oracle precision {precision!r}")
    cmd = ["gcc", *flags, "-I", _HERE, "-o", out_path, source, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return out_path


def build() -> None:
    """Build both oracle precisions and the OpenMP f32 build in place."""
    for p in ("f32", "f64", "f32_omp"):
        compile_oracle(lib_path(p), precision=p)


_F = np.float32
_D = np.float64
_PF = ctypes.POINTER(ctypes.c_float)
_PD = ctypes.POINTER(ctypes.c_double)
_PI = ctypes.POINTER(ctypes.c_int32)
_PL = ctypes.POINTER(ctypes.c_int64)


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctype)


class Oracle:
    """ctypes view of one compiled oracle library."""

    def __init__(self, path: str):
        self.path = path
        L = ctypes.CDLL(path)
        L.oracle_precision.restype = ctypes.c_char_p
        L.oracle_threads.argtypes = [ctypes.c_int]
        L.oracle_threads.restype = ctypes.c_int
        L.oracle_silu.argtypes = [ctypes.c_double]
        L.oracle_silu.restype = ctypes.c_double
        L.oracle_cats_mlp.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      _PF, _PF, _PF, ctypes.c_double, ctypes.c_int32, _PF,
                                      _PD, _PI, _PI, _PD, _PD]
        L.oracle_cats_mlp.restype = ctypes.c_int
        L.oracle_rmsnorm.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_double, _PD]
        L.oracle_rmsnorm.restype = ctypes.c_int
        L.oracle_sparse_input_gemv.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _PF,
                                               ctypes.c_double, _PF, _PD, _PI, _PI]
        L.oracle_sparse_input_gemv.restype = ctypes.c_int
        L.oracle_topk_thresholds.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _PF,
                                             ctypes.c_double, _PD]
        L.oracle_topk_thresholds.restype = ctypes.c_int
        _PPF = ctypes.POINTER(_PF)
        L.oracle_stack.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                   _PPF, _PPF, _PPF, _PD, ctypes.c_int32, ctypes.c_double, _PF, _PI]
        L.oracle_stack.restype = ctypes.c_int
        L.oracle_calib_acts.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _PF, _PD]
        L.oracle_calib_acts.restype = ctypes.c_int
        L.oracle_calib_acts_at.argtypes = [_PF, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           _PF, _PL, ctypes.c_int64, _PD]
        L.oracle_calib_acts_at.restype = ctypes.c_int
        L.oracle_cutoff_rank.argtypes = [ctypes.c_int64, ctypes.c_double]
        L.oracle_cutoff_rank.restype = ctypes.c_int64
        L.oracle_threshold.argtypes = [_PD, ctypes.c_int64, ctypes.c_double, _PD]
        L.oracle_threshold.restype = ctypes.c_int
        self._L = L
        self.precision = L.oracle_precision().decode()

    def threads(self, n: int = 0) -> int:
        """Set the thread count of an OpenMP build (n > 0); returns the count
        in use (1 for a sequential build)."""
        return int(self._L.oracle_threads(int(n)))

    def silu(self, z: float) -> float:
        return float(self._L.oracle_silu(float(z)))

    def cats_mlp(self, x, w_gate, w_up, w_down, t, dense=False, residual=None):
        """Run the CATS MLP on host arrays (math layouts, see the header).

        Returns a dict with y [B,d], v [B,m], and per row the ascending active
        index list, count and the matching h = v*u values.
        """
        x = np.ascontiguousarray(x, dtype=_F)
        if x.ndim == 1:
            x = x[None, :]
        B, d = x.shape
        w_gate = np.ascontiguousarray(w_gate, dtype=_F)
        w_up = np.ascontiguousarray(w_up, dtype=_F)
        w_down = np.ascontiguousarray(w_down, dtype=_F)
        m = w_gate.shape[1]
        assert w_gate.shape == (d, m) and w_up.shape == (d, m) and w_down.shape == (m, d)
        res = None if residual is None else np.ascontiguousarray(residual, dtype=_F).reshape(B, d)
        y = np.empty((B, d), _D)
        idx = np.empty((B, m), np.int32)
        cnt = np.empty((B,), np.int32)
        v = np.empty((B, m), _D)
        h = np.empty((B, m), _D)
        rc = self._L.oracle_cats_mlp(_ptr(x, _PF), B, d, m, _ptr(w_gate, _PF), _ptr(w_up, _PF),
                                     _ptr(w_down, _PF), float(t), int(bool(dense)), _ptr(res, _PF),
                                     _ptr(y, _PD), _ptr(idx, _PI), _ptr(cnt, _PI), _ptr(v, _PD),
                                     _ptr(h, _PD))
        if rc != 0:
            raise ValueError("oracle_cats_mlp rejected its arguments")
        return {
            "y": y,
            "v": v,
            "cnt": cnt.copy(),
            "idx": [idx[b, : cnt[b]].copy() for b in range(B)],
            "h": [h[b, : cnt[b]].copy() for b in range(B)],
        }

    def rmsnorm(self, x, eps=1e-5):
        x = np.ascontiguousarray(x, dtype=_F)
        if x.ndim == 1:
            x = x[None, :]
        out = np.empty(x.shape, _D)
        if self._L.oracle_rmsnorm(_ptr(x, _PF), x.shape[0], x.shape[1], float(eps), _ptr(out, _PD)) != 0:
            raise ValueError("oracle_rmsnorm rejected its arguments")
        return out

    def topk_thresholds(self, x, w_gate, k):
        """Per-row cutoffs of the top-k variant (see the header): t [B]."""
        x = np.ascontiguousarray(x, dtype=_F)
        if x.ndim == 1:
            x = x[None, :]
        B, d = x.shape
        w_gate = np.ascontiguousarray(w_gate, dtype=_F)
        m = w_gate.shape[1]
        t = np.empty((B,), _D)
        if self._L.oracle_topk_thresholds(_ptr(x, _PF), B, d, m, _ptr(w_gate, _PF), float(k), _ptr(t, _PD)) != 0:
            raise ValueError("oracle_topk_thresholds rejected its arguments")
        return t

    def topk_mlp(self, x, w_gate, w_up, w_down, k, residual=None):
        """The top-k variant: row b runs the CATS MLP at its own cutoff
        t_b = topk_thresholds(x, w_gate, k)[b].  Returns the cats_mlp dict
        of all rows plus "t" [B]."""
        x = np.ascontiguousarray(x, dtype=_F)
        if x.ndim == 1:
            x = x[None, :]
        B = x.shape[0]
        ts = self.topk_thresholds(x, w_gate, k)
        res = None if residual is None else np.asarray(residual, dtype=_F).reshape(B, -1)
        rows = [self.cats_mlp(x[b : b + 1], w_gate, w_up, w_down, ts[b],
                              residual=None if res is None else res[b : b + 1]) for b in range(B)]
        out = {"y": np.concatenate([r["y"] for r in rows]), "v": np.concatenate([r["v"] for r in rows]),
               "cnt": np.concatenate([r["cnt"] for r in rows]), "idx": [r["idx"][0] for r in rows],
               "h": [r["h"][0] for r in rows], "t": ts}
        return out

    def sparse_input_gemv(self, x, w, t, residual=None):
        """y = residual + CATS_t(x) W for W [d, n] (see the header).

        Returns a dict with y [B, n], the ascending kept channels of every row
        and their count."""
        x = np.ascontiguousarray(x, dtype=_F)
        if x.ndim == 1:
            x = x[None, :]
        B, d = x.shape
        w = np.ascontiguousarray(w, dtype=_F)
        assert w.shape[0] == d
        n = w.shape[1]
        res = None if residual is None else np.ascontiguousarray(residual, dtype=_F).reshape(B, n)
        y = np.empty((B, n), _D)
        idx = np.empty((B, d), np.int32)
        cnt = np.empty((B,), np.int32)
        rc = self._L.oracle_sparse_input_gemv(_ptr(x, _PF), B, d, n, _ptr(w, _PF), float(t), _ptr(res, _PF),
                                              _ptr(y, _PD), _ptr(idx, _PI), _ptr(cnt, _PI))
        if rc != 0:
            raise ValueError("oracle_sparse_input_gemv rejected its arguments")
        return {"y": y, "cnt": cnt.copy(), "idx": [idx[b, : cnt[b]].copy() for b in range(B)]}

    def stack(self, x0, layers, ts=None, eps=1e-5):
        """Residual stack x_{l+1} = x_l + MLP_l(RMSNorm(x_l)) (see the header).

        layers: list of (w_gate [d, m], w_up [d, m], w_down [m, d]) host
        arrays; ts: one threshold per layer, or None for the dense stack.
        Returns (x_all [(L+1), B, d] float32, active counts [L, B])."""
        x0 = np.ascontiguousarray(x0, dtype=_F)
        if x0.ndim == 1:
            x0 = x0[None, :]
        B, d = x0.shape
        L = len(layers)
        ws = [[np.ascontiguousarray(w, dtype=_F) for w in lw] for lw in layers]
        m = ws[0][0].shape[1] if L else 1
        for wg, wu, wd in ws:
            assert wg.shape == (d, m) and wu.shape == (d, m) and wd.shape == (m, d)
        PP = _PF * max(L, 1)
        pg = PP(*[w[0].ctypes.data_as(_PF) for w in ws])
        pu = PP(*[w[1].ctypes.data_as(_PF) for w in ws])
        pd = PP(*[w[2].ctypes.data_as(_PF) for w in ws])
        dense = ts is None
        tarr = None if dense else np.ascontiguousarray(ts, dtype=np.float64)
        assert dense or tarr.shape == (L,)
        x_all = np.empty((L + 1, B, d), _F)
        cnt = np.empty((max(L, 1), B), np.int32)
        rc = self._L.oracle_stack(_ptr(x0, _PF), B, d, m, L, pg, pu, pd, _ptr(tarr, _PD), int(dense),
                                  float(eps), _ptr(x_all, _PF), _ptr(cnt, _PI))
        if rc != 0:
            raise ValueError("oracle_stack rejected its arguments")
        return x_all, cnt[:L].copy()

    def calib_acts(self, X, w_gate):
        X = np.ascontiguousarray(X, dtype=_F)
        w_gate = np.ascontiguousarray(w_gate, dtype=_F)
        N, d = X.shape
        m = w_gate.shape[1]
        out = np.empty((N, m), _D)
        if self._L.oracle_calib_acts(_ptr(X, _PF), N, d, m, _ptr(w_gate, _PF), _ptr(out, _PD)) != 0:
            raise ValueError("oracle_calib_acts rejected its arguments")
        return out

    def calib_acts_at(self, X, w_gate, pairs):
        X = np.ascontiguousarray(X, dtype=_F)
        w_gate = np.ascontiguousarray(w_gate, dtype=_F)
        pairs = np.ascontiguousarray(pairs, dtype=np.int64).reshape(-1, 2)
        N, d = X.shape
        m = w_gate.shape[1]
        out = np.empty((pairs.shape[0],), _D)
        rc = self._L.oracle_calib_acts_at(_ptr(X, _PF), N, d, m, _ptr(w_gate, _PF),
                                          _ptr(pairs, _PL), pairs.shape[0], _ptr(out, _PD))
        if rc != 0:
            raise ValueError("oracle_calib_acts_at rejected its arguments")
        return out

    def cutoff_rank(self, n: int, k: float) -> int:
        return int(self._L.oracle_cutoff_rank(int(n), float(k)))

    def threshold(self, acts, k: float) -> float:
        a = np.ascontiguousarray(np.asarray(acts, dtype=_D).ravel())
        t = ctypes.c_double()
        if self._L.oracle_threshold(_ptr(a, _PD), a.size, float(k), ctypes.byref(t)) != 0:
            raise ValueError("oracle_threshold rejected its arguments")
        return float(t.value)


_cache: dict = {}


def load(precision: str = "f32") -> Oracle:
    """Load (building first if absent) the oracle of the given precision."""
    if precision not in _cache:
        path = lib_path(precision)
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(SOURCE):
            compile_oracle(path, precision=precision)
        _cache[precision] = Oracle(path)
    return _cache[precision]
