"""ctypes binding of libcats (the C ABI declared in include/cats.h).

Argument marshalling only: every function passes device pointers of torch
tensors and the current HIP stream to the library, which does all the work
in its own kernels.  torch supplies device memory and streams.  There is no
fallback: if libcats.so is missing the import fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

# torch is imported first so that libcats binds to the HIP runtime torch
# already loaded (both carry the soname libamdhip64.so.7); loading libcats
# first would pull in a second runtime.
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcats.so")

CATS_F32 = 0
CATS_BF16 = 1
# size of the fixed scratch array behind cats_mlp_forward_noalloc
NOALLOC_SCRATCH_BYTES = 32 << 20
STATUS_NAMES = {
    0: "CATS_OK", 1: "CATS_ERR_NULL", 2: "CATS_ERR_SHAPE", 3: "CATS_ERR_RANGE",
    4: "CATS_ERR_DTYPE", 5: "CATS_ERR_ALIGN", 6: "CATS_ERR_WORKSPACE", 7: "CATS_ERR_HIP",
    8: "CATS_ERR_UNIMPLEMENTED",
}


class CatsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class _Layer(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("m", ctypes.c_int32), ("wdtype", ctypes.c_int32),
                ("w_gate_t", ctypes.c_void_p), ("w_up_t", ctypes.c_void_p),
                ("w_down", ctypes.c_void_p)]


class _Aux(ctypes.Structure):
    _fields_ = [("active_idx", ctypes.c_void_p), ("active_cnt", ctypes.c_void_p),
                ("active_v", ctypes.c_void_p), ("active_h", ctypes.c_void_p)]


_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t
_f32 = ctypes.c_float
_f64 = ctypes.c_double

_SIGNATURES = {
    "cats_version": ([], _i32),
    "cats_status_string": ([_i32], ctypes.c_char_p),
    "cats_last_error": ([], ctypes.c_char_p),
    "cats_workspace_bytes": ([_i32, _i32, _i32, _i64], _sz),
    "cats_pack_weights": ([_vp, _vp, _i32, _i32, _i32, _vp], _i32),
    "cats_calib_activations": ([ctypes.POINTER(_Layer), _vp, _i32, _vp, _vp], _i32),
    "cats_threshold_from_acts": ([_vp, _i64, _f64, _vp, _sz, _vp, ctypes.POINTER(_f32)], _i32),
    "cats_calibrate_threshold": ([ctypes.POINTER(_Layer), _vp, _i32, _f64, _vp, _sz, _vp,
                                  ctypes.POINTER(_f32)], _i32),
    "cats_mlp_forward": ([ctypes.POINTER(_Layer), _vp, _i32, _f32, _vp, _vp, ctypes.POINTER(_Aux),
                          _vp, _sz, _vp], _i32),
    "cats_mlp_forward_noalloc": ([ctypes.POINTER(_Layer), _vp, _i32, _f32, _vp, _vp, ctypes.POINTER(_Aux), _vp],
                                 _i32),
    "cats_mlp_dense": ([ctypes.POINTER(_Layer), _vp, _i32, _vp, _vp, _vp, _sz, _vp], _i32),
    "cats_stack_forward": ([ctypes.POINTER(_Layer), _i32, ctypes.POINTER(_f32), _vp, _i32, _f32, _vp,
                            _vp, ctypes.POINTER(_Aux), _vp, _sz, _vp], _i32),
    "cats_calibrate_stack_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "cats_calibrate_stack": ([ctypes.POINTER(_Layer), _i32, _vp, _i32, _f64, _f32, _vp, _sz, _vp,
                              ctypes.POINTER(_f32)], _i32),
    "cats_sparse_input_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "cats_sparse_input_gemv": ([_vp, _i32, _i32, _i32, _vp, _i32, _f32, _vp, _vp, ctypes.POINTER(_Aux), _vp,
                                _sz, _vp], _i32),
    "cats_topk_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "cats_mlp_forward_topk": ([ctypes.POINTER(_Layer), _vp, _i32, _f64, _vp, _vp, ctypes.POINTER(_Aux), _vp, _sz,
                               _vp, _vp], _i32),
    "cats_unfused_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "cats_mlp_forward_unfused": ([ctypes.POINTER(_Layer), _vp, _i32, _f32, _i32, _vp, _vp, _vp, _sz, _vp], _i32),
    "cats_rmsnorm": ([_vp, _vp, _i32, _i32, _f32, _vp], _i32),
    "cats_stream_read": ([_vp, _sz, _i32, _i32, _i32, _vp, _vp], _i32),
    "cats_timer_enable": ([_i32], _i32),
    "cats_timer_reset": ([], _i32),
    "cats_timer_count": ([], _i32),
    "cats_timer_get": ([_i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_i64),
                        ctypes.POINTER(_f64)], _i32),
}

_lib: Optional[ctypes.CDLL] = None


def lib_path() -> str:
    return _LIB_PATH


def raw() -> ctypes.CDLL:
    """The loaded libcats handle (signatures set).  Raises if not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"libcats.so is not built ({_LIB_PATH}); run "
                              "`python -m paper_2404_08763_amd.build` first")
        L = ctypes.CDLL(_LIB_PATH, mode=ctypes.RTLD_GLOBAL)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        msg = raw().cats_last_error().decode(errors="replace")
        raise CatsError(status, msg)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, name: str, dtype=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _wdtype(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return CATS_BF16
    if dt == torch.float32:
        return CATS_F32
    raise ValueError(f"unsupported weight dtype {dt}")


@dataclass
class Layer:
    """One gated-MLP block in neuron-major layout (all [m, d] device tensors)."""
    w_gate_t: torch.Tensor
    w_up_t: torch.Tensor
    w_down: torch.Tensor

    def __post_init__(self):
        m, d = self.w_gate_t.shape
        for n, w in (("w_gate_t", self.w_gate_t), ("w_up_t", self.w_up_t), ("w_down", self.w_down)):
            _dev(w, n, self.w_gate_t.dtype)
            if tuple(w.shape) != (m, d):
                raise ValueError(f"{n} has shape {tuple(w.shape)}, expected {(m, d)}")
        self._c = _Layer(d, m, _wdtype(self.w_gate_t.dtype), self.w_gate_t.data_ptr(),
                         self.w_up_t.data_ptr(), self.w_down.data_ptr())

    @property
    def d(self) -> int:
        return int(self.w_gate_t.shape[1])

    @property
    def m(self) -> int:
        return int(self.w_gate_t.shape[0])

    @property
    def c(self):
        return ctypes.byref(self._c)


def version() -> int:
    return int(raw().cats_version())


def workspace_bytes(d: int, m: int, max_batch: int = 1, max_calib_values: int = 0) -> int:
    return int(raw().cats_workspace_bytes(d, m, max_batch, max_calib_values))


def workspace(d: int, m: int, max_batch: int = 1, max_calib_values: int = 0, device="cuda") -> torch.Tensor:
    """A zero-filled device byte buffer of cats_workspace_bytes(...) bytes."""
    n = workspace_bytes(d, m, max_batch, max_calib_values)
    if n == 0:
        raise ValueError("arguments outside the supported range")
    ws = torch.zeros(n, dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def pack_weights(w: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """[rows, cols] -> [cols, rows] transpose on the device (bit-exact)."""
    _dev(w, "w")
    rows, cols = w.shape
    if out is None:
        out = torch.empty((cols, rows), dtype=w.dtype, device=w.device)
    _dev(out, "out", w.dtype)
    _check(raw().cats_pack_weights(_ptr(w), _ptr(out), rows, cols, _wdtype(w.dtype), _stream()))
    return out


def layer_from_math(w_gate: torch.Tensor, w_up: torch.Tensor, w_down: torch.Tensor) -> Layer:
    """Build a Layer from math-layout weights (W_gate, W_up [d, m]; W_down [m, d])."""
    return Layer(pack_weights(w_gate), pack_weights(w_up), w_down.contiguous())


def calib_activations(layer: Layer, x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    N = _rows_of(x, layer.d)
    _numel_is(out, N * layer.m, "out")
    _dev(x, "x", torch.float32)
    if out is None:
        out = torch.empty((N, layer.m), dtype=torch.float32, device=x.device)
    _dev(out, "out", torch.float32)
    _numel_is(out, N * layer.m, "out")
    _check(raw().cats_calib_activations(layer.c, _ptr(x), N, _ptr(out), _stream()))
    return out


def threshold_from_acts(acts: torch.Tensor, sparsity: float, ws: Optional[torch.Tensor] = None) -> float:
    _dev(acts, "acts", torch.float32)
    if ws is None:
        ws = torch.empty(4096, dtype=torch.uint8, device=acts.device)
    t = _f32()
    _check(raw().cats_threshold_from_acts(_ptr(acts), acts.numel(), float(sparsity), _ptr(ws),
                                          ws.numel(), _stream(), ctypes.byref(t)))
    return float(t.value)


def calibrate_threshold(layer: Layer, calib_x: torch.Tensor, sparsity: float,
                        ws: Optional[torch.Tensor] = None) -> float:
    N = _rows_of(calib_x, layer.d, "calib_x")
    _dev(calib_x, "calib_x", torch.float32)
    if ws is None:
        ws = workspace(layer.d, layer.m, 1, N * layer.m, device=calib_x.device)
    t = _f32()
    _check(raw().cats_calibrate_threshold(layer.c, _ptr(calib_x), N, float(sparsity), _ptr(ws),
                                          ws.numel(), _stream(), ctypes.byref(t)))
    return float(t.value)


def _rows(x: torch.Tensor) -> int:
    return 1 if x.dim() == 1 else int(x.shape[0])


def _rows_of(x: torch.Tensor, d: int, name: str = "x") -> int:
    """Rows of a [B, d] (or [d]) activation tensor; raises before any call
    into the library when its width is not the layer's d, since the kernels
    read and write B * d floats through raw pointers."""
    if x.dim() not in (1, 2):
        raise ValueError(f"{name} must be [d] or [B, d], got shape {tuple(x.shape)}")
    if int(x.shape[-1]) != d:
        raise ValueError(f"{name} has width {int(x.shape[-1])}, the layer has d={d}")
    return _rows(x)


def _numel_is(t: Optional[torch.Tensor], n: int, name: str) -> None:
    if t is not None and t.numel() != n:
        raise ValueError(f"{name} must hold {n} elements, has {t.numel()}")


def _io_checks(x: torch.Tensor, d: int, out: Optional[torch.Tensor], residual: Optional[torch.Tensor],
               n_out: Optional[int] = None) -> int:
    """Validate x, out and residual of a [B, d] -> [B, n_out] call; returns B.
    Shapes are checked first, so a mismatch raises whatever the device."""
    B = _rows_of(x, d)
    n_out = d if n_out is None else n_out
    _numel_is(out, B * n_out, "out")
    _numel_is(residual, B * n_out, "residual")
    _dev(x, "x", torch.float32)
    if out is not None:
        _dev(out, "out", torch.float32)
    if residual is not None:
        _dev(residual, "residual", torch.float32)
    return B


def mlp_forward(layer: Layer, x: torch.Tensor, t: float, residual: Optional[torch.Tensor] = None,
                out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                aux: bool = False):
    """CATS MLP forward.  Returns y, or (y, aux dict) when aux=True.

    The aux dict holds per row b: idx[b, :cnt[b]] (ascending active neurons),
    v and h (= v * x.W_up[:, j]) aligned with idx, and cnt.
    """
    B = _io_checks(x, layer.d, out, residual)
    if out is None:
        out = torch.empty_like(x)
    if ws is None:
        ws = workspace(layer.d, layer.m, B, device=x.device)
    aux_c = None
    bufs = None
    if aux:
        m = layer.m
        bufs = {
            "idx": torch.empty((B, m), dtype=torch.int32, device=x.device),
            "cnt": torch.empty((B,), dtype=torch.int32, device=x.device),
            "v": torch.empty((B, m), dtype=torch.float32, device=x.device),
            "h": torch.empty((B, m), dtype=torch.float32, device=x.device),
        }
        aux_c = _Aux(bufs["idx"].data_ptr(), bufs["cnt"].data_ptr(), bufs["v"].data_ptr(),
                     bufs["h"].data_ptr())
    _check(raw().cats_mlp_forward(layer.c, _ptr(x), B, float(t), _ptr(residual), _ptr(out),
                                  ctypes.byref(aux_c) if aux_c is not None else None, _ptr(ws),
                                  ws.numel(), _stream()))
    if aux:
        return out, bufs
    return out


CATS_UNFUSED_MASK = 0
CATS_UNFUSED_INDEX = 1
_UNFUSED_MODES = {"mask": CATS_UNFUSED_MASK, "index": CATS_UNFUSED_INDEX}


def mlp_forward_unfused(layer: Layer, x: torch.Tensor, t: float, mode: str = "mask",
                        residual: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The forward in separate gate / up / down kernels; mode "mask" or "index"."""
    B = _io_checks(x, layer.d, out, residual)
    if mode not in _UNFUSED_MODES:
        raise ValueError(f"mode must be one of {sorted(_UNFUSED_MODES)}")
    if out is None:
        out = torch.empty_like(x)
    if ws is None:
        nbytes = int(raw().cats_unfused_workspace_bytes(layer.d, layer.m, B))
        if nbytes == 0:
            raise ValueError("arguments outside the supported range")
        ws = torch.zeros(nbytes, dtype=torch.uint8, device=x.device)
    _check(raw().cats_mlp_forward_unfused(layer.c, _ptr(x), B, float(t), _UNFUSED_MODES[mode], _ptr(residual),
                                          _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out


def mlp_forward_topk(layer: Layer, x: torch.Tensor, sparsity: float, residual: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, aux: bool = False):
    """Per-token top-k variant.  Returns (y, t [B]) or (y, t, aux dict)."""
    B = _io_checks(x, layer.d, out, residual)
    if out is None:
        out = torch.empty_like(x)
    if ws is None:
        nbytes = int(raw().cats_topk_workspace_bytes(layer.d, layer.m, B))
        if nbytes == 0:
            raise ValueError("arguments outside the supported range")
        ws = torch.zeros(nbytes, dtype=torch.uint8, device=x.device)
    t = torch.empty((B,), dtype=torch.float32, device=x.device)
    aux_c = None
    bufs = None
    if aux:
        m = layer.m
        bufs = {
            "idx": torch.empty((B, m), dtype=torch.int32, device=x.device),
            "cnt": torch.empty((B,), dtype=torch.int32, device=x.device),
            "v": torch.empty((B, m), dtype=torch.float32, device=x.device),
            "h": torch.empty((B, m), dtype=torch.float32, device=x.device),
        }
        aux_c = _Aux(bufs["idx"].data_ptr(), bufs["cnt"].data_ptr(), bufs["v"].data_ptr(), bufs["h"].data_ptr())
    _check(raw().cats_mlp_forward_topk(layer.c, _ptr(x), B, float(sparsity), _ptr(residual), _ptr(out),
                                       ctypes.byref(aux_c) if aux_c is not None else None, _ptr(ws), ws.numel(),
                                       _stream(), _ptr(t)))
    if aux:
        return out, t, bufs
    return out, t


def mlp_dense(layer: Layer, x: torch.Tensor, residual: Optional[torch.Tensor] = None,
              out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    B = _io_checks(x, layer.d, out, residual)
    if out is None:
        out = torch.empty_like(x)
    if ws is None:
        ws = workspace(layer.d, layer.m, B, device=x.device)
    _check(raw().cats_mlp_dense(layer.c, _ptr(x), B, _ptr(residual), _ptr(out), _ptr(ws), ws.numel(),
                                _stream()))
    return out


class Stack:
    """L blocks with one d, marshalled once for repeated stack calls.

    t: one threshold per layer, or None for the dense stack."""

    def __init__(self, layers, t=None):
        self.layers = list(layers)
        L = len(self.layers)
        if L == 0:
            raise ValueError("a stack needs at least one layer")
        self.d = self.layers[0].d
        self.max_m = max(l.m for l in self.layers)
        self._arr = (_Layer * L)(*[l._c for l in self.layers])
        self._t = None
        if t is not None:
            if len(t) != L:
                raise ValueError(f"{len(t)} thresholds for {L} layers")
            self._t = (_f32 * L)(*[float(v) for v in t])

    def __len__(self):
        return len(self.layers)


def stack_forward(stack: Stack, x0: torch.Tensor, eps: float = 1e-5, out: Optional[torch.Tensor] = None,
                  ws: Optional[torch.Tensor] = None, keep_all: bool = False, aux: bool = False):
    """x_{l+1} = x_l + MLP_l(RMSNorm(x_l)) over the stack's layers.

    Returns x_L, or a dict with "out", "x_all" [(L+1), B, d] (keep_all) and
    "aux" (a list of per-layer dicts as from mlp_forward, when aux=True)."""
    B = _rows_of(x0, stack.d, "x0")
    _numel_is(out, B * stack.d, "out")
    _dev(x0, "x0", torch.float32)
    L = len(stack)
    if out is None:
        out = torch.empty_like(x0)
    _dev(out, "out", torch.float32)
    if ws is None:
        ws = workspace(stack.d, stack.max_m, B, device=x0.device)
    x_all = torch.empty((L + 1,) + tuple(x0.shape), dtype=torch.float32, device=x0.device) if keep_all else None
    aux_bufs = None
    aux_c = None
    if aux:
        aux_bufs, cs = [], []
        for l in stack.layers:
            m = l.m
            b = {
                "idx": torch.empty((B, m), dtype=torch.int32, device=x0.device),
                "cnt": torch.empty((B,), dtype=torch.int32, device=x0.device),
                "v": torch.empty((B, m), dtype=torch.float32, device=x0.device),
                "h": torch.empty((B, m), dtype=torch.float32, device=x0.device),
            }
            aux_bufs.append(b)
            cs.append(_Aux(b["idx"].data_ptr(), b["cnt"].data_ptr(), b["v"].data_ptr(), b["h"].data_ptr()))
        aux_c = (_Aux * L)(*cs)
    _check(raw().cats_stack_forward(stack._arr, L, stack._t, _ptr(x0), B, float(eps), _ptr(out),
                                    _ptr(x_all), aux_c, _ptr(ws), ws.numel(), _stream()))
    if not keep_all and not aux:
        return out
    return {"out": out, "x_all": x_all, "aux": aux_bufs}


def calibrate_stack(stack: Stack, calib_x: torch.Tensor, sparsity: float, eps: float = 1e-5,
                    ws: Optional[torch.Tensor] = None) -> list:
    """Per-layer thresholds of a stack, the calibration vectors propagated
    densely through the earlier layers (cats_calibrate_stack)."""
    N = _rows_of(calib_x, stack.d, "calib_x")
    _dev(calib_x, "calib_x", torch.float32)
    L = len(stack)
    if ws is None:
        n = int(raw().cats_calibrate_stack_workspace_bytes(stack.d, stack.max_m, N))
        if n == 0:
            raise ValueError("arguments outside the supported range")
        ws = torch.zeros(n, dtype=torch.uint8, device=calib_x.device)
    t = (_f32 * L)()
    _check(raw().cats_calibrate_stack(stack._arr, L, _ptr(calib_x), N, float(sparsity), float(eps),
                                      _ptr(ws), ws.numel(), _stream(), t))
    return [float(v) for v in t]


def sparse_input_workspace(d: int, n: int, max_batch: int = 1, device="cuda") -> torch.Tensor:
    nbytes = int(raw().cats_sparse_input_workspace_bytes(d, n, max_batch))
    if nbytes == 0:
        raise ValueError("arguments outside the supported range")
    return torch.zeros(nbytes, dtype=torch.uint8, device=device)


def sparse_input_gemv(w: torch.Tensor, x: torch.Tensor, t: float, residual: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, aux: bool = False):
    """y = residual + CATS_t(x) W for W [d, n] (channel-major, bf16).

    Returns y, or (y, aux dict) with per row the ascending kept channels
    idx[b, :cnt[b]] and their values v (= h)."""
    if w.dim() != 2:
        raise ValueError(f"w must be [d, n], got shape {tuple(w.shape)}")
    d, n = int(w.shape[0]), int(w.shape[1])
    B = _io_checks(x, d, out, residual, n_out=n)
    _dev(w, "w", torch.bfloat16)
    if out is None:
        out = torch.empty((B, n), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = sparse_input_workspace(d, n, B, device=x.device)
    aux_c = None
    bufs = None
    if aux:
        bufs = {
            "idx": torch.empty((B, d), dtype=torch.int32, device=x.device),
            "cnt": torch.empty((B,), dtype=torch.int32, device=x.device),
            "v": torch.empty((B, d), dtype=torch.float32, device=x.device),
            "h": torch.empty((B, d), dtype=torch.float32, device=x.device),
        }
        aux_c = _Aux(bufs["idx"].data_ptr(), bufs["cnt"].data_ptr(), bufs["v"].data_ptr(), bufs["h"].data_ptr())
    _check(raw().cats_sparse_input_gemv(_ptr(w), d, n, CATS_BF16, _ptr(x), B, float(t), _ptr(residual),
                                        _ptr(out), ctypes.byref(aux_c) if aux_c is not None else None,
                                        _ptr(ws), ws.numel(), _stream()))
    if aux:
        return out, bufs
    return out


def rmsnorm(x: torch.Tensor, eps: float = 1e-5, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    _dev(x, "x", torch.float32)
    if x.dim() not in (1, 2):
        raise ValueError(f"x must be [d] or [B, d], got shape {tuple(x.shape)}")
    if out is None:
        out = torch.empty_like(x)
    _dev(out, "out", torch.float32)
    _numel_is(out, x.numel(), "out")
    B = _rows(x)
    d = int(x.shape[-1])
    _check(raw().cats_rmsnorm(_ptr(x), _ptr(out), B, d, float(eps), _stream()))
    return out


def stream_read(buf: torch.Tensor, blocks: int, inflight: int = 8, runs: bool = False,
                sink: Optional[torch.Tensor] = None) -> None:
    """Enqueue one plain read of a device tensor's bytes (attainable-bandwidth
    probe; time it with timer_* under the name "stream_read")."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    if sink is None:
        sink = torch.empty(blocks, dtype=torch.int32, device=buf.device)
    _check(raw().cats_stream_read(_ptr(buf), buf.numel() * buf.element_size(), int(blocks), int(inflight),
                                  1 if runs else 0, _ptr(sink), _stream()))


def timer_enable(on: bool = True) -> None:
    _check(raw().cats_timer_enable(1 if on else 0))


def timer_reset() -> None:
    _check(raw().cats_timer_reset())


def timer_read() -> dict:
    """{kernel name: (launches, total ms)} for the kernels timed so far."""
    L = raw()
    out = {}
    for i in range(int(L.cats_timer_count())):
        name = ctypes.c_char_p()
        n = _i64()
        ms = _f64()
        _check(L.cats_timer_get(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
        out[name.value.decode()] = (int(n.value), float(ms.value))
    return out
