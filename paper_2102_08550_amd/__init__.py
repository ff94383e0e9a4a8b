"""Oscars local-SGD hot path on MI355X (gfx950): Python binding.

A thin ctypes layer over the C ABI declared in ``include/oscars.h``.  It only
marshals arguments (torch tensors become device pointers, the current torch
stream becomes the HIP stream); every step of the hot path runs in the HIP
library ``_lib/liboscars.so``.  If that library is missing the import of this
package fails: there is no CPU fallback.

Build with ``python paper_2102_08550_amd/build.py`` (or
``__graft_entry__.build()``).
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "liboscars.so")

OK, E_INVALID, E_NOMEM, E_HIP, E_INFEASIBLE, E_STATE = 0, -1, -2, -3, -4, -5
FP32, BF16 = 0, 1
MAX_K = 64
EVAL_NOALLOC_MAX_ROWS = 262144
(KERNEL_CAST, KERNEL_FWD, KERNEL_SOFTMAX, KERNEL_DGRAD, KERNEL_WGRAD, KERNEL_AGGREGATE,
 KERNEL_BWD_FUSED) = range(7)
KERNEL_NAMES = ("cast_bf16", "gemm_fwd", "softmax_ce", "gemm_dgrad", "gemm_wgrad_update",
                "aggregate", "gemm_bwd_fused")

_i32, _i64, _u32, _u64, _f32, _vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                     ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p)
_P = ctypes.POINTER


class OscarsError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {_lib().oscars_status_str(status).decode()} (status {status}"
                         + (f", hip error {_lib().oscars_last_hip_error()}" if status == E_HIP
                            else "") + ")")


class _Model(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("dims", _P(_i32)), ("dtype", _i32)]


class _CnnModel(ctypes.Structure):
    _fields_ = [("height", _i32), ("width", _i32), ("channels", _i32), ("n_conv", _i32),
                ("conv_channels", _P(_i32)), ("conv_strides", _P(_i32)), ("classes", _i32),
                ("conv_skip", _P(_i32))]


class _Shards(ctypes.Structure):
    _fields_ = [("x", _vp), ("y", _vp), ("n_rows", _i64), ("offsets", _P(_i64)), ("seed", _u64)]


_LIB = None

# name -> (restype, argtypes)
_SIGS = {
    "oscars_create": (_i32, [_P(_vp), _P(_Model), _i32, _i32, _vp]),
    "oscars_create_cnn": (_i32, [_P(_vp), _P(_CnnModel), _i32, _i32, _vp]),
    "oscars_destroy": (None, [_vp]),
    "oscars_set_stream": (_i32, [_vp, _vp]),
    "oscars_num_params": (_i64, [_vp]),
    "oscars_layer_offsets": (_i32, [_vp, _i32, _P(_i64), _P(_i64)]),
    "oscars_load_balance": (_i32, [_P(_i64), _i32, _i64, _P(_i64), _P(_i32)]),
    "oscars_paper_weights": (_i32, [_P(_i32), _i32, _P(_f32)]),
    "oscars_shard_offsets": (_i32, [_i64, _i32, _P(_i64)]),
    "oscars_sample_indices": (_i32, [_P(_Shards), _i32, _i32, _i64, _i32, _i32, _P(_i64)]),
    "oscars_local_steps": (_i32, [_vp, _vp, _P(_Shards), _P(_i32), _f32, _i32]),
    "oscars_round": (_i32, [_vp, _vp, _vp, _P(_Shards), _P(_i32), _f32, _i32, _P(_f32)]),
    "oscars_round_losses": (_i32, [_vp, _P(_f32)]),
    "oscars_aggregate": (_i32, [_vp, _vp, _P(_f32), _i32, _i64, _i64, _i32, _vp]),
    "oscars_get_cursors": (_i32, [_vp, _P(_i64)]),
    "oscars_set_cursors": (_i32, [_vp, _P(_i64)]),
    "oscars_profile_begin": (_i32, [_vp, _u32]),
    "oscars_profile_end": (_i32, [_vp, _P(ctypes.c_double), _P(_i64)]),
    "oscars_set_gemm_tiling": (_i32, [_vp, _i32]),
    "oscars_tuning_pending": (_i32, [_vp, _P(_i32)]),
    "oscars_set_backward": (_i32, [_vp, _i32]),
    "oscars_backward_path": (_i32, [_vp, _i32, _i32, _i32, _P(_i32)]),
    "oscars_broadcast": (_i32, [_vp, _vp, _i32, _i64, _i64, _vp]),
    "oscars_plan_tau": (_i32, [_P(ctypes.c_double), _i32, _i32, _i64, _P(_i64), _P(_i64), _P(_i32)]),
    "oscars_evaluate": (_i32, [_vp, _vp, _vp, _vp, _i64, _P(ctypes.c_double), _P(_i64)]),
    "oscars_evaluate_noalloc": (_i32, [_vp, _vp, _vp, _vp, _i64, _P(ctypes.c_double),
                                       _P(_i64)]),
    "oscars_status_str": (ctypes.c_char_p, [_i32]),
    "oscars_last_hip_error": (_i32, []),
}


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"HIP library not built: {LIB_PATH} is missing "
                              "(run python paper_2102_08550_amd/build.py)")
        # torch first: the library then binds to the HIP runtime torch has
        # loaded, so that both share one runtime (and one view of the GPU).
        import torch  # noqa: F401
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


_lib()  # fail at import time when the library is absent


def _check(status: int, what: str):
    if status != OK:
        raise OscarsError(status, what)


def _arr(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(_P(np.ctypeslib.as_ctypes_type(dtype)))


def _stream_handle(stream=None) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dev_ptr(t, dtype=None, what="tensor") -> int:
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must have dtype {dtype}, got {t.dtype}")
    return t.data_ptr()


# ---------------------------------------------------------------- host-only calls

def load_balance(t_iter: Sequence[int], M: int) -> Tuple[int, List[int]]:
    """Algorithm 1: (T*, tau) for integer iteration times t_iter and bound M."""
    t, tp = _arr(t_iter, np.int64)
    tau = np.zeros(len(t), np.int32)
    T = _i64(0)
    _check(_lib().oscars_load_balance(tp, len(t), int(M), ctypes.byref(T),
                                      tau.ctypes.data_as(_P(_i32))), "oscars_load_balance")
    return int(T.value), tau.tolist()


def plan_tau(t_measured: Sequence[float], resolution: int, M: int):
    """The controller's plan from measured iteration times: (ticks, T*, tau).
    The tick is min(t) / resolution; Algorithm 1 then runs on the ticks."""
    t = np.ascontiguousarray(t_measured, dtype=np.float64)
    ticks = np.zeros(len(t), np.int64)
    tau = np.zeros(len(t), np.int32)
    T = _i64(0)
    _check(_lib().oscars_plan_tau(t.ctypes.data_as(_P(ctypes.c_double)), len(t), int(resolution),
                                  int(M), ticks.ctypes.data_as(_P(_i64)), ctypes.byref(T),
                                  tau.ctypes.data_as(_P(_i32))), "oscars_plan_tau")
    return ticks.tolist(), int(T.value), tau.tolist()


def paper_weights(K: int, staleness: Optional[Sequence[int]] = None) -> np.ndarray:
    w = np.zeros(K, np.float32)
    st = None
    if staleness is not None:
        st, stp = _arr(staleness, np.int32)
    else:
        stp = None
    _check(_lib().oscars_paper_weights(stp, int(K), w.ctypes.data_as(_P(_f32))),
           "oscars_paper_weights")
    return w


def shard_offsets(n_rows: int, K: int) -> List[int]:
    off = np.zeros(K + 1, np.int64)
    _check(_lib().oscars_shard_offsets(int(n_rows), int(K), off.ctypes.data_as(_P(_i64))),
           "oscars_shard_offsets")
    return off.tolist()


def _shards(x_ptr, y_ptr, n_rows, offsets, seed):
    off, offp = _arr(offsets, np.int64)
    sh = _Shards(x_ptr, y_ptr, int(n_rows), offp, ctypes.c_uint64(seed & (2**64 - 1)).value)
    return sh, off  # keep `off` alive with the struct


def sample_indices(n_rows: int, offsets: Sequence[int], seed: int, k: int, first_step: int,
                   steps: int, batch: int) -> np.ndarray:
    sh, keep = _shards(None, None, n_rows, offsets, seed)
    out = np.zeros((steps, batch), np.int64)
    _check(_lib().oscars_sample_indices(ctypes.byref(sh), len(offsets) - 1, int(k),
                                        int(first_step), int(steps), int(batch),
                                        out.ctypes.data_as(_P(_i64))), "oscars_sample_indices")
    return out


# ---------------------------------------------------------------- GPU calls

# Forward / backward-data GEMM tilings (oscars_set_gemm_tiling); results are
# bit-identical for every tiling.
TILING_AUTO, TILING_L, TILING_M, TILING_S, TILING_W, TILING_WS, TILING_VS, TILING_LS = range(8)
TILINGS = {"auto": TILING_AUTO, "L": TILING_L, "M": TILING_M, "S": TILING_S, "W": TILING_W,
           "WS": TILING_WS, "VS": TILING_VS, "LS": TILING_LS}



# Backward pass of hidden bf16 layers (oscars_set_backward); results are
# bit-identical in every mode.
BACKWARD_AUTO, BACKWARD_SEPARATE, BACKWARD_FUSED, BACKWARD_FUSED_SPLIT = range(4)
BACKWARDS = {"auto": BACKWARD_AUTO, "separate": BACKWARD_SEPARATE, "fused": BACKWARD_FUSED,
             "fused_split": BACKWARD_FUSED_SPLIT}



def aggregate(global_, replicas, weights: Sequence[float], K: int, n: int, ld: int,
              broadcast: bool = False, stream=None):
    """global_[i] = pairwise-tree sum_k w_k replicas[k*ld + i]; optional broadcast."""
    import torch
    gp = _dev_ptr(global_, torch.float32, "global")
    rp = _dev_ptr(replicas, torch.float32, "replicas")
    if global_.numel() < n or replicas.numel() < (K - 1) * ld + n:
        raise ValueError("buffers smaller than K, n, ld imply")
    w, wp = _arr(weights, np.float32)
    if len(w) != K:
        raise ValueError("one weight per replica")
    _check(_lib().oscars_aggregate(gp, rp, wp, int(K), int(n), int(ld), int(bool(broadcast)),
                                   _stream_handle(stream)), "oscars_aggregate")


def broadcast(global_, replicas, K: int, n: int, ld: int, stream=None):
    """replicas[k*ld + i] = global_[i] for k < K, i < n (the step after Eq. 4's average)."""
    import torch
    gp = _dev_ptr(global_, torch.float32, "global")
    rp = _dev_ptr(replicas, torch.float32, "replicas")
    if global_.numel() < n or replicas.numel() < (K - 1) * ld + n:
        raise ValueError("buffers smaller than K, n, ld imply")
    _check(_lib().oscars_broadcast(gp, rp, int(K), int(n), int(ld), _stream_handle(stream)),
           "oscars_broadcast")


class Context:
    """K replicas of a ReLU MLP (dims = (d, h_1, ..., C)) and their workspace;
    or, with ``cnn = (image, conv)``, of the convolutional model: image =
    (H, W, C), conv = ((out channels, stride[, shortcut]), ...), dims =
    (H W C, classes), fp32 (oscars_create_cnn; shortcut: the layer adds the
    output of the layer two before it)."""

    def __init__(self, dims: Sequence[int], dtype: int, K: int, max_batch: int, stream=None,
                 cnn=None):
        self.dims = [int(v) for v in dims]
        self.dtype = int(dtype)
        self.K = int(K)
        h = _vp()
        if cnn is None:
            self._dims_arr, dp = _arr(self.dims, np.int32)
            model = _Model(len(self.dims) - 1, dp, self.dtype)
            self.shapes = [(o, i) for i, o in zip(self.dims[:-1], self.dims[1:])]
            _check(_lib().oscars_create(ctypes.byref(h), ctypes.byref(model), self.K,
                                        int(max_batch), _stream_handle(stream)), "oscars_create")
        else:
            image = [int(v) for v in cnn[0]]
            conv = [(int(c[0]), int(c[1]), int(c[2]) if len(c) > 2 else 0) for c in cnn[1]]
            if self.dtype != FP32 or len(self.dims) != 2 or len(image) != 3:
                raise ValueError("convolutional models are fp32 with dims (H W C, classes)")
            self._ch, chp = _arr([c[0] for c in conv], np.int32)
            self._st, stp = _arr([c[1] for c in conv], np.int32)
            skp = None
            if any(c[2] for c in conv):
                self._sk, skp = _arr([c[2] for c in conv], np.int32)
            model = _CnnModel(image[0], image[1], image[2], len(conv), chp, stp, self.dims[-1], skp)
            self.shapes, cin = [], image[2]
            for o, *_ in conv:
                self.shapes.append((o, 3, 3, cin))
                cin = o
            self.shapes.append((self.dims[-1], cin))
            _check(_lib().oscars_create_cnn(ctypes.byref(h), ctypes.byref(model), self.K,
                                            int(max_batch), _stream_handle(stream)),
                   "oscars_create_cnn")
        self._h = h
        self.n_pad = int(_lib().oscars_num_params(h))

    def close(self):
        if getattr(self, "_h", None):
            _lib().oscars_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_stream(self, stream=None):
        _check(_lib().oscars_set_stream(self._h, _stream_handle(stream)), "oscars_set_stream")

    def layer_offsets(self, l: int) -> Tuple[int, int]:
        w, b = _i64(0), _i64(0)
        _check(_lib().oscars_layer_offsets(self._h, int(l), ctypes.byref(w), ctypes.byref(b)),
               "oscars_layer_offsets")
        return int(w.value), int(b.value)

    def pack(self, layers) -> np.ndarray:
        """Flat padded float32 vector from [(W, b), ...] in this model's layout."""
        flat = np.zeros(self.n_pad, np.float32)
        for l, (W, b) in enumerate(layers, start=1):
            wo, bo = self.layer_offsets(l)
            flat[wo:wo + W.size] = np.asarray(W, np.float32).ravel()
            flat[bo:bo + b.size] = np.asarray(b, np.float32)
        return flat

    def unpack(self, flat: np.ndarray):
        out = []
        for l, shape in enumerate(self.shapes, start=1):
            wo, bo = self.layer_offsets(l)
            size = int(np.prod(shape))
            out.append((flat[wo:wo + size].reshape(shape), flat[bo:bo + shape[0]]))
        return out

    def _step_args(self, replicas, x, y, offsets, seed, tau):
        import torch
        rp = _dev_ptr(replicas, torch.float32, "replicas")
        if replicas.numel() < self.K * self.n_pad:
            raise ValueError("replicas must hold K * n_pad floats")
        xdt = torch.bfloat16 if self.dtype == BF16 else torch.float32
        if x.dtype == torch.int16 or x.dtype == torch.uint16:
            xdt = x.dtype  # bf16 bit patterns
        xp = _dev_ptr(x, xdt, "x")
        yp = _dev_ptr(y, torch.int32, "y")
        if x.dim() != 2 or x.shape[1] != self.dims[0] or y.numel() != x.shape[0]:
            raise ValueError("x must be [n_rows][d] and y [n_rows]")
        sh, keep = _shards(xp, yp, x.shape[0], offsets, seed)
        t, tp = _arr(tau, np.int32)
        if len(t) != self.K or len(offsets) != self.K + 1:
            raise ValueError("tau needs K entries and offsets K + 1")
        return rp, sh, (keep, t), tp

    def local_steps(self, replicas, x, y, offsets: Sequence[int], seed: int, tau: Sequence[int],
                    lr: float, batch: int):
        rp, sh, keep, tp = self._step_args(replicas, x, y, offsets, seed, tau)
        _check(_lib().oscars_local_steps(self._h, rp, ctypes.byref(sh), tp, float(lr), int(batch)),
               "oscars_local_steps")

    def round(self, global_, replicas, x, y, offsets: Sequence[int], seed: int,
              tau: Sequence[int], lr: float, batch: int, weights: Sequence[float]):
        """One round of Eq. 4 from the global model (oscars_round)."""
        import torch
        gp = _dev_ptr(global_, torch.float32, "global")
        if global_.numel() < self.n_pad:
            raise ValueError("global must hold n_pad floats")
        rp, sh, keep, tp = self._step_args(replicas, x, y, offsets, seed, tau)
        w, wp = _arr(weights, np.float32)
        if len(w) != self.K:
            raise ValueError("one weight per worker")
        _check(_lib().oscars_round(self._h, gp, rp, ctypes.byref(sh), tp, float(lr), int(batch),
                                   wp), "oscars_round")

    def round_losses(self) -> np.ndarray:
        out = np.zeros(self.K, np.float32)
        _check(_lib().oscars_round_losses(self._h, out.ctypes.data_as(_P(_f32))),
               "oscars_round_losses")
        return out

    def evaluate(self, params, x, y, n_rows: Optional[int] = None, noalloc: bool = False):
        """Held-out (summed loss, correct count) of the flat model ``params``
        (device tensor [n_pad] fp32) on rows 0..n_rows-1 of x / y
        (oscars_evaluate, or with ``noalloc`` oscars_evaluate_noalloc)."""
        import torch
        n = int(x.shape[0] if n_rows is None else n_rows)
        if n > x.shape[0] or n > y.shape[0]:
            raise ValueError("n_rows exceeds the rows of x or y")
        loss = ctypes.c_double(0.0)
        hits = _i64(0)
        name = "oscars_evaluate_noalloc" if noalloc else "oscars_evaluate"
        _check(getattr(_lib(), name)(self._h, _dev_ptr(params, torch.float32, "params"),
                                     _dev_ptr(x, None, "x"), _dev_ptr(y, torch.int32, "y"), n,
                                     ctypes.byref(loss), ctypes.byref(hits)), name)
        return float(loss.value), int(hits.value)

    def cursors(self) -> List[int]:
        out = np.zeros(self.K, np.int64)
        _check(_lib().oscars_get_cursors(self._h, out.ctypes.data_as(_P(_i64))),
               "oscars_get_cursors")
        return out.tolist()

    def set_cursors(self, steps_done: Sequence[int]):
        a, ap = _arr(steps_done, np.int64)
        _check(_lib().oscars_set_cursors(self._h, ap), "oscars_set_cursors")

    def set_gemm_tiling(self, tiling: int):
        """Tiling of this context's forward / backward-data GEMMs (AUTO: tuned
        online per configuration, fastest kept); restarts the tuning."""
        _check(_lib().oscars_set_gemm_tiling(self._h, int(tiling)), "oscars_set_gemm_tiling")

    def tuning_pending(self) -> int:
        """This context's GEMM configurations whose AUTO tiling is still being
        tuned."""
        n = ctypes.c_int32(0)
        _check(_lib().oscars_tuning_pending(self._h, ctypes.byref(n)), "oscars_tuning_pending")
        return int(n.value)

    def set_backward(self, mode: int):
        """Backward of this context's hidden bf16 layers: AUTO (timed per
        configuration), SEPARATE, FUSED, FUSED_SPLIT."""
        _check(_lib().oscars_set_backward(self._h, int(mode)), "oscars_set_backward")

    def backward_path(self, layer: int, batch: int, replicas: int) -> int:
        """Backward of `layer` (1..L) with `replicas` active replicas: 1 fused,
        0 separate launches, -1 not timed yet (AUTO)."""
        out = _i32(0)
        _check(_lib().oscars_backward_path(self._h, int(layer), int(batch), int(replicas),
                                           ctypes.byref(out)), "oscars_backward_path")
        return int(out.value)

    def profile_begin(self, kinds: Sequence[int]):
        mask = 0
        for k in kinds:
            mask |= 1 << int(k)
        _check(_lib().oscars_profile_begin(self._h, mask), "oscars_profile_begin")

    def profile_end(self):
        k = len(KERNEL_NAMES)
        ms = (ctypes.c_double * k)()
        n = (_i64 * k)()
        _check(_lib().oscars_profile_end(self._h, ms, n), "oscars_profile_end")
        return {KERNEL_NAMES[i]: (ms[i], n[i]) for i in range(k)}
