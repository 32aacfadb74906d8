"""ctypes binding of liblstm_sd.so (C ABI in include/lstm_sd.h).

Argument marshalling only: every step of the computation runs in the
library's HIP kernels.  Functions keep the C names; device buffers are passed
as torch tensors (their data pointers are handed to the library) and the
stream defaults to torch's current stream.  A missing library raises: there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

from . import build as _build

LIB_PATH = _build.LIB

OK, EINVAL, EUNSUPPORTED, EHIP, EWORKSPACE = 0, -1, -2, -3, -4
DTYPE_F32, DTYPE_BF16 = 0, 1
MAX_K = 2048


class lstm_sd_dims(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("input_dim", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("seq_len", ctypes.c_int32), ("num_dirs", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("compact", ctypes.c_int32),
                ("p_nr", ctypes.c_double), ("p_rh", ctypes.c_double),
                ("p_nr_layer", ctypes.POINTER(ctypes.c_double)),
                ("p_rh_layer", ctypes.POINTER(ctypes.c_double))]


class lstm_sd_weights(ctypes.Structure):
    _fields_ = [("W", ctypes.POINTER(ctypes.c_void_p)), ("U", ctypes.POINTER(ctypes.c_void_p)),
                ("b", ctypes.POINTER(ctypes.c_void_p))]


class lstm_sd_grads(ctypes.Structure):
    _fields_ = [("dW", ctypes.POINTER(ctypes.c_void_p)), ("dU", ctypes.POINTER(ctypes.c_void_p)),
                ("db", ctypes.POINTER(ctypes.c_void_p))]


class lstm_sd_mask_layout(ctypes.Structure):
    _fields_ = [("sites", ctypes.c_int32), ("kmax", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("mask_off", ctypes.c_size_t),
                ("keep_off", ctypes.c_size_t), ("pos_off", ctypes.c_size_t),
                ("count_off", ctypes.c_size_t), ("drop_off", ctypes.c_size_t),
                ("dcount_off", ctypes.c_size_t), ("kseg_off", ctypes.c_size_t),
                ("dseg_off", ctypes.c_size_t), ("total_bytes", ctypes.c_size_t)]


class lstm_sd_head_dims(ctypes.Structure):
    _fields_ = [("features", ctypes.c_int32), ("vocab", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("seq_len", ctypes.c_int32), ("dtype", ctypes.c_int32), ("compact", ctypes.c_int32),
                ("stream_id", ctypes.c_int32), ("reserved", ctypes.c_int32), ("p_out", ctypes.c_double)]


_P = ctypes.c_void_p
_SZ = ctypes.c_size_t
_DIMS = ctypes.POINTER(lstm_sd_dims)
_HD = ctypes.POINTER(lstm_sd_head_dims)

# name -> (restype, argtypes); the header's declarations
SIGNATURES = {
    "lstm_sd_version": (ctypes.c_int, []),
    "lstm_sd_last_error": (ctypes.c_char_p, []),
    "lstm_sd_mask_bytes": (_SZ, [_DIMS]),
    "lstm_sd_reserve_bytes": (_SZ, [_DIMS]),
    "lstm_sd_workspace_bytes": (_SZ, [_DIMS]),
    "lstm_sd_mask_layout_get": (ctypes.c_int, [_DIMS, ctypes.POINTER(lstm_sd_mask_layout)]),
    "lstm_sd_mask_generate": (ctypes.c_int, [_DIMS, ctypes.c_uint64, ctypes.c_uint64, _P, _SZ, _P]),
    "lstm_sd_mask_compact": (ctypes.c_int, [_DIMS, _P, _SZ, _P]),
    "lstm_sd_mask_generate_fixed": (ctypes.c_int, [_DIMS, ctypes.c_uint64, ctypes.c_uint64, _P, _SZ, _P]),
    "lstm_sd_forward": (ctypes.c_int, [_DIMS, ctypes.POINTER(lstm_sd_weights), _P, _P, _P, _P, _P, _SZ,
                                       _P, _P, _P, _P, _SZ, _P, _SZ, _P]),
    "lstm_sd_backward": (ctypes.c_int, [_DIMS, ctypes.POINTER(lstm_sd_weights), _P, _P, _P, _P, _P, _SZ,
                                        _P, _SZ, _P, _P, _P, _P, _P, _P, ctypes.POINTER(lstm_sd_grads),
                                        _P, _SZ, _P]),
    "lstm_sd_mse_grad": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "lstm_sd_embedding_backward": (ctypes.c_int, [_DIMS, _P, ctypes.c_int, _P, _P, _SZ, _P, _P]),
    "lstm_sd_case1_dropout": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P,
                                             ctypes.c_int32, _P, _P, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                             ctypes.c_double, _P]),
    "lstm_sd_case1_dropout_backward": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P,
                                                      ctypes.c_double, _P, _P]),
    "lstm_sd_head_mask_bytes": (_SZ, [_HD]),
    "lstm_sd_head_workspace_bytes": (_SZ, [_HD]),
    "lstm_sd_head_mask_layout_get": (ctypes.c_int, [_HD, ctypes.POINTER(lstm_sd_mask_layout)]),
    "lstm_sd_head_mask_generate": (ctypes.c_int, [_HD, ctypes.c_uint64, ctypes.c_uint64, _P, _SZ, _P]),
    "lstm_sd_head_forward": (ctypes.c_int, [_HD, _P, _P, _P, _P, _SZ, _P, _P, _SZ, _P]),
    "lstm_sd_head_backward": (ctypes.c_int, [_HD, _P, _P, _P, _P, _SZ, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "lstm_sd_forward_static": (ctypes.c_int, [_DIMS, ctypes.POINTER(lstm_sd_weights), _P, _P, _P, _P, _P, _SZ,
                                              _P, _P, _P, _P, _SZ, _P]),
    "lstm_sd_status": (ctypes.c_int, [_DIMS, _P, _SZ, _P]),
    "lstm_sd_set_barrier_timeout": (ctypes.c_int, [ctypes.c_double]),
    "lstm_sd_kernel_timer_start": (ctypes.c_int, [ctypes.c_char_p]),
    "lstm_sd_kernel_timer_stop": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2106_12089_amd.build.build() "
                           "(no fallback implementation exists)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class LstmSdError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"lstm_sd error {code}: {msg}")
        self.code = code


def _check(rc):
    if rc != OK:
        raise LstmSdError(rc, load().lstm_sd_last_error().decode())
    return rc


def _rates(p, num_layers):
    """A scalar rate, or a per-layer sequence as a ctypes double array (the
    structure's pointer field keeps it alive)."""
    if isinstance(p, (list, tuple)):
        if len(p) != num_layers:
            raise ValueError(f"{len(p)} per-layer rates for {num_layers} layers")
        return float(p[0]), (ctypes.c_double * num_layers)(*[float(v) for v in p])
    return float(p), None


def make_dims(num_layers, input_dim, hidden, batch, seq_len, num_dirs=1, dtype=DTYPE_BF16,
              compact=1, p_nr=0.0, p_rh=0.0) -> lstm_sd_dims:
    """p_nr / p_rh: one rate for every layer, or a list of L rates."""
    nr, nr_arr = _rates(p_nr, num_layers)
    rh, rh_arr = _rates(p_rh, num_layers)
    d = lstm_sd_dims(num_layers, input_dim, hidden, batch, seq_len, num_dirs, dtype, compact, nr, rh)
    if nr_arr is not None:
        d.p_nr_layer = ctypes.cast(nr_arr, ctypes.POINTER(ctypes.c_double))
        d._keep_nr = nr_arr
    if rh_arr is not None:
        d.p_rh_layer = ctypes.cast(rh_arr, ctypes.POINTER(ctypes.c_double))
        d._keep_rh = rh_arr
    return d


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _ptr_array(ts):
    arr = (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])
    return arr


# --- size queries -----------------------------------------------------------
def lstm_sd_version() -> int:
    return load().lstm_sd_version()


def lstm_sd_last_error() -> str:
    return load().lstm_sd_last_error().decode()


def lstm_sd_mask_bytes(dims) -> int:
    n = load().lstm_sd_mask_bytes(ctypes.byref(dims))
    if n == 0:
        raise LstmSdError(EINVAL, lstm_sd_last_error())
    return n


def lstm_sd_reserve_bytes(dims) -> int:
    n = load().lstm_sd_reserve_bytes(ctypes.byref(dims))
    if n == 0:
        raise LstmSdError(EINVAL, lstm_sd_last_error())
    return n


def lstm_sd_workspace_bytes(dims) -> int:
    n = load().lstm_sd_workspace_bytes(ctypes.byref(dims))
    if n == 0:
        raise LstmSdError(EINVAL, lstm_sd_last_error())
    return n


def lstm_sd_mask_layout_get(dims) -> lstm_sd_mask_layout:
    out = lstm_sd_mask_layout()
    _check(load().lstm_sd_mask_layout_get(ctypes.byref(dims), ctypes.byref(out)))
    return out


# --- device calls -------------------------------------------------------------
def lstm_sd_mask_generate(dims, seed, step, mask_buf, stream=None):
    _check(load().lstm_sd_mask_generate(ctypes.byref(dims), ctypes.c_uint64(seed & (2**64 - 1)),
                                        ctypes.c_uint64(step), _ptr(mask_buf),
                                        mask_buf.numel() * mask_buf.element_size(), _stream(stream)))


def lstm_sd_mask_generate_fixed(dims, seed, step, mask_buf, stream=None):
    _check(load().lstm_sd_mask_generate_fixed(ctypes.byref(dims), ctypes.c_uint64(seed & (2**64 - 1)),
                                              ctypes.c_uint64(step), _ptr(mask_buf), _nbytes(mask_buf),
                                              _stream(stream)))


def lstm_sd_mask_compact(dims, mask_buf, stream=None):
    _check(load().lstm_sd_mask_compact(ctypes.byref(dims), _ptr(mask_buf),
                                       mask_buf.numel() * mask_buf.element_size(), _stream(stream)))


def _nbytes(t):
    return t.numel() * t.element_size()


def lstm_sd_forward(dims, W, U, b, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, workspace,
                    stream=None):
    keep = (_ptr_array(W), _ptr_array(U), _ptr_array(b))
    w = lstm_sd_weights(keep[0], keep[1], keep[2])
    _check(load().lstm_sd_forward(ctypes.byref(dims), ctypes.byref(w), _ptr(x), _ptr(lengths), _ptr(h0),
                                  _ptr(c0), _ptr(mask_buf), _nbytes(mask_buf), _ptr(y), _ptr(hT), _ptr(cT),
                                  _ptr(reserve), _nbytes(reserve), _ptr(workspace), _nbytes(workspace),
                                  _stream(stream)))


def lstm_sd_backward(dims, W, U, b, x, lengths, h0, c0, mask_buf, reserve, dy, dhT, dcT, dx, dh0, dc0,
                     dW, dU, db, workspace, stream=None):
    keep = (_ptr_array(W), _ptr_array(U), _ptr_array(b), _ptr_array(dW), _ptr_array(dU), _ptr_array(db))
    w = lstm_sd_weights(keep[0], keep[1], keep[2])
    g = lstm_sd_grads(keep[3], keep[4], keep[5])
    _check(load().lstm_sd_backward(ctypes.byref(dims), ctypes.byref(w), _ptr(x), _ptr(lengths), _ptr(h0),
                                   _ptr(c0), _ptr(mask_buf), _nbytes(mask_buf), _ptr(reserve),
                                   _nbytes(reserve), _ptr(dy), _ptr(dhT), _ptr(dcT), _ptr(dx), _ptr(dh0),
                                   _ptr(dc0), ctypes.byref(g), _ptr(workspace), _nbytes(workspace),
                                   _stream(stream)))


def lstm_sd_mse_grad(dims, y, target, lengths, dy, loss, workspace, stream=None):
    _check(load().lstm_sd_mse_grad(ctypes.byref(dims), _ptr(y), _ptr(target), _ptr(lengths), _ptr(dy),
                                   _ptr(loss), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def lstm_sd_embedding_backward(dims, tokens, vocab, dx, mask_buf, d_emb, stream=None):
    _check(load().lstm_sd_embedding_backward(ctypes.byref(dims), _ptr(tokens), int(vocab), _ptr(dx), _ptr(mask_buf),
                                             _nbytes(mask_buf), _ptr(d_emb), _stream(stream)))


def lstm_sd_case1_dropout(T, B, K, src_dtype, src, dst_dtype, dst, mask, seed, step, stream_id, p, stream=None):
    _check(load().lstm_sd_case1_dropout(T, B, K, src_dtype, _ptr(src), dst_dtype, _ptr(dst), _ptr(mask),
                                        ctypes.c_uint64(seed & (2**64 - 1)), ctypes.c_uint64(step), stream_id,
                                        float(p), _stream(stream)))


def lstm_sd_case1_dropout_backward(T, B, K, dx, mask, p, dsrc, stream=None):
    _check(load().lstm_sd_case1_dropout_backward(T, B, K, _ptr(dx), _ptr(mask), float(p), _ptr(dsrc),
                                                 _stream(stream)))


def make_head_dims(features, vocab, batch, seq_len, dtype=DTYPE_BF16, compact=1, stream_id=0,
                   p_out=0.0) -> lstm_sd_head_dims:
    return lstm_sd_head_dims(features, vocab, batch, seq_len, dtype, compact, stream_id, 0, float(p_out))


def lstm_sd_head_mask_bytes(hd) -> int:
    n = load().lstm_sd_head_mask_bytes(ctypes.byref(hd))
    if n == 0:
        raise LstmSdError(EINVAL, lstm_sd_last_error())
    return n


def lstm_sd_head_workspace_bytes(hd) -> int:
    n = load().lstm_sd_head_workspace_bytes(ctypes.byref(hd))
    if n == 0:
        raise LstmSdError(EINVAL, lstm_sd_last_error())
    return n


def lstm_sd_head_mask_layout_get(hd) -> lstm_sd_mask_layout:
    out = lstm_sd_mask_layout()
    _check(load().lstm_sd_head_mask_layout_get(ctypes.byref(hd), ctypes.byref(out)))
    return out


def lstm_sd_head_mask_generate(hd, seed, step, mask_buf, stream=None):
    _check(load().lstm_sd_head_mask_generate(ctypes.byref(hd), ctypes.c_uint64(seed & (2**64 - 1)),
                                             ctypes.c_uint64(step), _ptr(mask_buf), _nbytes(mask_buf),
                                             _stream(stream)))


def lstm_sd_head_forward(hd, W_fc, b_fc, y, mask_buf, logits, workspace, stream=None):
    _check(load().lstm_sd_head_forward(ctypes.byref(hd), _ptr(W_fc), _ptr(b_fc), _ptr(y), _ptr(mask_buf),
                                       _nbytes(mask_buf), _ptr(logits), _ptr(workspace), _nbytes(workspace),
                                       _stream(stream)))


def lstm_sd_head_backward(hd, W_fc, targets, lengths, mask_buf, logits, loss, dy, dW_fc, db_fc, workspace,
                          stream=None):
    _check(load().lstm_sd_head_backward(ctypes.byref(hd), _ptr(W_fc), _ptr(targets), _ptr(lengths),
                                        _ptr(mask_buf), _nbytes(mask_buf), _ptr(logits), _ptr(loss), _ptr(dy),
                                        _ptr(dW_fc), _ptr(db_fc), _ptr(workspace), _nbytes(workspace),
                                        _stream(stream)))


STATIC_WORKSPACE_MAX = 64 << 20


def lstm_sd_forward_static(dims, W, U, b, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, stream=None):
    """lstm_sd_forward with the library's own workspace (allocates nothing)."""
    keep = (_ptr_array(W), _ptr_array(U), _ptr_array(b))
    w = lstm_sd_weights(keep[0], keep[1], keep[2])
    _check(load().lstm_sd_forward_static(ctypes.byref(dims), ctypes.byref(w), _ptr(x), _ptr(lengths), _ptr(h0),
                                         _ptr(c0), _ptr(mask_buf), _nbytes(mask_buf), _ptr(y), _ptr(hT), _ptr(cT),
                                         _ptr(reserve), _nbytes(reserve), _stream(stream)))


def lstm_sd_status(dims, workspace, stream=None):
    """Waits for the stream; raises LstmSdError (EHIP) if a grid barrier of
    the step last run on this workspace timed out."""
    _check(load().lstm_sd_status(ctypes.byref(dims), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def lstm_sd_set_barrier_timeout(seconds: float):
    """Process-wide bound of a grid-barrier wait; < 0 restores the default,
    0 makes every wait fail at once (tests of the failure path)."""
    _check(load().lstm_sd_set_barrier_timeout(float(seconds)))


def lstm_sd_kernel_timer_start(kernel: str):
    _check(load().lstm_sd_kernel_timer_start(kernel.encode()))


def lstm_sd_kernel_timer_stop():
    """Returns (total milliseconds, number of launches)."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(load().lstm_sd_kernel_timer_stop(ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
