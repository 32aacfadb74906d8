"""The C ABI library loads without a GPU, exports every entry point that
include/lstm_sd.h declares, and rejects bad arguments before touching the
device (only size queries and validation paths are called here)."""
import ctypes
import os
import re

import pytest

from paper_2106_12089_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lstm_sd.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="library not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lstm_sd_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(B.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.SIGNATURES), "binding and header disagree"


def test_version():
    assert B.lstm_sd_version() == 1


def dims(**kw):
    base = dict(num_layers=2, input_dim=650, hidden=650, batch=20, seq_len=35, num_dirs=1,
                dtype=B.DTYPE_BF16, compact=1, p_nr=0.5, p_rh=0.0)
    base.update(kw)
    return B.make_dims(**base)


def test_sizes_positive_and_monotone():
    d = dims()
    m, r, w = B.lstm_sd_mask_bytes(d), B.lstm_sd_reserve_bytes(d), B.lstm_sd_workspace_bytes(d)
    assert m > 0 and r > 0 and w > 0
    d2 = dims(seq_len=70)
    assert B.lstm_sd_reserve_bytes(d2) > r
    lay = B.lstm_sd_mask_layout_get(d)
    assert lay.sites == 2 + 2 and lay.kmax == 650 and lay.seq_len == 35
    assert lay.mask_off < lay.keep_off < lay.pos_off < lay.count_off < lay.total_bytes == m
    assert all(o % 256 == 0 for o in (lay.keep_off, lay.pos_off, lay.count_off))
    # a bidirectional model has one RH site per direction and K_in = 2H above layer 0
    lay2 = B.lstm_sd_mask_layout_get(dims(num_layers=2, num_dirs=2, hidden=256, input_dim=300))
    assert lay2.sites == 2 + 4 and lay2.kmax == 512


@pytest.mark.parametrize("kw,code", [
    (dict(num_layers=0), B.EINVAL), (dict(hidden=0), B.EINVAL), (dict(batch=-1), B.EINVAL),
    (dict(num_dirs=3), B.EINVAL), (dict(p_nr=1.0), B.EINVAL), (dict(p_rh=-0.1), B.EINVAL),
    (dict(p_nr=float("nan")), B.EINVAL), (dict(compact=2), B.EINVAL),
    (dict(dtype=7), B.EUNSUPPORTED), (dict(hidden=4096), B.EUNSUPPORTED),
    (dict(num_layers=17), B.EUNSUPPORTED), (dict(num_dirs=2, hidden=1100), B.EUNSUPPORTED),
])
def test_invalid_dims_rejected(kw, code):
    lib = B.load()
    d = dims(**kw)
    assert lib.lstm_sd_mask_bytes(ctypes.byref(d)) == 0
    assert B.lstm_sd_last_error()
    lay = B.lstm_sd_mask_layout()
    assert lib.lstm_sd_mask_layout_get(ctypes.byref(d), ctypes.byref(lay)) == code
    # device entry points validate first and return the same code
    assert lib.lstm_sd_mask_generate(ctypes.byref(d), 1, 0, None, 0, None) == code
    assert lib.lstm_sd_forward(ctypes.byref(d), None, *([None] * 5), 0, None, None, None, None, 0,
                               None, 0, None) == code


def test_null_pointers_and_small_buffers_rejected():
    lib = B.load()
    d = dims()
    assert lib.lstm_sd_mask_generate(ctypes.byref(d), 1, 0, None, 10**9, None) == B.EINVAL
    fake = 4096  # never dereferenced: size checks fail first
    assert lib.lstm_sd_mask_generate(ctypes.byref(d), 1, 0, fake, 16, None) == B.EWORKSPACE
    assert lib.lstm_sd_mask_compact(ctypes.byref(d), fake, 16, None) == B.EWORKSPACE
    assert "mask_bytes" in B.lstm_sd_last_error()
    assert lib.lstm_sd_forward(ctypes.byref(d), None, *([None] * 5), 0, None, None, None, None, 0,
                               None, 0, None) == B.EINVAL
    assert lib.lstm_sd_mse_grad(ctypes.byref(d), None, None, None, None, None, None, 0, None) == B.EINVAL
    assert lib.lstm_sd_mse_grad(ctypes.byref(d), fake, fake, None, fake, fake, fake, 8, None) == B.EWORKSPACE
    assert lib.lstm_sd_backward(ctypes.byref(d), None, *([None] * 5), 0, None, 0, *([None] * 6),
                                None, None, 0, None) == B.EINVAL
    assert lib.lstm_sd_mask_layout_get(ctypes.byref(d), None) == B.EINVAL


def test_forward_rejects_small_reserve_before_device_work():
    lib = B.load()
    d = dims(num_layers=1, input_dim=8, hidden=8, batch=2, seq_len=3)
    fake = 4096
    arr = (ctypes.c_void_p * 1)(fake)
    w = B.lstm_sd_weights(arr, arr, arr)
    mb = B.lstm_sd_mask_bytes(d)
    rc = lib.lstm_sd_forward(ctypes.byref(d), ctypes.byref(w), fake, None, fake, fake, fake, mb, fake, fake,
                             fake, fake, 1, fake, 10**9, None)
    assert rc == B.EWORKSPACE and "reserve" in B.lstm_sd_last_error()


def head_dims(**kw):
    base = dict(features=650, vocab=10000, batch=20, seq_len=35, dtype=B.DTYPE_BF16, compact=1, stream_id=8,
                p_out=0.5)
    base.update(kw)
    return B.make_head_dims(**base)


def test_head_sizes_and_layout():
    hd = head_dims()
    mb = B.lstm_sd_head_mask_bytes(hd)
    lay = B.lstm_sd_head_mask_layout_get(hd)
    assert lay.sites == 1 and lay.kmax == 650 and lay.seq_len == 35 and lay.total_bytes == mb
    assert lay.mask_off == 0 and lay.keep_off >= 35 * 650
    ws = B.lstm_sd_head_workspace_bytes(hd)
    # at least: the prepared input twice and the loss gradient twice (compute type)
    assert ws >= 2 * (35 * 20 * 650 * 2) and ws >= 35 * 10000 * 32 * 2
    assert B.lstm_sd_head_workspace_bytes(head_dims(batch=40)) > ws


@pytest.mark.parametrize("kw,code", [
    (dict(features=0), B.EINVAL), (dict(vocab=0), B.EINVAL), (dict(p_out=1.0), B.EINVAL),
    (dict(compact=3), B.EINVAL), (dict(stream_id=-1), B.EINVAL), (dict(dtype=5), B.EUNSUPPORTED),
    (dict(features=4096), B.EUNSUPPORTED), (dict(vocab=10002), B.EUNSUPPORTED),
    (dict(features=2048, vocab=600000), B.EUNSUPPORTED),
])
def test_head_invalid_dims_rejected(kw, code):
    lib = B.load()
    hd = head_dims(**kw)
    assert lib.lstm_sd_head_mask_bytes(ctypes.byref(hd)) == 0
    assert lib.lstm_sd_head_workspace_bytes(ctypes.byref(hd)) == 0
    assert lib.lstm_sd_head_mask_generate(ctypes.byref(hd), 1, 0, None, 0, None) == code
    assert lib.lstm_sd_head_forward(ctypes.byref(hd), *([None] * 4), 0, None, None, 0, None) == code
    assert lib.lstm_sd_head_backward(ctypes.byref(hd), *([None] * 4), 0, *([None] * 6), 0, None) == code


def test_head_null_pointers_and_small_buffers_rejected():
    lib = B.load()
    hd = head_dims(features=16, vocab=64, batch=2, seq_len=3)
    fake = 4096  # never dereferenced: the checks fail first
    mb = B.lstm_sd_head_mask_bytes(hd)
    ws = B.lstm_sd_head_workspace_bytes(hd)
    assert lib.lstm_sd_head_mask_generate(ctypes.byref(hd), 1, 0, fake, mb - 1, None) == B.EWORKSPACE
    assert lib.lstm_sd_head_forward(ctypes.byref(hd), fake, None, fake, fake, mb, fake, fake, ws, None) == B.EINVAL
    assert lib.lstm_sd_head_forward(ctypes.byref(hd), fake, fake, fake, fake, mb, fake, fake, ws - 1,
                                    None) == B.EWORKSPACE
    assert lib.lstm_sd_head_backward(ctypes.byref(hd), fake, fake, None, fake, mb, fake, fake, fake, fake, None,
                                     fake, ws, None) == B.EINVAL
    assert lib.lstm_sd_head_backward(ctypes.byref(hd), fake, fake, None, fake, mb - 1, fake, fake, fake, fake,
                                     fake, fake, ws, None) == B.EWORKSPACE
    assert lib.lstm_sd_head_mask_layout_get(ctypes.byref(hd), None) == B.EINVAL


def test_case1_entry_points_validate_before_device_work():
    lib = B.load()
    fake = 4096  # never dereferenced: the checks fail first
    D = ctypes.c_double
    assert lib.lstm_sd_case1_dropout(0, 2, 3, 0, fake, 0, fake, fake, 1, 0, 0, D(0.5), None) == B.EINVAL
    assert lib.lstm_sd_case1_dropout(4, 2, 3, 0, fake, 0, fake, fake, 1, 0, 0, D(1.0), None) == B.EINVAL
    assert lib.lstm_sd_case1_dropout(4, 2, 3, 0, fake, 0, fake, fake, 1, 0, -1, D(0.5), None) == B.EINVAL
    assert lib.lstm_sd_case1_dropout(4, 2, 3, 3, fake, 0, fake, fake, 1, 0, 0, D(0.5), None) == B.EUNSUPPORTED
    assert lib.lstm_sd_case1_dropout(4, 2, 3, 0, None, 0, fake, fake, 1, 0, 0, D(0.5), None) == B.EINVAL
    assert lib.lstm_sd_case1_dropout_backward(4, 2, 3, fake, None, D(0.5), fake, None) == B.EINVAL
    assert lib.lstm_sd_case1_dropout_backward(4, 2, 0, fake, fake, D(0.5), fake, None) == B.EINVAL
    assert "dimensions" in B.lstm_sd_last_error()


def test_per_layer_rates_validated():
    lib = B.load()
    good = dims(num_layers=3, p_nr=[0.4, 0.25, 0.25], p_rh=[0.5, 0.5, 0.5])
    assert B.lstm_sd_mask_bytes(good) == B.lstm_sd_mask_bytes(dims(num_layers=3))
    for bad in (dict(p_nr=[0.4, 1.0, 0.25]), dict(p_rh=[0.5, -0.1, 0.5]), dict(p_nr=[0.4, float("nan"), 0.2])):
        d = dims(num_layers=3, **bad)
        assert lib.lstm_sd_mask_bytes(ctypes.byref(d)) == 0
        assert "per-layer" in B.lstm_sd_last_error()
        assert lib.lstm_sd_mask_generate(ctypes.byref(d), 1, 0, None, 0, None) == B.EINVAL
    with pytest.raises(ValueError):
        dims(num_layers=3, p_nr=[0.4, 0.25])


def test_status_and_timeout_validate_before_device_work():
    lib = B.load()
    d = dims()
    fake = 4096  # never dereferenced: the checks fail first
    assert lib.lstm_sd_status(ctypes.byref(d), None, 10**9, None) == B.EINVAL
    assert lib.lstm_sd_status(ctypes.byref(d), fake, 16, None) == B.EWORKSPACE
    assert lib.lstm_sd_status(ctypes.byref(dims(hidden=0)), fake, 10**9, None) == B.EINVAL
    assert lib.lstm_sd_set_barrier_timeout(ctypes.c_double(float("nan"))) == B.EINVAL
    assert lib.lstm_sd_set_barrier_timeout(ctypes.c_double(-1.0)) == B.OK
