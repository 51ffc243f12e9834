"""The C ABI on the host: the library loads without a GPU, exports every
function the header declares, sizes buffers, and rejects bad arguments
before anything is enqueued (all checks here run with no device)."""
import ctypes
import os
import re

import numpy as np
import pytest

import synth
from paper_2604_09752_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aio.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        import paper_2604_09752_amd.build as b
        b.build()
    return B.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(aio_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_function(L):
    names = declared_functions()
    assert "aio_decode_step" in names and "aio_verify" in names and "aio_argmax" in names
    for n in names:
        assert hasattr(L, n), n
    # and nothing from the oracle leaks into the product library
    with open(B.LIB_PATH, "rb") as f:
        blob = f.read()
    assert b"orc_decode_step" not in blob


def cfg7b(**kw):
    return B.make_config(synth.CONFIGS["7b"].with_(**kw))


def test_sizes(L):
    c = cfg7b()
    assert B.aio_kv_bytes(c) == 32 * 2 * 32 * c.max_ctx * 128 * 2
    ws = B.aio_workspace_bytes(c)
    assert 0 < ws < 64 << 20
    c1 = B.make_config(synth.CONFIGS["1b"])
    assert B.aio_kv_bytes(c1) == 24 * 2 * 8 * c1.max_ctx * 128 * 2


@pytest.mark.parametrize("field,value,code", [
    ("n_layers", 0, B.AIO_EINVAL),
    ("d_model", 100, B.AIO_EINVAL),
    ("n_kv_heads", 3, B.AIO_EINVAL),        # 32 % 3 != 0
    ("n_kv_heads", 2, B.AIO_EUNSUPPORTED),  # G = 16
    ("head_dim", 96, B.AIO_EUNSUPPORTED),
    ("ffn_dim", 1000, B.AIO_EINVAL),
    ("vocab", 0, B.AIO_EINVAL),
    ("max_ctx", 0, B.AIO_EINVAL),
    ("max_verify", 0, B.AIO_EINVAL),
    ("max_verify", 11, B.AIO_EINVAL),
    ("wfmt", 7, B.AIO_EINVAL),
    ("rms_eps", 0.0, B.AIO_EINVAL),
    ("rope_base", float("nan"), B.AIO_EINVAL),
])
def test_config_rejections(L, field, value, code):
    c = cfg7b()
    assert B.aio_check_config(c) == B.AIO_OK
    setattr(c, field, value)
    assert B.aio_check_config(c) == code
    assert B.aio_kv_bytes(c) == 0 and B.aio_workspace_bytes(c) == 0


def test_null_config(L):
    assert L.aio_check_config(None) == B.AIO_EINVAL
    assert L.aio_kv_bytes(None) == 0


def test_decode_ranges(L):
    c = cfg7b()
    assert B.aio_check_decode(c, 0, 0) == B.AIO_OK
    assert B.aio_check_decode(c, c.vocab - 1, c.max_ctx - 1) == B.AIO_OK
    for tok, pos in ((-1, 0), (c.vocab, 0), (0, -1), (0, c.max_ctx)):
        assert B.aio_check_decode(c, tok, pos) == B.AIO_ERANGE


def test_verify_ranges(L):
    c = cfg7b()
    d8 = np.arange(8, dtype=np.int32)
    assert B.aio_check_verify(c, 1, d8, 8, 100) == B.AIO_OK
    assert B.aio_check_verify(c, 1, None, 0, 100) == B.AIO_OK          # k = 0: one row
    assert B.aio_check_verify(c, 1, None, 2, 100) == B.AIO_EINVAL      # drafts missing
    assert B.aio_check_verify(c, 1, np.arange(10, dtype=np.int32), 10, 0) == B.AIO_ERANGE
    assert B.aio_check_verify(c, 1, d8, -1, 0) == B.AIO_ERANGE
    assert B.aio_check_verify(c, 1, d8, 8, c.max_ctx - 8) == B.AIO_ERANGE  # pos + k == max_ctx
    assert B.aio_check_verify(c, 1, d8, 8, c.max_ctx - 9) == B.AIO_OK
    bad = d8.copy()
    bad[5] = c.vocab
    assert B.aio_check_verify(c, 1, bad, 8, 0) == B.AIO_ERANGE
    assert B.aio_check_verify(c, -1, d8, 8, 0) == B.AIO_ERANGE


def test_strerror(L):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert B.aio_strerror(code)
    assert B.aio_strerror(-99) == "unknown error"


def test_entry_points_reject_before_any_device_call(L):
    vp = ctypes.c_void_p
    # null handle / pointers are rejected on the host
    assert L.aio_decode_step(None, 0, 0, vp(16)) == B.AIO_EINVAL
    assert L.aio_verify(None, 0, None, 0, 0, vp(16)) == B.AIO_EINVAL
    assert L.aio_argmax(None, vp(16), 1, 1, vp(16)) == B.AIO_EINVAL
    labels = (ctypes.c_int32 * 2)(0, 1)
    assert L.aio_category_entropy(None, vp(16), labels, 2, vp(16)) == B.AIO_EINVAL
    assert L.aio_decode_greedy(None, 0, 0, 1, vp(16), vp(16)) == B.AIO_EINVAL
    out = (ctypes.c_int32 * 4)()
    assert L.aio_pld_generate(None, None, 0, 0, 4, 3, 1, 2, vp(16), vp(16), out,
                              None) == B.AIO_EINVAL
    h = vp()
    c = cfg7b()
    w = B.aio_weights()
    assert L.aio_model_load(ctypes.byref(c), ctypes.byref(w), vp(256), vp(256), None,
                            ctypes.byref(h)) == B.AIO_EINVAL  # null weight pointers
    assert L.aio_model_load(None, ctypes.byref(w), vp(256), vp(256), None,
                            ctypes.byref(h)) == B.AIO_EINVAL
    # misaligned weight pointer
    layers = (B.aio_layer_weights * c.n_layers)()
    for l in range(c.n_layers):
        for n in ("attn_norm", "ffn_norm") + B.LINEARS:
            setattr(layers[l], n, 4096)
    w.embed, w.final_norm, w.lm_head = 4096, 4096, 4096 + 8
    w.layers = ctypes.cast(layers, ctypes.POINTER(B.aio_layer_weights))
    assert L.aio_model_load(ctypes.byref(c), ctypes.byref(w), vp(256), vp(256), None,
                            ctypes.byref(h)) == B.AIO_EINVAL
    # bf16 weights must not carry scales
    w.lm_head = 4096
    w.s_lm_head = 4096
    assert L.aio_model_load(ctypes.byref(c), ctypes.byref(w), vp(256), vp(256), None,
                            ctypes.byref(h)) == B.AIO_EINVAL
    # misaligned workspace
    w.s_lm_head = None
    assert L.aio_model_load(ctypes.byref(c), ctypes.byref(w), vp(256), vp(272), None,
                            ctypes.byref(h)) == B.AIO_EINVAL
