"""CPU oracle for the batch-1 decode step (ctypes wrapper over ``oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may use it; the GPU path never does.  It shares
no code with the GPU path: weights, prompt KV and tokens come in as numpy
arrays of storage bits (bf16 as uint16, int8, fp16 scales as uint16), and the
model shape from any object carrying the usual attribute names.

See ``oracle.h`` for the computed function, its precision, and the passages of
the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

LINEARS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def build(force: bool = True) -> str:
    """Compile ``liboracle.so`` with gcc (-O2, OpenMP).  No fast-math: the
    sums must run in the written order."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-fno-fast-math", "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Layer(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("ffn_norm", ctypes.c_void_p)] + \
               [(n, ctypes.c_void_p) for n in LINEARS] + \
               [("s_" + n, ctypes.c_void_p) for n in LINEARS]


class _Model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads",
                                            "head_dim", "ffn_dim", "vocab", "max_ctx", "wfmt")] + \
               [("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_double),
                ("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("s_lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(_Layer))]


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("AIO_ORACLE_LIB")  # a mutated copy, for the pin tests
        if not path:
            path = _LIB_PATH
            if not os.path.exists(path):
                build(force=False)
        L = ctypes.CDLL(path)
        vp, ci, cf = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
        L.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.orc_bf16_to_f32.restype = cf
        L.orc_f32_to_bf16.argtypes = [cf]
        L.orc_f32_to_bf16.restype = ctypes.c_uint16
        L.orc_fp16_to_f32.argtypes = [ctypes.c_uint16]
        L.orc_fp16_to_f32.restype = cf
        L.orc_rmsnorm.argtypes = [vp, vp, ci, cf, vp]
        L.orc_gemv.argtypes = [vp, vp, ci, ci, ci, vp, vp]
        L.orc_rope.argtypes = [vp, ci, ci, ctypes.c_double]
        L.orc_attention_head.argtypes = [vp, vp, vp, ci, ci, vp]
        L.orc_silu.argtypes = [ctypes.c_double]
        L.orc_silu.restype = ctypes.c_double
        L.orc_argmax.argtypes = [vp, ci]
        L.orc_argmax.restype = ci
        L.orc_decode_step.argtypes = [ctypes.POINTER(_Model), vp, ci, ci, vp]
        L.orc_decode_step_row.argtypes = [ctypes.POINTER(_Model), vp, ci, ci, vp, vp, vp]
        L.orc_verify.argtypes = [ctypes.POINTER(_Model), vp, vp, ci, ci, vp]
        L.orc_num_threads.restype = ci
        _lib = L
    return _lib


def _p(a):
    if a is None:
        return None
    assert isinstance(a, np.ndarray) and a.flags.c_contiguous, type(a)
    return a.ctypes.data


# ---------------------------------------------------------------- single ops

def rmsnorm(x: np.ndarray, g_bf16: np.ndarray, eps: float) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    g = np.ascontiguousarray(g_bf16, dtype=np.uint16)
    out = np.empty_like(x)
    lib().orc_rmsnorm(_p(x), _p(g), x.size, eps, _p(out))
    return out


def gemv(w: np.ndarray, x: np.ndarray, scale: np.ndarray | None = None) -> np.ndarray:
    """y = W x for bf16 bits (uint16) or int8 W [n_out][n_in] (+ fp16 scale)."""
    w = np.ascontiguousarray(w)
    x = np.ascontiguousarray(x, dtype=np.float32)
    n_out, n_in = w.shape
    assert x.size == n_in
    if w.dtype == np.uint16:
        fmt = 0
    elif w.dtype == np.int8:
        fmt = 1
        assert scale is not None and scale.dtype == np.uint16 and scale.size == n_out
        scale = np.ascontiguousarray(scale)
    else:
        raise TypeError(w.dtype)
    y = np.empty(n_out, dtype=np.float32)
    lib().orc_gemv(_p(w), _p(scale) if fmt else None, fmt, n_out, n_in, _p(x), _p(y))
    return y


def rope(u: np.ndarray, pos: int, base: float = 10000.0) -> np.ndarray:
    u = np.array(u, dtype=np.float32, copy=True)
    lib().orc_rope(_p(u), u.size, pos, base)
    return u


def attention_head(q: np.ndarray, k_bf16: np.ndarray, v_bf16: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k_bf16, dtype=np.uint16)
    v = np.ascontiguousarray(v_bf16, dtype=np.uint16)
    n, hd = k.shape
    out = np.empty(hd, dtype=np.float32)
    lib().orc_attention_head(_p(q), _p(k), _p(v), n, hd, _p(out))
    return out


def silu(z: float) -> float:
    return float(lib().orc_silu(z))


def argmax(x: np.ndarray) -> int:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return int(lib().orc_argmax(_p(x), x.size))


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32).ravel()
    return np.array([lib().orc_f32_to_bf16(float(v)) for v in x], dtype=np.uint16)


def num_threads() -> int:
    return int(lib().orc_num_threads())


# ------------------------------------------------------------- whole decoder

class OracleModel:
    """The decoder over host weights.  ``weights`` maps the tensor names
    ``embed``, ``final_norm``, ``lm_head`` (+ ``.scale``), and
    ``layers.{l}.{attn_norm, ffn_norm, wq, wk, wv, wo, w_gate, w_up, w_down}``
    (+ ``.scale`` for int8) to arrays of storage bits."""

    def __init__(self, cfg, weights: dict):
        self.cfg = cfg
        self._keep = []
        int8 = cfg.wfmt == "int8"

        def arr(name, dtype):
            a = weights[name]
            assert a.dtype == dtype and a.flags.c_contiguous, (name, a.dtype)
            self._keep.append(a)
            return a.ctypes.data

        wdt = np.int8 if int8 else np.uint16
        layers = (_Layer * cfg.n_layers)()
        for l in range(cfg.n_layers):
            p = "layers.%d." % l
            L = layers[l]
            L.attn_norm = arr(p + "attn_norm", np.uint16)
            L.ffn_norm = arr(p + "ffn_norm", np.uint16)
            for n in LINEARS:
                setattr(L, n, arr(p + n, wdt))
                setattr(L, "s_" + n, arr(p + n + ".scale", np.uint16) if int8 else None)
        self._layers = layers
        m = _Model()
        m.n_layers, m.d_model, m.n_heads = cfg.n_layers, cfg.d_model, cfg.n_heads
        m.n_kv_heads, m.head_dim, m.ffn_dim = cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim
        m.vocab, m.max_ctx, m.wfmt = cfg.vocab, cfg.max_ctx, 1 if int8 else 0
        m.rms_eps, m.rope_base = cfg.rms_eps, cfg.rope_base
        m.embed = arr("embed", np.uint16)
        m.final_norm = arr("final_norm", np.uint16)
        m.lm_head = arr("lm_head", wdt)
        m.s_lm_head = arr("lm_head.scale", np.uint16) if int8 else None
        m.layers = ctypes.cast(layers, ctypes.POINTER(_Layer))
        self._m = m

    def _check_kv(self, kv):
        c = self.cfg
        assert kv.dtype == np.uint16 and kv.flags.c_contiguous
        assert kv.shape == (c.n_layers, 2, c.n_kv_heads, c.max_ctx, c.head_dim), kv.shape

    def decode_step(self, kv: np.ndarray, token: int, pos: int) -> np.ndarray:
        """Consume ``token`` at ``pos`` (writes KV row pos); fp32 logits [V]."""
        self._check_kv(kv)
        logits = np.empty(self.cfg.vocab, dtype=np.float32)
        rc = lib().orc_decode_step(ctypes.byref(self._m), _p(kv), int(token), int(pos), _p(logits))
        if rc:
            raise ValueError("oracle decode_step rejected token=%d pos=%d" % (token, pos))
        return logits

    def decode_step_row(self, kv: np.ndarray, token: int, pos: int, row_in: np.ndarray):
        """decode_step with the cache entries at ``pos`` taken from ``row_in``
        (bf16 bits [n_layers][2][n_kv_heads][head_dim], any shape of that
        size) in place of the step's own roundings, layer by layer before the
        layer attends.  Returns (fp32 logits [V], the step's own row, same
        layout as ``row_in``)."""
        self._check_kv(kv)
        c = self.cfg
        rin = np.ascontiguousarray(row_in, dtype=np.uint16)
        assert rin.size == c.n_layers * 2 * c.n_kv_heads * c.head_dim, rin.shape
        own = np.empty_like(rin)
        logits = np.empty(c.vocab, dtype=np.float32)
        rc = lib().orc_decode_step_row(ctypes.byref(self._m), _p(kv), int(token), int(pos),
                                       _p(rin), _p(own), _p(logits))
        if rc:
            raise ValueError("oracle decode_step rejected token=%d pos=%d" % (token, pos))
        return logits, own

    def verify(self, kv: np.ndarray, toks, pos: int) -> np.ndarray:
        """Rows = toks at pos..pos+n-1; fp32 logits [n][V]."""
        self._check_kv(kv)
        t = np.ascontiguousarray(toks, dtype=np.int32)
        logits = np.empty((t.size, self.cfg.vocab), dtype=np.float32)
        rc = lib().orc_verify(ctypes.byref(self._m), _p(kv), _p(t), t.size, int(pos), _p(logits))
        if rc:
            raise ValueError("oracle verify rejected n=%d pos=%d" % (t.size, pos))
        return logits
