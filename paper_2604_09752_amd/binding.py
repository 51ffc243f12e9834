"""ctypes binding of ``libaio.so`` (C ABI in ``include/aio.h``).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of ``libaio.so``.  Torch provides device memory and streams.  If the
library is missing this module raises instead of computing anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libaio.so")

AIO_OK, AIO_EINVAL, AIO_ERANGE, AIO_EUNSUPPORTED, AIO_EHIP, AIO_ENOMEM, AIO_EDEVICE = \
    0, -1, -2, -3, -4, -5, -6
AIO_WFMT_BF16, AIO_WFMT_INT8 = 0, 1
AIO_MAX_VERIFY_ROWS = 10
LINEARS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")
SCALES = ("sq", "sk", "sv", "so", "s_gate", "s_up", "s_down")


class aio_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads",
                                              "head_dim", "ffn_dim", "vocab", "max_ctx",
                                              "max_verify", "wfmt")] + \
               [("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


class aio_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "ffn_norm") + LINEARS + SCALES]


class aio_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("s_lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(aio_layer_weights))]


class aio_pld_stats(ctypes.Structure):
    _fields_ = [("forwards", ctypes.c_int32), ("verifies", ctypes.c_int32),
                ("drafted", ctypes.c_int32), ("accepted", ctypes.c_int32)]


class aio_spec_stats(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_int32), ("drafted", ctypes.c_int32),
                ("accepted", ctypes.c_int32), ("draft_steps", ctypes.c_int32)]


class AioError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__("%s failed: %d (%s)%s" % (
            what, code, aio_strerror(code),
            "" if code != AIO_EHIP else ", hipError %d" % aio_last_hip_error()))


_lib = None


def lib():
    """The loaded library; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libaio.so is not built (run python -m paper_2604_09752_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        P = ctypes.POINTER
        L.aio_kv_bytes.argtypes = [P(aio_config)]
        L.aio_kv_bytes.restype = ctypes.c_size_t
        L.aio_workspace_bytes.argtypes = [P(aio_config)]
        L.aio_workspace_bytes.restype = ctypes.c_size_t
        L.aio_check_config.argtypes = [P(aio_config)]
        L.aio_check_decode.argtypes = [P(aio_config), i32, i32]
        L.aio_check_verify.argtypes = [P(aio_config), i32, vp, i32, i32]
        L.aio_strerror.argtypes = [ctypes.c_int]
        L.aio_strerror.restype = ctypes.c_char_p
        L.aio_last_hip_error.restype = ctypes.c_int
        L.aio_model_load.argtypes = [P(aio_config), P(aio_weights), vp, vp, vp, P(vp)]
        L.aio_model_free.argtypes = [vp]
        L.aio_model_free.restype = None
        L.aio_decode_step.argtypes = [vp, i32, i32, vp]
        L.aio_verify.argtypes = [vp, i32, vp, i32, i32, vp]
        L.aio_argmax.argtypes = [vp, vp, i32, i32, vp]
        L.aio_decode_greedy.argtypes = [vp, i32, i32, i32, vp, vp]
        L.aio_profile_step.argtypes = [vp, i32, i32, vp, vp, i32, P(i32)]
        L.aio_trace_step.argtypes = [vp, i32, i32, vp, vp, i32, P(i32)]
        L.aio_device_status.argtypes = [vp, P(i32)]
        L.aio_trace_barriers.argtypes = [vp, i32, i32, vp, vp, vp, i32, P(i32), P(i32)]
        L.aio_uses_step_kernel.argtypes = [vp]
        L.aio_pld_match.argtypes = [vp, i32, i32, i32, i32, vp, P(i32)]
        L.aio_pld_generate.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, vp,
                                       P(aio_pld_stats)]
        L.aio_tune_step.argtypes = [vp, i32, i32, vp, i32]
        L.aio_prefill.argtypes = [vp, vp, i32, i32, vp]
        L.aio_prefill_noalloc.argtypes = [vp, vp, i32, i32, vp]
        L.aio_prefill_noalloc_rows.argtypes = [P(aio_config)]
        L.aio_category_entropy.argtypes = [vp, vp, vp, i32, vp]
        L.aio_category_entropy.restype = i32
        L.aio_probe_route.argtypes = [vp, i32, i32, i32, i32, ctypes.c_float,
                                      P(ctypes.c_float), P(i32)]
        L.aio_spec_generate.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                        P(aio_spec_stats)]
        _lib = L
    return _lib


def make_config(cfg) -> aio_config:
    """aio_config from any object with the usual shape attributes."""
    c = aio_config()
    for n in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab",
              "max_ctx", "max_verify"):
        setattr(c, n, int(getattr(cfg, n)))
    if c.max_verify > AIO_MAX_VERIFY_ROWS:
        c.max_verify = AIO_MAX_VERIFY_ROWS
    c.wfmt = AIO_WFMT_INT8 if getattr(cfg, "wfmt", "bf16") == "int8" else AIO_WFMT_BF16
    c.rms_eps = float(cfg.rms_eps)
    c.rope_base = float(cfg.rope_base)
    return c


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _check(rc: int, what: str):
    if rc != AIO_OK:
        raise AioError(rc, what)


# ------------------------------------------------------------- pure host calls

def aio_kv_bytes(c: aio_config) -> int:
    return int(lib().aio_kv_bytes(ctypes.byref(c)))


def aio_workspace_bytes(c: aio_config) -> int:
    return int(lib().aio_workspace_bytes(ctypes.byref(c)))


def aio_check_config(c: aio_config) -> int:
    return int(lib().aio_check_config(ctypes.byref(c) if c is not None else None))


def aio_check_decode(c: aio_config, token: int, pos: int) -> int:
    return int(lib().aio_check_decode(ctypes.byref(c), token, pos))


def aio_check_verify(c: aio_config, token: int, drafts, k: int, pos: int) -> int:
    arr = None if drafts is None else np.ascontiguousarray(drafts, dtype=np.int32)
    return int(lib().aio_check_verify(ctypes.byref(c), token,
                                      None if arr is None else arr.ctypes.data, k, pos))


def aio_strerror(code: int) -> str:
    return lib().aio_strerror(code).decode()


def aio_last_hip_error() -> int:
    return int(lib().aio_last_hip_error())


# ------------------------------------------------------------ model handles

def aio_model_load(c: aio_config, w: aio_weights, kv: torch.Tensor, ws: torch.Tensor,
                   stream: int | None) -> int:
    h = ctypes.c_void_p()
    _check(lib().aio_model_load(ctypes.byref(c), ctypes.byref(w), _ptr(kv), _ptr(ws), stream,
                                ctypes.byref(h)), "aio_model_load")
    return h.value


def aio_model_free(handle: int) -> None:
    lib().aio_model_free(handle)


def aio_decode_step(handle: int, token: int, pos: int, logits: torch.Tensor) -> None:
    _check(lib().aio_decode_step(handle, int(token), int(pos), _ptr(logits)), "aio_decode_step")


def aio_verify(handle: int, token: int, drafts, k: int, pos: int, logits: torch.Tensor) -> None:
    arr = np.ascontiguousarray(drafts if drafts is not None else [], dtype=np.int32)
    _check(lib().aio_verify(handle, int(token), arr.ctypes.data if arr.size else None, int(k),
                            int(pos), _ptr(logits)), "aio_verify")


def aio_argmax(handle: int, logits: torch.Tensor, rows: int, n: int, out: torch.Tensor) -> None:
    _check(lib().aio_argmax(handle, _ptr(logits), int(rows), int(n), _ptr(out)), "aio_argmax")


def aio_decode_greedy(handle: int, token: int, pos: int, n_steps: int, tokens: torch.Tensor,
                      logits: torch.Tensor) -> None:
    _check(lib().aio_decode_greedy(handle, int(token), int(pos), int(n_steps), _ptr(tokens),
                                   _ptr(logits)), "aio_decode_greedy")


KERNELS_PER_LAYER = ("qkv", "attn", "merge", "o", "gateup", "down")


def aio_profile_step(handle: int, token: int, pos: int, logits: torch.Tensor,
                     max_kernels: int) -> np.ndarray:
    """Per-kernel event-to-event milliseconds of one decode step."""
    ms = np.zeros(max_kernels, dtype=np.float32)
    n = ctypes.c_int32(0)
    _check(lib().aio_profile_step(handle, int(token), int(pos), _ptr(logits), ms.ctypes.data,
                                  int(max_kernels), ctypes.byref(n)), "aio_profile_step")
    return ms[: n.value].copy()


def aio_trace_step(handle: int, token: int, pos: int, logits: torch.Tensor,
                   max_phases: int) -> np.ndarray:
    """Per-phase microseconds of one step of the persistent kernel."""
    us = np.zeros(max_phases, dtype=np.float64)
    n = ctypes.c_int32(0)
    _check(lib().aio_trace_step(handle, int(token), int(pos), _ptr(logits), us.ctypes.data,
                                int(max_phases), ctypes.byref(n)), "aio_trace_step")
    return us[: n.value].copy()


def aio_trace_barriers(handle: int, token: int, pos: int, logits: torch.Tensor, n_layers: int,
                       max_blocks: int = 1024):
    """(arrive, leave) device-clock times [barrier][workgroup] of one step."""
    cap = (5 * n_layers + 1) * max_blocks
    arr = np.zeros(cap, dtype=np.uint64)
    lev = np.zeros(cap, dtype=np.uint64)
    nb, nk = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().aio_trace_barriers(handle, int(token), int(pos), _ptr(logits), arr.ctypes.data,
                                    lev.ctypes.data, cap, ctypes.byref(nb), ctypes.byref(nk)),
           "aio_trace_barriers")
    n = nb.value * nk.value
    return arr[:n].reshape(nb.value, nk.value), lev[:n].reshape(nb.value, nk.value)


def aio_pld_match(hist, ngram_max: int, ngram_min: int, k: int) -> np.ndarray:
    """Prompt-lookup drafts for the history ``hist`` (pure host call)."""
    h = np.ascontiguousarray(hist, dtype=np.int32)
    out = np.zeros(max(int(k), 1), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib().aio_pld_match(h.ctypes.data if h.size else None, int(h.size), int(ngram_max),
                               int(ngram_min), int(k), out.ctypes.data, ctypes.byref(n)),
           "aio_pld_match")
    return out[: n.value].copy()


def aio_pld_generate(handle: int, history, pos: int, token: int, n_new: int, ngram_max: int,
                     ngram_min: int, k: int, logits: torch.Tensor, argmax_out: torch.Tensor):
    """Greedy generation with prompt-lookup decoding; returns (tokens, stats)."""
    h = np.ascontiguousarray(history, dtype=np.int32)
    assert h.size == pos
    out = np.zeros(int(n_new), dtype=np.int32)
    st = aio_pld_stats()
    _check(lib().aio_pld_generate(handle, h.ctypes.data if h.size else None, int(pos), int(token),
                                  int(n_new), int(ngram_max), int(ngram_min), int(k),
                                  _ptr(logits), _ptr(argmax_out), out.ctypes.data,
                                  ctypes.byref(st)), "aio_pld_generate")
    return out, {f: int(getattr(st, f)) for f, _ in aio_pld_stats._fields_}


def aio_spec_generate(target: int, draft: int, pos: int, token: int, n_new: int, k: int,
                      target_logits: torch.Tensor, draft_logits: torch.Tensor,
                      argmax_out: torch.Tensor, draft_tokens: torch.Tensor):
    """Greedy generation of the target with drafts from the draft model;
    returns (tokens, stats)."""
    out = np.zeros(int(n_new), dtype=np.int32)
    st = aio_spec_stats()
    _check(lib().aio_spec_generate(target, draft, int(pos), int(token), int(n_new), int(k),
                                   _ptr(target_logits), _ptr(draft_logits), _ptr(argmax_out),
                                   _ptr(draft_tokens), out.ctypes.data, ctypes.byref(st)),
           "aio_spec_generate")
    return out, {f: int(getattr(st, f)) for f, _ in aio_spec_stats._fields_}


def spec_generate(target: "DeviceModel", draft: "DeviceModel", pos: int, token: int, n_new: int,
                  k: int):
    """Draft-model speculative generation over two resident models (synchronous)."""
    tl = target.new_logits(k + 1)
    dl = draft.new_logits(1)
    am = torch.zeros(k + 1, dtype=torch.int32, device=target.device)
    dt = torch.zeros(max(k, 1), dtype=torch.int32, device=draft.device)
    return aio_spec_generate(target.handle, draft.handle, pos, token, n_new, k, tl, dl, am, dt)


def aio_probe_route(category_logits, code_category: int, ctx_len: int, ctx_limit: int = 2048,
                    tau: float = 0.45):
    """(route to the small model?, entropy in nats, category) of the probe."""
    x = np.ascontiguousarray(category_logits, dtype=np.float32)
    h, cat = ctypes.c_float(0.0), ctypes.c_int32(-1)
    rc = lib().aio_probe_route(x.ctypes.data, int(x.size), int(code_category), int(ctx_len),
                               int(ctx_limit), float(tau), ctypes.byref(h), ctypes.byref(cat))
    if rc < 0:
        raise AioError(rc, "aio_probe_route")
    return bool(rc), float(h.value), int(cat.value)


def aio_category_entropy(handle: int, logits: torch.Tensor, label_ids, out: torch.Tensor) -> None:
    """Enqueue H(X) and the category of the label tokens' logits into out[0:2]
    (device fp32)."""
    ids = np.ascontiguousarray(label_ids, dtype=np.int32)
    _check(lib().aio_category_entropy(handle, _ptr(logits), ids.ctypes.data, int(ids.size),
                                      _ptr(out)), "aio_category_entropy")


def aio_device_status(handle: int) -> int:
    st = ctypes.c_int32(0)
    _check(lib().aio_device_status(handle, ctypes.byref(st)), "aio_device_status")
    return int(st.value)


def aio_uses_step_kernel(handle: int) -> bool:
    return bool(lib().aio_uses_step_kernel(handle))


# ------------------------------------------------------------------ a model

def _to_device(a: np.ndarray, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).to(device)
        return t.view(torch.bfloat16)
    if a.dtype == np.int8:
        return torch.from_numpy(a).to(device)
    raise TypeError(a.dtype)


class DeviceModel:
    """Weights, KV cache and workspace in device memory plus a loaded handle.

    ``weights`` maps tensor names (``embed``, ``final_norm``, ``lm_head``,
    ``layers.{l}.{attn_norm, ffn_norm, wq, ...}``, ``*.scale``) to numpy
    arrays of storage bits; they are copied to the device once."""

    def __init__(self, cfg, weights: dict, kv_init: np.ndarray | None = None,
                 device: str = "cuda:0", stream: torch.cuda.Stream | None = None):
        self.cfg = cfg
        self.c = make_config(cfg)
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.Stream(device=self.device)
        int8 = self.c.wfmt == AIO_WFMT_INT8
        self.dev = {k: _to_device(v, self.device) for k, v in weights.items()}
        kvb, wsb = aio_kv_bytes(self.c), aio_workspace_bytes(self.c)
        if kvb == 0 or wsb == 0:
            raise AioError(aio_check_config(self.c), "config")
        if kv_init is not None:
            assert kv_init.nbytes == kvb and kv_init.dtype == np.uint16
            self.kv = _to_device(np.ascontiguousarray(kv_init).reshape(-1), self.device)
        else:
            self.kv = torch.zeros(kvb // 2, dtype=torch.bfloat16, device=self.device)
        self.ws = torch.zeros(wsb, dtype=torch.uint8, device=self.device)
        layers = (aio_layer_weights * self.c.n_layers)()
        for l in range(self.c.n_layers):
            p = "layers.%d." % l
            L = layers[l]
            L.attn_norm = _ptr(self.dev[p + "attn_norm"])
            L.ffn_norm = _ptr(self.dev[p + "ffn_norm"])
            for n, s in zip(LINEARS, SCALES):
                setattr(L, n, _ptr(self.dev[p + n]))
                setattr(L, s, _ptr(self.dev[p + n + ".scale"]) if int8 else None)
        self._layers = layers
        w = aio_weights()
        w.embed = _ptr(self.dev["embed"])
        w.final_norm = _ptr(self.dev["final_norm"])
        w.lm_head = _ptr(self.dev["lm_head"])
        w.s_lm_head = _ptr(self.dev["lm_head.scale"]) if int8 else None
        w.layers = ctypes.cast(layers, ctypes.POINTER(aio_layer_weights))
        self._w = w
        torch.cuda.synchronize(self.device)
        self.handle = aio_model_load(self.c, w, self.kv, self.ws, self.stream.cuda_stream)

    def kv_numpy(self) -> np.ndarray:
        """The device KV cache as uint16 bf16 bits in the oracle's layout."""
        c = self.c
        t = self.kv.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.reshape(c.n_layers, 2, c.n_kv_heads, c.max_ctx, c.head_dim)

    def kv_rows(self, lo: int, hi: int) -> np.ndarray:
        """Cache positions [lo, hi) as uint16 bf16 bits, [layer, K/V, kv head,
        position, head_dim] (only those rows cross to the host)."""
        c = self.c
        t = self.kv.view(torch.int16).view(c.n_layers, 2, c.n_kv_heads, c.max_ctx, c.head_dim)
        return t[:, :, :, lo:hi, :].cpu().numpy().view(np.uint16)

    def new_logits(self, rows: int = 1) -> torch.Tensor:
        return torch.empty((rows, self.c.vocab), dtype=torch.float32, device=self.device)

    def decode_step(self, token: int, pos: int, logits: torch.Tensor) -> None:
        aio_decode_step(self.handle, token, pos, logits)

    def verify(self, token: int, drafts, pos: int, logits: torch.Tensor) -> None:
        aio_verify(self.handle, token, drafts, len(drafts), pos, logits)

    def argmax(self, logits: torch.Tensor, rows: int, out: torch.Tensor) -> None:
        aio_argmax(self.handle, logits, rows, logits.shape[-1], out)

    def greedy(self, token: int, pos: int, n_steps: int, tokens: torch.Tensor,
               logits: torch.Tensor) -> None:
        aio_decode_greedy(self.handle, token, pos, n_steps, tokens, logits)

    def pld_generate(self, history, pos: int, token: int, n_new: int, ngram_max: int,
                     ngram_min: int, k: int):
        """Prompt-lookup greedy generation of n_new tokens (synchronous)."""
        logits = self.new_logits(k + 1)
        am = torch.zeros(k + 1, dtype=torch.int32, device=self.device)
        return aio_pld_generate(self.handle, history, pos, token, n_new, ngram_max, ngram_min, k,
                                logits, am)

    def prefill(self, tokens, pos: int, logits: torch.Tensor) -> None:
        """Consume tokens at pos.. in prompt-length matrix products; logits
        (fp32, at least [vocab]) receives the last token's logits."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        _check(lib().aio_prefill(self.handle, t.ctypes.data, int(t.size), int(pos), _ptr(logits)),
               "aio_prefill")

    def prefill_noalloc(self, tokens, pos: int, logits: torch.Tensor) -> None:
        """aio_prefill with the scratch in the library's fixed device array
        (no device allocation)."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        _check(lib().aio_prefill_noalloc(self.handle, t.ctypes.data, int(t.size), int(pos),
                                         _ptr(logits)), "aio_prefill_noalloc")

    @property
    def prefill_noalloc_rows(self) -> int:
        return int(lib().aio_prefill_noalloc_rows(ctypes.byref(self.c)))

    def tune(self, token: int, pos: int, logits: torch.Tensor, rounds: int = 4) -> None:
        """Calibrate the persistent kernel's gate/up split (aio_tune_step)."""
        _check(lib().aio_tune_step(self.handle, int(token), int(pos), _ptr(logits), int(rounds)),
               "aio_tune_step")

    def profile_step(self, token: int, pos: int, logits: torch.Tensor) -> np.ndarray:
        return aio_profile_step(self.handle, token, pos, logits, 6 * self.c.n_layers + 1)

    def trace_step(self, token: int, pos: int, logits: torch.Tensor) -> np.ndarray:
        return aio_trace_step(self.handle, token, pos, logits, 5 * self.c.n_layers + 1)

    @property
    def uses_step_kernel(self) -> bool:
        return aio_uses_step_kernel(self.handle)

    def status(self) -> int:
        """Device-side status word (0 = fine); synchronises."""
        return aio_device_status(self.handle)

    def sync(self) -> None:
        self.stream.synchronize()

    def close(self) -> None:
        if getattr(self, "handle", None):
            aio_model_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
