"""Seeded synthetic workloads for the batch-1 decode path.

Shared by the CPU oracle and the GPU path: model shapes, weights, synthetic
prompt KV and prompt tokens.  Nothing here computes any part of the decoder;
it only draws numbers (Philox4x32-10 streams in ``synth.c``) and rounds them to
the storage formats (bf16, int8, fp16).

The paper (Sections 2.1, 3.1 and 4.2) names 1B and 7B models, 2K and 32K
contexts, W8A16 storage and prompt-lookup verification but never the
architecture, so the five workloads below fix it: a Llama-style pre-norm
decoder with RMSNorm, rotate-half RoPE, SwiGLU and grouped-query attention.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``libsynth.so`` with gcc (OpenMP, -O2)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = ctypes.CDLL(_LIB_PATH)
        u64, vp = ctypes.c_uint64, ctypes.c_void_p
        L.synth_philox4x32_10.argtypes = [vp, vp, vp]
        L.synth_stream_id.argtypes = [ctypes.c_char_p]
        L.synth_stream_id.restype = u64
        L.synth_normal_bf16.argtypes = [u64, u64, vp, u64, ctypes.c_double, ctypes.c_double]
        L.synth_normal_f32.argtypes = [u64, u64, vp, u64, ctypes.c_double, ctypes.c_double]
        L.synth_int8_sym.argtypes = [u64, u64, vp, u64]
        L.synth_uniform_fp16.argtypes = [u64, u64, vp, u64, ctypes.c_double, ctypes.c_double]
        L.synth_tokens.argtypes = [u64, u64, vp, u64, ctypes.c_uint32]
        L.synth_uniform_index.argtypes = [u64, u64, u64, ctypes.c_uint32]
        L.synth_uniform_index.restype = ctypes.c_uint32
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags.c_contiguous
    return a.ctypes.data


def philox4x32_10(ctr, key) -> tuple:
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().synth_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return tuple(int(v) for v in out)


def stream_id(name: str) -> int:
    return int(lib().synth_stream_id(name.encode()))


def normal_bf16(seed: int, name: str, shape, mean=0.0, std=1.0) -> np.ndarray:
    """bf16 bit patterns (uint16) of mean + std * N(0, 1)."""
    out = np.empty(shape, dtype=np.uint16)
    lib().synth_normal_bf16(seed, stream_id(name), _ptr(out), out.size, mean, std)
    return out


def normal_f32(seed: int, name: str, shape, mean=0.0, std=1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    lib().synth_normal_f32(seed, stream_id(name), _ptr(out), out.size, mean, std)
    return out


def int8_sym(seed: int, name: str, shape) -> np.ndarray:
    out = np.empty(shape, dtype=np.int8)
    lib().synth_int8_sym(seed, stream_id(name), _ptr(out), out.size)
    return out


def uniform_fp16(seed: int, name: str, shape, lo: float, hi: float) -> np.ndarray:
    """IEEE binary16 bit patterns (uint16) uniform on (lo, hi)."""
    out = np.empty(shape, dtype=np.uint16)
    lib().synth_uniform_fp16(seed, stream_id(name), _ptr(out), out.size, lo, hi)
    return out


def tokens(seed: int, name: str, n: int, vocab: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    lib().synth_tokens(seed, stream_id(name), _ptr(out), n, vocab)
    return out


def uniform_index(seed: int, name: str, which: int, n: int) -> int:
    return int(lib().synth_uniform_index(seed, stream_id(name), which, n))


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (a storage-format view)."""
    return (u16.astype(np.uint32) << 16).view(np.float32)


def fp16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    return u16.view(np.float16).astype(np.float32)


# --------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class ModelConfig:
    """Shape and workload of one synthetic decoder.

    ``prompt_len`` positions of KV are present before the first measured
    decode step.  With ``prefill_by_model`` the prompt tokens are run through
    the model one by one (the oracle-scale workload); otherwise the prompt KV
    is drawn directly as bf16 N(0, 1) and taken as already rotated.
    """
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    prompt_len: int
    n_steps: int
    seed: int
    wfmt: str = "bf16"                 # "bf16" or "int8" (per-output-channel fp16 scale)
    prefill_by_model: bool = False
    verify_k: int = 8
    max_verify: int = 10
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    weight_std: float = 0.02
    max_ctx: int = field(default=0)

    def __post_init__(self):
        if self.max_ctx == 0:
            need = self.prompt_len + self.n_steps + self.max_verify
            object.__setattr__(self, "max_ctx", (need + 63) // 64 * 64)

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    def with_(self, **kw) -> "ModelConfig":
        kw.setdefault("max_ctx", 0)
        return replace(self, **kw)


CONFIGS = {
    # 2 layers, d 256, 4 x 64 MHA, FFN 1024, vocab 4096; 128 prompt tokens
    # prefilled through the model, then 32 greedy steps.
    "tiny": ModelConfig("tiny", 2, 256, 4, 4, 64, 1024, 4096, prompt_len=128, n_steps=32,
                        seed=0xA10, prefill_by_model=True),
    # 1B-class probe: 24 layers, d 2048, 16 heads / 8 KV heads x 128, FFN 5632.
    "1b": ModelConfig("1b", 24, 2048, 16, 8, 128, 5632, 32000, prompt_len=2048, n_steps=256,
                      seed=0xA11),
    # 7B-class backbone at 2K context: 32 layers, d 4096, 32 x 128 MHA, FFN 11008.
    "7b": ModelConfig("7b", 32, 4096, 32, 32, 128, 11008, 32000, prompt_len=2048, n_steps=256,
                      seed=0xA12),
    # Same backbone with 32768 positions of KV.
    "7b_32k": ModelConfig("7b_32k", 32, 4096, 32, 32, 128, 11008, 32000, prompt_len=32768,
                          n_steps=128, seed=0xA13),
    # Same backbone with int8 per-output-channel weights; plus one k=8 verify.
    "7b_int8": ModelConfig("7b_int8", 32, 4096, 32, 32, 128, 11008, 32000, prompt_len=2048,
                           n_steps=256, seed=0xA14, wfmt="int8"),
}


def linear_shapes(cfg: ModelConfig) -> dict:
    """(out, in) of every per-layer projection, nn.Linear convention."""
    d, hd = cfg.d_model, cfg.head_dim
    return {
        "wq": (cfg.n_heads * hd, d),
        "wk": (cfg.n_kv_heads * hd, d),
        "wv": (cfg.n_kv_heads * hd, d),
        "wo": (d, cfg.n_heads * hd),
        "w_gate": (cfg.ffn_dim, d),
        "w_up": (cfg.ffn_dim, d),
        "w_down": (d, cfg.ffn_dim),
    }


LAYER_LINEARS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def _linear(cfg: ModelConfig, name: str, shape, out: dict):
    if cfg.wfmt == "bf16":
        out[name] = normal_bf16(cfg.seed, name, shape, 0.0, cfg.weight_std)
    elif cfg.wfmt == "int8":
        out[name] = int8_sym(cfg.seed, name, shape)
        out[name + ".scale"] = uniform_fp16(cfg.seed, name + ".scale", (shape[0],), 0.001, 0.01)
    else:
        raise ValueError(cfg.wfmt)


def make_weights(cfg: ModelConfig) -> dict:
    """All weights as numpy arrays of storage bits.

    Linear and embedding weights ~ N(0, std) in bf16; norm gains
    bf16(1 + N(0, 0.02)) so that a dropped gain multiply is visible.  With
    ``wfmt == 'int8'`` the projections and the LM head are int8 uniform on
    [-127, 127] with fp16 per-output-channel scales uniform on (0.001, 0.01);
    the embedding and gains stay bf16.
    """
    w = {}
    d, V = cfg.d_model, cfg.vocab
    w["embed"] = normal_bf16(cfg.seed, "embed", (V, d), 0.0, cfg.weight_std)
    w["final_norm"] = normal_bf16(cfg.seed, "final_norm", (d,), 1.0, 0.02)
    _linear(cfg, "lm_head", (V, d), w)
    shapes = linear_shapes(cfg)
    for l in range(cfg.n_layers):
        p = "layers.%d." % l
        w[p + "attn_norm"] = normal_bf16(cfg.seed, p + "attn_norm", (d,), 1.0, 0.02)
        w[p + "ffn_norm"] = normal_bf16(cfg.seed, p + "ffn_norm", (d,), 1.0, 0.02)
        for nm in LAYER_LINEARS:
            _linear(cfg, p + nm, shapes[nm], w)
    return w


def kv_shape(cfg: ModelConfig) -> tuple:
    """KV cache layout: [layer][K or V][kv head][position][head dim], bf16."""
    return (cfg.n_layers, 2, cfg.n_kv_heads, cfg.max_ctx, cfg.head_dim)


def make_kv(cfg: ModelConfig, n_pos: int | None = None) -> np.ndarray:
    """bf16 KV cache with N(0, 1) keys and values at positions [0, n_pos).

    The synthetic prompt KV stands in for a prompt already run through the
    model (2K and 32K context); it is taken as already rotated.  Positions at
    and beyond ``n_pos`` are zero and are written by decode before any read.
    """
    if n_pos is None:
        n_pos = 0 if cfg.prefill_by_model else cfg.prompt_len
    kv = np.zeros(kv_shape(cfg), dtype=np.uint16)
    if n_pos:
        shp = (cfg.n_kv_heads, n_pos, cfg.head_dim)
        for l in range(cfg.n_layers):
            for t, nm in enumerate(("k", "v")):
                kv[l, t, :, :n_pos, :] = normal_bf16(cfg.seed + 1, "kv.%d.%s" % (l, nm), shp)
    return kv


def make_prompt(cfg: ModelConfig) -> np.ndarray:
    """Uniform random prompt token ids (length prompt_len)."""
    return tokens(cfg.seed + 2, "prompt", cfg.prompt_len, cfg.vocab)


def first_token(cfg: ModelConfig) -> int:
    """Seeded first decode input when the prompt KV is synthetic."""
    return int(tokens(cfg.seed + 2, "tau0", 1, cfg.vocab)[0])


def planted_drafts(cfg: ModelConfig, prompt: np.ndarray, tau0: int, k: int | None = None):
    """Prompt with a planted 3-gram match and the k drafts it yields.

    Uniform random prompts almost never repeat a 3-gram, so one is planted:
    for a seeded j, (prompt[P-2], prompt[P-1], tau0) is made equal to
    (prompt[j], prompt[j+1], prompt[j+2]); a prompt-lookup matcher then
    proposes prompt[j+3 : j+3+k] as drafts.  Returns (prompt', drafts).
    """
    k = cfg.verify_k if k is None else k
    P = len(prompt)
    p = prompt.copy()
    j = uniform_index(cfg.seed + 2, "plant", 0, P - 3 - k - 2)
    p[P - 2], p[P - 1] = p[j], p[j + 1]
    p[j + 2] = tau0
    drafts = p[j + 3: j + 3 + k].copy()
    return p, drafts
