"""Independent fp64 reference computations used to pin the oracle.

These are written in a different form from the oracle (matrix form over all
positions at once, numpy/torch library routines) so that a slip in the
oracle's loops shows up as a mismatch.  Test-only.
"""
from __future__ import annotations

import numpy as np
import torch


def bf16_to_f64(u16: np.ndarray) -> np.ndarray:
    return (np.asarray(u16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def fp16_to_f64(u16: np.ndarray) -> np.ndarray:
    return np.asarray(u16).view(np.float16).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 (round to nearest even, torch's conversion) -> fp64."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.to(torch.float64).numpy()


def dense(w: dict, name: str, wfmt: str) -> np.ndarray:
    if wfmt == "bf16":
        return bf16_to_f64(w[name])
    return w[name].astype(np.float64) * fp16_to_f64(w[name + ".scale"])[:, None]


def rope_tables(T: int, hd: int, base: float):
    i = np.arange(hd // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / hd)
    ang = np.arange(T, dtype=np.float64)[:, None] * theta[None, :]
    # the method's table: fp32 roundings of fp64 cos/sin
    return np.cos(ang).astype(np.float32).astype(np.float64), \
        np.sin(ang).astype(np.float32).astype(np.float64)


def apply_rope(X: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """X [T][n_heads][hd], rotate-half: pairs (i, i + hd/2)."""
    half = X.shape[-1] // 2
    a, b = X[..., :half], X[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rmsnorm_rows(X: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return X / np.sqrt(np.mean(X * X, axis=-1, keepdims=True) + eps) * g


def full_causal_logits(cfg, w: dict, toks: np.ndarray, hand_over=None) -> np.ndarray:
    """Logits at every position of ``toks`` with one causal-masked forward.

    K and V are rounded to bf16 (through fp32) before use, as the cache holds
    them.  ``hand_over``, if given, is applied to every activation a fused
    decode step passes from one group of workers to the next (the residual
    stream after each addition, the rotated queries, the attention output,
    the SwiGLU product).  Returns fp64 [T][V]."""
    ho = hand_over if hand_over is not None else (lambda a: a)
    T = len(toks)
    d, H, Hkv, hd = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    G = H // Hkv
    X = bf16_to_f64(w["embed"])[np.asarray(toks)]
    cos, sin = rope_tables(T, hd, cfg.rope_base)
    mask = np.triu(np.ones((T, T), dtype=bool), k=1)
    for l in range(cfg.n_layers):
        p = "layers.%d." % l
        Hn = rmsnorm_rows(X, bf16_to_f64(w[p + "attn_norm"]), cfg.rms_eps)
        Q = (Hn @ dense(w, p + "wq", cfg.wfmt).T).reshape(T, H, hd)
        K = (Hn @ dense(w, p + "wk", cfg.wfmt).T).reshape(T, Hkv, hd)
        Vv = (Hn @ dense(w, p + "wv", cfg.wfmt).T).reshape(T, Hkv, hd)
        Q = ho(apply_rope(Q, cos, sin))
        K = round_bf16(apply_rope(K, cos, sin))
        Vv = round_bf16(Vv)
        O = np.empty((T, H, hd))
        for h in range(H):
            S = Q[:, h, :] @ K[:, h // G, :].T / np.sqrt(hd)
            S[mask] = -np.inf
            S = S - S.max(axis=1, keepdims=True)
            A = np.exp(S)
            A /= A.sum(axis=1, keepdims=True)
            O[:, h, :] = A @ Vv[:, h // G, :]
        X = ho(X + ho(O).reshape(T, H * hd) @ dense(w, p + "wo", cfg.wfmt).T)
        H2 = rmsnorm_rows(X, bf16_to_f64(w[p + "ffn_norm"]), cfg.rms_eps)
        Gt = H2 @ dense(w, p + "w_gate", cfg.wfmt).T
        Up = H2 @ dense(w, p + "w_up", cfg.wfmt).T
        M = ho(Gt / (1.0 + np.exp(-Gt)) * Up)
        X = ho(X + M @ dense(w, p + "w_down", cfg.wfmt).T)
    Hf = rmsnorm_rows(X, bf16_to_f64(w["final_norm"]), cfg.rms_eps)
    return Hf @ dense(w, "lm_head", cfg.wfmt).T
