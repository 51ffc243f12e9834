"""Algorithmic HBM bytes of one decode step (host-side accounting).

The paper's bandwidth argument (Section 3.1) is that each generated token
streams every weight from HBM; with the KV cache read and the new row
appended, that fixes the bytes a decode step must move:

    B_tok(p) = sum_linear |W| * w_bytes  (+ 2 bytes per output channel: int8 scales)
             + 2 * (2L + 1) * d           (norm gains, bf16)
             + 2 * d                      (one embedding row)
             + 2 * L * Hkv * hd * (p + 1) * 2   (K and V read over positions 0..p)
             + 2 * L * Hkv * hd * 2             (K and V appended at p)

Activations and split-KV partials stay on chip or in L2 and are not counted.
"""
from __future__ import annotations


def linear_params(cfg) -> int:
    d, H, Hkv, hd, F, L = (cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                           cfg.ffn_dim, cfg.n_layers)
    per_layer = d * H * hd + 2 * d * Hkv * hd + H * hd * d + 3 * d * F
    return L * per_layer + cfg.vocab * d


def output_channels(cfg) -> int:
    d, H, Hkv, hd, F, L = (cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                           cfg.ffn_dim, cfg.n_layers)
    return L * (H * hd + 2 * Hkv * hd + d + 2 * F + d) + cfg.vocab


def weight_bytes(cfg) -> int:
    """Bytes of weights, gains and one embedding row read per token."""
    wb = 1 if cfg.wfmt == "int8" else 2
    b = linear_params(cfg) * wb
    if cfg.wfmt == "int8":
        b += 2 * output_channels(cfg)
    b += 2 * (2 * cfg.n_layers + 1) * cfg.d_model + 2 * cfg.d_model
    return b


def kv_bytes_per_position(cfg) -> int:
    """K and V bytes of one position across all layers."""
    return 2 * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2


def step_bytes(cfg, pos: int) -> int:
    """B_tok for the decode step that consumes a token at position ``pos``."""
    kvp = kv_bytes_per_position(cfg)
    return weight_bytes(cfg) + kvp * (pos + 1) + kvp


def run_bytes(cfg, first_pos: int, n_steps: int) -> int:
    """Sum of B_tok over positions first_pos .. first_pos + n_steps - 1."""
    kvp = kv_bytes_per_position(cfg)
    w = weight_bytes(cfg) + kvp
    p0, p1 = first_pos, first_pos + n_steps - 1
    reads = kvp * ((p1 + 1) * (p1 + 2) // 2 - p0 * (p0 + 1) // 2)
    return n_steps * w + reads


def verify_bytes(cfg, pos: int, rows: int) -> int:
    """One verify forward of ``rows`` tokens at pos..pos+rows-1: weights once,
    the cache read once up to the last row, every new row appended."""
    kvp = kv_bytes_per_position(cfg)
    return weight_bytes(cfg) + 2 * rows * cfg.d_model - 2 * cfg.d_model \
        + kvp * (pos + rows) + kvp * rows
