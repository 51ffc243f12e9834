"""Why the GPU parity tests compare every step from identical state (CPU,
oracle only).

A cache entry is the bf16 rounding of an fp32 value, rounded to nearest
even on append (reading c10).  The GPU and the oracle accumulate that value
in different orders, so where it lies within their difference of a rounding
boundary the two caches legitimately hold neighbouring bf16 values.  With
the int8 workload's weights (int8 uniform on [-127, 127] times scales in
0.001-0.01, about 20x the scale of N(0, 0.02) bf16 weights) queries and keys
are large and attention is very peaked, so such a one-ulp difference in a
single entry of an earlier row moves the next logits by more than the 2e-2
bound, on the oracle alone; with bf16 weights it moves them by far less.
The parity tests therefore hand the oracle the GPU's cache rows (each first
checked against the oracle's own row) before every compared step."""
import numpy as np
import pytest

import oracle
import synth


def _largest_change(wfmt: str, trials: int = 120) -> float:
    cfg = synth.CONFIGS["tiny"].with_(name="sens_" + wfmt, prompt_len=40, n_steps=8, wfmt=wfmt)
    w = synth.make_weights(cfg)
    orc = oracle.OracleModel(cfg, w)
    kv = synth.make_kv(cfg)
    prompt = synth.make_prompt(cfg)
    lg = None
    for p, t in enumerate(prompt):
        lg = orc.decode_step(kv, int(t), p)
    tok, P = oracle.argmax(lg), len(prompt)
    base = orc.decode_step(kv.copy(), tok, P).astype(np.float64)
    rng = np.random.default_rng(0)
    worst = 0.0
    for _ in range(trials):
        k2 = kv.copy()
        idx = (rng.integers(0, cfg.n_layers), rng.integers(0, 2), rng.integers(0, cfg.n_kv_heads),
               rng.integers(P - 8, P), rng.integers(0, cfg.head_dim))
        # the neighbouring bf16 value (one unit in the last place)
        k2[idx] = np.uint16(int(k2[idx]) + (1 if rng.random() < 0.5 else -1))
        worst = max(worst, float(np.abs(orc.decode_step(k2, tok, P) - base).max()))
    return worst


def test_one_ulp_cache_difference_exceeds_bound_with_int8_weights(oracle_lib, synth_lib):
    assert _largest_change("int8") > 2e-2


def test_one_ulp_cache_difference_is_small_with_bf16_weights(oracle_lib, synth_lib):
    assert _largest_change("bf16") < 1e-3
