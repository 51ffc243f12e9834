"""Measures how far a plain fp32 evaluation of a decode step lands from the
oracle on the int8 workload (7B-class, W8A16, 2048-position cache): the
arithmetic fact behind the int8 tolerances of the GPU parity tests.

    python tests/measure_int8_fp32.py [steps] > tests/golden/int8_fp32_conditioning.json

For each of the first `steps` greedy steps from the workload's first token,
the same step is evaluated twice from the same state: by the oracle (sums
in fp64, one rounding to fp32) and by numpy in float32 (every product and
sum in fp32, BLAS order).  Reported per step: the max-abs logit difference,
its ratio to the oracle's logit RMS, and the absolute term (times the row
maximum) the fp32 evaluation's new cache rows would need beyond one bf16
rounding.  Steps where the int8 model's attention nearly ties two keys of
very different values amplify fp32 rounding well beyond 2e-2.  Slow (about
40 s per step, 13 GB of host memory); not part of the test suite.
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402
from tests import ref_np as R  # noqa: E402


def fp32_step(cfg, w, kv, tok, pos, rows_out):
    """One decode step in float32 from the bf16 cache rows [0, pos); fills
    rows_out[l] = (K row, V row) as bf16-rounded values; kv is not modified."""
    f = np.float32
    H, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    G = H // Hkv

    def mat(n):
        if cfg.wfmt == "bf16":
            return R.bf16_to_f64(w[n]).astype(f)
        return w[n].astype(f) * R.fp16_to_f64(w[n + ".scale"]).astype(f)[:, None]

    def norm(x, g):
        return (x / np.sqrt(np.mean(x * x, dtype=f) + f(cfg.rms_eps))
                * R.bf16_to_f64(g).astype(f)).astype(f)

    theta = cfg.rope_base ** (-2.0 * np.arange(hd // 2) / hd)
    c, s = np.cos(pos * theta).astype(f), np.sin(pos * theta).astype(f)

    def rope(u):
        a, b = u[..., :hd // 2], u[..., hd // 2:]
        return np.concatenate([a * c - b * s, b * c + a * s], axis=-1).astype(f)

    x = R.bf16_to_f64(w["embed"][tok]).astype(f)
    with np.errstate(over="ignore"):
        for l in range(cfg.n_layers):
            p = "layers.%d." % l
            h = norm(x, w[p + "attn_norm"])
            q = rope((mat(p + "wq") @ h).reshape(H, hd))
            kb = R.round_bf16(rope((mat(p + "wk") @ h).reshape(Hkv, hd))).astype(f)
            vb = R.round_bf16((mat(p + "wv") @ h).reshape(Hkv, hd)).astype(f)
            rows_out[l] = (kb, vb)
            K = np.concatenate([synth.bf16_bits_to_f32(kv[l, 0, :, :pos, :]), kb[:, None]], axis=1)
            V = np.concatenate([synth.bf16_bits_to_f32(kv[l, 1, :, :pos, :]), vb[:, None]], axis=1)
            o = np.empty((H, hd), f)
            for hh in range(H):
                sc = (K[hh // G] @ q[hh]) / f(np.sqrt(hd))
                a = np.exp(sc - sc.max())
                o[hh] = (a / a.sum()) @ V[hh // G]
            x = (x + mat(p + "wo") @ o.reshape(-1)).astype(f)
            h2 = norm(x, w[p + "ffn_norm"])
            g, u = mat(p + "w_gate") @ h2, mat(p + "w_up") @ h2
            x = (x + mat(p + "w_down") @ ((g / (1 + np.exp(-g))) * u).astype(f)).astype(f)
    return mat("lm_head") @ norm(x, w["final_norm"])


def main():
    steps = int(sys.argv[1]) if len(sys.argv) > 1 else 8
    cfg = synth.CONFIGS["7b_int8"]
    w, kv = synth.make_weights(cfg), synth.make_kv(cfg)
    orc = oracle.OracleModel(cfg, w)
    tok, P = synth.first_token(cfg), cfg.prompt_len
    out = {"workload": "7b_int8, first %d greedy steps from position %d" % (steps, P),
           "evaluations": "oracle (fp64 sums) vs numpy float32, same state", "steps": []}
    for st in range(steps):
        t0 = time.time()
        rows = {}
        g = fp32_step(cfg, w, kv, tok, P + st, rows).astype(np.float64)
        r = orc.decode_step(kv, tok, P + st).astype(np.float64)
        need = 0.0
        for l, pair in rows.items():
            for j, a in enumerate(pair):
                o = synth.bf16_bits_to_f32(kv[l, j, :, P + st, :]).astype(np.float64)
                a = a.astype(np.float64)
                exc = np.abs(a - o) - 2.0 ** -7 * np.maximum(np.abs(a), np.abs(o))
                need = max(need, float((exc / np.abs(o).max(axis=-1, keepdims=True)).max()))
        err, rms = float(np.abs(g - r).max()), float(np.sqrt(np.mean(r * r)))
        out["steps"].append({"pos": P + st, "max_abs": err, "rel_rms": err / rms,
                             "kv_abs_need": need})
        print("pos %d: max-abs %.3e (%.2e of rms), KV need %.2e [%.0fs]"
              % (P + st, err, err / rms, need, time.time() - t0), file=sys.stderr, flush=True)
        tok = oracle.argmax(r)
    out["max_rel_rms"] = max(s["rel_rms"] for s in out["steps"])
    out["max_kv_abs_need"] = max(s["kv_abs_need"] for s in out["steps"])
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
