"""Pins for the CPU oracle: each check compares it with something other than
itself (closed forms, fp64 brute force, library routines, an independent
full causal recompute, invariants), chosen so that a dropped term, a wrong
sign or index, or a transposed operand in the oracle fails one of them."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import ref_np

RNG = np.random.default_rng(1234)


def rand_bf16(shape, std=1.0, seed=0, name="t"):
    return synth.normal_bf16(seed, name, shape, 0.0, std)


# ------------------------------------------------------------------ formats

def test_bf16_rounding_matches_torch(oracle_lib):
    x = RNG.standard_normal(20000).astype(np.float32) * 10.0 ** RNG.integers(-6, 6, 20000)
    # exact ties: values halfway between two bf16 numbers
    base = RNG.integers(0, 0x7F7F, 200).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, [0.0, -0.0, np.inf, -np.inf, 3.0e38]]).astype(np.float32)
    ours = oracle.f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    # NaN stays NaN (payloads are not compared)
    n = oracle.f32_to_bf16(np.array([np.nan], np.float32))[0]
    assert (n & 0x7F80) == 0x7F80 and (n & 0x7F) != 0


def test_fp16_widening_matches_numpy(oracle_lib):
    bits = np.arange(0, 1 << 16, dtype=np.uint16)
    fin = np.isfinite(bits.view(np.float16))
    ours = np.array([oracle.lib().orc_fp16_to_f32(int(b)) for b in bits[fin]], dtype=np.float32)
    assert np.array_equal(ours, bits[fin].view(np.float16).astype(np.float32))


# --------------------------------------------------------------------- GEMV

@pytest.mark.parametrize("shape", [(7, 13), (64, 256), (256, 1024), (33, 520)])
def test_gemv_bf16_vs_fp64(oracle_lib, shape):
    n, k = shape
    w = rand_bf16(shape, 0.02, name="w%dx%d" % shape)
    x = RNG.standard_normal(k).astype(np.float32)
    y = oracle.gemv(w, x)
    ref = ref_np.bf16_to_f64(w) @ x.astype(np.float64)
    # one fp32 rounding of a double-accumulated sum
    assert np.allclose(y, ref, rtol=2 ** -23, atol=1e-30)


def test_gemv_orientation(oracle_lib):
    """y_n reads row n of W: a one-hot row picks exactly one input."""
    w = np.zeros((5, 9), dtype=np.uint16)
    w[3, 7] = 0x3F80  # 1.0
    w[1, 2] = 0x4000  # 2.0
    x = np.arange(9, dtype=np.float32) + 1
    assert list(oracle.gemv(w, x)) == [0, 6, 0, 8, 0]


@pytest.mark.parametrize("shape", [(7, 16), (96, 512), (128, 1024)])
def test_gemv_int8_exact_integer(oracle_lib, shape):
    """int8 with unit scale and small-integer inputs: an exact integer dot."""
    q = synth.int8_sym(5, "q%dx%d" % shape, shape)
    s = np.full(shape[0], 0x3C00, dtype=np.uint16)  # fp16 1.0
    x = RNG.integers(-8, 9, shape[1]).astype(np.float32)
    y = oracle.gemv(q, x, s)
    ref = q.astype(np.int64) @ x.astype(np.int64)
    assert np.array_equal(y.astype(np.int64), ref)


def test_gemv_int8_scale_per_output_channel(oracle_lib):
    shape = (48, 256)
    q = synth.int8_sym(6, "qs", shape)
    s = synth.uniform_fp16(6, "ss", (shape[0],), 0.001, 0.01)
    x = RNG.standard_normal(shape[1]).astype(np.float32)
    y = oracle.gemv(q, x, s)
    ref = (q.astype(np.float64) @ x.astype(np.float64)) * ref_np.fp16_to_f64(s)
    assert np.allclose(y, ref, rtol=2 ** -23, atol=1e-30)


# ------------------------------------------------------------------ RMSNorm

def test_rmsnorm_constant_vector(oracle_lib):
    d, c, eps = 256, 0.37, 1e-6
    x = np.full(d, c, dtype=np.float32)
    g = synth.normal_bf16(1, "gain", (d,), 1.0, 0.02)
    out = oracle.rmsnorm(x, g, eps)
    cc = float(np.float32(c))
    ref = ref_np.bf16_to_f64(g) * cc / math.sqrt(cc * cc + float(np.float32(eps)))
    assert np.allclose(out, ref, rtol=2 ** -22, atol=0)


def test_rmsnorm_unit_rms_and_scale_invariance(oracle_lib):
    d = 4096
    x = RNG.standard_normal(d).astype(np.float32) * 3
    ones = np.full(d, 0x3F80, dtype=np.uint16)
    out = oracle.rmsnorm(x, ones, 1e-6).astype(np.float64)
    assert abs(math.sqrt(np.mean(out * out)) - 1.0) < 1e-6
    out2 = oracle.rmsnorm(x * 1000, ones, 1e-6)
    assert np.allclose(out, out2, rtol=1e-6, atol=1e-7)


def test_rmsnorm_eps_inside_sqrt(oracle_lib):
    """A zero vector stays zero; a tiny vector is damped by eps, not divided
    by its own tiny RMS."""
    d = 64
    ones = np.full(d, 0x3F80, dtype=np.uint16)
    assert np.all(oracle.rmsnorm(np.zeros(d, np.float32), ones, 1e-6) == 0)
    x = np.full(d, 1e-4, dtype=np.float32)
    out = oracle.rmsnorm(x, ones, 1e-6)
    ref = 1e-4 / math.sqrt(1e-8 + float(np.float32(1e-6)))
    assert np.allclose(out, ref, rtol=1e-6)


# --------------------------------------------------------------------- RoPE

@pytest.mark.parametrize("hd", [64, 128])
def test_rope_basis_vectors_closed_form(oracle_lib, hd):
    """e_i at position p -> cos(p theta_i) e_i + sin(p theta_i) e_{i+hd/2};
    e_{i+hd/2} -> -sin e_i + cos e_{i+hd/2}; theta_i = 10000^(-2i/hd)."""
    half = hd // 2
    for p in (1, 7, 2049, 32768):
        for i in (0, 1, half // 2, half - 1):
            th = 10000.0 ** (-2.0 * i / hd)
            c, s = math.cos(p * th), math.sin(p * th)
            u = np.zeros(hd, np.float32)
            u[i] = 1
            r = oracle.rope(u, p)
            exp = np.zeros(hd)
            exp[i], exp[i + half] = c, s
            assert np.allclose(r, exp, atol=1e-7), (p, i)
            u = np.zeros(hd, np.float32)
            u[i + half] = 1
            r = oracle.rope(u, p)
            exp = np.zeros(hd)
            exp[i], exp[i + half] = -s, c
            assert np.allclose(r, exp, atol=1e-7), (p, i)


def test_rope_identity_norm_and_relative_position(oracle_lib):
    hd = 128
    q = RNG.standard_normal(hd).astype(np.float32)
    k = RNG.standard_normal(hd).astype(np.float32)
    assert np.array_equal(oracle.rope(q, 0), q)
    for p in (1, 100, 4000, 32000):
        r = oracle.rope(q, p).astype(np.float64)
        assert abs(np.linalg.norm(r) - np.linalg.norm(q.astype(np.float64))) < 2e-6 * np.linalg.norm(q)
    # <R_p q, R_r k> depends only on p - r
    dots = [np.dot(oracle.rope(q, p + s).astype(np.float64), oracle.rope(k, s).astype(np.float64))
            for p, s in ((5, 0), (5, 17), (5, 300))]
    assert max(dots) - min(dots) < 1e-5


# ---------------------------------------------------------------- attention

def test_attention_single_key_returns_v_exactly(oracle_lib):
    hd = 128
    q = RNG.standard_normal(hd).astype(np.float32) * 5
    k = rand_bf16((1, hd), name="k1")
    v = rand_bf16((1, hd), name="v1")
    out = oracle.attention_head(q, k, v)
    assert np.array_equal(out, ref_np.bf16_to_f64(v[0]).astype(np.float32))


def test_attention_equal_keys_mean_of_v(oracle_lib):
    hd, n = 64, 37
    q = RNG.standard_normal(hd).astype(np.float32)
    k = np.tile(rand_bf16((1, hd), name="ke"), (n, 1))
    v = rand_bf16((n, hd), name="ve")
    out = oracle.attention_head(q, k, v)
    assert np.allclose(out, ref_np.bf16_to_f64(v).mean(axis=0), rtol=1e-6, atol=1e-7)


def test_attention_ones_v_and_dominant_key(oracle_lib):
    hd, n = 128, 300
    q = RNG.standard_normal(hd).astype(np.float32)
    k = rand_bf16((n, hd), name="kd")
    ones = np.full((n, hd), 0x3F80, dtype=np.uint16)
    assert np.all(oracle.attention_head(q, k, ones) == 1.0)  # weights sum to 1
    # key 123 aligned with a large q dominates every other score
    qd = np.zeros(hd, np.float32)
    qd[3] = 400.0
    k2 = np.zeros((n, hd), np.uint16)
    k2[123, 3] = 0x3F80
    v = rand_bf16((n, hd), name="vd")
    out = oracle.attention_head(qd, k2, v)
    assert np.allclose(out, ref_np.bf16_to_f64(v[123]), rtol=1e-6, atol=1e-6)


def test_attention_vs_fp64_softmax(oracle_lib):
    from scipy.special import softmax
    hd, n = 128, 2049
    q = RNG.standard_normal(hd).astype(np.float32)
    k = rand_bf16((n, hd), name="kb")
    v = rand_bf16((n, hd), name="vb")
    out = oracle.attention_head(q, k, v)
    a = softmax(ref_np.bf16_to_f64(k) @ q.astype(np.float64) / math.sqrt(hd))
    ref = a @ ref_np.bf16_to_f64(v)
    assert np.allclose(out, ref, rtol=1e-6, atol=1e-7)


# -------------------------------------------------------------- silu, argmax

def test_silu(oracle_lib):
    from scipy.special import expit
    assert oracle.silu(0.0) == 0.0
    assert abs(oracle.silu(40.0) - 40.0) < 1e-12
    assert abs(oracle.silu(-40.0)) < 1e-15
    for z in np.linspace(-12, 12, 97):
        assert abs(oracle.silu(z) - z * expit(z)) <= 4e-16 * max(1.0, abs(z))


def test_argmax_ties_inf_nan_match_torch(oracle_lib):
    cases = [
        np.array([1, 3, 3, 2], np.float32),
        np.array([-np.inf, -np.inf], np.float32),
        np.array([0, np.inf, 5, np.inf], np.float32),
        np.array([0, np.inf, np.nan, np.nan], np.float32),
        np.array([np.nan, 1], np.float32),
        np.array([-1e30, -0.0, 0.0], np.float32),
    ]
    r = np.random.default_rng(7)
    for _ in range(50):
        x = r.integers(-3, 4, 4096).astype(np.float32)  # many ties
        cases.append(x)
    for x in cases:
        assert oracle.argmax(x) == int(torch.argmax(torch.from_numpy(x))), x


# --------------------------------------------------------- the whole decoder

def _small(wfmt="bf16", **kw):
    base = synth.CONFIGS["tiny"].with_(**kw)
    return base.with_(wfmt=wfmt) if wfmt != base.wfmt else base


CASES = {
    "tiny": dict(),
    "gqa": dict(n_heads=4, n_kv_heads=2, name="gqa"),
    "hd128_gqa4": dict(n_heads=4, n_kv_heads=1, head_dim=128, d_model=256, name="hd128"),
    "int8": dict(wfmt="int8", name="int8"),
}


@pytest.mark.parametrize("case", list(CASES))
def test_decode_matches_full_causal_recompute(oracle_lib, case):
    kw = dict(CASES[case])
    wfmt = kw.pop("wfmt", "bf16")
    cfg = _small(wfmt, prompt_len=40, n_steps=24, **kw)
    w = synth.make_weights(cfg)
    m = oracle.OracleModel(cfg, w)
    kv = synth.make_kv(cfg)
    toks = list(synth.make_prompt(cfg))
    rows = []
    for p in range(cfg.prompt_len + cfg.n_steps):
        lg = m.decode_step(kv, toks[p], p)
        rows.append(lg)
        if p + 1 >= len(toks):
            toks.append(oracle.argmax(lg))
    got = np.stack(rows).astype(np.float64)
    ref = ref_np.full_causal_logits(cfg, w, np.array(toks[: len(rows)]))
    scale = max(np.abs(ref).max(), 1.0)
    per_pos = np.abs(got - ref).max(axis=1)
    # Typical positions agree to fp32 rounding.  With int8 weights the
    # activations are ~25x larger and attention is nearly one-hot, so a single
    # bf16 rounding flip of a cached K/V element (decided from slightly
    # different fp32 values on the two sides) can move one position's logits
    # by ~3e-4 of their scale; a dropped or misapplied scale moves them O(1).
    assert np.median(per_pos) <= 1e-5 * scale, (case, np.median(per_pos), scale)
    bound = 1e-3 if cfg.wfmt == "int8" else 1e-5
    assert per_pos.max() <= bound * scale, (case, per_pos.max(), scale)


def test_gqa_equals_mha_with_duplicated_kv_heads(oracle_lib):
    cfg_g = _small(n_heads=4, n_kv_heads=2, name="g", prompt_len=20, n_steps=0)
    w = synth.make_weights(cfg_g)
    cfg_m = cfg_g.with_(n_kv_heads=4)
    wm = dict(w)
    hd = cfg_g.head_dim
    for l in range(cfg_g.n_layers):
        for nm in ("wk", "wv"):
            a = w["layers.%d.%s" % (l, nm)].reshape(2, hd, -1)
            wm["layers.%d.%s" % (l, nm)] = np.ascontiguousarray(np.repeat(a, 2, axis=0).reshape(4 * hd, -1))
    mg, mm = oracle.OracleModel(cfg_g, w), oracle.OracleModel(cfg_m, wm)
    kvg, kvm = synth.make_kv(cfg_g), synth.make_kv(cfg_m)
    for p, t in enumerate(synth.make_prompt(cfg_g)):
        a, b = mg.decode_step(kvg, t, p), mm.decode_step(kvm, t, p)
        assert np.array_equal(a, b)


def test_verify_equals_sequential_decode(oracle_lib):
    cfg = _small(prompt_len=16, n_steps=0, name="v")
    w = synth.make_weights(cfg)
    m = oracle.OracleModel(cfg, w)
    prompt = synth.make_prompt(cfg)
    kv1, kv2 = synth.make_kv(cfg), synth.make_kv(cfg)
    for p, t in enumerate(prompt[:-3]):
        m.decode_step(kv1, t, p)
        m.decode_step(kv2, t, p)
    pos = len(prompt) - 3
    rows = [t for t in prompt[-3:]] + [11, 12, 13]
    ver = m.verify(kv1, rows, pos)
    seq = np.stack([m.decode_step(kv2, t, pos + i) for i, t in enumerate(rows)])
    assert np.array_equal(ver, seq)
    assert np.array_equal(kv1, kv2)


def test_decode_step_row_supplied_entries(oracle_lib):
    """The supplied-row step: given its own row back it is the plain step bit
    for bit; given a row with one layer-0 V entry moved by one bf16 ulp, it
    hands out the same layer-0 row, stores the supplied entries, and its
    logits move (the attention reads the stored entry)."""
    cfg = _small(prompt_len=12, n_steps=0, name="row")
    m = oracle.OracleModel(cfg, synth.make_weights(cfg))
    prompt = synth.make_prompt(cfg)
    kv = synth.make_kv(cfg)
    for p, t in enumerate(prompt[:-1]):
        m.decode_step(kv, t, p)
    pos, tok = len(prompt) - 1, prompt[-1]
    kv_plain = kv.copy()
    ref = m.decode_step(kv_plain, tok, pos)
    own_plain = np.ascontiguousarray(kv_plain[:, :, :, pos, :])
    kv_same = kv.copy()
    lg, own = m.decode_step_row(kv_same, tok, pos, own_plain)
    assert np.array_equal(lg.view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(own, own_plain)
    assert np.array_equal(kv_same, kv_plain)
    moved = own_plain.copy()
    moved[0, 1, 0, 3] += 1
    kv_moved = kv.copy()
    lg2, own2 = m.decode_step_row(kv_moved, tok, pos, moved)
    assert np.array_equal(own2[0], own_plain[0])
    assert np.array_equal(kv_moved[:, :, :, pos, :], moved)
    assert not np.array_equal(lg2, ref)


def test_oracle_rejects_out_of_range(oracle_lib):
    cfg = _small(prompt_len=4, n_steps=0, name="r")
    m = oracle.OracleModel(cfg, synth.make_weights(cfg))
    kv = synth.make_kv(cfg)
    for tok, pos in ((-1, 0), (cfg.vocab, 0), (0, -1), (0, cfg.max_ctx)):
        with pytest.raises(ValueError):
            m.decode_step(kv, tok, pos)
