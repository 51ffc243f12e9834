"""Parity of the one-forward verify path (MFMA skinny GEMM + causal multi-row
attention) with k+1 sequential oracle decode steps (needs an MI355X)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_cases import LOGIT_TOL, Pair, assert_kv_close, compare_logits, log

pytestmark = pytest.mark.gpu

BASE = synth.CONFIGS["tiny"].with_(prompt_len=40, n_steps=16)

CASES = {
    "tiny": dict(),
    "gqa2": dict(n_heads=4, n_kv_heads=2),
    "hd128_gqa4": dict(n_heads=4, n_kv_heads=1, head_dim=128),
    "ragged": dict(d_model=320, ffn_dim=192, vocab=1000, n_heads=5, n_kv_heads=5),
    "int8": dict(wfmt="int8"),
    # caches beyond 8K positions take the attention shape with two row
    # groups, and 128 splits per head leave most splits empty
    "long_cache": dict(max_ctx=8256),
    "long_cache_hd128": dict(n_heads=4, n_kv_heads=1, head_dim=128, max_ctx=8256),
}


def _tol(cfg, rms):
    return LOGIT_TOL * max(1.0, rms) if cfg.wfmt == "int8" else LOGIT_TOL


def _prefilled(cfg):
    pair = Pair(cfg)
    prompt = synth.make_prompt(cfg)
    for p, t in enumerate(prompt):
        pair.gpu_step(int(t), p)
        pair.oracle_step(int(t), p)
    return pair, prompt


@pytest.mark.parametrize("name", list(CASES))
def test_verify_equals_sequential_decode(name):
    cfg = BASE.with_(name="v_" + name, **CASES[name])
    pair, prompt = _prefilled(cfg)
    try:
        P = cfg.prompt_len
        rng = np.random.default_rng(11)
        for k in (0, 2, 3, 4, 5, 8, 9):
            token = int(rng.integers(0, cfg.vocab))
            drafts = rng.integers(0, cfg.vocab, k).astype(np.int32)
            kv_before = pair.kv_host.copy()
            ref = pair.orc.verify(pair.kv_host, [token] + list(drafts), P)
            pair.gpu.verify(token, drafts, P, pair.logits)
            pair.gpu.sync()
            got = pair.logits[: k + 1].cpu().numpy()
            worst = 0.0
            for i in range(k + 1):
                err, rms = compare_logits(got[i], ref[i])
                tol = _tol(cfg, rms)
                worst = max(worst, err / tol)
                assert err <= tol, (name, k, i, err, tol)
            ids = pair.gpu_argmax(k + 1)
            agree = int(np.sum(ids == [oracle.argmax(r) for r in ref]))
            log("verify %s k=%d: worst err/tol %.3e, argmax agree %d/%d"
                % (name, k, worst, agree, k + 1))
            # the k+1 appended KV rows match within one bf16 rounding
            kg = pair.gpu.kv_numpy()[:, :, :, P:P + k + 1, :]
            ko = pair.kv_host[:, :, :, P:P + k + 1, :]
            assert_kv_close(kg, ko, "verify %s k=%d" % (name, k))
            # roll back: the oracle's cache returns to the prefilled state
            pair.kv_host[...] = kv_before
    finally:
        pair.close()


def test_verify_argmax_and_rollback():
    """Greedy acceptance on the verify logits, then plain decode continues at
    pos + a + 1 with the oracle's logits (rollback by position)."""
    cfg = BASE.with_(name="v_rollback")
    pair, prompt = _prefilled(cfg)
    try:
        P = cfg.prompt_len
        # drafts = the oracle's own greedy continuation for 3 tokens, then junk
        kv = pair.kv_host.copy()
        tok = int(prompt[-1])
        r = pair.orc.decode_step(kv.copy(), tok, P - 1)
        t0 = oracle.argmax(r)
        greedy = [t0]
        kvg = kv.copy()
        for s in range(3):
            greedy.append(oracle.argmax(pair.orc.decode_step(kvg, greedy[-1], P + s)))
        drafts = np.array(greedy[1:4] + [7, 8, 9], dtype=np.int32)
        pair.gpu.verify(t0, drafts, P, pair.logits)
        ids = pair.gpu_argmax(len(drafts) + 1)
        a = 0
        while a < len(drafts) and ids[a] == drafts[a]:
            a += 1
        assert a >= 3, (ids, drafts)
        nxt = int(ids[a])
        # oracle: the same tokens sequentially
        seq = pair.orc.verify(pair.kv_host, [t0] + list(drafts[:a]), P)
        assert oracle.argmax(seq[-1]) == nxt
        # continue at P + a + 1 on both sides
        g = pair.gpu_step(nxt, P + a + 1)
        o = pair.oracle_step(nxt, P + a + 1)
        err, _ = compare_logits(g, o)
        assert err <= LOGIT_TOL
    finally:
        pair.close()
