"""Parity of the one-forward verify path (MFMA skinny GEMM + causal multi-row
attention) with k+1 sequential oracle decode steps (needs an MI355X)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_cases import (LOGIT_TOL, Pair, Tally, check_verify, compare_logits, log,
                             teacher_forced)

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
    # O (K = 1024) and down (K = 4096) products split over K, their slices
    # added in order by the next RMSNorm
    "split_k": dict(n_heads=16, n_kv_heads=4, ffn_dim=4096),
    # d 576: three 256-k stages per tile pair, the last one ragged; the QKV
    # and gate/up products deal out (tile pair, stage) units two per
    # workgroup, so tile pairs are shared by two workgroups
    "stream_k": dict(d_model=576, ffn_dim=192),
    "stream_k_int8": dict(d_model=576, ffn_dim=192, wfmt="int8"),
}


def _prefilled(cfg):
    """Both sides prefilled with the prompt, every step from identical state."""
    pair = Pair(cfg)
    prompt = synth.make_prompt(cfg)
    teacher_forced(pair, int(prompt[0]), 0, len(prompt), tokens=prompt)
    return pair, prompt


@pytest.mark.parametrize("name", list(CASES))
def test_verify_equals_sequential_decode(name):
    """Every row of a verify of k drafts equals the oracle's decode step of
    that row's token from identical state (the cache rows before it are the
    ones this verify wrote, each checked against the oracle's); the same
    verify again gives bit-identical logits and cache rows."""
    cfg = BASE.with_(name="v_" + name, **CASES[name])
    pair, prompt = _prefilled(cfg)
    try:
        P = cfg.prompt_len
        rng = np.random.default_rng(11)
        for k in (0, 2, 3, 4, 5, 8, 9):
            token = int(rng.integers(0, cfg.vocab))
            drafts = rng.integers(0, cfg.vocab, k).astype(np.int32)
            kv_before = pair.kv_host.copy()
            free = pair.kv_host.copy()
            tally = Tally()
            got = check_verify(pair, token, drafts, P, "verify %s k=%d" % (name, k), tally, free)
            log("verify %s k=%d: %s" % (name, k, tally.summary()))
            if cfg.wfmt != "int8":
                assert tally.worst_free <= LOGIT_TOL
            kg = pair.gpu.kv_rows(P, P + k + 1)
            # the same call again gives bit-identical logits and cache rows
            pair.gpu.verify(token, drafts, P, pair.logits)
            pair.gpu.sync()
            again = pair.logits[: k + 1].cpu().numpy()
            assert np.array_equal(got.view(np.uint32), again.view(np.uint32)), (name, k)
            assert np.array_equal(kg, pair.gpu.kv_rows(P, P + k + 1)), (name, k)
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
