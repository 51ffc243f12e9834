"""Prompt-lookup decoding loop on the GPU (needs an MI355X): the tokens
aio_pld_generate produces equal plain greedy decoding from the same state
(verification is lossless), with the paper's setting (n-gram window 6,
look-ahead 2) and the 3-gram / k = 8 setting, on the tiny decoder prefilled
with a prompt, and on the int8 7B decoder with a planted 3-gram."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_cases import Pair, log, top2_gap

pytestmark = pytest.mark.gpu


def _greedy_device(pair, token, pos, n):
    toks = torch.zeros(n, dtype=torch.int32, device=pair.gpu.device)
    pair.gpu.greedy(token, pos, n, toks, pair.logits[0])
    pair.gpu.sync()
    return toks.cpu().numpy().copy()


@pytest.mark.parametrize("ngram_max,k", [(6, 2), (3, 8)])
def test_tiny_pld_equals_greedy(ngram_max, k):
    cfg = synth.CONFIGS["tiny"].with_(name="pld", prompt_len=40, n_steps=48)
    pair = Pair(cfg)
    try:
        prompt = [int(t) for t in synth.make_prompt(cfg)]
        for p, t in enumerate(prompt[:-1]):
            pair.gpu_step(t, p)
            pair.oracle_step(t, p)
        pos, tok = len(prompt) - 1, prompt[-1]
        n_new = 48
        got, st = pair.gpu.pld_generate(prompt[:-1], pos, tok, n_new, ngram_max, 1, k)
        log("pld N=%d k=%d: %s" % (ngram_max, k, st))
        assert st["forwards"] + st["accepted"] == n_new  # a + 1 tokens per forward
        ref = _greedy_device(pair, tok, pos, n_new)
        assert list(got) == list(ref)
        # and the oracle's own greedy sequence, up to a near tie
        t = tok
        for i in range(n_new):
            lg = pair.oracle_step(t, pos + i)
            t = oracle.argmax(lg)
            if t != int(got[i]):
                assert top2_gap(lg) < 4e-2, (i, t, int(got[i]))
                break
    finally:
        pair.close()


def test_7b_int8_pld_with_planted_three_gram():
    cfg = synth.CONFIGS["7b_int8"]
    pair = Pair(cfg, with_oracle=False)
    try:
        P = cfg.prompt_len
        tau0 = synth.first_token(cfg)
        prompt, drafts = synth.planted_drafts(cfg, synth.make_prompt(cfg), tau0)
        n_new = 16
        got, st = pair.gpu.pld_generate([int(x) for x in prompt], P, tau0, n_new, 3, 1, 8)
        log("7b int8 pld: %s, first drafts %s" % (st, list(drafts[:4])))
        assert st["verifies"] >= 1 and st["drafted"] >= 8
        ref = _greedy_device(pair, tau0, P, n_new)
        assert list(got) == list(ref)
    finally:
        pair.close()
