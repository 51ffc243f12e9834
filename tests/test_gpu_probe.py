"""Prefill of a prompt through the verify forward in chunks (the probe's
single pass over its templated request), on the GPU: the logits after the
last token and the next decode step match the oracle (needs an MI355X)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_cases import LOGIT_TOL, Pair, compare_logits, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n", [1, 10, 23])
def test_prefill_matches_sequential_oracle(n):
    cfg = synth.CONFIGS["tiny"].with_(name="probe", prompt_len=24, n_steps=4)
    pair = Pair(cfg)
    try:
        prompt = [int(t) for t in synth.make_prompt(cfg)[:n]]
        pair.gpu.prefill(prompt, 0, pair.logits)
        pair.gpu.sync()
        got = pair.logits[0].cpu().numpy()
        ref = None
        for p, t in enumerate(prompt):
            ref = pair.oracle_step(t, p)
        err, _ = compare_logits(got, ref)
        log("prefill n=%d: last-token max-abs %.3e" % (n, err))
        assert err <= LOGIT_TOL
        # the cache it left is the one decode continues from
        nxt = oracle.argmax(ref)
        g = pair.gpu_step(nxt, n)
        r = pair.oracle_step(nxt, n)
        err2, _ = compare_logits(g, r)
        assert err2 <= LOGIT_TOL, err2
    finally:
        pair.close()
