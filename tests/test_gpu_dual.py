"""Two models resident together (the paper's 1B probe and 7B backbone share
one device, Section 5.3): handles are independent, so steps of one model
interleaved with steps of the other give each model's own results (needs an
MI355X)."""
import numpy as np
import pytest

import synth
from tests.gpu_cases import LOGIT_TOL, Pair, compare_logits, log

pytestmark = pytest.mark.gpu


def test_interleaved_models_match_their_oracles():
    ca = synth.CONFIGS["tiny"].with_(name="dual_a", prompt_len=24, n_steps=8)
    cb = synth.CONFIGS["tiny"].with_(name="dual_b", seed=0xB10, n_heads=4, n_kv_heads=2,
                                     prompt_len=24, n_steps=8)
    a, b = Pair(ca), Pair(cb)
    try:
        pa, pb = synth.make_prompt(ca), synth.make_prompt(cb)
        worst = 0.0
        for p in range(len(pa)):
            for pair, prompt in ((a, pa), (b, pb)):
                got = pair.gpu_step(int(prompt[p]), p)
                ref = pair.oracle_step(int(prompt[p]), p)
                err, _ = compare_logits(got, ref)
                worst = max(worst, err)
                assert err <= LOGIT_TOL, (pair.cfg.name, p, err)
        log("interleaved two-model decode: worst max-abs %.3e over %d steps each" % (worst, len(pa)))
        # the two models' caches hold their own rows
        assert not np.array_equal(a.gpu.kv_numpy()[0, 0, 0, :4], b.gpu.kv_numpy()[0, 0, 0, :4])
    finally:
        a.close()
        b.close()
