"""aio_prefill_noalloc, the prefill entry point that allocates nothing (its
scratch is the library's fixed device array), against aio_prefill (library-
allocated scratch) on the same inputs, through the C ABI (needs an MI355X).
Two calls in a row, the second with a smaller prompt: the first takes the
prompt in several passes of the array's capacity, the second in one."""
import numpy as np
import pytest

import synth
from tests.gpu_cases import (LOGIT_TOL, Pair, compare_logits, kv_check, kv_deep_abs, log)

pytestmark = pytest.mark.gpu

# 2 layers, d 1024, 8 x 128 heads, FFN 4096: about 32 KB of scratch per
# row, so the 32 MiB array takes 1021 rows per pass
CFG = synth.CONFIGS["tiny"].with_(name="noalloc", d_model=1024, n_heads=8, n_kv_heads=8,
                                  head_dim=128, ffn_dim=4096, prompt_len=1100, n_steps=8)


def test_noalloc_prefill_matches_allocating_prefill():
    ref = Pair(CFG, with_oracle=False)
    got = Pair(CFG, with_oracle=False)
    try:
        rows = got.gpu.prefill_noalloc_rows
        log("noalloc: %d rows per pass" % rows)
        assert 0 < rows < 1050
        prompt = [int(t) for t in synth.make_prompt(CFG)]
        # call 1: 1050 tokens from position 0 (two passes); call 2: 50
        # tokens continuing at 1050 (one pass)
        for start, n in ((0, 1050), (1050, 50)):
            toks = prompt[start:start + n]
            ref.gpu.prefill(toks, start, ref.logits)
            got.gpu.prefill_noalloc(toks, start, got.logits)
            ref.gpu.sync()
            got.gpu.sync()
            a = ref.logits[0].cpu().numpy()
            b = got.logits[0].cpu().numpy()
            err, rms = compare_logits(b, a)
            ka = ref.gpu.kv_rows(start, start + n)
            kb = got.gpu.kv_rows(start, start + n)
            need = kv_check(kb, ka, "noalloc prefill at %d" % start, kv_deep_abs(CFG))
            log("noalloc prefill of %d tokens at %d: logits max-abs %.3e vs aio_prefill "
                "(bit-identical %s), KV bit-identical %.5f, KV term needed %s"
                % (n, start, err, np.array_equal(a.view(np.uint32), b.view(np.uint32)),
                   float((ka == kb).mean()), " ".join("%.2e" % v for v in need)))
            assert err <= LOGIT_TOL
        # the two models' caches hold the same sequence: decoding continues alike
        a = ref.gpu_step(prompt[-1], 1100)
        b = got.gpu_step(prompt[-1], 1100)
        assert compare_logits(b, a)[0] <= LOGIT_TOL
    finally:
        ref.close()
        got.close()
