"""Draft-model speculative decoding over two resident models (needs an
MI355X): the generated tokens equal the target's plain greedy decoding on
the device and the oracle's greedy sequence of the target, whether the
draft is another model (few drafts accepted) or a second copy of the target
(every draft accepted, which exercises the catch-up step of the draft
model)."""
import pytest
import torch

import oracle
import synth
from paper_2604_09752_amd import binding
from tests.gpu_cases import NEAR_TIE, Pair, log, top2_gap

pytestmark = pytest.mark.gpu


def _prefill(pair, prompt):
    for p, t in enumerate(prompt):
        pair.gpu_step(int(t), p)
        if pair.orc is not None:
            pair.oracle_step(int(t), p)


def _oracle_greedy(pair, token, pos, n):
    """The oracle's greedy ids and each step's logits, on a copy of its cache."""
    kv = pair.kv_host.copy()
    ids, logits, t = [], [], token
    for i in range(n):
        lg = pair.orc.decode_step(kv, t, pos + i)
        t = oracle.argmax(lg)
        ids.append(t)
        logits.append(lg)
    return ids, logits


def _greedy(pair, token, pos, n):
    toks = torch.zeros(n, dtype=torch.int32, device=pair.gpu.device)
    pair.gpu.greedy(token, pos, n, toks, pair.logits[0])
    pair.gpu.sync()
    return [int(x) for x in toks.cpu().numpy()]


@pytest.mark.parametrize("same", [False, True])
def test_spec_equals_target_greedy(same):
    ct = synth.CONFIGS["tiny"].with_(name="spec_t", prompt_len=24, n_steps=40)
    cd = ct if same else ct.with_(name="spec_d", seed=0xD1, n_layers=1, n_kv_heads=2)
    target, draft = Pair(ct), Pair(cd, with_oracle=False)
    try:
        prompt = synth.make_prompt(ct)
        _prefill(target, prompt[:-1])
        _prefill(draft, prompt[:-1])
        pos, tok, n_new = len(prompt) - 1, int(prompt[-1]), 40
        orc_ids, orc_logits = _oracle_greedy(target, tok, pos, n_new)
        for k in (4, 8):
            got, st = binding.spec_generate(target.gpu, draft.gpu, pos, tok, n_new, k)
            log("spec same=%s k=%d: %s" % (same, k, st))
            assert st["rounds"] + st["accepted"] == n_new
            if same:
                assert st["accepted"] >= 0.9 * st["drafted"]
            ref = _greedy(target, tok, pos, n_new)
            assert list(got) == ref
            # the oracle's greedy sequence of the target: identical up to the
            # first near tie (after a divergence the sequences part ways)
            same_ids = 0
            for i in range(n_new):
                if int(got[i]) != orc_ids[i]:
                    assert top2_gap(orc_logits[i]) < NEAR_TIE, (i, int(got[i]), orc_ids[i])
                    break
                same_ids += 1
            log("spec same=%s k=%d: identical to the oracle's greedy ids for %d of %d tokens"
                % (same, k, same_ids, n_new))
    finally:
        target.close()
        draft.close()
