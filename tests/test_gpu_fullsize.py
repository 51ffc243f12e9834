"""Full-size workloads on the GPU (needs an MI355X): the 1B-class and
7B-class decoders at 2K context, the 7B at 32K context, and the int8 7B with
a k = 8 verify of drafts from a planted 3-gram.  The oracle runs the first
steps of each on the host (one 7B step costs it about a second), so parity
is checked on 32 teacher-forced steps (8 at 32K context), each from
identical state, every logit and every new cache row, in the launch
configuration the benchmark times.  The greedy device loop (what the
benchmark times) then decodes the same steps free running and must produce
the same ids."""
import math

import numpy as np
import pytest
import torch

import synth
from tests.gpu_cases import Pair, Tally, check_step, check_verify, log, teacher_forced

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _free_running(pair, token, pos, n):
    toks = torch.zeros(n, dtype=torch.int32, device=pair.gpu.device)
    pair.gpu.greedy(token, pos, n, toks, pair.logits[0])
    pair.gpu.sync()
    return [int(t) for t in toks.cpu().numpy()]


@pytest.mark.parametrize("name,n_steps", [("1b", 32), ("7b", 32), ("7b_int8", 32),
                                          ("7b_32k", 8)])
def test_fullsize_teacher_forced(name, n_steps):
    cfg = synth.CONFIGS[name]
    pair = Pair(cfg)
    try:
        tau0 = synth.first_token(cfg)
        P = cfg.prompt_len
        tf = teacher_forced(pair, tau0, P, n_steps)
        log("%s: %s" % (name, tf.summary()))
        assert tf.agree >= math.ceil(0.99 * n_steps)
        # Free running from the same state: the device loop feeds its own
        # argmax back.  While the teacher-forced ids agreed, both runs
        # consumed the same tokens, so the ids must be the same.
        got = _free_running(pair, tau0, P, n_steps)
        first_div = next((i for i in range(n_steps) if got[i] != tf.ref_ids[i]), n_steps)
        log("%s: free-running greedy ids identical to the oracle's for the first %d of %d steps"
            % (name, first_div, n_steps))
        agree_prefix = next((i for i in range(n_steps) if tf.gpu_ids[i] != tf.ref_ids[i]),
                            n_steps)
        assert got[:agree_prefix + 1] == tf.gpu_ids[:agree_prefix + 1]
        # one more greedy step continues from that state and matches the
        # oracle's next step
        if first_div == n_steps:
            pos = P + n_steps
            nxt = tf.next
            toks = torch.zeros(1, dtype=torch.int32, device=pair.gpu.device)
            pair.gpu.greedy(nxt, pos, 1, toks, pair.logits[0])
            pair.gpu.sync()
            g = pair.logits[0].cpu().numpy()
            check_step(pair, g, int(toks.item()), nxt, pos, name + " greedy loop", Tally())
    finally:
        pair.close()


@pytest.mark.parametrize("name", ["7b_int8", "7b", "1b", "7b_32k"])
def test_verify_planted_3gram(name):
    """k = 8 verify of the planted 3-gram's drafts at the full shapes (the
    launch configuration the verify bench times): every row's logits and
    cache rows against the oracle from identical state, then the same
    verify again, bit for bit.  At 32K positions the attention takes one
    workgroup per CU, each wave streaming 16 key blocks."""
    cfg = synth.CONFIGS[name]
    pair = Pair(cfg)
    try:
        P = cfg.prompt_len
        tau0 = synth.first_token(cfg)
        _, drafts = synth.planted_drafts(cfg, synth.make_prompt(cfg), tau0)
        assert len(drafts) == 8
        tally = Tally()
        got = check_verify(pair, tau0, drafts, P, name + " verify", tally)
        log("%s verify: %s" % (name, tally.summary()))
        kv_rows = pair.gpu.kv_rows(P, P + 9)
        # the same verify again: bit-identical logits and cache rows
        pair.gpu.verify(tau0, drafts, P, pair.logits)
        pair.gpu.sync()
        again = pair.logits[:9].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), again.view(np.uint32))
        assert np.array_equal(kv_rows, pair.gpu.kv_rows(P, P + 9))
    finally:
        pair.close()


def test_tuned_split_keeps_parity():
    """After aio_tune_step moves gate/up rows between workgroups, decode still
    matches the oracle (the 1B-class decoder, teacher-forced steps)."""
    cfg = synth.CONFIGS["1b"]
    pair = Pair(cfg)
    try:
        tau0 = synth.first_token(cfg)
        pair.gpu.tune(tau0, cfg.prompt_len, pair.logits[0], 4)
        tf = teacher_forced(pair, tau0, cfg.prompt_len, 8)
        log("1b tuned: " + tf.summary())
        assert tf.agree >= math.ceil(0.99 * 8)
    finally:
        pair.close()
