"""Prefill of a prompt in prompt-length matrix products with causal
attention (the probe's single forward over its templated request), on the
GPU: every cache row the prefill writes and the logits after the last token
match the oracle's decode step of the same token from identical state (the
oracle's cache holds the prefill's own earlier rows, each checked when its
step is compared), and the next decode step continues from that state
(needs an MI355X).  The drift of a free-running oracle over the same tokens
is logged beside it, and held to the logit bound for bf16 weights."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_cases import (Pair, check_argmax, compare_logits, kv_check, kv_deep_abs, log,
                             logit_tol, teacher_forced)

pytestmark = pytest.mark.gpu

TINY = synth.CONFIGS["tiny"]

CASES = {
    # name: (config changes, tokens already in the cache, prompt tokens)
    "n1": (dict(), 0, 1),
    # up to max_verify (10) tokens the prefill is the verify forward
    "n10": (dict(), 0, 10),
    "n23": (dict(), 0, 23),
    "n128": (dict(), 0, 128),
    # the full 2K-token request of the routing rule, several 64-row tiles
    "n2048": (dict(prompt_len=2048, n_steps=8), 0, 2048),
    # a prompt that continues a cache already holding 37 positions
    "after37": (dict(), 37, 90),
    # d 320, FFN 192, vocab 1000, 5 heads (an odd number of 64-dim heads)
    "ragged": (dict(d_model=320, ffn_dim=192, vocab=1000, n_heads=5, n_kv_heads=5), 0, 77),
    # head_dim 128 with 4 query heads per kv head
    "hd128_gqa4": (dict(n_heads=4, n_kv_heads=1, head_dim=128), 0, 100),
    "int8": (dict(wfmt="int8"), 0, 23),
    # d 1024, FFN 4096: at a short prompt every product (QKV and gate/up as
    # well as O and down) has fewer tiles than two per CU and splits K over
    # workgroups, the last slice adding the partial tiles in slice order
    "split_k": (dict(d_model=1024, ffn_dim=4096, n_heads=8, n_kv_heads=8, head_dim=128), 0, 23),
    "split_k_int8": (dict(d_model=1024, ffn_dim=4096, n_heads=8, n_kv_heads=8, head_dim=128,
                          wfmt="int8"), 0, 70),
    # 1100 prompt rows (18 tiles of 64): 256-row weight tiles of 8 waves; K
    # split in two for O and down, while QKV (216 workgroups) and gate/up
    # (576) run unsplit in the XCD-renumbered order, whose last band holds 2
    # of the 18 row tiles; attention gives each XCD one of the 8 heads
    "wide_tiles": (dict(d_model=1024, ffn_dim=4096, n_heads=8, n_kv_heads=8, head_dim=128,
                        prompt_len=1100), 0, 1100),
    # 16 query heads on 8 kv heads (G = 2), hd 64: attention gives each XCD
    # two heads, which share one kv head
    "xcd_heads_gqa": (dict(d_model=1024, ffn_dim=2048, n_heads=16, n_kv_heads=8, head_dim=64,
                           prompt_len=300), 0, 300),
}


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_matches_sequential_oracle(name):
    kw, before, n = CASES[name]
    cfg = TINY.with_(name="pf_" + name, **kw)
    pair = Pair(cfg)
    try:
        prompt = [int(t) for t in synth.make_prompt(cfg)]
        toks = (prompt * ((before + n) // len(prompt) + 1))[:before + n]
        if before:
            teacher_forced(pair, toks[0], 0, before, tokens=toks)
        pair.gpu.prefill(toks[before:], before, pair.logits)
        pair.gpu.sync()
        got = pair.logits[0].cpu().numpy().copy()
        kg = pair.gpu.kv_rows(before, before + n)
        free = pair.kv_host.copy()
        ref = ref_free = None
        need = np.zeros(cfg.n_layers)
        same = 0
        for i in range(n):
            p = before + i
            # row p from identical state: rows before it are the prefill's own
            ref = pair.oracle_step(toks[p], p)
            ko = pair.kv_host[:, :, :, p:p + 1, :]
            need = np.maximum(need, kv_check(kg[:, :, :, i:i + 1, :], ko, "prefill %s pos %d"
                                             % (name, p), kv_deep_abs(cfg)))
            same += int((kg[:, :, :, i:i + 1, :] == ko).sum())
            pair.kv_host[:, :, :, p:p + 1, :] = kg[:, :, :, i:i + 1, :]
            ref_free = pair.orc.decode_step(free, toks[p], p)
        err, rms = compare_logits(got, ref)
        err_free, _ = compare_logits(got, ref_free)
        gi = int(pair.gpu_argmax(1)[0])
        kind = check_argmax(gi, ref, err, "prefill " + name)
        log("prefill %s (n=%d after %d): last-token max-abs %.3e (%.2e of logit rms), argmax %s, "
            "free-running oracle %.3e; KV rows bit-identical %.5f, KV term needed per layer %s"
            % (name, n, before, err, err / rms, kind, err_free, same / kg.size,
               " ".join("%.2e" % v for v in need)))
        assert err <= logit_tol(cfg, rms)
        if cfg.wfmt != "int8":
            assert err_free <= logit_tol(cfg, rms)
        # the state it left is the one decode continues from
        nxt = oracle.argmax(ref)
        pos = before + n
        g = pair.gpu_step(nxt, pos)
        r = pair.oracle_step(nxt, pos)
        err2, rms2 = compare_logits(g, r)
        log("prefill %s: next decode step max-abs %.3e" % (name, err2))
        assert err2 <= logit_tol(cfg, rms2)
    finally:
        pair.close()


def test_prefill_repeats_bit_for_bit():
    """The same prefill twice: identical logits and cache rows (no atomics)."""
    cfg = TINY.with_(name="pf_repeat")
    pair = Pair(cfg, with_oracle=False)
    try:
        toks = [int(t) for t in synth.make_prompt(cfg)[:100]]
        outs = []
        for _ in range(2):
            pair.gpu.prefill(toks, 0, pair.logits)
            pair.gpu.sync()
            outs.append((pair.logits[0].cpu().numpy().copy(), pair.gpu.kv_rows(0, 100)))
        assert np.array_equal(outs[0][0].view(np.uint32), outs[1][0].view(np.uint32))
        assert np.array_equal(outs[0][1], outs[1][1])
    finally:
        pair.close()


def test_category_entropy_on_device_matches_host_rule():
    """H(X) and the category of the label tokens' logits, computed on the
    device (aio_category_entropy), equal the host routing rule's on the
    same logits: prefill logits of a prompt, and planted cases (one
    dominant label, two tied leaders, all equal)."""
    import torch
    from paper_2604_09752_amd import binding as B
    cfg = TINY.with_(name="pf_entropy")
    pair = Pair(cfg, with_oracle=False)
    try:
        toks = [int(t) for t in synth.make_prompt(cfg)[:40]]
        pair.gpu.prefill(toks, 0, pair.logits)
        pair.gpu.sync()
        row = pair.logits[0]
        out = torch.zeros(2, dtype=torch.float32, device=pair.gpu.device)
        cases = [list(range(3)), [5, 17, 901, 2, 77], list(range(0, cfg.vocab, cfg.vocab // 40))]
        planted = torch.zeros(cfg.vocab, dtype=torch.float32, device=pair.gpu.device)
        planted[:8] = torch.tensor([3.0, 3.0, -1.0, 0.5, 0.5, 0.5, 0.5, 0.5])
        for logits, labels in [(row, c) for c in cases] + [(planted, [0, 1, 2]), (planted, [3, 4, 5, 6])]:
            B.aio_category_entropy(pair.gpu.handle, logits, labels, out)
            pair.gpu.sync()
            h_dev, cat_dev = [float(v) for v in out.cpu().numpy()]
            _, h, cat = B.aio_probe_route(logits.cpu().numpy()[labels], 0, 10)
            assert int(cat_dev) == cat
            assert abs(h_dev - h) <= 1e-6 * max(1.0, abs(h)), (h_dev, h)
        # all equal: ln C exactly as the host gives it
        B.aio_category_entropy(pair.gpu.handle, planted, [3, 4, 5, 6], out)
        pair.gpu.sync()
        assert abs(float(out[0]) - np.log(4.0)) < 1e-6 and int(out[1]) == 0
    finally:
        pair.close()
