"""Shared helpers for the GPU parity tests: build the same seeded model for
the HIP path and the oracle, run steps on both from identical state, compare.

Identical state.  Each compared step gives both sides the same token (the
oracle's argmax of the step before: teacher forcing) and the same cache
history: before the oracle computes position p, its cache rows for the
positions this comparison already wrote are the GPU's rows, each of which
was checked against the oracle's own row when it was written.  The row at p
itself is the GPU's too: layer by layer the oracle rounds its own K and V
(handed out for the check) and stores the GPU's entries before the layer
attends.  A cache row is the bf16 rounding of fp32 values that the two sides
compute in different orders, so a value close to a rounding boundary may
legitimately round to neighbouring bf16 values on the two sides; with int8
weights, whose attention is very peaked, one such flip of one entry moves
the next logits by more than 2e-2 (pinned on the oracle alone in
tests/test_int8_sensitivity.py), and a query that attends strongly to its
own key moves its own logits the same way.  So every step is compared from
the same state, and the drift of free-running caches is logged beside it.

The bounds:
  * logits, bf16 weights: max-abs error <= 2e-2 over every logit of every
    compared step and verify row (fp32 accumulation);
  * logits, int8 weights: max-abs error <= max(2e-2, 5e-3 x the oracle's
    logit RMS).  The int8 workload's attention can nearly tie two keys of
    very different values; at such steps fp32 rounding of the scores moves
    the logits by more than 2e-2 whatever the summation order: a plain
    numpy float32 evaluation of the same step from the same state lands up
    to 1.24e-3 x RMS (3.5e-2) from the oracle
    (tests/golden/int8_fp32_conditioning.json, written by
    tests/measure_int8_fp32.py).  The bound is 4x that.  Steps above 2e-2
    are counted apart;
  * KV cache: an entry may differ from the oracle's by one bf16 rounding of
    its value plus an absolute term times the largest magnitude of its row,
    checked for every row when it is written: 2^-16 in layer 0 (one fp32
    dot product of identical inputs), 2^-14 in deeper layers (they inherit
    the fp32 error of the step's earlier layers; measured up to 3.3e-5), and
    2^-10 in deeper layers with int8 weights (the same plain fp32 evaluation
    needs up to 1.8e-4 there);
  * greedy ids: wherever the oracle's top-2 gap exceeds twice the step's
    measured max-abs error, the ids must be identical (the bound then makes
    any other outcome impossible); the rest are near ties, reported apart.
Every comparison logs its error (absolute and relative to the logit RMS), so
the margin under each bound is on record."""
from __future__ import annotations

import os
import sys
import time

import numpy as np
import torch

import oracle
import synth

LOGIT_TOL = 2e-2  # max-abs logit error, bf16 weights (fp32 accumulation)
INT8_LOGIT_REL = 5e-3  # int8 weights: times the oracle's logit RMS (see above)
# Absolute KV term, times the row's largest magnitude: layer 0's rows are one
# fp32 dot product of identical inputs; deeper layers' rows also inherit the
# fp32 error of the step's earlier layers (measured up to 3.3e-5 x row max).
KV_ABS = 2.0 ** -16
KV_ABS_DEEP = 2.0 ** -14
KV_ABS_DEEP_INT8 = 2.0 ** -10
NEAR_TIE = 4e-2  # oracle top-2 gap below which a step counts as a near tie


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class env_set:
    """Temporarily set environment variables (read by the library at load)."""

    def __init__(self, **kw):
        self.kw = {k: v for k, v in kw.items() if v is not None}

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kw}
        os.environ.update(self.kw)

    def __exit__(self, *exc):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


class Pair:
    """The HIP model and the oracle on identical seeded inputs.  mega="1" /
    "0" selects the persistent step kernel / the per-operation kernels."""

    def __init__(self, cfg, with_oracle: bool = True, mega: str | None = None):
        from paper_2604_09752_amd.binding import DeviceModel
        t0 = time.time()
        self.cfg = cfg
        self.w = synth.make_weights(cfg)
        self.kv_host = synth.make_kv(cfg)
        log("[%s] inputs generated in %.1fs" % (cfg.name, time.time() - t0))
        with env_set(AIO_MEGA=mega):
            self.gpu = DeviceModel(cfg, self.w, kv_init=self.kv_host)
        log("[%s] persistent step kernel: %s" % (cfg.name, self.gpu.uses_step_kernel))
        self.orc = oracle.OracleModel(cfg, self.w) if with_oracle else None
        self.logits = self.gpu.new_logits(cfg.max_verify)
        self.tok_out = torch.zeros(max(cfg.max_verify, 1), dtype=torch.int32,
                                   device=self.gpu.device)
        log("[%s] device model loaded in %.1fs" % (cfg.name, time.time() - t0))

    def gpu_step(self, token: int, pos: int) -> np.ndarray:
        self.gpu.decode_step(token, pos, self.logits)
        self.gpu.sync()
        return self.logits[0].cpu().numpy().copy()

    def gpu_argmax(self, rows: int = 1) -> np.ndarray:
        self.gpu.argmax(self.logits, rows, self.tok_out)
        self.gpu.sync()
        return self.tok_out[:rows].cpu().numpy().copy()

    def oracle_step(self, token: int, pos: int) -> np.ndarray:
        return self.orc.decode_step(self.kv_host, token, pos)

    def oracle_step_row(self, token: int, pos: int, row: np.ndarray):
        """The oracle's step with the GPU's cache row at pos in place of its
        own roundings; returns (logits, the oracle's own row)."""
        return self.orc.decode_step_row(self.kv_host, token, pos, row)

    def check_status(self):
        assert self.gpu.status() == 0, "a bounded wait of the step kernel gave up"

    def close(self):
        self.check_status()
        self.gpu.close()
        del self.gpu
        torch.cuda.empty_cache()


def logit_tol(cfg, ref_rms: float) -> float:
    """The max-abs logit bound of a step (see the module docstring)."""
    if cfg.wfmt == "int8":
        return max(LOGIT_TOL, INT8_LOGIT_REL * ref_rms)
    return LOGIT_TOL


def kv_deep_abs(cfg) -> float:
    return KV_ABS_DEEP_INT8 if cfg.wfmt == "int8" else KV_ABS_DEEP


def compare_logits(got: np.ndarray, ref: np.ndarray):
    """(max-abs error, RMS of the oracle's logits)."""
    err = float(np.max(np.abs(got.astype(np.float64) - ref.astype(np.float64))))
    rms = float(np.sqrt(np.mean(ref.astype(np.float64) ** 2)))
    return err, rms


def _kv_excess(kg: np.ndarray, ko: np.ndarray):
    """Per entry of two bf16 caches (uint16 bits, [layer, K/V, kv head,
    position, head_dim]): how far |gpu - oracle| exceeds one bf16 rounding
    of the value (2^-7 relative), in units of the row's largest magnitude."""
    fg = synth.bf16_bits_to_f32(kg).astype(np.float64)
    fo = synth.bf16_bits_to_f32(ko).astype(np.float64)
    row_scale = np.max(np.abs(fo), axis=-1, keepdims=True)
    excess = np.abs(fg - fo) - 2.0 ** -7 * np.maximum(np.abs(fg), np.abs(fo))
    rel = np.where(row_scale > 0, excess / np.where(row_scale > 0, row_scale, 1.0),
                   np.where(excess > 0, np.inf, 0.0))
    rel = np.where(np.isnan(fg) != np.isnan(fo), np.inf, rel)
    return rel, fg, fo


def kv_abs_need(kg: np.ndarray, ko: np.ndarray) -> np.ndarray:
    """Per layer, the smallest absolute term (times the row maximum) under
    which every entry of the layer would pass; 0 where one bf16 rounding
    already covers every entry."""
    rel, _, _ = _kv_excess(kg, ko)
    return np.maximum(rel.reshape(rel.shape[0], -1).max(axis=1), 0.0)


def kv_mismatches(kg: np.ndarray, ko: np.ndarray, deep: float = KV_ABS_DEEP):
    """Entries that differ by more than one bf16 rounding of the value plus
    the absolute term of their layer (KV_ABS for layer 0, `deep` beyond)
    times the largest magnitude of the row.  A cache entry is the
    bf16 rounding of an fp32 value; the two sides' fp32 values differ by
    accumulation order only, and a value within that difference of a bf16
    rounding boundary may round to the neighbouring bf16 value (one
    rounding).  The absolute term covers the accumulation error itself,
    which is on the scale of the row (a near-zero entry comes from
    cancellation)."""
    rel, fg, fo = _kv_excess(kg, ko)
    bound = np.full((kg.shape[0],) + (1,) * (kg.ndim - 1), deep)
    bound[0] = KV_ABS
    idx = np.argwhere(rel > bound)
    return idx, fg, fo


def kv_check(kg: np.ndarray, ko: np.ndarray, what: str, deep: float = KV_ABS_DEEP) -> np.ndarray:
    """Raises if any entry is out of bound; returns kv_abs_need per layer."""
    idx, fg, fo = kv_mismatches(kg, ko, deep)
    if len(idx):
        rows = ["%s: gpu %r oracle %r" % (tuple(i), fg[tuple(i)], fo[tuple(i)]) for i in idx[:12]]
        raise AssertionError("%s: %d KV entries differ by more than one bf16 rounding plus "
                             "%.2e (layer 0) / %.2e x row max (index = layer, K/V, kv head, "
                             "position, dim):\n%s"
                             % (what, len(idx), KV_ABS, deep, "\n".join(rows)))
    return kv_abs_need(kg, ko)


def top2_gap(x: np.ndarray) -> float:
    s = np.sort(x.astype(np.float64))
    return float(s[-1] - s[-2])


def check_argmax(gpu_id: int, ref: np.ndarray, err: float, what: str) -> str:
    """Compares a GPU argmax with the oracle's.  Returns "agree", "tie" (a
    disagreement where the oracle's top-2 gap is within twice the measured
    error, so the bound admits either id) or raises: with a larger gap the
    max-abs bound leaves only the oracle's id possible."""
    ri = oracle.argmax(ref)
    if gpu_id == ri:
        return "agree"
    gap = top2_gap(ref)
    assert gap <= 2 * err, ("%s: argmax %d vs oracle %d with top-2 gap %.3e > 2 x max-abs %.3e"
                            % (what, gpu_id, ri, gap, err))
    return "tie"


class Tally:
    """Running record of a sequence of compared steps."""

    def __init__(self):
        self.worst = self.worst_rel = self.worst_free = self.kv_need = self.kv_need0 = 0.0
        self.n = self.agree = self.near_ties = self.disagree = self.over_2e2 = 0
        self.kv_same = self.kv_total = 0
        self.kv_deep = KV_ABS_DEEP
        self.gpu_ids, self.ref_ids = [], []

    def summary(self) -> str:
        s = ("%d steps: worst max-abs %.3e (%.2e of logit rms; %d steps above 2e-2), "
             "argmax agree %d/%d "
             "(disagreements at near ties %d, near-tie steps %d), new KV rows bit-identical "
             "%.5f, largest absolute KV term needed %.2e in layer 0 (bound %.2e), %.2e beyond "
             "(bound %.2e)"
             % (self.n, self.worst, self.worst_rel, self.over_2e2, self.agree, self.n,
                self.disagree, self.near_ties, self.kv_same / max(self.kv_total, 1),
                self.kv_need0, KV_ABS, self.kv_need, self.kv_deep))
        if self.worst_free:
            s += ", free-running caches: worst max-abs %.3e" % self.worst_free
        return s


def check_step(pair: Pair, g: np.ndarray, gi: int, tok: int, pos: int, what: str,
               tally: Tally, free_kv: np.ndarray | None = None) -> int:
    """Compares GPU logits g (and argmax gi) of consuming `tok` at `pos` with
    the oracle's from identical state, the state including the cache row the
    GPU wrote at pos (the oracle stores it in place of its own roundings,
    layer by layer, before the layer attends); checks that row against the
    oracle's own.
    With free_kv (a second oracle cache that is never forced) also logs the
    drift of free-running caches.  Returns the oracle's argmax."""
    kg = pair.gpu.kv_rows(pos, pos + 1)
    r, ko = pair.oracle_step_row(tok, pos, kg)
    ri = oracle.argmax(r)
    err, rms = compare_logits(g, r)
    gap = top2_gap(r)
    kind = check_argmax(gi, r, err, "%s pos %d" % (what, pos))
    tol = logit_tol(pair.cfg, rms)
    tally.kv_deep = kv_deep_abs(pair.cfg)
    ko = ko.reshape(kg.shape)
    need = kv_check(kg, ko, "%s pos %d" % (what, pos), tally.kv_deep)
    tally.kv_same += int((kg == ko).sum())
    tally.kv_total += kg.size
    tally.kv_need0 = max(tally.kv_need0, float(need[0]))
    tally.kv_need = max(tally.kv_need, float(need[1:].max()) if len(need) > 1 else 0.0)
    assert np.array_equal(pair.kv_host[:, :, :, pos:pos + 1, :], kg)
    free = ""
    if free_kv is not None:
        ef, _ = compare_logits(g, pair.orc.decode_step(free_kv, tok, pos))
        tally.worst_free = max(tally.worst_free, ef)
        free = ", free-running caches %.3e" % ef
    tally.n += 1
    tally.worst = max(tally.worst, err)
    tally.over_2e2 += err > LOGIT_TOL
    tally.worst_rel = max(tally.worst_rel, err / max(rms, 1e-30))
    tally.near_ties += gap < NEAR_TIE
    tally.agree += kind == "agree"
    tally.disagree += kind != "agree"
    tally.gpu_ids.append(gi)
    tally.ref_ids.append(ri)
    log("[%s] pos %d: max-abs %.3e (%.2e of logit rms %.3f) top-2 gap %.3e argmax %d/%d, "
        "KV term needed %.2e%s" % (what, pos, err, err / max(rms, 1e-30), rms, gap, gi, ri,
                                   float(need.max()), free))
    assert err <= tol, "%s pos %d: max-abs %.3e > %.2e (rms %.3f)" % (what, pos, err, tol, rms)
    return ri


def teacher_forced(pair: Pair, first_token: int, first_pos: int, n: int,
                   tokens=None, free_kv: np.ndarray | None = None) -> Tally:
    """n decode steps from first_pos, each compared from identical state
    (check_step).  The token of step s is tokens[s] when given (a prompt),
    else the oracle's argmax of the step before.  Returns the Tally; its
    attribute `next` is the oracle's argmax after the last step."""
    tally = Tally()
    tok = first_token
    for s in range(n):
        if tokens is not None:
            tok = int(tokens[s])
        pos = first_pos + s
        g = pair.gpu_step(tok, pos)
        gi = int(pair.gpu_argmax(1)[0])
        tok = check_step(pair, g, gi, tok, pos, pair.cfg.name, tally, free_kv)
    tally.next = tok
    return tally


def check_verify(pair: Pair, token: int, drafts, pos: int, what: str, tally: Tally,
                 free_kv: np.ndarray | None = None) -> np.ndarray:
    """One GPU verify of [token, drafts] at pos; every row compared with the
    oracle's decode step from identical state (the rows before it in the
    cache are the GPU's, checked when compared).  Returns the GPU logits."""
    pair.gpu.verify(token, drafts, pos, pair.logits)
    pair.gpu.sync()
    rows = 1 + len(drafts)
    got = pair.logits[:rows].cpu().numpy().copy()
    ids = pair.gpu_argmax(rows)
    toks = [int(token)] + [int(d) for d in drafts]
    for i in range(rows):
        check_step(pair, got[i], int(ids[i]), toks[i], pos + i, what, tally, free_kv)
    return got
