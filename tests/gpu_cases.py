"""Shared helpers for the GPU parity tests: build the same seeded model for
the HIP path and the oracle, run teacher-forced steps on both, compare."""
from __future__ import annotations

import os
import sys
import time

import numpy as np
import torch

import oracle
import synth

LOGIT_TOL = 2e-2  # max-abs logit error for bf16 weights with fp32 accumulation


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

    def check_status(self):
        assert self.gpu.status() == 0, "a bounded wait of the step kernel gave up"

    def close(self):
        self.check_status()
        self.gpu.close()
        del self.gpu
        torch.cuda.empty_cache()


def compare_logits(got: np.ndarray, ref: np.ndarray):
    err = float(np.max(np.abs(got.astype(np.float64) - ref.astype(np.float64))))
    rms = float(np.sqrt(np.mean(ref.astype(np.float64) ** 2)))
    return err, rms


def kv_mismatches(kg: np.ndarray, ko: np.ndarray):
    """Entries of two bf16 caches (uint16 bits, [layer, K/V, kv head,
    position, head_dim]) that differ by more than one bf16 rounding of the
    value (2^-7 relative) plus an absolute term on the scale of the row.

    Layer 0 rows are computed from identical inputs on both sides, so the
    only difference is the fp32 accumulation error of the dot product that
    produced the entry; that error is absolute, on the scale of the row (a
    near-zero entry comes from cancellation), and is bounded by 2^-16 times
    the row's largest magnitude.

    Rows of deeper layers also inherit the earlier layers' cache: where an
    fp32 value lies within fp32 noise of a bf16 rounding boundary, the two
    sides may round it to neighbouring bf16 values (the one-rounding bound
    above), and attention over keys whose scores nearly tie amplifies such a
    one-ulp difference by the softmax's sensitivity.  Their absolute term is
    2^-6 times the row's largest magnitude."""
    fg = synth.bf16_bits_to_f32(kg).astype(np.float64)
    fo = synth.bf16_bits_to_f32(ko).astype(np.float64)
    row_scale = np.max(np.abs(fo), axis=-1, keepdims=True)
    absf = np.full((kg.shape[0],) + (1,) * (kg.ndim - 1), 2.0 ** -6)
    absf[0] = 2.0 ** -16
    bad = np.abs(fg - fo) > 2.0 ** -7 * np.maximum(np.abs(fg), np.abs(fo)) + absf * row_scale
    bad |= np.isnan(fg) != np.isnan(fo)
    idx = np.argwhere(bad)
    return idx, fg, fo


def assert_kv_close(kg: np.ndarray, ko: np.ndarray, what: str):
    idx, fg, fo = kv_mismatches(kg, ko)
    if len(idx):
        rows = ["%s: gpu %r oracle %r" % (tuple(i), fg[tuple(i)], fo[tuple(i)]) for i in idx[:12]]
        raise AssertionError("%s: %d KV entries differ by more than one bf16 rounding "
                             "(index = layer, K/V, kv head, position, dim):\n%s"
                             % (what, len(idx), "\n".join(rows)))


def top2_gap(x: np.ndarray) -> float:
    s = np.sort(x.astype(np.float64))
    return float(s[-1] - s[-2])


def logit_tol(cfg, ref_rms: float) -> float:
    """2e-2 for bf16 weights.  int8 weights (uniform on [-127, 127] times
    scales in (0.001, 0.01)) have ~20x the effective scale of N(0, 0.02)
    weights, so their logits are ~20x larger; the bound scales with the
    logit RMS (a bf16 model's logit RMS is about 1)."""
    return LOGIT_TOL * max(1.0, ref_rms) if cfg.wfmt == "int8" else LOGIT_TOL


def teacher_forced(pair: Pair, first_token: int, first_pos: int, n: int, tol=None):
    """n steps from first_pos; each step's token is the oracle's argmax of
    the previous step.  Returns (max err/tol, argmax agreement count, near
    ties, next token)."""
    tok, worst, agree, ties = first_token, 0.0, 0, 0
    for s in range(n):
        pos = first_pos + s
        g = pair.gpu_step(tok, pos)
        gi = int(pair.gpu_argmax(1)[0])
        r = pair.oracle_step(tok, pos)
        ri = oracle.argmax(r)
        err, rms = compare_logits(g, r)
        t = tol if tol is not None else logit_tol(pair.cfg, rms)
        worst = max(worst, err / t)
        if gi == ri:
            agree += 1
        elif top2_gap(r) < 4e-2:
            ties += 1
        log("[%s] step %d pos %d: max-abs %.3e (tol %.2e, logit rms %.3f) argmax %d/%d"
            % (pair.cfg.name, s, pos, err, t, rms, gi, ri))
        assert err <= t, "step %d pos %d: max-abs %.3e > %.1e (rms %.3f)" % (s, pos, err, t, rms)
        tok = ri
    return worst, agree, ties, tok
