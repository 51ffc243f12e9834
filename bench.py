#!/usr/bin/env python3
"""Batch-1 decode throughput on one MI355X.

A step is one decode step of the whole path -- embedding, every layer's
RMSNorm + QKV GEMV + RoPE + KV append, split-KV attention + merge, O GEMV,
RMSNorm + gate/up GEMV + SwiGLU, down GEMV, then final RMSNorm + LM head and
the greedy argmax that feeds the next step -- on the 7B-class decoder with
2048 positions of KV (the workload the paper's 7B TPS figures are quoted on).
Inputs (weights, KV cache) are resident in HBM before the timed region; the
loop is device-resident (captured graph replayed per step, argmax feeding the
next token on the device).

Prints one JSON line.  The HBM roofline figure is for the dominant kernel --
the persistent step kernel, which is the whole step (or, on the per-operation
path, the fused gate/up GEMV) -- timed with HIP events on the model's stream;
its `traffic` is the HBM bytes per launch that rocprofv3's FETCH_SIZE and
WRITE_SIZE counters read for this kernel (calibrated against a plain copy),
reported only while the kernel's device sources are the ones measured.  The
CPU baseline is the oracle, timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
PAPER_7B_TPS = 17.18   # A-IO Table core_perf: 7B FP16 decode at 2K on Ascend 910B
METRIC = "decode tokens/s at batch 1 and achieved HBM GB/s (% of peak), 7B-class @2K"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_name(cfg) -> str:
    return ("%s dense decoder (L%d d%d H%d/Hkv%d hd%d F%d V%d), %s weights, %d-position KV, "
            "batch 1, greedy decode" % (cfg.name, cfg.n_layers, cfg.d_model, cfg.n_heads,
                                        cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim, cfg.vocab,
                                        cfg.wfmt, cfg.prompt_len))


def measured_traffic(config: str, kernel_used: bool):
    """HBM bytes per step-kernel launch from the committed counter record of
    this workload, or None when there is none or the kernel's sources changed
    since it was taken."""
    from paper_2604_09752_amd import profile_record
    if not kernel_used or config not in profile_record.WORKLOADS:
        return None
    path = profile_record.record_path(config)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("sources_sha256") != profile_record.sources_sha256():
        return None
    return int(rec["traffic_bytes_per_launch"])


def calibrate_copy(nbytes: int) -> int:
    """A plain copy of a known number of bytes: read nbytes, write nbytes.
    Profiled with the same HBM counters as the decode step, it gives the
    factor between counter readings and bytes actually moved."""
    import torch
    if not torch.cuda.is_available():
        print("--calibrate-copy needs a GPU", file=sys.stderr)
        return 2
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    reps = 5
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    print(json.dumps({"copy_bytes": nbytes, "launches": reps + 1, "read_plus_write_gbs":
                      round(2 * nbytes / dt / 1e9, 1)}), flush=True)
    return 0


def pld_bench(dm, cfg, P, tau0, n, toks, logits) -> dict:
    """Prompt-lookup decoding (host loop over aio_verify) against plain greedy
    decoding of the same n tokens.  Random weights accept almost no drafts
    from a random prompt, so the history is also given with the greedy
    continuation planted behind a copy of its last two tokens and tau0: every
    draft is then accepted.  The two runs bound PLD's speed on this model."""
    import torch
    import synth
    k = min(cfg.verify_k, cfg.max_verify - 1)
    prompt = [int(t) for t in synth.make_prompt(cfg)]
    g = torch.zeros(n, dtype=torch.int32, device=dm.device)
    dm.greedy(tau0, P, n, g, logits)
    dm.sync()
    t0 = time.perf_counter()
    dm.greedy(tau0, P, n, g, logits)
    dm.sync()
    t_greedy = time.perf_counter() - t0
    cont = [int(x) for x in g.cpu().numpy()]
    j = 64
    planted = prompt[:j] + [prompt[-2], prompt[-1], tau0] + cont + prompt[j + 3 + n:]
    planted = planted[:P]
    out = {"tokens": n, "k": k, "ngram": 3, "greedy_tokens_per_s": round(n / t_greedy, 2)}
    for name, hist in (("random_prompt", prompt), ("planted_continuation", planted)):
        dm.pld_generate(hist, P, tau0, min(n, 8), 3, 1, k)  # warm-up
        t0 = time.perf_counter()
        got, st = dm.pld_generate(hist, P, tau0, n, 3, 1, k)
        dt = time.perf_counter() - t0
        out[name] = {"tokens_per_s": round(n / dt, 2), "identical_to_greedy": bool(list(got) == cont),
                     "acceptance": round(st["accepted"] / max(1, st["drafted"]), 3), **st}
        log("pld %s: %.1f tokens/s (greedy %.1f), %s" % (name, n / dt, n / t_greedy, st))
    return out


def dual_bench(r: int, rounds: int = 8) -> int:
    """Both models of the paper's deployment resident in HBM at once (its
    Section 5.3 measures 2.4 ms for switching between them): requests of r
    greedy tokens (one device-resident loop and a synchronisation each),
    first back to back on one model, then alternating between the 7B-class
    and the 1B-class decoder.  The switch cost is what an alternating pair
    of requests costs beyond one request of each on its own."""
    import torch
    import synth
    from paper_2604_09752_amd.binding import DeviceModel
    models = {}
    for name in ("7b", "1b"):
        cfg = synth.CONFIGS[name]
        dm = DeviceModel(cfg, synth.make_weights(cfg), kv_init=synth.make_kv(cfg))
        models[name] = (dm, cfg.prompt_len, synth.first_token(cfg), dm.new_logits(1)[0],
                        torch.zeros(r, dtype=torch.int32, device=dm.device))
        log("%s resident: %.1f GB of weights" % (name, sum(
            t.numel() * t.element_size() for t in dm.dev.values()) / 1e9))

    def request(name):
        dm, P, tau0, lg, toks = models[name]
        dm.greedy(tau0, P, r, toks, lg)
        dm.sync()

    for name in models:  # warm-up: graphs, kernels, caches
        request(name)
    alone = {}
    for name in models:
        t0 = time.perf_counter()
        for _ in range(rounds):
            request(name)
        alone[name] = (time.perf_counter() - t0) / rounds
    t0 = time.perf_counter()
    for _ in range(rounds):
        request("7b")
        request("1b")
    pair = (time.perf_counter() - t0) / rounds
    out = {"request_tokens": r, "rounds": rounds,
           "ms_per_request_7b": round(1e3 * alone["7b"], 3),
           "ms_per_request_1b": round(1e3 * alone["1b"], 3),
           "ms_per_alternating_pair": round(1e3 * pair, 3),
           "switch_us": round(1e6 * (pair - alone["7b"] - alone["1b"]) / 2, 1),
           "resident": {n: models[n][0].cfg.name for n in models}}
    rc = 0
    for dm, *_ in models.values():
        rc = rc or (3 if dm.status() != 0 else 0)
        dm.close()
    print(json.dumps(out), flush=True)
    return rc


def probe_bench(n: int, reps: int = 5) -> int:
    """The probe's front end (Section 3.2): the 1B-class decoder consumes an
    n-token request (seeded random tokens standing in for the templated
    prompt) from position 0 in prompt-length matrix products (aio_prefill),
    then the routing rule reads the logits of three seeded label tokens.  The
    paper measures 11.8 ms for its probe's prefill (Section 5.3).  Reported
    besides the time: the algorithmic flops of the prefill (2 n x the linear
    parameters, causal attention, the last row's LM head) per second, and the
    MFMA rate (the products run on two bf16 terms of every activation, twice
    the algorithmic flops of the linear layers)."""
    import torch
    import synth
    from paper_2604_09752_amd import binding
    from paper_2604_09752_amd.binding import DeviceModel
    cfg = synth.CONFIGS["1b"]
    n = min(n, cfg.max_ctx)
    dm = DeviceModel(cfg, synth.make_weights(cfg))
    toks = synth.tokens(cfg.seed + 3, "probe_request", n, cfg.vocab)
    labels = synth.tokens(cfg.seed + 3, "probe_labels", 3, cfg.vocab)
    lg = dm.new_logits(cfg.max_verify)
    dm.prefill(toks, 0, lg)
    dm.sync()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(dm.stream)
    for _ in range(reps):
        dm.prefill(toks, 0, lg)
    ev1.record(dm.stream)
    dm.sync()
    ms = ev0.elapsed_time(ev1) / reps
    # H(X) and the category on the device: only two floats cross to the host
    hc = torch.zeros(2, dtype=torch.float32, device=dm.device)
    binding.aio_category_entropy(dm.handle, lg[0], labels, hc)  # first launch loads the kernel
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    binding.aio_category_entropy(dm.handle, lg[0], labels, hc)
    h_dev, cat_dev = [float(v) for v in hc.cpu().numpy()]
    small = cat_dev == 0 and n <= 2048 and h_dev <= 0.45
    route_us = (time.perf_counter() - t0) * 1e6
    # the host rule on the same logits gives the same values
    _, h, cat = binding.aio_probe_route(lg[0].cpu().numpy()[labels], 0, n)
    if abs(h - h_dev) > 1e-6 * max(1.0, abs(h)) or cat != int(cat_dev):
        log("device entropy %r / category %r differ from the host's %r / %r" % (h_dev, cat_dev, h, cat))
        return 3
    d, hd, L = cfg.d_model, cfg.head_dim, cfg.n_layers
    lin = L * (d * cfg.n_heads * hd + 2 * d * cfg.n_kv_heads * hd + cfg.n_heads * hd * d
               + 3 * d * cfg.ffn_dim)
    attn = 4 * L * cfg.n_heads * hd * (n * (n + 1) // 2)
    flops = 2 * n * lin + attn + 2 * cfg.vocab * d
    out = {"request_tokens": n, "prefill_ms": round(ms, 3),
           "tokens_per_s": round(n / ms * 1e3, 1),
           "algorithmic_tflops": round(flops / ms / 1e9, 1),
           "mfma_tflops": round((4 * n * lin + 2 * attn) / ms / 1e9, 1),
           "entropy_nats": round(h_dev, 4), "category": int(cat_dev),
           "route_to_small_model": bool(small), "route_decision_us": round(route_us, 1),
           "workload": workload_name(cfg)}
    rc = 3 if dm.status() != 0 else 0
    dm.close()
    print(json.dumps(out), flush=True)
    return rc


def spec_bench(n: int, k: int = 4) -> int:
    """The paper's DraftModel baseline (Section 4.2; about 4 TPS on its
    system, Section 2.2): the 1B-class decoder drafts k tokens, the 7B-class
    decoder verifies them in one forward.  Both hold the same synthetic 2K
    context.  With unrelated random weights the target accepts almost
    nothing, so this times the mechanism's cost per token against the 7B's
    plain greedy loop."""
    import torch
    import synth
    from paper_2604_09752_amd import binding
    from paper_2604_09752_amd.binding import DeviceModel
    ct, cd = synth.CONFIGS["7b"], synth.CONFIGS["1b"]
    target = DeviceModel(ct, synth.make_weights(ct), kv_init=synth.make_kv(ct))
    draft = DeviceModel(cd, synth.make_weights(cd), kv_init=synth.make_kv(cd))
    P, tau0 = ct.prompt_len, synth.first_token(ct)
    n = min(n, ct.max_ctx - P - k - 1)
    lg = target.new_logits(1)[0]
    toks = torch.zeros(n, dtype=torch.int32, device=target.device)
    target.greedy(tau0, P, n, toks, lg)
    target.sync()
    t0 = time.perf_counter()
    target.greedy(tau0, P, n, toks, lg)
    target.sync()
    t_greedy = time.perf_counter() - t0
    ref = [int(x) for x in toks.cpu().numpy()]
    binding.spec_generate(target, draft, P, tau0, min(n, 8), k)  # warm-up
    t0 = time.perf_counter()
    got, st = binding.spec_generate(target, draft, P, tau0, n, k)
    dt = time.perf_counter() - t0
    out = {"tokens": n, "k": k, "target": "7b", "draft": "1b",
           "greedy_tokens_per_s": round(n / t_greedy, 2), "spec_tokens_per_s": round(n / dt, 2),
           "identical_to_greedy": list(got) == ref,
           "acceptance": round(st["accepted"] / max(1, st["drafted"]), 3), **st}
    rc = 3 if (target.status() != 0 or draft.status() != 0) else 0
    target.close()
    draft.close()
    print(json.dumps(out), flush=True)
    return rc


def verify_bench(dm, cfg, P, tau0, n) -> int:
    """Time n verify forwards (one warm-up first) of tau0 and the k drafts of
    the planted 3-gram at position P; one JSON line."""
    import torch
    import synth
    from paper_2604_09752_amd import traffic
    _, drafts = synth.planted_drafts(cfg, synth.make_prompt(cfg), tau0)
    k = len(drafts)
    lg = dm.new_logits(k + 1)
    dm.verify(tau0, drafts, P, lg)
    dm.sync()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(dm.stream)
    for _ in range(n):
        dm.verify(tau0, drafts, P, lg)
    ev1.record(dm.stream)
    dm.sync()
    ms = ev0.elapsed_time(ev1) / n
    b = traffic.verify_bytes(cfg, P, k + 1)
    status = dm.status()
    dm.close()
    print(json.dumps({"verify_rows": k + 1, "position": P, "runs": n, "ms_per_verify": round(ms, 4),
                      "bytes_per_verify": int(b), "gbs": round(b / (ms * 1e-3) / 1e9, 1),
                      "frac_of_peak": round(b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                      "workload": workload_name(cfg)}), flush=True)
    return 0 if status == 0 else 3


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", default="7b", help="tiny, 1b, 7b, 7b_32k or 7b_int8")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="wall-clock budget of the oracle's CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=3)
    ap.add_argument("--tune-rounds", type=int, default=4,
                    help="calibration steps of the step kernel's gate/up split before timing "
                         "(aio_tune_step); 0 keeps the even split")
    ap.add_argument("--pld", type=int, default=0, metavar="N",
                    help="also time N tokens of prompt-lookup decoding (3-gram drafts, k = 8), "
                         "with and without the greedy continuation planted in the history")
    ap.add_argument("--verify-runs", type=int, default=0, metavar="N",
                    help="instead of the decode bench, time N verify forwards of the token and "
                         "the k drafts of the planted 3-gram at the prompt's end, and exit")
    ap.add_argument("--dual", type=int, default=0, metavar="N",
                    help="instead of the decode bench, keep the 1B-class and the 7B-class "
                         "decoders resident together and time requests of N greedy tokens, back "
                         "to back on one model and alternating between them; one JSON line")
    ap.add_argument("--spec", type=int, default=0, metavar="N",
                    help="instead of the decode bench, time N tokens of the 7B-class decoder "
                         "with drafts (k = 4) from the resident 1B-class decoder, beside the "
                         "7B's plain greedy loop; one JSON line")
    ap.add_argument("--probe", type=int, default=0, metavar="N",
                    help="instead of the decode bench, time the 1B-class probe's prefill of an "
                         "N-token request and its routing decision; one JSON line")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="instead of the decode bench, run a plain device-to-device copy of "
                         "BYTES (the reference kernel for HBM counter calibration) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        return calibrate_copy(args.calibrate_copy)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the decode step runs on a single MI355X and has no "
              "multi-GPU path (requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world),
              file=sys.stderr)
        return 2

    import torch

    import synth
    from paper_2604_09752_amd import traffic
    from paper_2604_09752_amd.binding import KERNELS_PER_LAYER, DeviceModel

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    if args.dual > 0:
        return dual_bench(args.dual)
    if args.spec > 0:
        return spec_bench(args.spec)
    if args.probe > 0:
        return probe_bench(args.probe)
    cfg = synth.CONFIGS[args.config]
    P = cfg.prompt_len if not cfg.prefill_by_model else 0
    if args.verify_runs > 0 and P == 0:
        print("--verify-runs needs a workload with its prompt already in the cache", file=sys.stderr)
        return 2
    t0 = time.time()
    w = synth.make_weights(cfg)
    kv_host = synth.make_kv(cfg)
    log("inputs generated in %.1fs" % (time.time() - t0))
    dm = DeviceModel(cfg, w, kv_init=kv_host)
    log("device model ready in %.1fs" % (time.time() - t0))
    tau0 = synth.first_token(cfg)
    if args.verify_runs > 0:
        return verify_bench(dm, cfg, P, tau0, args.verify_runs)
    chunk = min(cfg.n_steps, cfg.max_ctx - P)
    logits = dm.new_logits(1)[0]
    toks = torch.zeros(max(chunk, args.warmup, 1), dtype=torch.int32, device=dm.device)

    # warm-up (graph capture happens on the first greedy call)
    if args.warmup > 0:
        dm.greedy(tau0, P, min(args.warmup, chunk), toks, logits)
    dm.sync()
    tuned = dm.uses_step_kernel and args.tune_rounds > 0
    if tuned:  # writes the same cache row at P that every timed chunk starts with
        dm.tune(tau0, P, logits, args.tune_rounds)

    # timed region: exactly args.steps steps, in chunks restarting at P
    plan, left = [], args.steps
    while left > 0:
        n = min(left, chunk)
        plan.append(n)
        left -= n
    first_tokens = None
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(dm.stream)
    t_start = time.perf_counter()
    for n in plan:
        dm.greedy(tau0, P, n, toks, logits)
    ev1.record(dm.stream)
    dm.sync()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    elapsed = t_end - t_start
    gpu_elapsed = ev0.elapsed_time(ev1) / 1e3
    first_tokens = toks[: plan[0]].cpu().numpy().copy()
    step_bytes = sum(traffic.run_bytes(cfg, P, n) for n in plan)
    tps = args.steps / elapsed
    log("timed %d steps: %.3f ms/step wall, %.3f ms/step events, %.1f tokens/s, %.0f GB/s"
        % (args.steps, 1e3 * elapsed / args.steps, 1e3 * gpu_elapsed / args.steps, tps,
           step_bytes / elapsed / 1e9))

    # dominant kernel, timed with HIP events on dm.stream
    L = cfg.n_layers
    wb = 1 if cfg.wfmt == "int8" else 2
    phases = None
    if dm.uses_step_kernel:
        # the whole step is one persistent kernel: its bytes are the step's
        kname = "k_step (whole decode step: all layers + LM head + argmax)"
        durs = [float(dm.profile_step(tau0, P, logits)[0]) for _ in range(args.profile_steps)]
        k_us = 1e3 * float(np.mean(durs))
        k_bytes = traffic.step_bytes(cfg, P)
        tr = np.stack([dm.trace_step(tau0, P, logits) for _ in range(args.profile_steps)]).mean(0)
        # between barrier exits: attention, O, gate/up, down, next layer's QKV
        names = ("attn", "o", "gateup", "down", "qkv")
        phases = {n: round(float(tr[i::5].mean()), 2) for i, n in enumerate(names)}
        log("per-phase average us: " + ", ".join("%s %.1f" % kv for kv in phases.items()))
        kinds = {"k_step": k_us}
    else:
        kname = "gate/up GEMV + RMSNorm prologue + SwiGLU epilogue"
        per_kernel = np.stack([dm.profile_step(tau0, P, logits)
                               for _ in range(args.profile_steps)])  # [iters][6L + 1] ms
        kinds = {}
        for i, name in enumerate(KERNELS_PER_LAYER):
            kinds[name] = float(per_kernel[:, i:6 * L:6].mean() * 1e3)
        kinds["lm_head"] = float(per_kernel[:, 6 * L].mean() * 1e3)
        k_bytes = 2 * cfg.ffn_dim * cfg.d_model * wb + 2 * cfg.d_model
        if cfg.wfmt == "int8":
            k_bytes += 2 * 2 * cfg.ffn_dim
        k_us = kinds["gateup"]
    achieved = k_bytes / (k_us * 1e-6) / 1e9
    log("dominant kernel %s: %.1f us per launch, %.0f GB/s" % (kname, k_us, achieved))

    result = {
        "metric": METRIC,
        "value": round(tps, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": round(tps / PAPER_7B_TPS, 2) if args.config == "7b" else None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": workload_name(cfg),
            "weights": cfg.wfmt,
            "kv_cache": "bf16",
            "prompt_positions": P,
            "steps_per_restart": chunk,
            "gate_up_split": "calibrated (%d steps)" % args.tune_rounds if tuned else "even",
        },
        "hbm_gbs": round(step_bytes / elapsed / 1e9, 1),
        "hbm_frac_of_peak": round(step_bytes / elapsed / 1e9 / HBM_PEAK_GBS, 4),
        "bytes_per_step": int(step_bytes // args.steps),
        "roofline": {
            "bound": "hbm",
            "kernel": kname,
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(args.config, dm.uses_step_kernel),
            "bytes_per_launch": int(k_bytes),
            "avg_launch_us": round(k_us, 2),
        },
        "kernel_avg_us": {k: round(v, 2) for k, v in kinds.items()},
        "phase_avg_us": phases,
    }
    if args.config == "7b":
        result["baseline_note"] = ("vs_baseline divides by the paper's 7B FP16 decode TPS at 2K "
                                   "(17.18, Ascend 910B, HF Transformers eager): context, "
                                   "another machine")

    if args.pld > 0:
        result["pld"] = pld_bench(dm, cfg, P, tau0, min(args.pld, cfg.max_ctx - P - 1), toks, logits)

    if not args.no_cpu_baseline:
        import oracle
        orc = oracle.OracleModel(cfg, w)
        kv_o = kv_host  # the oracle appends to the host copy
        tok, n_done, agree = tau0, 0, 0
        c0 = time.perf_counter()
        while n_done < args.steps and (n_done == 0 or time.perf_counter() - c0 < args.cpu_seconds):
            lg = orc.decode_step(kv_o, tok, P + n_done)
            tok = oracle.argmax(lg)
            if n_done < len(first_tokens) and tok == int(first_tokens[n_done]):
                agree += 1
            n_done += 1
        c1 = time.perf_counter()
        cpu_tps = n_done / (c1 - c0)
        result["cpu_baseline"] = {
            "value": round(cpu_tps, 4),
            "unit": "tokens/s",
            "cores": oracle.num_threads(),
            "cpu_model": cpu_model(),
            "kind": "oracle",
            "sample": "first %d greedy decode steps from position %d of the same workload "
                      "(%.1f s)" % (n_done, P, c1 - c0),
        }
        result["greedy_parity"] = {"steps": n_done, "identical_tokens": agree}
        log("oracle: %d steps in %.1fs (%.3f tokens/s, %d threads), greedy ids identical %d/%d"
            % (n_done, c1 - c0, cpu_tps, oracle.num_threads(), agree, n_done))
    status = dm.status()
    dm.close()
    if status != 0:
        print("device status %d: a bounded wait of the step kernel gave up; the run is invalid" % status,
              file=sys.stderr)
        return 3
    print(json.dumps(result), flush=True)
    return 0


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or the platform's processor."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


if __name__ == "__main__":
    sys.exit(main())
