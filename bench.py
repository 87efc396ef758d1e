"""Benchmark: scored tokens/s of the ACRL scoring path on one MI355X.

One step = the whole hot path over one batch already resident in HBM:
quantize H for mu (per-tensor FP8), score every valid token under pi (BF16)
and mu (FP8) with the fused log-softmax, merge, reduce the discrepancy per
sequence / group / batch, and apply the ACRL controller.  W's quantization
and its packed tile image happen once per weight version and are reported
separately.  After the headline workload (q8b), the other full-size
workloads (q17b, long, mx) run the same step and land under "workloads".

Usage: python bench.py [--gpus 1] [--steps 5] [--warmup 2] [--workload q8b]
Prints progress on stderr and ONE JSON line on stdout.

python bench.py --counters runs a plain copy of known size and one step, for
the FETCH_SIZE / WRITE_SIZE passes that give roofline.traffic (see
paper_2607_24062_amd/profiling.py); the traffic is read back from
profiles/score_<workload>_traffic.md while it matches the kernel sources.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

import inputs

PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}   # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def setup(torch, acrl, w, dev):
    """The workload resident in HBM: inputs, W's quantization and packed
    image (once per weight version, timed apart) and the rollout's ids drawn
    from mu (untimed)."""
    T = inputs.n_valid(w)
    d, V = w.d, w.V
    t0 = time.time()
    H = inputs.hidden_bf16_torch(w, T, dev)
    W = inputs.weights_bf16_torch(w, dev)
    slots = torch.from_numpy(inputs.valid_slots(w)).to(dev)
    mask = torch.from_numpy(inputs.mask(w).reshape(-1)).to(dev)
    groups = torch.from_numpy(inputs.group_of_seq(w)).to(dev)
    adv = torch.from_numpy(inputs.advantages(w)).to(dev)
    torch.cuda.synchronize()
    log("[%s] inputs generated in %.1fs" % (w.name, time.time() - t0))
    ev = lambda: torch.cuda.Event(enable_timing=True)
    a, b, c = ev(), ev(), ev()
    wq, ws = acrl.acrl_quantize_fp8(W, w.scaling)
    packed = acrl.acrl_pack_weights(W, wq, ws, w.scaling)
    torch.cuda.synchronize()
    a.record()
    acrl.acrl_quantize_fp8(W, w.scaling, q=wq, scales=ws)
    b.record()
    acrl.acrl_pack_weights(W, wq, ws, w.scaling, packed=packed)
    c.record()
    torch.cuda.synchronize()
    wq_ms, pw_ms = a.elapsed_time(b), b.elapsed_time(c)
    wq_bytes = V * d * (2 + 1) + (V * d * 2 if w.scaling == inputs.PER_TENSOR else 0)
    log("[%s] quantize W: %.3f ms (%.0f GB/s); pack W, Wq: %.3f ms" % (w.name, wq_ms, wq_bytes / wq_ms / 1e6, pw_ms))
    hq0, hs0 = acrl.acrl_quantize_fp8(H, w.scaling)
    a.record()
    ids, _ = acrl.acrl_sample_mu(hq0, hs0, wq, ws, w.scaling, seed=w.seed, inv_temperature=w.inv_temperature,
                                 want_logp=False, packed_weights=packed)
    b.record()
    torch.cuda.synchronize()
    sample_ms = a.elapsed_time(b)
    del hq0, hs0
    log("[%s] ids sampled from mu in %.1f ms" % (w.name, sample_ms))
    hq = torch.empty((T, d), dtype=torch.uint8, device=dev)
    if w.scaling == inputs.PER_TENSOR:
        hs = torch.empty(1, dtype=torch.float32, device=dev)
    elif w.scaling == inputs.PER_ROW:
        hs = torch.empty(T, dtype=torch.float32, device=dev)
    else:
        hs = torch.empty((T, d // 32), dtype=torch.uint8, device=dev)
    outs = {k: torch.zeros(w.slots, dtype=torch.float32, device=dev)
            for k in ("logp_pi", "logp_mu", "entropy_pi", "entropy_mu")}
    return dict(w=w, T=T, H=H, W=W, wq=wq, ws=ws, packed=packed, slots=slots, mask=mask, groups=groups, adv=adv,
                ids=ids, hq=hq, hs=hs, outs=outs, X=None, wq_ms=wq_ms, wq_bytes=wq_bytes, pw_ms=pw_ms,
                sample_ms=sample_ms)


def step(acrl, S, ev=None):
    """One pass of the hot path.  With ev (a list of 6 events) the pass is
    split at the call boundaries: quantize H | pi scoring | mu scoring |
    reduce | controller, pi and mu scored by separate calls (the same
    kernels the fused call launches) so that each can be timed alone."""
    w = S["w"]
    rec = (lambda k: ev[k].record()) if ev is not None else (lambda k: None)
    rec(0)
    acrl.acrl_quantize_fp8(S["H"], w.scaling, q=S["hq"], scales=S["hs"])
    rec(1)
    kw = dict(inv_temperature=w.inv_temperature, out_slot=S["slots"], n_slots=w.slots, outputs=S["outs"],
              want=("entropy",), packed_weights=S["packed"])
    args = (S["H"], S["W"], S["hq"], S["hs"], S["wq"], S["ws"], w.scaling, S["ids"])
    if ev is None:
        sc = acrl.acrl_score_pi_mu(*args, **kw)
    else:
        sc = acrl.acrl_score_pi_mu(*args, policies=acrl.POLICY_PI, **kw)
        rec(2)
        sc = acrl.acrl_score_pi_mu(*args, policies=acrl.POLICY_MU, **kw)
    rec(3)
    red = acrl.acrl_discrepancy_reduce(w.B, w.L, w.n_prompts, sc["logp_pi"], sc["logp_mu"], S["mask"], S["groups"],
                                       entropy_pi=sc["entropy_pi"], entropy_mu=sc["entropy_mu"], want_d_tok=False)
    rec(4)
    # X: the step-0 batch discrepancy (read once, outside the timed steps)
    X = S["X"] if S["X"] is not None else 1.0
    acrl.acrl_controller_step(w.B, w.L, w.n_prompts, S["mask"], S["groups"], sc["logp_pi"], sc["logp_mu"], S["adv"],
                              False, acrl.Y_GROUP, red["seq_mean_d"], red["group_y"], red["stats"], X, 0.65, 3.0,
                              want_alpha=False)
    rec(5)
    return red


def measure(torch, acrl, S, steps, warmup):
    """Warm-up (step 0 calibrates X, Sec. 4.1), the timed steps of the whole
    path, then one split pass per step for the per-kernel times."""
    w, T = S["w"], S["T"]
    d, V = w.d, w.V
    ev = lambda: torch.cuda.Event(enable_timing=True)
    t0 = time.time()
    red = step(acrl, S)
    torch.cuda.synchronize()
    S["X"] = max(float(red["stats"][0].item()), 1e-12)
    for _ in range(max(warmup - 1, 0)):
        step(acrl, S)
    torch.cuda.synchronize()
    log("[%s] warmup %d steps in %.1fs; X = %.4g" % (w.name, warmup, time.time() - t0, S["X"]))
    start, end = ev(), ev()
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        step(acrl, S)
    end.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / steps
    evs = [[ev() for _ in range(6)] for _ in range(steps)]
    for k in range(steps):
        red = step(acrl, S, evs[k])
    torch.cuda.synchronize()
    seg = lambda i, j: float(np.mean([evs[k][i].elapsed_time(evs[k][j]) for k in range(steps)]))
    t = {"quantize_h": seg(0, 1), "score_pi_call": seg(1, 2), "score_mu_call": seg(2, 3), "reduce": seg(3, 4),
         "controller": seg(4, 5)}
    stats = red["stats"].cpu().numpy()
    log("[%s] per step %.3f ms | " % (w.name, ms_per_step) + " | ".join("%s %.3f" % kv for kv in t.items()))
    log("[%s] batch stats:" % w.name, dict(zip(acrl.STAT_NAMES, [float(x) for x in stats])))
    flops = 2.0 * T * V * d           # per precision, algorithmic
    ideal_ms = (flops / (PEAK_TFLOPS["bf16"] * 1e12) + flops / (PEAK_TFLOPS["fp8"] * 1e12)) * 1e3
    return dict(ms_per_step=ms_per_step, kernel_ms=t, flops=flops, ideal_ms=ideal_ms,
                pi_frac=flops / (t["score_pi_call"] * 1e-3) / 1e12 / PEAK_TFLOPS["bf16"],
                mu_frac=flops / (t["score_mu_call"] * 1e-3) / 1e12 / PEAK_TFLOPS["fp8"],
                mfma_frac_combined=ideal_ms / ms_per_step, stats=stats)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="q8b", choices=sorted(inputs.WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline (0 = skip)")
    ap.add_argument("--no-divergence", action="store_true",
                    help="skip the full-vocabulary KL / Euclidean leg")
    ap.add_argument("--div-chunk", type=int, default=0,
                    help="rows per pass of the full-vocabulary measures (0 = the library's 16384)")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the surrogate + LM-head backward leg")
    ap.add_argument("--no-library", action="store_true",
                    help="skip the vendor-library GEMM leg (hipBLASLt through torch, no softmax)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other full-size workloads (q17b, long, mx after the headline)")
    ap.add_argument("--counters", action="store_true",
                    help="copy calibration + one step only (for rocprofv3 --pmc passes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this path runs on a single MI355X "
              "(multi-GPU sharding is design-only); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_24062_amd import acrl, profiling

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    acrl.lib()
    w = inputs.WORKLOADS[args.workload]
    log("workload:", w.describe(), "| valid tokens", inputs.n_valid(w), "of", w.slots, "slots")
    S = setup(torch, acrl, w, dev)
    T, d, V = S["T"], w.d, w.V
    H, W, hq, hs, wq, ws, ids, slots = S["H"], S["W"], S["hq"], S["hs"], S["wq"], S["ws"], S["ids"], S["slots"]

    if args.counters:
        # a plain copy of COPY_BYTES (read and written once), then one step
        src = torch.ones(profiling.COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        step(acrl, S)
        if not args.no_divergence:
            divergence_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, S["packed"], 0.0, reps=0,
                           div_chunk=args.div_chunk)
        if not args.no_backward:
            backward_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, S["mask"], S["groups"], S["adv"], 1.0,
                         reps=0)
        if not args.no_library:
            library_leg(torch, w, T, H, W, hq, hs, wq, ws, 1.0, 1.0, reps=0)
        torch.cuda.synchronize()
        log("counters run done")
        return

    R = measure(torch, acrl, S, args.steps, args.warmup)
    ms_per_step, t = R["ms_per_step"], R["kernel_ms"]
    t_pi, t_mu = t["score_pi_call"], t["score_mu_call"]
    flops = R["flops"]
    ach_pi = flops / (t_pi * 1e-3) / 1e12
    ach_mu = flops / (t_mu * 1e-3) / 1e12
    # achieved = 2 T V d FLOP per launch / the launch's duration, the duration
    # being the bench's own events around a call that launches the kernel and
    # the policy's strip merge (tens of microseconds)
    roof_pi = {"kernel": "score_kernel<bf16> (pi LM head + fused log-softmax)", "bound": "mfma",
               "achieved": round(ach_pi, 1), "peak": PEAK_TFLOPS["bf16"], "unit": "TFLOP/s",
               "frac": round(ach_pi / PEAK_TFLOPS["bf16"], 4), "traffic": None,
               "avg_ms": round(float(t_pi), 4), "flops_per_launch": flops}
    roof_mu = {"kernel": "score_kernel<fp8> (mu LM head + fused log-softmax)", "bound": "mfma",
               "achieved": round(ach_mu, 1), "peak": PEAK_TFLOPS["fp8"], "unit": "TFLOP/s",
               "frac": round(ach_mu / PEAK_TFLOPS["fp8"], 4), "traffic": None,
               "avg_ms": round(float(t_mu), 4), "flops_per_launch": flops}
    dominant = roof_pi if t_pi >= t_mu else roof_mu
    # HBM traffic of each score kernel from the committed counter summary, if current
    tr = profiling.load_traffic(os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                                             "score_%s_traffic.md" % w.name))
    mu_mode = {inputs.PER_TENSOR: 1, inputs.PER_ROW: 2, inputs.MX32: 3}[w.scaling]

    def scorer_row(mode):  # the scoring instantiation <mode, softmax epilogue, any wave count>
        if tr is None:
            return None
        keys = [k for k in tr["kernels"] if k.startswith("score_kernel<%d, 0" % mode)]
        return tr["kernels"][keys[0]] if keys else None

    for roof, mode in ((roof_pi, 0), (roof_mu, mu_mode)):
        row = scorer_row(mode)
        if row is not None:
            roof["traffic"] = round(row["traffic_bytes"])
            roof["traffic_unit"] = "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    q_bytes = T * d * 3 + (T * d * 2 if w.scaling == inputs.PER_TENSOR else 0)

    value = T / (ms_per_step * 1e-3)
    line = {
        "metric": "scored tokens/sec (pi+mu logprob+discrepancy) and %% of MFMA peak, d=%d V=%d" % (d, V),
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16(pi)+fp8e4m3(mu)",
        "data": "synthetic",
        "config": {"workload": w.describe(), "valid_tokens": T, "slots": w.slots,
                   "ids": "drawn from mu at tau (Gumbel-max with Philox4x32-10, seed %d), untimed" % w.seed,
                   "sample_mu_ms": round(S["sample_ms"], 3),
                   "mfma_frac_combined": round(R["mfma_frac_combined"], 4),
                   "kernel_ms": {k: round(v, 4) for k, v in t.items()},
                   "quantize_h_GBps": round(q_bytes / (t["quantize_h"] * 1e-3) / 1e9, 1),
                   "quantize_w_ms": round(S["wq_ms"], 4),
                   "quantize_w_GBps": round(S["wq_bytes"] / (S["wq_ms"] * 1e-3) / 1e9, 1),
                   "pack_w_ms": round(S["pw_ms"], 4),
                   # one step with the once-per-weight-version quantization and packing of W added in
                   "all_in_tokens_per_s": round(T / ((ms_per_step + S["wq_ms"] + S["pw_ms"]) * 1e-3), 1),
                   "X": S["X"]},
        "roofline": dominant,
        "roofline_other": roof_mu if dominant is roof_pi else roof_pi,
    }

    line["config"]["hbm_kernels"] = hbm_kernels(torch, acrl, dev, H, w)
    score_ms = t_pi + t_mu
    if not args.no_divergence:
        line["divergence"] = divergence_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, S["packed"],
                                            score_ms, div_chunk=args.div_chunk)
    if not args.no_backward:
        line["backward"] = backward_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, S["mask"], S["groups"],
                                        S["adv"], S["X"])
    if not args.no_library:
        line["library_gemm"] = library_leg(torch, w, T, H, W, hq, hs, wq, ws, t_pi, t_mu)

    # ---------------- CPU baseline: the oracle on host cores, bounded sample
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, T, H, W, args.cpu_seconds)
    del S, H, W, hq, hs, wq, ws, ids, slots
    torch.cuda.empty_cache()

    # ---------------- the other full-size workloads: the same step, fewer steps
    if not args.no_workloads:
        line["workloads"] = {}
        for name in ("q17b", "long", "mx"):
            if name == w.name:
                continue
            wl = inputs.WORKLOADS[name]
            S2 = setup(torch, acrl, wl, dev)
            R2 = measure(torch, acrl, S2, 2, 1)
            line["workloads"][name] = {
                "workload": wl.describe(), "valid_tokens": S2["T"], "steps": 2, "warmup": 1,
                "ms_per_step": round(R2["ms_per_step"], 3),
                "tokens_per_s": round(S2["T"] / (R2["ms_per_step"] * 1e-3), 1),
                "kernel_ms": {k: round(v, 3) for k, v in R2["kernel_ms"].items()},
                "pi_frac_of_bf16_peak": round(R2["pi_frac"], 4), "mu_frac_of_fp8_peak": round(R2["mu_frac"], 4),
                "mfma_frac_combined": round(R2["mfma_frac_combined"], 4)}
            del S2
            torch.cuda.empty_cache()
        log("workloads:", line["workloads"])
    print(json.dumps(line), flush=True)


def library_leg(torch, w, T, H, W, hq, hs, wq, ws, pi_ms, mu_ms, reps=2):
    """Context for the scorers' rates, not part of the path: the vendor
    library (hipBLASLt through torch) on the same two contractions with no
    softmax, logits = H W^T with bf16 output, in BF16 and (per-tensor
    scaling only) as the scaled FP8 product of the same quantized operands.
    Chunks of 32768 tokens keep the [T, V] logits it writes in HBM; the
    token count is cut to a multiple of 16 for the FP8 product."""
    d, V = w.d, w.V
    CH = 32768
    Tm = (T // 16) * 16
    chunks = [(s0, min(CH, Tm - s0)) for s0 in range(0, Tm, CH)]
    flops = 2.0 * Tm * V * d
    out = torch.empty((CH, V), dtype=torch.bfloat16, device=H.device)
    res = {"what": "torch.mm (hipBLASLt) logits = H W^T, bf16 out, and torch._scaled_mm on the FP8 operands; "
                   "no softmax; %d chunks of <= %d tokens" % (len(chunks), CH),
           "tokens": Tm, "flops": flops}

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        if reps == 0:  # one untimed pass (counter collection)
            return 1.0
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    def bf16():
        for s0, n in chunks:
            torch.mm(H[s0:s0 + n], W.t(), out=out[:n])

    ms = timed(bf16)
    tf = flops / (ms * 1e-3) / 1e12
    res["bf16"] = {"ms": round(ms, 3), "TFLOPs": round(tf, 1), "frac_of_peak": round(tf / 2500.0, 4),
                   "fused_pi_rate_over_library": round((T / float(pi_ms)) / (Tm / ms), 4)}
    log("library bf16: %.2f ms, %.0f TFLOP/s" % (ms, tf))
    if w.scaling == inputs.PER_TENSOR:
        try:
            f8 = torch.float8_e4m3fn
            hq8, wq8 = hq.view(f8), wq.view(f8)

            def fp8():
                for s0, n in chunks:
                    torch._scaled_mm(hq8[s0:s0 + n], wq8.t(), scale_a=hs, scale_b=ws,
                                     out_dtype=torch.bfloat16)

            ms = timed(fp8)
            tf = flops / (ms * 1e-3) / 1e12
            res["fp8"] = {"ms": round(ms, 3), "TFLOPs": round(tf, 1), "frac_of_peak": round(tf / 5000.0, 4),
                          "fused_mu_rate_over_library": round((T / float(mu_ms)) / (Tm / ms), 4)}
            log("library fp8: %.2f ms, %.0f TFLOP/s" % (ms, tf))
        except (RuntimeError, TypeError) as e:
            res["fp8"] = {"error": str(e)[:200]}
    del out
    torch.cuda.empty_cache()
    return res if reps else None


def divergence_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, packed, score_ms, reps=2, div_chunk=0):
    """The scoring call with the full-vocabulary measures (KL both ways,
    Euclidean distance) switched on: in passes of 16384 rows the mu kernel
    also stores its logits (4 B each) and the pi kernel reads them back and
    accumulates the measures in its epilogue (8 B per vocabulary entry and
    row in all)."""
    V = w.V
    outs = {}

    def run():
        return acrl.acrl_score_pi_mu(H, W, hq, hs, wq, ws, w.scaling, ids, inv_temperature=w.inv_temperature,
                                     out_slot=slots, n_slots=w.slots, outputs=outs, want=("entropy",),
                                     divergence=True, div_chunk=div_chunk, packed_weights=packed)

    outs.update(run())
    torch.cuda.synchronize()
    if reps == 0:  # one untimed pass (counter collection)
        return None
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        run()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    valid = slots.long()
    kl = outs["kl_pi_mu"][valid]
    res = {"what": "acrl_score_pi_mu with kl_pi_mu, kl_mu_pi and l2 over the batch's valid tokens",
           "ms": round(ms, 3), "score_ms_without": round(float(score_ms), 3),
           "overhead_ms": round(ms - float(score_ms), 3),
           "rows_per_pass": div_chunk or 16384,
           "logit_bytes_stored_and_read": 2 * 4 * T * V,
           "mean_kl_pi_mu": float(kl.double().mean().item()),
           "mean_kl_mu_pi": float(outs["kl_mu_pi"][valid].double().mean().item()),
           "mean_l2": float(outs["l2"][valid].double().mean().item())}
    log("divergence:", res)
    del outs
    torch.cuda.empty_cache()
    return res


def backward_leg(torch, acrl, w, T, H, W, hq, hs, wq, ws, ids, slots, mask, groups, adv, X, reps=2):
    """The training side of the step, after scoring: the ACRL-weighted
    surrogate's coefficients (from this batch's pi log-probs, the controller's
    weights and the advantages; logp_old = logp_new, the first update of a
    batch) and the LM-head backward dH = dZ W, dW = dZ^T H with dZ recomputed
    from the logits.  Roofline: 3 x 2 T V d FLOP (logits, dH, dW) at the BF16
    MFMA peak."""
    d, V = w.d, w.V
    sc = acrl.acrl_score_pi_mu(H, W, hq, hs, wq, ws, w.scaling, ids, inv_temperature=w.inv_temperature,
                               out_slot=slots, n_slots=w.slots, want=("entropy", "lse"))
    red = acrl.acrl_discrepancy_reduce(w.B, w.L, w.n_prompts, sc["logp_pi"], sc["logp_mu"], mask, groups,
                                       entropy_pi=sc["entropy_pi"], entropy_mu=sc["entropy_mu"], want_d_tok=False)
    _, weight = acrl.acrl_controller_step(w.B, w.L, w.n_prompts, mask, groups, sc["logp_pi"], sc["logp_mu"], adv,
                                          False, acrl.Y_GROUP, red["seq_mean_d"], red["group_y"], red["stats"],
                                          X, 0.65, 3.0, want_alpha=False)
    dh = torch.empty((T, d), dtype=torch.float32, device=H.device)
    dw = torch.empty((V, d), dtype=torch.float32, device=H.device)

    def run():
        coef, loss = acrl.acrl_surrogate(w.B, w.L, w.n_prompts, mask, groups, sc["logp_pi"], sc["logp_pi"], adv,
                                         False, weight=weight)
        acrl.acrl_lm_head_backward(H, W, ids, coef, sc["lse_pi"], inv_temperature=w.inv_temperature,
                                   row_slot=slots, dh=dh, dw=dw)
        return loss

    run()
    torch.cuda.synchronize()
    if reps == 0:  # one untimed pass (counter collection)
        return None
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        loss = run()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    flops = 3 * 2.0 * T * V * d
    ach = flops / (ms * 1e-3) / 1e12
    res = {"what": "acrl_surrogate + acrl_lm_head_backward (dH and dW) over the batch's valid tokens",
           "ms": round(ms, 3), "tokens_per_s": round(T / (ms * 1e-3), 1),
           "roofline": {"bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_TFLOPS["bf16"],
                        "unit": "TFLOP/s", "frac": round(ach / PEAK_TFLOPS["bf16"], 4),
                        "flops": flops, "flops_rule": "3 x 2 T V d (logits recomputed, dH, dW)"},
           "loss": float(loss.item()), "dw_abs_max": float(dw.abs().max().item())}
    log("backward:", res)
    del dh, dw
    torch.cuda.empty_cache()
    return res


def hbm_kernels(torch, acrl, dev, H, w, reps=5):
    """Achieved HBM bandwidth of the streaming kernels against 8 TB/s: the
    three quantizers on this workload's hidden states, and the discrepancy
    reduce on a dedicated 64M-slot batch (at the workload's 262k slots it is
    launch-bound)."""
    T, d = H.shape
    res = {}

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    for name, scaling, bytes_per_elt in (("quantize_h_per_tensor", inputs.PER_TENSOR, 5.0),
                                         ("quantize_h_per_row", inputs.PER_ROW, 3.0),
                                         ("quantize_h_mx32", inputs.MX32, 3.0 + 1.0 / 32)):
        q, sc = acrl.acrl_quantize_fp8(H, scaling)
        ms = timed(lambda: acrl.acrl_quantize_fp8(H, scaling, q=q, scales=sc))
        nbytes = T * d * bytes_per_elt
        res[name] = {"ms": round(ms, 4), "GBps": round(nbytes / ms / 1e6, 1),
                     "frac_of_8TBps": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4),
                     "bytes": int(nbytes)}
        del q, sc
    # reduce: 16384 sequences x 4096 slots, lengths U[1, 4096], 17 bytes per slot
    B, L, ng = 16384, 4096, 2048
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    lp_pi = -torch.rand(B * L, device=dev, generator=g) * 10
    lp_mu = lp_pi + 0.05 * torch.randn(B * L, device=dev, generator=g)
    ent = torch.rand(B * L, device=dev, generator=g) * 9
    lens = torch.randint(1, L + 1, (B,), device=dev, generator=g)
    mask = (torch.arange(L, device=dev)[None, :] < lens[:, None]).to(torch.uint8).reshape(-1)
    groups = (torch.arange(B, device=dev, dtype=torch.int32) // 8).contiguous()
    ms = timed(lambda: acrl.acrl_discrepancy_reduce(B, L, ng, lp_pi, lp_mu, mask, groups, entropy_pi=ent,
                                                    entropy_mu=ent, want_d_tok=False))
    nbytes = B * L * 17.0
    res["reduce_64M_slots"] = {"ms": round(ms, 4), "GBps": round(nbytes / ms / 1e6, 1),
                               "frac_of_8TBps": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4),
                               "bytes": int(nbytes)}
    del lp_pi, lp_mu, ent, mask
    # what a plain device copy reaches on this GPU (context for the figures
    # above): torch's copy (the runtime's blit kernel) and an elementwise
    # kernel, 1 GiB read + 1 GiB written each
    src = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    for name, fn in (("copy_1GiB", lambda: dst.copy_(src)), ("elementwise_neg_1GiB", lambda: torch.neg(src, out=dst))):
        ms = timed(fn)
        nbytes = 2.0 * (1 << 30)
        res[name] = {"ms": round(ms, 4), "GBps": round(nbytes / ms / 1e6, 1),
                     "frac_of_8TBps": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4), "bytes": int(nbytes)}
    del src, dst
    torch.cuda.empty_cache()
    log("HBM kernels:", res)
    return res


def cpu_baseline(w, T, H, W, budget_s):
    """The oracle on the host cores, on a bounded sample of this workload's
    valid tokens: its own quantization of W (once, timed apart) and of the
    sampled rows, then pi and mu scored at full V and d.  Ids are the seeded
    uniform draw (the scoring cost does not depend on them)."""
    import torch
    import oracle
    cores = len(os.sched_getaffinity(0))
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            model = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    log("cpu baseline: oracle on %d threads (%d cores in affinity, %s)" % (threads, cores, model))
    oracle.set_threads(threads)
    Wh = W.cpu().view(torch.int16).numpy().view(np.uint16)
    t0 = time.time()
    wq, ws = oracle.quantize_fp8(Wh, w.scaling)
    t_wq = time.time() - t0
    log("  oracle: W quantized in %.1fs" % t_wq)
    ids = inputs.uniform_ids(w, T)
    rng = np.random.default_rng(0)

    def run(n_threads, batch, seconds):
        oracle.set_threads(n_threads)
        done, t_total = 0, 0.0
        while t_total < seconds and done < T:
            rows = rng.choice(T, size=batch, replace=False)
            Hs = H.index_select(0, torch.from_numpy(rows).to(H.device)).cpu().view(torch.int16).numpy()
            Hs = Hs.view(np.uint16)
            t1 = time.time()
            # per-tensor: the scale of the sampled rows stands in for the whole H's (same cost)
            hq, hs = oracle.quantize_fp8(Hs, w.scaling)
            oracle.score(Hs, Wh, hq, hs, wq, ws, w.scaling, ids[rows], inv_temperature=w.inv_temperature)
            t_total += time.time() - t1
            done += batch
            log("  oracle (%d threads): %d rows in %.1fs" % (n_threads, done, t_total))
        return done, t_total

    done, t_total = run(threads, max(threads, 1), budget_s)
    done1, t1 = run(1, 1, min(budget_s / 3, 8.0))
    oracle.set_threads(threads)
    return {"value": round(done / t_total, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d valid tokens of the %s workload, full V=%d and d=%d, pi and mu "
                      "(the oracle's own FP8 quantization of each sampled row, fp64 logits + "
                      "log-softmax), %.1f s of wall time; W quantized by the oracle once "
                      "beforehand in %.1f s (not in the rate)" % (done, T, w.name, w.V, w.d, t_total, t_wq),
            "single_thread": {"value": round(done1 / t1, 4), "unit": "tokens/s",
                              "sample": "%d tokens in %.1f s" % (done1, t1)},
            "cpu_model": model}


if __name__ == "__main__":
    main()
