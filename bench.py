#!/usr/bin/env python3
"""Rollout throughput of the DASH hot path on one MI355X.

One step = one whole preemptive-sampling rollout of the workload (prefill of
every prompt, G samples each, gen_len decode steps with temperature sampling)
followed by the GRPO group advantage and the gradient-filter compaction of the
synthetic rewards.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps 3] [--warmup 1] [--workload 1.5b-b1024] [--eager]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0

# Memory traffic of one decode-attention launch of the 1.5B batch-1024 rollout, from the
# rocprofv3 read/write request counters (profiles/decode_attn_traffic__1.5b-b1024.md:
# 595.9 MB read + 3.15 MB written), valid for the attention sources it was measured with.
ATTN_TRAFFIC = {
    "workload": "1.5b-b1024",
    "bytes_per_launch": 599_100_000,
    "sources": {
        "paper_2505_17218_amd/csrc/attention.hip": "d7872754a3c4d32096cb2a52c0acccfe6ab0adc3234586060611604122336633",
        "paper_2505_17218_amd/csrc/common.h": "0f40c78e53eca25bf8577dd7eee24736429eac2b540ae38e76c22c6b64ed8147",
    },
}


class SclkSampler:
    """The shader clock the driver reports for this GPU (the current level of its
    pp_dpm_sclk), sampled every `period` seconds on a background thread while the timed
    steps run: observed, not pinned.  `result()` is None where the file is unavailable."""

    def __init__(self, period: float = 0.05):
        import glob
        import re
        import threading

        self.re = re.compile(r"(\d+)\s*mhz", re.IGNORECASE)
        self.period, self.samples, self.stop = period, [], threading.Event()
        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if len(paths) == 1 else self._match(paths)
        self.thread = threading.Thread(target=self._run, daemon=True)

    @staticmethod
    def _match(paths):
        # several cards visible: the one whose PCI bus is torch's device 0
        try:
            import torch

            bus = "%02x:" % torch.cuda.get_device_properties(0).pci_bus_id
            for p in paths:
                if os.path.basename(os.path.realpath(os.path.dirname(p))).split(":", 1)[-1].startswith(bus):
                    return p
        except Exception:
            pass
        return None

    def _read(self):
        with open(self.path) as f:
            for line in f:
                if "*" in line:
                    m = self.re.search(line)
                    return int(m.group(1)) if m else None
        return None

    def _run(self):
        while not self.stop.is_set():
            try:
                v = self._read()
                if v:
                    self.samples.append(v)
            except OSError:
                return
            self.stop.wait(self.period)

    def __enter__(self):
        if self.path:
            self.thread.start()
        return self

    def __exit__(self, *exc):
        self.stop.set()
        if self.thread.is_alive():
            self.thread.join()

    def result(self):
        if not self.samples:
            return None
        v = sorted(self.samples)
        return {"median": v[len(v) // 2], "max": v[-1], "samples": len(v), "source": "pp_dpm_sclk"}


def measured_attention_traffic(workload: str):
    """The counted bytes per attention launch, or None if the workload or the kernel sources differ."""
    import hashlib

    if workload != ATTN_TRAFFIC["workload"]:
        return None
    for rel, digest in ATTN_TRAFFIC["sources"].items():
        with open(os.path.join(ROOT, rel), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return ATTN_TRAFFIC["bytes_per_launch"]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def attention_bytes(wl, steps_run: int) -> tuple[float, float]:
    """Algorithmic bytes of all decode-attention launches of one rollout: (unique, logical).

    Per layer and decode step t (1..T-1, context P + t): every row reads its K/V
    (2 * n_kv * head_dim * 2 bytes per position), plus q and o (n_heads * head_dim
    * 2 bytes each).  'unique' counts the shared prompt pages once per group (the
    group's rows read the same physical pages); 'logical' counts them per row."""
    s = wl.shape
    kvb = 2 * s.n_kv_heads * s.head_dim * 2
    qo = 2 * s.n_heads * s.head_dim * 2
    N, P, G = wl.n_seqs, wl.prompt_len, wl.group
    uniq = logi = 0.0
    for t in range(1, steps_run):
        logi += N * (P + t) * kvb + N * qo
        uniq += (N // G) * P * kvb + N * t * kvb + N * qo
    return uniq * s.n_layers, logi * s.n_layers


def gemm_flops(wl, rows: int) -> dict:
    s = wl.shape
    d, hq = s.d_model, s.n_heads * s.head_dim
    qr = (s.n_heads + 2 * s.n_kv_heads) * s.head_dim
    L = s.n_layers
    return {"gemm_qkv": 2.0 * rows * qr * d * L, "gemm_o": 2.0 * rows * d * hq * L,
            "gemm_gate_up": 2.0 * rows * 2 * s.d_ff * d * L, "gemm_down": 2.0 * rows * d * s.d_ff * L,
            "gemm_lm_head": 2.0 * rows * s.vocab * d}


def cpu_baseline(wl, weights, prompts, seconds: float) -> dict:
    """The oracle (float64 full recompute + float32 sampler) generating tokens for the
    workload's first prompt until `seconds` have passed (at least one token); then the
    small fp32 configuration's whole rollout (16 sequences x 32 tokens) as `tiny_full`."""
    import dataclasses

    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import model as om
    from oracle import sampler as osm

    sd = dataclasses.asdict(wl.shape)
    seq = list(prompts[0])
    t0 = time.perf_counter()
    n = 0
    while True:
        lg = om.forward(sd, weights, np.array(seq, dtype=np.int32), positions=[len(seq) - 1])[0]
        tok, _ = osm.sample_row(lg.astype(np.float32), 0, n, wl.temperature, 2)
        seq.append(tok)
        n += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    # and the small fp32 configuration in full: every sequence and token of its rollout
    from paper_2505_17218_amd import synth

    tw = synth.WORKLOADS["tiny"]
    tsd, tww, tpr = dataclasses.asdict(tw.shape), synth.make_weights(tw.shape, 0), synth.make_prompts(tw, 0)
    t1 = time.perf_counter()
    for i in range(tw.n_seqs):
        tseq = list(tpr[i // tw.group])
        for t in range(tw.gen_len):
            lg = om.forward(tsd, tww, np.array(tseq, dtype=np.int32), positions=[len(tseq) - 1])[0]
            tok, _ = osm.sample_row(lg.astype(np.float32), i, t, tw.temperature, synth.sampler_seed(0))
            tseq.append(tok)
    tiny_dt = time.perf_counter() - t1
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    return {"value": n / dt, "unit": "generated tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{wl.shape.name} shape, 1 sequence, prompt {wl.prompt_len}, {n} tokens generated by "
                      f"full float64 recompute in {dt:.1f} s",
            "cpu_model": cpu_model, "host_cpus_available": len(os.sched_getaffinity(0)),
            "tiny_full": {"workload": tw.name, "sequences": tw.n_seqs, "tokens": tw.n_seqs * tw.gen_len,
                          "seconds": round(tiny_dt, 2), "tokens_per_s": round(tw.n_seqs * tw.gen_len / tiny_dt, 1)}}


def kl_leg(shape, model, kv, seqs, P, adv, kept, lp_rollout, kept_l, N, T):
    """KL regulariser after the filter: teacher-forced KL(base || policy) of the kept samples
    against an independently initialised base model of the same architecture, the
    regularised PPO loss (rollout log-probs as the old policy, beta 0.04, eps 0.2), and the
    row-KL kernel alone on a block of logits, timed with events on its stream."""
    import torch

    from paper_2505_17218_amd import engine, synth
    base = engine.Model(shape, synth.make_weights(shape, 1))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    lp, kl, _ = engine.teacher_forced_kl(model, base, kv, seqs, P, seqs_per_chunk=16, reverse=False)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    lp_full = torch.zeros((N, T), dtype=torch.float32, device="cuda")
    kl_full = torch.zeros((N, T), dtype=torch.float32, device="cuda")
    old_full = torch.zeros((N, T), dtype=torch.float32, device="cuda")
    lp_full[kept_l], kl_full[kept_l], old_full[kept_l] = lp, kl, lp_rollout
    loss, _ = engine.policy_loss(lp_full, adv, kept, logprobs_old=old_full, kl=kl_full, clip_eps=0.2, beta=0.04)
    n_tok = int(seqs.shape[0]) * int(seqs.shape[1])
    out = {"tokens_per_s": round(n_tok / dt, 1), "seconds": round(dt, 3), "mean_kl_per_token": float(kl.mean().item()),
           "policy_loss_ppo_kl": float(loss.item())}
    del base, lp, kl, lp_full, kl_full, old_full
    # the row-KL kernel alone: 4096 row pairs of vocabulary-wide fp32 logits
    rows, V = 4096, shape.vocab
    a = torch.randn(rows, V, dtype=torch.float32, device="cuda")
    b = a + 0.1 * torch.randn(rows, V, dtype=torch.float32, device="cuda")
    engine.logits_kl(a, b, reverse=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 5
    e0.record()
    for _ in range(reps):
        engine.logits_kl(a, b, reverse=True)
    e1.record()
    e1.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    nbytes = 2 * rows * V * 4 + 2 * rows * 4
    out["kl_rows_kernel"] = {"rows": rows, "vocab": V, "avg_launch_us": round(us, 1),
                             "GBs": round(nbytes / us / 1e3, 1), "frac_hbm": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)}
    del a, b
    return out


def workload_leg(wl, model, weights_seed: int = 0, kv_pages_extra: int = 8, budgets=None) -> dict:
    """One rollout of `wl` on an already created model: a short warm-up rollout (8 tokens,
    same batch) that loads the kernels, then one timed rollout of the full workload with the
    middle decoder layer's decode attention timed by events, and the advantage filter of
    the workload's rewards.  Returns tokens/s and the attention HBM fraction."""
    import dataclasses

    import numpy as np
    import torch

    from paper_2505_17218_amd import _lib as L
    from paper_2505_17218_amd import engine, synth

    s = wl.shape
    N, P, G, T = wl.n_seqs, wl.prompt_len, wl.group, wl.gen_len
    ps = 32
    if budgets is not None:
        pages = wl.n_prompts * (P // ps) + int(sum((P + int(b) + ps - 1) // ps - P // ps for b in budgets))
    else:
        pages = wl.n_prompts * (P // ps) + N * ((P + T + ps - 1) // ps - P // ps)
    kv = engine.KVCache(model, ps, N, P + T, pages + kv_pages_extra)
    prompts = torch.from_numpy(synth.make_prompts(wl, weights_seed)).cuda()
    rewards = torch.from_numpy(synth.make_rewards(wl.n_prompts, G, wl.reward, weights_seed)).cuda()
    seed = synth.sampler_seed(weights_seed)
    warm = engine.Rollout(model, kv, wl.n_prompts, P, G, 8)
    warm.run(prompts, wl.temperature, seed, budgets=None if budgets is None else np.minimum(budgets, 8),
             use_graph=budgets is None)
    torch.cuda.synchronize()
    del warm
    ro = engine.Rollout(model, kv, wl.n_prompts, P, G, T)
    layer = s.n_layers // 2
    L.dash_profile_read(reset=True)
    L.dash_profile_enable((1 << L.K["attn"]) | (1 << L.K["prefill"]))
    L.dash_profile_layer(layer)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ro.run(prompts, wl.temperature, seed, budgets=budgets, use_graph=budgets is None)
    _, kept = engine.advantage_filter(rewards, G, L.DASH_ADV_STD_SAMPLE, 1e-6, wl.tau)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    prof = L.dash_profile_read(reset=True)
    L.dash_profile_enable(0)
    L.dash_profile_layer(-1)
    gen = int(budgets.sum()) if budgets is not None else N * T
    out = {"workload": wl.name, "sequences": N, "prompt_len": P, "gen_len": T, "ragged": budgets is not None,
           "tokens": gen, "seconds": round(dt, 3), "tokens_per_s": round(gen / dt, 1),
           "prefill_ms": round(prof["prefill"][0], 1), "kept_fraction": kept.numel() / N,
           "attn_split_keys": kv.split_keys}
    attn_ms, attn_n = prof["attn"]
    if budgets is None and attn_n:
        uniq, _ = attention_bytes(wl, T)
        per_layer = uniq / s.n_layers
        achieved = per_layer / (attn_ms * 1e-3) / 1e9
        out["decode_attn"] = {"avg_launch_us": round(attn_ms / attn_n * 1e3, 2), "GBs": round(achieved, 1),
                              "frac_hbm": round(achieved / HBM_PEAK_GBS, 4)}
    del ro, kv
    torch.cuda.empty_cache()
    return out


def legs(main_model, main_wl, max_seconds: float) -> dict:
    """Compact legs over the other workloads, each timed once after a short warm-up: the 3B
    batch sweep (64, 256, 1024, 2048 sequences), the 0.5B workload, and the ragged 1.5B
    workload (its kept fraction reported).  Stops early once `max_seconds` have passed."""
    import torch

    from paper_2505_17218_amd import engine, synth

    t0 = time.perf_counter()
    out = {}

    def left():
        return max_seconds - (time.perf_counter() - t0)

    rw = synth.WORKLOADS["1.5b-ragged"]
    if main_wl.shape == rw.shape:
        budgets = synth.make_lengths(rw.n_seqs, rw.ragged_mean, rw.gen_len, 0)
        out[rw.name] = workload_leg(rw, main_model, budgets=budgets)
        log(f"leg {rw.name}: {out[rw.name]}")
    model = None
    for name in ("0.5b-b512", "3b-b64", "3b-b256", "3b-b1024", "3b-b2048"):
        if left() <= 0:
            out[name] = "skipped (time budget)"
            continue
        wl = synth.WORKLOADS[name]
        if model is None or model.shape != wl.shape:
            model = None
            torch.cuda.empty_cache()
            model = engine.Model(wl.shape, synth.make_weights(wl.shape, 0))
        out[name] = workload_leg(wl, model)
        log(f"leg {name}: {out[name]}")
    model = None
    torch.cuda.empty_cache()
    out["seconds"] = round(time.perf_counter() - t0, 1)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="1.5b-b1024")
    ap.add_argument("--gen-len", type=int, default=0, help="override the generation length (quick runs)")
    ap.add_argument("--eager", action="store_true", help="launch every decode step eagerly (default: HIP graph replay)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kl", action="store_true",
                    help="skip the KL regulariser leg (teacher-forced KL against a second model, PPO loss)")
    ap.add_argument("--no-recompute", action="store_true",
                    help="skip the teacher-forced log-prob recompute of the kept samples after the timed region")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the compact legs over the other workloads (3B batch sweep, 0.5B, ragged 1.5B)")
    ap.add_argument("--legs-seconds", type=float, default=240.0,
                    help="stop starting new legs after this many seconds")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain 1 GiB device-to-device copy (reference for HBM traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the rollout is "
              "data-parallel over prompt groups, so each GPU would run its own share of the groups; "
              "the multi-GPU launcher is not implemented)", file=sys.stderr)
        return 2

    import dataclasses

    import numpy as np
    import torch

    from paper_2505_17218_amd import _lib as L
    from paper_2505_17218_amd import engine, synth

    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 1 GiB device-to-device copy done")
        del src, dst

    wl = synth.WORKLOADS[args.workload]
    if args.gen_len:
        wl = dataclasses.replace(wl, gen_len=args.gen_len)
    s = wl.shape
    N, P, G, T = wl.n_seqs, wl.prompt_len, wl.group, wl.gen_len
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    weights = synth.make_weights(s, 0)
    prompts = synth.make_prompts(wl, 0)
    rewards = synth.make_rewards(wl.n_prompts, G, wl.reward, 0)
    budgets = None
    if wl.ragged_mean:
        budgets = synth.make_lengths(N, wl.ragged_mean, T, 0)
    log(f"inputs ready ({time.perf_counter() - t0:.1f} s): {s.name}, {N} sequences, prompt {P}, gen {T}")
    model = engine.Model(s, weights)
    ps = 32 if s.dtype == synth.DT_BF16 else 16
    max_ctx = P + T
    if budgets is not None:  # pages each sample can hold at its own budget (what the driver reserves)
        pages = wl.n_prompts * (P // ps) + int(sum((P + int(b) + ps - 1) // ps - P // ps for b in budgets)) + 8
    else:
        pages = wl.n_prompts * (P // ps) + N * ((max_ctx + ps - 1) // ps - P // ps) + 8
    kv = engine.KVCache(model, ps, N, max_ctx, pages)
    ro = engine.Rollout(model, kv, wl.n_prompts, P, G, T)
    d_prompts = torch.from_numpy(prompts).cuda()
    d_rewards = torch.from_numpy(rewards).cuda()
    seed = synth.sampler_seed(0)
    torch.cuda.synchronize()
    log(f"model + kv ready ({time.perf_counter() - t0:.1f} s): pool {kv.pool.numel() / 2**30:.1f} GiB")

    def step():
        ro.run(d_prompts, wl.temperature, seed, budgets=budgets, use_graph=not args.eager)
        return engine.advantage_filter(d_rewards, G, L.DASH_ADV_STD_SAMPLE, 1e-6, wl.tau)

    # warm-up with every kernel class timed: the per-class breakdown
    L.dash_profile_enable((1 << len(L.K_CLASSES)) - 1)
    kept = None
    for i in range(args.warmup):
        tw = time.perf_counter()
        _, kept = step()
        torch.cuda.synchronize()
        log(f"warmup {i}: {time.perf_counter() - tw:.2f} s")
    breakdown = L.dash_profile_read(reset=True)
    # timed region: decode attention (the roofline kernel) of one decoder layer is
    # bracketed by events; every layer runs the same attention on the same bytes
    prof_layer = s.n_layers // 2
    L.dash_profile_enable((1 << L.K["attn"]) | (1 << L.K["attn_combine"]) | (1 << L.K["prefill"]))
    L.dash_profile_layer(prof_layer)
    torch.cuda.synchronize()
    with SclkSampler() as sclk:
        t_start = time.perf_counter()
        step_ms = []
        for i in range(args.steps):
            t_i = time.perf_counter()
            _, kept = step()
            torch.cuda.synchronize()
            step_ms.append((time.perf_counter() - t_i) * 1e3)
            log(f"step {i}: {time.perf_counter() - t_start:.2f} s cumulative")
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
    timed = L.dash_profile_read(reset=True)
    L.dash_profile_enable(0)
    L.dash_profile_layer(-1)
    kept_frac = kept.numel() / N if kept is not None else None

    gen_tokens = int(budgets.sum()) if budgets is not None else N * T
    value = gen_tokens * args.steps / elapsed
    ms_per_step = elapsed / args.steps * 1e3
    # decode-only rate: tokens drawn in decode steps (all but each sample's first) over the
    # timed wall time minus the prefill launches' event time
    prefill_ms = timed["prefill"][0] / max(1, args.steps)
    decode_tps = (gen_tokens - N) / max(1e-9, (ms_per_step - prefill_ms) * 1e-3)

    # roofline of decode attention from the events of the timed region
    attn_ms, attn_n = timed["attn"]
    uniq, logi = attention_bytes(wl, T) if budgets is None else (None, None)
    roofline = None
    if attn_n and uniq:
        # the timed launches are one layer's: its bytes are 1/n_layers of the rollout's
        per_launch_ms = attn_ms / attn_n
        uniq_l, logi_l = uniq / s.n_layers * args.steps, logi / s.n_layers * args.steps
        achieved = uniq_l / (attn_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_attention_traffic(args.workload),
                    "kernel": "decode_attn_bf16_k", "timed_layer": prof_layer, "launches": attn_n,
                    "avg_launch_us": round(per_launch_ms * 1e3, 2),
                    "bytes_per_launch": round(uniq_l / attn_n),
                    "logical_GBs": round(logi_l / (attn_ms * 1e-3) / 1e9, 1)}
    # GEMM MFMA utilisation from the warm-up breakdown (decode launches only; rows = N)
    gemm = {}
    if budgets is None and args.warmup:
        fl = gemm_flops(wl, N)
        tot_f = tot_ms = 0.0
        for k, f in fl.items():
            ms, n = breakdown[k]
            if not n:
                continue
            f_all = f * (T - 1) * args.warmup  # per decode step, T - 1 steps per rollout
            tf = f_all / (ms * 1e-3) / 1e12
            gemm[k] = {"tflops": round(tf, 1), "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
                       "avg_launch_us": round(ms / n * 1e3, 1)}
            tot_f += f_all
            tot_ms += ms
        if tot_ms:
            gemm["weighted"] = {"tflops": round(tot_f / (tot_ms * 1e-3) / 1e12, 1),
                                "mfma_frac": round(tot_f / (tot_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
    per_step = {k: round(v[0] / max(1, args.warmup), 2) for k, v in breakdown.items() if v[1]}

    # after the timed region: teacher-forced log-probs of the kept samples (the forward
    # of the policy-gradient step that follows the filter) and the PG loss
    recompute = None
    if not args.no_recompute and budgets is None and kept is not None and kept.numel():
        toks, _ = ro.tokens, ro.logprobs
        kept_l = kept.long()
        seqs = torch.cat([d_prompts.repeat_interleave(G, dim=0)[kept_l], toks[kept_l]], dim=1).contiguous()
        adv, kept2 = engine.advantage_filter(d_rewards, G, L.DASH_ADV_STD_SAMPLE, 1e-6, wl.tau)
        torch.cuda.synchronize()
        tr = time.perf_counter()
        rec = engine.teacher_forced_logprobs(model, kv, seqs, P, seqs_per_chunk=16)
        torch.cuda.synchronize()
        dt = time.perf_counter() - tr
        lp_full = torch.zeros((N, T), dtype=torch.float32, device="cuda")
        lp_full[kept_l] = rec
        loss, _ = engine.pg_loss(lp_full, adv, kept2)
        n_tok = int(seqs.shape[0]) * int(seqs.shape[1])
        recompute = {"sequences": int(seqs.shape[0]), "tokens": n_tok, "seconds": round(dt, 3),
                     "tokens_per_s": round(n_tok / dt, 1), "pg_loss": float(loss.item()),
                     "identical_to_rollout_logprobs": bool(torch.equal(rec, ro.logprobs[kept_l])),
                     "max_abs_dlogprob_vs_rollout": float((rec - ro.logprobs[kept_l]).abs().max().item())}
        log(f"recompute: {recompute}")
        if not args.no_kl:
            recompute["kl"] = kl_leg(s, model, kv, seqs, P, adv, kept2, ro.logprobs[kept_l], kept_l, N, T)
            log(f"kl: {recompute['kl']}")

    other = None
    if not args.no_legs and args.workload == "1.5b-b1024" and not args.gen_len:
        del ro
        torch.cuda.empty_cache()
        log("legs: other workloads, one timed rollout each ...")
        other = legs(model, wl, args.legs_seconds)

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        cpu = cpu_baseline(wl, weights, prompts, args.cpu_seconds)

    metric = ("rollout tokens/sec at batch 1024 (1.5B-shape)" if args.workload == "1.5b-b1024"
              else f"rollout tokens/sec ({wl.name})")
    out = {
        "metric": metric,
        "value": round(value, 1),
        "unit": "generated tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 1),
        "step_ms": [round(x, 1) for x in step_ms],
        "median_step_ms": round(sorted(step_ms)[len(step_ms) // 2], 1),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if s.dtype == synth.DT_BF16 else "f32",
        "data": "synthetic (uniform prompt ids, N(0,0.02) random-init weights, Bernoulli rewards)",
        "config": {"workload": wl.name, "shape": s.name, "sequences": N, "group": G, "prompt_len": P,
                   "gen_len": T, "ragged": bool(budgets is not None), "page_size": ps,
                   "graph": not args.eager and budgets is None,
                   "attn_split_keys": kv.split_keys},
        "roofline": roofline,
        "gemm_mfma": gemm,
        "prefill_ms": round(prefill_ms, 1),
        "decode_tokens_per_s": round(decode_tps, 1),
        "observed_sclk_mhz": sclk.result(),
        "kernel_ms_per_rollout": per_step,
        "kept_fraction": kept_frac,
        "recompute": recompute,
        "legs": other,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
