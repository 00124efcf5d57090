#!/usr/bin/env python
"""Throughput of the batched speculative-verify pass on one MI355X.

One step = the whole verify pass (sd_verify_batch: embedding, 64 decoder
layers, lm_head, accept/resample) plus sd_accept, for every batch of the
workload, with all inputs resident in HBM.  Users are not committed between
steps, so every step verifies the same batch.  Reported value: accepted
tokens per second, sum over users of (a_m + 1) per step / seconds per step
(the numerator of DiP-SD's throughput, eq. 2 and eq. 22).

The headline workload is the 32-user ragged batch of the Qwen3-32B shape
(prefixes U{256..4096}, l_m U{1..12}); the 16-user batch (stochastic and
greedy) and the four pipelined 16-user batches (HIP graphs, two streams)
are timed in the same run and reported under "workloads".

Prints one JSON line (rank 0, one GPU).  Inputs are seeded synthetic stand-ins:
random-init Qwen3-shaped weights, synthetic cached KV, synthetic draft
distributions; no trained weights or prompts are used.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, vendor figure
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, vendor figure


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen3-32b-ragged32")
    ap.add_argument("--extra", default="qwen3-32b-b16,qwen3-32b-pipe4x16",
                    help="comma-separated workloads timed after the headline one ('none': skip)")
    ap.add_argument("--mode", default="stochastic", choices=["stochastic", "greedy"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=3,
                    help="decoder layers the CPU-baseline sample runs (extrapolated to all)")
    ap.add_argument("--breakdown", action="store_true", help="time every kernel class")
    ap.add_argument("--no-greedy", action="store_true",
                    help="skip the greedy-mode measurement that follows a stochastic run")
    ap.add_argument("--graph", type=int, default=-1, choices=[-1, 0, 1],
                    help="1: each batch's pass is replayed from a HIP graph (sd_verify_batch_graph); "
                         "0: eager launches; -1 (default): graphs for the pipelined multi-batch "
                         "workload, whose definition asks for them, eager otherwise")
    ap.add_argument("--q-topk", type=int, default=0,
                    help="K > 0: draft rows sent as sparse payloads (top-K tokens plus a uniform "
                         "remainder, drafts redrawn from them) and verified by sd_verify_batch_sparse")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy (scale reference for HBM byte counters)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Run:
    """One workload on the GPU: weights, verifier context, cached KV and
    device inputs, ready to time."""

    def __init__(self, name, args, torch, graph=-1, q_topk=0, mode="stochastic"):
        import workload as wl
        from workload.device import DeviceWeights, batch_to_device, kv_rows
        from paper_2604_20919_amd.verifier import Verifier
        self.torch = torch
        self.name = name
        self.mode = mode
        w = self.w = wl.workload(name)
        m = self.m = w.model
        self.graph = (1 if w.n_batches > 1 else 0) if graph < 0 else graph
        t0 = time.time()
        self.dw = DeviceWeights(m, w.seed)
        log(f"{name}: weights {self.dw.nbytes() / 1e9:.1f} GB generated on GPU in {time.time() - t0:.1f}s")
        names = {"wq": wl.W_Q, "wk": wl.W_K, "wv": wl.W_V, "wo": wl.W_O, "wg": wl.W_G, "wu": wl.W_U,
                 "wd": wl.W_D, "norm1": wl.N_1, "norm2": wl.N_2, "qnorm": wl.N_Q, "knorm": wl.N_K}
        dw = self.dw
        ptrs = {"embed": dw.ptr(wl.EMBED), "lm_head": dw.ptr(wl.LM_HEAD), "norm_f": dw.ptr(wl.NORM_F),
                "layers": [{f: dw.ptr(k, l) for f, k in names.items()} for l in range(m.n_layers)]}
        nb = self.nb = w.n_batches
        batches = self.batches = [w.batch(n) for n in range(nb)]
        max_ctx = int((w.prefix_len + w.draft_len).max()) + 1
        pages = sum((int(p) + int(l) + 1 + 15) // 16 for p, l in zip(w.prefix_len, w.draft_len)) + 16
        v = self.v = Verifier(m, ptrs, n_pages=pages, max_users=w.n_users, max_draft=int(w.draft_len.max()),
                              max_batch_users=max(len(b.users) for b in batches),
                              max_batch_tokens=max(b.T for b in batches), max_ctx=max_ctx,
                              max_pending=min(nb, 8))
        log(f"{name}: KV pool {v.kv_bytes / 1e9:.1f} GB, workspace {v.ws_bytes / 1e9:.2f} GB")
        t0 = time.time()
        dt = torch.int16 if m.dtype == "bf16" else torch.float32
        pmax = int(w.prefix_len.max())
        buf = (torch.empty((pmax, m.n_kv_heads, m.head_dim), dtype=dt, device="cuda"),
               torch.empty((pmax, m.n_kv_heads, m.head_dim), dtype=dt, device="cuda"))
        for b in batches:
            for i, u in enumerate(b.users):
                P = int(b.prefix_len[i])
                v.reset_user(int(u), P, int(b.root[i]))
                for l in range(m.n_layers):
                    k, vv = kv_rows(m, w.seed, l, int(u), P, out=buf)
                    v.write_kv(int(u), l, 0, k, vv)
        torch.cuda.synchronize()
        del buf
        self.kv_tokens = int(w.prefix_len.sum())
        log(f"{name}: cached KV of {self.kv_tokens} tokens written in {time.time() - t0:.1f}s")
        self.sparse = None
        self.q_topk = q_topk
        if q_topk > 0:
            self.sparse = []
            for b in batches:
                sr = wl.sparsify(b, q_topk, w.seed)   # redraws b.drafts from the sparse rows
                self.sparse.append(tuple(torch.from_numpy(a).cuda() for a in (sr.idx, sr.val, sr.rest)))
        self.dev_in = [batch_to_device(b) for b in batches]
        if mode == "greedy":
            plant_greedy_drafts(v, w, batches, self.dev_in, torch)
        self.streams = [torch.cuda.Stream() for _ in range(min(nb, 2))]
        self.verified_step = sum(b.T for b in batches)

    def step(self, one_stream=False, mode=None):
        # one_stream: every batch on the first stream, so that the event pairs
        # of the profiling passes time kernels that share the GPU with nothing
        mode = mode or self.mode
        w, v = self.w, self.v
        for n in range(self.nb):
            d, q, au = self.dev_in[n]
            st = self.streams[0] if one_stream else self.streams[n % len(self.streams)]
            if self.sparse is not None and mode == "stochastic":
                v.verify_sparse(n, w.assign, w.draft_len, d, *self.sparse[n], mode, seed=w.seed,
                                round_=0, accept_u=au, stream=st)
                continue
            v.verify(n, w.assign, w.draft_len, d, q, mode, seed=w.seed, round_=0,
                     accept_u=au if mode == "stochastic" else None, stream=st, graph=bool(self.graph))
        acc = 0
        for n in range(self.nb):
            n_acc, _ = v.accept(n, w.n_users)
            acc += int((n_acc[self.batches[n].users] + 1).sum())
        return acc

    def time(self, steps, warmup, mode=None):
        """Timed region: `steps` whole steps after `warmup` untimed ones,
        bracketed by device synchronisation; returns ms per step, accepted
        tokens per step and the per-step times."""
        torch = self.torch
        for _ in range(warmup):
            self.step(mode=mode)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        accepted = 0
        marks = [t0]
        for _ in range(steps):
            accepted += self.step(mode=mode)   # ends in sd_accept, which waits for the batch
            marks.append(time.perf_counter())
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        return 1e3 * elapsed / steps, accepted / steps, np.diff(np.array(marks)) * 1e3

    def close(self):
        self.v.close()
        del self.v, self.dw, self.dev_in, self.sparse
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2604_20919_amd import sdverify as sv

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    sv.lib()  # fails loudly if the HIP library is not built
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 3 x 1 GiB device-to-device copies done")
        del src, dst

    run = Run(args.workload, args, torch, graph=args.graph, q_topk=args.q_topk, mode=args.mode)
    w, m, v, nb, batches = run.w, run.m, run.v, run.nb, run.batches
    ms_step, acc_step, per_step = run.time(args.steps, args.warmup)
    verified_step = run.verified_step
    value = acc_step / (ms_step / 1e3)
    log(f"{args.workload}: {ms_step:.3f} ms/step, {acc_step:.1f} accepted / {verified_step} verified tokens per step")
    step = run.step

    # ---- roofline of the dominant kernel (gate/up GEMM + SwiGLU), timed live ----
    # Algorithmic bytes per launch: the layer's gate and up weights, read once
    # (2 x d_ffn x d_model bf16).  Time per launch: the average of HIP-event
    # pairs recorded around every gate/up launch on the stream it runs on.
    T = sum(b.T for b in batches) / nb   # slots per launch (the batches' mean)
    gu_bytes = 2 * m.d_ffn * m.d_model * m.wbytes
    gu_flops = 2.0 * T * 2 * m.d_ffn * m.d_model   # model FLOPs per launch
    prof_steps = max(3, args.steps // 2)
    sv.sd_profile_begin(v.ctx, sv.SD_K_GATEUP, prof_steps * nb * m.n_layers + 8)
    for _ in range(prof_steps):
        step(one_stream=True)
    gu_ms, gu_n = sv.sd_profile_end(v.ctx)
    # cost of an event pair with nothing between them, on the same stream (reported only)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(64)]
    for a, b in ev:
        a.record(run.streams[0])
        b.record(run.streams[0])
    torch.cuda.synchronize()
    pair_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    gu_avg_s = gu_ms / max(gu_n, 1) / 1e3
    achieved = gu_bytes / gu_avg_s / 1e9
    traffic = measured_traffic(args.workload)
    mfma_tf = gu_flops / gu_avg_s / 1e12
    roofline = {"bound": "hbm", "kernel": "gate/up GEMM with the SwiGLU epilogue (k_gemm16/k_gemm32)",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "traffic_over_algorithmic": round(traffic / gu_bytes, 4) if traffic else None,
                "bytes_per_launch": gu_bytes, "slots_per_launch": T, "avg_launch_us": round(gu_avg_s * 1e6, 2),
                "launches": gu_n, "empty_event_pair_us": round(pair_ms * 1e3, 2),
                "mfma_tflops": round(mfma_tf, 1), "mfma_frac_bf16": round(mfma_tf / BF16_PEAK_TFLOPS, 4)}

    # achievable peaks of this GPU (library calibration kernels): a read-only
    # stream and a copy of 1 GiB (4x the last-level cache), and a bf16 MFMA
    # loop with no memory traffic
    cal_buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    cal_sink = torch.empty(4, dtype=torch.float32, device="cuda")
    cs0 = run.streams[0].cuda_stream
    achievable = {"hbm_read_gbs": round(sv.sd_calib_hbm(cal_buf.data_ptr(), cal_buf.numel(), 1, 10, cs0), 1),
                  "hbm_copy_gbs": round(sv.sd_calib_hbm(cal_buf.data_ptr(), cal_buf.numel(), 0, 10, cs0), 1),
                  "mfma_bf16_tflops": round(sv.sd_calib_mfma(cal_sink.data_ptr(), 2048, cs0), 1),
                  "note": "sd_calib_hbm (1 GiB read-only stream; copy = bytes read + written) and "
                          "sd_calib_mfma (32x32x16 bf16 MFMA chains on every SIMD)"}
    del cal_buf, cal_sink
    hbm_ach = achievable["hbm_read_gbs"]
    roofline["frac_of_achievable"] = round(achieved / hbm_ach, 4)
    roofline["mfma_frac_of_achievable"] = round(mfma_tf / achievable["mfma_bf16_tflops"], 4)
    # the matrix cores run each product on both activation planes: twice the model's FLOPs
    roofline["mfma_issued_tflops"] = round(2 * mfma_tf, 1)
    roofline["mfma_issued_frac_bf16"] = round(2 * mfma_tf / BF16_PEAK_TFLOPS, 4)
    roofline["mfma_issued_frac_of_achievable"] = round(2 * mfma_tf / achievable["mfma_bf16_tflops"], 4)
    # MFMA work the counters saw (both planes and the last slot tile's padding),
    # over the live launch time, and the counted busy fraction of all SIMDs
    mm = measured_mfma(args.workload)
    if mm is not None:
        roofline["mfma_counted_tflops"] = round(mm[0] / gu_avg_s / 1e12, 1)
        roofline["mfma_counted_frac_bf16"] = round(mm[0] / gu_avg_s / 1e12 / BF16_PEAK_TFLOPS, 4)
        roofline["mfma_busy_frac_counted"] = mm[1]

    def class_ms(k, steps=3):
        """Per-step device time of one kernel class (sum of the event pairs
        around its launches)."""
        sv.sd_profile_begin(v.ctx, k, steps * nb * (4 * m.n_layers + 8))
        for _ in range(steps):
            step(one_stream=True)
        ms, n = sv.sd_profile_end(v.ctx)
        return max(ms, 1e-6) / steps

    # attention (all layers, KV streamed once per user) and sampler rates
    kv_read_step = sum(int(p + l + 1) for p, l in zip(w.prefix_len, w.draft_len)) * m.kv_bytes_per_token()
    attn_ms = class_ms(sv.SD_K_ATTN)
    nd_all = int(sum(int(b.draft_len.sum()) for b in batches))
    # phase A comes from the lm_head epilogue's statistics (no logits read);
    # phase B reads the stop slot's logits row and q row of every user
    if run.sparse is not None:
        # the stop rows; every sparse row's K entries (the accept lookups) and remainders
        samp_bytes = int(w.n_users) * m.vocab * 4 + nd_all * (args.q_topk * 8 + 4)
    else:
        samp_bytes = 2 * int(w.n_users) * m.vocab * 4
    samp_ms = class_ms(sv.SD_K_SAMPLER)
    kernels = {
        "attention": {"achieved": round(kv_read_step / (attn_ms / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                      "unit": "GB/s", "frac": round(kv_read_step / (attn_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                      "bytes_per_step": kv_read_step, "ms_per_step": round(attn_ms, 4),
                      "frac_of_achievable": round(kv_read_step / (attn_ms / 1e3) / 1e9 / hbm_ach, 4),
                      "note": "paged attention + chunk combine, all layers; bytes = cached and new K/V read once"},
        "sampler": {"achieved": round(samp_bytes / (samp_ms / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(samp_bytes / (samp_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                    "frac_of_achievable": round(samp_bytes / (samp_ms / 1e3) / 1e9 / hbm_ach, 4),
                    "bytes_per_step": samp_bytes, "ms_per_step": round(samp_ms, 4),
                    "note": ("phase-A merge of the lm_head statistics + accept/reject + resample "
                             "kernels; bytes = one fp32 logits row per user + "
                             + ("the sparse rows" if run.sparse is not None else "one q row per user"))},
    }

    breakdown = None
    if args.breakdown:
        breakdown = {}
        for name, k in (("qkv", sv.SD_K_QKV), ("attention", sv.SD_K_ATTN), ("o_proj", sv.SD_K_O),
                        ("gate_up", sv.SD_K_GATEUP), ("down", sv.SD_K_DOWN), ("lm_head", sv.SD_K_LMHEAD),
                        ("sampler", sv.SD_K_SAMPLER), ("small", sv.SD_K_SMALL)):
            breakdown[name] = round(class_ms(k), 4)
        log(f"per-step ms by kernel class: {breakdown}")

    # algorithmic bytes of one step: weights once per batch, each user's KV
    # once, logits and q rows once
    wbytes = (m.n_layers * m.layer_params() + 2 * m.vocab * m.d_model) * m.wbytes
    wbytes -= m.vocab * m.d_model * m.wbytes  # embedding: only T rows are read
    step_bytes = nb * wbytes + kv_read_step
    result = {
        "metric": "accepted tokens/s, Qwen3-32B-shaped batch verify; MFMA util + HBM GB/s",
        "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "ms_per_step_p10_p50_p90": [round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": m.dtype,
        "data": "synthetic (random-init weights N(0,0.02), synthetic KV N(0,1), synthetic draft q)",
        "config": {"workload": args.workload, "model": m.name, "mode": args.mode,
                   "users": int(w.n_users), "batches": nb, "verified_tokens_per_step": verified_step,
                   "prefix_tokens": run.kv_tokens, "hip_graph": bool(run.graph) and run.sparse is None,
                   "q_payload": (f"sparse top-{args.q_topk} + remainder" if run.sparse is not None
                                 else "dense fp32 rows"),
                   "q_payload_bytes_per_step": (nd_all * (args.q_topk * 8 + 4) if run.sparse is not None
                                                else nd_all * m.vocab * 4),
                   "streams": len(run.streams)},
        "verified_tokens_per_s": round(verified_step / (ms_step / 1e3), 1),
        "accepted_per_step": acc_step,
        "step_hbm_floor_ms": round(step_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 3),
        "step_algorithmic_gb": round(step_bytes / 1e9, 2),
        "step_effective_gbs": round(step_bytes / (ms_step / 1e3) / 1e9, 1),
        "roofline": roofline,
        "kernels": kernels,
        "achievable": achievable,
    }
    if breakdown is not None:
        result["breakdown_ms"] = breakdown
    if args.mode == "stochastic" and not args.no_greedy and "greedy" in w.modes:
        result["greedy"] = greedy_run(run, args.steps, args.warmup)
    cpu_batch = batches[0]
    run.close()
    del run

    extras = [x for x in args.extra.split(",") if x and x != "none" and x != args.workload]
    if extras:
        result["workloads"] = {}
    for name in extras:
        r = Run(name, args, torch)
        ms_x, acc_x, per_x = r.time(args.steps, args.warmup)
        rec = {"value": round(acc_x / (ms_x / 1e3), 2), "unit": "tokens/s", "ms_per_step": round(ms_x, 4),
               "ms_per_step_p10_p50_p90": [round(float(np.percentile(per_x, q)), 4) for q in (10, 50, 90)],
               "accepted_per_step": acc_x, "verified_tokens_per_step": r.verified_step,
               "verified_tokens_per_s": round(r.verified_step / (ms_x / 1e3), 1),
               "users": int(r.w.n_users), "batches": r.nb, "prefix_tokens": r.kv_tokens,
               "hip_graph": bool(r.graph), "streams": len(r.streams), "mode": "stochastic"}
        log(f"{name}: {ms_x:.3f} ms/step, {acc_x:.1f} accepted / {r.verified_step} verified tokens per step")
        if not args.no_greedy and "greedy" in r.w.modes:
            rec["greedy"] = greedy_run(r, args.steps, args.warmup)
        result["workloads"][name] = rec
        r.close()
        del r

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, cpu_batch, args.cpu_layers, acc_step / verified_step)
    print(json.dumps(result), flush=True)


def measured_mfma(workload):
    """MFMA work and busy fraction per gate/up launch from the committed SQ
    counter summary (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512, SQ_VALU_MFMA_BUSY_CYCLES),
    or None when it covers another workload or the GEMM source has changed."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"mfma_lds_counters_{workload}.md")
    src = os.path.join(ROOT, "paper_2604_20919_amd", "csrc", "k_gemm.hip")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    f = re.search(r"gateup_mfma_flop_per_launch: (\d+)", text)
    b = re.search(r"gateup_mfma_busy_frac: ([0-9.]+)", text)
    h = re.search(r"k_gemm.hip sha256: ([0-9a-f]{64})", text)
    if not (f and b and h) or hashlib.sha256(open(src, "rb").read()).hexdigest() != h.group(1):
        return None
    return int(f.group(1)), float(b.group(1))


def measured_traffic(workload):
    """HBM bytes per gate/up launch from the committed FETCH_SIZE/WRITE_SIZE
    summary, or None when it covers another workload or the GEMM source has
    changed since the counters were taken."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"k_gemm_gateup_{workload}_hbm_traffic.md")
    src = os.path.join(ROOT, "paper_2604_20919_amd", "csrc", "k_gemm.hip")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"traffic_bytes_per_launch: (\d+)", text)
    h = re.search(r"k_gemm.hip sha256: ([0-9a-f]{64})", text)
    if not (m and h):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != h.group(1):
        return None
    return int(m.group(1))


def greedy_run(run, steps, warmup):
    """The same workload in greedy mode (accept iff the draft is the
    target's argmax), with drafts planted to follow the target's own argmax
    for k_m ~ U{0..l_m} steps; timed like the stochastic run."""
    plant_greedy_drafts(run.v, run.w, run.batches, run.dev_in, run.torch)
    ms_step, acc_step, _ = run.time(steps, warmup, mode="greedy")
    log(f"{run.name} greedy: {ms_step:.3f} ms/step, {acc_step:.1f} accepted per step")
    return {"value": round(acc_step / (ms_step / 1e3), 2), "unit": "tokens/s",
            "ms_per_step": round(ms_step, 4), "accepted_per_step": acc_step,
            "drafts": "first k_m drafts follow the target's argmax, k_m ~ U{0..l_m}"}


def plant_greedy_drafts(v, w, batches, dev_in, torch):
    """Greedy workload: user m's first k_m drafts follow the target's own
    argmax continuation (k_m uniform in 0..l_m, seeded), then one random
    token; found with l_max greedy passes on the GPU: at pass j a user whose
    first j drafts already follow the argmax stops at slot j, where the
    returned token is the argmax (or later, when its draft j is the argmax
    already)."""
    import workload as wl
    for n, b in enumerate(batches):
        d, q, au = dev_in[n]
        k = wl._ints(len(b.users), w.seed, wl.S_LEN << 8, 0, int(b.draft_len.max()))
        k = np.minimum(k, b.draft_len)
        doff = np.concatenate([[0], np.cumsum(b.draft_len)]).astype(np.int64)
        drafts = b.drafts.copy()
        for j in range(int(b.draft_len.max())):
            d.copy_(torch.from_numpy(drafts))
            v.verify(n, w.assign, w.draft_len, d, q, "greedy")
            n_acc, tok = v.accept(n, w.n_users)
            for i, u in enumerate(b.users):
                if j < b.draft_len[i] and j < k[i]:
                    a = int(n_acc[u])
                    assert a >= j, "a planted argmax draft was rejected"
                    if a == j:
                        drafts[doff[i] + j] = tok[u]
        d.copy_(torch.from_numpy(drafts))
        b.drafts = drafts


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, b, n_layers_sample, acc_per_verified):
    """The oracle on the host cores: every user of the batch through
    n_layers_sample decoder layers, plus lm_head and the sampler, timed with
    weight generation excluded (and reported); the per-layer time is
    extrapolated to all layers (users are independent and every layer costs
    the same)."""
    import oracle
    m = w.model
    threads = oracle.omp_threads()
    t0 = time.perf_counter()
    ws = oracle.WeightSource(m, w.seed)
    layers = {l: ws.layer(l) for l in range(n_layers_sample)}
    t_gen = time.perf_counter() - t0

    class Cached(oracle.WeightSource):
        def __init__(self):
            self.m, self.seed, self.gamma, self._glob = m, w.seed, "ones", ws._glob

        def layer(self, l):
            return layers[l]

    import dataclasses
    ms = dataclasses.replace(m, n_layers=n_layers_sample)
    users, P, n = b.users, b.prefix_len, b.n_slots
    toks = b.slot_tokens()
    t0 = time.perf_counter()
    logits = oracle.forward(ms, Cached(), oracle.KVSource(ms, w.seed, users, P), P, n, toks)
    t_fwd = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.sample("stochastic", users, b.draft_len, logits, b.drafts, b.q, None, w.seed, 0)
    t_samp = time.perf_counter() - t0
    # split the measured forward into per-layer and lm_head parts: time the
    # lm_head alone with a zero-layer model
    m0 = dataclasses.replace(m, n_layers=0)
    t0 = time.perf_counter()
    oracle.forward(m0, Cached(), oracle.KVSource(m0, w.seed, users, P), P, n, toks)
    t_head = time.perf_counter() - t0
    t_layer = max(t_fwd - t_head, 0.0) / n_layers_sample
    per_batch = t_layer * m.n_layers + t_head + t_samp
    slots = int(n.sum())
    cpu_tok_s = slots * acc_per_verified / per_batch
    return {"value": round(cpu_tok_s, 4), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": _cpu_model(), "omp_threads": threads, "host_cpus": os.cpu_count(),
            "weight_generation_s": round(t_gen, 2), "per_batch_s_extrapolated": round(per_batch, 2),
            "sample": (f"all {len(users)} users of the batch ({slots} query slots, prefixes "
                       f"{int(P.min())}-{int(P.max())}): {n_layers_sample} of {m.n_layers} decoder layers "
                       f"timed ({t_layer:.2f} s/layer), lm_head {t_head:.2f} s and sampler {t_samp:.2f} s "
                       f"timed ({t_fwd + t_head + t_samp:.1f} s of CPU work on {threads} OpenMP threads), "
                       f"extrapolated to {per_batch:.1f} s per batch; accepted = verified x "
                       f"{acc_per_verified:.3f} (the GPU run's ratio); weight generation "
                       f"({t_gen:.1f} s for {n_layers_sample} layers) excluded")}


if __name__ == "__main__":
    main()
