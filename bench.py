"""Benchmark of one engine step of the large-v3-shaped ASR path on one MI355X.

A step is one pass of the whole hot path on one batch of synthetic input:

  * submit 64 requests of 30 s of seeded PCM (resident in HBM) and pop them
    from the duration-aware queue (SJF on duration, Section 3.2);
  * prefill them: log-mel front-end, conv stem, 32 encoder layers, ln_post,
    cross K/V of all 32 decoder layers into 64 fresh slots;
  * one teacher-forced decode step of 128 running sequences (self-attention
    caches pre-filled to lengths U[10, 400], 1500 cross positions each), with
    the vocabulary projection fused with argmax;
  * slot bookkeeping (the 64 prefill slots are released for the next step).

The 128 running sequences come from an SJF-ordered stream of 2000 requests
with lognormal durations.  Weights are random (seeded); no dataset is read.

Prints ONE JSON line.  `value` is audio-seconds of speech prefilled per
second of wall time over whole steps (the decode step riding along);
`decode_tokens_per_s` and `encoder_audio_s_per_s` use the phase times
measured with HIP events inside the same timed steps.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_bf16_large-v3_step_traffic.md")
# the GEMM kernels and the device helpers their epilogues inline
GEMM_SOURCES = [os.path.join(ROOT, "paper_2603_11273_amd", "csrc", f)
                for f in ("k_gemm.hip", "asr_device.h", "asr_kernels.h")]


def gemm_traffic_per_launch():
    """Counter-measured bytes per GEMM launch, or None once the kernel source
    differs from the one the counters were taken on."""
    import hashlib
    import re
    try:
        text = open(TRAFFIC_SUMMARY).read()
        rec = json.loads(re.search(r"```json\n(.*?)\n```", text, re.S).group(1))
        h = hashlib.sha256()
        for f in GEMM_SOURCES:
            h.update(open(f, "rb").read())
        sha = h.hexdigest()[:16]
    except Exception:
        return None
    return rec["gemm_bytes_per_launch"] if rec.get("kernel_source_sha256_16") == sha else None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--prefill", type=int, default=64)
    ap.add_argument("--decode", type=int, default=128)
    ap.add_argument("--breakdown-steps", type=int, default=3,
                    help="untimed-for-value steps with every launch timed (per-class table)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-serving", action="store_true",
                    help="skip the continuous-batching run and the serving simulation")
    ap.add_argument("--cpu-budget-s", type=float, default=25.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (3 times): the reference "
                         "reading for the FETCH_SIZE / WRITE_SIZE counters")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                          "(the path shards by request, see DESIGN.md)"}))
        sys.exit(2)
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "one GPU only"}))
        sys.exit(2)
    import torch
    from paper_2603_11273_amd import asr, synth

    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")      # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": src.numel() * 4, "copies": 3}))
        return

    if args.warmup + args.steps > 45:
        raise SystemExit("warmup + steps must stay <= 45 (decode positions stay below 448)")
    P, D = args.prefill, args.decode
    shape = synth.SHAPES["large-v3"]
    enc_wl = synth.WORKLOADS["large-v3-encoder"]
    dec_wl = synth.WORKLOADS["large-v3-decode"]
    dev = torch.device("cuda:0")

    # ---------------------------------------------------------------- context
    cfg = asr.model_cfg(shape, max_slots=D + P, max_prefill=P, max_decode=D, max_queue=4096)
    ctx = asr.Context(cfg, device=0)
    log(f"workspace {ctx.workspace_size() / 2**30:.1f} GiB")
    ctx.bind()
    t0 = time.time()
    params = synth.model_params(shape, enc_wl.seed, device=dev)
    ctx.load_weights(list(params.values()), on_device=True)
    torch.cuda.synchronize()
    log(f"weights generated + loaded in {time.time() - t0:.1f} s")

    # ------------------------------------------- the running decode sequences
    # SJF-ordered stream of 2000 lognormal requests (queue-only context)
    q = asr.Context(cfg, device=-1)
    q.set_policy(asr.SJF)
    n_req = dec_wl.extra["n_requests"]
    durs = synth.durations_lognormal(dec_wl.seed, n_req)
    ns = synth.n_samples_of(durs)
    arr = synth.poisson_arrivals_us(dec_wl.seed, n_req, 25.0)
    tq = time.perf_counter()
    for i in range(n_req):
        q.submit(i, None, n_samples=int(ns[i]), duration_us=int(ns[i]) * 10**6 // 16000,
                 arrival_us=int(arr[i]))
    running = q.pop_batch(int(arr[n_req // 2]), D)
    queue_us_per_req = (time.perf_counter() - tq) * 1e6 / n_req
    steps_left = [max(1, min(448, (27 * int(ns[i]) + 80000) // 160000)) for i in running]

    kv_len = synth.kv_lengths(dec_wl.seed, D, dec_wl.extra["kv_lo"], dec_wl.extra["kv_hi"])
    t0 = time.time()
    for s0 in range(0, D, P):
        idx = list(range(s0, min(D, s0 + P)))
        E = torch.stack([synth.encoder_output(dec_wl.seed, b, shape.d_model, device=dev)
                         for b in idx])
        ctx.debug_set_encoder_out(idx, [-1] * len(idx), [steps_left[b] for b in idx], E,
                                  on_device=True)
        del E
    for b in range(D):
        kv = synth.self_kv_prefix(dec_wl.seed, b, shape.n_dec, shape.n_head, device=dev)
        ctx.debug_set_self_kv(b, kv, int(kv_len[b]), on_device=True)
        del kv
    torch.cuda.synchronize()
    log(f"{D} decode slots filled in {time.time() - t0:.1f} s")

    # -------------------------------------------------- prefill audio in HBM
    pcm_host = np.stack([synth.pcm_clip(enc_wl.seed, i, synth.N_SAMPLES_30S)
                         for i in range(P)])
    pcm = torch.from_numpy(pcm_host).to(dev)
    toks = synth.token_ids(dec_wl.seed, (args.warmup + args.steps + max(1, args.breakdown_steps), D),
                           shape.vocab)
    del params
    torch.cuda.empty_cache()

    next_id = [10**6]
    vclock = [int(arr[-1]) + 1]

    def one_step(k):
        ids = []
        for i in range(P):
            ctx.submit(next_id[0], pcm[i], n_samples=synth.N_SAMPLES_30S,
                       arrival_us=vclock[0] + i, on_device=True)
            next_id[0] += 1
        popped = ctx.pop_batch(vclock[0] + P, P)
        vclock[0] += 10**6
        out = ctx.step(prefill_ids=popped, slots=list(range(D)), tokens=[int(t) for t in toks[k]])
        for s in out["slot_of"]:
            ctx.release_slot(int(s))
        return out

    ctx.set_policy(asr.SJF)
    for k in range(args.warmup):
        one_step(k)
    torch.cuda.synchronize()
    log("warmup done")

    # Timed region: event pairs only around the two phases of a step (the
    # encoder runs its two clip groups on two streams, so per-launch times
    # would overlap; kernels are timed in the pass below).
    ctx.reset_timing()
    ctx.set_timing((1 << asr.K_PREFILL) | (1 << asr.K_DECODE) | (1 << asr.K_ENCODE))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        one_step(args.warmup + k)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ctx.set_timing(False)
    tm = ctx.timing()
    log(f"timed {args.steps} steps in {wall:.3f} s")

    # Per-class breakdown and the rooflines on further steps with the encoder
    # as one stream (every launch owns the GPU) and every launch bracketed
    # (the extra events slow the many short decode launches a little).
    nb = max(1, args.breakdown_steps)
    ctx.set_encoder_streams(1)
    ctx.reset_timing()
    ctx.set_timing(True)
    for k in range(nb):
        one_step(args.warmup + args.steps + k)
    torch.cuda.synchronize()
    ctx.set_timing(False)
    ctx.set_encoder_streams(2)
    tb = ctx.timing()

    ms_step = wall * 1e3 / args.steps
    audio_s = P * 30.0
    enc_ms = tm["prefill"]["ms"] / args.steps
    encode_ms = tm["encode"]["ms"] / args.steps
    dec_ms = tm["decode"]["ms"] / args.steps
    # every MFMA GEMM launch: encoder and stem products plus the cross K/V product
    g = {k: tb["gemm"][k] + tb["xkv"][k] for k in ("ms", "flops", "launches")}
    gemm_tflops = g["flops"] / (g["ms"] * 1e-3) / 1e12 if g["ms"] else 0.0
    da = tb["dattn"]
    dattn_gbs = da["bytes"] / (da["ms"] * 1e-3) / 1e9 if da["ms"] else 0.0
    # algorithmic work of the timed steps, from the shapes alone
    work = algorithmic_work(shape, P, D, kv_len, args.warmup, args.steps)
    kernels = {k: {"ms_per_step": v["ms"] / nb, "launches_per_step": v["launches"] / nb}
               for k, v in tb.items()}

    result = {
        "metric": "encoder audio-sec/s + decode tokens/s at large-v3 shape; % MFMA peak / % HBM BW",
        "value": round(audio_s / (ms_step * 1e-3), 1),
        "unit": "audio-s/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded PCM, random-init weights; no dataset)",
        "config": {"workload": f"large-v3 step: prefill {P} x 30 s clips + decode {D} sequences "
                               "(self-KV U[10,400], 1500 cross positions)",
                   "prefill_clips": P, "decode_rows": D, "n_mels": 128, "d_model": 1280,
                   "layers": "32+32", "vocab": 51866, "parallelism": "none (1 GPU)"},
        "encoder_audio_s_per_s": round(audio_s / (encode_ms * 1e-3), 1) if encode_ms else None,
        "prefill_audio_s_per_s": round(audio_s / (enc_ms * 1e-3), 1) if enc_ms else None,
        "decode_tokens_per_s": round(D / (dec_ms * 1e-3), 1) if dec_ms else None,
        "prefill_ms": round(enc_ms, 3),
        "encoder_ms": round(encode_ms, 3),
        "cross_kv_ms": round(enc_ms - encode_ms, 3),
        "decode_ms": round(dec_ms, 3),
        # stem + encoder GEMMs + attention flops over the encoder's wall time
        # (mel .. ln_post); cross K/V reported on its own
        "encoder_mfma_frac": round(work["encoder_flops"] / (encode_ms * 1e-3) / 1e12
                                   / PEAK_BF16_TFLOPS, 4) if encode_ms else None,
        "cross_kv_mfma_frac": round(work["cross_kv_flops"] / ((enc_ms - encode_ms) * 1e-3)
                                    / 1e12 / PEAK_BF16_TFLOPS, 4) if enc_ms > encode_ms else None,
        # weights + cross K/V + self K/V at the timed steps' own positions
        "decode_bytes_per_step": round(work["decode_bytes"]),
        "decode_hbm_frac": round(work["decode_bytes"] / (dec_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        if dec_ms else None,
        "work_note": "encoder flops " + f"{work['encoder_flops']:.4g}" + " and decode bytes from "
                     "the model shape and the timed steps' cache lengths; the 64 clips' PCM is "
                     "resident in HBM before the timed region (its host-to-device copy is not "
                     "timed)",
        "queue_us_per_request": round(queue_us_per_req, 3),
        "kernels": kernels,
        "kernels_note": f"per-class breakdown and rooflines over {nb} further steps with the "
                        "encoder on one stream and every launch timed",
        "roofline": {"bound": "mfma", "kernel": "gemm_bf16 (encoder, stem, cross K/V)",
                     "achieved": round(gemm_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": gemm_traffic_per_launch(),
                     "flops_per_launch": round(g["flops"] / max(1, g["launches"])),
                     "avg_launch_us": round(g["ms"] * 1e3 / max(1, g["launches"]), 1)},
        "roofline_decode": {"bound": "hbm", "kernel": "decode attention (self + cross)",
                            "achieved": round(dattn_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": round(dattn_gbs / PEAK_HBM_GBS, 4), "traffic": None},
    }
    if not args.no_serving:
        result["serving"] = serving_section(ctx, D, P, enc_ms, dec_ms, toks,
                                            args.warmup + args.steps + nb)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(shape, enc_wl, dec_wl, pcm_host[0], P, D,
                                              ms_step, args.cpu_budget_s)
    print(json.dumps(result), flush=True)


def algorithmic_work(shape, P, D, kv_len, warmup, steps):
    """Algorithmic flops of the encoder and bytes of the decode step at the
    benchmark's shape (2 flops per multiply-add; each operand read once).

    Encoder (per clip): conv1 3000 x d x 3 n_mels, conv2 1500 x d x 3d; per
    layer QKV 1500 x 3d x d, out-projection 1500 x d x d, FC1 and FC2
    1500 x F x d; attention 4 x 1500^2 x 64 per head.  Cross K/V: 1500 x
    (L_dec 2 d) x d per clip.  Decode step: every decoder weight matrix and the
    token embedding (bf16), the cross K/V of all rows (1500 positions), and
    the self K/V of each row over its length + 1 positions at the timed
    steps (the cache grows by one position per step)."""
    d, F, H, M = shape.d_model, shape.d_ffn, shape.n_head, shape.n_mels
    Le, Ld, V = shape.n_enc, shape.n_dec, shape.vocab
    T = 1500
    stem = 2.0 * 3000 * d * 3 * M + 2.0 * T * d * 3 * d
    layer = 2.0 * T * d * (3 * d + d + 2 * F) + 4.0 * T * T * 64 * H
    enc = P * (stem + Le * layer)
    xkv = P * 2.0 * T * (Ld * 2 * d) * d
    w_bytes = 2.0 * (Ld * (3 * d * d + 3 * d * d + 2 * F * d) + V * d)
    cross_bytes = 2.0 * D * Ld * 2 * T * d
    keys = np.mean([np.sum(np.asarray(kv_len, np.int64) + warmup + k + 1) for k in range(steps)])
    self_bytes = 2.0 * Ld * 2 * keys * d
    return {"encoder_flops": enc, "cross_kv_flops": xkv,
            "decode_bytes": w_bytes + cross_bytes + self_bytes}


def serving_section(ctx, D, P, enc_ms, dec_ms, toks, steps_done):
    """Continuous batching at the large-v3 shape.

    1. Decode cost at 16 rows (the bench measured 128): a per-step and a
       per-row term for the virtual clock.
    2. A real burst on the GPU: 256 lognormal-duration requests (the LibriSpeech
       stand-in) through asr_serve_step with 128 slots and up to 64 prefills per
       step; wall-clock throughput, and the virtual clock's prediction of the
       same run with the measured costs.
    3. The paper's evaluation on that virtual clock (native simulator, queue-only
       context): 5-minute Poisson streams at 5 / 15 / 25 requests/s plus a
       500-request burst, FCFS / SJF / HRRN, P50 / P90 TTFT and E2EL and the
       change against FCFS; and the host cost of scheduling per request."""
    import numpy as np
    import torch
    from paper_2603_11273_amd import asr, synth
    from paper_2603_11273_amd import serving_metrics as SM

    # 1. decode cost at 16 rows (positions stay below 448: the bench's slots
    #    start at <= 400 and have advanced steps_done + 3 positions)
    rows = 16
    t16 = []
    for k in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctx.step(slots=list(range(rows)), tokens=[int(t) for t in toks[k % len(toks)][:rows]])
        t16.append(time.perf_counter() - t0)
    dec16_ms = min(t16) * 1e3
    row_us = max(0.0, (dec_ms - dec16_ms) * 1e3 / (D - rows))
    step_us = max(1.0, dec16_ms * 1e3 - rows * row_us)
    prefill_us = enc_ms * 1e3 / P
    cost = dict(prefill_us=int(round(prefill_us)), step_us=int(round(step_us)),
                row_us=int(round(row_us)))
    log(f"serving cost model: {cost}")

    # 2. a burst on the GPU
    for s in range(ctx.cfg.max_slots):
        ctx.release_slot(s)
    n_burst = 256
    seed = synth.WORKLOADS["large-v3-decode"].seed + 7
    ns = synth.n_samples_of(synth.durations_lognormal(seed, n_burst))
    clips = [synth.pcm_clip(seed, i, int(ns[i])) for i in range(n_burst)]
    def burst(overlap, id0):
        ctx.set_policy(asr.HRRN)
        ctx.serve_config(kv_capacity=0, cross_tokens=1500, max_admit=P, start_token=50258,
                         overlap=overlap)
        for i, pcm in enumerate(clips):
            ctx.submit(id0 + i, pcm, arrival_us=0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        done, n_steps, n_tok, t_virtual = 0, 0, 0, 0
        while done < n_burst:
            r = ctx.serve_step(0)
            n_steps += 1
            n_tok += len(r["decoded"])
            t_virtual += (cost["prefill_us"] * len(r["admitted"]) +
                          (cost["step_us"] + cost["row_us"] * len(r["decoded"])
                           if r["decoded"] else 0))
            for rid in r["finished"]:
                ctx.serve_tokens(rid)
            done += len(r["finished"])
        wall = time.perf_counter() - t0
        return {"requests": n_burst, "policy": "HRRN", "steps": n_steps, "output_tokens": n_tok,
                "wall_s": round(wall, 3), "req_per_s": round(n_burst / wall, 1),
                "tok_per_s": round(n_tok / wall, 1), "virtual_clock_s": round(t_virtual * 1e-6, 3)}

    gpu = burst(False, 10**7)
    log(f"GPU burst: {gpu}")

    # real-time Poisson serving on the GPU (arrivals on the wall clock), with
    # and without the prefill overlapped on a second stream: most steps then
    # admit a few requests while up to 128 others decode
    def realtime(overlap, id0, rate, seconds):
        n = int(rate * seconds)
        s3 = seed + 99
        n_s = synth.n_samples_of(synth.durations_lognormal(s3, n))
        arr = synth.poisson_arrivals_us(s3, n, rate)
        ctx.set_policy(asr.HRRN)
        ctx.serve_config(kv_capacity=0, cross_tokens=1500, max_admit=P, start_token=50258,
                         overlap=int(overlap))
        for i in range(n):
            ctx.submit(id0 + i, clips[i % n_burst][:int(n_s[i])], arrival_us=int(arr[i]))
        emit, steps, busy, n_fin = {}, 0, 0.0, 0
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        t_end = 0
        while n_fin < n:
            now = int((time.perf_counter() - t0) * 1e6)
            ts = time.perf_counter()
            r = ctx.serve_step(now)
            te = time.perf_counter()
            end_us = int((te - t0) * 1e6)
            if r["decoded"]:
                steps += 1
                busy += te - ts
            # every decoded row emits one token at the end of the step (no
            # preemption here: the pool is unbounded)
            for rid in r["decoded"]:
                emit.setdefault(rid, []).append(end_us)
            for rid in r["finished"]:
                ctx.serve_tokens(rid)
                n_fin += 1
                t_end = end_us
            if not r["decoded"] and not r["admitted"]:
                time.sleep(0.0002)
        ids = [id0 + i for i in range(n)]
        m = SM.latency_metrics(arr, [emit[i][0] for i in ids], [emit[i][-1] for i in ids],
                               [len(emit[i]) for i in ids], [t for i in ids for t in emit[i]],
                               t_end)
        return {"requests": n, "rate_per_s": rate,
                "ttft_p50_s": round(m["ttft_p50_us"] * 1e-6, 4),
                "ttft_p90_s": round(m["ttft_p90_us"] * 1e-6, 4),
                "e2el_p50_s": round(m["e2el_p50_us"] * 1e-6, 4),
                "e2el_p90_s": round(m["e2el_p90_us"] * 1e-6, 4),
                "tpot_mean_ms": round(m["tpot_mean_us"] * 1e-3, 3),
                "itl_p50_ms": round(m["itl_p50_us"] * 1e-3, 3),
                "itl_p90_ms": round(m["itl_p90_us"] * 1e-3, 3),
                "busy_steps": steps,
                "mean_busy_step_ms": round(busy * 1e3 / max(steps, 1), 3)}

    rt_rate = round(0.6 * gpu["req_per_s"], 1)
    rt = {"sequential": realtime(0, 3 * 10**7, rt_rate, 4.0),
          "overlapped_prefill": realtime(1, 4 * 10**7, rt_rate, 4.0),
          "overlapped_prefill_32_cus_reserved": realtime(32, 5 * 10**7, rt_rate, 4.0)}
    log(f"GPU real-time serving: {rt}")

    # 3. the paper's evaluation on the virtual clock
    DYNAMIC = 3

    def run(policy, n, rate, burst=False):
        q = asr.Context(asr.model_cfg(synth.SHAPES["large-v3"], max_slots=D, max_prefill=P,
                                      max_decode=D, max_queue=n + 1), device=-1)
        if policy == DYNAMIC:
            # FCFS while every eligible request is admitted this step, HRRN once
            # some request's response ratio passes 3, SJF otherwise
            q.serve_config(kv_capacity=0, cross_tokens=1500, max_admit=P, dynamic=True,
                           depth_low=P, starve=(3, 1))
        else:
            q.set_policy(policy)
            q.serve_config(kv_capacity=0, cross_tokens=1500, max_admit=P)
        s2 = seed + int(rate * 10)
        n_s = synth.n_samples_of(synth.durations_lognormal(s2, n))
        arr = np.zeros(n, np.int64) if burst else synth.poisson_arrivals_us(s2, n, rate)
        for i in range(n):
            q.submit(i, None, n_samples=int(n_s[i]), arrival_us=int(arr[i]))
        t0 = time.perf_counter()
        info, t_end = q.serve_simulate(list(range(n)), want_token_times=True, **cost)
        host_us = (time.perf_counter() - t0) * 1e6 / n
        m = SM.latency_metrics(arr, [info[i]["first_us"] for i in range(n)],
                               [info[i]["finish_us"] for i in range(n)],
                               [info[i]["n_tokens"] for i in range(n)],
                               [t for i in range(n) for t in info[i]["token_us"]], t_end)
        extra = {}
        if policy == DYNAMIC:
            st = q.serve_stats()
            extra["steps_fcfs_sjf_hrrn"] = st
        return {**extra, "ttft_p50_s": round(m["ttft_p50_us"] * 1e-6, 3),
                "ttft_p90_s": round(m["ttft_p90_us"] * 1e-6, 3),
                "e2el_p50_s": round(m["e2el_p50_us"] * 1e-6, 3),
                "e2el_p90_s": round(m["e2el_p90_us"] * 1e-6, 3),
                "tpot_mean_ms": round(m["tpot_mean_us"] * 1e-3, 3),
                "itl_p50_ms": round(m["itl_p50_us"] * 1e-3, 3),
                "itl_p90_ms": round(m["itl_p90_us"] * 1e-3, 3),
                "req_per_s": round(m["req_per_s"], 2), "tok_per_s": round(m["tok_per_s"], 1),
                "sched_host_us_per_request": round(host_us, 2)}

    names = {asr.FCFS: "fcfs", asr.SJF: "sjf", asr.HRRN: "hrrn", DYNAMIC: "dynamic"}
    sim = {"burst_500": {names[p]: run(p, 500, 0, burst=True) for p in names}}
    # Poisson streams (60 s each) at fractions of the engine's saturation rate
    # (the burst's throughput): the paper's 1-25 req/s span the A100 engine's
    # range up to and past its saturation; the same regimes here are higher.
    sat = sim["burst_500"]["fcfs"]["req_per_s"]
    for frac in (0.5, 0.9, 1.2):
        rate = round(sat * frac, 1)
        sim[f"poisson_{frac:g}x_saturation"] = dict(
            rate_per_s=rate, **{names[p]: run(p, int(rate * 60), rate) for p in names})
    for case in sim.values():
        base = case["fcfs"]
        for pol in ("sjf", "hrrn", "dynamic"):
            case[pol]["vs_fcfs_pct"] = {
                k: round(100.0 * (case[pol][k] - base[k]) / base[k], 1) if base[k] else None
                for k in ("ttft_p50_s", "ttft_p90_s", "e2el_p50_s", "e2el_p90_s",
                          "tpot_mean_ms", "itl_p50_ms", "itl_p90_ms")}
    return {"cost_model_us": cost, "decode_16_rows_ms": round(dec16_ms, 3), "gpu_burst": gpu,
            "gpu_realtime_poisson": rt,
            "simulation": sim,
            "note": "virtual clock with the costs measured above; lognormal durations stand in "
                    "for LibriSpeech test-clean; 128 slots, up to 64 prefills per step; "
                    "Poisson rates are fractions of the burst's (saturated) throughput"}


def cpu_baseline(shape, enc_wl, dec_wl, pcm0, P, D, ms_step, budget_s):
    """The oracle, as it stands, on a bounded sample of the same step: one clip
    through mel + encoder + cross K/V and one sequence through one decode step,
    extrapolated linearly to the P clips and D sequences of a step."""
    import torch
    from oracle import mel as OM
    from oracle import whisper as OW
    from paper_2603_11273_amd import synth
    cores = len(os.sched_getaffinity(0))
    torch.set_num_threads(cores)
    log(f"cpu baseline on {cores} cores")
    # parameters from the same generator (device copy brought to the host)
    params = {k: v.cpu() for k, v in synth.model_params(shape, enc_wl.seed, device="cuda").items()}
    t0 = time.perf_counter()
    mel = OM.log_mel(pcm0, shape.n_mels)
    E = OW.encode(mel, params, shape.n_enc, shape.n_head)
    ckv = OW.cross_kv(E, params, shape.n_dec)
    t_clip = time.perf_counter() - t0
    log(f"oracle: one clip prefill {t_clip:.1f} s")
    kv = synth.self_kv_prefix(dec_wl.seed, 0, shape.n_dec, shape.n_head).numpy().astype(np.float64)
    L = 205
    kp = [kv[l, 0, :, :L].transpose(1, 0, 2).reshape(L, -1) for l in range(shape.n_dec)]
    vp = [kv[l, 1, :, :L].transpose(1, 0, 2).reshape(L, -1) for l in range(shape.n_dec)]
    st = OW.DecoderState(shape.n_dec, shape.d_model, kp, vp)
    t0 = time.perf_counter()
    OW.decoder_step(1, st, ckv, params, shape.n_dec, shape.n_head)
    t_tok = time.perf_counter() - t0
    log(f"oracle: one sequence decode step {t_tok:.1f} s")
    step_s = P * t_clip + D * t_tok
    return {"value": round(P * 30.0 / step_s, 4), "unit": "audio-s/s", "cores": cores,
            "kind": "oracle",
            "sample": f"1 clip (30 s) mel+encoder+cross-K/V ({t_clip:.1f} s) and 1 sequence "
                      f"decode step at self-KV length 205 ({t_tok:.2f} s), fp64 numpy, "
                      f"extrapolated to {P} clips + {D} sequences per step",
            "extrapolated": True,
            "decode_tokens_per_s": round(1.0 / t_tok, 3),
            "encoder_audio_s_per_s": round(30.0 / t_clip, 3)}


if __name__ == "__main__":
    main()
