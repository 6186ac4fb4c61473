"""Parity at the five measured workloads' full sizes, in the launch
configurations the benchmark uses; the oracle checks sampled clips / rows
(batch elements are independent, so a sample is a complete check of them)."""
import numpy as np
import pytest
import torch

from oracle import mel as OM
from oracle import queue as OQ
from oracle import whisper as OW
from paper_2603_11273_amd import synth

from gpu_util import TOL, check_argmax, needs_gpu, rel_err

pytestmark = [pytest.mark.gpu, needs_gpu]


def _context(shape, seed, **cap):
    from paper_2603_11273_amd import asr
    ctx = asr.Context(asr.model_cfg(shape, **cap), device=0)
    ctx.bind()
    params = synth.model_params(shape, seed, device="cuda")
    ctx.load_weights(list(params.values()), on_device=True)
    torch.cuda.synchronize()
    # the oracle's copy comes from the same generator (device copy brought to the host)
    host = {k: v.cpu() for k, v in params.items()}
    del params
    torch.cuda.empty_cache()
    return ctx, host


@pytest.mark.parametrize("kmax,bits,offset,fine", [(141, 12, 0.0, False), (141, 12, 1.0, False),
                                                   (221, 7, 0.0, False), (141, 12, 0.0, True),
                                                   (141, 12, 1.0, True)])
def test_generator_is_device_independent(kmax, bits, offset, fine):
    """The device generator (libasr_synth.so) and the CPU route (torch
    integer ops) give bit-identical tensors, with and without the offset and
    the fine second draw; the length is not a multiple of the launch grid."""
    n = (1 << 20) + 77
    a = synth.grid_values(20260314, 77, (n,), kmax, bits, device="cuda", offset=offset,
                          fine=fine).cpu()
    b = synth.grid_values(20260314, 77, (n,), kmax, bits, device="cpu", offset=offset, fine=fine)
    assert torch.equal(a, b)


def _teacher_forced(ctx, P, shape, clips, ids, sample, tol, steps_cap=None):
    """Prefill `clips` (already popped as `ids`), decode every clip for its
    steps; the oracle follows the clips in `sample`.  Returns (worst rel err,
    near-ties)."""
    out = ctx.step(prefill_ids=ids)
    slots = list(out["slot_of"])
    steps = [OW.steps_for(len(p)) for p in clips]
    if steps_cap:
        steps = [min(s, steps_cap) for s in steps]
    toks = synth.token_ids(len(clips) * 7919, (len(clips), max(steps)), shape.vocab)
    st, ckv = {}, {}
    for b in sample:
        E = OW.encode(OM.log_mel(clips[b], shape.n_mels), P, shape.n_enc, shape.n_head)
        ckv[b] = OW.cross_kv(E, P, shape.n_dec)
        st[b] = OW.DecoderState(shape.n_dec, shape.d_model)
    worst, near = 0.0, 0
    for t in range(max(steps)):
        active = [b for b in range(len(clips)) if t < steps[b]]
        res = ctx.step(slots=[slots[b] for b in active], tokens=[int(toks[b, t]) for b in active],
                       want_logits=True)
        rows = [j for j, b in enumerate(active) if b in st]
        if not rows:
            continue
        ref = np.stack([OW.decoder_step(int(toks[active[j], t]), st[active[j]], ckv[active[j]], P,
                                        shape.n_dec, shape.n_head) for j in rows])
        got = res["logits"][rows]
        e = rel_err(got, ref)
        worst = max(worst, e)
        assert e <= tol, f"step {t}: {e:.3e}"
        near += check_argmax(res["argmax"][rows], got, ref, tol)
    for s in slots:
        ctx.release_slot(int(s))
    return worst, near


def test_tiny_fp32_workload():
    """Whisper-tiny shape, fp32: one 4-s clip, 16 teacher-forced steps."""
    wl = synth.WORKLOADS["tiny-fp32"]
    shape = synth.SHAPES[wl.shape]
    ctx, P = _context(shape, wl.seed, max_slots=1, max_prefill=1, max_decode=1)
    pcm = synth.pcm_clip(wl.seed, 0, int(wl.extra["clip_s"] * 16000))
    ctx.submit(0, pcm)
    ids = ctx.pop_batch(0, 1)
    worst, near = _teacher_forced(ctx, P, shape, [pcm], ids, [0], TOL["f32"],
                                  steps_cap=wl.extra["steps"])
    print(f"tiny-fp32: worst rel err {worst:.3e} near-ties {near}")


def test_base_bf16_workload():
    """Whisper-base shape, bf16: 8 lognormal-duration clips, ragged decode;
    the oracle follows the shortest and the longest clip."""
    wl = synth.WORKLOADS["base-bf16"]
    shape = synth.SHAPES[wl.shape]
    ctx, P = _context(shape, wl.seed, max_slots=8, max_prefill=8, max_decode=8)
    ns = synth.n_samples_of(synth.durations_lognormal(wl.seed, wl.batch))
    clips = [synth.pcm_clip(wl.seed, i, int(n)) for i, n in enumerate(ns)]
    for i, pcm in enumerate(clips):
        ctx.submit(i, pcm, arrival_us=i)
    ids = ctx.pop_batch(10**6, 8)
    sample = [int(np.argmin(ns)), int(np.argmax(ns))]
    worst, near = _teacher_forced(ctx, P, shape, [clips[i] for i in ids], ids,
                                  [ids.index(s) for s in sample], TOL["bf16"])
    print(f"base-bf16: worst rel err {worst:.3e} near-ties {near}")


def test_small_bf16_hrrn_workload():
    """Whisper-small shape, bf16: 256 Poisson requests (20/s, durations U[1,30]
    s), static batches of 32 popped by HRRN at each batch boundary on a
    virtual clock (0.05 s per prefill batch + 0.08 s per decode step).  The
    pop sequence is bit-exact against the oracle queue; the oracle follows
    one clip of the first batch through all its steps and spot-checks the
    first decode step of every batch."""
    from paper_2603_11273_amd import asr
    wl = synth.WORKLOADS["small-bf16-hrrn"]
    shape = synth.SHAPES[wl.shape]
    n_req = wl.extra["n_requests"]
    ctx, P = _context(shape, wl.seed, max_slots=32, max_prefill=32, max_decode=32, max_queue=n_req)
    ctx.set_policy(asr.HRRN)
    ref_q = OQ.Queue(OQ.HRRN)
    ns = synth.n_samples_of(synth.durations_uniform(wl.seed, n_req))
    arr = synth.poisson_arrivals_us(wl.seed, n_req, wl.extra["rate"])
    clips = {}
    for i in range(n_req):
        clips[i] = synth.pcm_clip(wl.seed, i, int(ns[i]))
        ctx.submit(i, clips[i], arrival_us=int(arr[i]))
        ref_q.submit(i, int(ns[i]), 16000, int(arr[i]))
    now = int(arr[31])                       # first batch once 32 requests are in
    batch_no = 0
    served = 0
    while ctx.queue_len() > 0:
        ids = ctx.pop_batch(now, 32)
        assert ids == ref_q.pop_batch(now, 32), f"batch {batch_no}: pop order differs"
        if not ids:
            now = int(min(arr[i] for i in ref_q.reqs))
            continue
        bclips = [clips[i] for i in ids]
        served += len(ids)
        if batch_no == 0:
            worst, near = _teacher_forced(ctx, P, shape, bclips, ids, [0], TOL["bf16"])
            print(f"small-bf16 batch 0 (oracle-followed clip): worst {worst:.3e} near-ties {near}")
        else:
            out = ctx.step(prefill_ids=ids)
            slots = list(out["slot_of"])
            toks = synth.token_ids(batch_no, len(ids), shape.vocab)
            res = ctx.step(slots=slots, tokens=[int(t) for t in toks], want_logits=True)
            j = batch_no % len(ids)
            E = OW.encode(OM.log_mel(bclips[j], shape.n_mels), P, shape.n_enc, shape.n_head)
            st = OW.DecoderState(shape.n_dec, shape.d_model)
            ref = OW.decoder_step(int(toks[j]), st, OW.cross_kv(E, P, shape.n_dec), P, shape.n_dec,
                                  shape.n_head)
            assert rel_err(res["logits"][j], ref) <= TOL["bf16"]
            check_argmax(res["argmax"][j:j + 1], res["logits"][j:j + 1], ref[None], TOL["bf16"])
            for s in slots:
                ctx.release_slot(int(s))
        steps = max(OW.steps_for(len(c)) for c in bclips)
        now += 50_000 + 80_000 * steps
        batch_no += 1
    assert served == n_req and ref_q.reqs == {}


def test_large_v3_encoder_workload():
    """large-v3 encoder, 64 full 30-s clips in one prefill (the benchmark's
    batch); the oracle checks clips 0 and 63."""
    wl = synth.WORKLOADS["large-v3-encoder"]
    shape = synth.reduced_shape(synth.SHAPES[wl.shape], 32, 0)
    ctx, P = _context(shape, wl.seed, max_slots=0, max_prefill=64, max_decode=0)
    pcm = torch.from_numpy(np.stack([synth.pcm_clip(wl.seed, i, synth.N_SAMPLES_30S)
                                     for i in range(64)])).cuda()
    E = ctx.debug_encode([pcm[i] for i in range(64)], on_device=True)
    for i in (0, 63):
        ref = OW.encode(OM.log_mel(pcm[i].cpu().numpy(), shape.n_mels), P, shape.n_enc,
                        shape.n_head)
        e = rel_err(E[i], ref)
        print(f"large-v3 encoder clip {i}: rel err {e:.3e}")
        assert e <= TOL["bf16"]


def test_large_v3_decode_workload():
    """large-v3 decode step, 128 rows with self-KV lengths U[10, 400] and 1500
    cross positions each (the benchmark's launch configuration); the oracle
    checks rows 0, 1 and 127."""
    wl = synth.WORKLOADS["large-v3-decode"]
    shape = synth.reduced_shape(synth.SHAPES[wl.shape], 0, 32)
    D = 128
    ctx, P = _context(shape, wl.seed, max_slots=D, max_prefill=64, max_decode=D)
    lens = synth.kv_lengths(wl.seed, D, wl.extra["kv_lo"], wl.extra["kv_hi"])
    for s0 in range(0, D, 64):
        idx = list(range(s0, s0 + 64))
        E = torch.stack([synth.encoder_output(wl.seed, b, shape.d_model, device="cuda") for b in idx])
        ctx.debug_set_encoder_out(idx, [-1] * 64, [10] * 64, E, on_device=True)
    for b in range(D):
        kv = synth.self_kv_prefix(wl.seed, b, shape.n_dec, shape.n_head, device="cuda")
        ctx.debug_set_self_kv(b, kv, int(lens[b]), on_device=True)
    toks = synth.token_ids(wl.seed, D, shape.vocab)
    res = ctx.step(slots=list(range(D)), tokens=[int(t) for t in toks], want_logits=True)
    rows = [0, 1, 127]
    ref = []
    for b in rows:
        kv = synth.self_kv_prefix(wl.seed, b, shape.n_dec, shape.n_head).numpy().astype(np.float64)
        L, d = int(lens[b]), shape.d_model
        kp = [kv[l, 0, :, :L].transpose(1, 0, 2).reshape(L, d) for l in range(shape.n_dec)]
        vp = [kv[l, 1, :, :L].transpose(1, 0, 2).reshape(L, d) for l in range(shape.n_dec)]
        st = OW.DecoderState(shape.n_dec, d, kp, vp)
        ckv = OW.cross_kv(synth.encoder_output(wl.seed, b, d).numpy(), P, shape.n_dec)
        ref.append(OW.decoder_step(int(toks[b]), st, ckv, P, shape.n_dec, shape.n_head))
    ref = np.stack(ref)
    got = res["logits"][rows]
    e = rel_err(got, ref)
    near = check_argmax(res["argmax"][rows], got, ref, TOL["bf16"])
    print(f"large-v3 decode: rel err {e:.3e} near-ties {near}")
    assert e <= TOL["bf16"]
    # the whole batch's argmax equals the argmax of its own logits
    lg = res["logits"]
    assert np.array_equal(res["argmax"], np.array([int(np.flatnonzero(r == r.max())[0]) for r in lg]))
