"""Parity with weights that bfloat16 cannot hold.

The default generator's values are exact in bf16, so the cases elsewhere
never ask a load path to round.  Here the weights carry a finer second draw
(18 significant bits): the fp32 path must keep them exactly (a load that
rounded or truncated them to bf16 would miss the 1e-4 tolerance, which the
first test checks on the oracle side); the bf16 path must round them to
nearest even, which the oracle reproduces by receiving the rounded matrices;
and the bf16 conversion itself is checked bit for bit on exact ties and their
neighbours."""
import numpy as np
import pytest

from oracle import whisper as OW
from paper_2603_11273_amd import synth

from gpu_util import TOL, check_argmax, cpu_params, make_context, needs_gpu, oracle_encode, rel_err

pytestmark = [pytest.mark.gpu, needs_gpu]


def test_fp32_fine_weights_teacher_forced():
    """Whisper-tiny widths, fp32, 2+2 layers, vocabulary 4096: one 3-s clip,
    8 teacher-forced steps with fine weights, logits within 1e-4 of the
    oracle on the same float32 weights.  The same oracle run on the weights
    rounded to bf16 differs from it by more than 1e-4, so a load path that
    rounded them would fail."""
    shape = synth.reduced_shape(synth.SHAPES["tiny"], 2, 2, vocab=4096)
    seed = 20260370
    ctx = make_context(shape, seed, max_slots=1, max_prefill=1, max_decode=1, fine=True)
    P = cpu_params(shape, seed, fine=True)
    Pr = cpu_params(shape, seed, fine=True, bf16_rounded=True)
    pcm = synth.pcm_clip(seed, 0, 48000)
    ctx.submit(1, pcm)
    ctx.pop_batch(0, 1)
    slot = int(ctx.step(prefill_ids=[1])["slot_of"][0])
    E, Er = oracle_encode(pcm, P, shape), oracle_encode(pcm, Pr, shape)
    ckv, ckvr = OW.cross_kv(E, P, shape.n_dec), OW.cross_kv(Er, Pr, shape.n_dec)
    st, str_ = OW.DecoderState(shape.n_dec, shape.d_model), OW.DecoderState(shape.n_dec, shape.d_model)
    toks = synth.token_ids(seed, 8, shape.vocab)
    worst, sep = 0.0, 0.0
    for t in range(8):
        res = ctx.step(slots=[slot], tokens=[int(toks[t])], want_logits=True)
        ref = OW.decoder_step(int(toks[t]), st, ckv, P, shape.n_dec, shape.n_head)
        rr = OW.decoder_step(int(toks[t]), str_, ckvr, Pr, shape.n_dec, shape.n_head)
        e = rel_err(res["logits"][0], ref)
        worst = max(worst, e)
        sep = max(sep, rel_err(rr, ref))
        assert e <= TOL["f32"], f"step {t}: rel err {e:.3e}"
        check_argmax(res["argmax"], res["logits"], ref[None], TOL["f32"])
    print(f"fine fp32: worst rel err {worst:.3e}; bf16-rounded weights move the oracle by {sep:.3e}")
    assert sep > 10 * TOL["f32"]


def test_bf16_encoder_fine_weights():
    """Whisper-base widths, bf16, 2 encoder layers, two clips, fine weights:
    the library rounds every matrix to bf16 (nearest even) at load; the
    oracle, given the rounded matrices and the float32 vectors, matches
    within the bf16 tolerance."""
    shape = synth.reduced_shape(synth.SHAPES["base"], 2, 0)
    seed = 20260371
    ctx = make_context(shape, seed, max_slots=0, max_prefill=2, max_decode=0, fine=True)
    clips = [synth.pcm_clip(seed, i, n) for i, n in enumerate([80000, 480000])]
    got = ctx.debug_encode(clips)
    P = cpu_params(shape, seed, fine=True, bf16_rounded=True)
    for i, pcm in enumerate(clips):
        e = rel_err(got[i], oracle_encode(pcm, P, shape))
        print(f"fine bf16 encoder clip {i}: rel err {e:.3e}")
        assert e <= TOL["bf16"]


def _rne_bf16(x):
    """float32 -> bfloat16 -> float32 with round to nearest, ties to even,
    on the bit pattern (finite inputs)."""
    u = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF
    return (r << 16).astype(np.uint32).view(np.float32)


def test_bf16_conversion_rounds_to_nearest_even():
    """The float32 -> bf16 conversion of the load and cache paths (the one
    asr_load_weights uses) on exact ties with an even and an odd kept bit,
    values one unit above and below a tie, negative values and exact bf16
    values, through a slot's self cache (written with asr_debug_set_self_kv,
    read back exactly with asr_debug_get_kv); compared bit for bit with a
    round-to-nearest-even written on the bit pattern."""
    shape = synth.reduced_shape(synth.SHAPES["tiny"], 0, 1, vocab=256, dtype="bf16")
    seed = 20260372
    ctx = make_context(shape, seed, max_slots=1, max_prefill=1, max_decode=1)
    ctx.debug_set_encoder_out([0], [-1], [1], synth.encoder_output(seed, 0, shape.d_model).numpy()[None])
    n = shape.n_dec * 2 * shape.n_head * 448 * 64
    rng = np.random.default_rng(seed)
    # kept halves: sign random, exponent in [2^-20, 2^20], mantissa random
    hi = (rng.integers(0, 2, n, dtype=np.uint32) << 15) | \
        (rng.integers(127 - 20, 127 + 20, n, dtype=np.uint32) << 7) | rng.integers(0, 128, n, dtype=np.uint32)
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    lo = lows[rng.integers(0, len(lows), n)]
    lo[: n // 4] = rng.integers(0, 1 << 16, n // 4, dtype=np.uint32)     # and arbitrary ones
    x = ((hi << 16) | lo).view(np.float32)
    ties_even = np.sum((lo == 0x8000) & ((hi & 1) == 0))
    ties_odd = np.sum((lo == 0x8000) & ((hi & 1) == 1))
    assert ties_even > 1000 and ties_odd > 1000
    src = x.reshape(shape.n_dec, 2, shape.n_head, 448, 64)
    ctx.debug_set_self_kv(0, src, 0)
    got = ctx.debug_get_kv(0, 0).reshape(-1)
    ref = _rne_bf16(x)
    bad = np.flatnonzero(got.view(np.uint32) != ref.view(np.uint32))
    assert bad.size == 0, f"{bad.size} mismatches, first {x[bad[0]]!r} -> {got[bad[0]]!r} (want {ref[bad[0]]!r})"
    # the reference itself: ties go to the even neighbour, everything else to the nearest
    t = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20,
                  1.0 + 2.0 ** -8 - 2.0 ** -20], np.float32)
    assert _rne_bf16(t).tolist() == [1.0, 1.0 + 4 * 2.0 ** -8, 1.0 + 2.0 ** -7, 1.0]
