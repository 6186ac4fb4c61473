"""Decode steps replayed from HIP graphs against the same steps launched
kernel by kernel: two contexts with the same weights, encoder outputs and
caches run the same sequence of steps (two row counts, with and without
logits, so shapes are seen a first time, captured at their second step and
replayed afterwards, with other shapes' direct steps and host
synchronisations in between); every step's logits and argmax must be
bit-identical."""
import numpy as np
import pytest

from paper_2603_11273_amd import synth

from gpu_util import make_context, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


@pytest.mark.parametrize("name,dtype", [("base", "bf16"), ("tiny", "f32")])
def test_graph_replay_matches_direct_launches(name, dtype):
    shape = synth.reduced_shape(synth.SHAPES[name], 0, 2, vocab=4096, dtype=dtype)
    seed = 20260390
    B = 6
    ctxs = []
    for graphs in (False, True):
        ctx = make_context(shape, seed, max_slots=B, max_prefill=B, max_decode=B)
        ctx.set_decode_graphs(graphs)
        E = np.stack([synth.encoder_output(seed, b, shape.d_model).numpy() for b in range(B)])
        ctx.debug_set_encoder_out(list(range(B)), [-1] * B, [40] * B, E)
        for b in range(B):
            kv = synth.self_kv_prefix(seed, b, shape.n_dec, shape.n_head).numpy()
            ctx.debug_set_self_kv(b, kv, 3 + 5 * b)
        ctxs.append(ctx)
    # (rows, logits) per step: the all-rows shape is direct at step 0,
    # captured at step 1 and replayed from step 2; the subset shape's
    # first, second and later steps fall in between
    plan = [(B, True), (B, True), (B, True), (3, True), (B, True), (3, True), (B, False),
            (3, True), (B, False), (B, True), (3, True), (B, False)]
    toks = synth.token_ids(seed, (len(plan), B), shape.vocab)
    for k, (rows, logits) in enumerate(plan):
        outs = [c.step(slots=list(range(rows)), tokens=[int(t) for t in toks[k, :rows]],
                       want_logits=logits) for c in ctxs]
        assert list(outs[0]["argmax"]) == list(outs[1]["argmax"]), f"step {k}"
        if logits:
            assert np.array_equal(outs[0]["logits"], outs[1]["logits"]), f"step {k}"
    for b in range(B):
        assert ctxs[0].slot_info(b)["position"] == ctxs[1].slot_info(b)["position"]
    for which in (0,):
        for b in (0, B - 1):
            assert np.array_equal(ctxs[0].debug_get_kv(b, which), ctxs[1].debug_get_kv(b, which))
