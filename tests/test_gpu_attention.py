"""Encoder attention kernel alone, through asr_debug_attention, against the
oracle's multi-head attention (Section 2's encoder self-attention over the
1500 positions of a segment).  The operands are bf16-exact, so both sides see
the same inputs; the cases include scores far from zero on the first key tile
and on a later one, and uniformly very negative scores, which take the
kernel's softmax-reference branches that random model weights never reach."""
import math

import numpy as np
import pytest

from oracle import whisper as OW
from paper_2603_11273_amd import synth

from gpu_util import make_context, needs_gpu, rel_err

pytestmark = [pytest.mark.gpu, needs_gpu]

# bf16 path: probabilities go through bf16 (relative 2^-9) before the PV
# product, fp32 everywhere else; fp32 path: fp32 throughout.
ATT_TOL = {"bf16": 1e-2, "f32": 1e-4}


@pytest.mark.parametrize("name", ["base", "tiny"])
@pytest.mark.parametrize("case", synth.ATTENTION_CASES)
def test_attention_matches_oracle(name, case):
    shape = synth.reduced_shape(synth.SHAPES[name], 1, 0)
    seed = 20260350
    n = 2
    ctx = make_context(shape, seed, max_slots=0, max_prefill=n, max_decode=0)
    q, k, v = synth.attention_operands(seed, n, shape.d_model, case)
    got = ctx.debug_attention(q, k, v)
    assert np.all(np.isfinite(got))
    # the kernel reads q in the exp2 domain: softmax_2(q k^T) equals the
    # oracle's softmax(q' k^T / sqrt(64)) for q' = q * 8 / log2(e)
    qn = q.astype(np.float64) * (8.0 / math.log2(math.e))
    worst = 0.0
    for b in range(n):
        ref = OW.attention(qn[b], k[b].astype(np.float64), v[b].astype(np.float64), shape.n_head)
        e = rel_err(got[b], ref)
        worst = max(worst, e)
        assert e <= ATT_TOL[shape.dtype], f"clip {b}: rel err {e:.3e}"
    print(f"attention {name} {case}: worst rel err {worst:.3e}")


@pytest.mark.parametrize("n", [1, 3])
def test_attention_block_count_not_a_multiple_of_eight(n):
    """The kernel deals its (query block, head, clip) work items to the 8
    XCDs in contiguous ranges; with 6 heads and 1 or 3 clips the block count
    (36, 108) leaves a remainder, so the first XCDs take one item more.
    Every item must still be computed exactly once."""
    shape = synth.reduced_shape(synth.SHAPES["tiny"], 1, 0, dtype="bf16")
    assert shape.n_head == 6
    seed = 20260351 + n
    ctx = make_context(shape, seed, max_slots=0, max_prefill=n, max_decode=0)
    q, k, v = synth.attention_operands(seed, n, shape.d_model, "small")
    got = ctx.debug_attention(q, k, v)
    assert np.all(np.isfinite(got))
    qn = q.astype(np.float64) * (8.0 / math.log2(math.e))
    for b in range(n):
        ref = OW.attention(qn[b], k[b].astype(np.float64), v[b].astype(np.float64), shape.n_head)
        e = rel_err(got[b], ref)
        assert e <= ATT_TOL["bf16"], f"clip {b}: rel err {e:.3e}"
