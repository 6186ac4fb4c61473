"""Shared helpers of the GPU parity tests (not collected: no test_ prefix).

The HIP path is driven only through the C ABI (paper_2603_11273_amd.asr); the
expected values come only from the oracle, on the same seeded inputs."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import mel as OM
from oracle import whisper as OW
from paper_2603_11273_amd import synth

try:
    import torch
    HAVE_GPU = torch.cuda.is_available()
except Exception:  # pragma: no cover
    HAVE_GPU = False

needs_gpu = pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")

# Relative tolerances on max|g - o| / max|o| per tensor: the fp32 path and the
# bf16 path (bf16 storage of weights and activations, fp32 accumulation).
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_err(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return float(np.abs(g - o).max() / max(np.abs(o).max(), 1e-30))


def make_context(shape, seed, max_slots=4, max_prefill=2, max_decode=4, fine=False):
    from paper_2603_11273_amd import asr
    ctx = asr.Context(asr.model_cfg(shape, max_slots=max_slots, max_prefill=max_prefill,
                                    max_decode=max_decode), device=0)
    ctx.bind()
    params = synth.model_params(shape, seed, device="cuda", fine=fine)
    tensors = list(params.values())
    assert len(tensors) == ctx.n_params()
    for i, t in enumerate(tensors):
        assert t.numel() == ctx.param_numel(i)
    ctx.load_weights(tensors, on_device=True)
    torch.cuda.synchronize()
    del params, tensors
    return ctx


def cpu_params(shape, seed, fine=False, bf16_rounded=False):
    """The oracle's parameters: the same generator on the CPU; bf16_rounded
    gives them as a bf16 context holds them (matrices rounded to nearest
    even)."""
    p = synth.model_params(shape, seed, device="cpu", fine=fine)
    return synth.bf16_rounded_params(p) if bf16_rounded else p


def check_logits(g, o, tol, label=""):
    """Per-step logits within tol; argmax bit-exact where the oracle's top-2
    margin exceeds 2*tol*max|o|; the GPU argmax always equals the argmax of the
    GPU's own logits (checked by the caller).  Returns (rel_err, n_near_ties)."""
    e = rel_err(g, o)
    assert e <= tol, f"{label}: logits rel err {e:.3e} > {tol:.1e}"
    return e


def check_argmax(am_gpu, logits_gpu, logits_ref, tol):
    """Argmax checks of one step.  Always: the GPU argmax is the argmax of the
    GPU's own logits (lowest index on ties), bit-exact.  Against the oracle:
    if every logit of a row is within eps of the oracle's and the oracle's
    top-2 margin exceeds 2*eps, the two argmaxes must be equal (no rounding
    within eps can reorder them); eps is the row's observed max |g - o|.
    Rows with a smaller margin are near-ties: the GPU pick must then be a
    maximal oracle logit within 2*eps.  Returns the number of near-ties."""
    near = 0
    for b in range(len(am_gpu)):
        g = np.asarray(logits_gpu[b])
        assert am_gpu[b] == int(np.flatnonzero(g == g.max())[0]), "argmax != argmax of own logits"
        o = np.asarray(logits_ref[b], np.float64)
        eps = float(np.abs(g.astype(np.float64) - o).max())
        assert eps <= tol * np.abs(o).max()
        top = np.sort(o)[-2:]
        if top[1] - top[0] > 2 * eps:
            assert am_gpu[b] == OW.argmax_first(o), f"row {b}: argmax {am_gpu[b]} != oracle"
        else:
            near += 1
            assert o[am_gpu[b]] >= o.max() - 2 * eps
    return near


def oracle_encode(pcm, P, shape):
    mel = OM.log_mel(pcm, shape.n_mels)
    return OW.encode(mel, P, shape.n_enc, shape.n_head)
