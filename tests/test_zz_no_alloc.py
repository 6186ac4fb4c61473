"""The allocation-free log-mel entry point (asr_logmel_noalloc) against the
existing one (asr_debug_logmel), through the C ABI: the same kernels on the
same clips, so the features must agree bit for bit; calls in a row, the
second with fewer and shorter clips (the shared scratch keeps the first
call's per-group maxima, which the second must overwrite before it reads
them), the third into an output one float past a 16-byte boundary (the
normalisation's unvectorised path)."""
import numpy as np
import pytest
import torch

from paper_2603_11273_amd import synth

from gpu_util import needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


def _ctx(n_mels, n):
    from paper_2603_11273_amd import asr
    shape = synth.ModelShape("mel", n_mels, 384, 1, 0, 6, 1536, 0, "f32")
    ctx = asr.Context(asr.model_cfg(shape, max_slots=0, max_prefill=n, max_decode=0), device=0)
    ctx.bind()
    return ctx


@pytest.mark.parametrize("n_mels", [80, 128])
def test_noalloc_logmel_matches_bound_entry_point(n_mels):
    from paper_2603_11273_amd import asr
    seed = 20260380 + n_mels
    first = [480000, 64000, 1, 16000, 123457, 480000]
    second = [32000, 7]
    ctx = _ctx(n_mels, len(first))
    for lengths, offset in ((first, 0), (second, 0), (second, 1)):
        clips = [synth.pcm_clip(seed, i, n) for i, n in enumerate(lengths)]
        if len(lengths) > 3:
            clips[3] = np.zeros(lengths[3], np.float32)        # silence: the constant floor
        dev = [torch.from_numpy(c).cuda() for c in clips]
        size = len(clips) * 3000 * n_mels
        buf = torch.full((size + offset,), float("nan"), dtype=torch.float32, device="cuda")
        out = buf[offset:].view(len(clips), 3000, n_mels)
        asr.logmel_noalloc(dev, n_mels, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ref = ctx.debug_logmel(clips)
        assert not np.isnan(got).any()
        assert np.array_equal(got, ref), f"max diff {np.abs(got - ref).max():.3e}"
        print(f"n_mels {n_mels}, {len(clips)} clips, output offset {offset}: "
              "bit-identical to asr_debug_logmel")


def test_noalloc_logmel_rejects_bad_sizes():
    from paper_2603_11273_amd import asr
    f32 = dict(dtype=torch.float32, device="cuda")
    clips = [torch.zeros(16000, **f32) for _ in range(65)]
    out = torch.empty((65, 3000, 80), **f32)
    with pytest.raises(asr.AsrError) as e:
        asr.logmel_noalloc(clips, 80, out)
    assert e.value.status == asr.ASR_EINVAL
    with pytest.raises(asr.AsrError) as e:
        asr.logmel_noalloc(clips[:2], 64, torch.empty((2, 3000, 64), **f32))
    assert e.value.status == asr.ASR_EINVAL
    big = [torch.zeros(480001, **f32)]
    with pytest.raises(asr.AsrError) as e:
        asr.logmel_noalloc(big, 80, torch.empty((1, 3000, 80), **f32))
    assert e.value.status == asr.ASR_EINVAL
