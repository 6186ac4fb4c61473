"""The seeded generators: the tensor hash equals its scalar definition, and
generated values are exact in bfloat16."""
import numpy as np
import pytest
import torch

from paper_2603_11273_amd import synth


def test_lowbias32_known_value_and_tensor_route():
    # the mixer is a bijection on 32 bits; 0 maps to 0
    assert synth.lowbias32_py(0) == 0
    idx = list(range(0, 5000, 7)) + [2**32 - 1, 2**31, 123456789]
    h = synth.hash_tensor(20260311, 5, 0, 5000)
    for i in idx[:-3]:
        assert int(h[i]) == synth.hash_py(20260311, 5, i)
    big = synth.hash_tensor(3, 1, 2**32 - 3, 3)
    assert [int(x) for x in big] == [synth.hash_py(3, 1, i) for i in range(2**32 - 3, 2**32)]


def test_grid_values_exact_in_bf16():
    v = synth.grid_values(1, 2, (4096,), 141, 12)
    assert torch.equal(v, v.to(torch.bfloat16).to(torch.float32))
    assert abs(float(v.std()) - 0.02) < 0.002
    g = synth.grid_values(1, 3, (4096,), 141, 12, offset=1.0)
    assert torch.equal(g - 1.0, (g - 1.0).to(torch.bfloat16).to(torch.float32))
    e = synth.encoder_output(5, 0, 64)
    assert torch.equal(e, e.to(torch.bfloat16).to(torch.float32))
    assert abs(float(e.std()) - 1.0) < 0.05


def test_chunking_does_not_change_values():
    a = synth.grid_values(7, 1, (1000,), 100, 8, chunk=1 << 24)
    b = synth.grid_values(7, 1, (1000,), 100, 8, chunk=97)
    assert torch.equal(a, b)


def test_workload_distributions():
    d = synth.durations_lognormal(1, 20000)
    assert 1.0 <= d.min() and d.max() <= 30.0
    assert 6.5 < d.mean() < 7.8 and np.median(d) < d.mean()       # right-skewed
    u = synth.durations_uniform(1, 20000)
    assert abs(u.mean() - 15.5) < 0.3
    a = synth.poisson_arrivals_us(1, 5000, 20.0)
    assert np.all(np.diff(a) >= 0) and abs(a[-1] / 1e6 / 5000 - 0.05) < 0.005


@pytest.mark.parametrize("case", synth.ATTENTION_CASES)
def test_attention_operands_exact_and_structured(case):
    """The attention operands are bf16-exact, and each case puts the scores
    (exp2 domain, one head) where its docstring says."""
    q, k, v = synth.attention_operands(5, 1, 128, case)
    for a in (q, k, v):
        t = torch.from_numpy(a)
        assert torch.equal(t.to(torch.bfloat16).to(torch.float32), t)
    s = q[0][:, :64].astype(np.float64) @ k[0][:, :64].T.astype(np.float64)
    first, late = s[:, :64].max(axis=1), s[:, 896:960].max(axis=1)
    if case == "small":
        assert np.abs(s).max() < 8
    elif case == "first_tile_large":
        assert first.min() > 64 and s[:, 64:].max() < 8
    elif case == "late_large":
        assert np.abs(first).max() < 8 and late.min() > 64
    elif case == "late_huge":
        # past 128: exp2 of these scores against a reference of 0 overflows fp32
        assert np.abs(first).max() < 8 and late.min() > 128
    else:
        assert s.max() < -64


def test_fine_values_exact_in_fp32_not_in_bf16():
    """The fine variant: the base draw plus j * 2^-22 (|j| <= 255) is a
    multiple of 2^-22 (exact in float32), moves almost every value off the
    bfloat16 grid, leaves the spread at ~0.02, and keeps the base draw (the
    fine term is at most 255 * 2^-22 < 2^-13 away from it)."""
    base = synth.grid_values(1, 2, (8192,), 141, 12)
    v = synth.grid_values(1, 2, (8192,), 141, 12, fine=True)
    scaled = v.double() * 2.0 ** 22
    assert torch.equal(scaled, scaled.round())
    off_grid = (v.to(torch.bfloat16).to(torch.float32) != v).float().mean()
    assert off_grid > 0.95
    assert abs(float(v.std()) - 0.02) < 0.002
    d = (v - base).double() * 2.0 ** 22
    assert float(d.abs().max()) <= 255 and float(d.abs().max()) > 200
    g = synth.grid_values(1, 3, (4096,), 141, 12, offset=1.0, fine=True)
    assert torch.equal((g.double() - 1.0) * 2.0 ** 22, ((g.double() - 1.0) * 2.0 ** 22).round())


def test_bf16_rounded_params_round_matrices_only():
    shape = synth.reduced_shape(synth.SHAPES["tiny"], 1, 1, vocab=64)
    p = synth.model_params(shape, 3, fine=True)
    r = synth.bf16_rounded_params(p)
    for name, t in p.items():
        if name.endswith(".w") or name == "tok_emb":
            assert torch.equal(r[name], t.to(torch.bfloat16).to(torch.float32)), name
            assert not torch.equal(r[name], t), name
        else:
            assert r[name] is t, name
