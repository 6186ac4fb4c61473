"""Pins for the model oracle: library routines, invariants, brute force and an
independent second implementation written here with torch CPU ops."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mel as OM
from oracle import whisper as W
from paper_2603_11273_amd import synth



@pytest.fixture(autouse=True)
def _float64_default():
    """These pins compare against torch in float64; the default dtype is
    restored afterwards so that other test modules keep torch's float32."""
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)


def test_gelu_layernorm_match_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 48)) * 3
    assert np.allclose(W.gelu(x), F.gelu(torch.tensor(x)).numpy(), rtol=1e-13, atol=1e-15)
    g, b = rng.standard_normal(48), rng.standard_normal(48)
    ref = F.layer_norm(torch.tensor(x), (48,), torch.tensor(g), torch.tensor(b), eps=1e-5)
    assert np.allclose(W.layer_norm(x, g, b), ref.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("stride", [1, 2])
def test_conv1d_matches_torch(stride):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((20, 6))
    w = rng.standard_normal((5, 6, 3))
    b = rng.standard_normal(5)
    ref = F.conv1d(torch.tensor(x.T)[None], torch.tensor(w), torch.tensor(b), stride=stride,
                   padding=1)[0].T.numpy()
    assert np.allclose(W.conv1d(x, w, b, stride), ref, rtol=1e-12, atol=1e-12)


def test_sinusoids():
    s = W.sinusoids(1500, 384)
    assert np.array_equal(s[0], np.r_[np.zeros(192), np.ones(192)])
    inc = math.log(10000.0) / 191
    assert s[7, 3] == pytest.approx(math.sin(7 * math.exp(-3 * inc)), abs=1e-15)
    assert s[1499, 192 + 191] == pytest.approx(math.cos(1499 * 1e-4), abs=1e-12)


def _naive_attention(q, k, v, n_head, causal=False):
    """Brute force with Python loops."""
    Tq, d = q.shape
    dh = d // n_head
    out = np.zeros((Tq, d))
    for h in range(n_head):
        for i in range(Tq):
            keys = range(i + 1) if causal else range(k.shape[0])
            s = [sum(q[i, h * dh + c] * k[j, h * dh + c] for c in range(dh)) / math.sqrt(dh)
                 for j in keys]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for c in range(dh):
                out[i, h * dh + c] = sum(e[jj] * v[j, h * dh + c] for jj, j in enumerate(keys)) / z
    return out


def test_attention_bruteforce_and_sdpa():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((6, 8)) for _ in range(3))
    assert np.allclose(W.attention(q, k, v, 2), _naive_attention(q, k, v, 2), rtol=1e-12)
    mask = np.tril(np.ones((6, 6), bool))
    assert np.allclose(W.attention(q, k, v, 2, mask), _naive_attention(q, k, v, 2, True), rtol=1e-12)
    qt = torch.tensor(q).view(6, 2, 4).transpose(0, 1)
    kt = torch.tensor(k).view(6, 2, 4).transpose(0, 1)
    vt = torch.tensor(v).view(6, 2, 4).transpose(0, 1)
    ref = F.scaled_dot_product_attention(qt, kt, vt).transpose(0, 1).reshape(6, 8).numpy()
    assert np.allclose(W.attention(q, k, v, 2), ref, rtol=1e-12)


def test_softmax_rows_and_permutation_invariance():
    rng = np.random.default_rng(4)
    s = rng.standard_normal((9, 1500)) * 10
    assert np.allclose(W.softmax(s).sum(axis=1), 1.0, atol=1e-12)
    q, k, v = rng.standard_normal((5, 128)), rng.standard_normal((30, 128)), rng.standard_normal((30, 128))
    p = rng.permutation(30)
    assert np.allclose(W.attention(q, k, v, 2), W.attention(q, k[p], v[p], 2), rtol=1e-12)


def test_uniform_cross_attention():
    """All encoder rows equal -> uniform weights -> output is that value row."""
    rng = np.random.default_rng(5)
    q = rng.standard_normal((3, 128))
    krow, vrow = rng.standard_normal(128), rng.standard_normal(128)
    out = W.attention(q, np.tile(krow, (1500, 1)), np.tile(vrow, (1500, 1)), 2)
    assert np.allclose(out, np.tile(vrow, (3, 1)), rtol=1e-12)


def _small_model(n_enc=2, n_dec=2, vocab=512, seed=9):
    shape = synth.reduced_shape(synth.SHAPES["tiny"], n_enc, n_dec, vocab=vocab)
    return shape, synth.model_params(shape, seed)


def test_causal_invariance_and_incremental_decode():
    shape, P = _small_model()
    E = synth.encoder_output(9, 0, shape.d_model).numpy().astype(np.float64)
    ckv = W.cross_kv(E, P, shape.n_dec)
    toks = synth.token_ids(9, 10, shape.vocab)
    full = W.decoder_forward_full(toks, ckv, P, shape.n_dec, shape.n_head)
    toks2 = toks.copy()
    toks2[6:] = (toks2[6:] + 17) % shape.vocab
    full2 = W.decoder_forward_full(toks2, ckv, P, shape.n_dec, shape.n_head)
    assert np.array_equal(full[:6], full2[:6])                 # positions <= 5 untouched
    assert not np.allclose(full[6:], full2[6:])
    st = W.DecoderState(shape.n_dec, shape.d_model)
    inc = np.stack([W.decoder_step(int(t), st, ckv, P, shape.n_dec, shape.n_head) for t in toks])
    assert st.length == 10
    assert np.allclose(inc, full, rtol=1e-10, atol=1e-10 * np.abs(full).max())


def test_argmax_first():
    assert W.argmax_first([1.0, 3.0, 3.0, 2.0]) == 1
    assert W.argmax_first(np.r_[np.zeros(5), 1.0]) == 5
    with pytest.raises(ValueError):
        W.argmax_first([1.0, float("nan")])


def test_steps_for():
    assert W.steps_for(16000) == 3                    # 2.7 -> 3
    assert W.steps_for(480000) == 81                  # 81.0
    assert W.steps_for(1) == 1
    assert W.steps_for(16000 * 5) == 14               # 13.5 rounds half up
    assert W.steps_for(10**9) == 448


# ----------------------------------------------------------------------------
# Independent second implementation of the whole forward (torch CPU, float64)
# ----------------------------------------------------------------------------
def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def _torch_mha(x_q, x_kv, wq, bq, wk, wv, bv, wo, bo, n_head, causal=False, k_cache=None):
    q = x_q @ wq.T + bq
    k = x_kv @ wk.T
    v = x_kv @ wv.T + bv
    Tq, d = q.shape
    dh = d // n_head
    qh = q.view(Tq, n_head, dh).transpose(0, 1)
    kh = k.view(-1, n_head, dh).transpose(0, 1)
    vh = v.view(-1, n_head, dh).transpose(0, 1)
    o = F.scaled_dot_product_attention(qh, kh, vh, is_causal=causal)
    return o.transpose(0, 1).reshape(Tq, d) @ wo.T + bo


def _torch_forward(pcm, toks, P, shape):
    T = {k: _t(v.numpy() if hasattr(v, "numpy") else v) for k, v in P.items()}
    d = shape.d_model
    mel = _t(OM.log_mel(pcm, shape.n_mels))
    x = F.gelu(F.conv1d(mel.T[None], T["conv1.w"], T["conv1.b"], padding=1))
    x = F.gelu(F.conv1d(x, T["conv2.w"], T["conv2.b"], stride=2, padding=1))[0].T
    half = d // 2
    inv = torch.exp(-math.log(10000.0) / (half - 1) * torch.arange(half, dtype=torch.float64))
    ang = torch.arange(1500, dtype=torch.float64)[:, None] * inv[None]
    x = x + torch.cat([ang.sin(), ang.cos()], 1)
    ln = lambda z, p: F.layer_norm(z, (d,), T[p + ".g"], T[p + ".b"], eps=1e-5)
    for l in range(shape.n_enc):
        p = f"enc.{l}."
        a = ln(x, p + "attn_ln")
        x = x + _torch_mha(a, a, T[p + "q.w"], T[p + "q.b"], T[p + "k.w"], T[p + "v.w"],
                           T[p + "v.b"], T[p + "o.w"], T[p + "o.b"], shape.n_head)
        m = ln(x, p + "mlp_ln")
        x = x + F.gelu(m @ T[p + "fc1.w"].T + T[p + "fc1.b"]) @ T[p + "fc2.w"].T + T[p + "fc2.b"]
    E = ln(x, "ln_post")
    n = len(toks)
    h = T["tok_emb"][torch.as_tensor(toks, dtype=torch.long)] + T["pos_emb"][:n]
    for l in range(shape.n_dec):
        p = f"dec.{l}."
        a = ln(h, p + "attn_ln")
        h = h + _torch_mha(a, a, T[p + "q.w"], T[p + "q.b"], T[p + "k.w"], T[p + "v.w"],
                           T[p + "v.b"], T[p + "o.w"], T[p + "o.b"], shape.n_head, causal=True)
        c = ln(h, p + "xattn_ln")
        h = h + _torch_mha(c, E, T[p + "xq.w"], T[p + "xq.b"], T[p + "xk.w"], T[p + "xv.w"],
                           T[p + "xv.b"], T[p + "xo.w"], T[p + "xo.b"], shape.n_head)
        m = ln(h, p + "mlp_ln")
        h = h + F.gelu(m @ T[p + "fc1.w"].T + T[p + "fc1.b"]) @ T[p + "fc2.w"].T + T[p + "fc2.b"]
    h = ln(h, "ln")
    return E.numpy(), (h @ T["tok_emb"].T).numpy()


def test_whole_forward_vs_torch_second_implementation():
    shape, P = _small_model(n_enc=2, n_dec=2, vocab=700, seed=11)
    pcm = synth.pcm_clip(11, 0, 64000)
    toks = synth.token_ids(11, 6, shape.vocab)
    mel = OM.log_mel(pcm, shape.n_mels)
    E = W.encode(mel, P, shape.n_enc, shape.n_head)
    ckv = W.cross_kv(E, P, shape.n_dec)
    st = W.DecoderState(shape.n_dec, shape.d_model)
    logits = np.stack([W.decoder_step(int(t), st, ckv, P, shape.n_dec, shape.n_head) for t in toks])
    E_ref, logits_ref = _torch_forward(pcm, toks, P, shape)
    assert np.abs(E - E_ref).max() <= 1e-9 * np.abs(E_ref).max()
    assert np.abs(logits - logits_ref).max() <= 1e-9 * np.abs(logits_ref).max()
