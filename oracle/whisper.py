"""Oracle for the Whisper-shaped encoder-decoder step (test infrastructure only).

The paper's workload is Whisper inference (Section 1, Section 4.1 setup:
whisper-large-v3, at most 448 output tokens); Section 3.1 describes its two
phases: the encoder runs once per fixed 30-s segment, then decoding emits one
token per step, which is where the time goes.  This module writes that
architecture out plainly, in float64, with no blocking or fusion:

* stem: conv1d(n_mels -> d, k3, pad 1) + GELU, conv1d(d -> d, k3, stride 2,
  pad 1) + GELU, + fixed sinusoidal positions (1500 rows);
* encoder block: x += Attn(LN(x)); x += MLP(LN(x)); LN_post at the end;
* cross K/V per decoder layer from the encoder output (k has no bias);
* decoder step: h = tok_emb[id] + pos_emb[p]; causal self-attention over the
  cache (this step's k, v written at p); cross-attention over 1500 encoder
  positions; MLP; final LN; logits = h . tok_emb^T (tied, no bias); argmax
  with the lowest index on ties.

Conventions: linear weights are [out][in] (y = x W^T + b); conv weights are
[out][in][tap]; LayerNorm uses the biased variance and eps 1e-5; GELU is the
exact erf form; attention scores are scaled by 1/sqrt(64).
"""
from __future__ import annotations

import math

import numpy as np

try:                                   # erf for arrays
    from scipy.special import erf as _erf
except Exception:                      # pragma: no cover
    _erf = np.vectorize(math.erf)

N_CTX = 1500
EPS = 1e-5


def f64(a) -> np.ndarray:
    """Parameters may arrive as torch tensors or numpy arrays; use float64."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.asarray(a, dtype=np.float64)


def gelu(x):
    return 0.5 * x * (1.0 + _erf(x / math.sqrt(2.0)))


def layer_norm(x, g, b):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + EPS) * g + b


def linear(x, w, b=None):
    y = x @ w.T
    return y if b is None else y + b


def conv1d(x, w, b, stride):
    """x [T][C_in], w [C_out][C_in][3], padding 1 -> [T_out][C_out]."""
    T = x.shape[0]
    xp = np.concatenate([np.zeros((1, x.shape[1])), x, np.zeros((1, x.shape[1]))], axis=0)
    t_out = (T + 2 - 3) // stride + 1
    y = np.zeros((t_out, w.shape[0]))
    for j in range(3):
        rows = xp[j + stride * np.arange(t_out)]              # input row t*stride + j - 1
        y += rows @ w[:, :, j].T
    return y + b


def sinusoids(length: int, channels: int) -> np.ndarray:
    half = channels // 2
    inc = math.log(10000.0) / (half - 1)
    inv = np.exp(-inc * np.arange(half))
    t = np.arange(length)[:, None] * inv[None, :]
    return np.concatenate([np.sin(t), np.cos(t)], axis=1)


def softmax(s, axis=-1):
    s = s - s.max(axis=axis, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=axis, keepdims=True)


def attention(q, k, v, n_head, mask=None):
    """Multi-head scaled dot-product attention; q [Tq][d], k/v [Tk][d]."""
    d = q.shape[1]
    dh = d // n_head
    out = np.zeros((q.shape[0], d))
    for h in range(n_head):
        sl = slice(h * dh, (h + 1) * dh)
        s = q[:, sl] @ k[:, sl].T / math.sqrt(dh)
        if mask is not None:
            s = np.where(mask, s, -np.inf)
        out[:, sl] = softmax(s) @ v[:, sl]
    return out


# ----------------------------------------------------------------------------
# Encoder
# ----------------------------------------------------------------------------
def stem(mel, P):
    """mel [3000][n_mels] -> x [1500][d]."""
    h = gelu(conv1d(mel, f64(P["conv1.w"]), f64(P["conv1.b"]), 1))
    h = gelu(conv1d(h, f64(P["conv2.w"]), f64(P["conv2.b"]), 2))
    return h + sinusoids(h.shape[0], h.shape[1])


def encoder_block(x, P, l, n_head):
    p = f"enc.{l}."
    g = lambda n: f64(P[p + n])
    a = layer_norm(x, g("attn_ln.g"), g("attn_ln.b"))
    q = linear(a, g("q.w"), g("q.b"))
    k = linear(a, g("k.w"))
    v = linear(a, g("v.w"), g("v.b"))
    x = x + linear(attention(q, k, v, n_head), g("o.w"), g("o.b"))
    m = layer_norm(x, g("mlp_ln.g"), g("mlp_ln.b"))
    x = x + linear(gelu(linear(m, g("fc1.w"), g("fc1.b"))), g("fc2.w"), g("fc2.b"))
    return x


def encode(mel, P, n_enc, n_head):
    """Normalised log-mel [3000][n_mels] -> encoder output E [1500][d]."""
    x = stem(mel, P)
    for l in range(n_enc):
        x = encoder_block(x, P, l, n_head)
    return layer_norm(x, f64(P["ln_post.g"]), f64(P["ln_post.b"]))


# ----------------------------------------------------------------------------
# Decoder
# ----------------------------------------------------------------------------
def cross_kv(E, P, n_dec):
    """Per decoder layer (K_c, V_c) = (E Wk^T, E Wv^T + bv), each [1500][d]."""
    E = f64(E)
    out = []
    for l in range(n_dec):
        p = f"dec.{l}."
        out.append((linear(E, f64(P[p + "xk.w"])),
                    linear(E, f64(P[p + "xv.w"]), f64(P[p + "xv.b"]))))
    return out


class DecoderState:
    """Per-sequence self-attention cache: keys/values [n_dec][length][d]."""

    def __init__(self, n_dec, d, k_prefix=None, v_prefix=None):
        if k_prefix is None:
            self.k = [np.zeros((0, d)) for _ in range(n_dec)]
            self.v = [np.zeros((0, d)) for _ in range(n_dec)]
        else:
            self.k = [f64(k_prefix[l]) for l in range(n_dec)]
            self.v = [f64(v_prefix[l]) for l in range(n_dec)]

    @property
    def length(self):
        return self.k[0].shape[0]


def decoder_step(token, state: DecoderState, ckv, P, n_dec, n_head):
    """One decoding step of one sequence at position state.length.

    Appends this step's self-attention key/value to `state` and returns the
    logits row [vocab]."""
    pos = state.length
    h = f64(P["tok_emb"])[token] + f64(P["pos_emb"])[pos]
    h = h[None, :]
    for l in range(n_dec):
        p = f"dec.{l}."
        g = lambda n: f64(P[p + n])
        a = layer_norm(h, g("attn_ln.g"), g("attn_ln.b"))
        q = linear(a, g("q.w"), g("q.b"))
        state.k[l] = np.concatenate([state.k[l], linear(a, g("k.w"))], axis=0)
        state.v[l] = np.concatenate([state.v[l], linear(a, g("v.w"), g("v.b"))], axis=0)
        h = h + linear(attention(q, state.k[l], state.v[l], n_head), g("o.w"), g("o.b"))
        c = layer_norm(h, g("xattn_ln.g"), g("xattn_ln.b"))
        qc = linear(c, g("xq.w"), g("xq.b"))
        kc, vc = ckv[l]
        h = h + linear(attention(qc, kc, vc, n_head), g("xo.w"), g("xo.b"))
        m = layer_norm(h, g("mlp_ln.g"), g("mlp_ln.b"))
        h = h + linear(gelu(linear(m, g("fc1.w"), g("fc1.b"))), g("fc2.w"), g("fc2.b"))
    h = layer_norm(h, f64(P["ln.g"]), f64(P["ln.b"]))
    return (h @ f64(P["tok_emb"]).T)[0]


def decoder_forward_full(tokens, ckv, P, n_dec, n_head):
    """All positions of one sequence at once under a causal mask: [n][vocab].

    A second route to the same logits as repeated decoder_step calls, used to
    pin the incremental cache against the plain causal definition."""
    n = len(tokens)
    h = f64(P["tok_emb"])[np.asarray(tokens)] + f64(P["pos_emb"])[:n]
    causal = np.tril(np.ones((n, n), dtype=bool))
    for l in range(n_dec):
        p = f"dec.{l}."
        g = lambda s: f64(P[p + s])
        a = layer_norm(h, g("attn_ln.g"), g("attn_ln.b"))
        q, k, v = linear(a, g("q.w"), g("q.b")), linear(a, g("k.w")), linear(a, g("v.w"), g("v.b"))
        h = h + linear(attention(q, k, v, n_head, causal), g("o.w"), g("o.b"))
        c = layer_norm(h, g("xattn_ln.g"), g("xattn_ln.b"))
        kc, vc = ckv[l]
        h = h + linear(attention(linear(c, g("xq.w"), g("xq.b")), kc, vc, n_head), g("xo.w"), g("xo.b"))
        m = layer_norm(h, g("mlp_ln.g"), g("mlp_ln.b"))
        h = h + linear(gelu(linear(m, g("fc1.w"), g("fc1.b"))), g("fc2.w"), g("fc2.b"))
    h = layer_norm(h, f64(P["ln.g"]), f64(P["ln.b"]))
    return h @ f64(P["tok_emb"]).T


def argmax_first(logits) -> int:
    """Index of the maximum, lowest index among equal maxima; NaN is an error."""
    logits = np.asarray(logits)
    if np.isnan(logits).any():
        raise ValueError("NaN logit")
    return int(np.flatnonzero(logits == logits.max())[0])


def steps_for(n_samples: int) -> int:
    """Teacher-forced steps of a clip: round-half-up of 2.7 tokens per second of
    audio (the kappa = 2.7 of Eq. 1), clamped to [1, 448]."""
    return max(1, min(448, (27 * n_samples + 80000) // 160000))
