"""fp64 oracle: the paper's verifier head over a request's input sequence.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Source: Pro-Router, Sec. 3.1, the paragraph after Eq. 3: the stacked
per-token tuples X (T rows, 4 columns) pass through a linear projection with
positional encoding (the sinusoidal encoding of Vaswani et al., 2017), a
transformer encoder, a mean pool over the tokens and a sigmoid layer that
outputs the request's shipping confidence p; the request ships iff p >= tau
(Sec. 3.1, with the gain, Eq. 1). Sec. 4.2 (the signal-latency paragraph and
Table "ablation") gives two encoder layers and about 67k parameters.

Readings where the paper is silent:

R17  Width d = 64 and feed-forward width 128: with biases and two LayerNorms
     per layer this is 67,329 parameters, the paper's "about 67k". The
     encoder layer is the original post-norm one: h <- LN(h + MHA(h)),
     h <- LN(h + W2 relu(W1 h + b1) + b2), LayerNorm over the 64 features with
     the biased variance and eps = 1e-5, 4 heads of 16 dimensions, scores
     scaled by 1/sqrt(16), softmax over every token of the same request (the
     verifier reads a finished request, so nothing is masked).
R18  The positional encoding of token t (1-based) is the sinusoid at
     position t - 1: PE[2i] = sin((t-1) / 10000^(2i/64)),
     PE[2i+1] = cos((t-1) / 10000^(2i/64)), added after the projection.
R19  The sigmoid layer is a linear map of the pooled 64 features to one
     logit, then the logistic sigmoid. An empty request has score NaN (it
     escalates).
R20  The paper publishes no weights: the head runs with seeded synthetic
     weights, so its scores are parity unpinned against the paper; the
     oracle is pinned against an independent implementation of the same
     architecture and against closed forms.

Weights are a flat float32 array (HEAD_WEIGHTS entries) in the order of
:data:`HEAD_LAYOUT`: each matrix row-major [out][in]; within the 192 rows of
a layer's QKV projection the queries come first, then the keys, then the
values, and head h owns rows 16h .. 16h+15 of each.
"""

from __future__ import annotations

import math

import numpy as np

HEAD_D = 64
HEAD_FF = 128
HEAD_HEADS = 4
HEAD_LAYERS = 2
HEAD_LN_EPS = 1e-5


def _layout():
    d, f = HEAD_D, HEAD_FF
    items = [("W_in", (d, 4)), ("b_in", (d,))]
    for l in range(HEAD_LAYERS):
        items += [(f"W_qkv{l}", (3 * d, d)), (f"b_qkv{l}", (3 * d,)), (f"W_o{l}", (d, d)), (f"b_o{l}", (d,)),
                  (f"ln1_g{l}", (d,)), (f"ln1_b{l}", (d,)), (f"W_1{l}", (f, d)), (f"b_1{l}", (f,)),
                  (f"W_2{l}", (d, f)), (f"b_2{l}", (d,)), (f"ln2_g{l}", (d,)), (f"ln2_b{l}", (d,))]
    items += [("w_out", (d,)), ("b_out", (1,))]
    return items


HEAD_LAYOUT = _layout()
HEAD_WEIGHTS = sum(int(np.prod(s)) for _, s in HEAD_LAYOUT)  # 67,329


def unpack_weights(flat) -> dict:
    """The named float64 arrays of a flat weight vector (HEAD_LAYOUT order)."""
    flat = np.asarray(flat, dtype=np.float64).reshape(-1)
    if flat.shape[0] != HEAD_WEIGHTS:
        raise ValueError(f"expected {HEAD_WEIGHTS} weights, got {flat.shape[0]}")
    out, k = {}, 0
    for name, shape in HEAD_LAYOUT:
        n = int(np.prod(shape))
        out[name] = flat[k:k + n].reshape(shape)
        k += n
    return out


def positional_encoding(T: int) -> np.ndarray:
    """Sinusoids of positions 0 .. T-1 (reading R18), float64 [T][64]."""
    pe = np.zeros((T, HEAD_D))
    for t in range(T):
        for i in range(HEAD_D // 2):
            angle = t / (10000.0 ** (2 * i / HEAD_D))
            pe[t, 2 * i] = math.sin(angle)
            pe[t, 2 * i + 1] = math.cos(angle)
    return pe


def layer_norm(h, g, b):
    """Per row over the 64 features: biased variance, eps = 1e-5 (R17)."""
    mu = h.mean(axis=1, keepdims=True)
    var = ((h - mu) ** 2).mean(axis=1, keepdims=True)
    return (h - mu) / np.sqrt(var + HEAD_LN_EPS) * g + b


def self_attention(h, Wqkv, bqkv, Wo, bo):
    """Multi-head attention over the T tokens of one request (no mask)."""
    T = h.shape[0]
    d, dh = HEAD_D, HEAD_D // HEAD_HEADS
    qkv = h @ Wqkv.T + bqkv
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    out = np.empty((T, d))
    for hd in range(HEAD_HEADS):
        c = slice(hd * dh, (hd + 1) * dh)
        s = q[:, c] @ k[:, c].T / math.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, c] = p @ v[:, c]
    return out @ Wo.T + bo


def encoder_layer(h, W, l):
    """One post-norm encoder layer (R17)."""
    a = self_attention(h, W[f"W_qkv{l}"], W[f"b_qkv{l}"], W[f"W_o{l}"], W[f"b_o{l}"])
    h = layer_norm(h + a, W[f"ln1_g{l}"], W[f"ln1_b{l}"])
    f = np.maximum(h @ W[f"W_1{l}"].T + W[f"b_1{l}"], 0.0) @ W[f"W_2{l}"].T + W[f"b_2{l}"]
    return layer_norm(h + f, W[f"ln2_g{l}"], W[f"ln2_b{l}"])


def head_score(X, W) -> float:
    """Shipping confidence p of one request from its input sequence X [T][4]
    (Sec. 3.1): projection + positional encoding, encoder layers, mean pool,
    sigmoid. NaN for an empty request (R19)."""
    X = np.asarray(X, dtype=np.float64)
    T = X.shape[0]
    if T == 0:
        return math.nan
    h = X @ W["W_in"].T + W["b_in"] + positional_encoding(T)
    for l in range(HEAD_LAYERS):
        h = encoder_layer(h, W, l)
    z = float(h.mean(axis=0) @ W["w_out"] + W["b_out"][0])
    return 1.0 / (1.0 + math.exp(-z))


def head_scores(X, offsets, weights) -> np.ndarray:
    """Scores of every request of a ragged batch (request i owns rows
    offsets[i] .. offsets[i+1]-1 of X [n_rows][4])."""
    W = unpack_weights(weights)
    X = np.asarray(X, dtype=np.float64)
    offsets = np.asarray(offsets, dtype=np.int64)
    return np.array([head_score(X[offsets[i]:offsets[i + 1]], W) for i in range(offsets.shape[0] - 1)])
