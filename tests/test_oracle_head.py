"""The oracle's verifier head (projection + positional encoding, two
post-norm encoder layers, mean pool, sigmoid) against PyTorch's own encoder
layer in float64, an independent implementation of the same architecture,
and against closed forms; planted mistakes in copies of it must be caught.
CPU only."""

import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import head as ohead
from paper_2608_28726_amd import workloads as wl

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def test_parameter_count():
    assert ohead.HEAD_WEIGHTS == 67329  # "about 67k parameters" (Sec. 4.2)
    assert wl.head_weights().shape == (67329,)


def test_positional_encoding_closed_forms():
    pe = ohead.positional_encoding(5)
    assert np.array_equal(pe[0], np.tile([0.0, 1.0], 32))  # position 0: sin 0, cos 0
    for t in range(5):
        assert pe[t, 0] == math.sin(t) and pe[t, 1] == math.cos(t)
        assert abs(pe[t, 63] - math.cos(t * 10000.0 ** (-62 / 64))) < 1e-15


def _torch_head(W, X):
    """The same head assembled from torch.nn modules (float64)."""
    d = ohead.HEAD_D
    layer = torch.nn.TransformerEncoderLayer(d_model=d, nhead=4, dim_feedforward=128, dropout=0.0,
                                             activation="relu", batch_first=True, norm_first=False,
                                             layer_norm_eps=1e-5, dtype=torch.float64)
    enc = torch.nn.TransformerEncoder(layer, num_layers=2, enable_nested_tensor=False)
    t = lambda a: torch.tensor(a, dtype=torch.float64)
    with torch.no_grad():
        for l, lay in enumerate(enc.layers):
            lay.self_attn.in_proj_weight.copy_(t(W[f"W_qkv{l}"]))
            lay.self_attn.in_proj_bias.copy_(t(W[f"b_qkv{l}"]))
            lay.self_attn.out_proj.weight.copy_(t(W[f"W_o{l}"]))
            lay.self_attn.out_proj.bias.copy_(t(W[f"b_o{l}"]))
            lay.linear1.weight.copy_(t(W[f"W_1{l}"]))
            lay.linear1.bias.copy_(t(W[f"b_1{l}"]))
            lay.linear2.weight.copy_(t(W[f"W_2{l}"]))
            lay.linear2.bias.copy_(t(W[f"b_2{l}"]))
            lay.norm1.weight.copy_(t(W[f"ln1_g{l}"]))
            lay.norm1.bias.copy_(t(W[f"ln1_b{l}"]))
            lay.norm2.weight.copy_(t(W[f"ln2_g{l}"]))
            lay.norm2.bias.copy_(t(W[f"ln2_b{l}"]))
        enc.eval()
        T = X.shape[0]
        pos = torch.arange(T, dtype=torch.float64)[:, None]
        div = torch.tensor([10000.0 ** (2 * i / d) for i in range(d // 2)], dtype=torch.float64)
        pe = torch.zeros(T, d, dtype=torch.float64)
        pe[:, 0::2] = torch.sin(pos / div)
        pe[:, 1::2] = torch.cos(pos / div)
        h = t(X) @ t(W["W_in"]).T + t(W["b_in"]) + pe
        h = enc(h[None])[0]
        z = h.mean(dim=0) @ t(W["w_out"]) + t(W["b_out"])[0]
        return float(torch.sigmoid(z))


def _requests(rng, lengths):
    X = np.concatenate([np.stack([rng.normal(-1, 1, n), rng.uniform(0, 1, n), -rng.uniform(0, 3, n),
                                  (np.arange(n) + 1) / max(n, 1)], axis=1) for n in lengths])
    off = np.concatenate([[0], np.cumsum(lengths)])
    return X, off


def pin_torch(mod, seeds=(0, 1, 2)):
    """Scores of requests of several lengths against the torch assembly."""
    fails = []
    for s in seeds:
        rng = np.random.default_rng(s)
        weights = wl.head_weights(seed=100 + s).astype(np.float64)
        W = ohead.unpack_weights(weights)
        lengths = [1, 2, 7, 40]
        X, off = _requests(rng, lengths)
        got = mod.head_scores(X, off, weights)
        for i in range(len(lengths)):
            ref = _torch_head(W, X[off[i]:off[i + 1]])
            if not abs(got[i] - ref) <= 1e-12:
                fails.append(f"seed {s} request {i} (T={lengths[i]}): {got[i]} vs torch {ref}")
    return fails


def pin_closed_forms(mod):
    """A zero output map gives sigmoid(b_out); an empty request gives NaN;
    a request's score does not depend on the other requests of the batch."""
    fails = []
    rng = np.random.default_rng(7)
    weights = wl.head_weights(seed=9).astype(np.float64)
    W = ohead.unpack_weights(weights)
    X, off = _requests(rng, [3, 5])
    w0 = weights.copy()
    n_out = 65  # w_out and b_out are the last 65 entries
    w0[-n_out:-1] = 0.0
    s0 = mod.head_scores(X, off, w0)
    expect = 1.0 / (1.0 + math.exp(-w0[-1]))
    if not np.allclose(s0, expect, rtol=0, atol=1e-15):
        fails.append(f"zero output map: {s0} != {expect}")
    e = mod.head_scores(X[:0], np.array([0, 0]), weights)
    if not math.isnan(e[0]):
        fails.append(f"empty request: {e[0]}")
    alone = mod.head_scores(X[3:8], np.array([0, 5]), weights)[0]
    batched = mod.head_scores(X, off, weights)[1]
    if alone != batched:
        fails.append(f"batch dependence: {alone} vs {batched}")
    return fails


def test_oracle_matches_torch_encoder():
    fails = pin_torch(ohead)
    assert not fails, "\n".join(fails)


def test_oracle_closed_forms():
    fails = pin_closed_forms(ohead)
    assert not fails, "\n".join(fails)


MUTANTS = {
    "pre-norm layer": ("    a = self_attention(h, W[f\"W_qkv{l}\"], W[f\"b_qkv{l}\"], W[f\"W_o{l}\"], W[f\"b_o{l}\"])\n"
                       "    h = layer_norm(h + a, W[f\"ln1_g{l}\"], W[f\"ln1_b{l}\"])",
                       "    a = self_attention(layer_norm(h, W[f\"ln1_g{l}\"], W[f\"ln1_b{l}\"]), W[f\"W_qkv{l}\"], "
                       "W[f\"b_qkv{l}\"], W[f\"W_o{l}\"], W[f\"b_o{l}\"])\n    h = h + a"),
    "unscaled scores": ("s = q[:, c] @ k[:, c].T / math.sqrt(dh)", "s = q[:, c] @ k[:, c].T"),
    "1-based positions": ("angle = t / (10000.0 ** (2 * i / HEAD_D))", "angle = (t + 1) / (10000.0 ** (2 * i / HEAD_D))"),
    "no relu": ("f = np.maximum(h @ W[f\"W_1{l}\"].T + W[f\"b_1{l}\"], 0.0)", "f = (h @ W[f\"W_1{l}\"].T + W[f\"b_1{l}\"])"),
    "sum pool": ("z = float(h.mean(axis=0) @ W[\"w_out\"]", "z = float(h.sum(axis=0) @ W[\"w_out\"]"),
    "unbiased variance": ("var = ((h - mu) ** 2).mean(axis=1, keepdims=True)",
                          "var = ((h - mu) ** 2).sum(axis=1, keepdims=True) / (h.shape[1] - 1)"),
    "keys and values swapped": ("q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]",
                                "q, v, k = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]"),
    "one head": ("    for hd in range(HEAD_HEADS):\n        c = slice(hd * dh, (hd + 1) * dh)",
                 "    for hd in range(1):\n        c = slice(0, d)"),
}


def _mutant(old, new):
    src = open(os.path.join(ORACLE_DIR, "head.py")).read()
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    mod = types.ModuleType("head_mutant")
    exec(compile(src.replace(old, new), "mutant:head.py", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_head_mutant_is_caught(name):
    mod = _mutant(*MUTANTS[name])
    assert pin_torch(mod, seeds=(0,)) or pin_closed_forms(mod), f"mutant '{name}' passed every pin"
