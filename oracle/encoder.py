"""fp64 CPU oracle of the response-length predictor's forward pass.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module;
only the test-suite, the smoke check and the benchmark's CPU-baseline leg do.

The predictor is a BERT-style bidirectional Transformer encoder (the paper
builds it on BGE, a BERT-family model: Sec. 3.1) followed by pooling and a
regression head that outputs the number of tokens the job still has to
generate (Sec. 3.2 uses the CLS vector; Sec. 4.2 uses mean pooling over all
token embeddings; Sec. 3.3 defines the target as the remaining tokens).

Everything is computed per sequence, in float64, in the order the method
defines it; numpy's matmul is the only library primitive used for the
contractions. The readings of points the paper leaves open are:
  * post-LayerNorm encoder layers with an embedding LayerNorm (BERT layout);
  * LayerNorm with biased variance and epsilon from the config (1e-12);
  * exact erf GELU in the feed-forward block;
  * one token-type row added to every token; no BERT tanh pooler;
  * position ids restart at 0 for every sequence of a packed batch;
  * prediction = out_shift + out_scale * head output.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

POOL_CLS = 0
POOL_MEAN = 1


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def layer_norm(z: np.ndarray, gain: np.ndarray, bias: np.ndarray, eps: float) -> np.ndarray:
    """Normalise each row to zero mean, unit (biased) variance, then scale and shift."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return _f64(gain) * (z - mu) / np.sqrt(var + eps) + _f64(bias)


def gelu(u: np.ndarray) -> np.ndarray:
    """GELU, exact form: u * Phi(u), Phi the standard normal CDF."""
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row-wise softmax, shifted by the row maximum."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def embed(ids: np.ndarray, m: dict, eps: float) -> np.ndarray:
    """Token embedding + learned position embedding (positions from 0) + type-0 row, then LayerNorm."""
    n = len(ids)
    e = _f64(m["word"][ids]) + _f64(m["pos"][:n]) + _f64(m["type0"])[None, :]
    return layer_norm(e, m["emb_ln_g"], m["emb_ln_b"], eps)


def self_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Bidirectional multi-head attention within one sequence.

    q, k, v are [n, d]; head h owns columns h*dh .. (h+1)*dh - 1. Every token
    attends to every token of the same sequence (no mask: an encoder sees the
    whole input). Returns the concatenated head outputs, [n, d].
    """
    n, d = q.shape
    dh = d // n_heads
    out = np.empty((n, d), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        s = (q[:, cols] @ k[:, cols].T) / math.sqrt(dh)
        p = softmax_rows(s)
        out[:, cols] = p @ v[:, cols]
    return out


def encoder_layer(x: np.ndarray, m: dict, l: int, n_heads: int, eps: float) -> np.ndarray:
    """One post-LN encoder layer: attention sub-block, then feed-forward sub-block."""
    d = x.shape[1]
    qkv = x @ _f64(m["w_qkv"][l]).T + _f64(m["b_qkv"][l])
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    a = self_attention(q, k, v, n_heads)
    x1 = layer_norm(x + a @ _f64(m["w_o"][l]).T + _f64(m["b_o"][l]), m["ln1_g"][l], m["ln1_b"][l], eps)
    f = gelu(x1 @ _f64(m["w_1"][l]).T + _f64(m["b_1"][l]))
    return layer_norm(x1 + f @ _f64(m["w_2"][l]).T + _f64(m["b_2"][l]), m["ln2_g"][l], m["ln2_b"][l], eps)


def encode_sequence(ids: np.ndarray, m: dict, shape) -> np.ndarray:
    """Final hidden states [n, d] of one sequence."""
    x = embed(np.asarray(ids), m, shape.ln_eps)
    for l in range(shape.n_layers):
        x = encoder_layer(x, m, l, shape.n_heads, shape.ln_eps)
    return x


def pool(h: np.ndarray, pooling: int) -> np.ndarray:
    """CLS pooling takes the first token's vector; mean pooling averages every token (CLS included)."""
    if pooling == POOL_CLS:
        return h[0].copy()
    if pooling == POOL_MEAN:
        return h.mean(axis=0)
    raise ValueError(pooling)


def _head_layers(shape) -> int:
    n = getattr(shape, "head_layers", 0)
    if n:
        return n
    return 2 if shape.head_hidden else 1


def regression_head(z: np.ndarray, m: dict, shape) -> float:
    """Fully connected layers on the pooled vector, then the affine map to tokens.

    One layer: y = w2 . z + b2. More: h = act(W1 z + b1), then head_layers - 2 times
    h = act(Wl h + bl), then y = w2 . h + b2, with act = ReLU (Sec. 4.2) or none
    (a stack of linear layers, Sec. 3.2)."""
    nl = _head_layers(shape)
    relu = getattr(shape, "head_act", 0) == 0
    act = (lambda v: np.maximum(v, 0.0)) if relu else (lambda v: v)
    h = z
    if nl >= 2:
        h = act(_f64(m["head_w1"]) @ h + _f64(m["head_b1"]))
        for w, b in zip(m.get("head_mid_w", []), m.get("head_mid_b", [])):
            h = act(_f64(w) @ h + _f64(b))
    y = float(_f64(m["head_w2"])[0] @ h + _f64(m["head_b2"])[0])
    return shape.out_shift + shape.out_scale * y


def oracle_forward(token_ids, cu_seqlens, m: dict, shape, want_hidden: bool = True,
                   seqs=None):
    """Predicted remaining tokens for every sequence of a packed batch.

    token_ids  int[T], cu_seqlens int[n+1]; m is the weight dict (fp32 values of record).
    seqs: optional subset of sequence indices to evaluate (others are NaN / absent).
    Returns (pred float64[n], hidden float64[T, d] or None). Rows of sequences not
    evaluated are NaN.
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    ids = np.asarray(token_ids, dtype=np.int64)
    n = len(cu) - 1
    pred = np.full(n, np.nan)
    hidden = np.full((int(cu[-1]), shape.d_model), np.nan) if want_hidden else None
    which = range(n) if seqs is None else seqs
    for s in which:
        h = encode_sequence(ids[cu[s]:cu[s + 1]], m, shape)
        if want_hidden:
            hidden[cu[s]:cu[s + 1]] = h
        pred[s] = regression_head(pool(h, shape.pooling), m, shape)
    return pred, hidden
