"""Pins of the fp64 encoder oracle against things other than itself.

* explicit-loop attention (pure Python) on tiny inputs;
* closed forms: one-token sequences, zero query/key projections, softmax sums;
* PyTorch CPU float64 modules (nn.Embedding, nn.LayerNorm,
  nn.TransformerEncoderLayer with post-LN and exact GELU), which implement the
  BERT encoder layer independently of this code;
* invariants: packing invariance, batch-permutation equivariance, LayerNorm
  moments.
"""
import copy
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import TINY, W_TINY, EncoderShape, make_batch, make_weights, pack
from workloads.configs import POOL_CLS, POOL_MEAN

torch.set_default_dtype(torch.float64)


def _rand_weights(shape: EncoderShape, seed: int):
    return make_weights(shape, seed).master


# A small shape with every feature switched on: MLP head, mean pooling, d_head 16.
SMALL_MEAN = EncoderShape("small_mean", 2, 64, 4, 128, 97, 40, POOL_MEAN, 24, True, ln_eps=1e-3,
                          out_scale=7.0, out_shift=-3.0)
SMALL_CLS = EncoderShape("small_cls", 3, 48, 3, 96, 50, 32, POOL_CLS, 0, True, ln_eps=1e-5,
                         out_scale=100.0, out_shift=250.0)


# ---------------------------------------------------------------------------- attention

def _loop_attention(q, k, v, n_heads):
    n, d = len(q), len(q[0])
    dh = d // n_heads
    out = [[0.0] * d for _ in range(n)]
    for h in range(n_heads):
        for i in range(n):
            s = []
            for j in range(n):
                acc = 0.0
                for c in range(h * dh, (h + 1) * dh):
                    acc += q[i][c] * k[j][c]
                s.append(acc / math.sqrt(dh))
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for c in range(h * dh, (h + 1) * dh):
                out[i][c] = sum(e[j] / z * v[j][c] for j in range(n))
    return out


@pytest.mark.parametrize("n,d,h", [(1, 8, 2), (5, 8, 2), (7, 12, 3), (4, 16, 1)])
def test_attention_matches_explicit_loops(n, d, h):
    rng = np.random.default_rng(n * 100 + d)
    q, k, v = (rng.standard_normal((n, d)) * 1.5 for _ in range(3))
    ref = np.array(_loop_attention(q.tolist(), k.tolist(), v.tolist(), h))
    got = oracle.self_attention(q, k, v, h)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(0)
    s = rng.standard_normal((50, 33)) * 30.0
    p = oracle.softmax_rows(s)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(axis=1) - 1.0)) < 1e-12
    # argmax of scores is argmax of probabilities
    assert np.array_equal(p.argmax(axis=1), s.argmax(axis=1))


def test_single_token_attention_returns_value():
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((1, 12)) for _ in range(3))
    assert np.array_equal(oracle.self_attention(q, k, v, 3), v)


def test_zero_query_key_gives_mean_of_values():
    rng = np.random.default_rng(2)
    n, d = 9, 16
    v = rng.standard_normal((n, d))
    zero = np.zeros((n, d))
    got = oracle.self_attention(zero, zero, v, 4)
    np.testing.assert_allclose(got, np.broadcast_to(v.mean(axis=0), (n, d)), rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------- elementwise

def test_gelu_known_values_and_torch():
    # GELU(x) = x * Phi(x); Phi(1) = 0.8413447460685429 (standard normal CDF table value).
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15
    assert abs(oracle.gelu(np.array([-1.0]))[0] + 0.15865525393145707) < 1e-15
    x = np.linspace(-8, 8, 1001)
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(oracle.gelu(x), ref, rtol=1e-14, atol=1e-15)


def test_layer_norm_moments_and_torch():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((20, 37)) * 4 + 2
    y = oracle.layer_norm(z, np.ones(37), np.zeros(37), 1e-12)
    assert np.max(np.abs(y.mean(axis=1))) < 1e-13
    assert np.max(np.abs(y.var(axis=1) - 1.0)) < 1e-10
    g, b = rng.standard_normal(37), rng.standard_normal(37)
    for eps in (1e-12, 1e-3, 0.5):
        ln = torch.nn.LayerNorm(37, eps=eps)
        with torch.no_grad():
            ln.weight.copy_(torch.from_numpy(g))
            ln.bias.copy_(torch.from_numpy(b))
            ref = ln(torch.from_numpy(z)).numpy()
        np.testing.assert_allclose(oracle.layer_norm(z, g, b, eps), ref, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------- torch model

def _torch_layer(shape, m, l):
    d = shape.d_model
    layer = torch.nn.TransformerEncoderLayer(d, shape.n_heads, shape.d_ff, dropout=0.0, activation="gelu",
                                             norm_first=False, layer_norm_eps=shape.ln_eps, batch_first=True)
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(m["w_qkv"][l]))
        layer.self_attn.in_proj_bias.copy_(t(m["b_qkv"][l]))
        layer.self_attn.out_proj.weight.copy_(t(m["w_o"][l]))
        layer.self_attn.out_proj.bias.copy_(t(m["b_o"][l]))
        layer.linear1.weight.copy_(t(m["w_1"][l]))
        layer.linear1.bias.copy_(t(m["b_1"][l]))
        layer.linear2.weight.copy_(t(m["w_2"][l]))
        layer.linear2.bias.copy_(t(m["b_2"][l]))
        layer.norm1.weight.copy_(t(m["ln1_g"][l]))
        layer.norm1.bias.copy_(t(m["ln1_b"][l]))
        layer.norm2.weight.copy_(t(m["ln2_g"][l]))
        layer.norm2.bias.copy_(t(m["ln2_b"][l]))
    layer.train(False)
    return layer


def _torch_predict(shape, m, ids):
    """Whole predictor from torch modules, float64, one sequence."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    d = shape.d_model
    word = torch.nn.Embedding(shape.vocab, d)
    pos = torch.nn.Embedding(shape.max_pos, d)
    ln = torch.nn.LayerNorm(d, eps=shape.ln_eps)
    with torch.no_grad():
        word.weight.copy_(t(m["word"]))
        pos.weight.copy_(t(m["pos"]))
        ln.weight.copy_(t(m["emb_ln_g"]))
        ln.bias.copy_(t(m["emb_ln_b"]))
        ids_t = torch.from_numpy(np.asarray(ids, dtype=np.int64))
        x = ln(word(ids_t) + pos(torch.arange(len(ids))) + t(m["type0"]))[None]
        for l in range(shape.n_layers):
            x = _torch_layer(shape, m, l)(x)
        h = x[0]
        z = h[0] if shape.pooling == POOL_CLS else h.mean(dim=0)
        if shape.head_hidden:
            lin1 = torch.nn.Linear(d, shape.head_hidden)
            lin1.weight.copy_(t(m["head_w1"]))
            lin1.bias.copy_(t(m["head_b1"]))
            z = torch.relu(lin1(z))
        lin2 = torch.nn.Linear(z.shape[0], 1)
        lin2.weight.copy_(t(m["head_w2"]))
        lin2.bias.copy_(t(m["head_b2"]))
        y = lin2(z)[0]
    return float(shape.out_shift + shape.out_scale * y), h.numpy()


@pytest.mark.parametrize("shape,seed", [(SMALL_MEAN, 11), (SMALL_CLS, 12)])
def test_encoder_layer_matches_torch(shape, seed):
    m = _rand_weights(shape, seed)
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((13, shape.d_model))
    for l in range(shape.n_layers):
        ref = _torch_layer(shape, m, l)(torch.from_numpy(x)[None]).detach().numpy()[0]
        np.testing.assert_allclose(oracle.encoder_layer(x, m, l, shape.n_heads, shape.ln_eps), ref,
                                   rtol=1e-10, atol=1e-10)


def test_embedding_matches_torch():
    shape = SMALL_MEAN
    m = _rand_weights(shape, 21)
    ids = np.array([5, 0, 96, 5, 17, 3])
    word = torch.nn.Embedding(shape.vocab, shape.d_model)
    pos = torch.nn.Embedding(shape.max_pos, shape.d_model)
    ln = torch.nn.LayerNorm(shape.d_model, eps=shape.ln_eps)
    with torch.no_grad():
        word.weight.copy_(torch.from_numpy(m["word"].astype(np.float64)))
        pos.weight.copy_(torch.from_numpy(m["pos"].astype(np.float64)))
        ln.weight.copy_(torch.from_numpy(m["emb_ln_g"].astype(np.float64)))
        ln.bias.copy_(torch.from_numpy(m["emb_ln_b"].astype(np.float64)))
        ref = ln(word(torch.from_numpy(ids)) + pos(torch.arange(len(ids)))
                 + torch.from_numpy(m["type0"].astype(np.float64))).numpy()
    np.testing.assert_allclose(oracle.embed(ids, m, shape.ln_eps), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape,seed", [(SMALL_MEAN, 31), (SMALL_CLS, 32), (TINY, 1001)])
def test_whole_forward_matches_torch_model(shape, seed):
    m = _rand_weights(shape, seed)
    rng = np.random.default_rng(seed)
    seqs = [rng.integers(1, shape.vocab, size=int(L)) for L in (1, 7, min(shape.max_pos, 29))]
    b = pack(seqs)
    pred, hid = oracle.oracle_forward(b.token_ids, b.cu_seqlens, m, shape)
    for s, ids in enumerate(seqs):
        p_ref, h_ref = _torch_predict(shape, m, ids)
        np.testing.assert_allclose(hid[b.cu_seqlens[s]:b.cu_seqlens[s + 1]], h_ref, rtol=1e-10, atol=1e-10)
        assert abs(pred[s] - p_ref) <= 1e-9 * max(1.0, abs(p_ref))


def test_head_hand_computed():
    shape = EncoderShape("h", 0, 4, 1, 4, 2, 2, POOL_CLS, 2, True, out_scale=10.0, out_shift=1.0)
    m = {"head_w1": np.array([[1.0, 0, 0, 0], [0, -1.0, 0, 0]]), "head_b1": np.array([0.5, 0.0]),
         "head_w2": np.array([[2.0, 3.0]]), "head_b2": np.array([0.25])}
    z = np.array([1.0, 2.0, 3.0, 4.0])
    # hidden = relu([1.5, -2.0]) = [1.5, 0]; y = 2*1.5 + 0.25 = 3.25; pred = 1 + 10*3.25
    assert oracle.regression_head(z, m, shape) == 33.5
    lin = EncoderShape("h", 0, 4, 1, 4, 2, 2, POOL_CLS, 0, True, out_scale=2.0, out_shift=0.0)
    m2 = {"head_w2": np.array([[1.0, -1.0, 0.5, 0.0]]), "head_b2": np.array([-1.0])}
    # y = 1 - 2 + 1.5 - 1 = -0.5; pred = -1
    assert oracle.regression_head(z, m2, lin) == -1.0


def test_pooling():
    h = np.arange(12.0).reshape(4, 3)
    assert np.array_equal(oracle.pool(h, POOL_CLS), h[0])
    np.testing.assert_allclose(oracle.pool(h, POOL_MEAN), [4.5, 5.5, 6.5])
    c = np.tile(np.array([[1.5, -2.0, 7.0]]), (9, 1))
    assert np.array_equal(oracle.pool(c, POOL_MEAN), c[0])


# ---------------------------------------------------------------------------- invariants

def test_packing_invariance_bitwise():
    shape = SMALL_MEAN
    m = _rand_weights(shape, 41)
    rng = np.random.default_rng(41)
    seqs = [rng.integers(1, shape.vocab, size=int(L)) for L in (3, 17, 1, 40, 8)]
    b = pack(seqs)
    pred, hid = oracle.oracle_forward(b.token_ids, b.cu_seqlens, m, shape)
    for s, ids in enumerate(seqs):
        alone = pack([ids])
        p1, h1 = oracle.oracle_forward(alone.token_ids, alone.cu_seqlens, m, shape)
        assert p1[0] == pred[s]
        assert np.array_equal(h1, hid[b.cu_seqlens[s]:b.cu_seqlens[s + 1]])


def test_batch_permutation_equivariance():
    shape = SMALL_CLS
    m = _rand_weights(shape, 42)
    rng = np.random.default_rng(42)
    seqs = [rng.integers(1, shape.vocab, size=int(L)) for L in (5, 9, 2, 12)]
    perm = [2, 0, 3, 1]
    b = pack(seqs)
    bp = pack([seqs[i] for i in perm])
    p, _ = oracle.oracle_forward(b.token_ids, b.cu_seqlens, m, shape)
    pp, _ = oracle.oracle_forward(bp.token_ids, bp.cu_seqlens, m, shape)
    assert np.array_equal(pp, p[perm])


def test_mean_pool_of_identical_tokens_equals_cls():
    # identical tokens and a zero position table make every row of the output equal
    shape = SMALL_MEAN
    m = copy.deepcopy(_rand_weights(shape, 43))
    m["pos"] = np.zeros_like(m["pos"])
    ids = np.full(6, 7)
    h = oracle.encode_sequence(ids, m, shape)
    np.testing.assert_allclose(h, np.broadcast_to(h[0], h.shape), rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.pool(h, POOL_MEAN), h[0], rtol=0, atol=1e-12)


def test_tiny_workload_runs():
    w = W_TINY
    b = make_batch(w)
    m = make_weights(w.shape, w.weight_seed).master
    pred, hid = oracle.oracle_forward(b.token_ids, b.cu_seqlens, m, w.shape)
    assert pred.shape == (8,) and np.all(np.isfinite(pred))
    assert hid.shape == (b.total, 128) and np.all(np.isfinite(hid))


# ------------------------------------------------------------------------------ deep heads (Sec. 3.2, Sec. 4.2)
def _deep_head(nl, hh, d, act, rng, nonneg=False):
    shape = EncoderShape("h", 0, d, 1, 64, 10, 8, POOL_CLS, hh, True, head_layers=nl, head_act=act)
    draw = (lambda *s: np.abs(rng.standard_normal(s))) if nonneg else (lambda *s: rng.standard_normal(s))
    m = {"head_w1": draw(hh, d) / math.sqrt(d), "head_b1": draw(hh) * 0.1,
         "head_mid_w": [draw(hh, hh) / math.sqrt(hh) for _ in range(nl - 2)],
         "head_mid_b": [draw(hh) * 0.1 for _ in range(nl - 2)],
         "head_w2": draw(1, hh) / math.sqrt(hh), "head_b2": draw(1) * 0.1}
    return shape, m


@pytest.mark.parametrize("act,nonneg", [(1, False), (0, True)])
def test_deep_head_equals_composed_affine_map(act, nonneg):
    """Eight linear layers collapse to one affine map W z + c (W = W8 ... W1); with ReLU
    the same holds when weights, biases and input are all non-negative."""
    rng = np.random.default_rng(11 + act)
    d, hh = 24, 16
    shape, m = _deep_head(8, hh, d, act, rng, nonneg)
    Ws = [m["head_w1"]] + m["head_mid_w"] + [m["head_w2"]]
    bs = [m["head_b1"]] + m["head_mid_b"] + [m["head_b2"]]
    W, c = np.eye(d), np.zeros(d)
    for w, b in zip(Ws, bs):
        W, c = w @ W, w @ c + b
    for _ in range(5):
        z = np.abs(rng.standard_normal(d)) if nonneg else rng.standard_normal(d)
        y = float((W @ z + c)[0])
        assert abs(oracle.regression_head(z, m, shape) - (shape.out_shift + shape.out_scale * y)) < 1e-9


def test_deep_head_matches_torch_sequential():
    rng = np.random.default_rng(5)
    d, hh = 32, 24
    shape, m = _deep_head(8, hh, d, 0, rng)
    Ws = [m["head_w1"]] + m["head_mid_w"] + [m["head_w2"]]
    bs = [m["head_b1"]] + m["head_mid_b"] + [m["head_b2"]]
    mods = []
    for i, (w, b) in enumerate(zip(Ws, bs)):
        lin = torch.nn.Linear(w.shape[1], w.shape[0], dtype=torch.float64)
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(w))
            lin.bias.copy_(torch.from_numpy(np.asarray(b)))
        mods.append(lin)
        if i < len(Ws) - 1:
            mods.append(torch.nn.ReLU())
    net = torch.nn.Sequential(*mods)
    for _ in range(5):
        z = rng.standard_normal(d)
        y = float(net(torch.from_numpy(z)).item())
        assert abs(oracle.regression_head(z, m, shape) - (shape.out_shift + shape.out_scale * y)) < 1e-9


def test_deep_head_workload_weights():
    from workloads import TINY_HEAD8, BERT_BASE_HEAD8, TINY_CLS_LIN8
    for shape in (TINY_HEAD8, TINY_CLS_LIN8):
        W = make_weights(shape, 1)
        assert shape.n_head_layers == 8
        assert len(W.master["head_mid_w"]) == 6 and len(W.device["head_mid_b"]) == 6
        assert W.master["head_w1"].shape == (shape.head_hidden, shape.d_model)
        assert W.master["head_mid_w"][0].shape == (shape.head_hidden, shape.head_hidden)
        assert W.master["head_w2"].shape == (1, shape.head_hidden)
    assert BERT_BASE_HEAD8.n_head_layers == 8 and BERT_BASE_HEAD8.head_hidden == 1024
    assert BERT_BASE_HEAD8.pooling == POOL_MEAN
    # the one- and two-layer heads keep their shapes
    assert TINY.n_head_layers == 1
