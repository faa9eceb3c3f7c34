"""The seeded generators: determinism, shapes, and the stated distributions."""
import numpy as np

from workloads import (BERT_BASE, S_ISRTF, TINY, W_BERT_B64, W_BERT_B256_ROUNDS, W_TINY, W_XLMR_B128,
                       bf16_bits_to_f32, f32_to_bf16_bits, make_batch, make_requests, make_weights)
from workloads.gen import RoundStream


def test_bf16_round_to_nearest_even():
    # bf16 keeps 7 explicit mantissa bits: one ulp at 1.0 is 2^-7.
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 1.0 + 2 ** -9, 1.0 + 3 * 2 ** -8],
                 dtype=np.float32)
    got = bf16_bits_to_f32(f32_to_bf16_bits(x))
    # 1 + 2^-8: exact tie, even mantissa (1.0) wins; 1 + 3*2^-8: tie between 1+2^-7 (odd)
    # and 1 + 2^-6 (even), goes up.
    exp = np.array([1.0, 1.0, 1.0 + 2 ** -7, -2.5, 1.0, 1.0 + 2 ** -6], dtype=np.float32)
    assert np.array_equal(got, exp)
    # and agrees with torch's float32 -> bfloat16 conversion on random values
    import torch
    r = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 10
    ref = torch.from_numpy(r).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(r), ref)


def test_batches_deterministic_and_valid():
    for w in (W_TINY, W_BERT_B64, W_XLMR_B128):
        a, b = make_batch(w), make_batch(w)
        assert np.array_equal(a.token_ids, b.token_ids) and np.array_equal(a.cu_seqlens, b.cu_seqlens)
        assert a.cu_seqlens[0] == 0 and a.cu_seqlens[-1] == len(a.token_ids)
        assert a.n == w.n_seqs and np.all(a.lengths >= 1)
        assert a.token_ids.min() >= 1 and a.token_ids.max() < w.shape.vocab
        assert a.max_seqlen <= w.shape.max_pos
        assert sorted(a.arrival_seq.tolist()) == list(range(w.n_seqs))


def test_length_distributions():
    t = make_batch(W_TINY)
    assert t.lengths.min() >= 16 and t.lengths.max() <= 64
    b = make_batch(W_BERT_B64)
    assert b.lengths.max() <= 512 and 250 < b.lengths.mean() < 470
    x = make_batch(W_XLMR_B128)
    assert x.lengths.max() <= 2048 and 500 < x.lengths.mean() < 1100
    # Zipf(1.1) ids: rank 1 is the most frequent id
    vals, counts = np.unique(x.token_ids, return_counts=True)
    assert vals[np.argmax(counts)] == 1


def test_round_stream_grows_by_one():
    rs = RoundStream(W_BERT_B256_ROUNDS)
    b0, b1 = rs.batch(0), rs.batch(1)
    L0, L1 = b0.lengths, b1.lengths
    assert np.all((L1 == L0 + 1) | (L1 == 512))
    # below the cap the new input extends the old one by exactly one token
    s = int(np.argmin(L0))
    assert np.array_equal(b1.seq(s)[:-1], b0.seq(s))
    # above the cap the first token is kept and the window slides
    capped = np.nonzero(L0 == 512)[0]
    if len(capped):
        s = int(capped[0])
        assert b1.seq(s)[0] == b0.seq(s)[0]
        assert np.array_equal(b1.seq(s)[1:-1], b0.seq(s)[2:])


def test_weights_shapes_and_bf16_record():
    w = make_weights(TINY, 1001)
    assert w.master["w_qkv"][0].shape == (384, 128) and w.device["w_qkv"][0].dtype == np.uint16
    # tiny keeps fp32 masters: the device copy is their rounding
    assert not np.array_equal(w.master["w_1"][0], bf16_bits_to_f32(w.device["w_1"][0]))
    g = w.master["emb_ln_g"]
    assert abs(g.mean() - 1.0) < 0.01 and 0.01 < g.std() < 0.03


def test_requests():
    r = make_requests(S_ISRTF, n=500)
    assert np.all(np.diff(r.arrival_t) >= 0)
    rate = len(r) / r.arrival_t[-1]
    assert 15 < rate < 25
    R = np.array([len(x) for x in r.response])
    assert R.max() <= 2048 and R.min() >= 1 and 150 < np.median(R) < 400


def test_policy_study_streams():
    from workloads import POLICY_STUDY as st, make_policy_requests
    a = make_policy_requests(st, 4, 3.0, 1)
    b = make_policy_requests(st, 4, 3.0, 1)
    assert np.array_equal(a.arrival_t, b.arrival_t)
    assert all(np.array_equal(x, y) for x, y in zip(a.response, b.response))
    c = make_policy_requests(st, 4, 3.0, 2)
    # the same request set in another order
    key = lambda r: sorted(tuple(x[:4].tolist()) + (len(x),) for x in r.response)
    assert key(a) == key(c) and not np.array_equal(a.arrival_t, c.arrival_t)
    assert len(a) == st.n_requests and np.all(np.diff(a.arrival_t) >= 0)
    # Gamma(0.73) intervals at the requested rate: mean 1 / rate, squared CV 1 / 0.73 (checked
    # on a long draw of the same recipe)
    rlen = np.array([len(x) for x in a.response])
    rate = 3.0 * 4 / (rlen.mean() * st.step_cost_s)
    rng = np.random.Generator(np.random.PCG64(0))
    g = rng.gamma(st.gamma_shape, 1.0 / (rate * st.gamma_shape), size=400000)
    assert abs(g.mean() * rate - 1) < 0.01 and abs(g.var() / g.mean() ** 2 - 1 / 0.73) < 0.03
    gaps = np.diff(np.concatenate([[0.0], a.arrival_t]))
    assert 0.5 < gaps.mean() * rate < 1.5


def test_accuracy_model_keys():
    from workloads import accuracy_model_keys
    jobs = np.arange(200000)
    k = accuracy_model_keys(3, jobs, np.zeros_like(jobs), np.full(jobs.shape, 100.0), 19.923)
    err = k.astype(np.float64) - 100.0
    assert abs(np.abs(err).mean() - 19.923) < 0.3          # Laplace(0, b): E|X| = b
    assert abs(np.median(err)) < 0.3 and abs(err.var() - 2 * 19.923 ** 2) < 30
    # a fixed function of (seed, job, generated): independent of batching
    one = accuracy_model_keys(3, [17], [50], [42.0], 19.923)
    many = accuracy_model_keys(3, [5, 17, 9], [0, 50, 7], [1.0, 42.0, 3.0], 19.923)
    assert one[0] == many[1] and k.dtype == np.float32
    assert accuracy_model_keys(4, [17], [50], [42.0], 19.923)[0] != one[0]
