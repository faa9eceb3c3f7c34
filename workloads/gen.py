"""Seeded synthetic inputs: encoder weights, packed token batches, request streams.

This module is the only code shared by the fp64 oracle and the GPU path. It
draws random numbers and lays them out; it performs none of the predictor's
or the scheduler's arithmetic.

Generator: numpy PCG64 throughout. ``lognormal(m, s)`` means
``round(exp(ln m + s * Z))`` with Z ~ N(0, 1), floored at 1.

Weight recipe (N(0, 0.02) everywhere, with LayerNorm gains centred on 1):
  matrices, embedding tables, biases, head:  N(0, 0.02)
  LayerNorm gain: 1 + N(0, 0.02); LayerNorm bias: N(0, 0.02)
  heads of more than two layers: matrices N(0, 2 / fan_in) (He), biases N(0, 0.02),
    so that a random deep head neither vanishes nor explodes
Matrices and embedding tables of the bf16 shapes are drawn in fp32 and rounded
to bf16 with round-to-nearest-even; the exact bf16 values are the weights of
record. The tiny shape keeps fp32 master weights; its device copy is the bf16
rounding of them.
"""
from __future__ import annotations

import functools
import math

import numpy as np

from .configs import POOL_CLS, EncoderShape, PolicyStudy, RequestStream, Workload

# Tensors that the device stores in bf16 (everything else is fp32).
BF16_TENSORS = ("word", "pos", "w_qkv", "w_o", "w_1", "w_2")


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even); return the 16-bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((b >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((b + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 values."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Weights:
    """Encoder + head parameters.

    ``master[name]``  fp32 numpy arrays: the weights of record (exact bf16 values
                      for the bf16 shapes; unrounded fp32 for the tiny shape).
    ``device[name]``  what a bf16 device path stores: uint16 bf16 bit patterns for
                      the tensors in BF16_TENSORS, fp32 for the rest.
    Per-layer tensors are lists indexed by layer. Matrices are [out, in].
    """

    def __init__(self, shape: EncoderShape, master: dict, device: dict):
        self.shape = shape
        self.master = master
        self.device = device


def _normal(rng: np.random.Generator, shape, std=0.02) -> np.ndarray:
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def _table(seed_seq: np.random.SeedSequence, rows: int, cols: int, chunk_rows: int = 1 << 15):
    """A large N(0, 0.02) table drawn in fixed chunks, each from its own child stream."""
    out = np.empty((rows, cols), dtype=np.float32)
    n_chunks = (rows + chunk_rows - 1) // chunk_rows
    for i, child in enumerate(seed_seq.spawn(n_chunks)):
        r0 = i * chunk_rows
        r1 = min(rows, r0 + chunk_rows)
        out[r0:r1] = _normal(np.random.Generator(np.random.PCG64(child)), (r1 - r0, cols))
    return out


@functools.lru_cache(maxsize=4)
def make_weights(shape: EncoderShape, seed: int) -> Weights:
    d, F, L = shape.d_model, shape.d_ff, shape.n_layers
    root = np.random.SeedSequence(seed)
    s_word, s_rest = root.spawn(2)
    rng = np.random.Generator(np.random.PCG64(s_rest))
    m: dict = {}
    m["word"] = _table(s_word, shape.vocab, d)
    m["pos"] = _normal(rng, (shape.max_pos, d))
    m["type0"] = _normal(rng, (d,))
    m["emb_ln_g"] = 1.0 + _normal(rng, (d,))
    m["emb_ln_b"] = _normal(rng, (d,))
    for name in ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b",
                 "w_1", "b_1", "w_2", "b_2", "ln2_g", "ln2_b"):
        m[name] = []
    for _ in range(L):
        m["w_qkv"].append(_normal(rng, (3 * d, d)))
        m["b_qkv"].append(_normal(rng, (3 * d,)))
        m["w_o"].append(_normal(rng, (d, d)))
        m["b_o"].append(_normal(rng, (d,)))
        m["ln1_g"].append(1.0 + _normal(rng, (d,)))
        m["ln1_b"].append(_normal(rng, (d,)))
        m["w_1"].append(_normal(rng, (F, d)))
        m["b_1"].append(_normal(rng, (F,)))
        m["w_2"].append(_normal(rng, (d, F)))
        m["b_2"].append(_normal(rng, (d,)))
        m["ln2_g"].append(1.0 + _normal(rng, (d,)))
        m["ln2_b"].append(_normal(rng, (d,)))
    nh, hh = shape.n_head_layers, shape.head_hidden
    if nh == 1:
        m["head_w2"] = _normal(rng, (1, d))
    elif nh == 2:
        m["head_w1"] = _normal(rng, (hh, d))
        m["head_b1"] = _normal(rng, (hh,))
        m["head_w2"] = _normal(rng, (1, hh))
    else:
        he = lambda shp: _normal(rng, shp, std=math.sqrt(2.0 / shp[1]))
        m["head_w1"] = he((hh, d))
        m["head_b1"] = _normal(rng, (hh,))
        m["head_mid_w"], m["head_mid_b"] = [], []
        for _ in range(nh - 2):
            m["head_mid_w"].append(he((hh, hh)))
            m["head_mid_b"].append(_normal(rng, (hh,)))
        m["head_w2"] = he((1, hh))
    m["head_b2"] = _normal(rng, (1,))

    dev: dict = {}
    for name, val in m.items():
        if name in BF16_TENSORS:
            if isinstance(val, list):
                dev[name] = [f32_to_bf16_bits(v) for v in val]
            else:
                dev[name] = f32_to_bf16_bits(val)
            if not shape.fp32_master:
                # bf16 shapes: the rounded values are the weights of record.
                if isinstance(val, list):
                    m[name] = [bf16_bits_to_f32(b) for b in dev[name]]
                else:
                    m[name] = bf16_bits_to_f32(dev[name])
        else:
            dev[name] = val
    return Weights(shape, m, dev)


# ----------------------------------------------------------------------------- batches

def _lognormal_int(rng: np.random.Generator, median: float, sigma: float, size: int) -> np.ndarray:
    z = rng.standard_normal(size)
    v = np.rint(np.exp(math.log(median) + sigma * z))
    return np.maximum(v, 1).astype(np.int64)


def draw_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    n = w.n_seqs
    if w.len_kind == "uniform":
        return rng.integers(w.len_lo, w.len_hi + 1, size=n).astype(np.int64)
    if w.len_kind == "prompt+gen":
        p = _lognormal_int(rng, w.prompt_median, w.prompt_sigma, n)
        g = rng.integers(0, w.gen_hi + 1, size=n)
        return np.minimum(w.max_len, p + g).astype(np.int64)
    if w.len_kind == "lognormal":
        return np.minimum(w.max_len, _lognormal_int(rng, w.len_median, w.len_sigma, n)).astype(np.int64)
    raise ValueError(w.len_kind)


@functools.lru_cache(maxsize=4)
def _zipf_cdf(vocab: int, s: float) -> np.ndarray:
    r = np.arange(1, vocab, dtype=np.float64)
    p = r ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def draw_ids(w: Workload, rng: np.random.Generator, count: int) -> np.ndarray:
    V = w.shape.vocab
    if w.id_kind == "uniform":
        return rng.integers(1, V, size=count).astype(np.int32)
    if w.id_kind == "zipf":
        cdf = _zipf_cdf(V, w.zipf_s)
        u = rng.random(count)
        rank = np.searchsorted(cdf, u, side="left") + 1
        return np.minimum(rank, V - 1).astype(np.int32)
    raise ValueError(w.id_kind)


class Batch:
    """A packed variable-length batch: ids of all sequences back to back.

    token_ids   int32[T]
    cu_seqlens  int32[n+1], cu_seqlens[0] = 0, cu_seqlens[n] = T
    arrival_seq int64[n]  arrival order of each in-flight job (a permutation)
    """

    def __init__(self, token_ids, cu_seqlens, arrival_seq):
        self.token_ids = np.ascontiguousarray(token_ids, dtype=np.int32)
        self.cu_seqlens = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.arrival_seq = np.ascontiguousarray(arrival_seq, dtype=np.int64)

    @property
    def n(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def total(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.cu_seqlens)

    @property
    def max_seqlen(self) -> int:
        return int(self.lengths.max()) if self.n else 0

    def seq(self, s: int) -> np.ndarray:
        return self.token_ids[self.cu_seqlens[s]:self.cu_seqlens[s + 1]]


def pack(seqs, arrival_seq=None) -> Batch:
    lens = np.array([len(s) for s in seqs], dtype=np.int64)
    cu = np.zeros(len(seqs) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    ids = np.concatenate([np.asarray(s, dtype=np.int32) for s in seqs]) if seqs else np.zeros(0, np.int32)
    if arrival_seq is None:
        arrival_seq = np.arange(len(seqs), dtype=np.int64)
    return Batch(ids, cu, arrival_seq)


def make_batch(w: Workload, seed: int | None = None) -> Batch:
    rng = np.random.Generator(np.random.PCG64(w.data_seed if seed is None else seed))
    lens = draw_lengths(w, rng)
    ids = draw_ids(w, rng, int(lens.sum()))
    cu = np.zeros(w.n_seqs + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    arrival = rng.permutation(w.n_seqs).astype(np.int64)
    return Batch(ids, cu, arrival)


class RoundStream:
    """In-flight sequences re-scored every round, each growing by one token per round.

    Sequence s owns a pre-drawn id stream of prompt_len + gen0 + rounds tokens.
    At round r its input is the first prompt_len + gen0 + r tokens of that
    stream; when that is longer than max_len, the first token is kept together
    with the most recent max_len - 1 tokens.
    """

    def __init__(self, w: Workload, seed: int | None = None):
        rng = np.random.Generator(np.random.PCG64(w.data_seed if seed is None else seed))
        n = w.n_seqs
        self.w = w
        self.prompt = _lognormal_int(rng, w.prompt_median, w.prompt_sigma, n)
        self.gen0 = rng.integers(0, w.gen_hi + 1, size=n).astype(np.int64)
        full = self.prompt + self.gen0 + w.rounds
        self.streams = [draw_ids(w, rng, int(f)) for f in full]
        self.arrival = rng.permutation(n).astype(np.int64)

    def lengths_at(self, r: int) -> np.ndarray:
        return self.prompt + self.gen0 + r

    def batch(self, r: int) -> Batch:
        L = self.w.max_len
        seqs = []
        for s, st in enumerate(self.streams):
            cur = int(self.prompt[s] + self.gen0[s] + r)
            x = st[:cur]
            if cur > L:
                x = np.concatenate([x[:1], x[cur - (L - 1):]])
            seqs.append(x)
        return pack(seqs, self.arrival)


class Requests:
    """Synthetic request stream (all arrays indexed by arrival order).

    arrival_t   float64[N] seconds, Poisson arrivals
    prompt      list of int32 arrays (prompt token ids)
    response    list of int32 arrays (the response the LLM would produce; its
                length is the true response length R)
    """

    def __init__(self, arrival_t, prompt, response):
        self.arrival_t = arrival_t
        self.prompt = prompt
        self.response = response

    def __len__(self):
        return len(self.arrival_t)


def make_requests(s: RequestStream, n: int | None = None, seed: int | None = None) -> Requests:
    rng = np.random.Generator(np.random.PCG64(s.data_seed if seed is None else seed))
    N = s.n_requests if n is None else n
    gaps = rng.exponential(1.0 / s.rate_per_s, size=N)
    arrival_t = np.cumsum(gaps)
    plen = _lognormal_int(rng, s.prompt_median, s.prompt_sigma, N)
    rlen = np.minimum(s.resp_cap, _lognormal_int(rng, s.resp_median, s.resp_sigma, N))
    V = s.shape.vocab
    prompt = [rng.integers(1, V, size=int(p)).astype(np.int32) for p in plen]
    response = [rng.integers(1, V, size=int(r)).astype(np.int32) for r in rlen]
    return Requests(arrival_t, prompt, response)


def make_policy_requests(st: PolicyStudy, batch_cap: int, rps_multiple: float, repetition: int) -> Requests:
    """One run of the policy study: the study's fixed request set, shuffled for this repetition,
    with Gamma(shape, scale) request intervals at rps_multiple x batch_cap / (mean(R) x step_cost)
    requests per second."""
    base = np.random.Generator(np.random.PCG64(st.data_seed))
    N = st.n_requests
    plen = _lognormal_int(base, st.prompt_median, st.prompt_sigma, N)
    rlen = np.minimum(st.resp_cap, _lognormal_int(base, st.resp_median, st.resp_sigma, N))
    prompt = [base.integers(1, st.vocab, size=int(p)).astype(np.int32) for p in plen]
    response = [base.integers(1, st.vocab, size=int(r)).astype(np.int32) for r in rlen]
    rng = np.random.Generator(np.random.PCG64([st.data_seed, repetition, batch_cap, int(round(rps_multiple * 1000))]))
    order = rng.permutation(N)
    rate = rps_multiple * batch_cap / (float(rlen.mean()) * st.step_cost_s)
    gaps = rng.gamma(st.gamma_shape, 1.0 / (rate * st.gamma_shape), size=N)
    return Requests(np.cumsum(gaps), [prompt[i] for i in order], [response[i] for i in order])


_M64 = (1 << 64) - 1


def _splitmix64(x: np.ndarray) -> np.ndarray:
    """splitmix64 finaliser (Steele, Lea, Flood 2014) on uint64 arrays."""
    with np.errstate(over="ignore"):
        z = x + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def accuracy_model_keys(seed: int, jobs, generated, remaining, mae: float) -> np.ndarray:
    """Stand-in for a trained predictor's outputs (float32): remaining + Laplace(0, mae) noise.

    The noise of job j after g generated tokens is a fixed function of (seed, j, g) (counter-based,
    so it does not depend on when or how often the job is re-scored): u = uniform (0, 1) from
    splitmix64, noise = -mae * sign(u - 1/2) * ln(1 - 2 |u - 1/2|). A Laplace(0, b) variable has
    mean absolute value b."""
    j = np.asarray(jobs, dtype=np.uint64)
    g = np.asarray(generated, dtype=np.uint64)
    with np.errstate(over="ignore"):
        x = _splitmix64(_splitmix64(np.uint64(seed) ^ (j * np.uint64(0xD1B54A32D192ED03))) ^ g)
    u = ((x >> np.uint64(11)).astype(np.float64) + 0.5) * 2.0 ** -53
    d = u - 0.5
    noise = -mae * np.sign(d) * np.log1p(-2.0 * np.abs(d))
    return (np.asarray(remaining, dtype=np.float64) + noise).astype(np.float32)


def head_is_linear(shape: EncoderShape) -> bool:
    return shape.head_hidden == 0


def pooling_is_cls(shape: EncoderShape) -> bool:
    return shape.pooling == POOL_CLS
