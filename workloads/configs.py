"""Named encoder shapes and workload recipes.

Pure data: sizes, distribution parameters and seeds. Nothing here computes
any part of the predictor or the scheduler.

The predictor is a BERT-style bidirectional encoder (the paper builds it on
BGE, a BERT-family model, Sec. 3.1) with a pooled regression head (Sec. 3.2
uses the CLS vector; Sec. 4.2 uses mean pooling). The shapes below are the
five workloads this implementation is measured and checked on.
"""
from __future__ import annotations

from dataclasses import dataclass, field

POOL_CLS = 0
POOL_MEAN = 1
ACT_RELU = 0
ACT_IDENTITY = 1


@dataclass(frozen=True)
class EncoderShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab: int
    max_pos: int
    pooling: int            # POOL_CLS or POOL_MEAN
    head_hidden: int        # width of the head's hidden layers; 0: one linear layer d->1
    fp32_master: bool       # True: weights drawn and kept in fp32 (device gets bf16 copies)
    ln_eps: float = 1e-12
    out_scale: float = 100.0
    out_shift: float = 250.0
    head_layers: int = 0    # FC layers of the head; 0: 1 when head_hidden == 0, else 2
    head_act: int = ACT_RELU  # activation between the head's layers

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads

    @property
    def n_head_layers(self) -> int:
        if self.head_layers:
            return self.head_layers
        return 2 if self.head_hidden else 1


TINY = EncoderShape("tiny", 2, 128, 4, 512, 1000, 128, POOL_CLS, 0, True)
BERT_BASE = EncoderShape("bert_base", 12, 768, 12, 3072, 30522, 512, POOL_CLS, 256, False)
XLMR_LARGE = EncoderShape("xlmr_large", 24, 1024, 16, 4096, 250002, 2048, POOL_MEAN, 0, False)
# The paper's predictor heads: eight FC layers of width 1024 with ReLU on mean pooling (Sec. 4.2),
# and eight linear layers on the CLS vector (Sec. 3.2, hidden width not stated: 1024 taken);
# tiny versions of both for full-batch parity.
BERT_BASE_HEAD8 = EncoderShape("bert_base_head8", 12, 768, 12, 3072, 30522, 512, POOL_MEAN, 1024, False,
                               head_layers=8)
TINY_HEAD8 = EncoderShape("tiny_head8", 2, 128, 4, 512, 1000, 128, POOL_MEAN, 64, True, head_layers=8)
TINY_CLS_LIN8 = EncoderShape("tiny_cls_lin8", 2, 128, 4, 512, 1000, 128, POOL_CLS, 64, True, head_layers=8,
                             head_act=ACT_IDENTITY)


@dataclass(frozen=True)
class Workload:
    """One synthetic workload. Lengths are drawn per sequence.

    len_kind:
      "uniform"       len ~ U{len_lo..len_hi}
      "prompt+gen"    len = min(max_len, lognormal(prompt_median, prompt_sigma) + U{0..gen_hi})
      "lognormal"     len = min(max_len, lognormal(len_median, len_sigma))
    id_kind:
      "uniform"       id ~ U{1..vocab-1}
      "zipf"          P(rank r) proportional to r^-zipf_s over ranks 1..vocab-1, rank r -> id r
    """
    name: str
    shape: EncoderShape
    n_seqs: int
    batch_cap: int
    len_kind: str
    id_kind: str = "uniform"
    len_lo: int = 0
    len_hi: int = 0
    prompt_median: float = 200.0
    prompt_sigma: float = 0.8
    gen_hi: int = 0
    len_median: float = 0.0
    len_sigma: float = 0.0
    max_len: int = 0
    zipf_s: float = 1.1
    rounds: int = 1
    data_seed: int = 0
    weight_seed: int = 0


W_TINY = Workload("tiny_b8", TINY, n_seqs=8, batch_cap=4, len_kind="uniform",
                  len_lo=16, len_hi=64, data_seed=1, weight_seed=1001)
W_BERT_B64 = Workload("bert_base_b64", BERT_BASE, n_seqs=64, batch_cap=32, len_kind="prompt+gen",
                      prompt_median=200.0, prompt_sigma=0.8, gen_hi=300, max_len=512,
                      data_seed=2, weight_seed=1002)
W_BERT_B256_ROUNDS = Workload("bert_base_b256_x100", BERT_BASE, n_seqs=256, batch_cap=128,
                              len_kind="prompt+gen", prompt_median=200.0, prompt_sigma=0.8,
                              gen_hi=300, max_len=512, rounds=100, data_seed=3, weight_seed=1002)
W_TINY_HEAD8 = Workload("tiny_head8_b8", TINY_HEAD8, n_seqs=8, batch_cap=4, len_kind="uniform",
                        len_lo=16, len_hi=64, data_seed=1, weight_seed=1005)
W_TINY_CLS_LIN8 = Workload("tiny_cls_lin8_b8", TINY_CLS_LIN8, n_seqs=8, batch_cap=4, len_kind="uniform",
                           len_lo=16, len_hi=64, data_seed=1, weight_seed=1007)
W_BERT_B64_HEAD8 = Workload("bert_base_head8_b64", BERT_BASE_HEAD8, n_seqs=64, batch_cap=32,
                            len_kind="prompt+gen", prompt_median=200.0, prompt_sigma=0.8, gen_hi=300,
                            max_len=512, data_seed=2, weight_seed=1006)
W_XLMR_B128 = Workload("xlmr_large_b128", XLMR_LARGE, n_seqs=128, batch_cap=64, len_kind="lognormal",
                       id_kind="zipf", len_median=600.0, len_sigma=0.9, max_len=2048,
                       data_seed=4, weight_seed=1004)


@dataclass(frozen=True)
class RequestStream:
    """Synthetic request stream for the one-node ISRTF round simulation."""
    name: str
    shape: EncoderShape
    n_requests: int = 4096
    rate_per_s: float = 20.0
    prompt_median: float = 200.0
    prompt_sigma: float = 0.8
    resp_median: float = 250.0
    resp_sigma: float = 1.0
    resp_cap: int = 2048
    window: int = 50            # tokens per scheduling iteration (Sec. 3.3, Sec. 4.1)
    step_cost_s: float = 0.008  # fixed synthetic LLM cost per decode step of a batch
    batch_cap: int = 64
    data_seed: int = 5
    weight_seed: int = 1002


S_ISRTF = RequestStream("isrtf_sim_4096", BERT_BASE)


@dataclass(frozen=True)
class PolicyStudy:
    """Synthetic analogue of the paper's scheduler comparison (Sec. 6.1-6.3, Fig. 5 and 6).

    The paper averages the JCT of 200 LMSYS prompts with Gamma-distributed request intervals,
    shuffling the same prompt set for each of three repetitions, at request rates that are
    multiples of (1000 / average latency in ms) x batch size, for batch sizes 1, 2 and 4.
    Here the prompts and responses are synthetic (lengths as in the ISRTF stream), the LLM is a
    fixed cost per decode step of the batch, and its average latency is mean(R) x step_cost.
    The Gamma shape is the paper's fitted 0.73; the scale follows from the target rate.
    Stand-in predictor ("accuracy model"): the true remaining length plus Laplace noise whose
    mean absolute error is the paper's final predictor MAE (Sec. 4.2), seeded per (job, tokens
    generated).
    """
    name: str = "policy_study_200"
    n_requests: int = 200
    batch_caps: tuple = (1, 2, 4)
    rps_multiples: tuple = (1.0, 3.0, 5.0)
    repetitions: int = 3
    gamma_shape: float = 0.73
    prompt_median: float = 200.0
    prompt_sigma: float = 0.8
    resp_median: float = 250.0
    resp_sigma: float = 1.0
    resp_cap: int = 2048
    vocab: int = 30522
    window: int = 50
    step_cost_s: float = 0.008
    accuracy_mae: float = 19.923    # tokens; the final predictor's MAE (Sec. 4.2)
    aging: float = 10.0             # tokens per second of waiting, for the starvation-control runs
    prefill_cost_s: float = 0.0001  # seconds per re-prefilled token, for the preemption-cost runs
    data_seed: int = 7


POLICY_STUDY = PolicyStudy()

WORKLOADS = {w.name: w for w in (W_TINY, W_BERT_B64, W_BERT_B256_ROUNDS, W_XLMR_B128, W_TINY_HEAD8,
                                  W_TINY_CLS_LIN8, W_BERT_B64_HEAD8)}
SHAPES = {s.name: s for s in (TINY, BERT_BASE, XLMR_LARGE, TINY_HEAD8, TINY_CLS_LIN8, BERT_BASE_HEAD8)}
