"""Seeded synthetic inputs shared by the oracle and the GPU path (data only)."""
from .configs import (ACT_IDENTITY, ACT_RELU, BERT_BASE, BERT_BASE_HEAD8, POLICY_STUDY, POOL_CLS, POOL_MEAN,
                      S_ISRTF, SHAPES,
                      TINY, TINY_CLS_LIN8, TINY_HEAD8, WORKLOADS, W_BERT_B64, W_BERT_B64_HEAD8,
                      W_BERT_B256_ROUNDS, W_TINY, W_TINY_CLS_LIN8, W_TINY_HEAD8, W_XLMR_B128, XLMR_LARGE,
                      EncoderShape, PolicyStudy, RequestStream, Workload)
from .gen import (BF16_TENSORS, Batch, Requests, RoundStream, Weights, accuracy_model_keys, bf16_bits_to_f32,
                  f32_to_bf16_bits, make_batch, make_policy_requests, make_requests, make_weights, pack)
