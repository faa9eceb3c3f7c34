"""Seeded synthetic inputs shared by the oracle and the GPU path (data only)."""
from .configs import (BERT_BASE, POOL_CLS, POOL_MEAN, S_ISRTF, SHAPES, TINY, WORKLOADS,
                      W_BERT_B64, W_BERT_B256_ROUNDS, W_TINY, W_XLMR_B128, XLMR_LARGE,
                      EncoderShape, RequestStream, Workload)
from .gen import (BF16_TENSORS, Batch, Requests, RoundStream, Weights, bf16_bits_to_f32,
                  f32_to_bf16_bits, make_batch, make_requests, make_weights, pack)
