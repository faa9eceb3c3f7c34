"""fp64 CPU oracle of the ELIS predictor, ISRTF selection and scheduling loop.

TEST INFRASTRUCTURE ONLY. Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import anything from this package. The GPU
path never does; it shares no code with the oracle (only the seeded input
generators in ``workloads`` serve both).

Parity pins (what fixes each function independently of itself) are in
tests/test_oracle_*.py. Every function here has at least one pin.
"""
from .encoder import (POOL_CLS, POOL_MEAN, embed, encode_sequence, encoder_layer, gelu,
                      layer_norm, oracle_forward, pool, regression_head, self_attention,
                      softmax_rows)
from .select import oracle_order, oracle_select
from .simulate import POLICIES, SimResult, aged_keys, job_input, simulate
