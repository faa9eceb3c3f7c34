"""Predictor checkpoints: round trip, and every mismatch rejected on save and on load."""
import numpy as np
import pytest

from paper_2505_09142_amd.checkpoint import PredictorConfig, load_predictor, save_predictor
from workloads import TINY, TINY_CLS_LIN8, TINY_HEAD8, make_weights


def _same(a, b):
    if isinstance(a, list):
        return len(a) == len(b) and all(_same(x, y) for x, y in zip(a, b))
    return a.dtype == b.dtype and a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("shape", [TINY, TINY_HEAD8, TINY_CLS_LIN8])
def test_round_trip(tmp_path, shape):
    W = make_weights(shape, 7)
    p = str(tmp_path / "pred.safetensors")
    save_predictor(p, shape, W.device)
    cfg, t = load_predictor(p)
    assert cfg == PredictorConfig.of(shape) and cfg.n_head_layers == shape.n_head_layers
    assert set(t) == set(W.device)
    for k in t:
        assert _same(t[k], W.device[k]), k


def test_rejects_mismatches(tmp_path):
    W = make_weights(TINY_HEAD8, 3)
    p = str(tmp_path / "x.safetensors")
    bad = dict(W.device)
    bad["w_o"] = list(bad["w_o"])
    bad["w_o"][1] = bad["w_o"][1][:, :64]
    with pytest.raises(ValueError, match="shape"):
        save_predictor(p, TINY_HEAD8, bad)
    bad = dict(W.device)
    bad["w_1"] = [x.astype(np.float32) for x in bad["w_1"]]  # not bf16 bit patterns
    with pytest.raises(ValueError, match="bf16"):
        save_predictor(p, TINY_HEAD8, bad)
    bad = dict(W.device)
    del bad["head_mid_b"]
    with pytest.raises(ValueError, match="missing"):
        save_predictor(p, TINY_HEAD8, bad)
    # a file whose config disagrees with its tensors, and a file of another format
    import torch
    from safetensors.torch import save_file
    save_predictor(p, TINY_HEAD8, W.device)
    from safetensors import safe_open
    with safe_open(p, framework="pt") as f:
        tensors = {k: f.get_tensor(k) for k in f.keys()}
        meta = dict(f.metadata())
    q = str(tmp_path / "y.safetensors")
    tensors.pop("head.mid.0.w")
    save_file(tensors, q, metadata=meta)
    with pytest.raises(ValueError, match="missing"):
        load_predictor(q)
    save_file({"a": torch.zeros(2)}, q, metadata={"format": "other"})
    with pytest.raises(ValueError, match="not an"):
        load_predictor(q)
