"""Predictor checkpoints: one safetensors file per predictor.

The file holds the encoder and head parameters in the layout libelis reads
(include/elis.h), plus the shape in the metadata, so a trained BGE/BERT-style
predictor can be converted once and loaded into HBM directly:

    metadata  "format": "elis-predictor", "version": "1",
              "config": JSON of PredictorConfig's fields
    tensors   word [vocab, d] BF16, pos [max_pos, d] BF16, type0 / emb_ln_g / emb_ln_b [d] F32,
              layers.{l}.w_qkv [3d, d] BF16 (rows: query | key | value, head h owns rows
              h*dh..(h+1)*dh-1 of each block), layers.{l}.w_o [d, d], layers.{l}.w_1 [F, d],
              layers.{l}.w_2 [d, F] BF16; layers.{l}.b_qkv / b_o / b_1 / b_2 and
              ln1_g / ln1_b / ln2_g / ln2_b F32;
              head.w1 [hidden, d], head.b1 [hidden], head.mid.{i}.w [hidden, hidden],
              head.mid.{i}.b [hidden], head.w2 [1, hidden or d], head.b2 [1], all F32.

Matrices are [out, in]. Loading validates every name, shape and dtype against the
config and raises ValueError on any mismatch.
"""
from __future__ import annotations

import dataclasses
import json

import numpy as np

FORMAT = "elis-predictor"
VERSION = "1"

POOL_CLS, POOL_MEAN = 0, 1
ACT_RELU, ACT_IDENTITY = 0, 1


@dataclasses.dataclass(frozen=True)
class PredictorConfig:
    """Encoder + head shape (the fields of elis_config)."""
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab: int
    max_pos: int
    pooling: int = POOL_CLS
    head_hidden: int = 0
    head_layers: int = 0        # 0: 1 when head_hidden == 0, else 2
    head_act: int = ACT_RELU
    ln_eps: float = 1e-12
    out_scale: float = 1.0
    out_shift: float = 0.0

    @property
    def n_head_layers(self) -> int:
        if self.head_layers:
            return self.head_layers
        return 2 if self.head_hidden else 1

    @classmethod
    def of(cls, shape) -> "PredictorConfig":
        """From any object carrying the same attribute names (e.g. a workload shape)."""
        return cls(**{f.name: getattr(shape, f.name) for f in dataclasses.fields(cls)})


_LAYER_BF16 = ("w_qkv", "w_o", "w_1", "w_2")
_LAYER_F32 = ("b_qkv", "b_o", "b_1", "b_2", "ln1_g", "ln1_b", "ln2_g", "ln2_b")


def _expected(cfg: PredictorConfig) -> dict:
    """name -> (shape, is_bf16) of every tensor the config needs."""
    d, F, L, hh, nh = cfg.d_model, cfg.d_ff, cfg.n_layers, cfg.head_hidden, cfg.n_head_layers
    e = {"word": ((cfg.vocab, d), True), "pos": ((cfg.max_pos, d), True), "type0": ((d,), False),
         "emb_ln_g": ((d,), False), "emb_ln_b": ((d,), False)}
    layer = {"w_qkv": (3 * d, d), "w_o": (d, d), "w_1": (F, d), "w_2": (d, F), "b_qkv": (3 * d,), "b_o": (d,),
             "b_1": (F,), "b_2": (d,), "ln1_g": (d,), "ln1_b": (d,), "ln2_g": (d,), "ln2_b": (d,)}
    for l in range(L):
        for k, shp in layer.items():
            e[f"layers.{l}.{k}"] = (shp, k in _LAYER_BF16)
    if nh >= 2:
        e["head.w1"] = ((hh, d), False)
        e["head.b1"] = ((hh,), False)
        for i in range(nh - 2):
            e[f"head.mid.{i}.w"] = ((hh, hh), False)
            e[f"head.mid.{i}.b"] = ((hh,), False)
    e["head.w2"] = ((1, hh if nh >= 2 else d), False)
    e["head.b2"] = ((1,), False)
    return e


def _flatten(tensors: dict) -> dict:
    """The package's in-memory layout (per-layer lists, head_* keys) -> file names."""
    out = {}
    for k, v in tensors.items():
        if k in _LAYER_BF16 + _LAYER_F32:
            for l, x in enumerate(v):
                out[f"layers.{l}.{k}"] = x
        elif k == "head_mid_w":
            for i, x in enumerate(v):
                out[f"head.mid.{i}.w"] = x
        elif k == "head_mid_b":
            for i, x in enumerate(v):
                out[f"head.mid.{i}.b"] = x
        elif k.startswith("head_"):
            out["head." + k[len("head_"):]] = v
        else:
            out[k] = v
    return out


def _nest(flat: dict, cfg: PredictorConfig) -> dict:
    """File names -> the package's in-memory layout (what DeviceWeights takes)."""
    t = {k: flat[k] for k in ("word", "pos", "type0", "emb_ln_g", "emb_ln_b")}
    for k in _LAYER_BF16 + _LAYER_F32:
        t[k] = [flat[f"layers.{l}.{k}"] for l in range(cfg.n_layers)]
    nh = cfg.n_head_layers
    if nh >= 2:
        t["head_w1"], t["head_b1"] = flat["head.w1"], flat["head.b1"]
    if nh > 2:
        t["head_mid_w"] = [flat[f"head.mid.{i}.w"] for i in range(nh - 2)]
        t["head_mid_b"] = [flat[f"head.mid.{i}.b"] for i in range(nh - 2)]
    t["head_w2"], t["head_b2"] = flat["head.w2"], flat["head.b2"]
    return t


def save_predictor(path: str, config, tensors: dict) -> None:
    """Write a predictor checkpoint. `tensors` is in the package's in-memory layout: bf16 bit
    patterns (uint16) for the embedding tables and the layer matrices, float32 for the rest,
    per-layer lists (as DeviceWeights takes them)."""
    import torch
    from safetensors.torch import save_file
    cfg = config if isinstance(config, PredictorConfig) else PredictorConfig.of(config)
    flat = _flatten(tensors)
    exp = _expected(cfg)
    if set(flat) != set(exp):
        raise ValueError(f"tensor set does not match the config: missing {sorted(set(exp) - set(flat))}, "
                         f"unexpected {sorted(set(flat) - set(exp))}")
    out = {}
    for k, (shp, bf16) in exp.items():
        a = np.ascontiguousarray(flat[k])
        if tuple(a.shape) != shp:
            raise ValueError(f"{k}: shape {a.shape}, expected {shp}")
        if bf16:
            if a.dtype != np.uint16:
                raise ValueError(f"{k}: expected bf16 bit patterns (uint16), got {a.dtype}")
            out[k] = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
        else:
            out[k] = torch.from_numpy(np.asarray(a, dtype=np.float32))
    meta = {"format": FORMAT, "version": VERSION, "config": json.dumps(dataclasses.asdict(cfg))}
    save_file(out, path, metadata=meta)


def load_predictor(path: str) -> tuple[PredictorConfig, dict]:
    """Read and validate a predictor checkpoint; returns (config, tensors in the in-memory layout)."""
    import torch
    from safetensors import safe_open
    with safe_open(path, framework="pt") as f:
        meta = f.metadata() or {}
        if meta.get("format") != FORMAT or meta.get("version") != VERSION:
            raise ValueError(f"{path}: not an {FORMAT} v{VERSION} checkpoint (metadata {meta})")
        cfg = PredictorConfig(**json.loads(meta["config"]))
        exp = _expected(cfg)
        keys = set(f.keys())
        if keys != set(exp):
            raise ValueError(f"{path}: missing {sorted(set(exp) - keys)}, unexpected {sorted(keys - set(exp))}")
        flat = {}
        for k, (shp, bf16) in exp.items():
            t = f.get_tensor(k)
            if tuple(t.shape) != shp:
                raise ValueError(f"{path}: {k} has shape {tuple(t.shape)}, expected {shp}")
            if bf16:
                if t.dtype != torch.bfloat16:
                    raise ValueError(f"{path}: {k} is {t.dtype}, expected bfloat16")
                flat[k] = t.view(torch.int16).numpy().view(np.uint16).copy()
            else:
                if t.dtype != torch.float32:
                    raise ValueError(f"{path}: {k} is {t.dtype}, expected float32")
                flat[k] = t.numpy().copy()
    return cfg, _nest(flat, cfg)
