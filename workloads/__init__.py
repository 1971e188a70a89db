"""Seeded synthetic workloads for the RKSC verify pass.

This module only describes shapes and draws random inputs; it holds none of
the method's arithmetic. Both the HIP path's tests/benchmark and the CPU oracle
are fed from it.

Recipe (one child seed per tensor, derived from the base seed and the tensor's
name):
  * weight matrices and the embedding table: N(0, init_std^2), then rounded to
    the model dtype (bf16 by round-to-nearest-even, as torch's cast does);
  * RMSNorm gains: exactly 1;
  * lm_head: N(0, (lm_head_scale * init_std)^2);
  * branch tokens: uniform over [0, vocab);
  * synthetic prefix K/V: N(0, (init_std * sqrt(d_model))^2), the magnitude a
    random-init projection of a unit-RMS row produces (RoPE is a rotation, so a
    Gaussian also stands in for post-RoPE keys).
"""
from __future__ import annotations

import dataclasses
import zlib
from dataclasses import dataclass
from typing import Optional

import torch

__all__ = [
    "ModelShape", "Workload", "WORKLOADS", "get", "ModelWeights", "PrefixKV",
    "make_model", "make_prefix_kv", "make_tokens", "make_hidden",
]


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    dtype: str                 # "f32" or "bf16": storage type of matrices and KV
    lm_head_scale: float       # lm_head std = lm_head_scale * init_std
    rms_eps: float = 1e-6
    rope_base: float = 1e4
    init_std: float = 0.02

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def params_per_layer(self) -> int:
        d, hd = self.d_model, self.head_dim
        return (d * self.qkv_rows + d * self.n_heads * hd + 3 * d * self.d_ff)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    n_branches: int
    prefix_len: int
    branch_len: int
    tau: float
    patience: int
    alpha: float
    share_threshold: Optional[float] = None   # ASKS gate S >= threshold
    description: str = ""

    def with_(self, **kw) -> "Workload":
        model_kw = {k: kw.pop(k) for k in list(kw) if k in ModelShape.__dataclass_fields__}
        model = dataclasses.replace(self.model, **model_kw) if model_kw else self.model
        return dataclasses.replace(self, model=model, **kw)


# lm_head scales for the 7B-class shapes: with unit-RMS normalised hidden rows,
# logits are i.i.d. N(0, sigma^2) with sigma = init_std*scale*sqrt(d_model); the
# scale is chosen so that the mean softmax entropy of V such logits is about
# 2 nats (workloads/calibrate_lm_head.py reproduces the numbers).
_TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                   d_ff=688, vocab=4096, dtype="f32", lm_head_scale=8.0)
_L7B = ModelShape(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                  d_ff=14336, vocab=128256, dtype="bf16", lm_head_scale=5.2)
_Q7B = ModelShape(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                  d_ff=18944, vocab=152064, dtype="bf16", lm_head_scale=5.5)
_B10 = ModelShape(n_layers=48, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                  d_ff=14336, vocab=256000, dtype="bf16", lm_head_scale=5.5)

WORKLOADS = {
    "tiny": Workload("tiny", _TINY, n_branches=4, prefix_len=64, branch_len=16,
                     tau=0.05, patience=1, alpha=0.5,
                     description="tiny fp32 decoder, 4 branches over a 64-token prefix"),
    # The tiny model with 8 layers, so that exits can happen before the last layer.
    "tiny_deep": Workload("tiny_deep", dataclasses.replace(_TINY, n_layers=8),
                          n_branches=4, prefix_len=64, branch_len=16,
                          tau=0.05, patience=1, alpha=0.5,
                          description="tiny fp32 decoder with 8 layers"),
    "7b_single": Workload("7b_single", _L7B, n_branches=1, prefix_len=1024, branch_len=128,
                          tau=0.02, patience=2, alpha=0.1,
                          description="7B shape, 1 branch, 1024-token prefix, 128 verify tokens"),
    "7b_tot": Workload("7b_tot", _L7B, n_branches=16, prefix_len=2048, branch_len=256,
                       tau=0.02, patience=2, alpha=0.1, share_threshold=0.9,
                       description="7B shape tree of thoughts, 16 leaves, 2048-token prefix, 256-token steps"),
    "7b_large_vocab": Workload("7b_large_vocab", _Q7B, n_branches=8, prefix_len=4096, branch_len=128,
                               tau=0.02, patience=2, alpha=0.1,
                               description="28-layer 28Q/4KV shape, vocab 152064, 8 branches, 4096-token prefix"),
    "10b_long": Workload("10b_long", _B10, n_branches=32, prefix_len=16384, branch_len=256,
                         tau=0.02, patience=3, alpha=0.1,
                         description="48-layer 10B shape, vocab 256000, 32 branches, 16384-token prefix"),
    # Supplemental points (not headline configs).
    # One verify token per branch over the long prefix: the decode regime, in
    # which the shared-prefix attention reads 67 MB of K/V per layer for only
    # G * B = 128 query rows per KV head and is HBM-bound.
    "10b_decode": Workload("10b_decode", _B10, n_branches=32, prefix_len=16384, branch_len=1,
                           tau=0.02, patience=3, alpha=0.1,
                           description="48-layer 10B shape, 32 branches x 1 token over a 16384-token prefix"),
    # The paper's own verify shape on the large-vocab model: 8 branches x 128
    # tokens over a 1024-token prefix.
    "7b_paper_verify": Workload("7b_paper_verify", _Q7B, n_branches=8, prefix_len=1024, branch_len=128,
                                tau=0.02, patience=2, alpha=0.1,
                                description="28-layer 28Q/4KV shape, 8 branches x 128 tokens, 1024-token prefix"),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def _child_seed(seed: int, name: str) -> int:
    return (int(seed) * 1_000_003 + zlib.crc32(name.encode())) & 0x7FFF_FFFF_FFFF


def _gen(seed: int, name: str, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_child_seed(seed, name))
    return g


def _normal(shape, std, seed, name, device, dtype):
    g = _gen(seed, name, device)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    t.mul_(std)
    return t.to(dtype) if dtype != torch.float32 else t


@dataclass
class ModelWeights:
    shape: ModelShape
    embed: torch.Tensor                 # [V, d]
    layers: list                        # list of dicts, see make_model
    final_norm: torch.Tensor            # [d] fp32
    lm_head: torch.Tensor               # [V, d]

    def to(self, device) -> "ModelWeights":
        return ModelWeights(self.shape, self.embed.to(device),
                            [{k: v.to(device) for k, v in lw.items()} for lw in self.layers],
                            self.final_norm.to(device), self.lm_head.to(device))


@dataclass
class PrefixKV:
    k: torch.Tensor     # [L, Hkv, n, hd] post-RoPE keys at positions 0..n-1
    v: torch.Tensor     # [L, Hkv, n, hd]

    @property
    def n_prefix(self) -> int:
        return int(self.k.shape[2])


def make_model(shape: ModelShape, seed: int = 42, device="cpu", n_layers: Optional[int] = None) -> ModelWeights:
    """Random-init decoder weights of the given shape (optionally only the first n_layers)."""
    dt = shape.torch_dtype
    d, F, V = shape.d_model, shape.d_ff, shape.vocab
    std = shape.init_std
    L = shape.n_layers if n_layers is None else n_layers
    layers = []
    for l in range(L):
        layers.append({
            "attn_norm": torch.ones(d, device=device, dtype=torch.float32),
            "w_qkv": _normal((shape.qkv_rows, d), std, seed, f"layer{l}.w_qkv", device, dt),
            "w_o": _normal((d, shape.n_heads * shape.head_dim), std, seed, f"layer{l}.w_o", device, dt),
            "ffn_norm": torch.ones(d, device=device, dtype=torch.float32),
            "w_gate_up": _normal((2 * F, d), std, seed, f"layer{l}.w_gate_up", device, dt),
            "w_down": _normal((d, F), std, seed, f"layer{l}.w_down", device, dt),
        })
    return ModelWeights(
        shape=shape,
        embed=_normal((V, d), std, seed, "embed", device, dt),
        layers=layers,
        final_norm=torch.ones(d, device=device, dtype=torch.float32),
        lm_head=_normal((V, d), std * shape.lm_head_scale, seed, "lm_head", device, dt),
    )


def make_prefix_kv(shape: ModelShape, n_prefix: int, seed: int = 42, device="cpu",
                   n_layers: Optional[int] = None) -> PrefixKV:
    """Synthetic post-RoPE prefix K/V of the magnitude a random-init model produces."""
    L = shape.n_layers if n_layers is None else n_layers
    std = shape.init_std * shape.d_model ** 0.5
    sz = (L, shape.n_kv_heads, n_prefix, shape.head_dim)
    return PrefixKV(_normal(sz, std, seed, "prefix.k", device, shape.torch_dtype),
                    _normal(sz, std, seed, "prefix.v", device, shape.torch_dtype))


def make_tokens(n: int, vocab: int, seed: int = 42, name: str = "branch_tokens", device="cpu",
                shape=None) -> torch.Tensor:
    """Uniform token ids over [0, vocab) as int32."""
    g = _gen(seed, name, device)
    shp = (n,) if shape is None else tuple(shape)
    return torch.randint(0, vocab, shp, generator=g, device=device, dtype=torch.int64).to(torch.int32)


def make_hidden(L: int, B: int, d: int, seed: int = 42, device="cpu", scale: float = 1.0) -> torch.Tensor:
    """Random fp32 per-layer hidden rows [L, B, d] for the similarity kernel."""
    return _normal((L, B, d), scale, seed, "asks.hidden", device, torch.float32)
