"""Seeded synthetic inputs for the verify step.

This module is the ONE piece of code shared by the HIP path's tests/bench and
the oracle's tests.  It only *creates inputs*: model weights, cached-context
KV values, token streams, context lengths and prior trajectories.  It holds
none of the decoder's arithmetic (no norm, projection, attention, softmax,
argmax or acceptance).

Random values come from a counter-based integer hash evaluated with torch
integer ops, so the same call gives bit-identical results on the CPU and on a
GPU: element ``i`` of stream ``s`` is a pure function of ``(seed, s, i)``.
The hash is Chris Wellons' ``lowbias32`` finaliser (published in his
"hash-prospector" notes), applied twice with a per-stream key.

Approximately normal values are the centred sum of the four bytes of one hash
word (an Irwin-Hall sum of four discrete uniforms, std sqrt(4*(256^2-1)/12)),
scaled to the requested std in fp32 and rounded to bf16 by torch's
round-to-nearest-even conversion.  Both the fp32 multiply and the conversion
are correctly rounded IEEE operations, so CPU and GPU agree bit for bit.

Workload shapes follow the paper's setting: multi-turn agent trajectories with
contexts of 10K-100K tokens (System Design, Overview), recurring code and
tool-call patterns (Evaluation, SuffixDecoding), several rollouts per prompt
that share a prompt prefix (System Design, Overview) and long-tailed
trajectory lengths (Background, rollout bottlenecks).  The paper's own SWE
dataset and Qwen3-32B weights are not available; these seeded inputs stand in
for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Sequence, Tuple

import numpy as np
import torch

# --------------------------------------------------------------------------
# model shapes
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    page_size: int = 16
    max_k: int = 15

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_dim(self) -> int:
        return self.q_dim + 2 * self.kv_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.kv_dim * 2

    def layer_params(self) -> int:
        d, F = self.d_model, self.ffn_dim
        return self.qkv_dim * d + d * self.q_dim + 3 * F * d

    def streamed_weight_bytes(self) -> int:
        """bf16 bytes of every matrix one verify step reads (embedding excluded:
        only T of its rows are gathered)."""
        return 2 * (self.n_layers * self.layer_params() + self.vocab * self.d_model)


# 2 layers, d 256, 4 q / 2 kv heads, head_dim 64, FFN 1024, vocab 4096.
TINY = ModelConfig(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                   ffn_dim=1024, vocab=4096)
# 36 layers, d 4096, 32 q / 8 kv heads, head_dim 128, FFN 12288, vocab 151936.
LARGE = ModelConfig(n_layers=36, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                    ffn_dim=12288, vocab=151936)


def reduced(cfg: ModelConfig, n_layers: int, vocab: int | None = None) -> ModelConfig:
    """Same layer shape with fewer layers (and optionally a smaller vocab)."""
    return dataclasses.replace(cfg, n_layers=n_layers, vocab=vocab or cfg.vocab)


# --------------------------------------------------------------------------
# counter-based hash (lowbias32) in torch integer ops
# --------------------------------------------------------------------------

_M32 = 0xFFFFFFFF
_NORM_DIV = math.sqrt(4.0 * (256.0 * 256.0 - 1.0) / 12.0)  # std of the byte sum


def _mul32_py(x: int, c: int) -> int:
    return (x * c) & _M32


def _lowbias32_py(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = _mul32_py(x, 0x7FEB352D)
    x ^= x >> 15
    x = _mul32_py(x, 0x846CA68B)
    x ^= x >> 16
    return x


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    # (x*c) mod 2^32 without int64 overflow: split c into 16-bit halves.
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def _lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def stream_key(*parts: int) -> Tuple[int, int]:
    """Two 32-bit keys for a stream named by a tuple of small integers."""
    k = 0x2545F491
    for p in parts:
        k = _lowbias32_py(k ^ _lowbias32_py((p * 0x9E3779B1 + 0x7F4A7C15) & _M32))
    return k, _lowbias32_py(k ^ 0xA511E9B3)


def hash_words(key: Tuple[int, int], idx: torch.Tensor) -> torch.Tensor:
    """32-bit hash word (as int64) for each int64 counter in ``idx`` (< 2^32)."""
    k1, k2 = key
    u = _lowbias32((idx ^ k1) & _M32)
    return _lowbias32(u ^ k2)


_CHUNK = 1 << 25


def normalish(key: Tuple[int, int], numel: int, std: float, device="cpu",
              offset: int = 0) -> torch.Tensor:
    """bf16 values, mean 0 and the given std, for counters offset..offset+numel-1."""
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    scale = torch.tensor(std / _NORM_DIV, dtype=torch.float32, device=device)
    for s in range(0, numel, _CHUNK):
        e = min(numel, s + _CHUNK)
        idx = torch.arange(offset + s, offset + e, dtype=torch.int64, device=device)
        u = hash_words(key, idx)
        b = (u & 255) + ((u >> 8) & 255) + ((u >> 16) & 255) + (u >> 24) - 510
        out[s:e] = (b.to(torch.float32) * scale).to(torch.bfloat16)
    return out


def uniform_ints(key: Tuple[int, int], numel: int, hi: int, device="cpu") -> torch.Tensor:
    """int64 values in [0, hi) (hi <= 2^16, modulo bias below 2^-16)."""
    idx = torch.arange(numel, dtype=torch.int64, device=device)
    return hash_words(key, idx) % hi


# --------------------------------------------------------------------------
# model weights
# --------------------------------------------------------------------------

LAYER_TENSORS = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate", "w_up", "w_down")
WEIGHT_STD = 0.02


def weight_shapes(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical tensor order.  Every matrix is [out, in], bf16.

    w_qkv stacks the query rows (head-major), then the key rows, then the value
    rows; w_gate and w_up are the two SwiGLU input projections.
    """
    d, F = cfg.d_model, cfg.ffn_dim
    shapes = [("embed", (cfg.vocab, d))]
    for l in range(cfg.n_layers):
        shapes += [
            (f"l{l}.attn_norm", (d,)),
            (f"l{l}.w_qkv", (cfg.qkv_dim, d)),
            (f"l{l}.w_o", (d, cfg.q_dim)),
            (f"l{l}.ffn_norm", (d,)),
            (f"l{l}.w_gate", (F, d)),
            (f"l{l}.w_up", (F, d)),
            (f"l{l}.w_down", (d, F)),
        ]
    shapes += [("final_norm", (d,)), ("w_lm", (cfg.vocab, d))]
    return shapes


def make_weight(cfg: ModelConfig, seed: int, index: int, name: str, shape, device="cpu",
                norm_std: float = 0.0, lm_std: float = WEIGHT_STD) -> torch.Tensor:
    numel = int(np.prod(shape))
    key = stream_key(seed, index)
    if name.endswith("norm"):
        if norm_std == 0.0:
            return torch.ones(shape, dtype=torch.bfloat16, device=device)
        return (1.0 + normalish(key, numel, norm_std, device).float()).to(torch.bfloat16).view(shape)
    std = lm_std if name == "w_lm" else WEIGHT_STD
    return normalish(key, numel, std, device).view(shape)


def model_weights(cfg: ModelConfig, seed: int, device="cpu", norm_std: float = 0.0,
                  lm_std: float = WEIGHT_STD) -> Dict[str, torch.Tensor]:
    """All weights of the decoder, bf16, in canonical order (dict keeps order).

    Matrices are approximately N(0, 0.02); norm gains are 1 (or 1 + N(0, norm_std)
    when ``norm_std`` > 0, used by tests to make the gains matter).  ``lm_std``
    rescales the LM head (tests use a larger value so that the top two logits
    of a row are rarely within rounding distance of each other).
    """
    return {name: make_weight(cfg, seed, i, name, shape, device, norm_std, lm_std)
            for i, (name, shape) in enumerate(weight_shapes(cfg))}


def layer_weight_names(l: int) -> List[str]:
    return [f"l{l}.{t}" for t in LAYER_TENSORS]


# --------------------------------------------------------------------------
# cached-context KV (the cached context is an input of the verify step)
# --------------------------------------------------------------------------

KV_STD = 1.0
_POS_STRIDE = 1 << 17


def kv_context(cfg: ModelConfig, seed: int, req: int, layer: int, pos0: int, n: int,
               device="cpu") -> torch.Tensor:
    """Keys and values of cached tokens pos0..pos0+n-1 of request ``req``.

    Returns bf16 [2, n_kv_heads, n, head_dim] (index 0 = keys, 1 = values),
    approximately N(0, 1), independent of how the tokens are paged.
    """
    H, D = cfg.n_kv_heads, cfg.head_dim
    assert pos0 + n <= _POS_STRIDE
    key = stream_key(seed, 7919, req, layer)
    kinds = torch.arange(2 * H, dtype=torch.int64, device=device).view(2 * H, 1, 1)
    pos = torch.arange(pos0, pos0 + n, dtype=torch.int64, device=device).view(1, n, 1)
    dd = torch.arange(D, dtype=torch.int64, device=device).view(1, 1, D)
    idx = ((kinds * _POS_STRIDE + pos) * D + dd).reshape(-1)
    out = torch.empty(idx.numel(), dtype=torch.bfloat16, device=device)
    scale = torch.tensor(KV_STD / _NORM_DIV, dtype=torch.float32, device=device)
    for s in range(0, idx.numel(), _CHUNK):
        u = hash_words(key, idx[s:s + _CHUNK])
        b = (u & 255) + ((u >> 8) & 255) + ((u >> 16) & 255) + (u >> 24) - 510
        out[s:s + _CHUNK] = (b.to(torch.float32) * scale).to(torch.bfloat16)
    return out.view(2, H, n, D)


# --------------------------------------------------------------------------
# token streams, context lengths, trajectories
# --------------------------------------------------------------------------


def uniform_tokens(seed: int, n: int, vocab: int) -> np.ndarray:
    return np.random.default_rng([seed, 11]).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def lognormal_contexts(seed: int, batch: int, median: float = 8192.0, sigma: float = 0.8,
                       lo: int = 1024, hi: int = 65536) -> np.ndarray:
    """Long-tailed context lengths: rint(lognormal(ln median, sigma)) clipped to [lo, hi]."""
    rng = np.random.default_rng(seed)
    x = np.rint(rng.lognormal(math.log(median), sigma, size=batch))
    return np.clip(x, lo, hi).astype(np.int64)


class MotifBank:
    """Recurring tool-call-like token patterns of length U[lo, hi]."""

    def __init__(self, seed: int, vocab: int, n_motifs: int = 256, lo: int = 64, hi: int = 512):
        rng = np.random.default_rng([seed, 23])
        self.motifs = [rng.integers(0, vocab, size=int(rng.integers(lo, hi + 1)), dtype=np.int64)
                       .astype(np.int32) for _ in range(n_motifs)]
        self.vocab, self.lo, self.hi = vocab, lo, hi

    def trajectory(self, seed: int, length: int, end_mid_motif: bool = False) -> np.ndarray:
        """Half motif tokens, half fresh 'observation' segments, in random order.

        With ``end_mid_motif`` the trajectory stops part-way into a motif, as a
        rollout that is in the middle of emitting a known pattern.
        """
        rng = np.random.default_rng([seed, 29])
        tail = np.zeros(0, dtype=np.int32)
        if end_mid_motif:
            m = self.motifs[int(rng.integers(len(self.motifs)))]
            tail = m[: int(rng.integers(16, len(m) - 8))]
        target = length - len(tail)
        segs, n = [], 0
        while n < target:
            if rng.random() < 0.5:
                s = self.motifs[int(rng.integers(len(self.motifs)))]
            else:
                s = rng.integers(0, self.vocab, size=int(rng.integers(self.lo, self.hi + 1)),
                                 dtype=np.int64).astype(np.int32)
            segs.append(s)
            n += len(s)
        body = np.concatenate(segs)[:target] if segs else np.zeros(0, np.int32)
        return np.concatenate([body, tail]).astype(np.int32)


def bernoulli_mask(seed: int, shape: Sequence[int], p: float) -> np.ndarray:
    return np.random.default_rng([seed, 31]).random(shape) < p
