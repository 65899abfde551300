"""GQA decoder forward over a block of new tokens -- oracle (test infrastructure only).

Plain definitions, float64, one request at a time:
  RMSNorm   y = x / sqrt(mean(x^2) + eps) * g          (Zhang & Sennrich 2019)
  RoPE      rotate-half form: pair (j, j + D/2) of a head is rotated by the angle
            p * base^(-2j/D) at absolute 0-based position p       (Su et al. 2021)
  attention each query head h reads key/value head floor(h / group)
            (grouped-query attention, Ainslie et al. 2023); scores q.k / sqrt(D);
            the query at position p sees keys at positions 0..p; softmax over them
  SwiGLU    silu(u W_gate^T) * (u W_up^T), silu(a) = a / (1 + e^-a)  (Shazeer 2020)
  residual  h += attention(...) W_o^T ;  h += swiglu(...) W_down^T
  logits    z = norm(h) W_lm^T (untied), float64
No biases, no QK-norm.

Precision contract (bf16 compute, fp32-or-better accumulate): with
``rounding=True`` the values that a bf16 kernel stores in bf16 are rounded to
bf16 here too -- every matrix-multiply input (each norm output, the attention
output, the SwiGLU product) and the rotated q, k and the v of the new tokens
(keys and values are cached in bf16).  Everything else (residual stream, norm
statistics, rotation, softmax, logits) stays float64.  ``rounding=False`` gives
the pure float64 decoder.

``precision="fp32"`` runs every matrix product and the attention in float32
(same rounding points).  It is the same algorithm at the accumulation
precision of a bf16 kernel, used to measure how far any fp32-accumulating
implementation drifts from the float64 result (the parity tolerance at full
depth is derived from that drift).

The verify step scores all new tokens of a request in ONE forward pass with a
causal mask inside the block (System Design, "SuffixDecoding": drafts verified
by the target in a single forward pass).
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from .bf16 import round_bf16


def to_f64(x) -> np.ndarray:
    """float64 numpy copy of a numpy array or of a (CPU) torch tensor."""
    if hasattr(x, "detach"):          # torch tensor, without importing torch
        x = x.detach().to("cpu").float().numpy()
    return np.asarray(x, dtype=np.float64)


class Weights:
    """Read-only view of the decoder weights (bf16 values held as float64).

    ``tensors`` maps the canonical names (embed, l{i}.attn_norm, l{i}.w_qkv,
    l{i}.w_o, l{i}.ffn_norm, l{i}.w_gate, l{i}.w_up, l{i}.w_down, final_norm,
    w_lm) to arrays; every matrix is [out, in].  Large models are converted
    layer by layer on use (``cache=False``) to bound host memory.
    """

    def __init__(self, cfg, tensors, cache: bool = True):
        self.cfg, self.t, self.cache = cfg, tensors, cache
        self._c: Dict[str, np.ndarray] = {}

    def get(self, name: str) -> np.ndarray:
        if name in self._c:
            return self._c[name]
        a = to_f64(self.t[name])
        if self.cache:
            self._c[name] = a
        return a

    def embed_rows(self, tokens: Sequence[int]) -> np.ndarray:
        e = self.t["embed"]
        idx = np.asarray(tokens, dtype=np.int64)
        if hasattr(e, "detach"):
            import torch  # only to index a torch tensor without converting all of it
            return to_f64(e[torch.as_tensor(idx)])
        return to_f64(np.asarray(e)[idx])


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """x [n, H, D], pos [n] absolute positions -> rotated copy (rotate-half)."""
    D = x.shape[-1]
    half = D // 2
    inv_freq = base ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]   # [n, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, q_pos: np.ndarray,
              group: int) -> np.ndarray:
    """q [n, Hq, D]; K, V [Hkv, S, D] hold keys/values at positions 0..S-1.

    Query i (position q_pos[i]) of head h attends keys 0..q_pos[i] of kv-head
    h // group.  Returns o [n, Hq, D] in the inputs' float type.
    """
    n, Hq, D = q.shape
    S = K.shape[1]
    scale = q.dtype.type(1.0 / np.sqrt(D))
    visible = np.arange(S)[None, :] <= np.asarray(q_pos)[:, None]      # [n, S]
    o = np.empty((n, Hq, D), dtype=q.dtype)
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ K[g].T) * scale                                # [n, S]
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        o[:, h, :] = p @ V[g]
    return o


KVGetter = Callable[[int], Tuple[np.ndarray, np.ndarray]]


def forward_block(cfg, W: Weights, tokens: Sequence[int], pos0: int, kv_get: KVGetter,
                  rounding: bool = True, want_logits: bool = True, precision: str = "fp64",
                  trace: Optional[Dict[str, np.ndarray]] = None):
    """Run tokens (at positions pos0, pos0+1, ...) through the decoder.

    ``kv_get(l)`` returns the cached keys and values of layer l for positions
    0..pos0-1 as [Hkv, pos0, D] arrays.  Returns (logits [n, V] or the final
    normalised hidden state when want_logits is False, new_kv) where new_kv[l]
    = (K_new [Hkv, n, D], V_new [Hkv, n, D]) for the block's own tokens.

    ``trace``, when given, receives every intermediate under a name (layer l's
    as "l{l}.<name>"): h0 (embedding rows), u1 (attention norm output), qkv
    (projection), q, k, v (after RoPE and rounding), o (attention output),
    h1 (residual after attention), u2 (FFN norm output), gate, up, y (SwiGLU
    product), h2 (residual after the FFN), then hf (final norm output) and
    logits.  Recording copies values only; it changes no arithmetic.
    """
    rb = round_bf16 if rounding else (lambda a: a)
    rec = (lambda name, a: trace.__setitem__(name, np.array(a, copy=True))) if trace is not None \
        else (lambda name, a: None)
    if precision == "fp64":
        mm = lambda x, Wt: x @ Wt.T
        attn = attention
    elif precision == "fp32":
        f32 = lambda a: np.asarray(a, dtype=np.float32)
        mm = lambda x, Wt: (f32(x) @ f32(Wt).T).astype(np.float64)
        attn = lambda q, K, V, p, g: attention(f32(q), f32(K), f32(V), p, g).astype(np.float64)
    else:
        raise ValueError(precision)
    n = len(tokens)
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    pos = pos0 + np.arange(n)
    h = W.embed_rows(tokens)                                             # [n, d]
    rec("h0", h)
    new_kv: List[Tuple[np.ndarray, np.ndarray]] = []
    for l in range(cfg.n_layers):
        p = f"l{l}."
        u = rb(rms_norm(h, W.get(p + "attn_norm"), cfg.rms_eps))
        rec(p + "u1", u)
        qkv = mm(u, W.get(p + "w_qkv"))                                 # [n, qkv]
        rec(p + "qkv", qkv)
        q = qkv[:, : Hq * D].reshape(n, Hq, D)
        k = qkv[:, Hq * D: (Hq + Hkv) * D].reshape(n, Hkv, D)
        v = qkv[:, (Hq + Hkv) * D:].reshape(n, Hkv, D)
        q = rb(rope(q, pos, cfg.rope_base))
        k = rb(rope(k, pos, cfg.rope_base))
        v = rb(v)
        rec(p + "q", q)
        rec(p + "k", k)
        rec(p + "v", v)
        Kc, Vc = kv_get(l)
        K = np.concatenate([Kc, k.transpose(1, 0, 2)], axis=1)          # [Hkv, pos0+n, D]
        V = np.concatenate([Vc, v.transpose(1, 0, 2)], axis=1)
        new_kv.append((k.transpose(1, 0, 2).copy(), v.transpose(1, 0, 2).copy()))
        o = rb(attn(q, K, V, pos, Hq // Hkv)).reshape(n, Hq * D)
        rec(p + "o", o)
        h = h + mm(o, W.get(p + "w_o"))
        rec(p + "h1", h)
        u = rb(rms_norm(h, W.get(p + "ffn_norm"), cfg.rms_eps))
        rec(p + "u2", u)
        gate, up = mm(u, W.get(p + "w_gate")), mm(u, W.get(p + "w_up"))
        rec(p + "gate", gate)
        rec(p + "up", up)
        y = rb(silu(gate) * up)
        rec(p + "y", y)
        h = h + mm(y, W.get(p + "w_down"))
        rec(p + "h2", h)
    hf = rb(rms_norm(h, W.get("final_norm"), cfg.rms_eps))
    rec("hf", hf)
    if not want_logits:
        return hf, new_kv
    z = mm(hf, W.get("w_lm"))
    rec("logits", z)
    return z, new_kv


class RequestKV:
    """Dense cached keys/values of one request, per layer [Hkv, length, D]."""

    def __init__(self, cfg, layers: Optional[List[Tuple[np.ndarray, np.ndarray]]] = None):
        self.cfg = cfg
        if layers is None:
            e = np.zeros((cfg.n_kv_heads, 0, cfg.head_dim))
            layers = [(e, e) for _ in range(cfg.n_layers)]
        self.layers = layers

    @property
    def length(self) -> int:
        return self.layers[0][0].shape[1]

    def get(self, l: int):
        return self.layers[l]

    def append(self, new_kv, count: int) -> None:
        """Keep the first ``count`` rows of a block's new keys/values."""
        self.layers = [(np.concatenate([K, nk[:, :count]], axis=1),
                        np.concatenate([V, nv[:, :count]], axis=1))
                       for (K, V), (nk, nv) in zip(self.layers, new_kv)]
