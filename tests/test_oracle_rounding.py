"""Pins of WHERE the oracle rounds to bfloat16 (the precision contract of the
verify step: bf16 compute, fp32-or-better accumulate).

The contract: every matrix-multiply input (each RMSNorm output, the attention
output, the SwiGLU product) and the rotated q, k and the v of the new tokens
(the KV cache holds bf16) are rounded to bf16 (nearest even); the residual
stream, the projections' outputs, the norm statistics, the rotation, the
softmax and the logits are not.

Three kinds of pin, none of which re-types the oracle's formulas:

* stage by stage: from the intermediates the oracle records (its ``trace``
  hook), each stage is recomputed with independent library routines --
  torch's ``rms_norm``, ``silu`` and ``scaled_dot_product_attention`` in
  float64, the rotate-half RoPE of Hugging Face ``transformers`` -- and the
  recorded output must equal that value rounded exactly where the contract
  says, and not rounded anywhere else;
* representability: the rounded intermediates are bf16 values (checked with
  torch's conversion), the unrounded ones almost never are;
* a hand-built one-token case whose cached key, read from the step's new KV,
  tells rounding after the rotation from rounding before it by a known amount.

``test_every_rounding_mutation_is_caught`` then plants each plausible mistake
in a copy of the oracle's decoder (a rounding point dropped, moved before the
rotation, or added where the contract keeps full precision) and checks that
the stage checks name it.
"""
import math
import os
import types

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.decoder as dec
from oracle.bf16 import round_bf16
from oracle.decoder import Weights, forward_block
from paper_2607_17299_amd import synth

CFG = synth.reduced(synth.TINY, 1)
SRC = os.path.join(os.path.dirname(dec.__file__), "decoder.py")


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def _is_bf16(a) -> np.ndarray:
    """Elementwise: is the float64 value a bfloat16 value (torch's conversion)."""
    x = _t(a)
    return (x.float().bfloat16().double() == x).numpy() & (x.float().double() == x).numpy()


def _hf_rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """x [n, H, D] rotated with transformers' rotate-half RoPE (float64 angles)."""
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    D = x.shape[-1]
    inv = 1.0 / (base ** (torch.arange(0, D, 2, dtype=torch.float64) / D))
    ang = torch.from_numpy(np.asarray(pos, np.float64))[:, None] * inv[None, :]
    emb = torch.cat([ang, ang], dim=-1)                               # [n, D]
    xt = _t(x).transpose(0, 1)[None]                                  # [1, H, n, D]
    out, _ = apply_rotary_pos_emb(xt, xt, emb.cos()[None], emb.sin()[None])
    return out[0].transpose(0, 1).numpy()


def _sdpa(q, K, V, pos, group):
    """o [n, Hq, D] from torch's float64 attention with an explicit position mask."""
    n, Hq, D = q.shape
    S = K.shape[1]
    mask = torch.from_numpy(np.arange(S)[None, :] <= np.asarray(pos)[:, None])
    Kx = _t(K).repeat_interleave(group, dim=0)                        # [Hq, S, D]
    Vx = _t(V).repeat_interleave(group, dim=0)
    o = F.scaled_dot_product_attention(_t(q).transpose(0, 1), Kx, Vx, attn_mask=mask)
    return o.transpose(0, 1).numpy()


class StageError(AssertionError):
    def __init__(self, stage, msg):
        super().__init__(f"{stage}: {msg}")
        self.stage = stage


def _rounded(stage, got, ref):
    """got must be ref rounded to bf16, and ref must not be bf16 already."""
    want = round_bf16(ref)
    bad = np.count_nonzero(got != want)
    if bad:
        raise StageError(stage, f"{bad} of {got.size} values are not bf16(library value)")
    # (a row that sees a single key has o = v, a bf16 value: only a majority counts)
    if _is_bf16(ref).mean() > 0.5:
        raise StageError(stage, "the value before rounding is already bf16 (rounded earlier)")


def _unrounded(stage, got, ref, rtol=1e-12):
    """got must equal ref (no rounding in between) and must not be bf16 values."""
    if not np.allclose(got, ref, rtol=rtol, atol=1e-13):
        raise StageError(stage, f"differs from the library value by {np.abs(got - ref).max():.3g}")
    if _is_bf16(got).mean() > 0.5:
        raise StageError(stage, "rounded to bf16, the contract keeps it unrounded")


def check_stages(cfg, W: Weights, tokens, pos0, kv_get, fwd=forward_block):
    """Run the decoder with its trace and check every stage (raises StageError)."""
    tr = {}
    logits, new_kv = fwd(cfg, W, tokens, pos0, kv_get, trace=tr)
    n, Hq, Hkv, D = len(tokens), cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    pos = pos0 + np.arange(n)
    eps = cfg.rms_eps

    def norm(x, g):
        return F.rms_norm(_t(x), (x.shape[-1],), _t(g), eps=eps).numpy()

    h = tr["h0"]
    if not (_is_bf16(h).all() and np.array_equal(h, W.embed_rows(tokens))):
        raise StageError("h0", "embedding rows are not the bf16 table rows")
    for l in range(cfg.n_layers):
        p = f"l{l}."
        _rounded(p + "u1", tr[p + "u1"], norm(h, W.get(p + "attn_norm")))
        qkv_ref = (_t(tr[p + "u1"]) @ _t(W.get(p + "w_qkv")).T).numpy()
        _unrounded(p + "qkv", tr[p + "qkv"], qkv_ref)
        qkv = tr[p + "qkv"]
        q0 = qkv[:, : Hq * D].reshape(n, Hq, D)
        k0 = qkv[:, Hq * D: (Hq + Hkv) * D].reshape(n, Hkv, D)
        v0 = qkv[:, (Hq + Hkv) * D:].reshape(n, Hkv, D)
        _rounded(p + "q", tr[p + "q"], _hf_rope(q0, pos, cfg.rope_base))
        _rounded(p + "k", tr[p + "k"], _hf_rope(k0, pos, cfg.rope_base))
        _rounded(p + "v", tr[p + "v"], v0)
        if not (np.array_equal(new_kv[l][0], tr[p + "k"].transpose(1, 0, 2)) and
                np.array_equal(new_kv[l][1], tr[p + "v"].transpose(1, 0, 2))):
            raise StageError(p + "kv", "the new KV is not the rounded k and v")
        Kc, Vc = kv_get(l)
        K = np.concatenate([Kc, tr[p + "k"].transpose(1, 0, 2)], axis=1)
        V = np.concatenate([Vc, tr[p + "v"].transpose(1, 0, 2)], axis=1)
        o_ref = _sdpa(tr[p + "q"], K, V, pos, Hq // Hkv).reshape(n, Hq * D)
        _rounded(p + "o", tr[p + "o"], o_ref)
        _unrounded(p + "h1", tr[p + "h1"], h + (_t(tr[p + "o"]) @ _t(W.get(p + "w_o")).T).numpy())
        h = tr[p + "h1"]
        _rounded(p + "u2", tr[p + "u2"], norm(h, W.get(p + "ffn_norm")))
        u2 = _t(tr[p + "u2"])
        _unrounded(p + "gate", tr[p + "gate"], (u2 @ _t(W.get(p + "w_gate")).T).numpy())
        _unrounded(p + "up", tr[p + "up"], (u2 @ _t(W.get(p + "w_up")).T).numpy())
        y_ref = (F.silu(_t(tr[p + "gate"])) * _t(tr[p + "up"])).numpy()
        _rounded(p + "y", tr[p + "y"], y_ref)
        _unrounded(p + "h2", tr[p + "h2"], h + (_t(tr[p + "y"]) @ _t(W.get(p + "w_down")).T).numpy())
        h = tr[p + "h2"]
    _rounded("hf", tr["hf"], norm(h, W.get("final_norm")))
    z_ref = (_t(tr["hf"]) @ _t(W.get("w_lm")).T).numpy()
    _unrounded("logits", tr["logits"], z_ref)
    if not np.array_equal(logits, tr["logits"]):
        raise StageError("logits", "returned logits differ from the recorded ones")
    return tr


@pytest.fixture(scope="module")
def W1():
    return Weights(CFG, synth.model_weights(CFG, seed=4, norm_std=0.1))


def _cached(cfg, n, seed=3):
    """A cached context of n tokens: bf16 keys/values, std 1."""
    rng = np.random.default_rng(seed)
    layers = [tuple(round_bf16(rng.standard_normal((cfg.n_kv_heads, n, cfg.head_dim))) for _ in range(2))
              for _ in range(cfg.n_layers)]
    return lambda l: layers[l]


def test_stages_of_a_fresh_block(W1):
    toks = synth.uniform_tokens(21, 12, CFG.vocab)
    check_stages(CFG, W1, toks, 0, _cached(CFG, 0))


def test_stages_of_a_block_over_a_cached_context(W1):
    toks = synth.uniform_tokens(22, 5, CFG.vocab)
    check_stages(CFG, W1, toks, 37, _cached(CFG, 37))


def test_stages_of_two_layers():
    cfg = synth.TINY
    W = Weights(cfg, synth.model_weights(cfg, seed=0, norm_std=0.1))
    toks = synth.uniform_tokens(23, 6, cfg.vocab)
    check_stages(cfg, W, toks, 19, _cached(cfg, 19, seed=5))


def test_rounded_intermediates_are_bf16_and_the_others_are_not(W1):
    tr = check_stages(CFG, W1, synth.uniform_tokens(24, 9, CFG.vocab), 11, _cached(CFG, 11))
    for name in ("l0.u1", "l0.q", "l0.k", "l0.v", "l0.o", "l0.u2", "l0.y", "hf"):
        assert _is_bf16(tr[name]).all(), name
    for name in ("l0.qkv", "l0.h1", "l0.gate", "l0.up", "l0.h2", "logits"):
        assert _is_bf16(tr[name]).mean() < 0.01, name


def _one_token_model(eps=0.0):
    """d = 4, one head of dim 4, vocab 2: token 0's embedding row is all ones, so
    with unit gains and eps = 0 the attention norm output is exactly 1."""
    cfg = synth.ModelConfig(n_layers=1, d_model=4, n_q_heads=1, n_kv_heads=1, head_dim=4,
                            ffn_dim=4, vocab=2, rms_eps=eps)
    one = np.ones(4)
    w_qkv = np.zeros((12, 4))
    # k = (1 + 2^-9, 0, 3 - 2^-7, 0): no rounding in the projection (exact sums of
    # bf16 entries), neither component is a bf16 value
    w_qkv[4, 0], w_qkv[4, 1] = 1.0, 2.0 ** -9
    w_qkv[6, 0], w_qkv[6, 1] = 3.0, -(2.0 ** -7)
    t = {"embed": np.stack([one, one]), "l0.attn_norm": one, "l0.w_qkv": w_qkv,
         "l0.w_o": np.zeros((4, 4)), "l0.ffn_norm": one, "l0.w_gate": np.zeros((4, 4)),
         "l0.w_up": np.zeros((4, 4)), "l0.w_down": np.zeros((4, 4)), "final_norm": one,
         "w_lm": np.zeros((2, 4))}
    return cfg, Weights(cfg, t)


def test_hand_built_key_is_rounded_after_the_rotation():
    """Key pair (k0, k2) = (1 + 2^-9, 3 - 2^-7) at position 1 turns by 1 rad
    (pair 0's frequency is 1): k0 cos 1 - k2 sin 1 = -1.97648..., k2 cos 1 +
    k0 sin 1 = 2.45980...  Rounding after the rotation gives (-1.9765625,
    2.453125); rounding the projection first, bf16(k0) = 1 and bf16(k2) = 3,
    gives (-1.984375, 2.46875): 2^-7 and 2^-6 apart.  Pair 1 is zero and
    stays zero."""
    cfg, W = _one_token_model()
    p = 1
    rng = np.random.default_rng(0)
    cached = round_bf16(rng.standard_normal((1, p, 4)))
    _, new_kv = forward_block(cfg, W, [0], p, lambda l: (cached, cached))
    k_out = new_kv[0][0][0, 0]                                         # [D]
    assert (k_out[0], k_out[2]) == (-1.9765625, 2.453125)
    assert (k_out[0], k_out[2]) != (-1.984375, 2.46875)
    assert k_out[1] == 0.0 and k_out[3] == 0.0
    # the same closed form from Python's math module, both orders
    k0, k2 = 1.0 + 2.0 ** -9, 3.0 - 2.0 ** -7
    c, s = math.cos(1.0), math.sin(1.0)
    assert (round_bf16(k0 * c - k2 * s), round_bf16(k2 * c + k0 * s)) == (-1.9765625, 2.453125)
    assert (round_bf16(c - 3 * s), round_bf16(3 * c + s)) == (-1.984375, 2.46875)


# ------------------------------------------------------------- mutation check
# Each mutant changes one line of the decoder's source: a rounding point
# dropped, moved before the rotation, or added where full precision is kept.
MUTANTS = {
    "drop u1": ("u = rb(rms_norm(h, W.get(p + \"attn_norm\"), cfg.rms_eps))",
                "u = rms_norm(h, W.get(p + \"attn_norm\"), cfg.rms_eps)", "l0.u1"),
    "drop q": ("q = rb(rope(q, pos, cfg.rope_base))", "q = rope(q, pos, cfg.rope_base)", "l0.q"),
    "drop k": ("k = rb(rope(k, pos, cfg.rope_base))", "k = rope(k, pos, cfg.rope_base)", "l0.k"),
    "drop v": ("v = rb(v)", "v = v", "l0.v"),
    "drop o": ("o = rb(attn(q, K, V, pos, Hq // Hkv))", "o = (attn(q, K, V, pos, Hq // Hkv))", "l0.o"),
    "drop u2": ("u = rb(rms_norm(h, W.get(p + \"ffn_norm\"), cfg.rms_eps))",
                "u = rms_norm(h, W.get(p + \"ffn_norm\"), cfg.rms_eps)", "l0.u2"),
    "drop y": ("y = rb(silu(gate) * up)", "y = silu(gate) * up", "l0.y"),
    "drop hf": ("hf = rb(rms_norm(h, W.get(\"final_norm\"), cfg.rms_eps))",
                "hf = rms_norm(h, W.get(\"final_norm\"), cfg.rms_eps)", "hf"),
    "q before rope": ("q = rb(rope(q, pos, cfg.rope_base))", "q = rope(rb(q), pos, cfg.rope_base)", "l0.q"),
    "k before rope": ("k = rb(rope(k, pos, cfg.rope_base))", "k = rope(rb(k), pos, cfg.rope_base)", "l0.k"),
    "q twice": ("q = rb(rope(q, pos, cfg.rope_base))", "q = rb(rope(rb(q), pos, cfg.rope_base))", "l0.q"),
    "norm before gain": ("u = rb(rms_norm(h, W.get(p + \"attn_norm\"), cfg.rms_eps))",
                         "u = rb(rms_norm(h, 1.0, cfg.rms_eps)) * W.get(p + \"attn_norm\")", "l0.u1"),
    "add qkv": ("qkv = mm(u, W.get(p + \"w_qkv\"))", "qkv = rb(mm(u, W.get(p + \"w_qkv\")))", "l0.qkv"),
    "add h1": ("h = h + mm(o, W.get(p + \"w_o\"))", "h = rb(h + mm(o, W.get(p + \"w_o\")))", "l0.h1"),
    "add gate": ("gate, up = mm(u, W.get(p + \"w_gate\")), mm(u, W.get(p + \"w_up\"))",
                 "gate, up = rb(mm(u, W.get(p + \"w_gate\"))), mm(u, W.get(p + \"w_up\"))", "l0.gate"),
    "add silu": ("y = rb(silu(gate) * up)", "y = rb(rb(silu(gate)) * up)", "l0.y"),
    "add h2": ("h = h + mm(y, W.get(p + \"w_down\"))", "h = rb(h + mm(y, W.get(p + \"w_down\")))", "l0.h2"),
    "add logits": ("z = mm(hf, W.get(\"w_lm\"))", "z = rb(mm(hf, W.get(\"w_lm\")))", "logits"),
}


def _mutant(old: str, new: str):
    src = open(SRC).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle._decoder_mutant")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), SRC, "exec"), mod.__dict__)
    return mod.forward_block


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_every_rounding_mutation_is_caught(W1, name):
    old, new, stage = MUTANTS[name]
    fwd = _mutant(old, new)
    toks = synth.uniform_tokens(25, 7, CFG.vocab)
    with pytest.raises(StageError) as e:
        check_stages(CFG, W1, toks, 13, _cached(CFG, 13), fwd=fwd)
    assert e.value.stage == stage, str(e.value)
