"""Pins of the oracle decoder and verify step.

* The pure-float64 decoder is compared with an independent library decoder
  (Hugging Face transformers' Llama: RMSNorm, rotate-half RoPE, GQA, SwiGLU, no
  biases) loaded with the same weights -- this fixes transposes, head mapping,
  the RoPE convention, the causal mask and the residual wiring.
* The verify step is pinned by the invariants that define greedy speculative
  verification: k = 0 is plain decode, drafts equal to the greedy continuation
  are all accepted, and iterated verify steps with arbitrary drafts emit
  exactly the token-by-token greedy stream (losslessness); prefill followed by
  an append and decode matches full recomputation.
"""
import numpy as np
import pytest
import torch

from oracle.accept import argmax_lowest
from oracle.decoder import RequestKV, Weights, forward_block
from oracle.verify import (commit_request, greedy_decode, prefill_request, verify_request)
from paper_2607_17299_amd import synth

CFG = synth.TINY


@pytest.fixture(scope="module")
def tiny_weights():
    return synth.model_weights(CFG, seed=0, norm_std=0.1)


@pytest.fixture(scope="module")
def W(tiny_weights):
    return Weights(CFG, tiny_weights)


def _hf_llama(tw):
    from transformers import LlamaConfig, LlamaForCausalLM
    c = LlamaConfig(vocab_size=CFG.vocab, hidden_size=CFG.d_model, intermediate_size=CFG.ffn_dim,
                    num_hidden_layers=CFG.n_layers, num_attention_heads=CFG.n_q_heads,
                    num_key_value_heads=CFG.n_kv_heads, head_dim=CFG.head_dim,
                    rms_norm_eps=CFG.rms_eps, rope_theta=CFG.rope_base,
                    max_position_embeddings=4096, tie_word_embeddings=False,
                    attention_bias=False, mlp_bias=False)
    c._attn_implementation = "eager"
    m = LlamaForCausalLM(c).double().eval()
    f = lambda t: t.detach().double()
    qd, kd = CFG.q_dim, CFG.kv_dim
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(f(tw["embed"]))
        for l, layer in enumerate(m.model.layers):
            w = tw[f"l{l}.w_qkv"]
            layer.self_attn.q_proj.weight.copy_(f(w[:qd]))
            layer.self_attn.k_proj.weight.copy_(f(w[qd:qd + kd]))
            layer.self_attn.v_proj.weight.copy_(f(w[qd + kd:]))
            layer.self_attn.o_proj.weight.copy_(f(tw[f"l{l}.w_o"]))
            layer.input_layernorm.weight.copy_(f(tw[f"l{l}.attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(f(tw[f"l{l}.ffn_norm"]))
            layer.mlp.gate_proj.weight.copy_(f(tw[f"l{l}.w_gate"]))
            layer.mlp.up_proj.weight.copy_(f(tw[f"l{l}.w_up"]))
            layer.mlp.down_proj.weight.copy_(f(tw[f"l{l}.w_down"]))
        m.model.norm.weight.copy_(f(tw["final_norm"]))
        m.lm_head.weight.copy_(f(tw["w_lm"]))
    return m


def _empty(l):
    e = np.zeros((CFG.n_kv_heads, 0, CFG.head_dim))
    return e, e


def test_float64_decoder_matches_transformers_llama(tiny_weights, W):
    m = _hf_llama(tiny_weights)
    toks = synth.uniform_tokens(5, 48, CFG.vocab)
    ours, _ = forward_block(CFG, W, toks, 0, _empty, rounding=False)
    with torch.no_grad():
        ref = m(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    # transformers evaluates RoPE angles and the norm statistics in float32
    np.testing.assert_allclose(ours, ref, atol=1e-5, rtol=0)
    # and greedy generation agrees token for token
    kv = RequestKV(CFG)
    r = prefill_request(CFG, W, kv, toks[:-1], rounding=False)
    stream = greedy_decode(CFG, W, kv, toks[-1], 6, rounding=False)
    with torch.no_grad():
        gen = m.generate(torch.from_numpy(toks.astype(np.int64))[None], max_new_tokens=6,
                         do_sample=False, pad_token_id=0)[0, len(toks):].tolist()
    assert stream == gen


def test_float32_mode_matches_transformers_llama_in_float32(tiny_weights, W):
    # the fp32-accumulation mode computes the same function at float32 precision
    m = _hf_llama(tiny_weights).float()
    toks = synth.uniform_tokens(15, 40, CFG.vocab)
    ours, _ = forward_block(CFG, W, toks, 0, _empty, rounding=False, precision="fp32")
    with torch.no_grad():
        ref = m(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].double().numpy()
    np.testing.assert_allclose(ours, ref, atol=1e-4, rtol=0)
    ours64, _ = forward_block(CFG, W, toks, 0, _empty, rounding=False)
    assert 0 < np.abs(ours - ours64).max() < 1e-4


def test_rounding_points_change_logits_only_at_bf16_scale(W):
    toks = synth.uniform_tokens(6, 32, CFG.vocab)
    a, _ = forward_block(CFG, W, toks, 0, _empty, rounding=False)
    b, _ = forward_block(CFG, W, toks, 0, _empty, rounding=True)
    d = np.abs(a - b).max()
    assert 1e-6 < d < 5e-2


def _prefilled(W, seed, n):
    kv = RequestKV(CFG)
    toks = synth.uniform_tokens(seed, n + 1, CFG.vocab)
    prefill_request(CFG, W, kv, toks[:-1])
    return kv, int(toks[-1])


def test_k0_is_plain_decode(W):
    kv, x = _prefilled(W, 7, 200)
    r = verify_request(CFG, W, kv, x, [])
    logits, _ = forward_block(CFG, W, [x], kv.length, kv.get)
    assert r["accept"] == 0 and r["logits"].shape == (1, CFG.vocab)
    np.testing.assert_array_equal(r["logits"], logits)
    assert r["next"] == int(argmax_lowest(logits)[0])


def test_verify_rows_equal_prefill_rows(W):
    # the causal mask inside the block: row i never sees rows > i
    kv, x = _prefilled(W, 8, 150)
    drafts = synth.uniform_tokens(9, 6, CFG.vocab).tolist()
    r = verify_request(CFG, W, kv, x, drafts)
    for i in range(len(drafts) + 1):
        li, _ = forward_block(CFG, W, ([x] + drafts)[: i + 1], kv.length, kv.get)
        np.testing.assert_allclose(r["logits"][i], li[-1], atol=1e-9, rtol=0)


def test_true_greedy_continuation_is_fully_accepted(W):
    kv, x = _prefilled(W, 10, 120)
    k = 5
    import copy
    cont = greedy_decode(CFG, W, copy.deepcopy(kv), x, k + 1)
    r = verify_request(CFG, W, kv, x, cont[:k])
    assert r["accept"] == k
    assert r["next"] == cont[k]


def test_losslessness_iterated_verify_equals_greedy_stream(W):
    import copy
    kv, x = _prefilled(W, 11, 64)
    ref = greedy_decode(CFG, W, copy.deepcopy(kv), x, 40)
    rng = np.random.default_rng(12)
    out, pos = [], 0
    while len(out) < 40:
        k = int(rng.integers(0, 6))
        # drafts: a prefix of the true stream, then junk (or all junk, or all true)
        good = int(rng.integers(0, k + 1))
        drafts = ref[pos: pos + good] + rng.integers(0, CFG.vocab, size=k - good).tolist()
        drafts = drafts[:k]
        r = verify_request(CFG, W, kv, x, drafts)
        commit_request(kv, r)
        emitted = drafts[: r["accept"]] + [r["next"]]
        out += emitted
        pos += len(emitted)
        x = r["next"]
    assert out[:40] == ref


def test_prefill_append_decode_equals_full_recompute(W):
    toks = synth.uniform_tokens(13, 401, CFG.vocab)
    kv_a = RequestKV(CFG)
    prefill_request(CFG, W, kv_a, toks[:300])
    ra = prefill_request(CFG, W, kv_a, toks[300:400])
    kv_b = RequestKV(CFG)
    rb = prefill_request(CFG, W, kv_b, toks[:400])
    np.testing.assert_allclose(ra["logits"][-1], rb["logits"][-1], atol=1e-9, rtol=0)
    assert ra["next"] == rb["next"]
    for (Ka, Va), (Kb, Vb) in zip(kv_a.layers, kv_b.layers):
        np.testing.assert_allclose(Ka, Kb, atol=1e-9, rtol=0)
        np.testing.assert_allclose(Va, Vb, atol=1e-9, rtol=0)
    assert greedy_decode(CFG, W, kv_a, toks[400], 5) == greedy_decode(CFG, W, kv_b, toks[400], 5)
