"""Pin of the oracle's decoder composition against an independent Llama implementation (CPU only).

The paper's targets are LLaMA-2 7B class decoders (Sec. 4.1, "Models"); the
oracle writes the Llama layer out from that family's definition.  Here the
oracle's block forward is compared with ``transformers.LlamaForCausalLM``
(float64, untied embedding and head) loaded with the same synthetic weights.
This pins what the layer-piece tests cannot: which of W_gate / W_up goes
through SiLU, where the two pre-norms sit, the final norm before the untied
head, the residual wiring, and the verify block's positions against a
committed cache.  RMSNorm gains are drawn away from 1 here so that a norm in
the wrong place changes the result.

The library computes its RoPE tables in float32, which sets the agreement
floor (about 1e-7 on these shapes); the bound is 1e-6.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import model as om
from paper_2608_10362_amd import synth

transformers = pytest.importorskip("transformers")

MHA = synth.ModelShape(2, 128, 4, 4, 32, 352, 512, dtype="f32")
GQA = synth.ModelShape(3, 128, 8, 2, 16, 256, 300, dtype="f32")
TOL = 1e-6


def _weights(shape, seed=11):
    """Synthetic weights with RMSNorm gains 1 + 0.2 N(0, 1) (test-local draws)."""
    W = synth.make_weights(shape, seed=seed)
    rng = np.random.default_rng([seed, 99])
    for L in W["layers"]:
        L["attn_norm"] = (1.0 + 0.2 * rng.standard_normal(shape.d_model)).astype(np.float32)
        L["ffn_norm"] = (1.0 + 0.2 * rng.standard_normal(shape.d_model)).astype(np.float32)
    W["final_norm"] = (1.0 + 0.2 * rng.standard_normal(shape.d_model)).astype(np.float32)
    return W


def _hf_model(shape, W):
    cfg = transformers.LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
        rope_theta=shape.rope_base, tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
        max_position_embeddings=1024)
    cfg._attn_implementation = "eager"
    m = transformers.LlamaForCausalLM(cfg).to(torch.float64).eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(W["embed"]))
        for l, L in enumerate(W["layers"]):
            layer = m.model.layers[l]
            layer.input_layernorm.weight.copy_(t(L["attn_norm"]))
            layer.self_attn.q_proj.weight.copy_(t(L["wq"]))
            layer.self_attn.k_proj.weight.copy_(t(L["wk"]))
            layer.self_attn.v_proj.weight.copy_(t(L["wv"]))
            layer.self_attn.o_proj.weight.copy_(t(L["wo"]))
            layer.post_attention_layernorm.weight.copy_(t(L["ffn_norm"]))
            layer.mlp.gate_proj.weight.copy_(t(L["w_gate"]))
            layer.mlp.up_proj.weight.copy_(t(L["w_up"]))
            layer.mlp.down_proj.weight.copy_(t(L["w_down"]))
        m.model.norm.weight.copy_(t(W["final_norm"]))
        m.lm_head.weight.copy_(t(W["lm_head"]))
    return m


def _hf_logits(m, tokens):
    with torch.no_grad():
        out = m(input_ids=torch.tensor(np.asarray(tokens)[None, :], dtype=torch.long), use_cache=False)
    return out.logits[0].numpy()


def _oracle_block(shape, W, tokens, start):
    """Oracle logits of tokens[start:] verified as one block after committing tokens[:start]."""
    model = om.Model(shape, W)
    kv = om.KVCache(shape, shape.n_layers, 128)
    if start:
        model.prefill(tokens[:start], kv)
    return model.forward_block(tokens[start:], kv.length, kv)


def _tokens(shape, n, seed=7):
    return np.random.default_rng(seed).integers(0, shape.vocab, n)


@pytest.mark.parametrize("shape", [MHA, GQA], ids=["mha", "gqa"])
def test_block_forward_matches_library_llama(shape):
    W = _weights(shape)
    tok = _tokens(shape, 48)
    ref = _hf_logits(_hf_model(shape, W), tok)
    got = _oracle_block(shape, W, tok, 0)
    assert np.abs(got - ref).max() < TOL
    # the comparison is sensitive: logits spread over several units
    assert np.abs(ref).max() > 0.05


@pytest.mark.parametrize("shape", [MHA, GQA], ids=["mha", "gqa"])
def test_verify_block_after_committed_context_matches_library(shape):
    # gamma + 1 = 5 rows at positions 43..47 against a 43-token committed cache
    W = _weights(shape)
    tok = _tokens(shape, 48, seed=8)
    ref = _hf_logits(_hf_model(shape, W), tok)[43:]
    got = _oracle_block(shape, W, tok, 43)
    assert np.abs(got - ref).max() < TOL


def _swap(W, a, b, scope="layers"):
    W2 = {k: v for k, v in W.items()}
    W2["layers"] = [dict(L) for L in W["layers"]]
    if scope == "layers":
        for L in W2["layers"]:
            L[a], L[b] = L[b], L[a]
    return W2


@pytest.mark.parametrize("mistake", ["gate_up", "norms", "final_norm", "q_k"])
def test_planted_composition_mistakes_fail_the_pin(mistake):
    """Composition mistakes planted in the oracle's input (so, in effect, in its
    wiring) make it disagree with the library by far more than the bound."""
    shape = GQA
    W = _weights(shape)
    tok = _tokens(shape, 48)
    ref = _hf_logits(_hf_model(shape, W), tok)
    if mistake == "gate_up":      # SiLU on the up projection instead of the gate
        W2 = _swap(W, "w_gate", "w_up")
    elif mistake == "norms":      # pre-attention and pre-FFN gains exchanged
        W2 = _swap(W, "attn_norm", "ffn_norm")
    elif mistake == "final_norm":  # no final RMSNorm gain before the head
        W2 = dict(W)
        W2["final_norm"] = np.ones_like(W["final_norm"])
    else:                          # keys projected with the query weights' key-sized slice
        W2 = _swap(W, "wq", "wq")
        for L in W2["layers"]:
            L["wk"] = L["wq"][: shape.kv_dim]
    got = _oracle_block(shape, W2, tok, 0)
    assert np.abs(got - ref).max() > 100 * TOL
