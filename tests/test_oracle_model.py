"""Pins for the oracle's decoder forward (CPU only).

Each layer piece is checked against an independent library routine or a
closed form; the verify pass over gamma+1 tokens is checked against gamma+1
single-token steps (the property the draft-and-verify iteration relies on).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model as om
from oracle.specdec import Sequence, greedy_decode
from paper_2608_10362_amd import synth


def test_round_to_bf16_matches_torch_on_float32_values():
    x = (np.random.default_rng(0).standard_normal(200000) * 3).astype(np.float32).astype(np.float64)
    ref = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(om.round_to_bf16(x), ref)
    # ties to even
    t = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8)])
    np.testing.assert_array_equal(om.round_to_bf16(t), [1.0, 1 + 2 ** -6, -1.0])


def test_bf16_bits_widen_exactly():
    bits = np.arange(0, 65536, 7, dtype=np.uint32).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]  # skip inf/nan
    ref = torch.tensor(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(om.bf16_bits_to_f64(bits), ref)


def test_rmsnorm_unit_rms_and_library():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((5, 64)) * 3
    y = om.rmsnorm(h, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(axis=1)), 1.0, rtol=1e-12)
    g = rng.standard_normal(64)
    ref = F.rms_norm(torch.tensor(h), (64,), torch.tensor(g), eps=1e-5).numpy()
    np.testing.assert_allclose(om.rmsnorm(h, g, 1e-5), ref, rtol=1e-12, atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 2, 32))
    np.testing.assert_allclose(om.rope(x, np.zeros(3), 10000.0), x, atol=0)
    y = om.rope(x, np.array([1, 17, 4000]), 10000.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    # q_m . k_n depends only on m - n
    q = rng.standard_normal((1, 1, 32))
    k = rng.standard_normal((1, 1, 32))
    dots = []
    for m, n in [(5, 2), (105, 102), (3003, 3000)]:
        qm = om.rope(q, np.array([m]), 10000.0)
        kn = om.rope(k, np.array([n]), 10000.0)
        dots.append(float((qm * kn).sum()))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-9)


def test_rope_equals_complex_rotation():
    # Pair (j, j+hd/2) as the complex number x_j + i x_{j+hd/2}, multiplied by e^{i pos theta_j}.
    rng = np.random.default_rng(3)
    hd = 64
    x = rng.standard_normal((4, 3, hd))
    pos = np.array([0, 1, 77, 2049])
    theta = 10000.0 ** (-np.arange(hd // 2) * 2.0 / hd)
    z = (x[..., : hd // 2] + 1j * x[..., hd // 2:]) * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    ref = np.concatenate([z.real, z.imag], axis=-1)
    np.testing.assert_allclose(om.rope(x, pos, 10000.0), ref, rtol=1e-12, atol=1e-12)


def test_silu_library():
    z = np.linspace(-20, 20, 1001)
    np.testing.assert_allclose(om.silu(z), F.silu(torch.tensor(z)).numpy(), rtol=1e-13, atol=1e-300)


@pytest.mark.parametrize("nh,nkv", [(4, 4), (8, 2)])
def test_attention_block_vs_sdpa(nh, nkv):
    rng = np.random.default_rng(4)
    n, T, hd = 5, 37, 16
    q = rng.standard_normal((n, nh, hd))
    K = rng.standard_normal((T, nkv, hd))
    V = rng.standard_normal((T, nkv, hd))
    q_pos = np.arange(T - n, T)
    out = om.attention_block(q, K, V, q_pos, nkv)
    group = nh // nkv
    Kr = np.repeat(K, group, axis=1)  # kv head for q head h is h // group
    Vr = np.repeat(V, group, axis=1)
    mask = np.arange(T)[None, :] <= q_pos[:, None]
    ref = F.scaled_dot_product_attention(
        torch.tensor(q).permute(1, 0, 2), torch.tensor(Kr).permute(1, 0, 2), torch.tensor(Vr).permute(1, 0, 2),
        attn_mask=torch.tensor(mask)).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 4, 8))
    K = rng.standard_normal((1, 2, 8))
    V = rng.standard_normal((1, 2, 8))
    out = om.attention_block(q, K, V, np.array([0]), 2)
    np.testing.assert_allclose(out[0], np.repeat(V[0], 2, axis=0), rtol=1e-15)


def _tiny():
    shape = synth.TINY
    return shape, synth.make_weights(shape)


def test_one_layer_first_token_closed_form():
    # With one layer and an empty cache, attention returns the stored v of the token itself.
    shape, W = _tiny()
    m = om.Model(shape, W, n_layers=1)
    kv = om.KVCache(shape, 1, 8)
    tok = 17
    logits = m.decode_step(tok, 0, kv)
    L = W["layers"][0]
    f = lambda a: np.asarray(a, np.float64)
    h = f(W["embed"][tok])
    x = h / np.sqrt((h * h).mean() + shape.rms_eps) * f(L["attn_norm"])
    v = om.store_kv(x @ f(L["wv"]).T, "f32")  # per head, kv head == q head here
    h = h + v @ f(L["wo"]).T
    x = h / np.sqrt((h * h).mean() + shape.rms_eps) * f(L["ffn_norm"])
    g = x @ f(L["w_gate"]).T
    h = h + (g / (1 + np.exp(-g)) * (x @ f(L["w_up"]).T)) @ f(L["w_down"]).T
    x = h / np.sqrt((h * h).mean() + shape.rms_eps) * f(W["final_norm"])
    np.testing.assert_allclose(logits, x @ f(W["lm_head"]).T, rtol=1e-10, atol=1e-12)


def test_verify_block_equals_sequential_steps():
    shape, W = _tiny()
    m = om.Model(shape, W)
    prompt = synth.make_prompt(20, shape.vocab)[0]
    kv_a = om.KVCache(shape, shape.n_layers, 64)
    m.prefill(prompt, kv_a)
    kv_b = kv_a.copy()
    toks = [5, 99, 300, 7, 511]
    block = m.forward_block(toks, kv_a.length, kv_a)
    seq = np.stack([m.decode_step(t, kv_b.length + i, kv_b) for i, t in enumerate(toks)])
    np.testing.assert_allclose(block, seq, rtol=1e-11, atol=1e-11)
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(kv_a.k[l], kv_b.k[l])
        np.testing.assert_array_equal(kv_a.v[l], kv_b.v[l])


def test_draft_is_target_prefix():
    shape, W = _tiny()
    full = om.Model(shape, W, n_layers=1)
    view = om.Model(shape, synth.draft_view(W, 1))
    kv1 = om.KVCache(shape, 1, 8)
    kv2 = om.KVCache(shape, 1, 8)
    np.testing.assert_array_equal(full.forward_block([1, 2, 3], 0, kv1), view.forward_block([1, 2, 3], 0, kv2))


def test_bf16_kv_rounding_is_the_only_mirror_point():
    # A bf16 model stores K/V rounded to bf16; widening then re-rounding is a no-op.
    shape = synth.ModelShape(1, 64, 2, 1, 32, 128, 97, dtype="bf16")
    W = synth.make_weights(shape)
    m = om.Model(shape, W)
    kv = om.KVCache(shape, 1, 8)
    m.forward_block([3, 4], 0, kv)
    k = kv.k[0][:2].astype(np.float64)
    np.testing.assert_array_equal(om.round_to_bf16(k), k)


def test_greedy_specdec_equals_greedy_decode():
    shape, W = _tiny()
    target = om.Model(shape, W)
    draft = om.Model(shape, W, n_layers=1)
    prompt = synth.make_prompt(64, shape.vocab)[0]
    ref = greedy_decode(target, prompt, 32, capacity=128)
    s = Sequence(target, draft, capacity=128)
    s.prefill(prompt)
    step = 0
    while len(s.emitted) < 32:
        s.iterate(4, 0.0, seed=2, step=step)
        step += 1
    assert s.emitted[:32] == ref


def test_rollback_leaves_no_stale_state():
    # After sampled iterations, the committed cache equals a fresh prefill over the committed text.
    shape, W = _tiny()
    target = om.Model(shape, W)
    draft = om.Model(shape, W, n_layers=1)
    prompt = list(synth.make_prompt(16, shape.vocab)[0])
    s = Sequence(target, draft, capacity=96)
    s.prefill(prompt)
    for step in range(6):
        s.iterate(4, 1.0, seed=2, step=step)
    text = prompt + s.emitted
    # target: committed = text[:-1]; draft: committed = text[:len]
    fresh_t = om.KVCache(shape, shape.n_layers, 96)
    target.prefill(text[:-1], fresh_t)
    assert fresh_t.length == s.st_t.length
    for l in range(shape.n_layers):
        np.testing.assert_allclose(s.kv_t.k[l][: fresh_t.length], fresh_t.k[l][: fresh_t.length], rtol=1e-6, atol=1e-6)
        np.testing.assert_allclose(s.kv_t.v[l][: fresh_t.length], fresh_t.v[l][: fresh_t.length], rtol=1e-6, atol=1e-6)
    fresh_d = om.KVCache(shape, 1, 96)
    draft.prefill(text[: s.st_d.length], fresh_d)
    np.testing.assert_allclose(s.kv_d.k[0][: s.st_d.length], fresh_d.k[0][: s.st_d.length], rtol=1e-6, atol=1e-6)
    assert text[s.st_d.length:] == s.st_d.pending
