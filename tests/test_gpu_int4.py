"""INT4 weights on the GPU (the paper's model precision, Sec. 4.1): the device
quantizer's image decoded on the host equals the oracle's codes and scales bit
for bit, and verify / draft passes over INT4 layer weights match the float64
oracle run on the effective weights q * s (tolerance of the bf16 models)."""
import numpy as np
import pytest

from oracle import model as om
from oracle import quant
from paper_2608_10362_amd import binding, synth
from tests.gpu_util import i32, install_context, log, oracle_caches, torch_cuda

pytestmark = pytest.mark.gpu

TOL = 2e-2
ALIGN = 256


def _align(x):
    return (x + ALIGN - 1) // ALIGN * ALIGN


def _matrices(shape):
    q, kv, d, f = shape.q_dim, shape.kv_dim, shape.d_model, shape.ffn_dim
    return [("wq", q, d), ("wk", kv, d), ("wv", kv, d), ("wo", d, q), ("w_gate", f, d), ("w_up", f, d),
            ("w_down", d, f)]


def _decode(img, off, soff, N, K):
    """Codes [N, K] and scale bits [N, ceil(K/128)] of one INT4 matrix of the image
    (layout as documented with specdec_pack_weights_fmt)."""
    T, G = N // 16, (K + 127) // 128
    words = img[off:off + T * G * 1024].view(np.uint32).reshape(T, G, 4, 16, 4)  # [t][G][c][i][j]
    codes = np.stack([((words >> np.uint32(4 * e)) & np.uint32(0xF)).astype(np.int16) for e in range(8)], -1)
    codes = np.where(codes >= 8, codes - 16, codes).astype(np.int8)               # [t][G][c][i][j][e]
    q = codes.transpose(0, 3, 1, 4, 2, 5).reshape(N, G * 128)                     # row 16t+i, col 128G+32j+8c+e
    assert not q[:, K:].any()                                                     # columns past K hold 0
    q = q[:, :K]
    s = img[soff:soff + T * G * 32].view(np.uint16).reshape(T, G, 16).transpose(0, 2, 1).reshape(N, G)
    return q, s


def _rope_rows(n_rows, hd):
    """Source row of each packed row of Wq / Wk: tile t of a head holds the RoPE
    pairs' rows 8t..8t+7 and hd/2 + 8t .. +7."""
    rows = np.empty(n_rows, np.int64)
    for n in range(n_rows):
        t, e = n // 16, n % 16
        head, tq = (16 * t) // hd, (16 * t) % hd // 16
        rows[n] = head * hd + (8 * tq + e if e < 8 else hd // 2 + 8 * tq + e - 8)
    return rows


def test_device_quantizer_matches_the_oracle_bit_for_bit():
    torch_cuda()
    shape = synth.LLAMA_1B
    W = synth.make_weights(shape, n_layers=1)
    dw = binding.DeviceWeights(shape, W, weight_format="int4")
    img = dw.packed.cpu().numpy()
    off = _align(shape.vocab * shape.d_model * 2)  # the bf16 LM head comes first
    for name, N, K in _matrices(shape):
        frag = _align(off + (N // 16) * ((K + 127) // 128) * 1024)
        q, s = _decode(img, off, frag, N, K)
        off = _align(frag + (N // 16) * ((K + 127) // 128) * 32)
        src = W["layers"][0][name]
        if name in ("wq", "wk"):
            src = src[_rope_rows(N, shape.head_dim)]
        q_ref, s_ref = quant.quantize_int4(src)
        assert np.array_equal(s, s_ref), name
        assert np.array_equal(q, q_ref), name
    assert off == img.size
    log(f"INT4 image of one 1.1B layer ({img.size} bytes) equals the oracle's codes and scales")


def _int4_case(shape, n_layers, lengths, g, seed):
    torch = torch_cuda()
    B = len(lengths)
    capacity = int(np.ceil((max(lengths) + g + 1) / 64) * 64)
    W = synth.make_weights(shape, n_layers=n_layers)
    ctx = synth.make_kv_context(shape, n_layers, lengths)
    dw = binding.DeviceWeights(shape, W, weight_format="int4")
    target = binding.Model(dw, n_layers, max_rows=B * (g + 1), max_ctx=capacity)
    kv = binding.KVCache(target, B, capacity)
    install_context(kv, ctx, lengths, n_layers, shape.dtype)
    pend = synth.make_prompt(1, shape.vocab, batch=B, seed=seed + 31)[:, 0]
    kv.set_state(np.asarray(lengths, np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
    drafts = synth.make_prompt(g, shape.vocab, batch=B, seed=seed + 32)
    logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, i32(drafts), g, logits)
    got = logits.cpu().numpy()
    assert kv.read_state()["status"] == 0
    m = om.Model(shape, quant.int4_model_weights(W, n_layers), n_layers=n_layers)
    m_bf16 = om.Model(shape, W, n_layers=n_layers)
    caches = oracle_caches(shape, n_layers, ctx, lengths, capacity)
    caches2 = oracle_caches(shape, n_layers, ctx, lengths, capacity)
    worst, moved = 0.0, 0.0
    for b in range(B):
        toks = [int(pend[b])] + list(drafts[b])
        ref = m.forward_block(toks, int(lengths[b]), caches[b])
        worst = max(worst, float(np.abs(got[b] - ref).max()))
        moved = max(moved, float(np.abs(m_bf16.forward_block(toks, int(lengths[b]), caches2[b]) - ref).max()))
    log(f"INT4 verify d={shape.d_model} B={B}: max-abs logit error {worst:.3g} "
        f"(quantization moves the logits by up to {moved:.3g})")
    assert worst < TOL
    assert moved > 10 * worst  # the comparison is sensitive to the quantized weights, not the bf16 ones
    return dw, W


@pytest.mark.parametrize("g", [4, 8])
def test_int4_7b_shape_verify(g):
    # 5 rows: x of every 4096-column GEMM in one LDS window, the down projection
    # in two; 9 rows: every GEMM over several windows
    _int4_case(synth.LLAMA_7B, 2, [2048], g=g, seed=0)


@pytest.mark.parametrize("lengths,g", [([1, 64, 300, 129], 4), ([1, 64, 300, 129], 3), ([517], 4)])
def test_int4_1b_shape_verify(lengths, g):
    # 20 rows: the skinny kernel's INT4 path; 16 rows: one group per wave and
    # window; one sequence: two SwiGLU units per block, 6 groups per wave of
    # the 5632-column down projection
    _int4_case(synth.LLAMA_1B, 2, lengths, g=g, seed=1)


def test_int4_draft_step_greedy():
    torch = torch_cuda()
    shape = synth.LLAMA_1B
    W = synth.make_weights(shape, n_layers=2)
    dw = binding.DeviceWeights(shape, W, weight_format="int4")
    # max_rows 64: the prompts are prefilled in 64-row passes (2 x 32 tokens: the
    # INT4 GEMMs' 4-row-tile variants), then a 2-row draft step
    draft = binding.Model(dw, 1, max_rows=64, max_ctx=256)
    kv = binding.KVCache(draft, 2, 256)
    prompts = synth.make_prompt(70, shape.vocab, batch=2, seed=5)
    binding.specdec_prefill(draft, kv, i32(prompts))
    g = 3
    d_out = torch.zeros((2, g), dtype=torch.int32, device="cuda")
    lo = torch.empty((2, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_draft_step(draft, kv, g, 0, 0.0, 0, 0, None, None, d_out, g, lo)
    got = lo.cpu().numpy()
    m = om.Model(shape, quant.int4_model_weights(W, 1), n_layers=1)
    for b in range(2):
        c = om.KVCache(shape, 1, 256)
        m.prefill(prompts[b, :-1], c)
        ref = m.forward_block([int(prompts[b, -1])], c.length, c)[0]
        assert np.abs(got[b] - ref).max() < TOL
        k, v = kv.read_context(0, b, 0, 69)
        assert np.abs(k.float().cpu().numpy() - c.k[0][:69]).max() < 0.05
        assert np.abs(v.float().cpu().numpy() - c.v[0][:69]).max() < 0.05
        # greedy: the proposed token is the argmax of the proposing row
        assert int(d_out[b, 0]) == int(np.argmax(got[b]))
