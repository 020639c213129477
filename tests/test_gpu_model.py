"""GPU parity of the forward passes (verify and draft step) against the oracle.

Logits must agree within max-abs 1e-4 (float32 model) / 2e-2 (bf16 model),
under teacher forcing: both sides get the same weights, resident context and
drafted tokens.
"""
import dataclasses

import numpy as np
import pytest

from oracle import model as om
from oracle import sampling
from oracle.specdec import greedy_decode
from paper_2608_10362_amd import binding, synth
from tests.gpu_util import (SOFTMAX_REL_ERR, accept_explained, f32, i32, install_context, log, oracle_caches,
                            torch_cuda, u32_tensor)

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


# ---------------------------------------------------------------- tiny float32 model
@pytest.fixture(scope="module")
def tiny():
    torch_cuda()
    shape = synth.TINY
    W = synth.make_weights(shape)
    dw = binding.DeviceWeights(shape, W)
    target = binding.Model(dw, 2, max_rows=64, max_ctx=512)
    draft = binding.Model(dw, 1, max_rows=64, max_ctx=512)
    return shape, W, target, draft


def test_tiny_prefill_and_verify(tiny):
    torch = torch_cuda()
    shape, W, target, _ = tiny
    B, g = 3, 4
    prompts = synth.make_prompt(64, shape.vocab, batch=B)
    drafts = synth.make_prompt(g, shape.vocab, batch=B, seed=77)
    kv = binding.KVCache(target, B, 256)
    binding.specdec_prefill(target, kv, i32(prompts))
    st = kv.read_state()
    assert (st["len"] == 63).all() and (st["pending"][:, 1] == prompts[:, -1]).all() and st["status"] == 0
    logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, i32(drafts), g, logits)
    got = logits.cpu().numpy()
    m = om.Model(shape, W)
    worst = 0.0
    for b in range(B):
        c = om.KVCache(shape, 2, 256)
        m.prefill(prompts[b, :-1], c)
        ref = m.forward_block([prompts[b, -1]] + list(drafts[b]), c.length, c)
        err = float(np.abs(got[b] - ref).max())
        worst = max(worst, err)
        for l in range(2):
            k, v = kv.read_context(l, b, 0, 68)
            assert np.abs(k.cpu().numpy() - c.k[l][:68]).max() < TOL_F32
            assert np.abs(v.cpu().numpy() - c.v[l][:68]).max() < TOL_F32
    log(f"tiny verify max-abs logit error {worst:.3g}")
    assert worst < TOL_F32


@pytest.fixture(scope="module")
def tiny_wide():
    """The tiny float32 model with a 50000-token vocabulary: the softmax and
    draw run over 49 chunks of 1021 (last one ragged)."""
    torch_cuda()
    shape = dataclasses.replace(synth.TINY, vocab=50000)
    W = synth.make_weights(shape)
    dw = binding.DeviceWeights(shape, W)
    return shape, W, binding.Model(dw, 1, max_rows=16, max_ctx=256)


@pytest.mark.parametrize("wide,T", [(False, 1.0), (True, 1.0), (False, 0.8), (True, 0.8)])
def test_tiny_draft_steps(tiny, tiny_wide, wide, T):
    torch = torch_cuda()
    if wide:
        shape, W, draft = tiny_wide
    else:
        shape, W, _, draft = tiny
    g, seed, step = 4, 2, 9
    prompt = synth.make_prompt(40, shape.vocab)
    kv = binding.KVCache(draft, 1, 256)
    binding.specdec_prefill(draft, kv, i32(prompt))
    m = om.Model(shape, W, n_layers=1)
    c = om.KVCache(shape, 1, 256)
    m.prefill(prompt[0, :-1], c)
    for n_pending in (1, 2):
        if n_pending == 2:  # the draft is one position behind after an all-accepted iteration
            kv.set_state([38], [[prompt[0, -2], prompt[0, -1]]], [2])
            pend, start = [prompt[0, -2], prompt[0, -1]], 38
        else:
            kv.set_state([39], [[0, prompt[0, -1]]], [1])
            pend, start = [prompt[0, -1]], 39
        c2 = c.copy()
        d = torch.zeros((1, g), dtype=torch.int32, device="cuda")
        q = torch.zeros((1, g, shape.vocab), dtype=torch.float32, device="cuda")
        lo = torch.zeros((1, shape.vocab), dtype=torch.float32, device="cuda")
        mismatched = 0
        for s in range(g):
            binding.specdec_draft_step(draft, kv, g, s, T, seed, step, None, q, d, g, lo)
            if s == 0:
                ref = m.forward_block(pend, start, c2)[-1]
            else:
                ref = m.decode_step(int(d[0, s - 1].item()), start + len(pend) + s - 1, c2)
            err = float(np.abs(lo.cpu().numpy()[0] - ref).max())
            q_ref = sampling.softmax(ref, T)
            qerr = float(np.abs(q.cpu().numpy()[0, s] - q_ref).max())
            tok_ref = sampling.draft_sample_philox(q_ref.astype(np.float32), seed, 0, step, s)
            mismatched += int(d[0, s].item()) != tok_ref
            log(f"draft n_pending={n_pending} slot={s} logit err {err:.3g} q err {qerr:.3g}")
            assert err < TOL_F32 and qerr < 1e-5
        assert mismatched == 0


def test_tiny_greedy_specdec_equals_oracle_greedy_decode(tiny):
    torch = torch_cuda()
    shape, W, target, draft = tiny
    g, n_new = 4, 32
    prompt = synth.make_prompt(64, shape.vocab)
    ref = greedy_decode(om.Model(shape, W), prompt[0], n_new, capacity=256)
    kv_t = binding.KVCache(target, 1, 256)
    kv_d = binding.KVCache(draft, 1, 256)
    binding.specdec_prefill(target, kv_t, i32(prompt))
    binding.specdec_prefill(draft, kv_d, i32(prompt))
    sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, 0.0, seed=2)
    out, step = [], 0
    while len(out) < n_new:
        sd.step(step)
        A = int(sd.n_acc[0].item())
        out += [int(x) for x in sd.d[0, :A].cpu().numpy()] + [int(sd.next[0].item())]
        step += 1
    log(f"greedy SD: {step} iterations for {len(out)} tokens")
    assert out[:n_new] == ref
    st_t, st_d = kv_t.read_state(), kv_d.read_state()
    assert st_t["len"][0] == 63 + len(out) and st_t["status"] == 0
    assert st_d["len"][0] + st_d["n_pending"][0] == st_t["len"][0] + 1


def test_tiny_verify_equals_sequential_steps(tiny):
    torch = torch_cuda()
    shape, W, target, _ = tiny
    g = 4
    prompt = synth.make_prompt(30, shape.vocab)
    toks = [int(prompt[0, -1])] + [11, 200, 3, 509]
    kv = binding.KVCache(target, 1, 256)
    binding.specdec_prefill(target, kv, i32(prompt))
    block = torch.empty((1, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, i32(np.array([toks[1:]])), g, block)
    one = torch.empty((1, 1, shape.vocab), dtype=torch.float32, device="cuda")
    rows = []
    for i, t in enumerate(toks):
        kv.set_state([29 + i], [[0, t]], [1])
        binding.specdec_verify(target, kv, 0, None, 0, one)
        rows.append(one.cpu().numpy()[0, 0].copy())
    seq = np.stack(rows)
    diff = float(np.abs(block.cpu().numpy()[0] - seq).max())
    log(f"verify block vs sequential steps max diff {diff:.3g} (bitwise={diff == 0.0})")
    assert diff <= 1e-6


def test_tiny_graph_of_whole_iterations_draws_fresh_words_each_replay(tiny):
    """One captured HIP graph of a whole sampled iteration (gamma draft steps,
    verify, accept, both commits), replayed R times with no library call in
    between: the Philox step comes from the target cache's commit counter, so
    replay i must equal the eager iteration run at explicit step c0 + i, token
    for token and bit for bit, and differ from iterations that reuse one step."""
    torch = torch_cuda()
    shape, W, target, draft = tiny
    B, g, R, T, cap = 2, 4, 5, 1.0, 256
    prompts = synth.make_prompt(48, shape.vocab, batch=B, seed=31)
    kv_t = binding.KVCache(target, B, cap)
    kv_d = binding.KVCache(draft, B, cap)
    binding.specdec_prefill(target, kv_t, i32(prompts))
    binding.specdec_prefill(draft, kv_d, i32(prompts))
    torch.cuda.synchronize()
    c0 = kv_t.read_step()
    assert c0 == 0
    # the host bound every launch below is sized from: the one R iterations reach
    bound_t, bound_d = kv_t.kv.len_upper + R * (g + 1), kv_d.kv.len_upper + R * (g + 1)
    saved_t, saved_d = kv_t.state.clone(), kv_d.state.clone()

    def restore():
        kv_t.state.copy_(saved_t)
        kv_d.state.copy_(saved_d)
        kv_t.kv.len_upper, kv_d.kv.len_upper = bound_t, bound_d

    def snap(sd):
        return [x.clone() for x in (sd.d, sd.n_acc, sd.next, sd.q)]

    def eager(steps):
        sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, T, seed=3)
        restore()
        out = []
        for st in steps:
            kv_t.kv.len_upper, kv_d.kv.len_upper = bound_t, bound_d
            sd.step(st)
            out.append(snap(sd))
        torch.cuda.synchronize()
        return out, kv_t.read_state(), kv_t.read_step()

    ref, ref_state, ref_count = eager([c0 + i for i in range(R)])
    assert ref_count == c0 + R          # every commit counts, whatever step the draws used
    stale, _, _ = eager([c0] * R)
    sdg = binding.SpecDecoder(target, draft, kv_t, kv_d, g, T, seed=3, device_step=True)
    assert sdg.step_dev == kv_t.step_word()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):       # warm-up launch off the capture
        restore()
        sdg.step(0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    restore()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sdg.step(0)
    restore()
    torch.cuda.synchronize()
    got = []
    for r in range(R):
        graph.replay()
        torch.cuda.synchronize()
        got.append(snap(sdg))
    n_acc = [[int(a) for a in x[1].cpu().numpy()] for x in got]
    same = [all(torch.equal(a, b) for a, b in zip(x, y)) for x, y in zip(got, ref)]
    fresh = [not all(torch.equal(a, b) for a, b in zip(x, y)) for x, y in zip(got, stale)]
    log(f"graph replays: accepted {n_acc}; equal to eager at steps c0+i {same}; differ from step c0 {fresh}")
    assert all(same)
    assert any(fresh[1:]) and not fresh[0]
    st = kv_t.read_state()
    assert (st["len"] == ref_state["len"]).all() and (st["pending"] == ref_state["pending"]).all()
    assert st["status"] == 0 and kv_t.read_step() == c0 + R


# ---------------------------------------------------------------- bf16 Llama-shaped prefixes
def _bf16_case(shape, n_layers, lengths, g, seed=0, capacity=None, return_logits=False):
    torch = torch_cuda()
    B = len(lengths)
    capacity = capacity or int(np.ceil((max(lengths) + g + 1) / 64) * 64)
    log(f"bf16 case d={shape.d_model} L={n_layers} B={B} ctx={list(lengths)[:4]} g={g}")
    W = synth.make_weights(shape, n_layers=n_layers)
    ctx = synth.make_kv_context(shape, n_layers, lengths)
    dw = binding.DeviceWeights(shape, W)
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
    m = om.Model(shape, W, n_layers=n_layers)
    caches = oracle_caches(shape, n_layers, ctx, lengths, capacity)
    worst = 0.0
    refs = []
    for b in range(B):
        ref = m.forward_block([int(pend[b])] + list(drafts[b]), int(lengths[b]), caches[b])
        refs.append(ref)
        worst = max(worst, float(np.abs(got[b] - ref).max()))
        # the drafted tokens' K/V were appended at [len, len+g]
        k, v = kv.read_context(n_layers - 1, b, int(lengths[b]), g + 1)
        kf = k.float().cpu().numpy()
        assert np.abs(kf - caches[b].k[n_layers - 1][lengths[b]:lengths[b] + g + 1]).max() < 0.05
    log(f"bf16 verify max-abs logit error {worst:.3g}")
    assert worst < TOL_BF16
    if return_logits:
        return got, np.stack(refs), drafts
    return worst


def test_bf16_1b_shape_verify():
    _bf16_case(synth.LLAMA_1B, 2, [517], g=4)


def test_bf16_1b_shape_ragged_batch():
    _bf16_case(synth.LLAMA_1B, 2, [1, 64, 300, 129], g=4, seed=1)


@pytest.mark.parametrize("g", [2, 4, 8])
def test_bf16_7b_shape_verify(g):
    _bf16_case(synth.LLAMA_7B, 2, [2048], g=g)


@pytest.fixture(scope="module")
def llama7b_2layer():
    torch_cuda()
    shape = synth.LLAMA_7B
    W = synth.make_weights(shape, n_layers=2)
    dw = binding.DeviceWeights(shape, W)
    return shape, binding.Model(dw, 2, max_rows=5, max_ctx=2240)


@pytest.mark.parametrize("length,bitwise", [(2171, True), (2172, False)])
def test_bf16_7b_shape_verify_block_vs_steps_across_an_attention_partition_change(llama7b_2layer, length, bitwise):
    """The attention kernel splits a head's keys into parts from the context
    bound (the block's bound is len + gamma + 1, a one-row step's len + i + 1),
    and its partials are merged part by part.  At len 2171 the block and its
    five one-row steps get the same partition (8 parts of 8 sub-chunks) and the
    block must equal the steps bit for bit; at len 2172 the block's bound
    (2177 keys, 69 sub-chunks) takes 11 parts of 6 while the first four steps
    keep 8 of 8, so the merge order differs and the rows agree within float32
    rounding of the attention sums instead."""
    torch = torch_cuda()
    shape, target = llama7b_2layer
    g, cap = 4, 2240
    ctx = synth.make_kv_context(shape, 2, [length])
    kv = binding.KVCache(target, 1, cap)
    install_context(kv, ctx, [length], 2, shape.dtype)
    pend = int(synth.make_prompt(1, shape.vocab, seed=51)[0, 0])
    drafts = [int(t) for t in synth.make_prompt(g, shape.vocab, seed=52)[0]]
    kv.set_state([length], [[0, pend]], [1])
    block = torch.empty((1, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, i32(np.array([drafts])), g, block)
    one = torch.empty((1, 1, shape.vocab), dtype=torch.float32, device="cuda")
    rows = []
    for i, t in enumerate([pend] + drafts):
        kv.set_state([length + i], [[0, t]], [1])
        binding.specdec_verify(target, kv, 0, None, 0, one)
        rows.append(one.cpu().numpy()[0, 0].copy())
    b = block.cpu().numpy()[0]
    diffs = [float(np.abs(b[i] - rows[i]).max()) for i in range(g + 1)]
    log(f"len {length}: block vs one-row steps max diff per row {diffs}")
    if bitwise:
        assert max(diffs) == 0.0
    else:
        assert max(diffs) <= 1e-4


def test_bf16_7b_shape_multi_request_ragged():
    # 16 sequences, ragged contexts, gamma 6: 112 rows (one launch of the wide GEMMs)
    lengths = synth.make_ragged_lengths(16, 40, 400)
    _bf16_case(synth.LLAMA_7B, 1, list(lengths), g=6, seed=2)


@pytest.mark.parametrize("B,g", [(2, 3), (2, 7), (3, 4)])
def test_bf16_1b_shape_stacked_operand_row_counts(B, g):
    # 8, 16 and 15 rows: passes of at most 16 rows hand x between kernels as the
    # stacked bf16 operand, one fragment (hi and lo rows of one MFMA) up to 8
    # rows and two fragments above; K = 2048 also takes the LDS-resident form
    lengths = synth.make_ragged_lengths(B, 50, 300, seed=7)
    _bf16_case(synth.LLAMA_1B, 2, list(lengths), g=g, seed=6)


@pytest.mark.parametrize("B,g", [(7, 4), (8, 7)])
def test_bf16_1b_shape_skinny_row_tiles(B, g):
    # 35 and 64 rows: the skinny kernels' four-row-tile variants (float32 x, no
    # stacked operand), up to the largest pass before the wide kernels (65 rows)
    lengths = synth.make_ragged_lengths(B, 1, 300, seed=9)
    _bf16_case(synth.LLAMA_1B, 2, list(lengths), g=g, seed=4)


def test_bf16_7b_shape_many_short_sequences():
    # 10 sequences of at most ~250 keys, gamma 6 (70 rows): more (kv head,
    # sequence) units than CUs and fewer than 12 sub-chunks of 32 keys per
    # sequence, so every attention part is a whole sequence, one wave per sub-chunk
    lengths = synth.make_ragged_lengths(10, 100, 250, seed=6)
    _bf16_case(synth.LLAMA_7B, 1, list(lengths), g=6, seed=5)


def test_bf16_7b_shape_long_context_looping_attention():
    # 2 sequences of 4500 and 6100 keys: 188 sub-chunks of 32 keys over 64
    # (kv head, sequence) units -> parts of 8 sub-chunks on 4-wave blocks, each
    # wave looping over 2 sub-chunks with the online softmax
    _bf16_case(synth.LLAMA_7B, 1, [4500, 6100], g=4, seed=4)


def test_bf16_7b_shape_attention_combine_modes_alternate_on_one_handle():
    # One model handle, two caches: 2 sequences of 4500 and 6100 keys (looping
    # attention: the fixed combining block polls tagged partial words, and the
    # launch advances the per-(sequence, tile, kv head) epochs) and one of 2048
    # keys (one-round attention: the last block to count combines).  Verifies
    # alternate between the two several times; every repeat of a verify from the
    # same state must give the same logits bit for bit, and the first of each
    # must match the oracle.
    torch = torch_cuda()
    shape, n_layers, g = synth.LLAMA_7B, 1, 4
    W = synth.make_weights(shape, n_layers=n_layers)
    dw = binding.DeviceWeights(shape, W)
    cases = [[4500, 6100], [2048]]
    cap = int(np.ceil((max(max(c) for c in cases) + g + 1) / 64) * 64)
    target = binding.Model(dw, n_layers, max_rows=2 * (g + 1), max_ctx=cap)
    m = om.Model(shape, W, n_layers=n_layers)
    setups = []
    for ci, lengths in enumerate(cases):
        B = len(lengths)
        ctx = synth.make_kv_context(shape, n_layers, lengths, seed=40 + ci)
        kv = binding.KVCache(target, B, cap)
        install_context(kv, ctx, lengths, n_layers, shape.dtype)
        pend = synth.make_prompt(1, shape.vocab, batch=B, seed=50 + ci)[:, 0]
        drafts = synth.make_prompt(g, shape.vocab, batch=B, seed=60 + ci)
        setups.append((lengths, ctx, kv, pend, drafts))

    def verify(ci):
        lengths, _, kv, pend, drafts = setups[ci]
        B = len(lengths)
        kv.set_state(np.asarray(lengths, np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
        logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
        binding.specdec_verify(target, kv, g, i32(drafts), g, logits)
        out = logits.cpu().numpy()
        assert kv.read_state()["status"] == 0
        return out

    first = [verify(0), verify(1)]
    for ci, (lengths, ctx, _, pend, drafts) in enumerate(setups):
        caches = oracle_caches(shape, n_layers, ctx, lengths, cap)
        for b in range(len(lengths)):
            ref = m.forward_block([int(pend[b])] + list(drafts[b]), int(lengths[b]), caches[b])
            err = float(np.abs(first[ci][b] - ref).max())
            log(f"case {ci} seq {b} ctx {lengths[b]}: max-abs logit error {err:.3g}")
            assert err < TOL_BF16
    for rep in range(3):
        for ci in (0, 1, 0):
            got = verify(ci)
            assert np.array_equal(got, first[ci]), (rep, ci)


def test_bf16_7b_shape_long_context_workload_launch_and_accept():
    # The exact launch of the 16-sequence long-context workload: contexts drawn
    # from U[1024, 8192] with the lengths seed (up to 8022 keys), gamma 6 (112
    # rows: the wide GEMMs and the looping attention), then the temperature-0.8
    # accept on the device's verify logits (LOGITS mode) against the oracle's
    # accept on its own logits, with synthetic draft distributions and words.
    torch = torch_cuda()
    B, g, V, T = 16, 6, synth.LLAMA_7B.vocab, 0.8
    lengths = synth.make_ragged_lengths(B, 1024, 8192)
    got, refs, _ = _bf16_case(synth.LLAMA_7B, 1, list(lengths), g=g, seed=8, return_logits=True)
    err = float(np.abs(got - refs).max())
    rng = np.random.default_rng(15)
    q = sampling.softmax(rng.standard_normal((B, g, V)) * 1.3 + refs[:, :g] * 0.5, T).astype(np.float32)
    d = np.array([[sampling.sample_fixed_point(q[b, i], int(rng.integers(0, 2 ** 32))) for i in range(g)]
                  for b in range(B)], np.int32)
    words = synth.make_rand_u32((B, g + 1), seed=14)
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    binding.specdec_accept(B, g, V, binding.INPUT_LOGITS, T, f32(got), f32(q), i32(d), g, u32_tensor(words), 0, 0,
                           nacc, nxt)
    A_dev, n_dev = nacc.cpu().numpy(), nxt.cpu().numpy()
    # the device's softmax starts from its own logits: exp(dl / T) moves a probability,
    # and its normaliser, by at most about err / T each
    rel = 2 * err / T + SOFTMAX_REL_ERR
    kinds = []
    for b in range(B):
        p = sampling.softmax(refs[b], T).astype(np.float32)
        kind, detail = accept_explained(p, q[b], d[b], words[b], A_dev[b], n_dev[b], rel=rel)
        log(f"seq {b} ctx {lengths[b]}: A device {A_dev[b]} next {n_dev[b]}: {kind} {detail}")
        kinds.append(kind)
    assert "mismatch" not in kinds and kinds.count("boundary") <= 2
    assert len(set(A_dev.tolist())) > 1  # ragged acceptance: commit/rollback differ per sequence


@pytest.mark.parametrize("B,g", [(13, 4), (16, 7), (25, 7)])
def test_bf16_1b_shape_wide_rows(B, g):
    # 65, 128 and 200 rows (128 + 72 in two launches): the wide GEMM path with
    # its 4-, 7- and 8-tile row variants, split-K residual GEMMs, head_dim 64 RoPE
    lengths = synth.make_ragged_lengths(B, 1, 300, seed=5)
    _bf16_case(synth.LLAMA_1B, 2, list(lengths), g=g, seed=3)


# ---------------------------------------------------------------- prefill in large chunks
@pytest.mark.parametrize("shape_name,B,rows,n", [("LLAMA_1B", 2, 256, 301), ("LLAMA_7B", 1, 256, 301),
                                                  ("LLAMA_1B", 2, 600, 301)])
def test_bf16_prefill_in_large_chunks(shape_name, B, rows, n):
    """Prefill of n-1 prompt tokens per sequence in chunks of rows/B tokens
    (1.1B: 128-token chunks of 2 sequences = 256-row passes, GQA with 64 query
    tiles per kv head; 7B: 256-token chunks, MHA; 1.1B in one 600-row pass:
    launches of three 256-row tiles, the last partial), then a verify: the
    caches and the verify logits against the oracle's prefill."""
    torch = torch_cuda()
    shape = getattr(synth, shape_name)
    L, g = 2, 4
    cap = 384
    W = synth.make_weights(shape, n_layers=L)
    dw = binding.DeviceWeights(shape, W)
    target = binding.Model(dw, L, max_rows=rows, max_ctx=cap)
    kv = binding.KVCache(target, B, cap)
    prompts = synth.make_prompt(n, shape.vocab, batch=B, seed=41)
    drafts = synth.make_prompt(g, shape.vocab, batch=B, seed=42)
    binding.specdec_prefill(target, kv, i32(prompts))
    st = kv.read_state()
    assert (st["len"] == n - 1).all() and (st["pending"][:, 1] == prompts[:, -1]).all() and st["status"] == 0
    logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, i32(drafts), g, logits)
    got = logits.cpu().numpy()
    m = om.Model(shape, W, n_layers=L)
    worst, worst_kv = 0.0, 0.0
    for b in range(B):
        c = om.KVCache(shape, L, cap)
        m.prefill(prompts[b, :-1], c)
        ref = m.forward_block([prompts[b, -1]] + list(drafts[b]), c.length, c)
        worst = max(worst, float(np.abs(got[b] - ref).max()))
        for layer in range(L):
            k, v = kv.read_context(layer, b, 0, n - 1)
            worst_kv = max(worst_kv, float(np.abs(k.float().cpu().numpy() - c.k[layer][:n - 1]).max()),
                           float(np.abs(v.float().cpu().numpy() - c.v[layer][:n - 1]).max()))
    log(f"{shape_name} prefill B={B} chunk {rows // B}: verify max-abs logit error {worst:.3g}, K/V {worst_kv:.3g}")
    assert worst < TOL_BF16 and worst_kv < 0.05


# ---------------------------------------------------------------- context copy and errors
def test_kv_context_roundtrip_is_exact(tiny):
    torch = torch_cuda()
    shape, _, target, _ = tiny
    kv = binding.KVCache(target, 2, 128)
    k = torch.randn((50, shape.n_kv_heads, shape.head_dim), device="cuda")
    v = torch.randn((50, shape.n_kv_heads, shape.head_dim), device="cuda")
    kv.write_context(1, 1, 10, k, v)
    k2, v2 = kv.read_context(1, 1, 10, 50)
    assert torch.equal(k, k2) and torch.equal(v, v2)
    with pytest.raises(binding.SpecdecError):
        kv.read_context(1, 1, 100, 50)


def test_device_and_host_errors(tiny):
    torch = torch_cuda()
    shape, _, target, _ = tiny
    kv = binding.KVCache(target, 1, 128)
    kv.set_state([10], [[0, 5]], [1])
    logits = torch.empty((1, 5, shape.vocab), dtype=torch.float32, device="cuda")
    bad = i32(np.array([[1, 2, shape.vocab + 3, 4]]))
    binding.specdec_verify(target, kv, 4, bad, 4, logits)
    assert binding.specdec_device_status(kv) == -7
    kv.set_state([124], [[0, 5]], [1])
    with pytest.raises(binding.SpecdecError) as e:
        binding.specdec_verify(target, kv, 4, i32(np.array([[1, 2, 3, 4]])), 4, logits)
    assert e.value.status == -3
    with pytest.raises(ValueError):
        binding.specdec_verify(target, kv, 4, np.array([[1, 2, 3, 4]], np.int32), 4, logits)
