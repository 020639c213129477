"""GPU checks of the whole 7B-shaped bf16 target (all 32 layers) at its benchmark
workload: batch 1, resident context of 2048 positions, gamma 2 / 4 / 8, the
4-layer draft that shares the embedding and LM head.

- the verify logits of the 32-layer model against the float64 oracle's forward
  (teacher forcing on the drafted tokens), and the K/V appended by the last layer;
- the draft's single-token steps (temperatures 1 and 0.8) against the oracle;
- the verify block against gamma+1 one-row verifies, bit for bit (Sec. 2: one
  target pass over the drafted block gives the same per-position distributions as
  decoding them one at a time; every reduction here has a fixed order that does not
  depend on the number of rows);
- replays of a HIP graph of verify + accept, the launch form the benchmark times,
  against the eager launches, bit for bit;
- greedy speculative decoding emits the target's own greedy decode, token for token.

The weights take about 13.5 GB on the host and the oracle's forward 20-40 s, so
the module allows several minutes.
"""
import numpy as np
import pytest

from oracle import model as om
from oracle import sampling
from paper_2608_10362_amd import binding, synth
from oracle.philox import PURPOSE_DRAFT, draw_u32
from tests.gpu_util import draw_near_boundary, i32, install_context, log, oracle_caches, torch_cuda

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

TOL_BF16 = 2e-2
SHAPE = synth.LLAMA_7B
CTX = 2048
DRAFT_LAYERS = 4
G_MAX = 8
CAP = ((CTX + G_MAX + 64 + 63) // 64) * 64   # room for a greedy run of 64 tokens


@pytest.fixture(scope="module")
def full7b():
    torch = torch_cuda()
    log(f"drawing the 32-layer 7B-shaped weights and a {CTX}-position context")
    W = synth.make_weights(SHAPE)
    ctx = synth.make_kv_context(SHAPE, SHAPE.n_layers, [CTX])
    dw = binding.DeviceWeights(SHAPE, W)
    target = binding.Model(dw, SHAPE.n_layers, max_rows=G_MAX + 1, max_ctx=CAP)
    draft = binding.Model(dw, DRAFT_LAYERS, max_rows=G_MAX + 1, max_ctx=CAP)
    kv_t = binding.KVCache(target, 1, CAP)
    kv_d = binding.KVCache(draft, 1, CAP)
    install_context(kv_t, ctx, [CTX], SHAPE.n_layers, SHAPE.dtype)
    install_context(kv_d, ctx, [CTX], DRAFT_LAYERS, SHAPE.dtype)
    torch.cuda.synchronize()
    log("model and caches on the device")
    return W, ctx, target, draft, kv_t, kv_d


def _pending(seed=31):
    return int(synth.make_prompt(1, SHAPE.vocab, seed=seed)[0, 0])


def _set(kv, length, pend):
    kv.set_state(np.array([length], np.int32), np.array([[0, pend]], np.int32), np.ones(1, np.int32))


def test_full_7b_verify_matches_oracle(full7b):
    torch = torch_cuda()
    W, ctx, target, _, kv_t, _ = full7b
    g = 4
    pend = _pending()
    drafts = synth.make_prompt(g, SHAPE.vocab, seed=32)
    _set(kv_t, CTX, pend)
    logits = torch.empty((1, g + 1, SHAPE.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv_t, g, i32(drafts), g, logits)
    got = logits.cpu().numpy()[0]
    assert kv_t.read_state()["status"] == 0
    k_dev, v_dev = kv_t.read_context(SHAPE.n_layers - 1, 0, CTX, g + 1)
    log("oracle forward over 32 layers")
    m = om.Model(SHAPE, W)
    cache = oracle_caches(SHAPE, SHAPE.n_layers, ctx, [CTX], CAP)[0]
    ref = m.forward_block([pend] + [int(t) for t in drafts[0]], CTX, cache)
    err = float(np.abs(got - ref).max())
    kerr = float(np.abs(k_dev.float().cpu().numpy() - cache.k[-1][CTX:CTX + g + 1]).max())
    verr = float(np.abs(v_dev.float().cpu().numpy() - cache.v[-1][CTX:CTX + g + 1]).max())
    log(f"32-layer verify: max-abs logit error {err:.3g} (logit range {ref.min():.2f}..{ref.max():.2f}); "
        f"last-layer K/V error {kerr:.3g} / {verr:.3g}")
    assert err < TOL_BF16
    assert kerr < 0.05 and verr < 0.05
    # the greedy decision of every position is the oracle's unless its top two are within the error
    for i in range(g + 1):
        top2 = np.sort(ref[i])[-2:]
        if top2[1] - top2[0] > 2 * err:
            assert int(np.argmax(got[i])) == int(np.argmax(ref[i]))


@pytest.mark.parametrize("T", [1.0, 0.8])
def test_full_7b_draft_steps_match_oracle(full7b, T):
    torch = torch_cuda()
    W, ctx, _, draft, _, kv_d = full7b
    g, seed, step = 4, 7, 3
    pend = _pending(33)
    _set(kv_d, CTX, pend)
    m = om.Model(SHAPE, W, n_layers=DRAFT_LAYERS)
    cache = oracle_caches(SHAPE, DRAFT_LAYERS, ctx, [CTX], CAP)[0]
    d = torch.zeros((1, g), dtype=torch.int32, device="cuda")
    q = torch.zeros((1, g, SHAPE.vocab), dtype=torch.float32, device="cuda")
    lo = torch.zeros((1, SHAPE.vocab), dtype=torch.float32, device="cuda")
    for s in range(g):
        binding.specdec_draft_step(draft, kv_d, g, s, T, seed, step, None, q, d, g, lo)
        if s == 0:
            ref = m.forward_block([pend], CTX, cache)[-1]
        else:  # teacher forcing: the oracle takes the device's proposal
            ref = m.decode_step(int(d[0, s - 1].item()), CTX + s, cache)
        err = float(np.abs(lo.cpu().numpy()[0] - ref).max())
        q_ref = sampling.softmax(ref, T)
        qerr = float(np.abs(q.cpu().numpy()[0, s] - q_ref).max())
        tok_ref = sampling.draft_sample_philox(q_ref.astype(np.float32), seed, 0, step, s)
        log(f"4-layer draft slot {s}: logit error {err:.3g}, q error {qerr:.3g}, "
            f"token {int(d[0, s].item())} (oracle {tok_ref})")
        assert err < TOL_BF16 and qerr < 1e-4
        if int(d[0, s].item()) != tok_ref:  # only where the oracle's draw is within the q error of an edge
            word = draw_u32(seed, 0, step, PURPOSE_DRAFT, s)
            assert draw_near_boundary(q_ref, word, tok_ref, rel=max(1e-5, 2 * qerr / float(q_ref.max())))


@pytest.mark.parametrize("g", [2, 4, 8])
def test_full_7b_verify_block_equals_one_row_verifies(full7b, g):
    torch = torch_cuda()
    _, _, target, _, kv_t, _ = full7b
    pend = _pending()
    drafts = [int(t) for t in synth.make_prompt(g, SHAPE.vocab, seed=40 + g)[0]]
    _set(kv_t, CTX, pend)
    block = torch.empty((1, g + 1, SHAPE.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv_t, g, i32(np.array([drafts])), g, block)
    one = torch.empty((1, 1, SHAPE.vocab), dtype=torch.float32, device="cuda")
    rows = []
    for i, t in enumerate([pend] + drafts):
        _set(kv_t, CTX + i, t)
        binding.specdec_verify(target, kv_t, 0, None, 0, one)
        rows.append(one.cpu().numpy()[0, 0].copy())
    blk, seq = block.cpu().numpy()[0], np.stack(rows)
    diff = float(np.abs(blk - seq).max())
    log(f"gamma {g}: verify block vs {g + 1} one-row verifies, max diff {diff:.3g} (bitwise={diff == 0.0})")
    assert diff == 0.0
    assert kv_t.read_state()["status"] == 0


def test_full_7b_graph_replays_equal_eager_verify(full7b):
    torch = torch_cuda()
    _, _, target, draft, kv_t, kv_d = full7b
    g = 4
    pend = _pending()
    _set(kv_t, CTX, pend)
    _set(kv_d, CTX, pend)
    sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, 1.0, seed=synth.SEED_SAMPLING)
    saved_t, saved_d = kv_t.state.clone(), kv_d.state.clone()

    def eager():
        kv_t.state.copy_(saved_t)
        kv_d.state.copy_(saved_d)
        sd.draft_phase(5)
        sd.verify_phase(5)

    eager()
    torch.cuda.synchronize()
    ref = (sd.d.clone(), sd.logits.clone(), sd.n_acc.clone(), sd.next.clone())
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sd.verify_phase(5)
    torch.cuda.current_stream().wait_stream(side)
    eager()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sd.verify_phase(5)
    for r in range(3):
        eager()                         # the library's own eager work between replays
        sd.logits.zero_()
        sd.n_acc.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        same = [torch.equal(sd.logits, ref[1]), torch.equal(sd.n_acc, ref[2]), torch.equal(sd.next, ref[3])]
        log(f"graph replay {r}: logits/A/next bitwise equal to eager = {same}")
        assert all(same)
    assert int(sd.status.item()) == 0


@pytest.mark.parametrize("draft_layers", [DRAFT_LAYERS, 32])
def test_full_7b_greedy_specdec_emits_target_greedy_decode(full7b, draft_layers):
    """With the 4-layer draft almost every proposal is rejected; a draft that is the
    target itself has every proposal accepted (the all-accepted commit and the
    draft's two pending tokens on every iteration)."""
    torch = torch_cuda()
    _, ctx, target, draft, kv_t, kv_d = full7b
    if draft_layers != DRAFT_LAYERS:
        draft = binding.Model(target.dw, draft_layers, max_rows=G_MAX + 1, max_ctx=CAP)
        kv_d = binding.KVCache(draft, 1, CAP)
        install_context(kv_d, ctx, [CTX], draft_layers, SHAPE.dtype)
    g, n_new = 4, 48
    pend = _pending(34)
    # the target alone: one-row verifies, argmax, the next position
    one = torch.empty((1, 1, SHAPE.vocab), dtype=torch.float32, device="cuda")
    ref, t = [], pend
    for i in range(n_new):
        _set(kv_t, CTX + i, t)
        binding.specdec_verify(target, kv_t, 0, None, 0, one)
        t = int(np.argmax(one.cpu().numpy()[0, 0]))
        ref.append(t)
    # speculative decoding with the 4-layer draft, temperature 0
    _set(kv_t, CTX, pend)
    _set(kv_d, CTX, pend)
    sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, 0.0, seed=2)
    out, step = [], 0
    while len(out) < n_new:
        sd.step(step)
        A = int(sd.n_acc[0].item())
        out += [int(x) for x in sd.d[0, :A].cpu().numpy()] + [int(sd.next[0].item())]
        step += 1
        kv_t.read_state()   # refresh the host's bound on the lengths (a commit raises it by gamma+1)
        kv_d.read_state()
    log(f"greedy SD, {draft_layers}-layer draft: {step} iterations for {len(out)} tokens")
    # the verify rows are bitwise the one-row verifies, so the tokens are exactly the same
    assert out[:n_new] == ref
    st_t, st_d = kv_t.read_state(), kv_d.read_state()
    assert st_t["status"] == 0 and st_d["status"] == 0
    assert st_t["len"][0] == CTX + len(out)
    if draft_layers == SHAPE.n_layers:
        assert step == -(-n_new // (g + 1))   # every proposal accepted
