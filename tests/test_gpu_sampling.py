"""GPU parity of the integer-exact pieces: Philox draws, the fixed-point
sampler, accept / resample and KV commit -- bit-exact against the oracle when
fed identical probabilities and 32-bit words."""
import numpy as np
import pytest

from oracle import kvstate, philox, sampling
from paper_2608_10362_amd import binding, synth
from tests.gpu_util import accept_explained, f32, i32, log, torch_cuda, u32_tensor

pytestmark = pytest.mark.gpu


def test_draw_u32_bit_exact():
    torch = torch_cuda()
    B = 300
    out = torch.zeros(B, dtype=torch.int32, device="cuda")
    for seed, step, purpose, index in [(0, 0, 0, 0), (2, 17, 1, 3), (2 ** 40 + 5, 2 ** 33 + 9, 2, 0), (7, 1, 0, 31)]:
        log(f"draw seed={seed} step={step} purpose={purpose} index={index}")
        binding.specdec_draw_u32(B, seed, step, purpose, index, out)
        got = out.cpu().numpy().view(np.uint32)
        ref = [philox.draw_u32(seed, b, step, purpose, index) for b in range(B)]
        np.testing.assert_array_equal(got, np.array(ref, np.uint32))


@pytest.mark.parametrize("V,zero_frac,conc", [(7, 0.3, 1.0), (1000, 0.5, 0.3), (32000, 0.0, 0.05), (32000, 0.9, 1.0),
                                              (4097, 0.0, 1.0)])
def test_sample_bit_exact(V, zero_frac, conc):
    torch = torch_cuda()
    B = 24
    log(f"sample V={V} zero_frac={zero_frac}")
    probs = synth.make_prob_rows(B, V, seed=V + 11, concentration=conc, zero_frac=zero_frac)
    probs[3] = 0.0  # an all-zero row
    words = synth.make_rand_u32(B, seed=V)
    words[0], words[1] = 0, 0xFFFFFFFF
    out = torch.zeros(B, dtype=torch.int32, device="cuda")
    binding.specdec_sample(f32(probs), u32_tensor(words), 0, 0, 0, 0, out)
    got = out.cpu().numpy()
    for b in range(B):
        ref = sampling.sample_fixed_point(probs[b], int(words[b]))
        assert got[b] == (-1 if ref is None else ref), (b, got[b], ref)


def _accept_inputs(B, g, V, seed, agree=0.7):
    """p, q rows with partial agreement, drafts drawn from q by the oracle sampler, random words."""
    rng = np.random.default_rng(seed)
    p = synth.make_prob_rows(B * (g + 1), V, seed=seed, concentration=0.2).reshape(B, g + 1, V)
    noise = synth.make_prob_rows(B * g, V, seed=seed + 1, concentration=0.2).reshape(B, g, V)
    q = (agree * p[:, :g].astype(np.float64) + (1 - agree) * noise).astype(np.float32)
    words = synth.make_rand_u32((B, g + 1), seed=seed + 2)
    d = np.zeros((B, g), np.int32)
    for b in range(B):
        for i in range(g):
            d[b, i] = sampling.sample_fixed_point(q[b, i], int(rng.integers(0, 2 ** 32)))
    return p, q, d, words


@pytest.mark.parametrize("g,V", [(1, 512), (4, 32000), (8, 2048), (6, 32000), (4, 50000), (2, 128256), (3, 65)])
def test_accept_sampling_bit_exact(g, V):
    torch = torch_cuda()
    B = 16
    counts = np.zeros(g + 1, int)
    for seed in range(3):
        log(f"accept g={g} V={V} seed={seed}")
        p, q, d, words = _accept_inputs(B, g, V, seed=100 * g + seed)
        nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
        nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d), g, u32_tensor(words),
                               0, 0, nacc, nxt, status)
        A_gpu, n_gpu = nacc.cpu().numpy(), nxt.cpu().numpy()
        assert int(status.item()) == 0
        for b in range(B):
            A, n = sampling.accept_sampling(p[b], q[b], d[b], [int(w) for w in words[b, :g]], int(words[b, g]))
            assert (A_gpu[b], n_gpu[b]) == (A, n), (b, A_gpu[b], n_gpu[b], A, n)
            counts[A] += 1
    log(f"accept-length histogram {counts.tolist()}")
    assert counts[g] > 0 and counts[:g].sum() > 0  # both branches exercised


def test_accept_philox_mode_bit_exact():
    torch = torch_cuda()
    B, g, V = 16, 4, 3000
    p, q, d, _ = _accept_inputs(B, g, V, seed=7)
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    for step in (0, 5, 2 ** 35):
        binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d), g, None, 2, step, nacc, nxt)
        A_gpu, n_gpu = nacc.cpu().numpy(), nxt.cpu().numpy()
        for b in range(B):
            assert (A_gpu[b], n_gpu[b]) == sampling.accept_philox(p[b], q[b], d[b], 2, b, step)


def test_accept_greedy_and_special_cases():
    torch = torch_cuda()
    B, g, V = 8, 5, 777
    rng = np.random.default_rng(3)
    scores = rng.standard_normal((B, g + 1, V)).astype(np.float32)
    am = scores.argmax(axis=2)
    d = am[:, :g].astype(np.int32).copy()
    for b in range(B):
        if b < g:
            d[b, b] = (am[b, b] + 1) % V   # first mismatch at position b
    scores[B - 1, 2, [3, 9]] = scores[B - 1, 2].max() + 1.0  # tie: lowest index wins
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    for kind in (binding.INPUT_PROBS, binding.INPUT_LOGITS):
        binding.specdec_accept(B, g, V, kind, 0.0, f32(scores), None, i32(d), g, None, 0, 0, nacc, nxt)
        A_gpu, n_gpu = nacc.cpu().numpy(), nxt.cpu().numpy()
        for b in range(B):
            assert (A_gpu[b], n_gpu[b]) == sampling.accept_greedy(scores[b], d[b])
    # p == q: everything accepted, bonus drawn from p_{g+1}
    p, _, _, words = _accept_inputs(B, g, V, seed=9)
    q = p[:, :g].copy()
    d2 = p[:, :g].argmax(axis=2).astype(np.int32)  # p(d) = q(d) > 0
    words[:, :g] = 0xFFFFFFFF
    binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d2), g, u32_tensor(words), 0, 0,
                           nacc, nxt)
    assert (nacc.cpu().numpy() == g).all()
    for b in range(B):
        assert nxt[b].item() == sampling.sample_fixed_point(p[b, g], int(words[b, g]))


def test_accept_nonfinite_sets_status():
    torch = torch_cuda()
    B, g, V = 2, 3, 100
    p, q, d, words = _accept_inputs(B, g, V, seed=4)
    p[1, 0, 5] = np.nan
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d), g, u32_tensor(words), 0, 0,
                           nacc, nxt, status)
    assert status.item() == -4
    assert nacc[1].item() == -1 and nacc[0].item() >= 0
    with pytest.raises(sampling.NonFiniteError):
        sampling.accept_sampling(p[1], q[1], d[1], [int(w) for w in words[1, :g]], int(words[1, g]))
    # an Inf in a draft row the decision never reaches is still an error (every
    # input row is checked, as the oracle does)
    p, q, d, words = _accept_inputs(B, g, V, seed=4)
    q[0, g - 1, 7] = np.inf
    status.zero_()
    binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d), g, u32_tensor(words), 0, 0,
                           nacc, nxt, status)
    assert status.item() == -4 and nacc[0].item() == -1 and nxt[0].item() == -1 and nacc[1].item() >= 0
    with pytest.raises(sampling.NonFiniteError):
        sampling.accept_sampling(p[0], q[0], d[0], [int(w) for w in words[0, :g]], int(words[0, g]))
    # greedy: a NaN in the bonus row
    scores = np.random.default_rng(5).standard_normal((B, g + 1, V)).astype(np.float32)
    scores[1, g, 3] = np.nan
    status.zero_()
    binding.specdec_accept(B, g, V, binding.INPUT_LOGITS, 0.0, f32(scores), None, i32(d), g, None, 0, 0,
                           nacc, nxt, status)
    assert status.item() == -4 and nacc[1].item() == -1 and nacc[0].item() >= 0
    with pytest.raises(sampling.NonFiniteError):
        sampling.accept_greedy(scores[1], d[1])


def test_accept_logits_mode_matches_oracle():
    torch = torch_cuda()
    B, g, V, T = 16, 4, 32000, 0.8
    rng = np.random.default_rng(12)
    logits = (rng.standard_normal((B, g + 1, V)) * 1.3).astype(np.float32)
    q = sampling.softmax(rng.standard_normal((B, g, V)) * 1.3 + logits[:, :g] * 0.5, T).astype(np.float32)
    d = np.array([[sampling.sample_fixed_point(q[b, i], int(rng.integers(0, 2 ** 32))) for i in range(g)]
                  for b in range(B)], np.int32)
    words = synth.make_rand_u32((B, g + 1), seed=13)
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    binding.specdec_accept(B, g, V, binding.INPUT_LOGITS, T, f32(logits), f32(q), i32(d), g, u32_tensor(words), 0, 0,
                           nacc, nxt)
    A_gpu, n_gpu = nacc.cpu().numpy(), nxt.cpu().numpy()
    kinds = []
    for b in range(B):
        p = sampling.softmax(logits[b].astype(np.float64), T).astype(np.float32)
        kind, detail = accept_explained(p, q[b], d[b], words[b], A_gpu[b], n_gpu[b])
        if kind != "equal":
            log(f"row {b}: {kind}: {detail}")
        kinds.append(kind)
    # float32 softmax on the GPU vs float64 in the oracle: a decision may only
    # differ where the oracle's own decision is within the float32 error of flipping
    assert "mismatch" not in kinds
    assert kinds.count("boundary") <= 1


@pytest.mark.parametrize("role", [binding.ROLE_TARGET, binding.ROLE_DRAFT])
def test_kv_commit_all_accept_counts(role):
    torch = torch_cuda()
    shape = synth.TINY.with_layers(1)
    W = synth.make_weights(synth.TINY, n_layers=1)
    dw = binding.DeviceWeights(shape, W)
    model = binding.Model(dw, 1, max_rows=64, max_ctx=256)
    g = 6
    B = 2 * (g + 1)
    kv = binding.KVCache(model, B, 256)
    lens = np.arange(B, dtype=np.int32) * 3 + 10
    npend = np.array([1 + (b % 2) for b in range(B)], np.int32)
    pend = np.stack([np.full(B, 5), np.arange(B) + 100], axis=1).astype(np.int32)
    if role == binding.ROLE_TARGET:
        npend[:] = 1
    kv.set_state(lens, pend, npend)
    A = np.array([b % (g + 1) for b in range(B)], np.int32)
    nxt = np.arange(B, dtype=np.int32) + 400
    d = (np.arange(B * g, dtype=np.int32).reshape(B, g) + 1000)
    binding.specdec_kv_commit(kv, g, role, i32(A), i32(d), g, i32(nxt))
    st = kv.read_state()
    for b in range(B):
        s0 = kvstate.SeqState(int(lens[b]), [int(x) for x in pend[b, 2 - npend[b]:]])
        if role == binding.ROLE_TARGET:
            ref = kvstate.commit_target(s0, int(A[b]), g, int(nxt[b]))
        else:
            ref = kvstate.commit_draft(s0, int(A[b]), g, d[b], int(nxt[b]))
        assert st["len"][b] == ref.length
        n = st["n_pending"][b]
        assert list(st["pending"][b, 2 - n:]) == ref.pending
    # an accept error (A = -1) leaves the cache untouched
    kv.set_state(lens, pend, npend)
    binding.specdec_kv_commit(kv, g, role, i32(np.full(B, -1, np.int32)), i32(d), g, i32(nxt))
    np.testing.assert_array_equal(kv.read_state()["len"], lens)


def _chi2_pvalue(counts, expected):
    """Pearson chi-square p-value; bins with expected count below 5 are pooled."""
    from scipy import stats
    counts, expected = np.asarray(counts, float), np.asarray(expected, float)
    small = expected < 5
    if small.any():
        counts = np.append(counts[~small], counts[small].sum())
        expected = np.append(expected[~small], expected[small].sum())
    chi2 = ((counts - expected) ** 2 / expected).sum()
    return float(stats.chi2.sf(chi2, len(counts) - 1))


def test_accept_distribution_matches_the_closed_form():
    """Statistics of the device accept over many independent sequences (Philox
    draws): with d_i ~ q_i, position i is accepted with probability
    alpha_i = sum_x min(p_i(x), q_i(x)), so P(A = k) = alpha_1..alpha_k (1 - alpha_{k+1})
    and P(A = gamma) = prod alpha_i (Sec. 2, speculative sampling); and the first
    emitted token (d_1 when accepted, else the residual draw) is distributed
    as p_1 exactly."""
    torch = torch_cuda()
    B, g, V, steps = 8192, 3, 50, 3
    p1 = synth.make_prob_rows(g + 1, V, seed=41, concentration=0.8).astype(np.float64)
    noise = synth.make_prob_rows(g, V, seed=42, concentration=0.8).astype(np.float64)
    q1 = 0.6 * p1[:g] + 0.4 * noise
    p1 = (p1 / p1.sum(axis=1, keepdims=True)).astype(np.float32)
    q1 = (q1 / q1.sum(axis=1, keepdims=True)).astype(np.float32)
    p = np.broadcast_to(p1, (B, g + 1, V)).copy()
    q = np.broadcast_to(q1, (B, g, V)).copy()
    rng = np.random.default_rng(43)
    nacc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = binding.accept_workspace(B, g, V)
    A_all, first = [], []
    for step in range(steps):
        # drafts d_i ~ q_i (the draws of the draft model, here independent test inputs)
        cdf = np.cumsum(q1.astype(np.float64), axis=1)
        u = rng.random((B, g))
        d = np.stack([np.minimum(np.searchsorted(cdf[i], u[:, i] * cdf[i, -1], side="right"), V - 1)
                      for i in range(g)], axis=1).astype(np.int32)
        binding.specdec_accept(B, g, V, binding.INPUT_PROBS, 1.0, f32(p), f32(q), i32(d), g, None, 9, step, nacc, nxt,
                               status, ws)
        A, n = nacc.cpu().numpy(), nxt.cpu().numpy()
        assert int(status.item()) == 0
        A_all.append(A)
        first.append(np.where(A >= 1, d[:, 0], n))
    A_all, first = np.concatenate(A_all), np.concatenate(first)
    N = A_all.size
    alpha = np.minimum(p1[:g].astype(np.float64), q1.astype(np.float64)).sum(axis=1)
    pk = [np.prod(alpha[:k]) * (1 - alpha[k]) for k in range(g)] + [np.prod(alpha)]
    hist_a = np.bincount(A_all, minlength=g + 1)
    pa = _chi2_pvalue(hist_a, N * np.array(pk))
    hist_t = np.bincount(first, minlength=V)
    pt = _chi2_pvalue(hist_t, N * p1[0].astype(np.float64))
    log(f"accept lengths {hist_a.tolist()} vs expected {np.round(N * np.array(pk)).astype(int).tolist()} "
        f"(chi-square p = {pa:.3g}); first-token chi-square p = {pt:.3g} over {N} sequences")
    assert pa > 1e-3 and pt > 1e-3
