"""Pins for the speculative-sampling accept/resample rule in the oracle (CPU only).

The central property (Leviathan et al. ICML'23, the rule the paper's draft-
and-verify iteration relies on to preserve output quality): the tokens
emitted by draft-and-verify are distributed exactly as the target's own
autoregressive samples.  We compute the exact output distribution of the
oracle's discrete implementation (by counting, over the 32-bit words, which
ones lead to each branch -- every call goes through ``accept_sampling`` and
``sample_fixed_point``) and compare it with the target distribution.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from oracle.sampling import accept_greedy, accept_sampling, sample_fixed_point

TOP = 2 ** 32


def _first_true(pred, lo, hi):
    """Smallest x in [lo, hi] with pred(x) true for a monotone predicate (hi if none)."""
    while lo < hi:
        mid = (lo + hi) // 2
        if pred(mid):
            hi = mid
        else:
            lo = mid + 1
    return lo


def sampler_dist(r):
    """Exact distribution of sample_fixed_point(r, x) over x uniform in [0, 2^32) (Fractions)."""
    V = len(r)
    out = {}
    start = 0
    for j in range(V):
        end = _first_true(lambda x: sample_fixed_point(r, x) > j, start, TOP)
        if end > start:
            out[j] = Fraction(end - start, TOP)
        start = end
    return out


def accept_prob(p_row, q_row, tok):
    """P(accept) of the oracle's test over the 2^24-point uniform grid, via accept_sampling with g=1."""
    p1 = np.stack([p_row, p_row])  # p_1 and (unused) p_2
    q1 = q_row[None, :]

    def rejects(x):
        A, _ = accept_sampling(p1, q1, [tok], [x], 0)
        return A == 0
    # acceptance is monotone: small u accept.  Count accepted 24-bit grid points.
    first_reject = _first_true(lambda k: rejects(k << 8), 0, 2 ** 24)
    return Fraction(first_reject, 2 ** 24)


def resample_dist(p_row, q_row, tok):
    """Distribution of the emitted token given rejection at this position (via accept_sampling)."""
    p1 = np.stack([p_row, p_row])
    q1 = q_row[None, :]
    u_rej = 0xFFFFFFFF
    A, _ = accept_sampling(p1, q1, [tok], [u_rej], 0)
    if A != 0:
        return None  # rejection impossible at this position
    V = len(p_row)
    out = {}
    start = 0
    for j in range(V):
        end = _first_true(lambda x: accept_sampling(p1, q1, [tok], [u_rej], x)[1] > j, start, TOP)
        if end > start:
            out[j] = Fraction(end - start, TOP)
        start = end
    return out


def _dist_rows(V, seed, ctx_tokens, spiky=False):
    """A deterministic context-dependent distribution (float32), seeded by the prefix."""
    rng = np.random.default_rng([seed] + list(ctx_tokens))
    g = rng.gamma(0.7 if spiky else 1.5, size=V)
    g[rng.random(V) < 0.2] = 0
    if g.sum() == 0:
        g[0] = 1
    return (g / g.sum()).astype(np.float32)


def emitted_first_two(V, gamma, seed_p, seed_q):
    """Exact P(first two emitted tokens) for draft-and-verify starting from an empty context.

    One iteration emits A+1 tokens; if it emits only one, the second comes
    from the next iteration started at the new context.
    """
    P = lambda ctx: _dist_rows(V, seed_p, ctx)
    Q = lambda ctx: _dist_rows(V, seed_q, ctx, spiky=True)
    cache = {}

    def sdist(r):
        key = r.tobytes()
        if key not in cache:
            cache[key] = sampler_dist(r)
        return cache[key]

    def one_iteration(ctx):
        """Distribution over emitted tuples of one iteration from context ctx."""
        res = {}

        def rec(drafts, prob):
            if len(drafts) < gamma:
                qd = sdist(Q(ctx + drafts))
                for t, pr in qd.items():
                    rec(drafts + (t,), prob * pr)
                return
            # verification of the full draft tuple
            acc_prob = prob
            for i in range(gamma):
                pre = ctx + drafts[:i]
                p_row, q_row = P(pre), Q(pre)
                a = accept_prob(p_row, q_row, drafts[i])
                rej = 1 - a
                if rej > 0:
                    rd = resample_dist(p_row, q_row, drafts[i])
                    for t, pr in rd.items():
                        key = drafts[:i] + (t,)
                        res[key] = res.get(key, 0) + acc_prob * rej * pr
                acc_prob = acc_prob * a
                if acc_prob == 0:
                    return
            for t, pr in sdist(P(ctx + drafts)).items():
                key = drafts + (t,)
                res[key] = res.get(key, 0) + acc_prob * pr

        rec((), Fraction(1))
        return res

    first = one_iteration(())
    two = {}
    for emitted, pr in first.items():
        if len(emitted) >= 2:
            k = emitted[:2]
            two[k] = two.get(k, 0) + pr
        else:
            for emitted2, pr2 in one_iteration(emitted).items():
                k = emitted + emitted2[:1]
                two[k] = two.get(k, 0) + pr * pr2
    return two, P


@pytest.mark.parametrize("V,gamma", [(3, 1), (3, 2), (4, 2)])
def test_output_distribution_equals_target(V, gamma):
    two, P = emitted_first_two(V, gamma, seed_p=101, seed_q=202)
    assert abs(float(sum(two.values())) - 1.0) < 1e-12
    worst = 0.0
    for t1, t2 in itertools.product(range(V), range(V)):
        target = float(Fraction(float(P(())[t1]))) * float(P((t1,))[t2])
        got = float(two.get((t1, t2), 0))
        worst = max(worst, abs(got - target))
    # discretisation: 2^-24 per accept decision, V*2^-40 + 2^-32 per draw, float32 p
    assert worst < 2e-6


def test_p_equals_q_accepts_everything():
    rng = np.random.default_rng(5)
    g, V = 4, 50
    p = rng.random((g + 1, V)).astype(np.float32)
    p /= p.sum(axis=1, keepdims=True)
    q = p[:g].copy()
    d = [int(np.argmax(p[i])) for i in range(g)]
    for x in [0, 0xFFFFFFFF, 12345]:
        A, _ = accept_sampling(p, q, d, [0xFFFFFFFF] * g, x)
        assert A == g


def test_onehot_q_with_zero_p_rejects_and_resamples_from_p():
    V = 6
    p = np.array([[0.0, 0.5, 0.25, 0.25, 0.0, 0.0]] * 2, np.float32)
    q = np.zeros((1, V), np.float32)
    q[0, 0] = 1.0
    A, _ = accept_sampling(p, q, [0], [0], 0)
    assert A == 0
    dist = resample_dist(p[0], q[0], 0)
    assert dist == {1: Fraction(1, 2), 2: Fraction(1, 4), 3: Fraction(1, 4)}


def test_greedy_is_argmax_match_prefix():
    rng = np.random.default_rng(9)
    g, V = 5, 40
    for A_true in range(g + 1):
        scores = rng.standard_normal((g + 1, V))
        am = scores.argmax(axis=1)
        d = list(am[:g])
        if A_true < g:
            d[A_true] = (am[A_true] + 1) % V
        A, nxt = accept_greedy(scores, d)
        assert A == A_true
        assert nxt == am[A_true]
    # ties: lowest index wins
    s = np.zeros((2, 5))
    s[0, [1, 3]] = 2.0
    assert accept_greedy(s, [3]) == (0, 1)


def test_greedy_is_sampling_with_onehot_distributions():
    rng = np.random.default_rng(4)
    g, V = 4, 12
    for trial in range(20):
        am = rng.integers(0, V, g + 1)
        d = [int(am[i]) if rng.random() < 0.7 else int((am[i] + 1) % V) for i in range(g)]
        p = np.zeros((g + 1, V), np.float32)
        p[np.arange(g + 1), am] = 1
        q = np.zeros((g, V), np.float32)
        q[np.arange(g), d] = 1
        words = rng.integers(0, 2 ** 32, g + 1, dtype=np.uint64)
        assert accept_sampling(p, q, d, [int(w) for w in words[:g]], int(words[g])) == accept_greedy(p, d)


def test_expected_accept_length_closed_form():
    # i.i.d. positions with acceptance alpha = sum min(p, q): E[A+1] = (1 - alpha^(g+1)) / (1 - alpha).
    V, g = 5, 3
    p_row = np.array([0.1, 0.2, 0.3, 0.25, 0.15], np.float32)
    q_row = np.array([0.3, 0.3, 0.1, 0.2, 0.1], np.float32)
    qd = sampler_dist(q_row)
    # P(accept one position) = sum_d q(d) * P(accept | d)
    a = sum(pr * accept_prob(p_row, q_row, t) for t, pr in qd.items())
    alpha = float(np.minimum(p_row.astype(np.float64), q_row.astype(np.float64)).sum())
    assert abs(float(a) - alpha) < 1e-6
    EA1 = sum(float(a) ** k for k in range(g + 1))
    assert abs(EA1 - (1 - alpha ** (g + 1)) / (1 - alpha)) < 1e-5


def test_nonfinite_is_an_error():
    from oracle.sampling import NonFiniteError
    p = np.full((2, 4), 0.25, np.float32)
    q = np.full((1, 4), 0.25, np.float32)
    p[1, 2] = np.nan
    with pytest.raises(NonFiniteError):
        accept_sampling(p, q, [0], [0], 0)


# ---------------------------------------------------------------- temperature (closed forms)
def _temperature_pin_holds(softmax_fn) -> bool:
    """softmax(l / T) against closed forms: logits (0, T ln 2) give (1/3, 2/3);
    logits T ln w give w / sum(w); a constant shift changes nothing."""
    ok = True
    for T in (0.8, 1.0, 2.0, 0.25):
        got = softmax_fn(np.array([0.0, T * np.log(2.0)]), T)
        ok &= np.allclose(got, [1 / 3, 2 / 3], rtol=0, atol=1e-14)
        w = np.array([1.0, 2.0, 3.0, 4.0, 10.0])
        got = softmax_fn(T * np.log(w), T)
        ok &= np.allclose(got, w / w.sum(), rtol=0, atol=1e-14)
        got2 = softmax_fn(T * np.log(w) + 37.5, T)
        ok &= np.allclose(got2, w / w.sum(), rtol=0, atol=1e-14)
    return bool(ok)


def test_softmax_temperature_closed_form():
    from oracle.sampling import softmax
    assert _temperature_pin_holds(softmax)
    # T = 0 is the greedy mode, never a softmax
    with pytest.raises(ValueError):
        softmax(np.zeros(3), 0.0)


def test_planted_temperature_mistake_fails_the_pin():
    def times_t(logits, T):  # multiplies by T instead of dividing
        z = np.asarray(logits, dtype=np.float64) * T
        e = np.exp(z - z.max())
        return e / e.sum()
    assert not _temperature_pin_holds(times_t)


# ---------------------------------------------------------------- degenerate residual (reading S4)
# q dominates p everywhere, so the residual max(0, p - q) is all zero and a
# rejection has nothing to draw from; the reading falls back to p itself with
# the same word.  p is not proportional to q, so a fallback to q is told apart.
_P_DOM = np.array([0.1, 0.3, 0.2], np.float32)
_Q_DOM = np.array([0.5, 0.3, 0.2], np.float32)


def _fallback_pin_holds(accept_fn) -> bool:
    p1 = np.stack([_P_DOM, _P_DOM])
    q1 = _Q_DOM[None, :]
    # accept iff u * 0.5 < 0.1, i.e. u < 0.2: word 0 accepts, the top word rejects
    if accept_fn(p1, q1, [0], [0], 0)[0] != 1 or accept_fn(p1, q1, [0], [0xFFFFFFFF], 0)[0] != 0:
        return False
    # emitted-token distribution given rejection, counted exactly over the resample word
    out, start = {}, 0
    for j in range(3):
        end = _first_true(lambda x: accept_fn(p1, q1, [0], [0xFFFFFFFF], x)[1] > j, start, TOP)
        out[j] = Fraction(end - start, TOP)
        start = end
    target = _P_DOM.astype(np.float64) / _P_DOM.astype(np.float64).sum()
    # fixed-point weights of float32 p: within 2^-32 + 3 * 2^-40 of p / sum(p)
    return all(abs(float(out[j]) - target[j]) < 1e-9 for j in range(3))


def test_degenerate_residual_falls_back_to_p():
    assert _fallback_pin_holds(accept_sampling)


def test_planted_fallback_to_q_fails_the_pin():
    def to_q(p, q, d, u, x):
        A, nxt = accept_sampling(p, q, d, u, x)
        if A < len(d) and not np.any(np.maximum(0, p[A] - q[A]) > 0):
            nxt = sample_fixed_point(q[A], x)
        return A, nxt
    assert not _fallback_pin_holds(to_q)
