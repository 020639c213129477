"""Temperature softmax, fixed-point sampler and the speculative accept rule
(TEST INFRASTRUCTURE ONLY).

The paper runs greedy decoding at batch 1 (Sec. 4.1, "Runtime configuration")
and defers the verification rule to the speculative-decoding works it cites
(Leviathan et al. ICML'23; Chen et al. 2023).  That rule, per sequence, with
target distributions p_1..p_{g+1}, draft distributions q_1..q_g and drafted
tokens d_1..d_g:
  * for i = 1..g: accept d_i with probability min(1, p_i(d_i) / q_i(d_i));
  * at the first rejection i: emit a token drawn from norm(max(0, p_i - q_i));
  * if all g are accepted: emit a bonus token drawn from p_{g+1}.
A = number of accepted drafts; A + 1 tokens are emitted per iteration
(Sec. 2.1, Eq. (1) uses E[A] as the throughput lever).

Readings where the sources are silent (one choice each, shared with the GPU
path through this documentation, not through code):
  * the test "with probability min(1, p/q)" is carried out as
    fl32(u * q_i(d_i)) < p_i(d_i) with a uniform u in [0, 1) taken from a
    32-bit word as (x >> 8) * 2^-24, one rounded float32 multiply, strict <;
  * a draw from weights r (probabilities or the residual) uses a fixed-point
    inverse CDF: R_j = floor(r_j * 2^40), S = sum R_j,
    t = floor(x * S / 2^32) for the 32-bit word x, token = the smallest j
    with R_0 + ... + R_j > t.  Integer sums make the draw independent of
    summation order;
  * the residual is r_j = max(0, fl32(p_j - q_j)); if all R_j are 0 the draw
    falls back to p_i with the same word;
  * greedy (temperature 0): argmax with the lowest index on ties; A is the
    length of the prefix where the drafted token equals the target argmax,
    the emitted token is the target argmax at position A+1;
  * NaN or Inf in p or q is an error.
"""
from __future__ import annotations

import numpy as np

from .philox import PURPOSE_ACCEPT, PURPOSE_DRAFT, PURPOSE_RESAMPLE, draw_u32, uniform_from_u32

TWO40 = float(2 ** 40)


class NonFiniteError(ValueError):
    pass


def softmax(logits: np.ndarray, temperature: float) -> np.ndarray:
    """softmax(logits / T) along the last axis, float64."""
    if temperature <= 0:
        raise ValueError("temperature must be > 0 for a softmax")
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def fixed_point_weights(r: np.ndarray) -> np.ndarray:
    """R_j = floor(r_j * 2^40) as uint64 (r_j >= 0, at most 1)."""
    r = np.asarray(r, dtype=np.float64)
    return np.floor(r * TWO40).astype(np.uint64)


def sample_fixed_point(r: np.ndarray, x: int):
    """Inverse-CDF draw from weights r with the 32-bit word x; None if all weights are 0."""
    R = fixed_point_weights(r)
    S = int(R.sum(dtype=np.uint64))
    if S == 0:
        return None
    t = (int(x) * S) >> 32
    cum = np.cumsum(R, dtype=np.uint64)
    return int(np.searchsorted(cum, np.uint64(t), side="right"))


def argmax_first(scores: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties."""
    return int(np.argmax(np.asarray(scores)))


def _check_finite(*arrays):
    for a in arrays:
        if a is not None and not np.all(np.isfinite(a)):
            raise NonFiniteError("non-finite probability")


def accept_sampling(p: np.ndarray, q: np.ndarray, d, u_accept, x_resample: int):
    """Speculative-sampling verification for one sequence.

    p: float32 [g+1, V], q: float32 [g, V], d: [g] drafted tokens,
    u_accept: [g] 32-bit words for the accept tests, x_resample: the 32-bit
    word for the resample / bonus draw.  Returns (A, next_token).
    """
    p = np.asarray(p, dtype=np.float32)
    q = np.asarray(q, dtype=np.float32)
    _check_finite(p, q)
    g = q.shape[0]
    for i in range(g):
        tok = int(d[i])
        u = uniform_from_u32(u_accept[i])
        if not (np.float32(u * q[i, tok]) < p[i, tok]):
            resid = np.maximum(np.float32(0), (p[i] - q[i]).astype(np.float32))
            nxt = sample_fixed_point(resid, x_resample)
            if nxt is None:
                nxt = sample_fixed_point(p[i], x_resample)
            return i, nxt
    return g, sample_fixed_point(p[g], x_resample)


def accept_greedy(scores_p: np.ndarray, d):
    """Greedy verification: argmax-match prefix and the target argmax after it."""
    scores_p = np.asarray(scores_p)
    _check_finite(scores_p)
    g = len(d)
    for i in range(g):
        a = argmax_first(scores_p[i])
        if a != int(d[i]):
            return i, a
    return g, argmax_first(scores_p[g])


def accept_philox(p, q, d, seed: int, b: int, step: int):
    """accept_sampling with the words drawn from Philox4x32-10 (see ``philox``)."""
    g = len(d)
    u = [draw_u32(seed, b, step, PURPOSE_ACCEPT, i) for i in range(g)]
    x = draw_u32(seed, b, step, PURPOSE_RESAMPLE, 0)
    return accept_sampling(p, q, d, u, x)


def draft_sample_philox(q_row: np.ndarray, seed: int, b: int, step: int, slot: int) -> int:
    """Draft token at ``slot`` drawn from q with the Philox word for that slot."""
    tok = sample_fixed_point(q_row, draw_u32(seed, b, step, PURPOSE_DRAFT, slot))
    if tok is None:
        raise NonFiniteError("all-zero draft distribution")
    return tok
