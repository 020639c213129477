"""Helpers shared by the GPU parity tests (imported by tests only)."""
from __future__ import annotations

import sys

import numpy as np

from paper_2608_10362_amd import binding, synth


def log(msg: str):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    return torch


def u32_tensor(words: np.ndarray):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(words, dtype=np.uint32).view(np.int32)).cuda()


def f32(x):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def i32(x):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def kv_to_device(arr, dtype: str):
    """A synth K/V block (float32 or bf16 bits) as a device tensor of the storage type."""
    torch = torch_cuda()
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def install_context(kv: binding.KVCache, ctx, lengths, n_layers: int, dtype: str):
    """Write a synthetic resident context (synth.make_kv_context) into a device cache."""
    for l in range(n_layers):
        for b, L in enumerate(lengths):
            if L == 0:
                continue
            kv.write_context(l, b, 0, kv_to_device(ctx[l][b]["k"], dtype), kv_to_device(ctx[l][b]["v"], dtype))


def oracle_caches(shape, n_layers: int, ctx, lengths, capacity: int):
    from oracle.model import KVCache
    caches = []
    for b, L in enumerate(lengths):
        c = KVCache(shape, n_layers, capacity)
        for l in range(n_layers):
            if L:
                c.load(l, ctx[l][b]["k"], ctx[l][b]["v"])
        c.length = int(L)
        caches.append(c)
    return caches


# Relative error allowed on a float32 softmax probability computed on the device
# against the oracle's float64 one, rounded to float32: the exponentials round
# to within a few ulps and the row sum is a fixed-order float32 sum over the
# vocabulary; 1e-5 is about 170 ulps.
SOFTMAX_REL_ERR = 1e-5


def accept_explained(p, q, d, words, A_dev, n_dev, rel=SOFTMAX_REL_ERR):
    """Compare a device accept result with the oracle's on float32 p rows
    (the oracle's softmax rounded to float32).

    Returns (kind, detail): kind "equal" when (A, next) agree; "boundary"
    when they differ and the first diverging decision of the oracle sits
    within the probability error ``rel`` of flipping: an accept test with
    |fl(u q(d)) - p(d)| <= rel p(d), or a draw whose scaled word t lies within
    the shift that relative errors of ``rel`` on p can cause of the edge of the
    oracle's token interval; "mismatch" otherwise (a real disagreement).
    """
    from oracle import sampling
    g = len(d)
    A, n = sampling.accept_sampling(p, q, d, [int(w) for w in words[:g]], int(words[g]))
    if (A, n) == (int(A_dev), int(n_dev)):
        return "equal", ""
    for i in range(min(A, g) + (1 if A < g else 0)):
        u = sampling.uniform_from_u32(int(words[i]))
        lhs = float(np.float32(u * q[i, int(d[i])]))
        rhs = float(p[i, int(d[i])])
        if abs(lhs - rhs) <= rel * max(abs(rhs), 1e-30):
            return "boundary", f"accept test {i}: u*q = {lhs:.9g}, p = {rhs:.9g}"
    if A != int(A_dev):
        return "mismatch", f"A oracle {A} device {A_dev}, no accept test near its boundary"
    # the same A: the draw differs; distance of t to the edges of the oracle's interval
    if A < g:
        r = np.maximum(np.float32(0), (p[A] - q[A]).astype(np.float32))
        if not np.any(sampling.fixed_point_weights(r) > 0):
            r = p[A]
    else:
        r = p[g]
    R = sampling.fixed_point_weights(r)
    S = int(R.sum(dtype=np.uint64))
    t = (int(words[g]) * S) >> 32
    cum = np.cumsum(R, dtype=np.uint64)
    lo = int(cum[n - 1]) if n > 0 else 0
    hi = int(cum[n])
    # relative errors of `rel` on p move every cumulative weight, and S, by at
    # most rel * 2^40 * sum(p) (the residual's entries by at most rel * p_j)
    shift = 2 * rel * sampling.TWO40 * float(np.asarray(p[A if A < g else g], np.float64).sum()) + 2
    dist = min(t - lo, hi - 1 - t)
    if dist <= shift:
        return "boundary", f"draw: t = {t} within {dist} of [{lo}, {hi}) (allowed {shift:.3g})"
    return "mismatch", f"draw: next oracle {n} device {n_dev}, t = {t} is {dist} from the edges of [{lo}, {hi})"


def draw_near_boundary(r, x, n_oracle, rel=SOFTMAX_REL_ERR):
    """Whether the oracle's fixed-point draw from weights r with word x lies
    within the shift that relative errors of ``rel`` on r can cause of the edge
    of its token's interval (then a device draw on its own float32 weights may
    pick the neighbouring token)."""
    from oracle import sampling
    R = sampling.fixed_point_weights(np.asarray(r, np.float32))
    S = int(R.sum(dtype=np.uint64))
    t = (int(x) * S) >> 32
    cum = np.cumsum(R, dtype=np.uint64)
    lo = int(cum[n_oracle - 1]) if n_oracle > 0 else 0
    hi = int(cum[n_oracle])
    shift = 2 * rel * sampling.TWO40 * float(np.asarray(r, np.float64).sum()) + 2
    return min(t - lo, hi - 1 - t) <= shift
