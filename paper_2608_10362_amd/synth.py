"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle.

This module only *draws* inputs: model weights, prompt token ids, resident KV
contexts, ragged lengths, 32-bit random words and the draft-switch schedule.
It contains none of the method's arithmetic (no normalisation, attention,
softmax, sampling or acceptance), so that the oracle and the GPU path share
data, never code.

The paper (Sec. 4.1, "Models" and "Workloads") evaluates trained LLaMA-2 7B /
Qwen2.5 7B targets on five public datasets; neither the weights nor the
datasets are used here.  Llama-shaped decoders with N(0, 0.02^2) weights and
uniform-random prompt ids stand in for them.

Generator definition (one reading, since the paper gives none):
  * tensor order: embedding E, then for every layer
    [attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down],
    then final_norm, lm_head; each tensor has an index in that order;
  * every matrix is ``default_rng([seed, idx]).standard_normal(shape, float32) * 0.02``,
    stored [out, in] row-major, rounded to bf16 (round-to-nearest-even) for
    bf16 models;
  * RMSNorm gains are the constant 1.0 (they take an index, draw nothing);
  * a draft model is the first k layers of the target plus the shared
    embedding, final norm and LM head (untied E and H).
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional

import numpy as np

SEED_WEIGHTS = 0
SEED_PROMPT = 1
SEED_SAMPLING = 2
SEED_SCHEDULE = 3
SEED_LENGTHS = 4
SEED_KV = 5
SEED_RAND = 6


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Shape of a Llama-style decoder (names follow the usual notation)."""

    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    dtype: str = "bf16"  # "f32" or "bf16": storage type of weights and KV

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n)


# The five workloads: shapes of the target (drafts are layer prefixes).
TINY = ModelShape(2, 128, 4, 4, 32, 512, 512, dtype="f32")
LLAMA_1B = ModelShape(22, 2048, 32, 4, 64, 5632, 32000)
LLAMA_7B = ModelShape(32, 4096, 32, 32, 128, 11008, 32000)

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _tensor_shape(shape: ModelShape, name: str):
    d, f = shape.d_model, shape.ffn_dim
    return {
        "attn_norm": (d,),
        "ffn_norm": (d,),
        "wq": (shape.q_dim, d),
        "wk": (shape.kv_dim, d),
        "wv": (shape.kv_dim, d),
        "wo": (d, shape.q_dim),
        "w_gate": (f, d),
        "w_up": (f, d),
        "w_down": (d, f),
    }[name]


def _draw(seed: int, idx: int, shp, dtype: str, literal_gain: bool, is_gain: bool):
    if is_gain and not literal_gain:
        a = np.ones(shp, dtype=np.float32)
    else:
        a = np.random.default_rng([seed, idx]).standard_normal(shp, dtype=np.float32)
        a *= np.float32(0.02)
    if dtype == "bf16":
        return f32_to_bf16_bits(a)
    return a


def make_weights(shape: ModelShape, seed: int = SEED_WEIGHTS, n_layers: Optional[int] = None,
                 literal_gain: bool = False, threads: int = 8) -> Dict:
    """Draw the weights of ``shape`` (or of its first ``n_layers`` layers).

    Returns a dict with numpy arrays: float32 for f32 models, uint16 bf16 bit
    patterns for bf16 models.  Layout: 'embed' [V,d], 'lm_head' [V,d],
    'final_norm' [d], 'layers': list of dicts keyed by LAYER_TENSORS.
    Tensor indices do not depend on ``n_layers``, so a prefix drawn alone is
    identical to the same layers drawn as part of the full model.
    """
    L = shape.n_layers if n_layers is None else n_layers
    jobs = [("embed", None, 0, (shape.vocab, shape.d_model), False)]
    for l in range(L):
        for t, name in enumerate(LAYER_TENSORS):
            idx = 1 + l * len(LAYER_TENSORS) + t
            jobs.append((name, l, idx, _tensor_shape(shape, name), name.endswith("norm")))
    base = 1 + shape.n_layers * len(LAYER_TENSORS)
    jobs.append(("final_norm", None, base, (shape.d_model,), True))
    jobs.append(("lm_head", None, base + 1, (shape.vocab, shape.d_model), False))

    def run(job):
        name, l, idx, shp, is_gain = job
        return job, _draw(seed, idx, shp, shape.dtype, literal_gain, is_gain)

    out: Dict = {"layers": [dict() for _ in range(L)], "dtype": shape.dtype}
    with ThreadPoolExecutor(max(1, threads)) as ex:
        for (name, l, _, _, _), arr in ex.map(run, jobs):
            if l is None:
                out[name] = arr
            else:
                out["layers"][l][name] = arr
    return out


def draft_view(weights: Dict, k: int) -> Dict:
    """The draft: first k layers of the target with the shared E, final norm and H."""
    d = dict(weights)
    d["layers"] = weights["layers"][:k]
    return d


def make_prompt(n_tokens: int, vocab: int, batch: int = 1, seed: int = SEED_PROMPT) -> np.ndarray:
    """Uniform-random prompt ids in [0, vocab), int32 [batch, n_tokens]."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab, size=(batch, n_tokens), dtype=np.int64).astype(np.int32)


def make_ragged_lengths(batch: int, lo: int, hi: int, seed: int = SEED_LENGTHS) -> np.ndarray:
    """Context lengths drawn uniformly from [lo, hi] inclusive, int32 [batch]."""
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=batch, dtype=np.int64).astype(np.int32)


def make_kv_context(shape: ModelShape, n_layers: int, lengths, seed: int = SEED_KV,
                    sigma: Optional[float] = None, threads: int = 8) -> List[List[Dict]]:
    """A resident KV context drawn directly (instead of by prefill).

    For every layer and sequence b: K and V of shape [lengths[b], n_kv_heads, head_dim],
    N(0, sigma^2) with sigma = 0.02*sqrt(d_model) by default (the spread a
    projection of a unit-RMS row by N(0, 0.02^2) weights has), in the model's
    storage type (float32 or bf16 bits).  Returns kv[layer][b] = {'k':..., 'v':...}.
    """
    if sigma is None:
        sigma = 0.02 * float(np.sqrt(shape.d_model))
    lengths = [int(x) for x in np.asarray(lengths).reshape(-1)]

    def run(job):
        l, b = job
        rng = np.random.default_rng([seed, l, b])
        shp = (lengths[b], shape.n_kv_heads, shape.head_dim)
        out = {}
        for name in ("k", "v"):
            a = rng.standard_normal(shp, dtype=np.float32) * np.float32(sigma)
            out[name] = f32_to_bf16_bits(a) if shape.dtype == "bf16" else a
        return job, out

    kv = [[None] * len(lengths) for _ in range(n_layers)]
    jobs = [(l, b) for l in range(n_layers) for b in range(len(lengths))]
    with ThreadPoolExecutor(max(1, threads)) as ex:
        for (l, b), out in ex.map(run, jobs):
            kv[l][b] = out
    return kv


def make_rand_u32(shape, seed: int = SEED_RAND) -> np.ndarray:
    """Explicit 32-bit random words (used in place of the counter-based generator)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2**32, size=shape, dtype=np.uint64).astype(np.uint32)


def make_markov_schedule(n_steps: int, n_states: int = 3, start: int = 1, stay: float = 0.8,
                         seed: int = SEED_SCHEDULE) -> np.ndarray:
    """Per-iteration active-draft index: stay with prob ``stay``, else move to another state uniformly."""
    rng = np.random.default_rng(seed)
    s = np.empty(n_steps, dtype=np.int32)
    cur = start
    for i in range(n_steps):
        s[i] = cur
        if rng.random() >= stay:
            others = [j for j in range(n_states) if j != cur]
            cur = others[int(rng.integers(0, len(others)))]
    return s


def make_prob_rows(n_rows: int, vocab: int, seed: int, concentration: float = 1.0,
                   zero_frac: float = 0.0) -> np.ndarray:
    """Random probability rows (float32 [n_rows, vocab]) for sampler/accept tests.

    Drawn as Dirichlet-like rows: gamma(concentration) draws normalised in
    float64 then stored as float32; ``zero_frac`` of the entries are set to 0
    before normalising.  These are test inputs, not part of the method.
    """
    rng = np.random.default_rng(seed)
    g = rng.gamma(concentration, size=(n_rows, vocab))
    if zero_frac > 0:
        g[rng.random((n_rows, vocab)) < zero_frac] = 0.0
        empty = g.sum(axis=1) == 0
        g[empty, 0] = 1.0
    return (g / g.sum(axis=1, keepdims=True)).astype(np.float32)
