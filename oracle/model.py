"""Llama-style decoder forward in float64 (TEST INFRASTRUCTURE ONLY).

The paper evaluates LLaMA-2 7B (and Qwen2.5 7B) targets with small drafts
(Sec. 4.1, "Models"); its draft-and-verify iteration (Sec. 2.1, Eq. (1); Sec.
3.4, Alg. 3) runs the draft, then verifies the drafted tokens with one
target pass.  The paper states no model arithmetic, so this module writes
out the standard Llama decoder:

    h   = E[token]
    per layer l:
        x   = RMSNorm(h; g_attn)             x * g / sqrt(mean(x^2) + eps)
        q,k,v = x Wq^T, x Wk^T, x Wv^T
        q,k = RoPE(q, k, pos)                rotate-half pairs (j, j + hd/2),
                                             theta_j = base^(-2j/hd)
        K[pos], V[pos] = k, v                stored in the cache's storage type
        o   = softmax(q K^T / sqrt(hd)) V    causal, kv head = q_head // (h/h_kv)
        h  += o Wo^T
        x   = RMSNorm(h; g_ffn)
        h  += (silu(x Wg^T) * (x Wu^T)) Wd^T   silu(z) = z / (1 + exp(-z))
    logits = RMSNorm(h; g_final) H^T

Everything is float64 except one mirror point fixed by the storage format:
K and V are rounded to the cache's storage type (float32, or bfloat16 by
round-to-nearest-even) when written, and attention reads the stored values.
The verify pass over n tokens is computed as one block with a causal mask
(``forward_block``); tests pin it against n single-token steps.
"""
from __future__ import annotations

import numpy as np

LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


# ---------------------------------------------------------------- storage types
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64 (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), returned as float64.

    bfloat16 keeps 8 significant bits (exponent range of float32): with
    x = m * 2^e, 0.5 <= |m| < 1, the spacing of representable values near x
    is q = 2^(e-8) (clamped at the subnormal spacing 2^-133), and the stored
    value is q * rint(x / q), rint rounding halves to even.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    q = np.ldexp(1.0, e - 8)
    out = np.rint(x / q) * q
    return np.where(np.isfinite(x), out, x)


def weight_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """A stored weight tensor (float32 array or bf16 bits) as float64; float64
    arrays (effective weights of a quantized model, quant.py) are used as given."""
    if isinstance(arr, np.ndarray) and arr.dtype == np.float64:
        return arr
    if dtype == "bf16":
        return bf16_bits_to_f64(arr)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def store_kv(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a K/V value to the cache storage type (the one mirror point)."""
    if dtype == "bf16":
        return round_to_bf16(x)
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


# ---------------------------------------------------------------- layer pieces
def rmsnorm(h: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm: h / sqrt(mean(h^2) + eps) * g."""
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps) * g


def rope_angles(pos: np.ndarray, head_dim: int, base: float):
    """cos and sin of pos * base^(-2j/hd) for j < hd/2 (float64)."""
    half = head_dim // 2
    inv_freq = base ** (-2.0 * np.arange(half, dtype=np.float64) / head_dim)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half RoPE on x [n, heads, hd] at positions pos [n].

    Pair (j, j + hd/2) is rotated by the angle pos * theta_j:
        out_j        = x_j cos - x_{j+hd/2} sin
        out_{j+hd/2} = x_{j+hd/2} cos + x_j sin
    """
    n, nh, hd = x.shape
    half = hd // 2
    c, s = rope_angles(pos, hd, base)
    c = c[:, None, :]
    s = s[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def attention_block(q: np.ndarray, K: np.ndarray, V: np.ndarray, q_pos: np.ndarray,
                    n_kv_heads: int) -> np.ndarray:
    """Causal GQA attention of n queries against one sequence's cache.

    q [n, h, hd]; K, V [T, h_kv, hd] (stored values); query i may attend to
    keys 0..q_pos[i].  Scale 1/sqrt(hd); query head h uses kv head
    h // (h / h_kv).  Returns o [n, h, hd].
    """
    n, nh, hd = q.shape
    group = nh // n_kv_heads
    T = K.shape[0]
    out = np.empty_like(q)
    key_pos = np.arange(T)
    for head in range(nh):
        kvh = head // group
        s = q[:, head, :] @ K[:, kvh, :].T / np.sqrt(hd)          # [n, T]
        mask = key_pos[None, :] <= np.asarray(q_pos)[:, None]
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, head, :] = p @ V[:, kvh, :]
    return out


# ---------------------------------------------------------------- KV cache
class KVCache:
    """One sequence's cache: per layer K, V [capacity, h_kv, hd] of stored values.

    Values are kept as float32 arrays (every float32 or bf16 value is exact
    there) and widened to float64 for arithmetic.  ``length`` counts committed
    positions; entries at or beyond it are speculative.
    """

    def __init__(self, shape, n_layers: int, capacity: int):
        self.shape = shape
        self.n_layers = n_layers
        self.capacity = capacity
        self.k = [np.zeros((capacity, shape.n_kv_heads, shape.head_dim), np.float32) for _ in range(n_layers)]
        self.v = [np.zeros((capacity, shape.n_kv_heads, shape.head_dim), np.float32) for _ in range(n_layers)]
        self.length = 0

    def load(self, layer: int, k: np.ndarray, v: np.ndarray):
        """Install a resident context for ``layer`` at positions [0, len(k))."""
        n = k.shape[0]
        if n > self.capacity:
            raise ValueError("context longer than capacity")
        self.k[layer][:n] = weight_f64(k, self.shape.dtype)
        self.v[layer][:n] = weight_f64(v, self.shape.dtype)

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c.shape, c.n_layers, c.capacity, c.length = self.shape, self.n_layers, self.capacity, self.length
        c.k = [a.copy() for a in self.k]
        c.v = [a.copy() for a in self.v]
        return c


# ---------------------------------------------------------------- forward
class Model:
    """A decoder over stored weights (dict from the synthetic generator).

    ``n_layers`` selects the first layers (a draft is a prefix of the target
    sharing E, final norm and H).  Weights are widened to float64 layer by
    layer when used, so large models need only one layer in float64 at a time.
    """

    def __init__(self, shape, weights: dict, n_layers: int | None = None):
        self.shape = shape
        self.w = weights
        self.n_layers = len(weights["layers"]) if n_layers is None else n_layers
        if self.n_layers > len(weights["layers"]):
            raise ValueError("model has fewer layers than requested")
        self.dtype = shape.dtype

    def _wt(self, arr):
        return weight_f64(arr, self.dtype)

    def embed(self, tokens) -> np.ndarray:
        tokens = np.asarray(tokens, dtype=np.int64)
        if tokens.min() < 0 or tokens.max() >= self.shape.vocab:
            raise ValueError("token id out of range")
        return self._wt(self.w["embed"][tokens])

    def layer(self, l: int, h: np.ndarray, pos: np.ndarray, kv: KVCache) -> np.ndarray:
        """One decoder layer over rows h [n, d] at positions pos [n] (block-causal)."""
        s = self.shape
        W = self.w["layers"][l]
        n = h.shape[0]
        x = rmsnorm(h, self._wt(W["attn_norm"]), s.rms_eps)
        q = (x @ self._wt(W["wq"]).T).reshape(n, s.n_heads, s.head_dim)
        k = (x @ self._wt(W["wk"]).T).reshape(n, s.n_kv_heads, s.head_dim)
        v = (x @ self._wt(W["wv"]).T).reshape(n, s.n_kv_heads, s.head_dim)
        q = rope(q, pos, s.rope_base)
        k = rope(k, pos, s.rope_base)
        top = int(np.max(pos)) + 1
        if top > kv.capacity:
            raise ValueError("KV capacity exceeded")
        kv.k[l][pos] = store_kv(k, self.dtype)
        kv.v[l][pos] = store_kv(v, self.dtype)
        K = kv.k[l][:top].astype(np.float64)
        V = kv.v[l][:top].astype(np.float64)
        o = attention_block(q, K, V, pos, s.n_kv_heads).reshape(n, s.q_dim)
        h = h + o @ self._wt(W["wo"]).T
        x = rmsnorm(h, self._wt(W["ffn_norm"]), s.rms_eps)
        u = silu(x @ self._wt(W["w_gate"]).T) * (x @ self._wt(W["w_up"]).T)
        return h + u @ self._wt(W["w_down"]).T

    def head(self, h: np.ndarray) -> np.ndarray:
        x = rmsnorm(h, self._wt(self.w["final_norm"]), self.shape.rms_eps)
        return x @ self._wt(self.w["lm_head"]).T

    def forward_block(self, tokens, start_pos: int, kv: KVCache) -> np.ndarray:
        """Process tokens at positions start_pos.. as one causal block.

        Writes their K/V into ``kv`` (without changing ``kv.length``) and
        returns float64 logits [n, V], row i being the next-token scores after
        token i.  This is the verify pass when tokens = [last committed token,
        d_1..d_gamma] and start_pos = committed length.
        """
        tokens = np.asarray(tokens).reshape(-1)
        pos = start_pos + np.arange(tokens.size)
        h = self.embed(tokens)
        for l in range(self.n_layers):
            h = self.layer(l, h, pos, kv)
        return self.head(h)

    def decode_step(self, token: int, pos: int, kv: KVCache) -> np.ndarray:
        """Single-token step (the draft's step): logits [V] for the token at ``pos``."""
        return self.forward_block([token], pos, kv)[0]

    def prefill(self, tokens, kv: KVCache, chunk: int = 256):
        """Commit tokens into the cache from position kv.length (logits discarded)."""
        tokens = np.asarray(tokens).reshape(-1)
        for i in range(0, tokens.size, chunk):
            part = tokens[i:i + chunk]
            self.forward_block(part, kv.length, kv)
            kv.length += part.size
