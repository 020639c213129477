"""One draft-and-verify iteration end to end (TEST INFRASTRUCTURE ONLY).

The inner loop of the paper's runtime (Sec. 3.4, Alg. 3: run the active
draft, then verify with the target) for a single sequence:
  1. draft: for slot s = 0..g-1 the draft processes its pending tokens
     (slot 0) or its previous token d_s (slot s > 0) and proposes
     d_{s+1} ~ q_{s+1} = softmax(draft logits / T) (argmax when T = 0);
  2. verify: one target pass over [x_last, d_1..d_g] gives p_1..p_{g+1};
  3. accept / resample (``sampling``);
  4. commit both caches (``kvstate``).
"""
from __future__ import annotations

import numpy as np

from .kvstate import SeqState, commit_draft, commit_target
from .model import KVCache, Model
from .philox import PURPOSE_ACCEPT, PURPOSE_RESAMPLE, draw_u32
from .sampling import (accept_greedy, accept_sampling, argmax_first, draft_sample_philox,
                       softmax)


class Sequence:
    """Target and draft caches plus bookkeeping for one sequence."""

    def __init__(self, target: Model, draft: Model, capacity: int):
        self.target, self.draft = target, draft
        self.kv_t = KVCache(target.shape, target.n_layers, capacity)
        self.kv_d = KVCache(draft.shape, draft.n_layers, capacity)
        self.st_t = SeqState(0, [])
        self.st_d = SeqState(0, [])
        self.emitted = []

    def prefill(self, prompt):
        """Commit prompt[:-1] to both caches; the last prompt token is pending."""
        prompt = [int(t) for t in np.asarray(prompt).reshape(-1)]
        self.target.prefill(prompt[:-1], self.kv_t)
        self.draft.prefill(prompt[:-1], self.kv_d)
        self.st_t = SeqState(self.kv_t.length, [prompt[-1]])
        self.st_d = SeqState(self.kv_d.length, [prompt[-1]])

    def draft_phase(self, g: int, temperature: float, seed: int, step: int, b: int = 0):
        """Run the draft for g slots: returns (d [g], q float32 [g, V] or None, draft logits [g, V])."""
        ds, qs, logit_rows = [], [], []
        n = len(self.st_d.pending)
        for s in range(g):
            if s == 0:
                logits = self.draft.forward_block(self.st_d.pending, self.st_d.length, self.kv_d)[-1]
            else:
                logits = self.draft.decode_step(ds[-1], self.st_d.length + n + s - 1, self.kv_d)
            logit_rows.append(logits)
            if temperature == 0:
                ds.append(argmax_first(logits))
            else:
                q = softmax(logits, temperature).astype(np.float32)
                qs.append(q)
                ds.append(draft_sample_philox(q, seed, b, step, s))
        q = np.stack(qs) if qs else None
        return ds, q, np.stack(logit_rows)

    def verify_phase(self, ds):
        """Target pass over [x_last, d_1..d_g]; returns float64 logits [g+1, V]."""
        tokens = [self.st_t.pending[-1]] + list(ds)
        return self.target.forward_block(tokens, self.st_t.length, self.kv_t)

    def iterate(self, g: int, temperature: float, seed: int, step: int, b: int = 0):
        """One full iteration; returns (A, next_token, drafted tokens)."""
        ds, q, _ = self.draft_phase(g, temperature, seed, step, b)
        logits = self.verify_phase(ds)
        if temperature == 0:
            A, nxt = accept_greedy(logits, ds)
        else:
            p = softmax(logits, temperature).astype(np.float32)
            u = [draw_u32(seed, b, step, PURPOSE_ACCEPT, i) for i in range(g)]
            x = draw_u32(seed, b, step, PURPOSE_RESAMPLE, 0)
            A, nxt = accept_sampling(p, q, ds, u, x)
        self.st_t = commit_target(self.st_t, A, g, nxt)
        self.st_d = commit_draft(self.st_d, A, g, ds, nxt)
        self.kv_t.length = self.st_t.length
        self.kv_d.length = self.st_d.length
        self.emitted.extend(list(ds[:A]) + [nxt])
        return A, nxt, ds


def greedy_decode(model: Model, prompt, n_new: int, capacity: int):
    """Plain autoregressive greedy decoding (no drafts): the tokens after the prompt."""
    kv = KVCache(model.shape, model.n_layers, capacity)
    prompt = [int(t) for t in np.asarray(prompt).reshape(-1)]
    model.prefill(prompt[:-1], kv)
    tok = prompt[-1]
    out = []
    for _ in range(n_new):
        logits = model.decode_step(tok, kv.length, kv)
        kv.length += 1
        tok = argmax_first(logits)
        out.append(tok)
    return out
