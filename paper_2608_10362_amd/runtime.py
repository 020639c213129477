"""Host-side draft scheduling over the C ABI.

The paper's contribution around the draft-and-verify engine is host policy:

- a resident draft cache of capacity K, refreshed at every scheduling point
  (Sec. 3.3, Alg. 2): the top-K drafts of the predicted ranking form the
  target set; a missing one is prefetched asynchronously into a free slot,
  evicting, when space is needed, the lowest-scored resident draft outside
  the target set and never the active draft;
- a runtime loop that never waits for a draft still loading (Sec. 3.4,
  Alg. 3): every N iterations it re-ranks the drafts and runs the best
  *resident* one for the next interval.

Here the ranking comes from a seeded synthetic score stream (the paper's
BERT predictor and its training data are not available), the backing storage
is pinned host memory holding the packed image, and a prefetch is an H2D copy
on a side stream (specdec_load_async) whose completion an event reports.

A draft that becomes active after an absence first runs a catch-up forward
over the committed tokens it missed (its KV cache stays its own; the
target's cache is never copied into it).

Every device computation runs in libspecdec.so; this module only sequences
calls and keeps the host-side token log.
"""
from __future__ import annotations

import ctypes
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import binding


# ---------------------------------------------------------------- Alg. 2: cache policy (pure host logic)
class CachePolicy:
    """Resident set of at most K drafts; each entry is 'loading' or 'resident'."""

    def __init__(self, capacity: int):
        if capacity < 1:
            raise ValueError("capacity must be >= 1")
        self.K = capacity
        self.state: Dict[int, str] = {}

    @staticmethod
    def ranking(scores: Dict[int, float]) -> List[int]:
        """R_i: drafts by decreasing score (ties: lower id first)."""
        return sorted(scores, key=lambda d: (-scores[d], d))

    def update(self, scores: Dict[int, float], active: Optional[int]) -> List[tuple]:
        """One cache update (Alg. 2).  Returns the actions taken, in order:
        ("evict", d) and ("prefetch", d).  The caller issues the prefetches."""
        target = self.ranking(scores)[:self.K]
        actions = []
        for d in target:
            if d in self.state:  # resident or being prefetched
                continue
            while len(self.state) == self.K:
                victims = [e for e in self.state if e not in target and e != active]
                if not victims:
                    break
                e = min(victims, key=lambda e: (scores[e], e))
                del self.state[e]
                actions.append(("evict", e))
            if len(self.state) < self.K:
                self.state[d] = "loading"
                actions.append(("prefetch", d))
        return actions

    def mark_resident(self, d: int):
        if self.state.get(d) == "loading":
            self.state[d] = "resident"

    def resident(self) -> List[int]:
        return [d for d, s in self.state.items() if s == "resident"]

    def select(self, scores: Dict[int, float], current: Optional[int]) -> Optional[int]:
        """Alg. 3: the best-scored draft among those resident now (never a
        loading one); keeps `current` when nothing is resident."""
        res = self.resident()
        if not res:
            return current
        return min(res, key=lambda d: (-scores[d], d))


# ---------------------------------------------------------------- the bandit baseline (pure host logic)
class UCBPolicy:
    """MAB-Async's draft selection (the exploration-based baseline of Sec. 4.1):
    explore every draft once, in order, then pick the draft maximising
    mean reward + c * sqrt(ln t / n_d) over the rewards observed so far
    (t = observations made, n_d = observations of draft d; ties: lower id)."""

    def __init__(self, n_drafts: int, c: float = 2.0):
        if n_drafts < 1:
            raise ValueError("need at least one draft")
        self.n = np.zeros(n_drafts, np.int64)
        self.total = np.zeros(n_drafts, np.float64)
        self.c = float(c)

    def observe(self, d: int, reward: float):
        self.n[d] += 1
        self.total[d] += float(reward)

    def select(self) -> int:
        unexplored = np.flatnonzero(self.n == 0)
        if unexplored.size:
            return int(unexplored[0])
        t = float(self.n.sum())
        index = self.total / self.n + self.c * np.sqrt(np.log(t) / self.n)
        return int(np.argmax(index))  # (first maximum: lower id on ties)


def observed_utility(schedule: Sequence[int], n_drafts: int, noise: float = 0.1, seed: int = 13):
    """Per scheduling interval, the utility a run of each draft would show
    (the reward a bandit observes for the draft it ran): 1.0 for the draft
    the schedule prefers in that interval, 0.5 for the others, plus
    N(0, noise^2).  Random weights give every draft the same acceptance, so
    this synthetic signal stands in for the measured acceptance."""
    rng = np.random.default_rng(seed)
    return [{d: (1.0 if d == s else 0.5) + float(rng.normal(0.0, noise)) for d in range(n_drafts)}
            for s in schedule]


# ---------------------------------------------------------------- synthetic prediction
def score_stream(schedule: Sequence[int], n_drafts: int, noise: float = 0.1, seed: int = 11):
    """Per scheduling point, a score per draft: the draft the schedule prefers
    at that point scores 1.0, the others 0.5, plus N(0, noise^2) (a stand-in
    for the predictor's probabilities P(d | x_i))."""
    rng = np.random.default_rng(seed)
    out = []
    for s in schedule:
        out.append({d: (1.0 if d == s else 0.5) + float(rng.normal(0.0, noise)) for d in range(n_drafts)})
    return out


# ---------------------------------------------------------------- device side
class HostImage:
    """Pinned host copy of the target's packed image prefix (LM head + the first
    `max_layers` layers): the backing storage of every draft."""

    def __init__(self, dw: binding.DeviceWeights, max_layers: int):
        import torch
        self.shape = dw.shape.with_layers(dw.n_layers)
        off0, nb = binding.packed_range(self.shape, 0, max_layers)
        self.nbytes = off0 + nb
        self.head_bytes = off0
        self.host = torch.empty(self.nbytes, dtype=torch.uint8, pin_memory=True)
        self.host.copy_(dw.packed[:self.nbytes])
        torch.cuda.current_stream().synchronize()


class Slot:
    """One resident slot: a device buffer in the packed-image format holding the
    shared LM head (copied once) and the layers of the draft loaded into it."""

    def __init__(self, image: HostImage, dw: binding.DeviceWeights):
        import torch
        self.image = image
        self.buf = torch.empty(image.nbytes, dtype=torch.uint8, device=dw.packed.device)
        self.buf[:image.head_bytes].copy_(dw.packed[:image.head_bytes])
        torch.cuda.current_stream().synchronize()
        self.event = binding.Event()
        self.draft: Optional[int] = None

    def load_async(self, draft: int, n_layers: int, copy_stream) -> int:
        off, nb = binding.packed_range(self.image.shape, 0, n_layers)
        binding._check(binding.lib().specdec_load_async(self.buf.data_ptr() + off, self.image.host.data_ptr() + off,
                                                        nb, binding._stream(copy_stream), self.event.handle),
                       "specdec_load_async")
        self.draft = draft
        return nb


@dataclass
class RunStats:
    iterations: int = 0
    tokens: int = 0
    switches: int = 0
    reloads: int = 0
    reload_bytes: int = 0
    blocked_ms: float = 0.0       # host time spent waiting for a reload (naive switching)
    catchup_tokens: int = 0
    wall_ms: float = 0.0
    active: List[int] = field(default_factory=list)    # draft run in each interval
    desired: List[int] = field(default_factory=list)   # the schedule's preferred draft
    selected: List[int] = field(default_factory=list)  # the policy's choice (runs unless still loading)
    # Execution time breakdown (Sec. 4.3, "Execution Breakdown"): host wall time of
    # the intervals decoded with the policy's preferred draft (desired) or with
    # another resident draft while the preferred one is not available (fallback),
    # and of the scheduling decisions themselves (prediction).  An interval runs
    # from the end of its scheduling decision to the synchronising drain of its
    # iteration log at the next point, so its GPU work is inside it.
    desired_ms: float = 0.0
    fallback_ms: float = 0.0
    prediction_ms: float = 0.0

    def fallback_fraction(self) -> float:
        """Intervals spent on another draft than the one the policy selected
        (its selection not resident yet): the paper's fallback execution."""
        if not self.active:
            return 0.0
        return float(np.mean([a != s for a, s in zip(self.active, self.selected)]))

    def time_breakdown(self) -> Dict[str, float]:
        """Fractions of desired execution, fallback execution and prediction time."""
        total = self.desired_ms + self.fallback_ms + self.prediction_ms
        if total <= 0:
            return {"desired": 0.0, "fallback": 0.0, "prediction": 0.0}
        return {"desired": self.desired_ms / total, "fallback": self.fallback_ms / total,
                "prediction": self.prediction_ms / total}


class SwitchingRunner:
    """Greedy or sampled speculative decoding of one sequence with a draft that
    changes at scheduling points (every `interval` iterations).

    mode "resident": every draft runs from the resident target image; the active
        draft is the preferred one at each point (switch cost: catch-up only).
    mode "reload": one slot; switching to a draft that is not in it blocks on
        its reload (naive dynamic switching).
    mode "memspec": `capacity` slots managed by CachePolicy (Alg. 2), prefetches
        overlapped with decoding, and the best resident draft runs (Alg. 3).
    mode "mab": `capacity` slots and the MAB-Async baseline: UCBPolicy picks a
        draft from the utilities observed for the drafts it ran; a selection
        that is not resident is loaded asynchronously (into a free slot, else
        the slot of the least recently run draft other than the active one)
        while decoding continues with the active draft.
    """

    def __init__(self, dw, target, kv_t, draft_layers: Sequence[int], gamma: int, temperature: float, seed: int,
                 capacity_ctx: int, mode: str, slots: int = 1, image: Optional[HostImage] = None):
        import torch
        self.dw, self.target, self.kv_t = dw, target, kv_t
        self.layers = list(draft_layers)
        self.gamma, self.T, self.seed, self.mode = gamma, temperature, seed, mode
        self.rows = max(64, gamma + 1)  # (draft handles: catch-up forwards in chunks of up to 64 tokens)
        self.cap = capacity_ctx
        self.copy = torch.cuda.Stream()
        # per draft: its own KV cache (layer count of the draft)
        self.kv = {}
        self.models_resident = {}
        for d, k in enumerate(self.layers):
            m = binding.Model(dw, k, max_rows=self.rows, max_ctx=capacity_ctx)
            self.models_resident[d] = m
            self.kv[d] = binding.KVCache(m, 1, capacity_ctx)
        self.slots: List[Slot] = []
        if mode not in ("resident", "reload", "memspec", "mab"):
            raise ValueError(f"unknown mode {mode!r}")
        if mode in ("reload", "memspec", "mab"):
            if image is None:
                image = HostImage(dw, max(self.layers))
            self.slots = [Slot(image, dw) for _ in range(slots)]
        self.policy = CachePolicy(slots) if mode == "memspec" else None
        self._slot_models = {}
        self.sd = None
        self.text: List[int] = []

    # -- models and KV
    def _model(self, d: int):
        if self.mode == "resident":
            return self.models_resident[d]
        s = next(i for i, sl in enumerate(self.slots) if sl.draft == d)
        key = (d, s)
        if key not in self._slot_models:
            self._slot_models[key] = binding.Model(self.dw, self.layers[d], max_rows=self.rows,
                                                   max_ctx=self.cap, packed=self.slots[s].buf)
        return self._slot_models[key]

    def prefill(self, prompt: np.ndarray):
        """Commit the prompt into the target and every draft (set-up, untimed)."""
        import torch
        tok = torch.from_numpy(np.ascontiguousarray(prompt.reshape(1, -1), dtype=np.int32)).cuda()
        binding.specdec_prefill(self.target, self.kv_t, tok)
        for d in range(len(self.layers)):
            binding.specdec_prefill(self.models_resident[d], self.kv[d], tok)
        self.text = [int(t) for t in prompt.reshape(-1)]
        torch.cuda.synchronize()

    def start_from_context(self, length: int, pending: int):
        """Start from a resident context of `length` positions already installed in
        the target's and every draft's cache (tokens unknown: only tokens after it
        are ever re-processed) with `pending` as the next input token."""
        for kv in [self.kv_t] + [self.kv[d] for d in range(len(self.layers))]:
            kv.set_state([length], [[0, pending]], [1])
        self.text = [-1] * length + [int(pending)]

    def _catch_up(self, d: int, model, stats: RunStats):
        """Bring draft d's cache up to the committed text: a forward over the
        tokens it has not processed; its pending token becomes the target's."""
        import torch
        st = self.kv[d].read_state()
        n_done = int(st["len"][0])
        missing = self.text[n_done:]
        if len(missing) <= int(st["n_pending"][0]) and st["pending"][0, -1] == self.text[-1]:
            return  # already in step
        tok = torch.tensor([missing], dtype=torch.int32, device="cuda")
        binding.specdec_prefill(model, self.kv[d], tok)
        stats.catchup_tokens += len(missing) - 1

    def _ensure_in_slot_blocking(self, d: int, stats: RunStats):
        """Naive switching: load d into the (only) slot and wait for it."""
        sl = self.slots[0]
        if sl.draft == d and sl.event.query():
            return
        t0 = time.perf_counter()
        stats.reload_bytes += sl.load_async(d, self.layers[d], self.copy)
        stats.reloads += 1
        sl.event.wait()  # the compute stream waits for the copy
        import torch
        torch.cuda.current_stream().synchronize()
        stats.blocked_ms += (time.perf_counter() - t0) * 1e3

    # -- the loop
    def run(self, n_iterations: int, schedule: Sequence[int], scores: Sequence[Dict[int, float]], interval: int,
            max_tokens: Optional[int] = None, utility: Optional[Sequence[Dict[int, float]]] = None,
            ucb_c: float = 2.0) -> RunStats:
        """`scores`: the predictor's per-point scores (memspec); `utility`: the
        per-interval utility a bandit observes for the draft it ran (mab)."""
        import torch
        stats = RunStats()
        g = self.gamma
        if self.sd is None:
            self.sd = binding.SpecDecoder(self.target, self.models_resident[0], self.kv_t, self.kv[0], g, self.T,
                                          self.seed)
        sd = self.sd
        active = None
        if self.mode == "memspec":
            # Alg. 3, set-up: rank with the first prediction, load the initial draft, prepare the cache
            first = CachePolicy.ranking(scores[0])[0]
            self.policy.state[first] = "loading"
            self.slots[0].load_async(first, self.layers[first], self.copy)
            stats.reloads += 1
            stats.reload_bytes += binding.packed_range(self.slots[0].image.shape, 0, self.layers[first])[1]
            self.slots[0].event.wait()
            torch.cuda.current_stream().synchronize()
            self.policy.mark_resident(first)
            active = first
            self._issue(self.policy.update(scores[0], active), stats)
        bandit = None
        last_run = {}
        if self.mode == "mab":
            if utility is None:
                raise ValueError("mode 'mab' needs the observed utility stream")
            bandit = UCBPolicy(len(self.layers), ucb_c)
            first = bandit.select()
            self._load_into_slot(first, active=None, last_run=last_run, stats=stats)
            self.slots[0].event.wait()
            torch.cuda.current_stream().synchronize()
            active = first
        # Device-side log of each iteration's outcome (drafted tokens, A, next),
        # read by the host once per scheduling point (no per-iteration sync).
        log_d = torch.zeros((interval, g), dtype=torch.int32, device="cuda")
        log_a = torch.zeros(interval, dtype=torch.int32, device="cuda")
        log_n = torch.zeros(interval, dtype=torch.int32, device="cuda")
        pending_log = 0

        def drain():
            nonlocal pending_log
            if pending_log == 0:
                return False
            d_h, a_h, n_h = log_d[:pending_log].cpu().numpy(), log_a[:pending_log].cpu().numpy(), \
                log_n[:pending_log].cpu().numpy()
            for j in range(pending_log):
                A = int(a_h[j])
                if A < 0:
                    raise RuntimeError("non-finite distribution during the run")
                self.text += [int(x) for x in d_h[j, :A]] + [int(n_h[j])]
                stats.tokens += A + 1
            pending_log = 0
            return max_tokens is not None and stats.tokens >= max_tokens

        t_exec = None          # start of the interval being decoded
        exec_fallback = False  # whether it runs another draft than the policy's choice

        def close_interval(now):
            if t_exec is not None:
                if exec_fallback:
                    stats.fallback_ms += (now - t_exec) * 1e3
                else:
                    stats.desired_ms += (now - t_exec) * 1e3

        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for it in range(n_iterations):
            if it % interval == 0:
                stop = drain()
                now = time.perf_counter()
                close_interval(now)
                t_exec = None
                if stop:
                    break
                t_pred, blocked0 = now, stats.blocked_ms
                point = it // interval
                desired = schedule[point]
                if self.mode == "mab":
                    if point > 0:
                        bandit.observe(active, utility[point - 1][active])
                    sel = bandit.select()
                    resident = [sl.draft for sl in self.slots if sl.draft is not None and sl.event.query()]
                    if sel in resident:
                        nxt = sel
                    else:
                        if all(sl.draft != sel for sl in self.slots):  # not already loading
                            self._load_into_slot(sel, active, last_run, stats)
                        nxt = active  # fallback: keep decoding with the active draft
                    stats.selected.append(int(sel))
                elif self.mode == "memspec":
                    for sl in self.slots:  # loads that completed since the last point
                        if sl.draft is not None and self.policy.state.get(sl.draft) == "loading" and sl.event.query():
                            self.policy.mark_resident(sl.draft)
                    nxt = self.policy.select(scores[point], active)
                    self._issue(self.policy.update(scores[point], nxt), stats)
                    stats.selected.append(int(CachePolicy.ranking(scores[point])[0]))
                else:
                    nxt = desired
                    if self.mode == "reload":
                        self._ensure_in_slot_blocking(nxt, stats)
                    stats.selected.append(int(desired))
                # (a blocking reload is counted in blocked_ms, not as prediction)
                stats.prediction_ms += (time.perf_counter() - t_pred) * 1e3 - (stats.blocked_ms - blocked0)
                if nxt != active:
                    if active is not None:
                        stats.switches += 1
                    model = self._model(nxt)
                    self._catch_up(nxt, model, stats)
                    sd.draft, sd.kv_d = model, self.kv[nxt]
                    active = nxt
                stats.desired.append(int(desired))
                stats.active.append(int(active))
                last_run[active] = point
                t_exec = time.perf_counter()
                exec_fallback = active != stats.selected[-1]
            sd.step(it)
            log_d[pending_log].copy_(sd.d[0])
            log_a[pending_log:pending_log + 1].copy_(sd.n_acc[:1])
            log_n[pending_log:pending_log + 1].copy_(sd.next[:1])
            pending_log += 1
            stats.iterations += 1
        drain()
        torch.cuda.synchronize()
        now = time.perf_counter()
        close_interval(now)
        stats.wall_ms = (now - t0) * 1e3
        return stats

    def _load_into_slot(self, d: int, active: Optional[int], last_run: Dict[int, int], stats: RunStats):
        """MAB-Async's reactive load: a free slot, else the slot of the least
        recently run draft that is not the active one (none: no load)."""
        free = [sl for sl in self.slots if sl.draft is None]
        if free:
            sl = free[0]
        else:
            victims = [sl for sl in self.slots if sl.draft != active]
            if not victims:
                return
            sl = min(victims, key=lambda x: (last_run.get(x.draft, -1), x.draft))
        stats.reload_bytes += sl.load_async(d, self.layers[d], self.copy)
        stats.reloads += 1

    def _issue(self, actions, stats: RunStats):
        """Carry out the policy's actions: an evicted draft frees its slot; a
        prefetch goes into a free slot on the copy stream (non-blocking)."""
        for kind, d in actions:
            if kind == "evict":
                for sl in self.slots:
                    if sl.draft == d:
                        sl.draft = None
            else:
                sl = next(s for s in self.slots if s.draft is None)
                stats.reload_bytes += sl.load_async(d, self.layers[d], self.copy)
                stats.reloads += 1
