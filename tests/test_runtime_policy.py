"""The draft cache policy (Sec. 3.3, Alg. 2) and the best-resident selection
(Sec. 3.4, Alg. 3), checked on scripted score sequences against what the
paper's text prescribes: the target set is the top K of the ranking; a missing
target draft is prefetched into a free slot; when the cache is full the
lowest-scored resident draft outside the target set is evicted, never the
active one; a draft still loading is never selected."""
import pytest

from paper_2608_10362_amd.runtime import CachePolicy, score_stream


def test_ranking_is_descending_with_id_ties():
    assert CachePolicy.ranking({0: 0.2, 1: 0.9, 2: 0.9, 3: 0.1}) == [1, 2, 0, 3]


def test_prefetches_the_top_k_into_free_slots():
    p = CachePolicy(2)
    acts = p.update({0: 0.1, 1: 0.8, 2: 0.6, 3: 0.3}, active=None)
    assert acts == [("prefetch", 1), ("prefetch", 2)]
    assert p.state == {1: "loading", 2: "loading"}
    assert p.update({0: 0.1, 1: 0.8, 2: 0.6, 3: 0.3}, active=None) == []  # nothing new


def test_evicts_lowest_scored_outside_the_target_set():
    p = CachePolicy(2)
    p.state = {0: "resident", 1: "resident"}
    # targets {2, 3}; 0 is active (protected), so 1 goes, and only one slot frees up
    acts = p.update({0: 0.1, 1: 0.2, 2: 0.9, 3: 0.8}, active=0)
    assert acts == [("evict", 1), ("prefetch", 2)]
    assert p.state == {0: "resident", 2: "loading"}
    # next point: 0 no longer active -> it can make room for 3
    acts = p.update({0: 0.1, 1: 0.2, 2: 0.9, 3: 0.8}, active=2)
    assert acts == [("evict", 0), ("prefetch", 3)]


def test_eviction_order_is_by_ascending_score():
    p = CachePolicy(3)
    p.state = {0: "resident", 1: "resident", 2: "resident"}
    acts = p.update({0: 0.5, 1: 0.3, 2: 0.4, 3: 0.9, 4: 0.8}, active=None)
    # targets {3, 4, 0}: 1 (0.3) then 2 (0.4) are evicted
    assert acts == [("evict", 1), ("prefetch", 3), ("evict", 2), ("prefetch", 4)]


def test_active_draft_is_protected_even_when_everything_else_is_wanted():
    p = CachePolicy(1)
    p.state = {0: "resident"}
    assert p.update({0: 0.0, 1: 1.0}, active=0) == []  # no victim: no prefetch, no blocking
    assert p.state == {0: "resident"}


def test_select_only_resident_drafts():
    p = CachePolicy(2)
    p.state = {0: "resident", 1: "loading"}
    scores = {0: 0.2, 1: 0.9, 2: 0.5}
    assert p.select(scores, current=0) == 0  # the better one is still loading
    p.mark_resident(1)
    assert p.select(scores, current=0) == 1
    q = CachePolicy(2)
    q.state = {1: "loading"}
    assert q.select(scores, current=None) is None


def test_score_stream_prefers_the_scheduled_draft():
    sched = [0, 2, 1, 1]
    s = score_stream(sched, 3, noise=0.05, seed=3)
    assert [CachePolicy.ranking(x)[0] for x in s] == sched


# ---------------------------------------------------------------- MAB-Async's UCB selection
def test_ucb_explores_every_draft_once_in_order():
    from paper_2608_10362_amd.runtime import UCBPolicy
    u = UCBPolicy(3, c=2.0)
    seen = []
    for r in (0.2, 0.9, 0.5):
        d = u.select()
        seen.append(d)
        u.observe(d, r)
    assert seen == [0, 1, 2]


def test_ucb_index_matches_the_formula_by_hand():
    import math
    from paper_2608_10362_amd.runtime import UCBPolicy
    u = UCBPolicy(3, c=2.0)
    obs = [(0, 1.0), (1, 0.5), (2, 0.6), (0, 0.8), (1, 0.7)]
    for d, r in obs:
        u.observe(d, r)
    t = 5.0
    idx = [(1.0 + 0.8) / 2 + 2.0 * math.sqrt(math.log(t) / 2),
           (0.5 + 0.7) / 2 + 2.0 * math.sqrt(math.log(t) / 2),
           0.6 + 2.0 * math.sqrt(math.log(t) / 1)]
    assert u.select() == max(range(3), key=lambda d: (idx[d], -d))  # draft 2: its bonus term dominates
    u2 = UCBPolicy(2, c=0.0)  # no exploration bonus: the higher mean, ties to the lower id
    u2.observe(0, 0.5)
    u2.observe(1, 0.5)
    assert u2.select() == 0


def test_ucb_settles_on_the_best_draft_of_a_stationary_stream():
    import numpy as np
    from paper_2608_10362_amd.runtime import UCBPolicy
    rng = np.random.default_rng(0)
    means = [0.5, 0.8, 0.55]
    u = UCBPolicy(3, c=0.5)
    picks = []
    for _ in range(400):
        d = u.select()
        u.observe(d, means[d] + rng.normal(0, 0.1))
        picks.append(d)
    assert np.mean(np.array(picks[-100:]) == 1) > 0.9


def test_observed_utility_prefers_the_scheduled_draft():
    from paper_2608_10362_amd.runtime import observed_utility
    sched = [0, 2, 1, 1]
    util = observed_utility(sched, 3, noise=0.0)
    for s, u in zip(sched, util):
        assert u[s] == 1.0 and all(u[d] == 0.5 for d in range(3) if d != s)
