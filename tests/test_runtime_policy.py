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
