"""Pins for KV commit / rollback bookkeeping (CPU only): exhaustive over A."""
import pytest

from oracle.kvstate import SeqState, commit_draft, commit_target


@pytest.mark.parametrize("g", [1, 2, 4, 6, 8])
@pytest.mark.parametrize("n_pending", [1, 2])
def test_commit_all_accept_counts(g, n_pending):
    L = 100
    d = list(range(1000, 1000 + g))
    for A in range(g + 1):
        t = commit_target(SeqState(L, [7]), A, g, 55)
        assert t.length == L + A + 1 and t.pending == [55]
        # the draft is one behind when it still holds two pending tokens
        dl = L + 1 - n_pending
        pend = [9] * n_pending
        dr = commit_draft(SeqState(dl, pend), A, g, d, 55)
        # invariant: draft committed + pending == target committed + pending
        assert dr.length + len(dr.pending) == t.length + len(t.pending)
        if A == g:
            assert dr.pending == [d[-1], 55] and dr.length == t.length - 1
        else:
            assert dr.pending == [55] and dr.length == t.length


def test_commit_rejects_bad_counts():
    with pytest.raises(ValueError):
        commit_target(SeqState(0, [1]), 5, 4, 0)
    with pytest.raises(ValueError):
        commit_draft(SeqState(0, [1, 2, 3]), 0, 4, [0] * 4, 0)
