"""KV commit / rollback bookkeeping after one draft-and-verify iteration
(TEST INFRASTRUCTURE ONLY).

The paper keeps one target and the active draft in memory and runs
draft-then-verify iterations (Sec. 3.4, Alg. 3); it does not describe the
caches.  The bookkeeping below follows from what each model has processed:

Target.  The verify pass consumed [x_last, d_1..d_g] at positions
len..len+g.  With A accepted drafts the committed text grows by
[x_last, d_1..d_A] (their K/V are already in place) and the emitted
token ``next`` becomes the single pending token:
    len' = len + A + 1,  pending' = [next].

Draft.  Its step at slot 0 consumed its n pending tokens (1 or 2), slots
1..g-1 consumed d_1..d_{g-1}; d_g was never fed to the draft.  Hence
    len' = len + n + min(A, g - 1),
    pending' = [d_g, next] if A == g else [next].
Rollback is truncation: entries at or beyond len' are overwritten later.
"""
from __future__ import annotations

import dataclasses
from typing import List


@dataclasses.dataclass
class SeqState:
    length: int
    pending: List[int]


def commit_target(st: SeqState, A: int, g: int, next_token: int) -> SeqState:
    if not 0 <= A <= g:
        raise ValueError("accepted count out of range")
    if len(st.pending) != 1:
        raise ValueError("target holds exactly one pending token")
    return SeqState(st.length + A + 1, [int(next_token)])


def commit_draft(st: SeqState, A: int, g: int, d, next_token: int) -> SeqState:
    if not 0 <= A <= g:
        raise ValueError("accepted count out of range")
    n = len(st.pending)
    if n not in (1, 2):
        raise ValueError("draft holds one or two pending tokens")
    new_len = st.length + n + min(A, g - 1)
    pending = [int(d[g - 1]), int(next_token)] if A == g else [int(next_token)]
    return SeqState(new_len, pending)
