"""Oracle: microbatch Orders for one pipeline stage and their validity rules.

`Split` replicates a stage's Chunks per microbatch and `Order` adds temporal
edges between consecutive entries (Piper Section 4.1). The worker runs
entries in that order and keeps a forward's activations until the matching
backward consumes them (Section 4.3.2, "Memory management"). Piper rejects
schedules in which a downstream worker would see microbatches in a different
order than the upstream produced them (Section 4.3.2, "Communication
management"); on one stage this means the F entries and the B entries each
appear in increasing microbatch order.

Status values mirror the C library: OK, BAD_ORDER, STASH_FULL.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

OK, BAD_ORDER, STASH_FULL = "OK", "BAD_ORDER", "STASH_FULL"


def one_f_one_b(M: int, P: int, s: int) -> List[Tuple[int, str]]:
    """1F1B for stage s of a P-stage pipeline over M microbatches.

    Warm-up: W = min(P - s - 1, M) forwards; steady state: M - W pairs
    (forward of the next microbatch, backward of the oldest); cool-down: the
    last W backwards.
    """
    W = min(P - s - 1, M)
    out = [(i, "F") for i in range(W)]
    for i in range(M - W):
        out.append((W + i, "F"))
        out.append((i, "B"))
    out.extend((i, "B") for i in range(M - W, M))
    return out


def gpipe(M: int) -> List[Tuple[int, str]]:
    """All forwards, then all backwards."""
    return [(i, "F") for i in range(M)] + [(i, "B") for i in range(M)]


def validate(entries: Sequence[Tuple[int, str]], M: int, max_in_flight: int):
    """Check an Order. Returns (status, peak number of stashed microbatches).

    Rules: every (mb, F) and (mb, B) with 0 <= mb < M appears exactly once;
    F(mb) precedes B(mb); F entries and B entries are each in increasing mb
    order; the number of microbatches between their F and B never exceeds
    max_in_flight (else STASH_FULL).
    """
    if M <= 0 or len(entries) != 2 * M:
        return BAD_ORDER, 0
    seen_f, seen_b = set(), set()
    last_f = last_b = -1
    live = peak = 0
    for mb, ps in entries:
        if not (0 <= mb < M) or ps not in ("F", "B"):
            return BAD_ORDER, peak
        if ps == "F":
            if mb in seen_f or mb <= last_f:
                return BAD_ORDER, peak
            seen_f.add(mb)
            last_f = mb
            live += 1
            peak = max(peak, live)
            if live > max_in_flight:
                return STASH_FULL, peak
        else:
            if mb in seen_b or mb not in seen_f or mb <= last_b:
                return BAD_ORDER, peak
            seen_b.add(mb)
            last_b = mb
            live -= 1
    return OK, peak


def parse(text: str) -> List[Tuple[int, str]]:
    """'F0 F1 B0 B1' -> [(0,'F'), (1,'F'), (0,'B'), (1,'B')]."""
    out = []
    for tok in text.split():
        out.append((int(tok[1:]), tok[0]))
    return out
