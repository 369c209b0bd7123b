"""Oracle: microbatch Orders for one pipeline stage and their validity rules.

`Split` replicates a stage's Chunks per microbatch and `Order` adds temporal
edges between consecutive entries (Piper Section 4.1). The worker runs
entries in that order and keeps a forward's activations until the matching
backward consumes them (Section 4.3.2, "Memory management"). Piper rejects
schedules in which a downstream worker would see microbatches in a different
order than the upstream produced them (Section 4.3.2, "Communication
management"); on one stage this means the F entries and the B entries each
appear in increasing microbatch order.

The PASS dimension also has Bi (backward for the inputs) and Bw (backward for
the weights), which split B for schedules such as ZeroBubble (Section 4.1,
Split). Reading of the rules for split backwards: a microbatch has either
one B or one Bi followed later by one Bw; Bi produces the input gradient the
upstream stage consumes, so B and Bi entries together are in increasing
microbatch order; Bw only adds into the local gradient accumulator, so Bw
entries may come in any order (the accumulator receives them in that
order). A microbatch keeps its stashed activations from F until its B or
Bw, and its saved output gradients from Bi until its Bw.

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


def one_f_one_b_split(M: int, P: int, s: int, w_delay: int) -> List[Tuple[int, str]]:
    """1F1B with every B split into Bi and Bw: Bw(mb) follows Bi(mb + w_delay)
    (or the last Bi); the remaining Bw entries close the Order in microbatch
    order. w_delay = 0 puts each Bw right after its Bi."""
    out = []
    pending = []
    for mb, ps in one_f_one_b(M, P, s):
        if ps == "F":
            out.append((mb, "F"))
            continue
        out.append((mb, "Bi"))
        pending.append(mb)
        if mb - pending[0] >= w_delay:
            out.append((pending.pop(0), "Bw"))
    out.extend((mb, "Bw") for mb in pending)
    return out


def validate(entries: Sequence[Tuple[int, str]], M: int, max_in_flight: int,
             max_w_pending: int = 1 << 30):
    """Check an Order. Returns (status, peak number of stashed microbatches).

    Rules: for every 0 <= mb < M, (mb, F) appears once and either (mb, B)
    once or (mb, Bi) and (mb, Bw) once each; F(mb) precedes B(mb) / Bi(mb),
    and Bi(mb) precedes Bw(mb); F entries are in increasing mb order, and so
    are the B and Bi entries taken together; the number of microbatches
    between their F and their B or Bw never exceeds max_in_flight, nor the
    number between their Bi and Bw max_w_pending (else STASH_FULL).
    """
    if M <= 0 or not (2 * M <= len(entries) <= 3 * M):
        return BAD_ORDER, 0
    seen = {k: set() for k in ("F", "B", "Bi", "Bw")}
    last_f = last_b = -1
    live = peak = wlive = 0
    for mb, ps in entries:
        if not (0 <= mb < M) or ps not in seen:
            return BAD_ORDER, peak
        if mb in seen[ps]:
            return BAD_ORDER, peak
        if ps == "F":
            if mb <= last_f:
                return BAD_ORDER, peak
            last_f = mb
            live += 1
            peak = max(peak, live)
            if live > max_in_flight:
                return STASH_FULL, peak
        elif ps in ("B", "Bi"):
            if mb not in seen["F"] or mb <= last_b or mb in seen["B"] or mb in seen["Bi"]:
                return BAD_ORDER, peak
            last_b = mb
            if ps == "B":
                live -= 1
            else:
                wlive += 1
                if wlive > max_w_pending:
                    return STASH_FULL, peak
        else:  # Bw
            if mb not in seen["Bi"]:
                return BAD_ORDER, peak
            live -= 1
            wlive -= 1
        seen[ps].add(mb)
    for mb in range(M):
        if mb not in seen["F"] or (mb in seen["B"]) == (mb in seen["Bw"]):
            return BAD_ORDER, peak
    return OK, peak


def parse(text: str) -> List[Tuple[int, str]]:
    """'F0 F1 B0 Bi1 Bw1' -> [(0,'F'), (1,'F'), (0,'B'), (1,'Bi'), (1,'Bw')]."""
    out = []
    for tok in text.split():
        k = 2 if tok[:2] in ("Bi", "Bw") else 1
        out.append((int(tok[k:]), tok[:k]))
    return out
