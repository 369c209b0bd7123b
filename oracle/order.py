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

An Order may also nest two entries to mark them overlappable (Section 4.1,
Order: a nested list of filters; the runtime interleaves the two sub-DAGs,
Section 4.3.1). Reading for one stage: a nested pair holds two entries of
different microbatches, at most one of which uses the backward's working
buffers (B, Bi) and at most one of which adds into the gradient accumulator
(B, Bw): {F, B}, {F, Bi}, {F, Bw} or {Bi, Bw}. As both may run at once, the
pair takes its stash and weight-pass slots before it frees any: the rules
are checked on the pair with its acquiring entry (F, Bi) first.

Status values mirror the C library: OK, BAD_ORDER, STASH_FULL.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple, Union

Entry = Tuple[int, str]

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


def one_f_one_b_overlap(M: int, P: int, s: int) -> list:
    """1F1B with every steady-state (forward of the next microbatch, backward
    of the oldest) pair nested as an overlapped pair; with no warm-up (W = 0)
    each such pair is one microbatch's F and B, which cannot overlap, and the
    Order stays flat."""
    W = min(P - s - 1, M)
    out: list = [(i, "F") for i in range(W)]
    for i in range(M - W):
        pair = [(W + i, "F"), (i, "B")]
        if W > 0:
            out.append(pair)
        else:
            out.extend(pair)
    out.extend((i, "B") for i in range(M - W, M))
    return out


def one_f_one_b_split_overlap(M: int, P: int, s: int, w_delay: int) -> list:
    """The split 1F1B Order with each Bi that another microbatch's Bw directly
    follows nested with that Bw as an overlapped pair (the weight pass runs
    beside the next input pass); an entry joins at most one pair."""
    seq = one_f_one_b_split(M, P, s, w_delay)
    out: list = []
    i = 0
    while i < len(seq):
        nxt = seq[i + 1] if i + 1 < len(seq) else None
        if seq[i][1] == "Bi" and nxt is not None and nxt[1] == "Bw" and nxt[0] != seq[i][0]:
            out.append([seq[i], nxt])
            i += 2
        else:
            out.append(seq[i])
            i += 1
    return out


_PAIRS = ({"F", "B"}, {"F", "Bi"}, {"F", "Bw"}, {"Bi", "Bw"})


def pair_ok(pair) -> bool:
    """A nested pair: two entries, different microbatches, an allowed kind."""
    if len(pair) != 2:
        return False
    (m0, p0), (m1, p1) = pair
    return m0 != m1 and {p0, p1} in _PAIRS


def flatten(entries) -> List[Entry]:
    """The Order as a flat sequence, each nested pair with its acquiring
    entry (F, Bi) first."""
    out: List[Entry] = []
    for e in entries:
        if isinstance(e, list):
            out.extend(sorted(e, key=lambda x: 0 if x[1] in ("F", "Bi") else 1))
        else:
            out.append(e)
    return out


def validate(entries, M: int, max_in_flight: int, max_w_pending: int = 1 << 30):
    """Check an Order. Returns (status, peak number of stashed microbatches).

    Rules: for every 0 <= mb < M, (mb, F) appears once and either (mb, B)
    once or (mb, Bi) and (mb, Bw) once each; F(mb) precedes B(mb) / Bi(mb),
    and Bi(mb) precedes Bw(mb); F entries are in increasing mb order, and so
    are the B and Bi entries taken together; the number of microbatches
    between their F and their B or Bw never exceeds max_in_flight, nor the
    number between their Bi and Bw max_w_pending (else STASH_FULL). Nested
    pairs must satisfy pair_ok and are checked in their flatten() order.
    """
    for e in entries:
        if isinstance(e, list) and not pair_ok(e):
            return BAD_ORDER, 0
    entries = flatten(entries)
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


def parse(text: str) -> list:
    """'F0 F1 B0 Bi1 Bw1' -> [(0,'F'), (1,'F'), (0,'B'), (1,'Bi'), (1,'Bw')];
    a bracketed group '[F1 B0]' becomes a nested list [(1,'F'), (0,'B')]."""
    out: list = []
    group = None
    for tok in text.replace("[", " [ ").replace("]", " ] ").split():
        if tok == "[":
            group = []
            continue
        if tok == "]":
            out.append(group)
            group = None
            continue
        k = 2 if tok[:2] in ("Bi", "Bw") else 1
        e = (int(tok[k:]), tok[:k])
        (out if group is None else group).append(e)
    return out
