"""Pins for the Order oracle (oracle/order.py): the Orders printed in the
paper's DualPipe listing (Piper Section 4.1) as a golden fixture, and 1F1B
sequences listed by hand."""
import os

import pytest

from oracle import order as OO

HERE = os.path.dirname(os.path.abspath(__file__))


def golden_cases():
    out = []
    with open(os.path.join(HERE, "golden", "listing2_orders.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            head, body = line.split(":")
            _, M, status, peak = head.split()
            out.append((int(M), status, int(peak), body.strip()))
    return out


@pytest.mark.parametrize("M,status,peak,body", golden_cases())
def test_listing_orders(M, status, peak, body):
    st, pk = OO.validate(OO.parse(body), M, max_in_flight=M)
    assert st == status
    if status == "OK":
        assert pk == peak


HAND = {
    (4, 2, 0): "F0 F1 B0 F2 B1 F3 B2 B3",
    (3, 5, 1): "F0 F1 F2 B0 B1 B2",
    (16, 8, 7): " ".join(f"F{i} B{i}" for i in range(16)),
    (16, 8, 0): " ".join([f"F{i}" for i in range(7)]
                         + [f"F{7 + i} B{i}" for i in range(9)]
                         + [f"B{i}" for i in range(9, 16)]),
}


@pytest.mark.parametrize("key", sorted(HAND))
def test_1f1b_hand_listed(key):
    M, P, s = key
    seq = OO.one_f_one_b(M, P, s)
    assert seq == OO.parse(HAND[key])
    st, pk = OO.validate(seq, M, max_in_flight=M)
    assert st == "OK" and pk == min(P - s, M)


def test_stash_limit():
    seq = OO.one_f_one_b(16, 8, 0)
    assert OO.validate(seq, 16, 8) == ("OK", 8)
    assert OO.validate(seq, 16, 7)[0] == "STASH_FULL"
    assert OO.validate(OO.gpipe(4), 4, 3)[0] == "STASH_FULL"
    assert OO.validate(OO.gpipe(4), 4, 4) == ("OK", 4)


# Split backwards (PASS values Bi, Bw): 1F1B with every B split, Bw(j) right
# after Bi(j + w_delay), listed by hand.
SPLIT_HAND = {
    (4, 2, 0, 0): "F0 F1 Bi0 Bw0 F2 Bi1 Bw1 F3 Bi2 Bw2 Bi3 Bw3",
    (4, 2, 0, 1): "F0 F1 Bi0 F2 Bi1 Bw0 F3 Bi2 Bw1 Bi3 Bw2 Bw3",
    (3, 5, 1, 5): "F0 F1 F2 Bi0 Bi1 Bi2 Bw0 Bw1 Bw2",
    (3, 1, 0, 1): "F0 Bi0 F1 Bi1 Bw0 F2 Bi2 Bw1 Bw2",
}


@pytest.mark.parametrize("key", sorted(SPLIT_HAND))
def test_1f1b_split_hand_listed(key):
    M, P, s, wd = key
    seq = OO.one_f_one_b_split(M, P, s, wd)
    assert seq == OO.parse(SPLIT_HAND[key])
    # removing the Bw entries and renaming Bi to B gives plain 1F1B
    plain = [(mb, "B" if ps == "Bi" else ps) for mb, ps in seq if ps != "Bw"]
    assert plain == OO.one_f_one_b(M, P, s)
    st, pk = OO.validate(seq, M, max_in_flight=M)
    assert st == "OK"
    need_w = min(wd + 1, M)
    assert OO.validate(seq, M, M, max_w_pending=need_w)[0] == "OK"
    assert OO.validate(seq, M, M, max_w_pending=need_w - 1)[0] == "STASH_FULL"


# (M, Order, status, peak in flight when OK), from the rules: one B or one
# Bi + Bw per microbatch, Bi before Bw, F in order, B and Bi together in
# order, Bw in any order; a microbatch holds its stash until B or Bw.
SPLIT_RULES = [
    (1, "F0 Bi0 Bw0", "OK", 1),
    (1, "F0 Bw0", "BAD_ORDER", 0),
    (1, "F0 Bi0", "BAD_ORDER", 0),
    (1, "F0 Bi0 B0", "BAD_ORDER", 0),
    (1, "F0 Bw0 Bi0", "BAD_ORDER", 0),
    (1, "Bi0 F0 Bw0", "BAD_ORDER", 0),
    (2, "F0 F1 Bi1 Bi0 Bw0 Bw1", "BAD_ORDER", 0),
    (2, "F0 F1 Bi1 B0 Bw1", "BAD_ORDER", 0),
    (2, "F0 F1 B0 Bi1 Bw1", "OK", 2),
    (2, "F0 F1 Bi0 B1 Bw0", "OK", 2),
    (2, "F0 F1 Bi0 Bi1 Bw1 Bw0", "OK", 2),
    (2, "F0 Bi0 F1 Bw0 Bi1 Bw1", "OK", 2),
    (2, "F0 Bi0 Bw0 F1 Bi1 Bw1", "OK", 1),
    (2, "F0 Bi0 Bi0 F1 Bi1 Bw1", "BAD_ORDER", 0),
    (2, "F0 F1 Bi0 Bw0 Bw0 B1", "BAD_ORDER", 0),
]


@pytest.mark.parametrize("M,body,status,peak", SPLIT_RULES)
def test_split_order_rules(M, body, status, peak):
    st, pk = OO.validate(OO.parse(body), M, max_in_flight=M)
    assert st == status
    if status == "OK":
        assert pk == peak


def test_split_pending_weight_passes_hold_the_stash():
    # Bw(0) after F(1): microbatch 0 still holds its stash, so two slots
    seq = OO.parse("F0 Bi0 F1 Bw0 Bi1 Bw1")
    assert OO.validate(seq, 2, 1)[0] == "STASH_FULL"
    assert OO.validate(OO.parse("F0 Bi0 Bw0 F1 Bi1 Bw1"), 2, 1) == ("OK", 1)
    # two pending weight passes need two weight slots
    seq = OO.parse("F0 F1 Bi0 Bi1 Bw0 Bw1")
    assert OO.validate(seq, 2, 2, max_w_pending=1)[0] == "STASH_FULL"
    assert OO.validate(seq, 2, 2, max_w_pending=2) == ("OK", 2)


# Overlapped pairs (nested lists in the Order): two entries of different
# microbatches, F with B/Bi/Bw or Bi with Bw; slots are taken before freed.
PAIR_RULES = [
    (2, "F0 [F1 B0] B1", "OK", 2),
    (2, "F0 [B0 F1] B1", "OK", 2),
    (2, "[F0 F1] B0 B1", "BAD_ORDER", 0),
    (2, "F0 F1 [B0 B1]", "BAD_ORDER", 0),
    (2, "F0 [F1 B1] B0", "BAD_ORDER", 0),
    (2, "[F0 B0] F1 B1", "BAD_ORDER", 0),
    (3, "F0 [F1 Bi0] [F2 Bw0] Bi1 Bi2 Bw1 Bw2", "OK", 3),
    (2, "F0 F1 Bi0 [Bi1 Bw0] Bw1", "OK", 2),
    (2, "F0 F1 [Bi0 Bw1] Bi1 Bw0", "BAD_ORDER", 0),
    (2, "F0 F1 [Bi0 Bi1] Bw0 Bw1", "BAD_ORDER", 0),
    (2, "F0 F1 [B0 Bw1] B1", "BAD_ORDER", 0),
    (3, "F0 [F1 B0] [F2 B1] B2", "OK", 2),
    (2, "F0 [F1 B0 B1]", "BAD_ORDER", 0),
]


@pytest.mark.parametrize("M,body,status,peak", PAIR_RULES)
def test_overlapped_pair_rules(M, body, status, peak):
    st, pk = OO.validate(OO.parse(body), M, max_in_flight=M)
    assert st == status
    if status == "OK":
        assert pk == peak


def test_overlapped_pairs_take_slots_before_freeing():
    assert OO.validate(OO.parse("F0 B0 F1 B1"), 2, 1) == ("OK", 1)
    assert OO.validate(OO.parse("F0 [F1 B0] B1"), 2, 1)[0] == "STASH_FULL"
    seq = OO.parse("F0 F1 Bi0 [Bi1 Bw0] Bw1")
    assert OO.validate(seq, 2, 2, max_w_pending=1)[0] == "STASH_FULL"
    assert OO.validate(OO.parse("F0 F1 Bi0 Bw0 Bi1 Bw1"), 2, 2, max_w_pending=1)[0] == "OK"


@pytest.mark.parametrize("M,P,s", [(4, 2, 0), (16, 8, 0), (3, 5, 1), (2, 2, 0), (5, 1, 0)])
def test_1f1b_overlap_nests_the_steady_state(M, P, s):
    seq = OO.one_f_one_b_overlap(M, P, s)
    assert OO.flatten(seq) == OO.one_f_one_b(M, P, s)
    W = min(P - s - 1, M)
    pairs = [e for e in seq if isinstance(e, list)]
    assert pairs == ([[(W + i, "F"), (i, "B")] for i in range(M - W)] if W else [])
    st, pk = OO.validate(seq, M, M)
    assert st == "OK" and pk == min(P - s, M)


@pytest.mark.parametrize("M,P,s,wd", [(8, 4, 0, 1), (8, 4, 0, 0), (16, 8, 0, 2), (3, 5, 1, 1),
                                      (4, 1, 0, 1), (1, 1, 0, 0)])
def test_split_overlap_nests_bi_with_the_next_bw(M, P, s, wd):
    seq = OO.one_f_one_b_split_overlap(M, P, s, wd)
    assert OO.flatten(seq) == OO.one_f_one_b_split(M, P, s, wd)
    for e in seq:
        if isinstance(e, list):
            (m1, p1), (m2, p2) = e
            assert (p1, p2) == ("Bi", "Bw") and m1 != m2
    st, pk = OO.validate(seq, M, M, M)
    assert st == "OK"
    # w_delay 1 in the steady state: Bi(j) beside Bw(j - 1)
    if wd == 1 and M - min(P - s - 1, M) > 1:
        assert any(isinstance(e, list) for e in seq)
