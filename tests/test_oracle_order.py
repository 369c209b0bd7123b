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
