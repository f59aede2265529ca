"""Parsers for the text fixtures under tests/golden/."""

import math
import os
from fractions import Fraction

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _in_token(t):
    if t.startswith("ln"):
        return math.log(int(t[2:]))
    return float(t)  # handles inf, -inf, nan and plain numbers


def _out_token(t):
    if t == "nan":
        return float("nan")
    return float(Fraction(t))


def hand_values():
    cases = []
    cur = None
    with open(os.path.join(HERE, "softmax_hand_values.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = dict(name=tok[1], R=int(tok[2]), C=int(tok[3]))
                cases.append(cur)
            elif tok[0] == "in":
                cur["x"] = [_in_token(t) for t in tok[1:]]
            elif tok[0] == "out":
                cur["y"] = [_out_token(t) for t in tok[1:]]
    for c in cases:
        assert len(c["x"]) == len(c["y"]) == c["R"] * c["C"], c["name"]
    return cases


def paper_bank_table():
    banks = None
    rows = []
    with open(os.path.join(HERE, "paper_bank_table.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "banks":
                banks = int(tok[1])
            elif tok[0] == "batch":
                rows.append(dict(name=tok[1], offset=int(tok[2]), R=int(tok[3]), C=int(tok[4]),
                                 flags=[int(t) for t in tok[5:5 + banks]],
                                 overlap=int(tok[5 + banks])))
    return banks, rows


def backward_hand_values():
    """Cases of tests/golden/softmax_backward_hand_values.txt: dicts with name, R, C, dyadic,
    y, dy, dx (floats; dx exact fractions converted once)."""
    cases = []
    cur = None
    with open(os.path.join(HERE, "softmax_backward_hand_values.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = dict(name=tok[1], R=int(tok[2]), C=int(tok[3]), dyadic="dyadic" in tok[4:])
                cases.append(cur)
            elif tok[0] in ("y", "dy", "dx"):
                cur[tok[0]] = [_out_token(t) for t in tok[1:]]
    for c in cases:
        assert len(c["y"]) == len(c["dy"]) == len(c["dx"]) == c["R"] * c["C"], c["name"]
    return cases
