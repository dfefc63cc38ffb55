"""Readers for the hand-computed fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def hand_values():
    """[(fmt_name, {field: int}, expected_bits, expected_value)]"""
    out = []
    for tok in _lines("hand_values.txt"):
        fields = {}
        for t in tok[1:-2]:
            k, v = t.split("=")
            fields[k] = int(v, 0)
        out.append((tok[0], fields, int(tok[-2], 16), float(tok[-1])))
    return out


def scale_record():
    d = {tok[0]: tok[1:] for tok in _lines("q4k_scale_record.txt")}
    return ([int(v) for v in d["sc"]], [int(v) for v in d["m"]], bytes(int(v, 16) for v in d["bytes"]))


def plane_sizes():
    return [(t[0], int(t[1]), int(t[2]), int(t[3]), int(t[4])) for t in _lines("plane_sizes.txt")]


def plane_sizes4():
    return [(t[0], int(t[1]), int(t[2]), int(t[3]), int(t[4]), int(t[5])) for t in _lines("plane_sizes4.txt")]
