"""Readers for the small text fixtures under tests/golden/."""
import os
from fractions import Fraction

from conftest import GOLDEN


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                yield line


def read_matrices(name):
    """Return (points, {"AT": rows, "BT": rows, "G": rows}) as Fractions."""
    it = iter(_lines(name))
    points = None
    mats = {}
    for line in it:
        if line.startswith("points:"):
            points = [Fraction(t) for t in line.split(":", 1)[1].split()]
            continue
        name_, rows, cols = line.split()
        mat = []
        for _ in range(int(rows)):
            row = [Fraction(t) for t in next(it).split()]
            assert len(row) == int(cols)
            mat.append(row)
        mats[name_] = mat
    return points, mats


def read_table1():
    rows = {}
    for line in _lines("table1.txt"):
        tok = line.split()
        rows[tok[0]] = dict(D=int(tok[1]), G=int(tok[2]), S=int(tok[3]),
                            zA=float(tok[4]), zB=float(tok[5]), zC=float(tok[6]),
                            su2=float(tok[7]), su3=float(tok[8]))
    return rows


def read_kv(name):
    out = {}
    for line in _lines(name):
        k, v = line.split(":", 1)
        out[k.strip()] = [Fraction(t) for t in v.split()]
    return out
