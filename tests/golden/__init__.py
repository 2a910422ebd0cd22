"""Loader for the hand-derived fixtures in this folder.

Each fixture is a text file: '#' lines hold the derivation and the passage of
the paper it follows; 'key: value' lines hold scalars or matrices, with rows
separated by ';' and entries written as exact rationals ('4/3') or 'inf'.
"""
import os
from fractions import Fraction

HERE = os.path.dirname(os.path.abspath(__file__))


def _num(tok):
    if tok in ("inf", "+inf"):
        return float("inf")
    if tok in ("exact", "paper_eq6"):
        return tok
    return Fraction(tok)


def load(name):
    out = {}
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            rows = [r.split() for r in val.split(";")]
            vals = [[_num(t) for t in r] for r in rows]
            if len(vals) == 1 and len(vals[0]) == 1:
                out[key.strip()] = vals[0][0]
            elif len(vals) == 1:
                out[key.strip()] = vals[0]
            else:
                out[key.strip()] = vals
    return out
