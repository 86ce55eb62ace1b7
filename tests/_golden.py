"""Reader for the worked-example fixtures under tests/golden/."""

from __future__ import annotations

import os
from fractions import Fraction


def _num(tok: str):
    if "/" in tok:
        return Fraction(tok)
    if tok.startswith("."):
        tok = "0" + tok
    return Fraction(tok)


def load(name: str, raw: bool = False) -> dict:
    """Parse ``key = v1 v2 ...`` lines; ``raw`` keeps the printed tokens."""
    path = os.path.join(os.path.dirname(__file__), "golden", name)
    out = {}
    with open(path) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, _, val = line.partition("=")
            vals = val.split() if raw else [_num(t) for t in val.split()]
            out[key.strip()] = vals[0] if len(vals) == 1 else vals
    return out


def printed_tolerance(printed: str) -> float:
    """Half a unit in the last printed digit."""
    if "." in printed:
        decimals = len(printed.split(".")[1])
    else:
        decimals = 0
    return 0.5 * 10.0 ** (-decimals)
