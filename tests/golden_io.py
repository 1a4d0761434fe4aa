"""Reader for the small text fixtures under tests/golden/.

Each fixture line is `key value value ...`; values may be integers, decimals
or fractions (5/3).  Repeated keys accumulate in order.  Lines starting with
# are comments (the citation of the passage the fixture follows).
"""
import os
from fractions import Fraction

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out.setdefault(key, []).append([Fraction(v) for v in vals])
    return out


def scalar(fx, key):
    return fx[key][0][0]
