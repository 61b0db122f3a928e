"""Reader for the hand-worked text fixtures under tests/golden/ (no method arithmetic)."""
import os
from fractions import Fraction

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_blocks(fname):
    blocks, cur = [], {}
    with open(os.path.join(GOLDEN, fname)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key == "name" and cur:
                blocks.append(cur)
                cur = {}
            cur[key] = vals
    if cur:
        blocks.append(cur)
    return blocks


def ints(v):
    return [int(x) for x in v]


def fracs(v):
    return [Fraction(x) for x in v]
