"""Parse the exact-value fixtures in tests/golden/ (fractions, optionally times sqrt(3))."""
import json
import math
import os
from fractions import Fraction

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def value(s: str) -> float:
    s = s.strip()
    if s == "ln2":
        return math.log(2.0)
    if s.startswith("pi"):
        return math.pi / float(s.split("/")[1]) if "/" in s else math.pi
    if s.endswith("*s3"):
        return float(Fraction(s[:-3])) * math.sqrt(3.0)
    return float(Fraction(s))
