"""Reader for the small text fixtures under tests/golden/."""
from fractions import Fraction
import os

import numpy as np

GOLDEN_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name: str) -> dict:
    g = {"score": [], "sig": [], "D": []}
    with open(os.path.join(GOLDEN_DIR, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key in ("score", "D"):
                g[key].append([float(v) for v in vals])
            elif key == "sig":
                g[key].append(vals[0])
            elif key in ("E", "k", "N", "sum", "sumsq"):
                g[key] = int(vals[0])
            else:
                g[key] = float(Fraction(vals[0]))
    g["scores"] = np.array(g.pop("score"), dtype=np.float32)
    g["D"] = np.array(g["D"], dtype=np.uint32)
    g["F"] = np.array([[int(c) for c in s] for s in g.pop("sig")], dtype=np.uint8)
    return g
