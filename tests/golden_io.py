"""Readers for the text fixtures under tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def appendix_cases():
    """Parse appendix_a_5x5.txt into a list of (params dict, expected array)."""
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "appendix_a_5x5.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("case"):
                parts = line.split()
                prm = dict(name=parts[1])
                for kv in parts[2:]:
                    k, v = kv.split("=")
                    prm[k] = int(v, 0)
                cur = (prm, [])
                cases.append(cur)
            else:
                cur[1].append([float(v) for v in line.split()])
    return [(p, np.array(rows)) for p, rows in cases]


def ppk1_small():
    out = {}
    with open(os.path.join(GOLDEN, "ppk1_small.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = [float(v) if "." in v else int(v) for v in vals]
    return out
