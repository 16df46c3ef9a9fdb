"""Parser for the hand-worked fixture ``hand_example.txt``."""
import fractions
import os

import numpy as np

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_example.txt")


def load(path=PATH):
    d = {"tables": [], "sum": {}, "wsum": {}, "mean": {}}
    cur = None
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            if key in ("T", "B", "R", "C"):
                d[key] = int(rest[0])
                cur = None
            elif key == "table":
                cur = []
                d["tables"].append(cur)
            elif key in ("offsets", "indices", "flags", "flags_per_table"):
                d[key] = [int(x) for x in rest]
                cur = None
            elif key == "weights":
                d[key] = [float(x) for x in rest]
                cur = None
            elif key in ("sum", "wsum", "mean"):
                r, s, *vals = rest
                # exact rationals, rounded once to the nearest double
                d[key][(int(r), int(s))] = [float(fractions.Fraction(x)) for x in vals]
                cur = None
            else:
                cur.append([float(x) for x in [key] + rest])
    R, B = d["R"], d["B"]
    S = B // R
    for k in ("sum", "wsum", "mean"):
        arr = np.zeros((R, S, len(next(iter(d[k].values())))))
        for (r, s), v in d[k].items():
            arr[r, s] = v
        d[k] = arr
    return d


GEMV_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gemv_hand.txt")


def load_gemv(path=GEMV_PATH):
    """Parse the hand-worked GEMV + AllReduce fixture: per-rank A rows and x,
    and the expected y and sum of |terms|."""
    A, x = {}, {}
    d = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            vals = [float(v) for v in rest]
            if key.startswith("A"):
                A.setdefault(int(key[1:]), []).append(vals)
            elif key.startswith("x"):
                x[int(key[1:])] = vals
            else:
                d[key] = np.array(vals)
    R = len(A)
    d["A"] = [np.array(A[r]) for r in range(R)]
    d["x"] = [np.array(x[r]) for r in range(R)]
    return d


BACKWARD_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "backward_hand.txt")


def load_backward(path=BACKWARD_PATH):
    """Parse the hand-worked backward fixture: the pooled gradient rows and
    the expected per-lookup rows (exact rationals rounded once to fp32) for
    the sum, weighted-sum and mean modes."""
    d = {"grad": [], "sum": [], "wsum": [], "mean": []}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            d[key].append([float(fractions.Fraction(v)) for v in rest])
    out = {"grad": np.array(d["grad"], dtype=np.float32)}
    for k in ("sum", "wsum", "mean"):
        out[k] = np.array(d[k], dtype=np.float64).astype(np.float32)
    return out
