"""Loads the hand-derived check cases of check_cases.json into storage arrays."""
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
STORAGE = {"f32": np.float32, "bf16": np.uint16, "f16": np.uint16, "f8": np.uint8}


def _arr(case, side):
    dt = case["dt" + side]
    if side + "_bits" in case:
        return np.array(case[side + "_bits"], dtype=STORAGE[dt])
    vals = [float(v) for v in case[side]]
    return np.array(vals, dtype=np.float32)


def _val(v):
    return float(v) if isinstance(v, str) else v


def check_cases():
    with open(os.path.join(HERE, "check_cases.json")) as f:
        data = json.load(f)
    out = []
    for c in data["cases"]:
        exp = {k: _val(v) for k, v in c["expect"].items()}
        out.append((c["name"], _arr(c, "a"), c["dta"], _arr(c, "b"), c["dtb"], c["rtol"], c["atol"], exp))
    return out
