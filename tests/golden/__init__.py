"""Readers for the text fixtures in this folder (values cited in each file)."""
from __future__ import annotations

import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def load_worked_example(name: str = "worked_example_eq10_eq11.txt") -> dict:
    rows: dict[str, list] = {}
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            rows.setdefault(key, []).append([float(v) for v in vals])
    N, K = int(rows["N"][0][0]), int(rows["K"][0][0])
    S = np.array(rows["S"][0], dtype=np.int32)
    nS = S.size
    return {
        "N": N,
        "K": K,
        "trits": np.array(rows["trits"], dtype=np.int8),
        "alpha": np.array(rows["alpha"][0], dtype=np.float16),
        "v": np.array(rows["v"][0], dtype=np.float16),
        "x": np.array(rows["x"], dtype=np.float16),
        "S": S,
        "R": np.array(rows["R"], dtype=np.float16).reshape(nS, N // 4),
        "idx": np.array(rows["idx"], dtype=np.uint8).reshape(nS, N // 4),
        "codes": np.array(rows["codes"], dtype=np.uint8),
        "y": np.array(rows["y"], dtype=np.float64),
    }
