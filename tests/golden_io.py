"""Reader for the hand-derived fixtures in tests/golden/."""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name: str) -> dict:
    rows = []
    out: dict = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, val = line.partition(":")
            key, val = key.strip(), val.strip()
            if key == "row":
                rows.append([float(v) for v in val.split()])
            elif key == "clusters":
                out[key] = [[int(v) for v in grp.split()] for grp in val.split("|")]
            elif key in ("grid_w", "window"):
                out[key] = int(val)
            elif key in ("layout", "stage1_rows", "stage2_rows"):
                out[key] = val.split()
            elif key.startswith("block_") or key == "angles_deg":
                out[key] = [float(v) for v in val.split()]
            else:
                vals = [int(v) for v in val.split()]
                out[key] = vals[0] if key.startswith("count") else vals
    if rows:
        out["x"] = np.array(rows, dtype=np.float64)
    if "angles_deg" in out:
        t = np.deg2rad(np.array(out["angles_deg"]))
        out["x"] = np.stack([np.cos(t), np.sin(t)], axis=1)
    if "onehot" in out:
        n, d = out["onehot"]
        out["x"] = np.eye(n, d)
    if "layout" in out:
        blocks = {k[len("block_"):]: np.array(v) for k, v in out.items() if k.startswith("block_")}
        out["blocks"] = blocks
        out["x"] = np.stack([blocks[c] for c in out["layout"]])
    return out


def all_merge_cases():
    return sorted(f for f in os.listdir(GOLDEN) if f.startswith("h") and f.endswith(".txt"))


def window_cases():
    return sorted(f for f in os.listdir(GOLDEN) if f.startswith("w") and f.endswith(".txt"))
