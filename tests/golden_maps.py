"""Reader for the hand-worked map files under tests/golden/ (stripe_maps.txt: one-dimensional
blocks; psablock_maps.txt: 3D PSABlocks)."""
import os

import numpy as np

INF = 2 ** 31 - 1
PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "stripe_maps.txt")
PSABLOCK_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "psablock_maps.txt")


def load(path=PATH):
    cases, cur, in_map = [], None, False
    with open(path) as f:
        for raw in f:
            line = raw.strip()
            if not line or line.startswith("#"):
                in_map = False if not line else in_map
                continue
            if line.startswith("["):
                cur = {"name": line.strip("[]"), "empty": None, "map": None}
                cases.append(cur)
                in_map = False
                continue
            if in_map:
                cur["map"].append([int(c) for c in line])
                continue
            key, _, val = (x.strip() for x in line.partition("="))
            if key == "grid":
                cur["grid"] = tuple(int(x) for x in val.split())
            elif key == "pb":
                cur["pb"] = tuple(int(x) for x in val.split())
            elif key == "m":
                cur["m"] = tuple(INF if x == "inf" else int(x) for x in val.split())
            elif key == "kept":
                cur["kept"] = int(val)
            elif key == "empty":
                cur["empty"] = [int(x) for x in val.split()]
            elif key == "map":
                cur["map"], in_map = [], True
    for c in cases:
        if c["map"] is not None:
            c["map"] = np.array(c["map"], dtype=np.uint8)
    return cases
