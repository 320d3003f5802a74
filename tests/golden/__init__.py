"""Fixtures: hand-derived values and (for larger cases) files written by
``make_golden.py``, which calls only the oracle."""
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def _expand(tokens, parse):
    out = []
    i = 0
    while i < len(tokens):
        if tokens[i] in ("zeros", "negzeros"):
            n = int(tokens[i + 1])
            out.extend([parse("-0.0" if tokens[i] == "negzeros" else "0")] * n)
            i += 2
        else:
            out.append(parse(tokens[i]))
            i += 1
    return out


def _parse_value(tok):
    return float.fromhex(tok) if tok.lower().lstrip("-").startswith("0x") else float(tok)


def load_hand_blocks():
    """Blocks of tests/golden/mxfp4_hand_blocks.txt as dicts."""
    blocks = []
    cur = None
    with open(os.path.join(HERE, "mxfp4_hand_blocks.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            if key == "block":
                cur = {"name": rest[0], "what": rest[1] if len(rest) > 1 else ""}
            elif key == "values":
                cur["values"] = np.array(_expand(rest, _parse_value), dtype=np.float32)
            elif key == "scale":
                cur["scale"] = int(rest[0])
            elif key == "codes":
                cur["codes"] = np.array(_expand(rest, lambda t: int(t, 16)), dtype=np.uint8)
            elif key == "packed":
                cur["packed"] = np.array(_expand(rest, lambda t: int(t, 16)), dtype=np.uint8)
            elif key == "end":
                for k, n in (("values", 32), ("codes", 32), ("packed", 16)):
                    assert cur[k].shape == (n,), (cur["name"], k, cur[k].shape)
                blocks.append(cur)
                cur = None
    return blocks
