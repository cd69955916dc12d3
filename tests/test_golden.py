"""The oracle against hand-derived closed-form cases stored under tests/golden/ (CPU only)."""
import json
import os

import numpy as np

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _rle(pairs, dtype):
    return np.concatenate([np.full(n, v, dtype=dtype) for n, v in pairs])


def test_hand_derived_cases():
    with open(os.path.join(HERE, "golden", "hand_small.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        x = _rle(c["x_rle"], np.uint16).reshape(c["M"], c["K"])
        if c["fmt"] == 0:
            ks = np.arange(c["K"])
            q = np.stack([ks - 16, np.full(c["K"], 127)]).astype(np.int8)
            wq = q
        else:
            wq = _rle(c["wq_bytes_rle"], np.uint8).reshape(c["N"], c["K"] // 2)
        s = np.array(c["scales"], dtype=np.float16)
        y, b = oracle.dense(x, wq, s, c["fmt"])
        assert np.array_equal(y, np.array(c["y"])), c["name"]
        assert np.array_equal(b, np.array(c["bound"])), c["name"]
