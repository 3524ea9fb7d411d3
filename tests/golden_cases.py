"""Load the hand-derived fixtures in tests/golden/ into arrays."""
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        fx = json.load(f)
    toks = np.array([fx["tokens"]], np.int32)
    T = toks.shape[1]
    d = fx["d"]
    H = np.zeros((1, T, d), np.float32)
    for r, v in fx["hidden_rows"].items():
        H[0, int(r)] = v
    A = None
    if "attn_rows" in fx:
        A = np.zeros((1, len(fx["attn_rows"]), T), np.float32)
        for r, row in enumerate(fx["attn_rows"]):
            for k, v in row.items():
                A[0, r, int(k)] = v
    return fx, toks, np.array([T], np.int32), H, A


def verify_case(vc):
    Z = np.array([vc["logits"]], np.float32)
    return Z, np.array([vc["draft"]], np.int32), np.array([vc["draft_len"]], np.int32)
