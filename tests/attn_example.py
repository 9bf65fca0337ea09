"""Inputs of the exact FP8 attention example (App. C.6), shared by oracle and GPU tests.

Builds Q, K, V, dO and the saved output for one (sigma, h) setting. No part of
the method's arithmetic is here: only the construction the paper describes.
"""
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fp8_attention_example.json")


def load():
    with open(GOLDEN) as f:
        return json.load(f)


def inputs(ex, dh=64):
    n = ex["keys"]
    Q = np.zeros((1, 1, n, dh), np.float32)
    K = np.zeros((1, 1, n, dh), np.float32)
    V = np.zeros((1, 1, n, dh), np.float32)
    K[..., 0] = 1.0                      # every key's first coordinate is 1
    Q[..., 1] = 1.0                      # every query is orthogonal to every key
    V[0, 0, :, 0] = np.where(np.arange(n) % 2 == 0, 1.0, 1.5)
    return Q, K, V


def saved_and_grad(ex, O, sign, h, dh=64):
    """Saved output with the active entry moved to s + sign*a, and dO = h at that entry."""
    n = ex["keys"]
    Os = O.astype(np.float32).copy()
    Os[0, 0, n - 1, 0] = ex["s"] + sign * ex["a"]
    dO = np.zeros((1, 1, n, dh), np.float32)
    dO[0, 0, n - 1, 0] = h
    return Os, dO
