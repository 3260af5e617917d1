"""Hand-worked fixtures (tests/golden/*.json, each carrying its derivation)."""
import json
import math
import os

import numpy as np

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_attention_hand_case():
    g = _load("attention_hand_case.json")
    q = np.array(g["q"]).reshape(1, 3, 1, 1)
    k = np.array(g["k"]).reshape(1, 3, 1, 1)
    v = np.array(g["v"]).reshape(1, 3, 1, 1)
    O, P = oracle.causal_attention_forward(q, k, v)
    assert np.allclose(P[0, 0], np.array(g["P"]), rtol=0, atol=1e-14)
    assert np.allclose(O.ravel(), g["O"], rtol=0, atol=1e-13)
    dO = np.array(g["dO"]).reshape(1, 3, 1, 1)
    dq, dk, dv = oracle.causal_attention_backward(dO, q, k, v, P)
    assert np.allclose(dv.ravel(), g["dV"], rtol=0, atol=1e-14)
    assert np.allclose(dk.ravel(), g["dK"], rtol=0, atol=1e-13)
    assert np.allclose(dq.ravel(), g["dQ"], rtol=0, atol=1e-13)
    assert math.isclose(g["dQ"][2], -2 / 3 * math.log(2) + 2 * math.log(3), rel_tol=1e-15)


def test_layernorm_hand_case():
    g = _load("layernorm_hand_case.json")
    z = np.array(g["z"])
    out, xhat, _ = oracle.layer_norm_forward(z, np.array(g["gamma"]), np.array(g["beta"]), 0.0)
    assert np.allclose(xhat, g["xhat"], rtol=0, atol=1e-15)
    assert np.allclose(out, g["out"], rtol=0, atol=1e-15)
    _, xh, rs = oracle.layer_norm_forward(z, np.ones(4), np.zeros(4), 0.0)
    dz, _, _ = oracle.layer_norm_backward(np.ones(4), xh, rs, np.ones(4))
    assert np.max(np.abs(dz)) < 1e-15
