"""Brute-force per-token evaluation of a top-k MoE layer (numpy, fp64).

Token-major and written independently of the expert-major C oracle: for
each token, for each of its k slots, apply that expert's SwiGLU FFN with
numpy matrix-vector products and add the gate-weighted result.
"""
import numpy as np


def silu(z):
    return z / (1.0 + np.exp(-z))


def moe_per_token(ids, w, x, weights_f64_of):
    """ids [T,k] int, w [T,k] float, x [T,H] float64; weights_f64_of(e) -> (W1, W3, W2) float64."""
    T, k = ids.shape
    H = x.shape[1]
    y = np.zeros((T, H), np.float64)
    cache = {}
    for t in range(T):
        for j in range(k):
            e = int(ids[t, j])
            if e not in cache:
                cache[e] = weights_f64_of(e)
            W1, W3, W2 = cache[e]
            h = silu(W1 @ x[t]) * (W3 @ x[t])
            y[t] += float(w[t, j]) * (W2 @ h)
    return y
