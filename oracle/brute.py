"""Brute-force dense formulation of the MoE layer, for tiny shapes only -- TEST INFRASTRUCTURE.

Independent of moe_oracle.c (shares no code with it): every expert runs on every token
and a routing mask keeps the picked ones, i.e. y[t] = sum_e m[t,e] * FFN_e(x[t]) with
m[t,e] the gate weight of expert e if e is among token t's picks and 0 otherwise.  This is
the dense form that the paper's sparse grouped computation (Algorithm 1, Steps 2-5) must
reproduce.  Routing is done with Python's sort on exact rational keys where possible.
"""
from __future__ import annotations

import math

import numpy as np


def route(x, wg, k, sel_bias=None, renorm=0):
    x = np.asarray(x, np.float64)
    wg = np.asarray(wg, np.float64)
    T, E = x.shape[0], wg.shape[0]
    logits = np.einsum("tj,ej->te", x, wg)
    bias = np.zeros((T, E)) if sel_bias is None else np.broadcast_to(np.asarray(sel_bias, np.float64), (T, E))
    idx = np.empty((T, k), np.int64)
    w = np.empty((T, k))
    for t in range(T):
        score = [logits[t, e] + bias[t, e] for e in range(E)]
        order = sorted(range(E), key=lambda e: (-score[e], e))
        z = [math.exp(v - max(logits[t])) for v in logits[t]]
        s = math.fsum(z)
        picks = order[:k]
        ws = [z[e] / s for e in picks]
        if renorm:
            tot = math.fsum(ws)
            ws = [v / tot for v in ws]
        idx[t] = picks
        w[t] = ws
    return idx, w, logits


def _act(u, g, act):
    if act == "gelu":
        return np.array([v * 0.5 * (1.0 + math.erf(v / math.sqrt(2.0))) for v in u.ravel()]).reshape(u.shape)
    if act == "gelu_tanh":
        c = math.sqrt(2.0 / math.pi)
        return np.array([0.5 * v * (1.0 + math.tanh(c * (v + 0.044715 * v ** 3)))
                         for v in u.ravel()]).reshape(u.shape)
    if act == "swiglu":
        sig = np.array([1.0 / (1.0 + math.exp(-v)) for v in u.ravel()]).reshape(u.shape)
        return u * sig * g
    raise ValueError(act)


def dense_layer(x, wg, w1, w3, w2, k, act="gelu", sel_bias=None, renorm=0, col0=0, f=None):
    """All experts on all tokens, masked by the routing: returns (y, idx, w)."""
    x = np.asarray(x, np.float64)
    E = wg.shape[0]
    F = w1.shape[2]
    if f is None:
        f = F - col0
    idx, w, _ = route(x, wg, k, sel_bias, renorm)
    T, h = x.shape
    mask = np.zeros((T, E))
    for t in range(T):
        for j in range(k):
            mask[t, idx[t, j]] += w[t, j]
    y = np.zeros((T, h))
    for e in range(E):
        W1 = np.asarray(w1[e], np.float64)[:, col0:col0 + f]
        W2 = np.asarray(w2[e], np.float64)[col0:col0 + f, :]
        u = x @ W1
        g = x @ np.asarray(w3[e], np.float64)[:, col0:col0 + f] if act == "swiglu" else None
        out = _act(u, g, act) @ W2
        y += mask[:, e:e + 1] * out
    return y, idx, w
