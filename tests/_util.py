"""Shared helpers of the GPU tests: device transfer, error metrics, routing-certainty rule."""
from __future__ import annotations

import numpy as np

U_F32 = 2.0 ** -23  # unit roundoff with margin: covers round-to-nearest and truncating adds


def to_dev(a, dtype, device="cuda"):
    import torch
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device=device).to(dtype)


def normwise(got, ref) -> float:
    """max_i |got_i - ref_i| / max_i |ref_i| over the whole tensor."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300))


def rowwise(got, ref) -> float:
    """Largest per-row normwise error (each row scaled by its own max |ref|)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    num = np.max(np.abs(got - ref), axis=1)
    den = np.maximum(np.max(np.abs(ref), axis=1), 1e-300)
    return float(np.max(num / den))


def route_certainty(x, wg, sel_bias, logits, idx, k, exact_products: bool):
    """Tokens whose top-k picks are fixed despite fp32 accumulation on the GPU.

    The GPU's logit for expert e differs from the fp64 one by at most
    gamma_n * sum_j |x_j wg_ej| (Higham, Accuracy and Stability of Numerical Algorithms,
    Sec. 3.1; n = h, or h + 1 when the products themselves round) plus one rounding of the
    bias add.  A token's order is certain when every gap between consecutive candidates
    among the first k + 1 scores exceeds the sum of their two error bounds; its pick set is
    certain when the gap between the k-th and (k+1)-th score does.
    Returns (order_certain [T], set_certain [T], err [T, E], score [T, E]).
    """
    x = np.asarray(x, np.float64)
    wg = np.asarray(wg, np.float64)
    h = x.shape[1]
    n = h if exact_products else h + 1
    gamma = n * U_F32 / (1 - n * U_F32)
    S = np.abs(x) @ np.abs(wg).T
    score = logits + (0.0 if sel_bias is None else np.asarray(sel_bias, np.float64))
    err = gamma * S + U_F32 * np.abs(score) + 1e-30
    T, E = logits.shape
    order = np.argsort(-score, axis=1, kind="stable")
    m = min(k + 1, E)
    cand = order[:, :m]
    s = np.take_along_axis(score, cand, axis=1)
    e = np.take_along_axis(err, cand, axis=1)
    ok = np.ones(T, bool)
    for j in range(m - 1):
        ok &= (s[:, j] - s[:, j + 1]) > (e[:, j] + e[:, j + 1])
    set_ok = np.ones(T, bool) if m == k else (s[:, k - 1] - s[:, k]) > (e[:, k - 1] + e[:, k])
    return ok, set_ok, err, score


def compare_routing(gi, gw, oi, ow, x, wg, sel_bias, logits, k, exact_products):
    """Check the GPU's picks and weights against the oracle's under the rounding margin.

    Order-certain tokens must match exactly; tokens whose order is within rounding must
    pick the same set; every other token's picks must be a valid greedy top-k under the
    error bounds: no expert left out of the first j picks may beat pick j by more than
    their two bounds.  Weights are compared per expert id.  Returns (same_set, order_ok).
    """
    order_ok, set_ok, err, score = route_certainty(x, wg, sel_bias, logits, oi, k, exact_products)
    assert np.array_equal(gi[order_ok], oi[order_ok])
    same_set = np.all(np.sort(gi, axis=1) == np.sort(oi, axis=1), axis=1)
    assert same_set[set_ok].all()
    for t in np.nonzero(~order_ok)[0]:
        assert len(set(gi[t].tolist())) == k
        left = np.ones(score.shape[1], bool)
        for j in range(k):
            a = gi[t, j]
            assert np.all(score[t, left] <= score[t, a] + err[t, left] + err[t, a])
            left[a] = False
    if same_set.any():
        go = np.argsort(gi[same_set], axis=1)
        oo = np.argsort(oi[same_set], axis=1)
        np.testing.assert_allclose(np.take_along_axis(gw[same_set], go, 1), np.take_along_axis(ow[same_set], oo, 1),
                                   rtol=1e-5, atol=1e-7)
    return same_set, order_ok


def by_expert(a, idx):
    """Reorder each token's k entries of `a` by ascending expert id."""
    return np.take_along_axis(a, np.argsort(idx, axis=1), axis=1)
