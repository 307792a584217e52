"""Pins of the fp64 oracle against facts other than itself (CPU only).

Each test ties the oracle to something it cannot simply restate: hand-worked fixtures,
published table values, library routines, a second independent dense formulation, the
paper's sharding identity (Section 3.2) and exact-integer special cases.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special as sps
import scipy.stats as sst
from hypothesis import given, settings, strategies as st

import oracle
from oracle import brute
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def _rand_layer(rng, T, h, E, k, f, act="gelu", std=0.3):
    x = rng.standard_normal((T, h)).astype(np.float32)
    wg = (rng.standard_normal((E, h)) * std).astype(np.float32)
    w1 = (rng.standard_normal((E, h, f)) * std).astype(np.float32)
    w3 = (rng.standard_normal((E, h, f)) * std).astype(np.float32) if act == "swiglu" else None
    w2 = (rng.standard_normal((E, f, h)) * std).astype(np.float32)
    return x, wg, w1, w3, w2


def _oracle_layer(x, wg, w1, w3, w2, k, act, bias=None, renorm=0, col0=0, f=None):
    idx, w, _ = oracle.route(x, wg, k, bias, renorm)
    counts, offsets, row_src, pos_of = oracle.dispatch(idx, wg.shape[0])
    y_perm = oracle.expert_ffn(x[row_src], offsets, w1, w3, w2, act, col0, f)
    return oracle.combine(y_perm, pos_of, w), idx, w


# ---------------------------------------------------------------- hand-worked fixtures

def test_dispatch_matches_hand_worked_example():
    g = _golden("dispatch_worked_example.json")
    counts, offsets, row_src, pos_of = oracle.dispatch(np.array(g["idx"]), g["E"])
    assert counts.tolist() == g["counts"]
    assert offsets.tolist() == g["offsets"]
    assert row_src.tolist() == g["row_src"]
    assert pos_of.tolist() == g["pos_of"]


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_route_matches_hand_worked_example(k):
    g = _golden("route_worked_example.json")
    x = np.array(g["x"], np.float32)
    wg = np.array(g["wg"], np.float32)
    idx, w, logits = oracle.route(x, wg, k)
    assert logits.tolist() == g["logits"]
    assert idx.tolist() == g[f"top{k}"]


# ---------------------------------------------------------------- activations

@pytest.mark.parametrize("u", ["1.0", "2.0", "0.5", "-1.5", "3.0", "-1.0"])
def test_gelu_against_normal_cdf_table(u):
    phi = _golden("activation_points.json")["phi"][u]
    v = float(u)
    one = np.ones((1, 1, 1), np.float32)
    y = oracle.ffn_rows(np.array([[v]], np.float32), [0], one, None, one, "gelu")[0, 0]
    assert abs(y - v * phi) < 1e-9
    # and against scipy's independent normal CDF to full precision
    assert abs(y - v * sst.norm.cdf(v)) < 1e-15 * max(1.0, abs(v))


@pytest.mark.parametrize("z", ["1.0", "-2.0"])
def test_swiglu_against_logistic_table(z):
    sig = _golden("activation_points.json")["sigma"][z]
    v = float(z)
    one = np.ones((1, 1, 1), np.float32)
    three = np.full((1, 1, 1), 3.0, np.float32)
    # silu(v * 1) * (v * 3), then times W2 = 1
    y = oracle.ffn_rows(np.array([[v]], np.float32), [0], one, three, one, "swiglu")[0, 0]
    assert abs(y - v * sig * 3 * v) < 1e-9
    assert abs(y - v * sps.expit(v) * 3 * v) < 1e-15


def test_gelu_tanh_is_within_published_deviation_of_gelu():
    bound = _golden("activation_points.json")["gelu_tanh_max_abs_dev_from_gelu"]
    u = np.linspace(-8, 8, 801, dtype=np.float32)[:, None]
    one = np.ones((1, 1, 1), np.float32)
    e = np.zeros(u.shape[0], np.int32)
    g = oracle.ffn_rows(u, e, one, None, one, "gelu")[:, 0]
    t = oracle.ffn_rows(u, e, one, None, one, "gelu_tanh")[:, 0]
    assert np.max(np.abs(g - t)) < bound
    assert np.max(np.abs(g - t)) > 1e-5  # really the approximate form, not the erf one
    assert t[400] == 0.0 and g[400] == 0.0  # u = 0


def test_gelu_tanh_against_torch_float64():
    """The tanh form against an independent implementation of the same published formula
    (PyTorch's GELU with approximate="tanh", evaluated in float64 on the CPU): a slip in
    either coefficient (sqrt(2/pi), 0.044715) moves values far more than rounding."""
    torch = pytest.importorskip("torch")
    u = np.concatenate([np.linspace(-8, 8, 1601), [-0.75, 0.3, 1.7, 2.9]]).astype(np.float32)[:, None]
    one = np.ones((1, 1, 1), np.float32)
    e = np.zeros(u.shape[0], np.int32)
    t = oracle.ffn_rows(u, e, one, None, one, "gelu_tanh")[:, 0]
    ref = torch.nn.functional.gelu(torch.from_numpy(u[:, 0].astype(np.float64)), approximate="tanh").numpy()
    np.testing.assert_allclose(t, ref, rtol=1e-13, atol=1e-15)
    # sensitivity: 0.0447 instead of 0.044715 would differ by more than 1e-6 near |u| = 2
    c = math.sqrt(2.0 / math.pi)
    slip = 0.5 * u[:, 0] * (1.0 + np.tanh(c * (u[:, 0] + 0.0447 * u[:, 0] ** 3)))
    assert np.max(np.abs(slip - ref)) > 1e-6


# ---------------------------------------------------------------- P1: dense == sparse

@settings(max_examples=25, deadline=None)
@given(T=st.integers(0, 12), h=st.integers(1, 9), E=st.integers(1, 6), f=st.integers(1, 7),
       kk=st.integers(1, 6), act=st.sampled_from(["gelu", "gelu_tanh", "swiglu"]),
       renorm=st.integers(0, 1), use_bias=st.booleans(), seed=st.integers(0, 2**31 - 1))
def test_dense_bruteforce_equals_grouped_sparse(T, h, E, f, kk, act, renorm, use_bias, seed):
    k = min(kk, E)
    rng = np.random.default_rng(seed)
    x, wg, w1, w3, w2 = _rand_layer(rng, T, h, E, k, f, act)
    bias = (rng.standard_normal((T, E)) * 2).astype(np.float32) if use_bias else None
    y, idx, w = _oracle_layer(x, wg, w1, w3, w2, k, act, bias, renorm)
    yb, idxb, wb = brute.dense_layer(x, wg, w1, w3, w2, k, act, bias, renorm)
    assert np.array_equal(idx, idxb)
    np.testing.assert_allclose(w, wb, rtol=1e-13, atol=0)
    scale = max(np.max(np.abs(yb)), 1e-300) if yb.size else 1.0
    assert (np.max(np.abs(y - yb)) if y.size else 0.0) <= 1e-12 * scale


def test_layer_tokens_equals_grouped_path():
    rng = np.random.default_rng(7)
    x, wg, w1, w3, w2 = _rand_layer(rng, 40, 16, 5, 2, 12, "swiglu")
    y, idx, w = _oracle_layer(x, wg, w1, w3, w2, 2, "swiglu", renorm=1)
    toks = np.array([0, 3, 39, 17])
    yt = oracle.layer_tokens(toks, x, idx, w, w1, w3, w2, "swiglu")
    np.testing.assert_allclose(yt, y[toks], rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------------- P2: shard sum

@pytest.mark.parametrize("act", ["gelu", "gelu_tanh", "swiglu"])
@pytest.mark.parametrize("widths", [[10, 27], [8, 8], [3, 5, 7, 1], [4] * 8])
def test_shard_partials_sum_to_unsharded_output(act, widths):
    rng = np.random.default_rng(len(widths) * 100 + sum(widths))
    F = sum(widths)
    x, wg, w1, w3, w2 = _rand_layer(rng, 30, 12, 4, 2, F, act)
    full, _, _ = _oracle_layer(x, wg, w1, w3, w2, 2, act, renorm=1)
    parts, col0 = [], 0
    for f in widths:
        y, _, _ = _oracle_layer(x, wg, w1, w3, w2, 2, act, renorm=1, col0=col0, f=f)
        parts.append(y)
        col0 += f
    np.testing.assert_allclose(sum(parts), full, rtol=0, atol=1e-12 * np.abs(full).max())


@pytest.mark.parametrize("g", [0, 1])
def test_shard_reads_only_its_own_slice(g):
    """Section 3.2's two-GPU example: 4 inner columns, GPU 0 owns columns 0-1 of W_i and
    rows 0-1 of W_o, GPU 1 owns the rest.  Poisoning the other GPU's slice with NaN must
    leave this shard's partial finite and unchanged."""
    rng = np.random.default_rng(3)
    x, wg, w1, w3, w2 = _rand_layer(rng, 6, 5, 3, 1, 4, "gelu")
    ref = oracle.expert_ffn(x, np.array([0, 2, 4, 6]), w1, None, w2, "gelu", col0=2 * g, f=2)
    other = slice(2, 4) if g == 0 else slice(0, 2)
    w1p, w2p = w1.copy(), w2.copy()
    w1p[:, :, other] = np.nan
    w2p[:, other, :] = np.nan
    got = oracle.expert_ffn(x, np.array([0, 2, 4, 6]), w1p, None, w2p, "gelu", col0=2 * g, f=2)
    assert np.isfinite(got).all()
    assert np.array_equal(got, ref)


def test_zero_padding_of_inner_width_changes_nothing():
    rng = np.random.default_rng(11)
    x, wg, w1, w3, w2 = _rand_layer(rng, 9, 6, 3, 1, 10, "gelu")
    w1p = np.concatenate([w1, np.zeros((3, 6, 13), np.float32)], axis=2)
    w2p = np.concatenate([w2, np.zeros((3, 13, 6), np.float32)], axis=1)
    off = np.array([0, 4, 4, 9])
    a = oracle.expert_ffn(x, off, w1, None, w2, "gelu")
    b = oracle.expert_ffn(x, off, w1p, None, w2p, "gelu")
    assert np.array_equal(a, b)


# ---------------------------------------------------------------- P3/P4: counts, permutation

@settings(max_examples=40, deadline=None)
@given(T=st.integers(0, 200), E=st.integers(1, 40), kk=st.integers(1, 8), seed=st.integers(0, 2**31 - 1))
def test_counts_and_permutation_invariants(T, E, kk, seed):
    k = min(kk, E)
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) if T else np.zeros((0, k), np.int32)
    counts, offsets, row_src, pos_of = oracle.dispatch(idx, E)
    assert np.array_equal(counts, np.bincount(idx.ravel(), minlength=E))
    assert offsets[0] == 0 and offsets[-1] == T * k == counts.sum()
    assert np.array_equal(np.diff(offsets), counts)
    # pos_of is a bijection onto [0, A); row_src inverts it; stable order per expert
    assert np.array_equal(np.sort(pos_of.ravel()), np.arange(T * k))
    assert np.array_equal(row_src[pos_of.ravel()], np.repeat(np.arange(T), k))
    assert np.array_equal(row_src, np.argsort(idx.ravel(), kind="stable") // k)
    x = rng.standard_normal((T, 3)).astype(np.float32)
    x_perm = x[row_src]
    for j in range(k):
        assert np.array_equal(x_perm[pos_of[:, j]], x)  # unpermute(permute(x)) == x


def test_route_picks_are_distinct_and_weights_renormalise():
    rng = np.random.default_rng(5)
    x, wg, *_ = _rand_layer(rng, 300, 20, 16, 4, 1)
    idx, w, _ = oracle.route(x, wg, 4, renorm=1)
    assert all(len(set(r)) == 4 for r in idx.tolist())
    np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-15)


# ---------------------------------------------------------------- P5: exact routing

def test_exact_integer_routing_with_ties():
    rng = np.random.default_rng(2)
    T, h, E = 64, 12, 10
    x = rng.integers(-8, 9, (T, h)).astype(np.float32)
    x[5] = 0  # all-zero row: every logit equal -> ids 0..k-1
    wg = rng.integers(-8, 9, (E, h)).astype(np.float32)
    wg[7] = wg[2]  # duplicated gate rows: equal logits, the lower id must win
    wg[9] = wg[4]
    for k in (1, 3, E):
        idx, _, logits = oracle.route(x, wg, k)
        exact = [[sum(int(a) * int(b) for a, b in zip(x[t], wg[e])) for e in range(E)] for t in range(T)]
        assert np.array_equal(logits, np.array(exact, np.float64))
        for t in range(T):
            ref = sorted(range(E), key=lambda e: (-exact[t][e], e))[:k]
            assert idx[t].tolist() == ref
        assert idx[5].tolist() == list(range(k))
        pos = {e: i for i, e in enumerate(idx[0].tolist())} if k == E else None
        if pos is not None:
            assert pos[2] < pos[7] and pos[4] < pos[9]


def test_weights_equal_softmax_of_unbiased_logits():
    rng = np.random.default_rng(9)
    x, wg, *_ = _rand_layer(rng, 50, 24, 12, 12, 1)
    bias = (rng.standard_normal((50, 12)) * 5).astype(np.float32)
    idx, w, logits = oracle.route(x, wg, 12, sel_bias=bias)
    np.testing.assert_allclose(logits, x.astype(np.float64) @ wg.astype(np.float64).T, rtol=1e-12, atol=1e-12)
    p = sps.softmax(logits, axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(p, idx.astype(np.int64), axis=1), rtol=1e-12, atol=0)
    # the bias changed the order: picks follow logits + bias, not the logits alone
    assert not np.array_equal(idx[:, 0], np.argmax(logits, axis=1))
    assert np.array_equal(idx[:, 0], np.argmax(logits + bias, axis=1))


# ---------------------------------------------------------------- P6: closed forms

def test_single_expert_is_a_dense_mlp():
    rng = np.random.default_rng(4)
    x, wg, w1, w3, w2 = _rand_layer(rng, 20, 8, 1, 1, 6, "gelu")
    y, idx, w = _oracle_layer(x, wg, w1, w3, w2, 1, "gelu")
    assert np.all(idx == 0) and np.all(w == 1.0)
    u = x.astype(np.float64) @ w1[0].astype(np.float64)
    ref = (u * sst.norm.cdf(u)) @ w2[0].astype(np.float64)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14)


def test_two_expert_top1_weight_is_sigmoid_of_logit_gap():
    rng = np.random.default_rng(6)
    x, wg, *_ = _rand_layer(rng, 100, 10, 2, 1, 1)
    idx, w, logits = oracle.route(x, wg, 1)
    gap = np.abs(logits[:, 0] - logits[:, 1])
    np.testing.assert_allclose(w[:, 0], sps.expit(gap), rtol=1e-14)


def test_combine_is_linear_in_the_gate_weights():
    rng = np.random.default_rng(8)
    y_perm = rng.standard_normal((12, 5))
    pos_of = rng.permutation(12).reshape(6, 2).astype(np.int32)
    w = rng.random((6, 2))
    a = oracle.combine(y_perm, pos_of, w)
    b = oracle.combine(y_perm, pos_of, 2 * w)
    assert np.array_equal(b, 2 * a)
    # and against a numpy gather-and-weight of the same definition
    ref = w[:, :1] * y_perm[pos_of[:, 0]] + w[:, 1:] * y_perm[pos_of[:, 1]]
    np.testing.assert_allclose(a, ref, rtol=1e-15, atol=0)


# ---------------------------------------------------------------- the generator

def test_bf16_rounding_known_bit_patterns():
    vals = np.array([1.0, -2.0, 3.140625], np.float32)
    assert synth.f32_to_bf16_bits(vals).tolist() == [0x3F80, 0xC000, 0x4049]
    ties = np.array([0x3F808000, 0x3F818000, 0x3F808001], np.uint32).view(np.float32)
    assert synth.f32_to_bf16_bits(ties).tolist() == [0x3F80, 0x3F82, 0x3F81]


def test_paper_router_frequencies_follow_its_formula():
    """Section 4.1's router: p_i proportional to 1/|E| + alpha_r for the k_r skewed experts."""
    cfg = synth.LayerConfig("t", T=200000, h=8, E=16, k=1, F=8, routing=("paper", 3, 0.6))
    tg = synth.routing_targets(cfg, seed=1)
    cnt = np.bincount(tg.ravel(), minlength=16)
    hot = np.argsort(-cnt)[:3]
    p = np.full(16, 1 / 16)
    p[hot] += 0.6
    p /= p.sum()
    chi2 = sst.chisquare(cnt, p * cfg.T)
    assert chi2.pvalue > 1e-4


def test_zipf_and_pair_routing_shapes():
    cfg = synth.LayerConfig("t", T=100000, h=8, E=64, k=1, F=8, routing=("zipf", 1.0))
    cnt = np.sort(np.bincount(synth.routing_targets(cfg, 0).ravel(), minlength=64))[::-1]
    ranks = np.arange(1, 65)
    p = (1 / ranks) / (1 / ranks).sum()
    assert abs(cnt[0] / cfg.T - p[0]) < 0.01 and abs(cnt[-1] / cfg.T - p[-1]) < 0.002
    cfg = synth.LayerConfig("t", T=20000, h=8, E=64, k=2, F=8, routing=("pair", 0.95))
    tg = synth.routing_targets(cfg, 0)
    assert np.all(tg[:, 0] < tg[:, 1])
    hot = tuple(np.unique(tg, axis=0, return_counts=True)[0][np.argmax(np.unique(tg, axis=0, return_counts=True)[1])])
    share = np.mean((tg[:, 0] == hot[0]) & (tg[:, 1] == hot[1]))
    assert 0.94 < share < 0.96


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_bias_injection_selects_exactly_the_sampled_targets(name):
    layer = synth.make(name, seed=0, weights=False, T=512)
    idx, _, _ = oracle.route(layer.x, layer.wg, layer.cfg.k, layer.sel_bias, layer.cfg.renorm)
    assert np.array_equal(np.sort(idx, axis=1), layer.targets)


def test_shard_weights_concatenate_to_the_full_layer():
    cfg = synth.CONFIGS["c3"].with_(T=4, E=2, h=16, F=64)
    w1, _, w2 = synth.full_width_weights(cfg)
    for g in range(cfg.G):
        part = synth.make(cfg.with_(shard=g))
        assert np.array_equal(part.w1, w1[:, :, g * cfg.f:(g + 1) * cfg.f])
        assert np.array_equal(part.w2, w2[:, g * cfg.f:(g + 1) * cfg.f, :])
