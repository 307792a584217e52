"""GPU parity of every step of the layer against the fp64 oracle (needs an MI355X).

Stage tests feed each kernel the oracle's inputs for that stage, so a failure points at
one kernel; end-to-end tests run the whole layer on the five workloads.  Integers are
compared bit-exactly; floats with the normwise error of each output row against the
oracle: <= 2e-2 for bf16 paths, <= 1e-5 for the fp32 path.
"""
import numpy as np
import pytest

import oracle
import synth
from _util import by_expert, compare_routing, normwise, rowwise, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2503_08467_amd as moe  # noqa: E402

TOL = {"bf16": 2e-2, "f32": 1e-5}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    moe.load()
    yield
    torch.cuda.synchronize()


def tdt(cfg_dtype):
    return torch.bfloat16 if cfg_dtype == "bf16" else torch.float32


def np_of(t):
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


# ------------------------------------------------------------------------------- route

def _check_route(x, wg, bias, k, renorm, dtype, exact_products):
    dt = tdt(dtype)
    idx, w = moe.route(to_dev(x, dt), to_dev(wg, dt), k, to_dev(bias, torch.float32), renorm)
    torch.cuda.synchronize()
    gi, gw = idx.cpu().numpy(), w.cpu().numpy()
    oi, ow, logits = oracle.route(x, wg, k, bias, renorm)
    same_set, order_ok = compare_routing(gi, gw, oi, ow, x, wg, bias, logits, k, exact_products)
    return gi, int((~order_ok).sum())


@pytest.mark.parametrize("name,T", [("c1", 512), ("c2", 8192), ("c3", 16384), ("c4", 4096), ("c5", 32768),
                                    ("c5dec", 64), ("paper128", 30000)])
def test_route_parity_on_workloads(name, T):
    L = synth.make(name, seed=0, weights=False, T=T)
    gi, unsure = _check_route(L.x, L.wg, L.sel_bias, L.cfg.k, L.cfg.renorm, L.cfg.dtype, L.cfg.dtype == "bf16")
    print(f"{name}: {unsure} tokens within the fp32 rounding margin")
    if L.targets is not None:  # the injected routing is exactly what the kernel picked
        assert np.array_equal(np.sort(gi, axis=1), L.targets)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T,h,E,k", [(1, 8, 1, 1), (17, 72, 3, 2), (100, 256, 16, 16), (65, 136, 17, 4),
                                     (130, 64, 64, 2), (33, 512, 200, 8), (64, 96, 256, 3), (257, 1024, 128, 1),
                                     (16449, 64, 136, 2),  # more 64-token workgroups than CUs
                                     # the persistent kernel (h % 256 == 0, E % 8 == 0, E <= 128, k <= 8):
                                     # several tiles per workgroup, partial last tiles, one to sixteen
                                     # chunks per row, one to four 32-expert blocks
                                     (1000, 768, 64, 2), (70, 4096, 8, 2), (5000, 1024, 64, 8), (33, 512, 16, 3),
                                     (9000, 2048, 40, 4), (20000, 256, 24, 2), (300, 1536, 96, 5),
                                     (70000, 256, 32, 2)])  # more than 8 tiles per workgroup
@pytest.mark.parametrize("bias_kind", ["none", "row", "shared"])
def test_route_shapes_and_bias(dtype, T, h, E, k, bias_kind):
    rng = np.random.default_rng(T * 1000 + E)
    x = rng.standard_normal((T, h)).astype(np.float32)
    wg = (rng.standard_normal((E, h)) * 0.05).astype(np.float32)
    if dtype == "bf16":
        x, wg = synth.round_to_bf16(x), synth.round_to_bf16(wg)
    bias = {"none": None, "row": rng.standard_normal((T, E)).astype(np.float32),
            "shared": rng.standard_normal(E).astype(np.float32)}[bias_kind]
    _check_route(x, wg, bias, k, int(k > 1), dtype, dtype == "bf16")


@pytest.mark.parametrize("T,h,E,k", [(1, 128, 40, 1), (17, 256, 64, 2), (64, 1024, 64, 2), (64, 128, 128, 8),
                                     (33, 64, 256, 5), (50, 192, 100, 3),
                                     (65, 128, 64, 2), (64, 128, 64, 9), (40, 128, 32, 2)])  # separate launches
@pytest.mark.parametrize("bias_kind", ["none", "row", "shared"])
def test_route_dispatch_matches_two_calls(T, h, E, k, bias_kind):
    """moe_route_dispatch = moe_route + moe_dispatch (indices only), every output bit for bit:
    one launch when a single workgroup routes the batch (T <= 64, k <= 8, 32 < E), the two
    launches otherwise."""
    rng = np.random.default_rng(T * 1000 + E + k)
    x = synth.round_to_bf16(rng.standard_normal((T, h)).astype(np.float32))
    wg = synth.round_to_bf16((rng.standard_normal((E, h)) * 0.05).astype(np.float32))
    bias = {"none": None, "row": rng.standard_normal((T, E)).astype(np.float32),
            "shared": rng.standard_normal(E).astype(np.float32)}[bias_kind]
    xd, wgd, bd = to_dev(x, torch.bfloat16), to_dev(wg, torch.bfloat16), to_dev(bias, torch.float32)
    renorm = k > 1
    idx1, w1 = moe.route(xd, wgd, k, bd, renorm)
    d1 = moe.dispatch(idx1, xd, E, x_perm=False)
    d2, ws = moe.alloc_dispatch(T, k, E, h, torch.bfloat16, xd.device, x_perm=False)
    for key in ("counts", "offsets", "row_src", "pos_of"):
        getattr(d2, key).fill_(-7)
    idx2, w2, d2 = moe.route_dispatch(xd, wgd, k, bd, renorm, disp=d2, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(idx1, idx2)
    assert torch.equal(w1.view(torch.int32), w2.view(torch.int32))
    n = int(d1.offsets[-1].item())
    for key in ("counts", "offsets", "pos_of"):
        assert torch.equal(getattr(d1, key), getattr(d2, key)), key
    assert torch.equal(d1.row_src[:n], d2.row_src[:n])
    assert np.array_equal(d2.counts.cpu().numpy(), np.bincount(idx2.cpu().numpy().ravel(), minlength=E))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_route_exact_ties_go_to_lower_expert(dtype):
    rng = np.random.default_rng(5)
    T, h, E = 200, 64, 40
    x = rng.integers(-4, 5, (T, h)).astype(np.float32)  # exact logits in fp32 and fp64
    x[3] = 0
    wg = rng.integers(-3, 4, (E, h)).astype(np.float32)
    wg[30] = wg[7]
    wg[39] = wg[0]
    for k in (1, 5, E):
        idx, _ = moe.route(to_dev(x, tdt(dtype)), to_dev(wg, tdt(dtype)), k)
        oi, _, _ = oracle.route(x, wg, k)
        assert np.array_equal(idx.cpu().numpy(), oi)
        assert idx[3].tolist() == list(range(k))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("h,E,k", [(1024, 64, 2), (768, 128, 1), (4096, 8, 2), (256, 256, 4), (136, 40, 3)])
def test_route_does_not_depend_on_batch_position(dtype, h, E, k):
    """A token's picks and weights are the same bits whatever its position in the batch and
    the batch size: the gate product sums every token in one fixed order."""
    rng = np.random.default_rng(h + E)
    T = 700
    x = rng.standard_normal((T, h)).astype(np.float32)
    wg = (rng.standard_normal((E, h)) * 0.02).astype(np.float32)
    if dtype == "bf16":
        x, wg = synth.round_to_bf16(x), synth.round_to_bf16(wg)
    xd, wd = to_dev(x, tdt(dtype)), to_dev(wg, tdt(dtype))
    i_all, w_all = moe.route(xd, wd, k, renorm=k > 1)
    for off, n in ((37, 300), (1, 64), (129, 571), (650, 50)):
        i_sub, w_sub = moe.route(xd[off:off + n].contiguous(), wd, k, renorm=k > 1)
        assert torch.equal(i_sub, i_all[off:off + n]), (off, n)
        assert torch.equal(w_sub, w_all[off:off + n]), (off, n)


# ------------------------------------------------------------------------------- dispatch

def _check_dispatch(idx, E, h=64, dtype=torch.bfloat16):
    T, k = idx.shape
    rng = np.random.default_rng(T + E)
    xd = to_dev(rng.standard_normal((T, h)).astype(np.float32), dtype)
    d = moe.dispatch(to_dev(idx, torch.int32), xd, E)
    torch.cuda.synchronize()
    gc, go, gr, gp = (d.counts.cpu().numpy(), d.offsets.cpu().numpy(), d.row_src.cpu().numpy(),
                      d.pos_of.cpu().numpy())
    flat = idx.ravel()
    keep = (flat >= 0) & (flat < E)
    if keep.all():
        counts, offsets, row_src, pos_of = oracle.dispatch(idx, E)
        assert np.array_equal(gc, counts)
        assert np.array_equal(go, offsets)
        assert np.array_equal(gr, row_src)
        assert np.array_equal(gp, pos_of)
    else:
        # invalid ids are dropped: counts and order are those of the valid ids alone
        order = np.argsort(np.where(keep, flat, E), kind="stable")[:keep.sum()]
        assert np.array_equal(gc, np.bincount(flat[keep], minlength=E))
        assert go[-1] == keep.sum()
        assert np.array_equal(gr[:keep.sum()], order // k)
        exp_pos = np.full(T * k, -1)
        exp_pos[order] = np.arange(keep.sum())
        assert np.array_equal(gp.ravel(), exp_pos)
    A = int(keep.sum())
    src = torch.from_numpy(gr[:A].astype(np.int64)).to(xd.device)
    assert torch.equal(d.x_perm[:A], xd[src])


# up to 16384 assignments one fused kernel dispatches, above it three kernels: both sides of
# that boundary are covered (8192 x 2, 16384 x 1 fused; 16385 x 1 and larger not), as are
# chunk edges and large skewed batches
@pytest.mark.parametrize("T,k,E", [(0, 1, 8), (1, 1, 1), (5, 2, 5), (1000, 1, 64), (1023, 2, 7), (1024, 2, 256),
                                   (3000, 3, 100), (8192, 2, 3), (16384, 1, 128), (16385, 1, 64), (32768, 2, 64),
                                   (4096, 8, 256), (4097, 1, 2), (131072, 2, 64), (131073, 2, 64),
                                   (70000, 4, 256)])
def test_dispatch_bit_exact(T, k, E):
    rng = np.random.default_rng(T + 7 * E)
    p = rng.dirichlet(np.full(E, 0.3))  # skewed popularity, many empty experts
    # k distinct ids per token drawn without replacement with probabilities p (Gumbel top-k)
    keys = np.log(np.maximum(p, 1e-300))[None, :] - np.log(-np.log(rng.random((T, E))))
    idx = np.argsort(-keys, axis=1, kind="stable")[:, :k].astype(np.int32)
    _check_dispatch(idx, E)


def test_dispatch_fused_skew_and_invalid_ids():
    """95 % of the assignments on one expert and some ids invalid, over many dispatch
    chunks: counts and ranks stay exact."""
    rng = np.random.default_rng(11)
    T, k, E = 30000, 2, 64
    idx = np.where(rng.random((T, k)) < 0.95, 17, rng.integers(0, E, (T, k))).astype(np.int32)
    idx[:, 1] = np.where(idx[:, 1] == idx[:, 0], (idx[:, 0] + 1) % E, idx[:, 1])
    idx[::97, 0] = -5
    idx[::89, 1] = E + 2
    _check_dispatch(idx, E)


def test_dispatch_golden_example():
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "dispatch_worked_example.json")))
    d = moe.dispatch(to_dev(np.array(g["idx"], np.int32), torch.int32),
                     torch.zeros((g["T"], 16), dtype=torch.bfloat16, device="cuda"), g["E"])
    assert d.counts.tolist() == g["counts"] and d.offsets.tolist() == g["offsets"]
    assert d.row_src.tolist() == g["row_src"] and d.pos_of.tolist() == g["pos_of"]


def test_dispatch_drops_invalid_ids():
    rng = np.random.default_rng(1)
    idx = rng.integers(0, 9, (700, 2)).astype(np.int32)
    idx[::7, 0] = -1
    idx[::11, 1] = 9 + 3
    _check_dispatch(idx, 9, h=32, dtype=torch.float32)


# ------------------------------------------------------------------------------- expert FFN

def _ffn_case(rng, counts, h, f, act, dtype, F=None, col0=0):
    E = len(counts)
    F = F or f
    A = int(sum(counts))
    std = 0.05
    x = rng.standard_normal((A, h)).astype(np.float32)
    w1 = (rng.standard_normal((E, h, F)) * std).astype(np.float32)
    w3 = (rng.standard_normal((E, h, F)) * std).astype(np.float32) if act == "swiglu" else None
    w2 = (rng.standard_normal((E, F, h)) * std).astype(np.float32)
    if dtype == "bf16":
        x, w1, w2 = synth.round_to_bf16(x), synth.round_to_bf16(w1), synth.round_to_bf16(w2)
        w3 = None if w3 is None else synth.round_to_bf16(w3)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return x, w1, w3, w2, offsets


def _run_ffn(x, w1, w3, w2, offsets, act, dtype, out_dtype=None, col0=0, f=None):
    dt = tdt(dtype)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), to_dev(w3, dt), col0=col0, f=f, act=act)
    y = moe.expert_ffn_shard(to_dev(x, dt), to_dev(offsets, torch.int32), packed, out_dtype=out_dtype)
    torch.cuda.synchronize()
    return np_of(y)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ["gelu", "gelu_tanh", "swiglu"])
@pytest.mark.parametrize("counts,h,f", [
    ([300, 0, 5, 129, 128, 1], 256, 200),     # ragged rows and a ragged inner width
    ([1], 64, 37),
    ([0, 0, 77], 72, 128),                     # h not a multiple of the 64-wide K step
    ([513, 40, 0, 255], 768, 512),
    ([700, 333], 256, 200),                    # >= 512 rows per expert: 256-row tiles, ragged
    ([1100, 0, 1500, 3], 512, 384),
    ([60, 0, 50, 9], 128, 1000),               # <= 128 rows: 128-column up tiles, K of the down in 4 parts
    ([100, 7, 0, 120], 192, 2048),             # <= 256 rows: down K in 8 parts
    ([200, 0, 61, 3], 256, 2048),              # <= 512 rows: down K in 4 parts
])
def test_ffn_parity(dtype, act, counts, h, f):
    rng = np.random.default_rng(sum(counts) + h + f)
    x, w1, w3, w2, offsets = _ffn_case(rng, counts, h, f, act, dtype)
    got = _run_ffn(x, w1, w3, w2, offsets, act, dtype)
    ref = oracle.expert_ffn(x, offsets, w1, w3, w2, act)
    assert rowwise(got, ref) <= TOL[dtype], (rowwise(got, ref), normwise(got, ref))


def _random_ffn_shapes(n, seed=2024):
    rng = np.random.default_rng(seed)
    shapes = []
    for i in range(n):
        E = int(rng.integers(1, 41))
        A = int(rng.integers(0, 701))
        counts = rng.multinomial(A, rng.dirichlet(np.full(E, 0.5))).tolist()
        h = int(rng.choice([8, 64, 72, 136, 256, 520]))
        f = int(rng.integers(1, 601))
        shapes.append((i, counts, h, f, ["gelu", "gelu_tanh", "swiglu"][i % 3], ["bf16", "f32"][(i // 3) % 2]))
    return shapes


@pytest.mark.parametrize("i,counts,h,f,act,dtype", _random_ffn_shapes(12))
def test_ffn_parity_on_random_shapes(i, counts, h, f, act, dtype):
    """Seeded random shapes: expert count, ragged segments (some empty), hidden sizes off the
    tile multiples, any inner width (split and unsplit second products)."""
    rng = np.random.default_rng(100 + i)
    x, w1, w3, w2, offsets = _ffn_case(rng, counts, h, f, act, dtype)
    got = _run_ffn(x, w1, w3, w2, offsets, act, dtype)
    ref = oracle.expert_ffn(x, offsets, w1, w3, w2, act)
    if len(ref):
        assert rowwise(got, ref) <= TOL[dtype], (rowwise(got, ref), normwise(got, ref))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("A,f", [(3000, 128), (300, 1024)])
def test_ffn_parity_at_the_expert_limit(dtype, act, A, f):
    """256 experts (the most the library takes), most of them with a handful of rows or none:
    the row-tile table at its full size, in the grouped launch and, below 512 rows, with the
    second product's K split."""
    rng = np.random.default_rng(A + f)
    counts = rng.multinomial(A, rng.dirichlet(np.full(256, 0.2))).tolist()
    assert len(counts) == 256 and 0 in counts
    x, w1, w3, w2, offsets = _ffn_case(rng, counts, 64, f, act, dtype)
    got = _run_ffn(x, w1, w3, w2, offsets, act, dtype)
    ref = oracle.expert_ffn(x, offsets, w1, w3, w2, act)
    assert rowwise(got, ref) <= TOL[dtype], (rowwise(got, ref), normwise(got, ref))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("counts,h,f", [
    ([300, 0, 5, 129, 128, 1], 256, 200),
    ([0, 0, 77], 72, 128),
    ([700, 333, 0], 256, 200),
    ([60, 0, 50, 9], 128, 1000),  # split down-projection K: both paths split alike
])
def test_per_expert_launches_match_grouped(dtype, act, counts, h, f):
    """The per-expert-launch ablation computes the same tiles as the grouped launch: equal
    bit for bit, and within tolerance of the oracle."""
    rng = np.random.default_rng(7 + sum(counts) + h)
    x, w1, w3, w2, offsets = _ffn_case(rng, counts, h, f, act, dtype)
    dt = tdt(dtype)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), to_dev(w3, dt), f=f, act=act)
    xd, od = to_dev(x, dt), to_dev(offsets, torch.int32)
    y_grouped = moe.expert_ffn_shard(xd, od, packed)
    y_each = moe.expert_ffn_shard_per_expert(xd, od, packed)
    torch.cuda.synchronize()
    ib = torch.int16 if dt == torch.bfloat16 else torch.int32
    assert torch.equal(y_grouped.view(ib), y_each.view(ib))
    ref = oracle.expert_ffn(x, offsets, w1, w3, w2, act)
    assert rowwise(np_of(y_each), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("T,k,E,h,f", [(700, 2, 6, 256, 200), (90, 1, 3, 72, 128), (1500, 1, 4, 768, 384),
                                        (50, 2, 5, 128, 1024)])
def test_gathered_rows_match_x_perm(dtype, act, T, k, E, h, f):
    """The expert step reading x[row_src[p]] itself equals the one reading x_perm, bit for
    bit; some ids are invalid (dropped), so row_src has unwritten entries past offsets[E]."""
    rng = np.random.default_rng(T + h)
    x = rng.standard_normal((T, h)).astype(np.float32)
    w1 = (rng.standard_normal((E, h, f)) * 0.05).astype(np.float32)
    w3 = (rng.standard_normal((E, h, f)) * 0.05).astype(np.float32) if act == "swiglu" else None
    w2 = (rng.standard_normal((E, f, h)) * 0.05).astype(np.float32)
    if dtype == "bf16":
        x, w1, w2 = synth.round_to_bf16(x), synth.round_to_bf16(w1), synth.round_to_bf16(w2)
        w3 = None if w3 is None else synth.round_to_bf16(w3)
    idx = np.stack([rng.permutation(E + 1)[:k] for _ in range(T)]).astype(np.int32)  # id E is invalid
    dt = tdt(dtype)
    xd = to_dev(x, dt)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), to_dev(w3, dt), f=f, act=act)
    d_full = moe.dispatch(to_dev(idx, torch.int32), xd, E)
    d_idx = moe.dispatch(to_dev(idx, torch.int32), xd, E, x_perm=False)
    d_idx.row_src.fill_(-123456)  # poison, then dispatch again: entries past offsets[E] stay poisoned
    d_idx = moe.dispatch(to_dev(idx, torch.int32), xd, E, out=d_idx,
                         ws=torch.empty(moe.dispatch_workspace_size(T, k, E), dtype=torch.uint8, device="cuda"))
    y_perm = moe.expert_ffn_shard(d_full.x_perm, d_full.offsets, packed)
    y_gath = moe.expert_ffn_shard_gather(xd, d_idx.row_src, d_idx.offsets, packed)
    torch.cuda.synchronize()
    n = int(d_full.offsets[-1].item())
    assert n < T * k
    ib = torch.int16 if dt == torch.bfloat16 else torch.int32
    assert torch.equal(y_perm[:n].view(ib), y_gath[:n].view(ib))
    offsets = d_full.offsets.cpu().numpy()
    ref = oracle.expert_ffn(x[d_full.row_src.cpu().numpy()[:n]], offsets, w1, w3, w2, act)
    assert rowwise(np_of(y_gath[:n]), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype,out_dtype", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("T,k,E,h,f,split", [
    (64, 2, 8, 256, 1024, {"bf16": True, "f32": True}),     # decode-sized: split second product
    (64, 2, 8, 256, 512, {"bf16": True, "f32": False}),     # fp32 K too short to split (16 steps)
    (300, 2, 6, 128, 1024, {"bf16": False, "f32": True}),   # 600 rows: split only in fp32 (<= 1024)
    (700, 3, 5, 64, 256, {"bf16": False, "f32": False}),    # 2100 rows: never split
    (1, 4, 9, 64, 1024, {"bf16": True, "f32": True}),       # one token
])
def test_gather_combine_matches_two_calls(dtype, out_dtype, T, k, E, h, f, split):
    """moe_expert_ffn_shard_gather_combine = moe_expert_ffn_shard_gather + moe_combine, bit
    for bit (one launch for the split sum and the combine when K is split, y_perm then left
    unwritten), and within tolerance of the oracle; dropped picks are skipped."""
    rng = np.random.default_rng(T * 10 + k + h)
    x = rng.standard_normal((T, h)).astype(np.float32)
    w1 = (rng.standard_normal((E, h, f)) * 0.05).astype(np.float32)
    w2 = (rng.standard_normal((E, f, h)) * 0.05).astype(np.float32)
    if dtype == "bf16":
        x, w1, w2 = synth.round_to_bf16(x), synth.round_to_bf16(w1), synth.round_to_bf16(w2)
    idx = np.stack([rng.permutation(E + 1)[:k] for _ in range(T)]).astype(np.int32)  # id E: dropped
    wt = rng.uniform(0.1, 1.0, size=(T, k)).astype(np.float32)
    dt, odt = tdt(dtype), tdt(out_dtype)
    xd = to_dev(x, dt)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), f=f, act="gelu")
    d = moe.dispatch(to_dev(idx, torch.int32), xd, E, x_perm=False)
    wd = to_dev(wt, torch.float32)
    y_perm = moe.expert_ffn_shard_gather(xd, d.row_src, d.offsets, packed, A_max=T * k)
    y_two = moe.combine(y_perm, d.pos_of, wd, out_dtype=odt)
    scratch = torch.full((T * k, h), 5.0, dtype=dt, device="cuda")
    y_one, written = moe.expert_ffn_shard_gather_combine(xd, d.row_src, d.offsets, d.pos_of, wd, packed,
                                                         y_perm=scratch, out_dtype=odt)
    torch.cuda.synchronize()
    ib = torch.int16 if odt == torch.bfloat16 else torch.int32
    assert torch.equal(y_one.view(ib), y_two.view(ib))
    assert (written is None) == split[dtype]
    if split[dtype]:
        assert bool((scratch == 5.0).all())
    offsets = d.offsets.cpu().numpy()
    row_src = d.row_src.cpu().numpy()[:offsets[-1]]
    ref_perm = oracle.expert_ffn(x[row_src], offsets, w1, None, w2, "gelu")
    pos = d.pos_of.cpu().numpy()
    ref = np.zeros((T, h))
    for j in range(k):  # dropped picks (pos -1) contribute nothing
        keep = pos[:, j] >= 0
        ref[keep] += wt[keep, j:j + 1].astype(np.float64) * ref_perm[pos[keep, j]]
    assert rowwise(np_of(y_one), ref) <= TOL["bf16" if "bf16" in (dtype, out_dtype) else "f32"]


@pytest.mark.parametrize("dtype,out_dtype", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("T,E,h,f", [(700, 6, 256, 200), (90, 3, 72, 128), (1300, 5, 768, 384),
                                     (100, 3, 128, 1024)])  # split down K: weighted sum in the reduce
def test_top1_step_writes_weighted_rows(dtype, out_dtype, act, T, E, h, f):
    """moe_expert_ffn_shard_top1 = the expert step plus the top-1 combine: y[t] = w[t] *
    FFN_e(x[t]).  Tokens whose only pick is invalid are dropped and left unwritten."""
    rng = np.random.default_rng(T + E + h)
    x = rng.standard_normal((T, h)).astype(np.float32)
    w1 = (rng.standard_normal((E, h, f)) * 0.05).astype(np.float32)
    w3 = (rng.standard_normal((E, h, f)) * 0.05).astype(np.float32) if act == "swiglu" else None
    w2 = (rng.standard_normal((E, f, h)) * 0.05).astype(np.float32)
    if dtype == "bf16":
        x, w1, w2 = synth.round_to_bf16(x), synth.round_to_bf16(w1), synth.round_to_bf16(w2)
        w3 = None if w3 is None else synth.round_to_bf16(w3)
    idx = rng.integers(0, E + 1, size=(T, 1)).astype(np.int32)  # id E is invalid: dropped
    wt = rng.uniform(0.1, 1.0, size=(T, 1)).astype(np.float32)
    dt, odt = tdt(dtype), tdt(out_dtype)
    xd = to_dev(x, dt)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), to_dev(w3, dt), f=f, act=act)
    d = moe.dispatch(to_dev(idx, torch.int32), xd, E, x_perm=False)
    y = torch.full((T, h), 7.0, dtype=odt, device="cuda")
    moe.expert_ffn_shard_top1(xd, d.row_src, to_dev(wt, torch.float32).view(-1), d.offsets, packed, out=y)
    torch.cuda.synchronize()
    y = np_of(y)
    valid = idx[:, 0] < E
    assert (~valid).any() and valid.any()
    offsets = d.offsets.cpu().numpy()
    row_src = d.row_src.cpu().numpy()[:offsets[-1]]
    y_perm = oracle.expert_ffn(x[row_src], offsets, w1, w3, w2, act)
    ref = np.zeros((T, h))
    ref[row_src] = y_perm * wt[row_src]
    assert rowwise(y[valid], ref[valid]) <= TOL[out_dtype if dtype == "bf16" and out_dtype == "bf16" else dtype]
    assert np.all(y[~valid] == 7.0)


@pytest.mark.parametrize("g", [0, 1, 2, 3])
def test_ffn_shard_slice_of_full_weights(g):
    """moe_pack_weights cuts shard g (inner columns [g*f, (g+1)*f)) out of the full weights;
    the shard partials, summed over g in fp32 on the host, give the unsharded output."""
    rng = np.random.default_rng(42)
    F, f = 4 * 96, 96
    x, w1, w3, w2, offsets = _ffn_case(rng, [70, 3, 0, 190], 128, F, "gelu", "bf16")
    got = _run_ffn(x, w1, w3, w2, offsets, "gelu", "bf16", out_dtype=torch.float32, col0=g * f, f=f)
    ref = oracle.expert_ffn(x, offsets, w1, w3, w2, "gelu", col0=g * f, f=f)
    assert rowwise(got, ref) <= TOL["bf16"]


def test_shard_partials_sum_to_full_layer_on_gpu():
    rng = np.random.default_rng(43)
    F, G = 300, 3
    x, w1, w3, w2, offsets = _ffn_case(rng, [100, 0, 31, 250], 192, F, "swiglu", "bf16")
    parts = [_run_ffn(x, w1, w3, w2, offsets, "swiglu", "bf16", out_dtype=torch.float32, col0=g * 100, f=100)
             for g in range(G)]
    full = oracle.expert_ffn(x, offsets, w1, w3, w2, "swiglu")
    assert rowwise(sum(parts), full) <= TOL["bf16"]


def test_ffn_with_no_rows():
    rng = np.random.default_rng(0)
    x, w1, w3, w2, offsets = _ffn_case(rng, [0, 0, 0], 64, 64, "gelu", "bf16")
    dt = torch.bfloat16
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), act="gelu")
    y = moe.expert_ffn_shard(torch.zeros((0, 64), dtype=dt, device="cuda"), to_dev(offsets, torch.int32), packed)
    torch.cuda.synchronize()
    assert y.shape == (0, 64)


# ------------------------------------------------------------------------------- combine

@pytest.mark.parametrize("ydt,odt", [("bf16", "bf16"), ("f32", "f32"), ("bf16", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("T,k,h", [(1, 1, 8), (333, 2, 768), (64, 8, 136)])
def test_combine_parity(ydt, odt, T, k, h):
    rng = np.random.default_rng(T * k + h)
    y_perm = rng.standard_normal((T * k, h)).astype(np.float32)
    if ydt == "bf16":
        y_perm = synth.round_to_bf16(y_perm)
    pos_of = rng.permutation(T * k).reshape(T, k).astype(np.int32)
    w = rng.random((T, k)).astype(np.float32)
    out = moe.combine(to_dev(y_perm, tdt(ydt)), to_dev(pos_of, torch.int32), to_dev(w, torch.float32),
                      out_dtype=tdt(odt))
    torch.cuda.synchronize()
    ref = oracle.combine(y_perm, pos_of, w)
    tol = TOL["bf16"] if "bf16" in (odt,) else TOL["f32"]
    assert rowwise(np_of(out), ref) <= tol


# ------------------------------------------------------------------------------- whole layer

def _gpu_layer(L, partial_dtype=None, fused_gather=True):
    cfg = L.cfg
    dt = tdt(cfg.dtype)
    packed = moe.pack_weights(to_dev(L.w1, dt), to_dev(L.w2, dt), to_dev(L.w3, dt), act=cfg.act)
    layer = moe.MoEShardLayer(to_dev(L.wg, dt), packed, cfg.k, bool(cfg.renorm), max_tokens=cfg.T,
                              partial_dtype=partial_dtype, fused_gather=fused_gather)
    x = to_dev(L.x, dt)
    bias = to_dev(L.sel_bias, torch.float32)
    y = layer(x, bias)
    torch.cuda.synchronize()
    return layer, x, bias, y


SMALL = [("c1", None), ("c2", 1536), ("c3", 4096), ("c4", 160), ("c5", 600), ("c5dec", None)]


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("name,T", SMALL)
def test_layer_end_to_end(name, T, fused):
    L = synth.make(name, seed=0, **({"T": T} if T else {}))
    cfg = L.cfg
    layer, x, bias, y = _gpu_layer(L, fused_gather=fused)
    ref = oracle.forward(L)
    last = layer.last
    gi = last["idx"].cpu().numpy()
    same_set, order_ok = compare_routing(gi, last["w"].cpu().numpy(), ref["idx"], ref["w"], L.x, L.wg, L.sel_bias,
                                         ref["logits"], cfg.k, cfg.dtype == "bf16")
    tol = TOL[cfg.dtype]
    d = last["dispatch"]
    if same_set.all():
        # same pick sets: grouping is unique (order inside a token does not move rows)
        for key in ("counts", "offsets", "row_src"):
            assert np.array_equal(getattr(d, key).cpu().numpy(), ref[key]), key
        assert np.array_equal(by_expert(d.pos_of.cpu().numpy(), gi), by_expert(ref["pos_of"], ref["idx"]))
        if d.x_perm is not None:
            assert np.array_equal(np_of(d.x_perm), ref["x_perm"])
        if last["y_perm"] is not None:  # top-1 with the fused gather writes y directly
            assert rowwise(np_of(last["y_perm"]), ref["y_perm"]) <= tol
    else:
        print(f"{name}: {(~same_set).sum()} tokens picked a different but equally valid set")
    assert rowwise(np_of(y)[same_set], ref["y"][same_set]) <= tol


FULL = ["c1", "c2", "c3", "c4", "c5", "c3u", "c5u", "paper128", "c5dec"]


@pytest.mark.parametrize("name", FULL)
def test_layer_full_size_every_token(name):
    """Full-size workload in the benchmark's launch configuration (rows gathered by the
    expert step; top-1 combine folded into it), and the same layer with x_perm written by
    the dispatch: routing, counts, offsets, the permutation and x_perm bit-exact, and every
    row of y_perm and y within tolerance of the fp64 oracle's whole-layer forward."""
    L = synth.make(name, seed=0)
    cfg = L.cfg
    dt = tdt(cfg.dtype)
    packed = moe.pack_weights(to_dev(L.w1, dt), to_dev(L.w2, dt), to_dev(L.w3, dt), act=cfg.act)
    x = to_dev(L.x, dt)
    bias = to_dev(L.sel_bias, torch.float32)
    ref = oracle.forward(L)
    tol = TOL[cfg.dtype]
    for fused in (True, False):
        layer = moe.MoEShardLayer(to_dev(L.wg, dt), packed, cfg.k, bool(cfg.renorm), max_tokens=cfg.T,
                                  fused_gather=fused)
        y = np_of(layer(x, bias))
        last = layer.last
        gi = last["idx"].cpu().numpy()
        same_set, _ = compare_routing(gi, last["w"].cpu().numpy(), ref["idx"], ref["w"], L.x, L.wg, L.sel_bias,
                                      ref["logits"], cfg.k, cfg.dtype == "bf16")
        print(f"{name} fused={fused}: {(~same_set).sum()} tokens picked another valid set")
        if L.targets is not None:  # the injected skew leaves no token within the rounding margin
            assert same_set.all()
        if same_set.all():
            d = last["dispatch"]
            for key in ("counts", "offsets", "row_src"):
                assert np.array_equal(getattr(d, key).cpu().numpy(), ref[key]), key
            assert np.array_equal(by_expert(d.pos_of.cpu().numpy(), gi), by_expert(ref["pos_of"], ref["idx"]))
            if d.x_perm is not None:
                assert np.array_equal(np_of(d.x_perm), ref["x_perm"])
            if last["y_perm"] is not None:
                err = rowwise(np_of(last["y_perm"]), ref["y_perm"])
                print(f"  y_perm: {cfg.A} rows, max row error {err:.2e}")
                assert err <= tol
        err = rowwise(y[same_set], ref["y"][same_set])
        print(f"  y: {same_set.sum()} of {cfg.T} rows, max row error {err:.2e}")
        assert err <= tol
        del layer


def test_layer_is_deterministic():
    L = synth.make("c5", seed=0, T=3000)
    layer, x, bias, y1 = _gpu_layer(L)
    y1 = y1.clone()
    y2 = layer(x, bias)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_layer_call_smaller_than_its_capacity():
    """A layer sized for 600 tokens, called with 256 (512 assignments, so the second product
    splits its K): the workspace sized for the larger bound holds the split's partials."""
    L = synth.make("c5dec", seed=0, T=256)
    cfg = L.cfg
    dt = torch.bfloat16
    packed = moe.pack_weights(to_dev(L.w1, dt), to_dev(L.w2, dt), act=cfg.act)
    layer = moe.MoEShardLayer(to_dev(L.wg, dt), packed, cfg.k, bool(cfg.renorm), max_tokens=600)
    y = layer(to_dev(L.x, dt), to_dev(L.sel_bias, torch.float32))
    torch.cuda.synchronize()
    ref = oracle.forward(L)
    same_set, _ = compare_routing(layer.last["idx"].cpu().numpy(), layer.last["w"].cpu().numpy(), ref["idx"],
                                  ref["w"], L.x, L.wg, L.sel_bias, ref["logits"], cfg.k, True)
    assert same_set.sum() > 0.9 * cfg.T
    assert rowwise(np_of(y)[same_set], ref["y"][same_set]) <= TOL["bf16"]


def test_layer_is_deterministic_with_split_k():
    """Decode-sized layer (split second product): two calls give the same bits."""
    L = synth.make("c5dec", seed=1)
    layer, x, bias, y1 = _gpu_layer(L)
    y1 = y1.clone()
    y2 = layer(x, bias)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("name,T", [("c5dec", None), ("c2", 1024)])
def test_layer_replays_from_a_graph(name, T):
    """A whole layer forward captured into a HIP graph (the library records no memset and
    never synchronises) replays to the eager result, bit for bit, every time; eager work
    clobbers the output between the replays."""
    L = synth.make(name, seed=2, **({"T": T} if T else {}))
    layer, x, bias, y_eager = _gpu_layer(L)
    y_eager = y_eager.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer(x, bias)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        y_graph = layer(x, bias)
    for r in range(3):
        layer.y.fill_(float(r + 1))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y_graph, y_eager), r


def test_layer_with_no_tokens():
    L = synth.make("c2", seed=0, T=8, E=8)
    dt = torch.bfloat16
    packed = moe.pack_weights(to_dev(L.w1, dt), to_dev(L.w2, dt), act="gelu")
    layer = moe.MoEShardLayer(to_dev(L.wg, dt), packed, 1, max_tokens=8)
    y = layer(torch.zeros((0, L.cfg.h), dtype=dt, device="cuda"))
    torch.cuda.synchronize()
    assert y.shape == (0, L.cfg.h)
    assert layer.last["dispatch"].counts.sum().item() == 0
