"""The no-allocation expert step (moe_expert_ffn_shard_noalloc) against moe_expert_ffn_shard.

Both run the same kernels; the no-allocation call keeps its workspace in the library's
static per-device array.  Two calls in a row, the second with fewer rows, so that the
second call runs over what the first left in the array; every output is compared bit for
bit with the workspace entry point and within tolerance with the fp64 oracle.
"""
import numpy as np
import pytest

import oracle
import synth
from _util import rowwise, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2503_08467_amd as moe  # noqa: E402
from paper_2503_08467_amd import _lib  # noqa: E402

TOL = {"bf16": 2e-2, "f32": 1e-5}


def _case(seed, counts, h, f, act, dtype):
    rng = np.random.default_rng(seed)
    E, A = len(counts), int(sum(counts))
    x = rng.standard_normal((A, h)).astype(np.float32)
    w1 = (rng.standard_normal((E, h, f)) * 0.03).astype(np.float32)
    w3 = (rng.standard_normal((E, h, f)) * 0.03).astype(np.float32) if act == "swiglu" else None
    w2 = (rng.standard_normal((E, f, h)) * 0.03).astype(np.float32)
    if dtype == "bf16":
        x, w1, w2 = synth.round_to_bf16(x), synth.round_to_bf16(w1), synth.round_to_bf16(w2)
        w3 = None if w3 is None else synth.round_to_bf16(w3)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return x, w1, w3, w2, offsets


def _noalloc(x, offsets, packed, out):
    """The raw C-ABI call: pointers, sizes, the current stream; no workspace argument."""
    _lib.call("moe_expert_ffn_shard_noalloc", x.data_ptr(), offsets.data_ptr(), x.shape[0], packed.E, packed.h,
              packed.f, _lib.ACTS[packed.act], _lib.MOE_BF16 if packed.dtype == torch.bfloat16 else _lib.MOE_F32,
              packed.buf.data_ptr(), out.data_ptr(),
              _lib.MOE_BF16 if out.dtype == torch.bfloat16 else _lib.MOE_F32,
              torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("dtype,act,h,f,first,second", [
    # 3000 rows (one part per K), then 200 (K of the second product in 8 parts)
    ("bf16", "gelu", 1024, 4096, [1400, 0, 1500, 3, 97], [120, 0, 70, 9, 1]),
    # SwiGLU; 700 rows, then 300 (K in 4 parts)
    ("bf16", "swiglu", 512, 1792, [300, 200, 0, 200], [100, 0, 180, 20]),
    ("f32", "gelu", 256, 512, [250, 150, 7], [31, 0, 2]),
])
def test_noalloc_matches_workspace_entry_point(dtype, act, h, f, first, second):
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, w1, w3, w2, off1 = _case(len(first) + h, first, h, f, act, dtype)
    packed = moe.pack_weights(to_dev(w1, dt), to_dev(w2, dt), to_dev(w3, dt), act=act)
    for counts in (first, second):
        off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        xs = x[:off[-1]]
        xd, od = to_dev(xs, dt), to_dev(off, torch.int32)
        ws_out = moe.expert_ffn_shard(xd, od, packed)
        na_out = torch.full_like(ws_out, float("nan"))
        _noalloc(xd, od, packed, na_out)
        torch.cuda.synchronize()
        ib = torch.int16 if dt == torch.bfloat16 else torch.int32
        assert torch.equal(na_out.view(ib), ws_out.view(ib)), counts
        ref = oracle.expert_ffn(xs, off, w1, w3, w2, act)
        got = na_out.float().cpu().numpy()
        assert rowwise(got, ref) <= TOL[dtype], counts


def test_noalloc_rejects_calls_beyond_its_array():
    """bf16, f = 4096: 10000 rows need about 82 MB of scratch, more than the array holds;
    nothing is launched and the output keeps its contents."""
    h, f, E = 64, 4096, 2
    need = _lib.load().moe_ffn_workspace_size(10000, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16)
    assert need > _lib.MOE_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((10000, h), dtype=torch.bfloat16, device="cuda")
    off = torch.tensor([0, 5000, 10000], dtype=torch.int32, device="cuda")
    packed = moe.pack_weights(torch.zeros((E, h, f), dtype=torch.bfloat16, device="cuda"),
                              torch.zeros((E, f, h), dtype=torch.bfloat16, device="cuda"))
    out = torch.full((10000, h), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(moe.MoeError) as e:
        _noalloc(x, off, packed, out)
    assert e.value.status == _lib.MOE_ERR_TOO_LARGE
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
