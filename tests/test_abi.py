"""The C ABI library loads, exports every declared symbol and rejects bad arguments on the
host before launching anything (CPU only: every call below fails validation, so no HIP
call is made)."""
import ctypes
import os
import re

import pytest

import paper_2503_08467_amd as moe
from paper_2503_08467_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moeshard.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2503_08467_amd import build
        build.build()
    return _lib.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\*?\s*(moe_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) == 16, names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib.SIGNATURES)


def test_status_strings(lib):
    for st in range(6):
        assert _lib.status_string(st).startswith("MOE_")
    assert "unknown" in _lib.status_string(99)


A16 = 0x10000  # a 16-byte aligned non-null address; never dereferenced (validation fails first)


def _route(lib, **kw):
    a = dict(x=A16, xdt=_lib.MOE_BF16, T=8, h=64, wg=A16, E=8, k=2, bias=None, stride=0, renorm=0,
             idx=A16, w=A16, s=None)
    a.update(kw)
    return lib.moe_route(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(k=9), _lib.MOE_ERR_INVALID_ARG),        # k > E
    (dict(k=0), _lib.MOE_ERR_INVALID_ARG),
    (dict(E=0, k=0), _lib.MOE_ERR_INVALID_ARG),
    (dict(E=300, k=2), _lib.MOE_ERR_UNSUPPORTED),  # beyond MOE_MAX_EXPERTS
    (dict(T=-1), _lib.MOE_ERR_INVALID_ARG),
    (dict(h=60), _lib.MOE_ERR_INVALID_ARG),        # h % 8 != 0
    (dict(xdt=7), _lib.MOE_ERR_INVALID_ARG),
    (dict(x=A16 + 4), _lib.MOE_ERR_INVALID_ARG),   # misaligned
    (dict(x=None), _lib.MOE_ERR_INVALID_ARG),      # null required pointer
    (dict(stride=3), _lib.MOE_ERR_INVALID_ARG),    # bias stride neither 0 nor E
    (dict(renorm=2), _lib.MOE_ERR_INVALID_ARG),
])
def test_route_rejects_bad_arguments(lib, kw, status):
    assert _route(lib, **kw) == status


def test_route_with_no_tokens_is_a_noop(lib):
    assert _route(lib, T=0, x=None, idx=None, w=None) == _lib.MOE_OK


def test_dispatch_rejects_small_workspace(lib):
    need = lib.moe_dispatch_workspace_size(100, 2, 16)
    assert need > 0
    st = lib.moe_dispatch(A16, 100, 2, 16, A16, _lib.MOE_BF16, 64, A16, A16, A16, A16, A16, A16, need - 1, None)
    assert st == _lib.MOE_ERR_WORKSPACE
    st = lib.moe_dispatch(A16, 100, 3, 2, A16, _lib.MOE_BF16, 64, A16, A16, A16, A16, A16, A16, need, None)
    assert st == _lib.MOE_ERR_INVALID_ARG  # k > E


def test_pack_rejects_bad_slices(lib):
    E, h, F = 4, 64, 100
    size = lib.moe_packed_weights_size(E, h, 50, _lib.MOE_ACT_GELU, _lib.MOE_BF16)
    args = lambda col0, f, w3=None, act=_lib.MOE_ACT_GELU, nbytes=size: (
        A16, w3, A16, E, h, F, col0, f, act, _lib.MOE_BF16, A16, nbytes, None)
    assert lib.moe_pack_weights(*args(60, 50)) == _lib.MOE_ERR_INVALID_ARG  # col0 + f > F
    assert lib.moe_pack_weights(*args(-1, 50)) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_pack_weights(*args(0, 0)) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_pack_weights(*args(0, 50, nbytes=size - 1)) == _lib.MOE_ERR_WORKSPACE
    assert lib.moe_pack_weights(*args(0, 50, act=_lib.MOE_ACT_SWIGLU)) == _lib.MOE_ERR_INVALID_ARG  # no w3


def test_sizes_follow_the_padded_layout(lib):
    assert lib.moe_padded_inner_width(1) == 128
    assert lib.moe_padded_inner_width(512) == 512
    assert lib.moe_padded_inner_width(1792) == 1792
    assert lib.moe_padded_inner_width(37) == 128
    # W1^T + W2^T (+ W3^T) of E x fp x h elements
    assert lib.moe_packed_weights_size(8, 768, 3072, _lib.MOE_ACT_GELU, _lib.MOE_BF16) == 2 * 8 * 3072 * 768 * 2
    assert lib.moe_packed_weights_size(8, 4096, 1792, _lib.MOE_ACT_SWIGLU, _lib.MOE_BF16) == 3 * 8 * 1792 * 4096 * 2
    assert lib.moe_ffn_workspace_size(1000, 8, 768, 3072, _lib.MOE_ACT_GELU, _lib.MOE_F32) >= 1000 * 3072 * 4


def test_ffn_workspace_holds_split_partials(lib):
    """Small calls split the second product's K: fp32 partials of S x A_max x h follow H
    (bf16: up to 8 parts up to 512 rows; fp32: 4 parts up to 1024 rows)."""
    al = lambda v: (v + 255) // 256 * 256
    ws = lambda A, h, f, dt=_lib.MOE_BF16: lib.moe_ffn_workspace_size(A, 64, h, f, _lib.MOE_ACT_GELU, dt)
    # decode-sized: 128 rows, fp = 4096 (128 K steps of 32) -> 8 parts
    assert ws(128, 1024, 4096) == al(128 * 4096 * 2) + al(8 * 128 * 1024 * 4) + 256
    assert ws(256, 1024, 4096) == al(256 * 4096 * 2) + al(8 * 256 * 1024 * 4) + 256
    assert ws(512, 768, 3072) == al(512 * 3072 * 2) + al(4 * 512 * 768 * 4) + 256
    # fp = 1792: 56 K steps, 8 parts would leave 7 per part -> 4 parts
    assert ws(128, 4096, 1792) == al(128 * 1792 * 2) + al(4 * 128 * 4096 * 4) + 256
    # short K: fp = 128 has 4 steps, too few to split
    assert ws(128, 1024, 128) == al(128 * 128 * 2) + 256
    # larger calls do not split but keep the room (a workspace sized for a bound serves
    # every smaller call)
    assert ws(513, 768, 3072) == al(513 * 3072 * 2) + al(2048 * 768 * 4) + 256
    assert ws(128, 1024, 4096, _lib.MOE_F32) == al(128 * 4096 * 4) + al(4 * 128 * 1024 * 4) + 256
    assert ws(1025, 768, 3072, _lib.MOE_F32) == al(1025 * 3072 * 4) + al(4 * 1024 * 768 * 4) + 256
    # fp32 with fp = 512: 16 K steps, 4 parts would leave 4 each -> no split
    assert ws(128, 1024, 512, _lib.MOE_F32) == al(128 * 512 * 4) + 256
    for dt in (_lib.MOE_BF16, _lib.MOE_F32):
        for h, f in [(1024, 4096), (4096, 1792), (768, 3072), (64, 128), (72, 1000)]:
            sizes = [ws(a, h, f, dt) for a in range(0, 1300, 7)]
            assert sizes == sorted(sizes), (h, f, dt)


def test_ffn_and_combine_reject_bad_arguments(lib):
    ws = lib.moe_ffn_workspace_size(64, 8, 64, 32, _lib.MOE_ACT_GELU, _lib.MOE_BF16)
    ok_args = [A16, A16, 64, 8, 64, 32, _lib.MOE_ACT_GELU, _lib.MOE_BF16, A16, A16, _lib.MOE_BF16, A16, ws, None]
    bad = list(ok_args); bad[11 + 1] = ws - 1
    assert lib.moe_expert_ffn_shard(*bad) == _lib.MOE_ERR_WORKSPACE
    bad = list(ok_args); bad[6] = 5
    assert lib.moe_expert_ffn_shard(*bad) == _lib.MOE_ERR_INVALID_ARG
    bad = list(ok_args); bad[3] = 257
    assert lib.moe_expert_ffn_shard(*bad) == _lib.MOE_ERR_UNSUPPORTED
    bad = list(ok_args); bad[8] = A16 + 8
    assert lib.moe_expert_ffn_shard(*bad) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(A16, _lib.MOE_BF16, A16, A16, 4, 0, 64, A16, _lib.MOE_BF16, None) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(A16, _lib.MOE_BF16, A16, A16, 4, 1, 12, A16, _lib.MOE_BF16, None) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(None, _lib.MOE_BF16, None, None, 0, 1, 64, None, _lib.MOE_BF16, None) == _lib.MOE_OK


def test_per_expert_ffn_rejects_bad_host_offsets(lib):
    """The per-expert variant checks its host copy of the offsets before any launch."""
    E = 4
    ws = lib.moe_ffn_workspace_size(64, E, 64, 32, _lib.MOE_ACT_GELU, _lib.MOE_BF16)

    def call(offs):
        host = None if offs is None else (ctypes.c_int32 * len(offs))(*offs)
        addr = None if host is None else ctypes.addressof(host)
        return lib.moe_expert_ffn_shard_per_expert(A16, A16, addr, 64, E, 64, 32, _lib.MOE_ACT_GELU, _lib.MOE_BF16,
                                                   A16, A16, _lib.MOE_BF16, A16, ws, None)

    assert call(None) == _lib.MOE_ERR_INVALID_ARG
    assert call([0, 10, 5, 20, 30]) == _lib.MOE_ERR_INVALID_ARG   # decreasing
    assert call([-1, 10, 20, 30, 40]) == _lib.MOE_ERR_INVALID_ARG  # negative start
    assert call([0, 10, 20, 30, 65]) == _lib.MOE_ERR_INVALID_ARG   # past A_max
    bad_ws = lib.moe_expert_ffn_shard_per_expert(A16, A16, None, 64, E, 64, 32, _lib.MOE_ACT_GELU, _lib.MOE_BF16,
                                                 A16, A16, _lib.MOE_BF16, A16, ws - 1, None)
    assert bad_ws == _lib.MOE_ERR_WORKSPACE


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensor"):
        moe.route(x, torch.zeros(8, 64, dtype=torch.bfloat16), 1)


def test_bench_names_the_expert_step_kernels():
    # the counter summaries pick the expert-step launches out of a profile by name
    import bench
    up = ["void moe::(anonymous namespace)::gemm_up_pairs<0>(moe::(anonymous namespace)::GroupedGemm)",
          "void moe::(anonymous namespace)::gemm_bf16_lds<128, 256, 32, 3, 2, true, 2>(moe::(anonymous namespace)::GroupedGemm)",
          "void moe::(anonymous namespace)::gemm_f32<0, false>(moe::(anonymous namespace)::GroupedGemm)"]
    down = ["void moe::(anonymous namespace)::gemm_bf16_lds<128, 384, 32, 3, 3, true, 4>(moe::(anonymous namespace)::GroupedGemm)",
            "void moe::(anonymous namespace)::gemm_bf16_lds<128, 256, 32, 3, 3, false, 2>(moe::(anonymous namespace)::GroupedGemm)",
            "void moe::(anonymous namespace)::gemm_f32<3, true>(moe::(anonymous namespace)::GroupedGemm)",
            "void moe::(anonymous namespace)::split_reduce<true>(float const*, int, long, int, int const*, int, "
            "void*, int, int const*, float const*, long)"]
    assert all(bench.is_ffn_kernel(n) for n in up + down)
    assert not bench.is_ffn_kernel("void moe::(anonymous namespace)::route_lds_kernel<1>(unsigned short const*)")
    assert [bench.ffn_matrix(n) for n in up] == ["up"] * 3
    assert [bench.ffn_matrix(n) for n in down] == ["down"] * 4
    # the other layer steps are summarised separately; packing, casts and the probe are not steps
    assert bench.is_layer_kernel("void moe::(anonymous namespace)::route_lds_kernel<1>(unsigned short const*)")
    assert bench.is_layer_kernel("moe::(anonymous namespace)::dispatch_fused(int const*, long)")
    assert bench.is_layer_kernel("void moe::(anonymous namespace)::combine_kernel<true, true>(void const*)")
    assert not bench.is_layer_kernel("void moe::(anonymous namespace)::transpose_pad<unsigned short>(int)")
    assert not bench.is_layer_kernel("void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel>")


def test_bench_stage_bytes():
    """Algorithmic bytes of the non-GEMM steps: inputs read once, outputs written once."""
    import bench
    import synth
    c2, c5 = synth.CONFIGS["c2"], synth.CONFIGS["c5"]
    b = bench.stage_bytes(c2, fused_gather=True, top1_fused=True, bias_per_row=True)
    assert b["route"] == 8192 * 768 * 2 + 64 * 768 * 2 + 8192 * 64 * 4 + 8192 * 8
    assert b["dispatch"] == 3 * 8192 * 4 + 129 * 4 and b["combine"] == 0
    b = bench.stage_bytes(c5, fused_gather=False, top1_fused=False, bias_per_row=False)
    A = 32768 * 2
    assert b["dispatch"] == 3 * A * 4 + 129 * 4 + 2 * A * 1024 * 2
    assert b["combine"] == A * 1024 * 2 + 32768 * 1024 * 2 + 32768 * 16


def test_bench_refuses_more_than_one_gpu():
    """Only one GPU is measured: --gpus above 1 exits with a message before touching a GPU."""
    import subprocess
    import sys
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_bench_cpu_baseline_is_bounded():
    """The oracle leg of the bench line: a bounded sample, its size and thread count stated."""
    import bench
    rec = bench.cpu_baseline("c1", 0, budget_s=2.0)
    assert rec["kind"] == "oracle" and rec["unit"] == "tokens/s" and rec["value"] > 0
    assert rec["cores"] >= 1 and "tokens of workload c1" in rec["sample"]


def test_noalloc_rejects_calls_beyond_its_static_array(lib):
    """The no-allocation expert step refuses, before touching the GPU, a call whose scratch
    would not fit the static array; a call that fits passes validation (not run here)."""
    h, f, E = 64, 4096, 2
    big, small = 10000, 4000
    assert lib.moe_ffn_workspace_size(big, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16) > _lib.MOE_NOALLOC_SCRATCH_BYTES
    assert lib.moe_ffn_workspace_size(small, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16) <= \
        _lib.MOE_NOALLOC_SCRATCH_BYTES
    st = lib.moe_expert_ffn_shard_noalloc(A16, A16, big, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16, A16, A16,
                                          _lib.MOE_BF16, None)
    assert st == _lib.MOE_ERR_TOO_LARGE
    # ordinary argument errors come first
    st = lib.moe_expert_ffn_shard_noalloc(A16 + 4, A16, big, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16, A16, A16,
                                          _lib.MOE_BF16, None)
    assert st == _lib.MOE_ERR_INVALID_ARG


def test_gather_combine_rejects_bad_arguments(lib):
    """The one-call expert step plus combine checks k, the output dtype and its pointers
    before any launch."""
    T, k, E, h, f = 64, 2, 4, 64, 32
    ws = lib.moe_ffn_workspace_size(T * k, E, h, f, _lib.MOE_ACT_GELU, _lib.MOE_BF16)
    flag = ctypes.c_int32(7)

    def call(k=k, pos=A16, w=A16, y=A16, out_dt=_lib.MOE_BF16, T=T):
        return lib.moe_expert_ffn_shard_gather_combine(A16, T, A16, A16, pos, w, k, E, h, f, _lib.MOE_ACT_GELU,
                                                       _lib.MOE_BF16, A16, A16, _lib.MOE_BF16, y, out_dt,
                                                       ctypes.addressof(flag), A16, ws, None)
    assert call(k=0) == _lib.MOE_ERR_INVALID_ARG
    assert call(pos=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(w=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(w=A16 + 2) == _lib.MOE_ERR_INVALID_ARG
    assert call(y=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(out_dt=9) == _lib.MOE_ERR_INVALID_ARG
    assert flag.value == 7  # untouched by a rejected call
    # no tokens: nothing to launch, nothing written
    assert call(T=0, pos=None, w=None, y=None) == _lib.MOE_OK
    assert flag.value == 1


def test_route_dispatch_checks_both_steps_arguments(lib):
    """The one-call route and dispatch rejects what either call would, before any launch."""
    T, h, E, k = 64, 128, 64, 2
    ws = lib.moe_dispatch_workspace_size(T, k, E)

    def call(k=k, E=E, counts=A16, ws_bytes=ws, renorm=0, stride=0):
        return lib.moe_route_dispatch(A16, _lib.MOE_BF16, T, h, A16, E, k, None, stride, renorm, A16, A16, counts,
                                      A16, A16, A16, A16, ws_bytes, None)
    assert call(k=0) == _lib.MOE_ERR_INVALID_ARG
    assert call(k=E + 1) == _lib.MOE_ERR_INVALID_ARG
    assert call(E=300, k=2) == _lib.MOE_ERR_UNSUPPORTED
    assert call(counts=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(ws_bytes=ws - 1) == _lib.MOE_ERR_WORKSPACE
    assert call(renorm=2) == _lib.MOE_ERR_INVALID_ARG
    assert call(stride=5) == _lib.MOE_ERR_INVALID_ARG
