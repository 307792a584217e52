"""Python face of the C ABI: the calls of the layer plus the one-time shard packing.

Argument marshalling only -- every step of the layer runs in the HIP kernels of
libmoeshard.so.  Tensors must be contiguous CUDA (HIP) tensors; torch provides the device
memory and the stream (the current stream of the tensors' device unless one is given).
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import Optional

import torch

from . import _lib

_DT = {torch.bfloat16: _lib.MOE_BF16, torch.float32: _lib.MOE_F32}


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}: use torch.bfloat16 or torch.float32") from None


def _torch_dtype(code: int) -> torch.dtype:
    return torch.bfloat16 if code == _lib.MOE_BF16 else torch.float32


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (no CPU path exists)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(t: torch.Tensor, stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(t.device)
    return s.cuda_stream


def route(x: torch.Tensor, w_gate: torch.Tensor, k: int, sel_bias: Optional[torch.Tensor] = None,
          renorm: bool = False, out=None, stream=None):
    """Step 1: returns (topk_idx [T,k] int32, topk_w [T,k] float32)."""
    _dev(x, "x"), _dev(w_gate, "w_gate")
    T, h = x.shape
    E = w_gate.shape[0]
    if w_gate.shape[1] != h or w_gate.dtype != x.dtype:
        raise ValueError("w_gate must be [E, h] with the dtype of x")
    stride = 0
    if sel_bias is not None:
        _dev(sel_bias, "sel_bias")
        if sel_bias.dtype != torch.float32:
            raise TypeError("sel_bias must be float32")
        stride = 0 if sel_bias.dim() == 1 else E
        if sel_bias.numel() != (E if stride == 0 else T * E):
            raise ValueError("sel_bias must be [E] or [T, E]")
    if out is None:
        idx = torch.empty((T, k), dtype=torch.int32, device=x.device)
        w = torch.empty((T, k), dtype=torch.float32, device=x.device)
    else:
        idx, w = out
    _lib.call("moe_route", _ptr(x), _dt(x), T, h, _ptr(w_gate), E, k, _ptr(sel_bias), stride,
              int(bool(renorm)), _ptr(idx), _ptr(w), _stream(x, stream))
    return idx, w


@dataclasses.dataclass
class Dispatch:
    counts: torch.Tensor  # [E] int32
    offsets: torch.Tensor  # [E+1] int32
    row_src: torch.Tensor  # [A] int32
    pos_of: torch.Tensor  # [T,k] int32
    x_perm: Optional[torch.Tensor]  # [A,h]; None when the expert step gathers the rows itself


def dispatch_workspace_size(T: int, k: int, E: int) -> int:
    return int(_lib.load().moe_dispatch_workspace_size(T, k, E))


def alloc_dispatch(T: int, k: int, E: int, h: int, dtype, device, x_perm: bool = True) -> tuple:
    """Output buffers and workspace of moe_dispatch (x_perm=False: indices only)."""
    d = Dispatch(counts=torch.empty(E, dtype=torch.int32, device=device),
                 offsets=torch.empty(E + 1, dtype=torch.int32, device=device),
                 row_src=torch.empty(T * k, dtype=torch.int32, device=device),
                 pos_of=torch.empty((T, k), dtype=torch.int32, device=device),
                 x_perm=torch.empty((T * k, h), dtype=dtype, device=device) if x_perm else None)
    ws = torch.empty(max(dispatch_workspace_size(T, k, E), 16), dtype=torch.uint8, device=device)
    return d, ws


def dispatch(topk_idx: torch.Tensor, x: torch.Tensor, E: int, out: Optional[Dispatch] = None,
             ws: Optional[torch.Tensor] = None, stream=None, x_perm: bool = True) -> Dispatch:
    """Step 2: group the T*k assignments per expert (stable in (t, j) order).  With
    x_perm=False (or out.x_perm None) only the indices are written."""
    _dev(topk_idx, "topk_idx"), _dev(x, "x")
    if topk_idx.dtype != torch.int32:
        raise TypeError("topk_idx must be int32")
    T, k = topk_idx.shape
    h = x.shape[1]
    if out is None or ws is None:
        out, ws = alloc_dispatch(T, k, E, h, x.dtype, x.device, x_perm=x_perm)
    _lib.call("moe_dispatch", _ptr(topk_idx), T, k, E, _ptr(x), _dt(x), h, _ptr(out.counts),
              _ptr(out.offsets), _ptr(out.row_src), _ptr(out.pos_of), _ptr(out.x_perm), _ptr(ws),
              ws.numel(), _stream(x, stream))
    return out


def route_dispatch(x: torch.Tensor, w_gate: torch.Tensor, k: int, sel_bias: Optional[torch.Tensor] = None,
                   renorm: bool = False, out=None, disp: Optional[Dispatch] = None, ws: Optional[torch.Tensor] = None,
                   stream=None):
    """Steps 1 and 2 in one call (one launch for decode-sized batches); the dispatch writes
    indices only (no x_perm).  Returns (topk_idx, topk_w, Dispatch)."""
    _dev(x, "x"), _dev(w_gate, "w_gate")
    T, h = x.shape
    E = w_gate.shape[0]
    if w_gate.shape[1] != h or w_gate.dtype != x.dtype:
        raise ValueError("w_gate must be [E, h] with the dtype of x")
    stride = 0
    if sel_bias is not None:
        _dev(sel_bias, "sel_bias")
        if sel_bias.dtype != torch.float32:
            raise TypeError("sel_bias must be float32")
        stride = 0 if sel_bias.dim() == 1 else E
        if sel_bias.numel() != (E if stride == 0 else T * E):
            raise ValueError("sel_bias must be [E] or [T, E]")
    if out is None:
        idx = torch.empty((T, k), dtype=torch.int32, device=x.device)
        w = torch.empty((T, k), dtype=torch.float32, device=x.device)
    else:
        idx, w = out
    if disp is None or ws is None:
        disp, ws = alloc_dispatch(T, k, E, h, x.dtype, x.device, x_perm=False)
    _lib.call("moe_route_dispatch", _ptr(x), _dt(x), T, h, _ptr(w_gate), E, k, _ptr(sel_bias), stride,
              int(bool(renorm)), _ptr(idx), _ptr(w), _ptr(disp.counts), _ptr(disp.offsets), _ptr(disp.row_src),
              _ptr(disp.pos_of), _ptr(ws), ws.numel(), _stream(x, stream))
    return idx, w, disp


def padded_inner_width(f: int) -> int:
    return int(_lib.load().moe_padded_inner_width(f))


@dataclasses.dataclass
class PackedShard:
    """One device's shard of every expert, laid out for the grouped GEMM."""
    buf: torch.Tensor
    E: int
    h: int
    f: int
    act: str
    dtype: torch.dtype


def pack_weights(w1: torch.Tensor, w2: torch.Tensor, w3: Optional[torch.Tensor] = None,
                 col0: int = 0, f: Optional[int] = None, act: str = "gelu", stream=None) -> PackedShard:
    """loadShard: slice inner columns [col0, col0+f) of W1/W3 [E,h,F] and rows of W2 [E,F,h]."""
    _dev(w1, "w1"), _dev(w2, "w2")
    E, h, F = w1.shape
    if f is None:
        f = F - col0
    if w2.shape != (E, F, h) or w2.dtype != w1.dtype:
        raise ValueError("w2 must be [E, F, h] with the dtype of w1")
    a = _lib.ACTS[act]
    if a == _lib.MOE_ACT_SWIGLU:
        if w3 is None or w3.shape != w1.shape or w3.dtype != w1.dtype:
            raise ValueError("SwiGLU needs w3 shaped and typed like w1")
        _dev(w3, "w3")
    lib = _lib.load()
    nbytes = int(lib.moe_packed_weights_size(E, h, f, a, _dt(w1)))
    buf = torch.empty(nbytes, dtype=torch.uint8, device=w1.device)
    _lib.call("moe_pack_weights", _ptr(w1), _ptr(w3) if a == _lib.MOE_ACT_SWIGLU else None, _ptr(w2), E, h,
              F, col0, f, a, _dt(w1), _ptr(buf), nbytes, _stream(w1, stream))
    return PackedShard(buf, E, h, f, act, w1.dtype)


def ffn_workspace_size(A_max: int, packed: PackedShard) -> int:
    return int(_lib.load().moe_ffn_workspace_size(A_max, packed.E, packed.h, packed.f,
                                                  _lib.ACTS[packed.act], _DT[packed.dtype]))


def expert_ffn_shard(x_perm: torch.Tensor, offsets: torch.Tensor, packed: PackedShard,
                     out_dtype: Optional[torch.dtype] = None, A_max: Optional[int] = None,
                     out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """Step 4: y_perm[p] = act(x_perm[p] . W1_e^g) . W2_e^g for every grouped row p."""
    _dev(x_perm, "x_perm"), _dev(offsets, "offsets")
    if x_perm.dtype != packed.dtype:
        raise TypeError("x_perm must have the packed weights' dtype")
    A = x_perm.shape[0]
    A_max = A if A_max is None else A_max
    if A_max > A:
        raise ValueError("A_max exceeds the rows of x_perm")
    out_dtype = out_dtype or x_perm.dtype
    if out is None:
        out = torch.empty((A, packed.h), dtype=out_dtype, device=x_perm.device)
    if ws is None:
        ws = torch.empty(max(ffn_workspace_size(A_max, packed), 16), dtype=torch.uint8, device=x_perm.device)
    _lib.call("moe_expert_ffn_shard", _ptr(x_perm), _ptr(offsets), A_max, packed.E, packed.h, packed.f,
              _lib.ACTS[packed.act], _DT[packed.dtype], _ptr(packed.buf), _ptr(out), _dt(out), _ptr(ws),
              ws.numel(), _stream(x_perm, stream))
    return out


def expert_ffn_shard_noalloc(x_perm: torch.Tensor, offsets: torch.Tensor, packed: PackedShard,
                             out: torch.Tensor, A_max: Optional[int] = None, stream=None) -> torch.Tensor:
    """Step 4 as expert_ffn_shard, with no workspace: the library's static per-device scratch
    array holds it (calls on one GPU must not overlap).  The caller passes the output."""
    _dev(x_perm, "x_perm"), _dev(offsets, "offsets"), _dev(out, "out")
    if x_perm.dtype != packed.dtype:
        raise TypeError("x_perm must have the packed weights' dtype")
    A = x_perm.shape[0]
    A_max = A if A_max is None else A_max
    if A_max > A or out.shape != (A, packed.h):
        raise ValueError("A_max exceeds the rows of x_perm, or out is not [A, h]")
    _lib.call("moe_expert_ffn_shard_noalloc", _ptr(x_perm), _ptr(offsets), A_max, packed.E, packed.h, packed.f,
              _lib.ACTS[packed.act], _DT[packed.dtype], _ptr(packed.buf), _ptr(out), _dt(out),
              _stream(x_perm, stream))
    return out


def expert_ffn_shard_gather(x: torch.Tensor, row_src: torch.Tensor, offsets: torch.Tensor, packed: PackedShard,
                            out_dtype: Optional[torch.dtype] = None, A_max: Optional[int] = None,
                            out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                            stream=None) -> torch.Tensor:
    """Step 4 reading grouped row p from x[row_src[p]] (the dispatch gather folded in)."""
    _dev(x, "x"), _dev(row_src, "row_src"), _dev(offsets, "offsets")
    if x.dtype != packed.dtype:
        raise TypeError("x must have the packed weights' dtype")
    if row_src.dtype != torch.int32:
        raise TypeError("row_src must be int32")
    T = x.shape[0]
    A = row_src.shape[0]
    A_max = A if A_max is None else A_max
    if A_max > A:
        raise ValueError("A_max exceeds the rows of row_src")
    out_dtype = out_dtype or x.dtype
    if out is None:
        out = torch.empty((A, packed.h), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = torch.empty(max(ffn_workspace_size(A_max, packed), 16), dtype=torch.uint8, device=x.device)
    _lib.call("moe_expert_ffn_shard_gather", _ptr(x), T, _ptr(row_src), _ptr(offsets), A_max, packed.E, packed.h,
              packed.f, _lib.ACTS[packed.act], _DT[packed.dtype], _ptr(packed.buf), _ptr(out), _dt(out), _ptr(ws),
              ws.numel(), _stream(x, stream))
    return out


def expert_ffn_shard_gather_combine(x: torch.Tensor, row_src: torch.Tensor, offsets: torch.Tensor,
                                    pos_of: torch.Tensor, topk_w: torch.Tensor, packed: PackedShard,
                                    y_perm: Optional[torch.Tensor] = None, out_dtype: Optional[torch.dtype] = None,
                                    out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                                    stream=None):
    """Steps 4 and 5 for any k: the gathered expert step and the weighted combine in one call
    (one launch for both when the second product's K is split).  Returns (y, y_perm or None
    when y_perm was not written)."""
    _dev(x, "x"), _dev(row_src, "row_src"), _dev(offsets, "offsets"), _dev(pos_of, "pos_of"), _dev(topk_w, "topk_w")
    if x.dtype != packed.dtype:
        raise TypeError("x must have the packed weights' dtype")
    if row_src.dtype != torch.int32 or pos_of.dtype != torch.int32 or topk_w.dtype != torch.float32:
        raise TypeError("row_src and pos_of must be int32, topk_w float32")
    T = x.shape[0]
    if pos_of.dim() != 2 or pos_of.shape[0] != T or topk_w.shape != pos_of.shape:
        raise ValueError("pos_of and topk_w must be [T, k]")
    k = pos_of.shape[1]
    if row_src.numel() < T * k:
        raise ValueError("row_src needs T * k entries")
    out_dtype = out_dtype or x.dtype
    if y_perm is None:
        y_perm = torch.empty((T * k, packed.h), dtype=x.dtype, device=x.device)
    if out is None:
        out = torch.empty((T, packed.h), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = torch.empty(max(ffn_workspace_size(T * k, packed), 16), dtype=torch.uint8, device=x.device)
    written = ctypes.c_int32(0)
    _lib.call("moe_expert_ffn_shard_gather_combine", _ptr(x), T, _ptr(row_src), _ptr(offsets), _ptr(pos_of),
              _ptr(topk_w), k, packed.E, packed.h, packed.f, _lib.ACTS[packed.act], _DT[packed.dtype],
              _ptr(packed.buf), _ptr(y_perm), _dt(y_perm), _ptr(out), _dt(out), ctypes.addressof(written),
              _ptr(ws), ws.numel(), _stream(x, stream))
    return out, (y_perm if written.value else None)


def expert_ffn_shard_top1(x: torch.Tensor, row_src: torch.Tensor, topk_w: torch.Tensor, offsets: torch.Tensor,
                          packed: PackedShard, out_dtype: Optional[torch.dtype] = None,
                          out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                          stream=None) -> torch.Tensor:
    """Steps 4 and 5 for top-1 routing: y[t] = topk_w[t] * FFN_shard(x[t]) in one call."""
    _dev(x, "x"), _dev(row_src, "row_src"), _dev(topk_w, "topk_w"), _dev(offsets, "offsets")
    if x.dtype != packed.dtype:
        raise TypeError("x must have the packed weights' dtype")
    if row_src.dtype != torch.int32 or topk_w.dtype != torch.float32:
        raise TypeError("row_src must be int32 and topk_w float32")
    T = x.shape[0]
    if row_src.numel() != T or topk_w.numel() != T:
        raise ValueError("top-1: row_src and topk_w must have one entry per token")
    out_dtype = out_dtype or x.dtype
    if out is None:
        out = torch.empty((T, packed.h), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = torch.empty(max(ffn_workspace_size(T, packed), 16), dtype=torch.uint8, device=x.device)
    _lib.call("moe_expert_ffn_shard_top1", _ptr(x), T, _ptr(row_src), _ptr(topk_w), _ptr(offsets), packed.E,
              packed.h, packed.f, _lib.ACTS[packed.act], _DT[packed.dtype], _ptr(packed.buf), _ptr(out), _dt(out),
              _ptr(ws), ws.numel(), _stream(x, stream))
    return out


def expert_ffn_shard_per_expert(x_perm: torch.Tensor, offsets: torch.Tensor, packed: PackedShard,
                                out_dtype: Optional[torch.dtype] = None, A_max: Optional[int] = None,
                                out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                                offsets_host: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Step 4 as one launch pair per expert (the ablation of the grouped operation).  The
    per-expert row counts come from a host copy of the offsets; without one, the offsets are
    read back here (a synchronization, as the per-expert loop needs)."""
    _dev(x_perm, "x_perm"), _dev(offsets, "offsets")
    if x_perm.dtype != packed.dtype:
        raise TypeError("x_perm must have the packed weights' dtype")
    A = x_perm.shape[0]
    A_max = A if A_max is None else A_max
    if A_max > A:
        raise ValueError("A_max exceeds the rows of x_perm")
    if offsets_host is None:
        offsets_host = offsets.to("cpu")
    offsets_host = offsets_host.to(torch.int32).contiguous()
    if offsets_host.device.type != "cpu" or offsets_host.numel() != packed.E + 1:
        raise ValueError("offsets_host must be a host tensor of E + 1 offsets")
    out_dtype = out_dtype or x_perm.dtype
    if out is None:
        out = torch.empty((A, packed.h), dtype=out_dtype, device=x_perm.device)
    if ws is None:
        ws = torch.empty(max(ffn_workspace_size(A_max, packed), 16), dtype=torch.uint8, device=x_perm.device)
    _lib.call("moe_expert_ffn_shard_per_expert", _ptr(x_perm), _ptr(offsets), offsets_host.data_ptr(), A_max,
              packed.E, packed.h, packed.f, _lib.ACTS[packed.act], _DT[packed.dtype], _ptr(packed.buf), _ptr(out),
              _dt(out), _ptr(ws), ws.numel(), _stream(x_perm, stream))
    return out


def combine(y_perm: torch.Tensor, pos_of: torch.Tensor, topk_w: torch.Tensor,
            out_dtype: Optional[torch.dtype] = None, out: Optional[torch.Tensor] = None,
            stream=None) -> torch.Tensor:
    """Step 5: y[t] = sum_j topk_w[t,j] * y_perm[pos_of[t,j]] in fp32, rounded once."""
    _dev(y_perm, "y_perm"), _dev(pos_of, "pos_of"), _dev(topk_w, "topk_w")
    T, k = pos_of.shape
    h = y_perm.shape[1]
    if out is None:
        out = torch.empty((T, h), dtype=out_dtype or y_perm.dtype, device=y_perm.device)
    _lib.call("moe_combine", _ptr(y_perm), _dt(y_perm), _ptr(pos_of), _ptr(topk_w), T, k, h, _ptr(out),
              _dt(out), _stream(y_perm, stream))
    return out


class MoEShardLayer:
    """One device's MoE layer: replicated gate + this device's shard of every expert.

    forward() issues the library calls on the current stream into buffers that are
    allocated once for a maximum token count: with fused_gather (the default) routing and
    grouping in one call, then the expert step with the combine in one call (top-1: the
    expert step writing y); without it route, dispatch with x_perm, expert step, combine.
    """

    def __init__(self, w_gate: torch.Tensor, packed: PackedShard, k: int, renorm: bool = False,
                 max_tokens: int = 0, out_dtype: Optional[torch.dtype] = None,
                 partial_dtype: Optional[torch.dtype] = None, fused_gather: bool = True):
        self.w_gate = _dev(w_gate, "w_gate")
        self.packed = packed
        self.E, self.h = w_gate.shape
        self.k = k
        self.renorm = renorm
        self.out_dtype = out_dtype or w_gate.dtype
        self.partial_dtype = partial_dtype or w_gate.dtype
        # fold the dispatch row gather into the expert step (no x_perm buffer)
        self.fused_gather = fused_gather
        self._cap = 0
        if max_tokens:
            self._alloc(max_tokens)

    def _alloc(self, T: int):
        dev = self.w_gate.device
        k, E, h = self.k, self.E, self.h
        self.idx = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.w = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.disp, self.dws = alloc_dispatch(T, k, E, h, self.w_gate.dtype, dev, x_perm=not self.fused_gather)
        self.y_perm = torch.empty((T * k, h), dtype=self.partial_dtype, device=dev)
        self.fws = torch.empty(max(ffn_workspace_size(T * k, self.packed), 16), dtype=torch.uint8, device=dev)
        self.y = torch.empty((T, h), dtype=self.out_dtype, device=dev)
        self._cap = T

    def forward(self, x: torch.Tensor, sel_bias: Optional[torch.Tensor] = None) -> torch.Tensor:
        T = x.shape[0]
        if T > self._cap:
            self._alloc(T)
        k = self.k
        idx, w = self.idx[:T], self.w[:T]
        d = Dispatch(self.disp.counts, self.disp.offsets, self.disp.row_src[:T * k], self.disp.pos_of[:T],
                     None if self.disp.x_perm is None else self.disp.x_perm[:T * k])
        if d.x_perm is None:
            # Steps 1 and 2 in one call (one launch when a single workgroup routes the batch)
            route_dispatch(x, self.w_gate, k, sel_bias, self.renorm, out=(idx, w), disp=d, ws=self.dws)
        else:
            route(x, self.w_gate, k, sel_bias, self.renorm, out=(idx, w))
            dispatch(idx, x, self.E, out=d, ws=self.dws)
        if d.x_perm is None and k == 1:
            # top-1: the expert step writes the weighted rows straight into y
            y_perm = None
            y = expert_ffn_shard_top1(x, d.row_src, w.view(-1), d.offsets, self.packed, out=self.y[:T], ws=self.fws)
        else:
            if d.x_perm is None:
                # Steps 4 and 5 in one call (one launch for the split sum and the combine when
                # the second product's K is split; y_perm is then not written)
                y, y_perm = expert_ffn_shard_gather_combine(x, d.row_src, d.offsets, d.pos_of, w, self.packed,
                                                            y_perm=self.y_perm[:T * k], out=self.y[:T], ws=self.fws)
            else:
                y_perm = expert_ffn_shard(d.x_perm, d.offsets, self.packed, A_max=T * k, out=self.y_perm[:T * k],
                                          ws=self.fws)
                y = combine(y_perm, d.pos_of, w, out=self.y[:T])
        self.last = dict(idx=idx, w=w, dispatch=d, y_perm=y_perm)
        return y

    __call__ = forward
