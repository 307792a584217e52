"""fp64 CPU oracle of the sharded expert-FFN MoE layer -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
package.  The product path (the HIP library and its Python binding) never does.

`moe_oracle.c` holds the arithmetic (plain fp64 loops following Algorithm 1 and Sections
3.1-3.2 of the paper); this module builds it with gcc on first use and wraps it with
numpy.  `brute.py` is a second, independent dense formulation used to pin it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB = os.path.join(_HERE, "libmoe_oracle.so")
_lock = threading.Lock()
_lib = None

ACTS = {"gelu": 0, "gelu_tanh": 1, "swiglu": 2}


def build(force: bool = False) -> str:
    """Compile the oracle (gcc -O3: element-wise loops vectorise, reductions keep their order; OpenMP, no fast-math) into oracle/libmoe_oracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O3", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
                               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
            lib.oracle_route.argtypes = [P, P, I64, I64, I32, I32, P, I64, I32, P, P, P]
            lib.oracle_dispatch.argtypes = [P, I64, I32, I32, P, P, P, P]
            lib.oracle_ffn_rows.argtypes = [I64, P, P, I32, P, P, P, I64, I64, I64, I64, I32, P]
            lib.oracle_expert_ffn.argtypes = [P, P, I32, P, P, P, I64, I64, I64, I64, I32, P]
            lib.oracle_combine.argtypes = [P, P, P, I64, I32, I64, P]
            lib.oracle_layer_tokens.argtypes = [I64, P, P, P, P, I32, I32, P, P, P, I64, I64,
                                                I64, I64, I32, P]
            for fn in ("oracle_route", "oracle_dispatch", "oracle_ffn_rows", "oracle_expert_ffn",
                       "oracle_combine", "oracle_layer_tokens", "oracle_num_threads"):
                getattr(lib, fn).restype = ctypes.c_int
            _lib = lib
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def route(x, wg, k, sel_bias=None, renorm=0):
    """Step 1.  x [T,h], wg [E,h], sel_bias None | [E] | [T,E].
    Returns idx [T,k] int32, w [T,k] float64, logits [T,E] float64."""
    x, wg = _f32(x), _f32(wg)
    T, h = x.shape
    E = wg.shape[0]
    stride = 0
    if sel_bias is not None:
        sel_bias = _f32(sel_bias)
        stride = 0 if sel_bias.ndim == 1 else E
    idx = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float64)
    logits = np.empty((T, E), np.float64)
    rc = _load().oracle_route(_ptr(x), _ptr(wg), T, h, E, k, _ptr(sel_bias), stride, int(renorm),
                              _ptr(idx), _ptr(w), _ptr(logits))
    if rc:
        raise ValueError("oracle_route: invalid arguments")
    return idx, w, logits


def dispatch(idx, E):
    """Step 2.  Returns counts [E], offsets [E+1], row_src [A], pos_of [T,k] (int32)."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    T, k = idx.shape
    counts = np.empty(E, np.int32)
    offsets = np.empty(E + 1, np.int32)
    row_src = np.empty(T * k, np.int32)
    pos_of = np.empty((T, k), np.int32)
    rc = _load().oracle_dispatch(_ptr(idx), T, k, E, _ptr(counts), _ptr(offsets), _ptr(row_src),
                                 _ptr(pos_of))
    if rc:
        raise ValueError("oracle_dispatch: expert id out of range")
    return counts, offsets, row_src, pos_of


def _shard_args(w1, w2, col0, f):
    F = w1.shape[2]
    if f is None:
        f = F - col0
    return F, col0, f


def ffn_rows(rows, expert, w1, w3, w2, act="gelu", col0=0, f=None):
    """Step 4 on independent rows: rows [n,h] through expert[r]'s shard [col0, col0+f)."""
    rows, w1, w2 = _f32(rows), _f32(w1), _f32(w2)
    w3 = None if w3 is None else _f32(w3)
    expert = np.ascontiguousarray(expert, dtype=np.int32)
    n, h = rows.shape
    E = w1.shape[0]
    F, col0, f = _shard_args(w1, w2, col0, f)
    out = np.empty((n, h), np.float64)
    rc = _load().oracle_ffn_rows(n, _ptr(rows), _ptr(expert), E, _ptr(w1), _ptr(w3), _ptr(w2), h,
                                 F, col0, f, ACTS[act], _ptr(out))
    if rc:
        raise ValueError("oracle_ffn_rows: invalid arguments")
    return out


def expert_ffn(x_perm, offsets, w1, w3, w2, act="gelu", col0=0, f=None):
    """Step 4 over grouped rows: y_perm[p] = FFN_e(x_perm[p]) for p in expert e's segment."""
    x_perm, w1, w2 = _f32(x_perm), _f32(w1), _f32(w2)
    w3 = None if w3 is None else _f32(w3)
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    A, h = x_perm.shape
    E = w1.shape[0]
    assert offsets.shape[0] == E + 1 and offsets[-1] == A
    F, col0, f = _shard_args(w1, w2, col0, f)
    y = np.empty((A, h), np.float64)
    rc = _load().oracle_expert_ffn(_ptr(x_perm), _ptr(offsets), E, _ptr(w1), _ptr(w3), _ptr(w2), h,
                                   F, col0, f, ACTS[act], _ptr(y))
    if rc:
        raise ValueError("oracle_expert_ffn: invalid arguments")
    return y


def combine(y_perm, pos_of, w):
    """Step 5.  y[t] = sum_j w[t,j] * y_perm[pos_of[t,j]] (j ascending)."""
    y_perm = np.ascontiguousarray(y_perm, dtype=np.float64)
    pos_of = np.ascontiguousarray(pos_of, dtype=np.int32)
    w = np.ascontiguousarray(w, dtype=np.float64)
    T, k = pos_of.shape
    h = y_perm.shape[1]
    y = np.empty((T, h), np.float64)
    _load().oracle_combine(_ptr(y_perm), _ptr(pos_of), _ptr(w), T, k, h, _ptr(y))
    return y


def layer_tokens(toks, x, idx, w, w1, w3, w2, act="gelu", col0=0, f=None):
    """Layer output of the listed tokens straight from the definition (no grouping)."""
    toks = np.ascontiguousarray(toks, dtype=np.int64)
    x, w1, w2 = _f32(x), _f32(w1), _f32(w2)
    w3 = None if w3 is None else _f32(w3)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    w = np.ascontiguousarray(w, dtype=np.float64)
    k = idx.shape[1]
    h = x.shape[1]
    E = w1.shape[0]
    F, col0, f = _shard_args(w1, w2, col0, f)
    y = np.empty((toks.shape[0], h), np.float64)
    rc = _load().oracle_layer_tokens(toks.shape[0], _ptr(toks), _ptr(x), _ptr(idx), _ptr(w), k, E,
                                     _ptr(w1), _ptr(w3), _ptr(w2), h, F, col0, f, ACTS[act], _ptr(y))
    if rc:
        raise ValueError("oracle_layer_tokens: invalid arguments")
    return y


def forward(layer, col0=0, f=None):
    """Whole layer on a synth.Layer: returns a dict of every intermediate (fp64 / int32)."""
    cfg = layer.cfg
    idx, w, logits = route(layer.x, layer.wg, cfg.k, layer.sel_bias, cfg.renorm)
    counts, offsets, row_src, pos_of = dispatch(idx, cfg.E)
    x_perm = layer.x[row_src]
    y_perm = expert_ffn(x_perm, offsets, layer.w1, layer.w3, layer.w2, cfg.act, col0, f)
    y = combine(y_perm, pos_of, w)
    return dict(idx=idx, w=w, logits=logits, counts=counts, offsets=offsets, row_src=row_src,
                pos_of=pos_of, x_perm=x_perm, y_perm=y_perm, y=y)
