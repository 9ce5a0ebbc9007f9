"""Plain fp64 CPU oracle of the verify hot path (C, loaded with ctypes).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library (``paper_2609_37532_amd``) and never imports it.

Functions take numpy arrays; bf16 tensors are ``uint16`` arrays holding the
upper half of IEEE binary32 values.  See ``oracle.c`` for the definitions and
the paper passages each one follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_HDR = os.path.join(_HERE, "oracle.h")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``liboracle.so`` with gcc (strict IEEE double, no fast-math)."""
    if not force and os.path.exists(LIB_PATH) and os.path.getmtime(LIB_PATH) >= max(
        os.path.getmtime(_SRC), os.path.getmtime(_HDR)
    ):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    lib = ctypes.CDLL(LIB_PATH)
    p = ctypes.c_void_p
    i32 = ctypes.c_int32
    lib.oracle_verify_attn.argtypes = [p, p, p, p, p, p, i32, i32, i32, i32, i32,
                                       i32, i32, i32, ctypes.c_double]
    lib.oracle_verify_attn.restype = ctypes.c_int
    lib.oracle_row_argmax.argtypes = [p, i32, i32, i32, p]
    lib.oracle_row_argmax.restype = ctypes.c_int
    lib.oracle_accept.argtypes = [p, i32, p, p, p, p, i32, i32, i32]
    lib.oracle_accept.restype = ctypes.c_int
    lib.oracle_accept_stochastic.argtypes = [p, i32, p, p, p, ctypes.c_double, p, p, p, p,
                                             i32, i32, i32]
    lib.oracle_accept_stochastic.restype = ctypes.c_int
    lib.oracle_successor_interval.argtypes = [p, i32, i32, i32, i32, ctypes.c_double, i32,
                                              p, p]
    lib.oracle_successor_interval.restype = ctypes.c_int
    lib.oracle_dvl_scores.argtypes = [p, i32, i32, p, p, p]
    lib.oracle_dvl_adjust.argtypes = [p, p, i32, i32, i32, p, p]
    lib.oracle_dvl_pack.argtypes = [p, i32, i32, i32, i32, p, p, p, p, p, p, p, p]
    lib.oracle_predictor_forward.argtypes = [p, i32, i32, p, p, p, p, i32, i32, i32, p]
    for f in (lib.oracle_dvl_scores, lib.oracle_dvl_adjust, lib.oracle_dvl_pack,
              lib.oracle_predictor_forward):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def verify_attn(q, cu_qlens, kv_pages, page_table, ctx_lens, *, num_q_heads,
                num_kv_heads, head_dim, page_size, scale, capacity=None):
    """fp64 verify attention; returns ``out`` float64 [capacity, Hq, D].

    ``q`` uint16 [cap, Hq, D]; ``kv_pages`` uint16 [P, 2, Hkv, page*D];
    ``page_table`` int32 [B, P_max]; ``cu_qlens`` int32 [B+1];
    ``ctx_lens`` int32 [B].
    """
    lib = _load()
    q = _c(q, np.uint16)
    kv = _c(kv_pages, np.uint16)
    cu = _c(cu_qlens, np.int32)
    pt = _c(page_table, np.int32)
    ctx = _c(ctx_lens, np.int32)
    cap = q.shape[0] if capacity is None else capacity
    B = ctx.shape[0]
    assert cu.shape[0] == B + 1 and pt.shape[0] == B
    out = np.empty((cap, num_q_heads, head_dim), dtype=np.float64)
    rc = lib.oracle_verify_attn(_ptr(q), _ptr(cu), _ptr(kv), _ptr(pt), _ptr(ctx),
                                _ptr(out), B, cap, num_q_heads, num_kv_heads,
                                head_dim, page_size, pt.shape[1], kv.shape[0],
                                float(scale))
    if rc != 0:
        raise ValueError("oracle_verify_attn rejected its input (rc=%d)" % rc)
    return out


def _logits_args(logits, dtype):
    if dtype == "f32":
        return _c(logits, np.float32), 0
    if dtype == "bf16":
        return _c(logits, np.uint16), 1
    raise ValueError(dtype)


def row_argmax(logits, dtype):
    """Lowest-index argmax of each row; ``dtype`` is 'f32' or 'bf16' (uint16 bits)."""
    lib = _load()
    lg, code = _logits_args(logits, dtype)
    rows, vocab = lg.shape
    idx = np.empty(rows, dtype=np.int32)
    rc = lib.oracle_row_argmax(_ptr(lg), code, rows, vocab, _ptr(idx))
    if rc != 0:
        raise ValueError("oracle_row_argmax rejected its input (rc=%d)" % rc)
    return idx


def accept(logits, dtype, cu_qlens, draft_tokens):
    """Greedy acceptance; returns ``(accept_len, next_token)`` int32 [B]."""
    lib = _load()
    lg, code = _logits_args(logits, dtype)
    cu = _c(cu_qlens, np.int32)
    dr = _c(draft_tokens, np.int32)
    cap, vocab = lg.shape
    B = cu.shape[0] - 1
    a = np.empty(B, dtype=np.int32)
    nxt = np.empty(B, dtype=np.int32)
    rc = lib.oracle_accept(_ptr(lg), code, _ptr(cu), _ptr(dr), _ptr(a), _ptr(nxt),
                           B, cap, vocab)
    if rc != 0:
        raise ValueError("oracle_accept rejected its input (rc=%d)" % rc)
    return a, nxt


# ---------------------------------------------------------------- DVL (Sec. III-C)
def dvl_scores(pred_logits, w):
    """Prefix scores, estimates and initial lengths (Alg. 1, Eqs. (6)-(7)).

    ``pred_logits`` float32 [n, w-1]; returns ``(q [n, w] f32, ell [n] f32,
    k0 [n] i32)``."""
    lib = _load()
    lg = _c(pred_logits, np.float32).reshape(-1, w - 1)
    n = lg.shape[0]
    q = np.zeros((n, w), np.float32)
    ell = np.zeros(n, np.float32)
    k0 = np.zeros(n, np.int32)
    rc = lib.oracle_dvl_scores(_ptr(lg), n, w, _ptr(q), _ptr(ell), _ptr(k0))
    if rc != 0:
        raise ValueError("oracle_dvl_scores rejected its input (rc=%d)" % rc)
    return q, ell, k0


def dvl_adjust(q, k0, budget):
    """Budget adjustment (Eqs. (8)-(9)); returns ``(k [n] i32, updates)``."""
    lib = _load()
    q = _c(q, np.float32)
    n, w = q.shape
    k0 = _c(k0, np.int32)
    k = np.zeros(n, np.int32)
    upd = ctypes.c_int32(0)
    rc = lib.oracle_dvl_adjust(_ptr(q), _ptr(k0), n, w, int(budget), _ptr(k),
                               ctypes.byref(upd))
    if rc != 0:
        raise ValueError("oracle_dvl_adjust rejected its input (rc=%d)" % rc)
    return k, int(upd.value)


def dvl_pack(k_live, n_bs, w, m_bs, tokens, positions, kv_refs):
    """Offsets, packing, sentinels and tail placeholders (Eqs. (10)-(11)).

    Fields are int32 [n_bs, w]; returns a dict with ``k`` [n_bs],
    ``offsets`` [n_bs+1] and ``tokens``, ``positions``, ``kv_refs`` [m_bs]."""
    lib = _load()
    kl = _c(k_live, np.int32)
    fields = [_c(f, np.int32).reshape(n_bs, w) for f in (tokens, positions, kv_refs)]
    k = np.zeros(n_bs, np.int32)
    off = np.zeros(n_bs + 1, np.int32)
    packed = [np.zeros(m_bs, np.int32) for _ in range(3)]
    rc = lib.oracle_dvl_pack(_ptr(kl), kl.shape[0], n_bs, w, m_bs, *[_ptr(f) for f in fields],
                             _ptr(k), _ptr(off), *[_ptr(p) for p in packed])
    if rc != 0:
        raise ValueError("oracle_dvl_pack rejected its input (rc=%d)" % rc)
    return dict(k=k, offsets=off, tokens=packed[0], positions=packed[1], kv_refs=packed[2])


def dvl_allocate_pack(pred_logits, n_live, tokens, positions, kv_refs, w=16):
    """Alg. 1 end to end for a bucket of ``n_bs`` requests of which the first
    ``n_live`` are live: budget M_live = w*n_live/2, capacity M_bs = w*n_bs/2.

    Returns the :func:`dvl_pack` dict plus ``q`` [n_bs, w] (zero rows for
    sentinels), ``k0`` [n_live], ``ell`` [n_live] and ``updates``."""
    lg = _c(pred_logits, np.float32).reshape(-1, w - 1)
    n_bs = lg.shape[0]
    n = int(n_live)
    assert 0 <= n <= n_bs and w % 2 == 0
    q = np.zeros((n_bs, w), np.float32)
    if n > 0:
        ql, ell, k0 = dvl_scores(lg[:n], w)
        q[:n] = ql
        k, upd = dvl_adjust(ql, k0, w * n // 2)
    else:
        ell, k0, k, upd = (np.zeros(0, np.float32), np.zeros(0, np.int32),
                           np.zeros(0, np.int32), 0)
    res = dvl_pack(k, n_bs, w, w * n_bs // 2, tokens, positions, kv_refs)
    res.update(q=q, k0=k0, ell=ell, updates=upd)
    return res


def accept_stochastic(logits, dtype, cu_qlens, draft_tokens, uniforms, temperature):
    """Stochastic prefix verifier (Sec. III-D); ``uniforms`` float32 [cap, 2].
    Returns ``(accept_len, next_token, margin_accept, margin_sample)``."""
    lib = _load()
    lg, code = _logits_args(logits, dtype)
    cu = _c(cu_qlens, np.int32)
    dr = _c(draft_tokens, np.int32)
    un = _c(uniforms, np.float32)
    cap, vocab = lg.shape
    assert un.shape == (cap, 2)
    B = cu.shape[0] - 1
    a = np.empty(B, dtype=np.int32)
    nxt = np.empty(B, dtype=np.int32)
    ma = np.empty(B, dtype=np.float64)
    ms = np.empty(B, dtype=np.float64)
    rc = lib.oracle_accept_stochastic(_ptr(lg), code, _ptr(cu), _ptr(dr), _ptr(un),
                                      float(temperature), _ptr(a), _ptr(nxt), _ptr(ma),
                                      _ptr(ms), B, cap, vocab)
    if rc != 0:
        raise ValueError("oracle_accept_stochastic rejected its input (rc=%d)" % rc)
    return a, nxt, ma, ms


def successor_interval(logits, dtype, row, removed, temperature, token):
    """Cumulative-probability interval ``(lo, hi)`` of ``token`` in the
    successor distribution of packed row ``row`` (without ``removed``)."""
    lib = _load()
    lg, code = _logits_args(logits, dtype)
    lo, hi = ctypes.c_double(0), ctypes.c_double(0)
    rc = lib.oracle_successor_interval(_ptr(lg), code, int(row), lg.shape[1], int(removed),
                                       float(temperature), int(token), ctypes.byref(lo),
                                       ctypes.byref(hi))
    if rc != 0:
        raise ValueError("oracle_successor_interval rejected its input (rc=%d)" % rc)
    return lo.value, hi.value


def predictor_forward(features, n_live, w1, b1, w2, b2):
    """Acceptance predictor forward (Eq. (5)) in float64: features [n, in],
    W1 [in, hidden], W2 [hidden, out]; rows past ``n_live`` are zero."""
    lib = _load()
    f = _c(features, np.float32)
    w1, b1, w2, b2 = (_c(x, np.float32) for x in (w1, b1, w2, b2))
    n, in_dim = f.shape
    hidden, out_dim = w2.shape
    assert w1.shape == (in_dim, hidden) and b1.shape == (hidden,) and b2.shape == (out_dim,)
    out = np.empty((n, out_dim), np.float64)
    rc = lib.oracle_predictor_forward(_ptr(f), int(n_live), n, _ptr(w1), _ptr(b1), _ptr(w2),
                                      _ptr(b2), in_dim, hidden, out_dim, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_predictor_forward rejected its input (rc=%d)" % rc)
    return out
