"""ctypes binding of libdsv.so: argument marshalling only.

Every step of the verify path runs in the HIP kernels of ``libdsv.so``;
PyTorch supplies device memory and streams.  There is no fallback: if the
library is not built, ``load()`` raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdsv.so")

DSV_OK = 0
DSV_F32 = 0
DSV_BF16 = 1
MAX_QLEN = 16
PAGE_SIZE = 16
TIMING_KINDS = ("attn_split", "attn_combine", "accept_argmax", "accept_prefix", "dvl",
                "sample_stats", "sample_draw", "predictor")
PRED_HIDDEN = 64
DVL_MAX_REQS = 1024


class DSVError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (fn, status_string(status), status))


class AttnDims(ctypes.Structure):
    """Mirror of ``dsv_attn_dims``."""
    _fields_ = [("num_reqs", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pages_per_req", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("max_kv_len", ctypes.c_int32), ("scale", ctypes.c_float)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


_lib = None


def load():
    """Load ``libdsv.so`` (built in-tree); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libdsv.so is not built (expected at %s); run "
                           "`python -m paper_2609_37532_amd.build`" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    PD = ctypes.POINTER(AttnDims)
    sig = {
        "dsv_verify_attn_workspace_bytes": (SZ, [PD]),
        "dsv_verify_attn": (ctypes.c_int, [P, P, P, P, P, P, PD, P, SZ, P]),
        "dsv_accept_workspace_bytes": (SZ, [I32, I32, I32]),
        "dsv_accept": (ctypes.c_int, [P, I32, P, P, P, P, I32, I32, I32, P, SZ, P]),
        "dsv_accept_noalloc": (ctypes.c_int, [P, I32, P, P, P, P, I32, I32, I32, P]),
        "dsv_validate_metadata": (ctypes.c_int, [P, P, P, PD, P, P]),
        "dsv_accept_stochastic_workspace_bytes": (SZ, [I32, I32, I32]),
        "dsv_accept_stochastic": (ctypes.c_int, [P, I32, P, P, P, ctypes.c_float, P, P, I32,
                                                 I32, I32, P, SZ, P]),
        "dsv_predictor_workspace_bytes": (SZ, [I32, I32]),
        "dsv_predictor_forward": (ctypes.c_int, [P, P, P, P, P, P, P, I32, I32, I32, I32, P,
                                                 SZ, P]),
        "dsv_dvl_allocate_pack": (ctypes.c_int, [P, P, P, P, P, P, P, P, P, P, P, I32, I32, P]),
        "dsv_graph_capture_begin": (ctypes.c_int, [P]),
        "dsv_graph_capture_end": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_void_p)]),
        "dsv_graph_replay": (ctypes.c_int, [P, P]),
        "dsv_graph_destroy": (ctypes.c_int, [P]),
        "dsv_read_probe": (ctypes.c_int, [P, I32, P, I32, P, I32, P]),
        "dsv_timing_start": (ctypes.c_int, [I32]),
        "dsv_timing_stop": (ctypes.c_int, [ctypes.POINTER(ctypes.c_float),
                                           ctypes.POINTER(ctypes.c_int32)]),
        "dsv_timing_stop_each": (ctypes.c_int, [ctypes.POINTER(ctypes.c_float),
                                                ctypes.POINTER(ctypes.c_int32), I32,
                                                ctypes.POINTER(ctypes.c_int32)]),
        "dsv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().dsv_status_string(int(status)).decode()


def _check(fn: str, status: int) -> None:
    if status != DSV_OK:
        raise DSVError(fn, status)


# ---------------------------------------------------------------- marshalling
def _ptr(t) -> Optional[int]:
    """Device address of a tensor (or None)."""
    return None if t is None else int(t.data_ptr())


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _require(t, name: str, dtypes, ndim: int):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.dtype not in dtypes:
        raise ValueError("%s has dtype %s, expected one of %s" % (name, t.dtype, dtypes))
    if t.dim() != ndim:
        raise ValueError("%s must have %d dims, got %d" % (name, ndim, t.dim()))


def attn_dims(q_packed, kv_pages, page_table, *, max_kv_len: Optional[int] = None,
              scale: Optional[float] = None) -> AttnDims:
    """``dsv_attn_dims`` from tensor shapes: q [cap, Hq, D],
    kv_pages [P, 2, Hkv, 16*D], page_table [B, P_max]."""
    cap, hq, d = q_packed.shape
    num_pages, two, hkv, tile = kv_pages.shape
    if two != 2 or tile % d != 0:
        raise ValueError("kv_pages must be [P, 2, Hkv, page*D]")
    B, pmax = page_table.shape
    return AttnDims(num_reqs=B, capacity=cap, num_q_heads=hq, num_kv_heads=hkv,
                    head_dim=d, page_size=tile // d, max_pages_per_req=pmax,
                    num_pages=num_pages,
                    max_kv_len=int(max_kv_len if max_kv_len is not None else pmax * (tile // d)),
                    scale=float(scale if scale is not None else 1.0 / math.sqrt(d)))


def verify_attn_workspace_bytes(dims: AttnDims) -> int:
    return int(load().dsv_verify_attn_workspace_bytes(ctypes.byref(dims)))


def accept_workspace_bytes(capacity: int, num_reqs: int, vocab: int) -> int:
    return int(load().dsv_accept_workspace_bytes(capacity, num_reqs, vocab))


def alloc_workspace(nbytes: int, device=None):
    """A zero-filled, 256-byte aligned uint8 device buffer of at least ``nbytes``
    (workspaces start zeroed once; the kernels leave them reusable)."""
    import torch
    dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
    buf = torch.zeros(max(1, nbytes) + 256, dtype=torch.uint8, device=dev)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + max(1, nbytes)]


def _bf16_like(torch):
    return (torch.bfloat16, torch.int16, torch.uint16)


def verify_attn(q_packed, cu_qlens, kv_pages, page_table, ctx_lens, out, *,
                max_kv_len: Optional[int] = None, scale: Optional[float] = None,
                workspace=None, stream=None, dims: Optional[AttnDims] = None) -> None:
    """Enqueue ``dsv_verify_attn`` on ``stream`` (default: torch's current)."""
    import torch
    bf = _bf16_like(torch)
    _require(q_packed, "q_packed", bf, 3)
    _require(kv_pages, "kv_pages", bf, 4)
    _require(out, "out", bf, 3)
    _require(cu_qlens, "cu_qlens", (torch.int32,), 1)
    _require(page_table, "page_table", (torch.int32,), 2)
    _require(ctx_lens, "ctx_lens", (torch.int32,), 1)
    if dims is None:
        dims = attn_dims(q_packed, kv_pages, page_table, max_kv_len=max_kv_len, scale=scale)
    if tuple(out.shape) != tuple(q_packed.shape):
        raise ValueError("out must have the shape of q_packed")
    if cu_qlens.numel() != dims.num_reqs + 1 or ctx_lens.numel() != dims.num_reqs:
        raise ValueError("cu_qlens must have B+1 entries and ctx_lens B")
    need = verify_attn_workspace_bytes(dims)
    if workspace is None:
        workspace = alloc_workspace(need, q_packed.device)
    nbytes = workspace.numel() * workspace.element_size()
    _check("dsv_verify_attn", load().dsv_verify_attn(
        _ptr(q_packed), _ptr(cu_qlens), _ptr(kv_pages), _ptr(page_table),
        _ptr(ctx_lens), _ptr(out), ctypes.byref(dims), _ptr(workspace), nbytes,
        _stream_handle(stream)))


def accept(logits_packed, cu_qlens, draft_tokens, accept_len, next_token, *,
           workspace=None, stream=None) -> None:
    """Enqueue ``dsv_accept``; logits are float32 or bfloat16 [cap, vocab]."""
    import torch
    _require(logits_packed, "logits_packed", (torch.float32, torch.bfloat16), 2)
    for t, n in ((cu_qlens, "cu_qlens"), (draft_tokens, "draft_tokens"),
                 (accept_len, "accept_len"), (next_token, "next_token")):
        _require(t, n, (torch.int32,), 1)
    cap, vocab = logits_packed.shape
    B = cu_qlens.numel() - 1
    if draft_tokens.numel() != cap or accept_len.numel() != B or next_token.numel() != B:
        raise ValueError("draft_tokens must be [cap]; accept_len, next_token [B]")
    dtype = DSV_BF16 if logits_packed.dtype == torch.bfloat16 else DSV_F32
    if workspace is None:
        workspace = alloc_workspace(accept_workspace_bytes(cap, B, vocab), logits_packed.device)
    nbytes = workspace.numel() * workspace.element_size()
    _check("dsv_accept", load().dsv_accept(
        _ptr(logits_packed), dtype, _ptr(cu_qlens), _ptr(draft_tokens), _ptr(accept_len),
        _ptr(next_token), B, cap, vocab, _ptr(workspace), nbytes, _stream_handle(stream)))


def accept_noalloc(logits_packed, cu_qlens, draft_tokens, accept_len, next_token, *,
                   stream=None) -> None:
    """Enqueue ``dsv_accept_noalloc``: ``accept`` with the library's fixed
    device scratch in place of a workspace (for callers that cannot
    allocate; calls that overlap on one GPU race)."""
    import torch
    _require(logits_packed, "logits_packed", (torch.float32, torch.bfloat16), 2)
    for t, n in ((cu_qlens, "cu_qlens"), (draft_tokens, "draft_tokens"),
                 (accept_len, "accept_len"), (next_token, "next_token")):
        _require(t, n, (torch.int32,), 1)
    cap, vocab = logits_packed.shape
    B = cu_qlens.numel() - 1
    if draft_tokens.numel() != cap or accept_len.numel() != B or next_token.numel() != B:
        raise ValueError("draft_tokens must be [cap]; accept_len, next_token [B]")
    dtype = DSV_BF16 if logits_packed.dtype == torch.bfloat16 else DSV_F32
    _check("dsv_accept_noalloc", load().dsv_accept_noalloc(
        _ptr(logits_packed), dtype, _ptr(cu_qlens), _ptr(draft_tokens), _ptr(accept_len),
        _ptr(next_token), B, cap, vocab, _stream_handle(stream)))


def accept_stochastic_workspace_bytes(capacity: int, num_reqs: int, vocab: int) -> int:
    return int(load().dsv_accept_stochastic_workspace_bytes(capacity, num_reqs, vocab))


def accept_stochastic(logits_packed, cu_qlens, draft_tokens, uniforms, temperature: float,
                      accept_len, next_token, *, workspace=None, stream=None) -> None:
    """Enqueue ``dsv_accept_stochastic`` (temperature > 0); ``uniforms`` is a
    float32 [cap, 2] device tensor of values in [0, 1)."""
    import torch
    _require(logits_packed, "logits_packed", (torch.float32, torch.bfloat16), 2)
    _require(uniforms, "uniforms", (torch.float32,), 2)
    for t, n in ((cu_qlens, "cu_qlens"), (draft_tokens, "draft_tokens"),
                 (accept_len, "accept_len"), (next_token, "next_token")):
        _require(t, n, (torch.int32,), 1)
    cap, vocab = logits_packed.shape
    B = cu_qlens.numel() - 1
    if draft_tokens.numel() != cap or accept_len.numel() != B or next_token.numel() != B:
        raise ValueError("draft_tokens must be [cap]; accept_len, next_token [B]")
    if tuple(uniforms.shape) != (cap, 2):
        raise ValueError("uniforms must be [cap, 2]")
    dtype = DSV_BF16 if logits_packed.dtype == torch.bfloat16 else DSV_F32
    if workspace is None:
        workspace = alloc_workspace(accept_stochastic_workspace_bytes(cap, B, vocab),
                                    logits_packed.device)
    nbytes = workspace.numel() * workspace.element_size()
    _check("dsv_accept_stochastic", load().dsv_accept_stochastic(
        _ptr(logits_packed), dtype, _ptr(cu_qlens), _ptr(draft_tokens), _ptr(uniforms),
        float(temperature), _ptr(accept_len), _ptr(next_token), B, cap, vocab, _ptr(workspace),
        nbytes, _stream_handle(stream)))


def validate_metadata(cu_qlens, ctx_lens, page_table, dims: AttnDims, err_word,
                      stream=None) -> None:
    _check("dsv_validate_metadata", load().dsv_validate_metadata(
        _ptr(cu_qlens), _ptr(ctx_lens), _ptr(page_table), ctypes.byref(dims),
        _ptr(err_word), _stream_handle(stream)))


def predictor_workspace_bytes(bucket_reqs: int, in_dim: int) -> int:
    return int(load().dsv_predictor_workspace_bytes(bucket_reqs, in_dim))


def predictor_forward(features, num_live, w1, b1, w2, b2, pred_logits, *, workspace=None,
                      stream=None) -> None:
    """Enqueue ``dsv_predictor_forward`` (Eq. (5)): features float32
    [N_bs, in_dim], W1 [in_dim, 64], b1 [64], W2 [64, out], b2 [out] ->
    pred_logits float32 [N_bs, out]; ``num_live`` int32 [1] on the device."""
    import torch
    f32 = (torch.float32,)
    _require(features, "features", f32, 2)
    _require(w1, "w1", f32, 2)
    _require(w2, "w2", f32, 2)
    _require(b1, "b1", f32, 1)
    _require(b2, "b2", f32, 1)
    _require(pred_logits, "pred_logits", f32, 2)
    _require(num_live, "num_live", (torch.int32,), 1)
    n_bs, in_dim = features.shape
    hidden, out_dim = w2.shape
    if tuple(w1.shape) != (in_dim, hidden) or b1.numel() != hidden or b2.numel() != out_dim:
        raise ValueError("weight shapes do not chain")
    if tuple(pred_logits.shape) != (n_bs, out_dim) or num_live.numel() != 1:
        raise ValueError("pred_logits must be [N_bs, out]; num_live one int32")
    if workspace is None:
        workspace = alloc_workspace(predictor_workspace_bytes(n_bs, in_dim), features.device)
    nbytes = workspace.numel() * workspace.element_size()
    _check("dsv_predictor_forward", load().dsv_predictor_forward(
        _ptr(features), _ptr(num_live), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2),
        _ptr(pred_logits), n_bs, in_dim, hidden, out_dim, _ptr(workspace), nbytes,
        _stream_handle(stream)))


def dvl_allocate_pack(pred_logits, num_live, tokens, positions, kv_refs, k_out, cu_qlens,
                      packed_tokens, packed_positions, packed_kv_refs, scores_out=None, *,
                      stream=None) -> None:
    """Enqueue ``dsv_dvl_allocate_pack`` (Sec. III-C, Alg. 1).

    ``pred_logits`` float32 [N_bs, W-1]; ``num_live`` int32 [1] (device);
    ``tokens``, ``positions``, ``kv_refs`` int32 [N_bs, W]; ``k_out`` int32
    [N_bs]; ``cu_qlens`` int32 [N_bs+1]; packed outputs int32 [W*N_bs/2];
    ``scores_out`` float32 [N_bs, W] or None."""
    import torch
    _require(pred_logits, "pred_logits", (torch.float32,), 2)
    n_bs, wm1 = pred_logits.shape
    w = wm1 + 1
    _require(num_live, "num_live", (torch.int32,), 1)
    for t, n in ((tokens, "tokens"), (positions, "positions"), (kv_refs, "kv_refs")):
        _require(t, n, (torch.int32,), 2)
        if tuple(t.shape) != (n_bs, w):
            raise ValueError("%s must be [N_bs, W]" % n)
    for t, n, size in ((k_out, "k_out", n_bs), (cu_qlens, "cu_qlens", n_bs + 1),
                       (packed_tokens, "packed_tokens", w * n_bs // 2),
                       (packed_positions, "packed_positions", w * n_bs // 2),
                       (packed_kv_refs, "packed_kv_refs", w * n_bs // 2)):
        _require(t, n, (torch.int32,), 1)
        if t.numel() != size:
            raise ValueError("%s must have %d entries" % (n, size))
    if num_live.numel() != 1:
        raise ValueError("num_live must hold one int32")
    if scores_out is not None:
        _require(scores_out, "scores_out", (torch.float32,), 2)
        if tuple(scores_out.shape) != (n_bs, w):
            raise ValueError("scores_out must be [N_bs, W]")
    _check("dsv_dvl_allocate_pack", load().dsv_dvl_allocate_pack(
        _ptr(pred_logits), _ptr(num_live), _ptr(tokens), _ptr(positions), _ptr(kv_refs),
        _ptr(k_out), _ptr(cu_qlens), _ptr(packed_tokens), _ptr(packed_positions),
        _ptr(packed_kv_refs), _ptr(scores_out), n_bs, w, _stream_handle(stream)))



PROBE_TILE_BYTES = 4096


def read_probe(buf, order, sink, *, stream=None) -> None:
    """Read-rate probe (not part of the verify path): reads the 4 KiB tiles
    of ``buf`` that ``order`` names, one workgroup per entry of ``sink``,
    which receives the XOR of the 32-bit words each workgroup read."""
    import torch
    _require(buf, "buf", (torch.uint8, torch.int32, torch.float32, torch.bfloat16,
                          torch.float16, torch.int64), 1)
    nbytes = buf.numel() * buf.element_size()
    if nbytes % PROBE_TILE_BYTES or nbytes // PROBE_TILE_BYTES >= 2 ** 31:
        raise ValueError("buf must hold a whole number of 4096-byte tiles (< 2^31 of them)")
    _require(order, "order", (torch.int32,), 1)
    _require(sink, "sink", (torch.int32,), 1)
    _check("dsv_read_probe", load().dsv_read_probe(
        _ptr(buf), nbytes // PROBE_TILE_BYTES, _ptr(order), order.numel(), _ptr(sink),
        sink.numel(), _stream_handle(stream)))


class Graph:
    """One captured hipGraph (Alg. 2: capture once, replay each step)."""

    def __init__(self):
        self._exec = ctypes.c_void_p(None)

    def capture(self, fn, stream) -> "Graph":
        """Record everything ``fn()`` enqueues on ``stream`` (not the null stream)."""
        h = _stream_handle(stream)
        _check("dsv_graph_capture_begin", load().dsv_graph_capture_begin(h))
        try:
            fn()
        finally:
            rc = load().dsv_graph_capture_end(h, ctypes.byref(self._exec))
        _check("dsv_graph_capture_end", rc)
        return self

    def replay(self, stream) -> None:
        _check("dsv_graph_replay", load().dsv_graph_replay(self._exec, _stream_handle(stream)))

    def close(self) -> None:
        if self._exec.value:
            load().dsv_graph_destroy(self._exec)
            self._exec = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KernelTimer:
    """HIP-event timing of the library's eager kernel launches."""

    def __init__(self, max_launches: int = 4096):
        self.max_launches = max_launches
        self.result = None

    def __enter__(self):
        _check("dsv_timing_start", load().dsv_timing_start(self.max_launches))
        return self

    def __exit__(self, *exc):
        cap = self.max_launches
        ms = (ctypes.c_float * cap)()
        kinds = (ctypes.c_int32 * cap)()
        count = ctypes.c_int32(0)
        _check("dsv_timing_stop_each", load().dsv_timing_stop_each(ms, kinds, cap,
                                                                   ctypes.byref(count)))
        self.samples = {k: [] for k in TIMING_KINDS}
        for n in range(count.value):
            if 0 <= kinds[n] < len(TIMING_KINDS):
                self.samples[TIMING_KINDS[kinds[n]]].append(float(ms[n]))
        self.result = {k: (float(sum(v)), len(v)) for k, v in self.samples.items()}
        return False

    def mean_ms(self, kind: str) -> float:
        total, count = self.result[kind]
        return total / count if count else float("nan")

    def median_ms(self, kind: str) -> float:
        v = sorted(self.samples[kind])
        if not v:
            return float("nan")
        h = len(v) // 2
        return v[h] if len(v) % 2 else 0.5 * (v[h - 1] + v[h])

    def count(self, kind: str) -> int:
        return self.result[kind][1]
