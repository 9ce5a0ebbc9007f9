"""Seeded synthetic workloads shaped like the paper's verify step.

The paper evaluates Qwen3-8B / Qwen3-4B targets with a W = 16 block (one
anchor + 15 DFlash candidates, Sec. II) at concurrency 8-32 (Sec. IV-A).
Weights, drafters and datasets are not used: every tensor here is drawn from
a seeded ``numpy.random.Generator`` (PCG64), with the shapes of those models'
attention layers (32 query / 8 KV heads, head_dim 128, vocabulary 151,936)
and length distributions from a geometric acceptance model.

Draw order inside one preset (fixed, so a seed pins every byte):
  1. verify lengths (if sampled), 2. context lengths (if sampled),
  3. physical page permutation, 4. q values, 5. KV pool values,
  6. acceptance: draft tokens, planted accept lengths, rejection tokens,
     logit noise.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

SEED_BASE = 20260901
BF16_NAN = np.uint16(0x7FC0)
PAGE_SIZE = 16
BLOCK_WIDTH = 16  # W: anchor + 15 candidates


# --------------------------------------------------------------------------
# bf16 storage helpers (format conversion of inputs, not method arithmetic)
# --------------------------------------------------------------------------
def bf16_bits(x) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, scale: float = 1.0,
                 chunk: int = 1 << 24) -> np.ndarray:
    """N(0, scale^2) draws stored as bf16, generated in chunks to bound memory."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = rng.standard_normal(e - s, dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        out[s:e] = bf16_bits(x)
    return out.reshape(shape)


# --------------------------------------------------------------------------
# KV page layout of the library contract (where slot s, dim c of a tile lives)
# --------------------------------------------------------------------------
def k_tile_offset(slot, dim, page_size: int = PAGE_SIZE):
    """Element offset of (slot, dim) inside a K tile: 8-wide dim chunks."""
    slot = np.asarray(slot)
    dim = np.asarray(dim)
    return ((dim // 8) * page_size + slot) * 8 + dim % 8


def v_tile_offset(slot, dim, page_size: int = PAGE_SIZE):
    """Element offset of (slot, dim) inside a V tile: dim-major."""
    slot = np.asarray(slot)
    dim = np.asarray(dim)
    return dim * page_size + slot


# --------------------------------------------------------------------------
# lengths and offsets
# --------------------------------------------------------------------------
def verify_lengths(rng: np.random.Generator, num_reqs: int, capacity: int,
                   p: float = 0.25, width: int = BLOCK_WIDTH) -> np.ndarray:
    """Per-request verify lengths: anchor + truncated geometric prefix.

    k_i = min(G_i, W) with G_i ~ Geometric(p) on {1, 2, ...}, i.e.
    1 + min(G_i - 1, W - 1).  Only if the total exceeds ``capacity``: scale
    proportionally (floor, at least 1), then decrement the largest (lowest
    index first) until the total fits.
    """
    g = rng.geometric(p, size=num_reqs)
    k = np.minimum(g, width).astype(np.int64)
    total = int(k.sum())
    if total > capacity:
        if capacity < num_reqs:
            raise ValueError("capacity below one row per request")
        k = np.maximum(1, (k * capacity) // total)
        while int(k.sum()) > capacity:
            k[int(np.argmax(k))] -= 1
    return k.astype(np.int32)


def cu_from_lengths(lengths: Sequence[int]) -> np.ndarray:
    """Packed row offsets: (0, k_0, k_0+k_1, ...) as int32 [B+1]."""
    k = np.asarray(lengths, dtype=np.int64)
    cu = np.zeros(k.shape[0] + 1, dtype=np.int64)
    cu[1:] = np.cumsum(k)
    return cu.astype(np.int32)


# --------------------------------------------------------------------------
# attention inputs
# --------------------------------------------------------------------------
@dataclass
class AttnInputs:
    q: np.ndarray            # uint16 [capacity, Hq, D]
    cu_qlens: np.ndarray     # int32 [B+1]
    kv_pages: np.ndarray     # uint16 [num_pages, 2, Hkv, page*D]
    page_table: np.ndarray   # int32 [B, P_max]; -1 beyond a request's pages
    ctx_lens: np.ndarray     # int32 [B]
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    max_kv_len: int
    scale: float
    meta: dict = field(default_factory=dict)

    @property
    def num_reqs(self) -> int:
        return int(self.ctx_lens.shape[0])

    @property
    def capacity(self) -> int:
        return int(self.q.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.kv_pages.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def qlens(self) -> np.ndarray:
        return np.diff(self.cu_qlens).astype(np.int32)

    def dims(self) -> dict:
        return dict(num_reqs=self.num_reqs, capacity=self.capacity,
                    num_q_heads=self.num_q_heads, num_kv_heads=self.num_kv_heads,
                    head_dim=self.head_dim, page_size=self.page_size,
                    max_pages_per_req=self.max_pages, num_pages=self.num_pages,
                    max_kv_len=self.max_kv_len, scale=self.scale)

    def oracle_kwargs(self) -> dict:
        return dict(num_q_heads=self.num_q_heads, num_kv_heads=self.num_kv_heads,
                    head_dim=self.head_dim, page_size=self.page_size,
                    scale=self.scale)


def make_attn_inputs(rng: np.random.Generator, *, ctx_lens, qlens, capacity: int,
                     num_q_heads: int, num_kv_heads: int, head_dim: int,
                     page_size: int = PAGE_SIZE, max_kv_len: Optional[int] = None,
                     scale: Optional[float] = None, permute_pages: bool = True,
                     spare_pages: int = 0, poison: bool = True,
                     q_scale: float = 1.0) -> AttnInputs:
    """Paged attention inputs with Q, K, V ~ N(0,1) in bf16.

    Request i owns ceil((ctx_i + k_i) / page) pages; physical ids are a random
    permutation of the pool when ``permute_pages``.  With ``poison``, every
    element that verify attention must NOT read is set to bf16 NaN: tail rows
    of q, slots at or beyond ctx_i + k_i in a request's last page, and
    ``spare_pages`` extra pool pages nobody references.
    """
    ctx = np.asarray(ctx_lens, dtype=np.int32)
    k = np.asarray(qlens, dtype=np.int32)
    B = ctx.shape[0]
    assert k.shape[0] == B
    cu = cu_from_lengths(k)
    if int(cu[-1]) > capacity:
        raise ValueError("packed rows exceed capacity")
    keys = ctx.astype(np.int64) + k
    if max_kv_len is None:
        max_kv_len = int(max(1, keys.max()))
    if int(keys.max()) > max_kv_len:
        raise ValueError("ctx + k exceeds max_kv_len")
    max_pages = -(-max_kv_len // page_size)
    need = [(-(-int(L) // page_size)) if kk > 0 else 0 for L, kk in zip(keys, k)]
    used = int(sum(need))
    num_pages = max(1, used + spare_pages)
    ids = rng.permutation(num_pages).astype(np.int32) if permute_pages else \
        np.arange(num_pages, dtype=np.int32)
    page_table = np.full((B, max_pages), -1, dtype=np.int32)
    pos = 0
    for i in range(B):
        page_table[i, :need[i]] = ids[pos:pos + need[i]]
        pos += need[i]

    q = _normal_bf16(rng, (capacity, num_q_heads, head_dim), q_scale)
    kv = _normal_bf16(rng, (num_pages, 2, num_kv_heads, page_size * head_dim))

    if poison:
        q[int(cu[-1]):] = BF16_NAN
        for p in ids[used:]:
            kv[p] = BF16_NAN
        dims = np.arange(head_dim)
        for i in range(B):
            if need[i] == 0:
                continue
            last = page_table[i, need[i] - 1]
            first_dead = int(keys[i]) - (need[i] - 1) * page_size
            for s in range(first_dead, page_size):
                kv[last, 0, :, k_tile_offset(s, dims, page_size)] = BF16_NAN
                kv[last, 1, :, v_tile_offset(s, dims, page_size)] = BF16_NAN
    if scale is None:
        scale = 1.0 / float(np.sqrt(head_dim))
    return AttnInputs(q=q, cu_qlens=cu, kv_pages=kv, page_table=page_table,
                      ctx_lens=ctx, num_q_heads=num_q_heads,
                      num_kv_heads=num_kv_heads, head_dim=head_dim,
                      page_size=page_size, max_kv_len=int(max_kv_len),
                      scale=float(scale))


def repack(inp: AttnInputs, order: Sequence[int], capacity: Optional[int] = None,
           gaps: Optional[Sequence[int]] = None, poison: bool = True) -> AttnInputs:
    """The same requests packed differently (input rearrangement only).

    Request ``order[n]`` of ``inp`` becomes the n-th live request; its q rows,
    context length and page-table row move with it and the KV pool is shared
    unchanged.  ``gaps[n]`` sentinel requests (k = 0) are inserted before it;
    ``gaps`` may carry one extra trailing entry.  ``meta['moves']`` lists
    (old_request, new_request, old_row, new_row, k) for the live requests.
    """
    order = list(order)
    gaps = list(gaps) if gaps is not None else []
    gaps += [0] * (len(order) + 1 - len(gaps))
    entries = []
    for n, i in enumerate(order):
        entries += [None] * gaps[n]
        entries.append(i)
    entries += [None] * gaps[len(order)]
    old_cu = inp.cu_qlens
    new_k = [0 if e is None else int(old_cu[e + 1] - old_cu[e]) for e in entries]
    cu = cu_from_lengths(new_k)
    cap = capacity if capacity is not None else max(1, int(cu[-1]))
    if int(cu[-1]) > cap:
        raise ValueError("packed rows exceed capacity")
    q = np.full((cap, inp.num_q_heads, inp.head_dim),
                BF16_NAN if poison else 0, dtype=np.uint16)
    page_table = np.full((len(entries), inp.max_pages), -1, dtype=np.int32)
    ctx = np.zeros(len(entries), dtype=np.int32)
    moves = []
    for r, e in enumerate(entries):
        if e is None:
            continue
        kk = new_k[r]
        o_old, o_new = int(old_cu[e]), int(cu[r])
        q[o_new:o_new + kk] = inp.q[o_old:o_old + kk]
        page_table[r] = inp.page_table[e]
        ctx[r] = inp.ctx_lens[e]
        moves.append((e, r, o_old, o_new, kk))
    out = AttnInputs(q=q, cu_qlens=cu, kv_pages=inp.kv_pages, page_table=page_table,
                     ctx_lens=ctx, num_q_heads=inp.num_q_heads,
                     num_kv_heads=inp.num_kv_heads, head_dim=inp.head_dim,
                     page_size=inp.page_size, max_kv_len=inp.max_kv_len,
                     scale=inp.scale)
    out.meta["moves"] = moves
    return out


# --------------------------------------------------------------------------
# acceptance inputs (planted scheme)
# --------------------------------------------------------------------------
@dataclass
class AcceptInputs:
    logits: np.ndarray          # float32 [cap, V] or uint16 bf16 bits [cap, V]
    dtype: str                  # 'f32' | 'bf16'
    cu_qlens: np.ndarray        # int32 [B+1]
    draft_tokens: np.ndarray    # int32 [cap]
    planted_accept_len: np.ndarray  # int32 [B]
    planted_next: np.ndarray        # int32 [B]

    @property
    def vocab(self) -> int:
        return int(self.logits.shape[1])

    @property
    def capacity(self) -> int:
        return int(self.logits.shape[0])

    @property
    def num_reqs(self) -> int:
        return int(self.cu_qlens.shape[0] - 1)


def make_accept_inputs(rng: np.random.Generator, *, cu_qlens, capacity: int,
                       vocab: int, dtype: str = "f32", p_accept: float = 0.3,
                       boost: float = 10.0, poison: bool = True) -> AcceptInputs:
    """Planted acceptance: logits ~ N(0,1); for request i (o = cu[i], k = k_i)
    draw a_i = min(G - 1, k - 1), G ~ Geometric(p_accept); add ``boost`` to
    the logit of draft_tokens[o+j+1] at row o+j for j < a_i, and to a token
    x_i at row o+a_i, with x_i != draft_tokens[o+a_i+1] when a_i < k-1.  By
    construction the greedy verifier accepts a_i candidates and emits x_i
    (barring a noise draw that beats the boosted one).  Draft tokens are
    uniform in [0, vocab).  Tail rows are NaN when ``poison``.
    """
    cu = np.asarray(cu_qlens, dtype=np.int32)
    B = cu.shape[0] - 1
    draft = rng.integers(0, vocab, size=capacity, dtype=np.int64).astype(np.int32)
    a = np.zeros(B, dtype=np.int32)
    nxt = np.full(B, -1, dtype=np.int32)
    for i in range(B):
        k = int(cu[i + 1] - cu[i])
        if k == 0:
            continue
        g = int(rng.geometric(p_accept))
        a[i] = min(g - 1, k - 1)
    for i in range(B):
        o, k = int(cu[i]), int(cu[i + 1] - cu[i])
        if k == 0:
            continue
        if a[i] < k - 1:
            avoid = int(draft[o + a[i] + 1])
            x = (avoid + 1 + int(rng.integers(0, vocab - 1))) % vocab
        else:
            x = int(rng.integers(0, vocab))
        nxt[i] = x
    logits = np.empty((capacity, vocab), dtype=np.float32)
    for r0 in range(0, capacity, 64):
        r1 = min(capacity, r0 + 64)
        logits[r0:r1] = rng.standard_normal((r1 - r0, vocab), dtype=np.float32)
    for i in range(B):
        o, k = int(cu[i]), int(cu[i + 1] - cu[i])
        if k == 0:
            continue
        for j in range(int(a[i])):
            logits[o + j, draft[o + j + 1]] += np.float32(boost)
        logits[o + int(a[i]), nxt[i]] += np.float32(boost)
    if poison:
        logits[int(cu[-1]):] = np.nan
    if dtype == "bf16":
        stored = bf16_bits(logits)
        if poison:
            stored[int(cu[-1]):] = BF16_NAN
    elif dtype == "f32":
        stored = logits
    else:
        raise ValueError(dtype)
    return AcceptInputs(logits=stored, dtype=dtype, cu_qlens=cu, draft_tokens=draft,
                        planted_accept_len=a, planted_next=nxt)


# --------------------------------------------------------------------------
# the workload presets
# --------------------------------------------------------------------------
CONFIGS = {
    1: dict(name="tiny", num_reqs=2, num_q_heads=4, num_kv_heads=1, head_dim=64,
            capacity=32, ctx=[37, 100], qlens=[16, 5], vocab=1000,
            accept_dtype="f32", p_accept=0.3),
    2: dict(name="qwen3-4b-shape unpacked", num_reqs=8, num_q_heads=32,
            num_kv_heads=8, head_dim=128, capacity=128, ctx_range=(256, 2048),
            qlens="full"),
    3: dict(name="qwen3-8b-shape packed", num_reqs=16, num_q_heads=32,
            num_kv_heads=8, head_dim=128, capacity=128, ctx_range=(512, 4096),
            qlens="geometric"),
    4: dict(name="qwen3-8b-shape verify+accept c32", num_reqs=32, num_q_heads=32,
            num_kv_heads=8, head_dim=128, capacity=256, ctx_range=(1024, 8192),
            qlens="geometric", vocab=151936, accept_dtype="bf16", p_accept=0.3),
}


def config_rng(index: int) -> np.random.Generator:
    return np.random.default_rng(SEED_BASE + index)


def config_attn_inputs(index: int, rng: Optional[np.random.Generator] = None,
                       poison: bool = True) -> AttnInputs:
    """Attention inputs of preset ``index`` (draws 1-5 of the fixed order)."""
    c = CONFIGS[index]
    rng = config_rng(index) if rng is None else rng
    B = c["num_reqs"]
    if c.get("qlens") == "full":
        k = np.full(B, BLOCK_WIDTH, dtype=np.int32)
    elif c.get("qlens") == "geometric":
        k = verify_lengths(rng, B, c["capacity"], p=0.25)
    else:
        k = np.asarray(c["qlens"], dtype=np.int32)
    if "ctx_range" in c:
        lo, hi = c["ctx_range"]
        ctx = rng.integers(lo, hi + 1, size=B).astype(np.int32)
        max_kv_len = hi + BLOCK_WIDTH
    else:
        ctx = np.asarray(c["ctx"], dtype=np.int32)
        max_kv_len = int((ctx + k).max())
    inp = make_attn_inputs(rng, ctx_lens=ctx, qlens=k, capacity=c["capacity"],
                           num_q_heads=c["num_q_heads"],
                           num_kv_heads=c["num_kv_heads"], head_dim=c["head_dim"],
                           max_kv_len=max_kv_len, poison=poison)
    inp.meta["config"] = index
    inp.meta["name"] = c["name"]
    return inp


def config_accept_inputs(index: int, cu_qlens, rng: np.random.Generator,
                         poison: bool = True) -> AcceptInputs:
    """Acceptance inputs of preset ``index`` (draw 6), after its attention draws."""
    c = CONFIGS[index]
    return make_accept_inputs(rng, cu_qlens=cu_qlens, capacity=c["capacity"],
                              vocab=c["vocab"], dtype=c["accept_dtype"],
                              p_accept=c["p_accept"], poison=poison)


# --------------------------------------------------------------------------
# config 5: graph-replay stress (host side of the plan)
# --------------------------------------------------------------------------
CONFIGS[5] = dict(name="graph-replay stress", num_layers=36, num_reqs=32, num_q_heads=32,
                  num_kv_heads=8, head_dim=128, capacity=256, ctx_range=(512, 4096),
                  steps=100, vocab=151936, accept_dtype="bf16", p_accept=0.3)


def plant_boosts(rng: np.random.Generator, cu_qlens, draft_tokens, vocab: int,
                 p_accept: float):
    """The planted acceptance of :func:`make_accept_inputs` for drafts that
    are already given, as a list of logit boosts to add on the device: per
    live request (o = cu[i], k = k_i) a_i = min(G - 1, k - 1) with
    G ~ Geometric(p_accept); rows o+j (j < a_i) boost draft[o+j+1]; row o+a_i
    boosts a token x_i != draft[o+a_i+1] (any token when a_i = k-1).
    Returns (accept_len, next_token, boost_rows, boost_tokens)."""
    cu = np.asarray(cu_qlens, dtype=np.int64)
    draft = np.asarray(draft_tokens)
    B = cu.shape[0] - 1
    a = np.zeros(B, dtype=np.int32)
    nxt = np.full(B, -1, dtype=np.int32)
    rows, toks = [], []
    for i in range(B):
        o, kk = int(cu[i]), int(cu[i + 1] - cu[i])
        if kk == 0:
            continue
        a[i] = min(int(rng.geometric(p_accept)) - 1, kk - 1)
        for j in range(int(a[i])):
            rows.append(o + j)
            toks.append(int(draft[o + j + 1]))
        if a[i] < kk - 1:
            avoid = int(draft[o + a[i] + 1])
            x = (avoid + 1 + int(rng.integers(0, vocab - 1))) % vocab
        else:
            x = int(rng.integers(0, vocab))
        nxt[i] = x
        rows.append(o + int(a[i]))
        toks.append(x)
    return a, nxt, np.asarray(rows, np.int64), np.asarray(toks, np.int64)


@dataclass
class StressStep:
    """One step's inputs: verify lengths, packed offsets, packed draft tokens,
    and the planted acceptance (accepted count and successor per request)
    with the (row, token) logits it boosts."""
    qlens: np.ndarray
    cu_qlens: np.ndarray
    draft_tokens: np.ndarray
    planted_accept_len: np.ndarray
    planted_next: np.ndarray
    boost_rows: np.ndarray
    boost_tokens: np.ndarray


class StressPlan:
    """Seeded host plan of the stress run: initial contexts, one page table
    (logical page -> physical page, a random permutation of the pool, shared
    by every layer's pool) sized for the longest context the run can reach,
    and per step the lengths, drafts and planted acceptances.  Contexts grow
    by the accepted count plus one after every step."""

    def __init__(self, steps: Optional[int] = None, num_layers: Optional[int] = None,
                 num_reqs: Optional[int] = None, rng: Optional[np.random.Generator] = None):
        c = CONFIGS[5]
        self.rng = config_rng(5) if rng is None else rng
        self.steps = c["steps"] if steps is None else steps
        self.num_layers = c["num_layers"] if num_layers is None else num_layers
        self.B = c["num_reqs"] if num_reqs is None else num_reqs
        self.capacity = c["capacity"]
        self.vocab = c["vocab"]
        self.p_accept = c["p_accept"]
        lo, hi = c["ctx_range"]
        self.ctx0 = self.rng.integers(lo, hi + 1, size=self.B).astype(np.int32)
        # the longest context: start + steps * (up to W per step) + one block
        self.max_kv_len = int(hi + (self.steps + 1) * BLOCK_WIDTH)
        self.max_pages = -(-self.max_kv_len // PAGE_SIZE)
        self.num_pages = self.B * self.max_pages
        self.page_table = self.rng.permutation(self.num_pages).astype(np.int32).reshape(
            self.B, self.max_pages)

    def draw_step(self) -> StressStep:
        B, cap, V = self.B, self.capacity, self.vocab
        k = verify_lengths(self.rng, B, cap, p=0.25)
        cu = cu_from_lengths(k)
        draft = self.rng.integers(0, V, size=cap, dtype=np.int64).astype(np.int32)
        a, nxt, rows, toks = plant_boosts(self.rng, cu, draft, V, self.p_accept)
        return StressStep(qlens=k, cu_qlens=cu, draft_tokens=draft, planted_accept_len=a,
                          planted_next=nxt, boost_rows=rows, boost_tokens=toks)


# --------------------------------------------------------------------- DVL
@dataclass
class DvlInputs:
    """Inputs of the DVL allocator and packer for one bucket of ``n_bs``
    request slots, the first ``n_live`` live.

    ``pred_logits`` float32 [n_bs, W-1]: synthetic predictor outputs.  Each
    live request draws a per-position acceptance rate r ~ U(rate_range)
    (default U(0.85, 0.995), which puts the mean estimate near the W/2 budget
    per request, so both growing and shrinking occur); its
    logit at draft position j is log(r^j / (1 - r^j)) plus N(0, noise) noise
    (default 0.5),
    so the sigmoid profile decays like the geometric acceptance model with
    some non-monotone noise for the running minimum to remove.  With
    ``ties`` the logits are rounded to a 0.5 grid so that equal scores across
    requests are common.  Sentinel rows hold NaN (never read).
    ``tokens`` [n_bs, W]: the anchor plus W-1 drafts, uniform over the
    vocabulary.  ``positions`` [n_bs, W]: ctx_i + j.  ``kv_refs`` [n_bs, W]:
    flat cache slots (page * 16 + slot) of those positions under a random
    page assignment."""
    pred_logits: np.ndarray
    n_live: int
    tokens: np.ndarray
    positions: np.ndarray
    kv_refs: np.ndarray
    width: int


def make_dvl_inputs(rng: np.random.Generator, *, n_bs: int, n_live: int,
                    width: int = BLOCK_WIDTH, vocab: int = 151936,
                    ctx_range=(256, 4096), noise: float = 0.5,
                    rate_range=(0.85, 0.995), ties: bool = False) -> DvlInputs:
    if not (0 <= n_live <= n_bs):
        raise ValueError("need 0 <= n_live <= n_bs")
    w = width
    rate = rng.uniform(rate_range[0], rate_range[1], size=(n_bs, 1))
    j = np.arange(1, w, dtype=np.float64)[None, :]
    p = np.clip(rate ** j, 1e-6, 1 - 1e-6)
    logits = np.log(p / (1 - p)) + rng.normal(0.0, noise, size=(n_bs, w - 1))
    if ties:
        logits = np.round(logits * 2.0) / 2.0
    logits = logits.astype(np.float32)
    logits[n_live:] = np.nan
    tokens = rng.integers(0, vocab, size=(n_bs, w), dtype=np.int64).astype(np.int32)
    ctx = rng.integers(ctx_range[0], ctx_range[1] + 1, size=(n_bs, 1))
    positions = (ctx + np.arange(w)[None, :]).astype(np.int32)
    pages_per_req = -(-(ctx_range[1] + w) // PAGE_SIZE)
    page_of = rng.permutation(n_bs * pages_per_req).reshape(n_bs, pages_per_req)
    kv_refs = np.take_along_axis(page_of, positions // PAGE_SIZE, axis=1) * PAGE_SIZE \
        + positions % PAGE_SIZE
    return DvlInputs(pred_logits=logits, n_live=int(n_live), tokens=tokens,
                     positions=positions, kv_refs=kv_refs.astype(np.int32), width=w)


# -------------------------------------------------------------- predictor
PREDICTOR_DIMS = (1735, 64, 15)  # features, hidden units, draft positions


@dataclass
class PredictorInputs:
    """Acceptance-predictor inputs for a bucket of ``n_bs`` slots (first
    ``n_live`` live) and random weights of the 1735-64-15 shape.

    Features follow the paper's layout: per draft position (15) the top
    logit ~ N(14, 3), its 15 gaps to ranks 2..16 (sorted |N(0, 2)| partial
    sums), the top token's log-probability -|N(0, 1)| and the entropy
    U(0, 4) (270 values); 960 hidden-state projections ~ N(0, 1); 480 logit
    projections ~ N(0, 1); a 25-value batch context with the live count
    first, 1 in the fourth entry and zeros elsewhere.  Weights: W1 ~ N(0,
    2/1735), b1 ~ N(0, 0.1), W2 ~ N(0, 1/64), b2 ~ N(1, 0.5) (the trained
    weights are not available).  Sentinel feature rows are NaN."""
    features: np.ndarray
    n_live: int
    w1: np.ndarray
    b1: np.ndarray
    w2: np.ndarray
    b2: np.ndarray


def make_predictor_inputs(rng: np.random.Generator, *, n_bs: int, n_live: int,
                          dims=PREDICTOR_DIMS) -> PredictorInputs:
    in_dim, hidden, out_dim = dims
    f = np.zeros((n_bs, in_dim), np.float32)
    pos = out_dim
    if in_dim == 1735:
        conf = np.zeros((n_bs, pos, 18), np.float32)
        conf[:, :, 0] = rng.normal(14.0, 3.0, size=(n_bs, pos))
        conf[:, :, 1:16] = np.cumsum(np.abs(rng.normal(0, 2.0, size=(n_bs, pos, 15))), axis=2)
        conf[:, :, 16] = -np.abs(rng.normal(0, 1.0, size=(n_bs, pos)))
        conf[:, :, 17] = rng.uniform(0, 4.0, size=(n_bs, pos))
        f[:, :270] = conf.reshape(n_bs, 270)
        f[:, 270:1710] = rng.normal(0, 1.0, size=(n_bs, 1440))
        f[:, 1710] = n_live
        f[:, 1713] = 1.0
    else:
        f[:] = rng.normal(0, 1.0, size=(n_bs, in_dim))
    f[n_live:] = np.nan
    w1 = rng.normal(0, np.sqrt(2.0 / in_dim), size=(in_dim, hidden)).astype(np.float32)
    b1 = rng.normal(0, 0.1, size=hidden).astype(np.float32)
    w2 = rng.normal(0, np.sqrt(1.0 / hidden), size=(hidden, out_dim)).astype(np.float32)
    b2 = rng.normal(1.0, 0.5, size=out_dim).astype(np.float32)
    return PredictorInputs(features=f, n_live=int(n_live), w1=w1, b1=b1, w2=w2, b2=b2)
