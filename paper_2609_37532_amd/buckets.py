"""Multi-bucket capture set: fixed-address buffers and captured graphs for a
finite set of request-bucket sizes (Sec. III-D, Alg. 2, Eqs. (13)-(15)).

For every bucket size N_bs the set allocates, once, every buffer the decision
step and the verify step touch (so their addresses and shapes never change,
Eq. (13)), and captures two graphs:

* the decision graph: the acceptance predictor (``predictor_forward``, when
  weights are given) and DVL allocation and packing (``dvl_allocate_pack``),
  which writes the lengths, offsets and packed rows into the bucket's buffers;
* the verify graph: verify attention for every layer, then greedy
  acceptance, reading the offsets and packed tokens the decision graph wrote.

Each step picks the smallest bucket that holds the live requests (Eq. (14)),
stages that step's inputs into the bucket's buffers, and replays the two
graphs.  Slots past the live count are sentinels with length 0, so the
bucket's packed capacity stays 8 N_bs (W N_bs / 2) whatever the live count
(Eq. (15)).  Host code here only allocates, copies inputs in and launches:
every step of the path runs in libdsv's kernels.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence

from . import _lib


def select_bucket(buckets: Iterable[int], n: int) -> int:
    """Eq. (14): the smallest captured bucket size that is at least ``n``."""
    fits = [b for b in buckets if b >= n]
    if n < 1 or not fits:
        raise ValueError("no bucket holds %d live requests (buckets %s)" % (n, sorted(buckets)))
    return min(fits)


class Bucket:
    """Buffers and graphs of one bucket size ``n_bs``."""

    def __init__(self, n_bs: int, *, kv_pools: Sequence, max_pages: int, max_kv_len: int,
                 num_q_heads: int, head_dim: int, vocab: int, width: int, device,
                 ws_attn=None, ws_acc=None, predictor: Optional[dict] = None, ws_pred=None):
        import torch

        self.torch = torch
        self.n_bs = n_bs
        self.width = w = width
        self.capacity = cap = w * n_bs // 2
        self.kv_pools = list(kv_pools)
        L = len(self.kv_pools)
        i32, f32, bf = torch.int32, torch.float32, torch.bfloat16
        z = lambda *shape, dtype=i32: torch.zeros(shape, dtype=dtype, device=device)
        # decision step: inputs staged each step, outputs written by the graph
        self.pred_logits = z(n_bs, w - 1, dtype=f32)
        self.predictor = predictor
        self.features = None
        if predictor is not None:
            in_dim = predictor["w1"].shape[0]
            if predictor["w2"].shape[1] != w - 1:
                raise ValueError("the predictor must output W-1 logits")
            self.features = z(n_bs, in_dim, dtype=f32)
            need = _lib.predictor_workspace_bytes(n_bs, in_dim)
            if ws_pred is not None and ws_pred.numel() < need:
                raise ValueError("shared workspace too small")
            self.ws_pred = ws_pred if ws_pred is not None else _lib.alloc_workspace(need, device)
        self.num_live = z(1)
        self.tokens, self.positions, self.kv_refs = z(n_bs, w), z(n_bs, w), z(n_bs, w)
        self.k, self.cu = z(n_bs), z(n_bs + 1)
        self.packed_tokens, self.packed_positions, self.packed_kv_refs = z(cap), z(cap), z(cap)
        # verify step: request state staged each step; q and logits stand in
        # for the target model's activations at the packed rows
        self.ctx_lens = z(n_bs)
        self.page_table = z(n_bs, max_pages)
        self.q = z(L, cap, num_q_heads, head_dim, dtype=bf)
        self.out = z(L, cap, num_q_heads, head_dim, dtype=bf)
        self.logits = z(cap, vocab, dtype=bf)
        self.accept_len, self.next_token = z(n_bs), z(n_bs)
        self.dims = _lib.attn_dims(self.q[0], self.kv_pools[0], self.page_table,
                                   max_kv_len=max_kv_len, scale=1.0 / math.sqrt(head_dim))
        # workspaces may be shared by buckets: one step replays one bucket,
        # and the kernels leave a workspace ready for the next call
        need_attn = _lib.verify_attn_workspace_bytes(self.dims)
        need_acc = _lib.accept_workspace_bytes(cap, n_bs, vocab)
        for ws, need in ((ws_attn, need_attn), (ws_acc, need_acc)):
            if ws is not None and ws.numel() < need:
                raise ValueError("shared workspace too small")
        self.ws_attn = ws_attn if ws_attn is not None else _lib.alloc_workspace(need_attn, device)
        self.ws_acc = ws_acc if ws_acc is not None else _lib.alloc_workspace(need_acc, device)
        self.graph_dec: Optional[_lib.Graph] = None
        self.graph_ver: Optional[_lib.Graph] = None
        self.graph_bytes = {"decision": 0, "verify": 0}

    # -------------------------------------------------------------- enqueue
    def enqueue_decision(self, stream) -> None:
        if self.predictor is not None:
            p = self.predictor
            _lib.predictor_forward(self.features, self.num_live, p["w1"], p["b1"], p["w2"],
                                   p["b2"], self.pred_logits, workspace=self.ws_pred,
                                   stream=stream)
        _lib.dvl_allocate_pack(self.pred_logits, self.num_live, self.tokens, self.positions,
                               self.kv_refs, self.k, self.cu, self.packed_tokens,
                               self.packed_positions, self.packed_kv_refs, stream=stream)

    def enqueue_verify(self, stream) -> None:
        for layer, kv in enumerate(self.kv_pools):
            _lib.verify_attn(self.q[layer], self.cu, kv, self.page_table, self.ctx_lens,
                             self.out[layer], dims=self.dims, workspace=self.ws_attn,
                             stream=stream)
        _lib.accept(self.logits, self.cu, self.packed_tokens, self.accept_len, self.next_token,
                    workspace=self.ws_acc, stream=stream)

    def capture(self, stream) -> None:
        """Run both steps once eagerly (all slots sentinels), then capture
        each as a graph, recording the device memory the instantiation took."""
        torch = self.torch
        self.num_live.zero_()
        torch.cuda.synchronize()
        self.enqueue_decision(stream)
        self.enqueue_verify(stream)
        torch.cuda.synchronize()
        for name, fn in (("decision", self.enqueue_decision), ("verify", self.enqueue_verify)):
            free0 = torch.cuda.mem_get_info()[0]
            g = _lib.Graph().capture(lambda: fn(stream), stream)
            torch.cuda.synchronize()
            self.graph_bytes[name] = max(0, free0 - torch.cuda.mem_get_info()[0])
            if name == "decision":
                self.graph_dec = g
            else:
                self.graph_ver = g

    # --------------------------------------------------------------- staging
    def stage_decision(self, n_live: int, pred_logits, tokens, positions, kv_refs) -> None:
        """Copy one step's decision inputs for the first ``n_live`` slots
        (host arrays or device tensors of n_live rows); the sentinel rows
        keep whatever they held (they are not used).  With a predictor,
        ``pred_logits`` is the feature matrix [n_live, in_dim] instead (the
        predictor computes the logits inside the graph).  The copies go on
        torch's current stream; the caller has synchronised the previous
        step's replays (Alg. 2 reads its outputs first)."""
        torch = self.torch
        if not 0 <= n_live <= self.n_bs:
            raise ValueError("live count %d outside bucket %d" % (n_live, self.n_bs))
        self.num_live.fill_(n_live)
        first = self.features if self.predictor is not None else self.pred_logits
        for dst, src in ((first, pred_logits), (self.tokens, tokens),
                         (self.positions, positions), (self.kv_refs, kv_refs)):
            if n_live:
                dst[:n_live].copy_(torch.as_tensor(src)[:n_live], non_blocking=False)

    def stage_verify(self, n_live: int, ctx_lens, page_rows) -> None:
        """Copy the live requests' committed context lengths and page-table
        rows (the historyKV gather of Alg. 2); sentinel slots get length 0
        and page 0, which nothing reads."""
        torch = self.torch
        self.ctx_lens.zero_()
        self.page_table.zero_()
        if n_live:
            self.ctx_lens[:n_live].copy_(torch.as_tensor(ctx_lens)[:n_live])
            rows = torch.as_tensor(page_rows)[:n_live]
            self.page_table[:n_live, :rows.shape[1]].copy_(rows)

    # ---------------------------------------------------------------- replay
    def replay_decision(self, stream) -> None:
        """Replay the decision graph on ``stream`` after the staging copies
        enqueued on torch's current stream."""
        stream.wait_stream(self.torch.cuda.current_stream())
        self.graph_dec.replay(stream)

    def replay_verify(self, stream) -> None:
        stream.wait_stream(self.torch.cuda.current_stream())
        self.graph_ver.replay(stream)

    def close(self) -> None:
        for g in (self.graph_dec, self.graph_ver):
            if g is not None:
                g.close()
        self.graph_dec = self.graph_ver = None

    # ---------------------------------------------------------------- memory
    def memory(self) -> Dict[str, int]:
        """Device bytes held by this bucket: decision and verify metadata,
        workspaces, the activation stand-ins (q, out, logits) and the two
        graph instantiations."""
        nb = lambda *ts: int(sum(t.numel() * t.element_size() for t in ts))
        extra = (self.features,) if self.features is not None else ()
        meta = nb(self.pred_logits, self.num_live, self.tokens, self.positions, self.kv_refs,
                  *extra,
                  self.k, self.cu, self.packed_tokens, self.packed_positions,
                  self.packed_kv_refs, self.ctx_lens, self.page_table, self.accept_len,
                  self.next_token)
        return {"n_bs": self.n_bs, "capacity_rows": self.capacity, "metadata_bytes": meta,
                "workspace_bytes": nb(self.ws_attn, self.ws_acc),
                "activation_bytes": nb(self.q, self.out, self.logits),
                "graph_decision_bytes": int(self.graph_bytes["decision"]),
                "graph_verify_bytes": int(self.graph_bytes["verify"])}


class BucketSet:
    """The capture set B of Alg. 2: one :class:`Bucket` per size, sharing the
    per-layer KV pools."""

    def __init__(self, buckets: Iterable[int], *, kv_pools: Sequence, max_pages: int,
                 max_kv_len: int, num_q_heads: int, head_dim: int, vocab: int,
                 width: int = _lib.MAX_QLEN, device=None, predictor: Optional[dict] = None):
        """``predictor``: optional dict of device tensors w1 [in, 64], b1 [64],
        w2 [64, W-1], b2 [W-1]; with it each decision graph runs the predictor
        on staged features before DVL (Alg. 2's Features -> DVL pipeline)."""
        import torch

        sizes = sorted(set(int(b) for b in buckets))
        if not sizes or sizes[0] < 1 or sizes[-1] > _lib.DVL_MAX_REQS:
            raise ValueError("bucket sizes must lie in [1, %d]" % _lib.DVL_MAX_REQS)
        if width % 2 or not 2 <= width <= _lib.MAX_QLEN:
            raise ValueError("block width must be even and in [2, %d]" % _lib.MAX_QLEN)
        dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.sizes: List[int] = sizes
        # one attention and one acceptance workspace, sized for the largest
        # bucket and shared by all of them (a step replays a single bucket)
        big = max(sizes)
        hkv = kv_pools[0].shape[2]
        dims = _lib.AttnDims(num_reqs=big, capacity=width * big // 2, num_q_heads=num_q_heads,
                             num_kv_heads=hkv, head_dim=head_dim, page_size=_lib.PAGE_SIZE,
                             max_pages_per_req=max_pages, num_pages=kv_pools[0].shape[0],
                             max_kv_len=max_kv_len, scale=1.0 / math.sqrt(head_dim))
        need_attn = max(_lib.verify_attn_workspace_bytes(dims), 1)
        need_acc = max(_lib.accept_workspace_bytes(width * b // 2, b, vocab) for b in sizes)
        self.ws_attn = _lib.alloc_workspace(need_attn, dev)
        self.ws_acc = _lib.alloc_workspace(need_acc, dev)
        self.ws_pred = None
        if predictor is not None:
            self.ws_pred = _lib.alloc_workspace(
                _lib.predictor_workspace_bytes(big, predictor["w1"].shape[0]), dev)
        self.buckets: Dict[int, Bucket] = {
            b: Bucket(b, kv_pools=kv_pools, max_pages=max_pages, max_kv_len=max_kv_len,
                      num_q_heads=num_q_heads, head_dim=head_dim, vocab=vocab, width=width,
                      device=dev, ws_attn=self.ws_attn, ws_acc=self.ws_acc,
                      predictor=predictor, ws_pred=self.ws_pred)
            for b in sizes}

    def select(self, n: int) -> int:
        return select_bucket(self.sizes, n)

    def __getitem__(self, n_bs: int) -> Bucket:
        return self.buckets[n_bs]

    def capture(self, stream) -> None:
        for b in self.sizes:
            self.buckets[b].capture(stream)

    def close(self) -> None:
        for b in self.buckets.values():
            b.close()

    def memory(self) -> Dict[str, object]:
        """Per-bucket figures (their workspace entry is the shared pair) and
        the set's totals."""
        per = [self.buckets[b].memory() for b in self.sizes]
        ws = int(self.ws_attn.numel() + self.ws_acc.numel()
                 + (self.ws_pred.numel() if self.ws_pred is not None else 0))
        keys = ("metadata_bytes", "activation_bytes", "graph_decision_bytes",
                "graph_verify_bytes")
        total = {k: int(sum(m[k] for m in per)) for k in keys}
        total["shared_workspace_bytes"] = ws
        total["all_bytes"] = ws + sum(total[k] for k in keys)
        return {"buckets": per, "total": total}
