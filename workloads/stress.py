"""Device side of the graph-replay stress run (preset 5): the per-layer KV
pools, q rows and outputs, the fixed-address metadata buffers, and one
captured hipGraph holding every layer's verify attention plus acceptance.

Each step writes that step's lengths, drafts and planted logits into the
fixed buffers (input staging, outside the graph), replays the graph, reads
the acceptance back and grows the contexts by the accepted count plus one.
Inputs are seeded and synthetic: K/V pools and q are N(0,1) bf16 drawn on the
device, logits N(0,1) bf16 with the plan's planted boosts.  Nothing here
computes the method's arithmetic; every step of the path runs in libdsv.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

from .gen import BLOCK_WIDTH, PAGE_SIZE, SEED_BASE, StressPlan, StressStep

BOOST = 10.0


class StressRun:
    def __init__(self, plan: StressPlan, device="cuda:0", num_q_heads: int = 32,
                 num_kv_heads: int = 8, head_dim: int = 128):
        import torch

        import paper_2609_37532_amd as dsv

        self.torch, self.dsv = torch, dsv
        self.plan = plan
        self.dev = torch.device(device)
        self.hq, self.hkv, self.d = num_q_heads, num_kv_heads, head_dim
        L, B, cap, V = plan.num_layers, plan.B, plan.capacity, plan.vocab
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(SEED_BASE + 5)
        bf = torch.bfloat16
        self.kv = [torch.randn((plan.num_pages, 2, self.hkv, PAGE_SIZE * self.d),
                               generator=self.gen, device=self.dev, dtype=bf)
                   for _ in range(L)]
        self.q = torch.randn((L, cap, self.hq, self.d), generator=self.gen, device=self.dev,
                             dtype=bf)
        self.out = torch.zeros((L, cap, self.hq, self.d), device=self.dev, dtype=bf)
        # fixed-address metadata (Eq. (13): same address and shape every step)
        i32 = torch.int32
        self.cu = torch.zeros(B + 1, dtype=i32, device=self.dev)
        self.ctx = torch.from_numpy(plan.ctx0.copy()).to(self.dev)
        self.pt = torch.from_numpy(plan.page_table).to(self.dev)
        self.draft = torch.zeros(cap, dtype=i32, device=self.dev)
        self.logits = torch.zeros((cap, V), dtype=bf, device=self.dev)
        self.a = torch.zeros(B, dtype=i32, device=self.dev)
        self.nxt = torch.zeros(B, dtype=i32, device=self.dev)
        self.dims = dsv.attn_dims(self.q[0], self.kv[0], self.pt, max_kv_len=plan.max_kv_len,
                                  scale=1.0 / math.sqrt(self.d))
        self.ws_attn = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(self.dims), self.dev)
        self.ws_acc = dsv.alloc_workspace(dsv.accept_workspace_bytes(cap, B, V), self.dev)
        self.stream = torch.cuda.Stream(device=self.dev)
        self.ctx_host = plan.ctx0.astype(np.int64).copy()
        self.graph = None

    # ------------------------------------------------------------ one step
    def _enqueue(self):
        s = self.stream
        for layer in range(self.plan.num_layers):
            self.dsv.verify_attn(self.q[layer], self.cu, self.kv[layer], self.pt, self.ctx,
                                 self.out[layer], dims=self.dims, workspace=self.ws_attn,
                                 stream=s)
        self.dsv.accept(self.logits, self.cu, self.draft, self.a, self.nxt,
                        workspace=self.ws_acc, stream=s)

    def stage(self, st: StressStep):
        """Input staging: this step's metadata and logits into the fixed
        buffers (and the grown contexts), then wait for the copies."""
        torch = self.torch
        if int((self.ctx_host + st.qlens).max()) > self.plan.max_kv_len:
            raise RuntimeError("context outgrew the plan")
        self.ctx_step = self.ctx_host.copy()  # the contexts this step reads
        self.cu.copy_(torch.from_numpy(st.cu_qlens))
        self.draft.copy_(torch.from_numpy(st.draft_tokens))
        self.ctx.copy_(torch.from_numpy(self.ctx_host.astype(np.int32)))
        self.logits.normal_(generator=self.gen)
        rows = torch.from_numpy(st.boost_rows).to(self.dev)
        toks = torch.from_numpy(st.boost_tokens).to(self.dev)
        self.logits.index_put_((rows, toks), torch.full_like(rows, 0, dtype=self.logits.dtype)
                               + BOOST, accumulate=True)
        torch.cuda.synchronize(self.dev)

    def capture(self):
        """Eager run once, then capture the whole step as one graph."""
        self._enqueue()
        self.torch.cuda.synchronize(self.dev)
        self.graph = self.dsv.Graph().capture(self._enqueue, self.stream)

    def replay(self):
        self.graph.replay(self.stream)

    def finish(self, st: StressStep):
        """Read this step's acceptance and grow the contexts (state commit)."""
        self.torch.cuda.synchronize(self.dev)
        a = self.a.cpu().numpy()
        nxt = self.nxt.cpu().numpy()
        live = st.qlens > 0
        self.ctx_host[live] += a[live].astype(np.int64) + 1
        return a, nxt

    def close(self):
        if self.graph is not None:
            self.graph.close()
            self.graph = None

    # ------------------------------------------------------------ checking
    def gather_request_inputs(self, layer: int, reqs, st: StressStep):
        """Host copies of what requests ``reqs`` read in ``layer`` this step,
        repacked as a small batch: q rows, their pages (renumbered), page
        table, contexts, offsets.  For an independent check of their rows."""
        torch = self.torch
        ks = [int(st.qlens[i]) for i in reqs]
        cu = np.zeros(len(reqs) + 1, np.int32)
        cu[1:] = np.cumsum(ks)
        q_rows, pages, pt_rows = [], [], []
        for n, i in enumerate(reqs):
            o = int(st.cu_qlens[i])
            q_rows.append(self.q[layer, o:o + ks[n]])
            keys = int(self.ctx_step[i]) + ks[n]
            npg = -(-keys // PAGE_SIZE)
            ids = self.plan.page_table[i, :npg]
            base = sum(len(p) for p in pages)
            pages.append(ids)
            pt_rows.append(np.arange(base, base + npg, dtype=np.int32))
        all_ids = np.concatenate(pages)
        kv = self.kv[layer][torch.from_numpy(all_ids.astype(np.int64)).to(self.dev)]
        q = torch.cat(q_rows).contiguous()
        P = max(len(r) for r in pt_rows)
        pt = np.full((len(reqs), P), -1, np.int32)
        for n, r in enumerate(pt_rows):
            pt[n, :len(r)] = r
        as_bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        ctx = np.asarray([int(self.ctx_step[i]) for i in reqs], np.int32)
        out_rows = torch.cat([self.out[layer, int(st.cu_qlens[i]):int(st.cu_qlens[i]) + ks[n]]
                              for n, i in enumerate(reqs)])
        return dict(q=as_bits(q), cu_qlens=cu, kv_pages=as_bits(kv), page_table=pt,
                    ctx_lens=ctx, out_bits=as_bits(out_rows))
