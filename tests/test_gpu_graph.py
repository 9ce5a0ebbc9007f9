"""Fixed-address workspace + one captured hipGraph replayed across steps
(Alg. 2; Eq. (13): the buffers keep their address and shape, only their
contents change).  Each replay must equal eager calls on the same inputs
(bitwise) and the oracle (attention within tolerance, acceptance exact)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, assert_attn_close, bf16_dev, bf16_host, i32_dev, say
except Exception:  # pragma: no cover
    pass

B, CAP, HQ, HKV, D, VOCAB = 8, 64, 32, 8, 128, 5000
MAX_KV = 3000 + 16
POOL = 8 * ((MAX_KV + 15) // 16) + 4


def step_inputs(seed):
    rng = np.random.default_rng(seed)
    k = W.verify_lengths(rng, B, CAP)
    k[seed % B] = 0  # a sentinel
    # short contexts on even seeds, long ones on odd seeds: with 8 requests
    # and 8 KV heads the short steps fall below the stream-K minimum share
    # and take the small-batch plan, so one captured graph replays both plans
    lo, hi = (0, 600) if seed % 2 == 0 else (2400, 3000)
    ctx = rng.integers(lo, hi, size=B).astype(np.int32)
    keys = ctx.astype(np.int64) + k
    used = int(sum(-(-int(L) // 16) for L, kk in zip(keys, k) if kk > 0))
    attn = W.make_attn_inputs(rng, ctx_lens=ctx, qlens=k, capacity=CAP, num_q_heads=HQ,
                              num_kv_heads=HKV, head_dim=D, max_kv_len=MAX_KV,
                              spare_pages=POOL - used)
    acc = W.make_accept_inputs(rng, cu_qlens=attn.cu_qlens, capacity=CAP, vocab=VOCAB,
                               dtype="bf16")
    return attn, acc


class Buffers:
    """Every device array the step touches, allocated once."""

    def __init__(self):
        P = (MAX_KV + 15) // 16
        self.q = torch.zeros(CAP, HQ, D, dtype=torch.bfloat16, device=DEV)
        self.cu = torch.zeros(B + 1, dtype=torch.int32, device=DEV)
        self.kv = torch.zeros(POOL, 2, HKV, 16 * D, dtype=torch.bfloat16, device=DEV)
        self.pt = torch.zeros(B, P, dtype=torch.int32, device=DEV)
        self.ctx = torch.zeros(B, dtype=torch.int32, device=DEV)
        self.out = torch.zeros(CAP, HQ, D, dtype=torch.bfloat16, device=DEV)
        self.logits = torch.zeros(CAP, VOCAB, dtype=torch.bfloat16, device=DEV)
        self.draft = torch.zeros(CAP, dtype=torch.int32, device=DEV)
        self.a = torch.zeros(B, dtype=torch.int32, device=DEV)
        self.nxt = torch.zeros(B, dtype=torch.int32, device=DEV)
        self.dims = dsv.attn_dims(self.q, self.kv, self.pt, max_kv_len=MAX_KV)
        self.ws = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(self.dims), DEV)
        self.ws2 = dsv.alloc_workspace(dsv.accept_workspace_bytes(CAP, B, VOCAB), DEV)

    def addresses(self):
        return [t.data_ptr() for t in (self.q, self.cu, self.kv, self.pt, self.ctx,
                                       self.out, self.logits, self.draft, self.a,
                                       self.nxt, self.ws, self.ws2)]

    def load(self, attn, acc):
        # contents change, addresses do not
        self.q.copy_(bf16_dev(attn.q))
        self.cu.copy_(i32_dev(attn.cu_qlens))
        self.kv.copy_(bf16_dev(attn.kv_pages))
        self.pt.copy_(i32_dev(attn.page_table))
        self.ctx.copy_(i32_dev(attn.ctx_lens))
        self.logits.copy_(bf16_dev(acc.logits))
        self.draft.copy_(i32_dev(acc.draft_tokens))
        self.out.fill_(float("nan"))
        self.a.fill_(-7)
        self.nxt.fill_(-7)

    def enqueue(self, stream):
        dsv.verify_attn(self.q, self.cu, self.kv, self.pt, self.ctx, self.out,
                        dims=self.dims, workspace=self.ws, stream=stream)
        dsv.accept(self.logits, self.cu, self.draft, self.a, self.nxt, workspace=self.ws2,
                   stream=stream)

    def snapshot(self):
        torch.cuda.synchronize()
        return bf16_host(self.out), self.a.cpu().numpy(), self.nxt.cpu().numpy()


def test_capture_once_replay_many_steps():
    buf = Buffers()
    stream = torch.cuda.Stream()
    addrs = buf.addresses()
    attn0, acc0 = step_inputs(100)
    buf.load(attn0, acc0)
    torch.cuda.synchronize()
    say("graph", "capture")
    graph = dsv.Graph().capture(lambda: buf.enqueue(stream), stream)
    for step in range(4):
        attn, acc = step_inputs(101 + step)
        say("graph", "step", step, "k", list(attn.qlens))
        buf.load(attn, acc)
        torch.cuda.synchronize()
        graph.replay(stream)
        out_g, a_g, n_g = buf.snapshot()
        # eager calls on the same buffers, between replays
        buf.out.fill_(float("nan"))
        buf.enqueue(torch.cuda.current_stream())
        out_e, a_e, n_e = buf.snapshot()
        assert np.array_equal(out_g, out_e) and np.array_equal(a_g, a_e) and \
            np.array_equal(n_g, n_e)
        ref = oracle.verify_attn(attn.q, attn.cu_qlens, attn.kv_pages, attn.page_table,
                                 attn.ctx_lens, **attn.oracle_kwargs())
        assert_attn_close(out_g, ref, attn)
        ra, rn = oracle.accept(acc.logits, "bf16", acc.cu_qlens, acc.draft_tokens)
        assert np.array_equal(a_g, ra) and np.array_equal(n_g, rn)
        assert buf.addresses() == addrs
    # replay again after eager work: the graph still computes the last inputs
    graph.replay(stream)
    out_g2, a_g2, n_g2 = buf.snapshot()
    assert np.array_equal(out_g2, out_e) and np.array_equal(a_g2, a_e)
    graph.close()
