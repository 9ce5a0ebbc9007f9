"""Device-side helpers shared by the GPU tests (marshalling only)."""
import sys

import numpy as np
import torch

import paper_2609_37532_amd as dsv
import workloads as W

DEV = "cuda:0"


def say(*a):
    """Flushed progress line naming the case (survives a dead box)."""
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def bf16_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)


def i32_dev(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def bf16_host(t: torch.Tensor) -> np.ndarray:
    """bf16 device tensor -> float64 numpy (exact)."""
    bits = t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
    return W.bf16_to_f32(bits).astype(np.float64)


class AttnDev:
    """An AttnInputs uploaded once; `run()` enqueues verify_attn."""

    def __init__(self, inp: W.AttnInputs, fill_out: float = float("nan")):
        self.inp = inp
        self.q = bf16_dev(inp.q)
        self.cu = i32_dev(inp.cu_qlens)
        self.kv = bf16_dev(inp.kv_pages)
        self.pt = i32_dev(inp.page_table)
        self.ctx = i32_dev(inp.ctx_lens)
        self.out = torch.full(tuple(inp.q.shape), fill_out, dtype=torch.bfloat16, device=DEV)
        self.dims = dsv.attn_dims(self.q, self.kv, self.pt, max_kv_len=inp.max_kv_len,
                                  scale=inp.scale)
        self.ws = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(self.dims), DEV)

    def run(self, stream=None):
        dsv.verify_attn(self.q, self.cu, self.kv, self.pt, self.ctx, self.out,
                        dims=self.dims, workspace=self.ws, stream=stream)

    def result(self) -> np.ndarray:
        torch.cuda.synchronize()
        return bf16_host(self.out)


def run_attn(inp: W.AttnInputs) -> np.ndarray:
    d = AttnDev(inp)
    d.run()
    return d.result()


def attn_errors(got: np.ndarray, ref: np.ndarray, inp: W.AttnInputs):
    live = int(inp.cu_qlens[-1])
    err = np.abs(got[:live] - ref[:live])
    return float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0


def bf16_spacing(x):
    """Distance between neighbouring bf16 values at magnitude |x|: 2^(e-7)
    for |x| in [2^e, 2^(e+1)) (8 significant bits); 0 at x = 0."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    _, e = np.frexp(x)  # x = f * 2^e with f in [0.5, 1): the binade is [2^(e-1), 2^e)
    return np.where(x > 0, np.ldexp(1.0, e - 8), 0.0)


def attn_bound(ref, max_abs=1e-2):
    """Per-element bound on |out - oracle|: max_abs, except where the bf16
    output format cannot meet it.  The output is rounded once to bf16
    (nearest even), which moves an element of magnitude |r| by up to half
    the bf16 spacing there, 2^(floor(log2 |r|) - 8): at most 0.0078 on
    [2, 4), so max_abs stays attainable below |r| = 4, and 0.0156 on
    [4, 8), where no bf16 output can meet 1e-2.  The bound is that half
    spacing plus 2e-3 for the arithmetic, or max_abs if larger; it equals
    max_abs below |r| = 4."""
    return np.maximum(max_abs, 0.5 * bf16_spacing(ref) + 2e-3)


# Two runs of one request that differ only in how the batch around it is
# packed (or in how many rows it has) may cut its segments at other points
# and stack its rows with other tile-mates.  The running maximum is an
# integer, so that moves its weights and partial sums by exact powers of two
# only; what remains is fp32 summation order and, rarely, a weight whose
# bf16 rounding flips because the exponent argument rounded differently
# (each such flip moves the output by at most 2^-8 of that weight's share).
# The final bf16 rounding can then land one spacing apart.  This is the
# slack for the fp32 part.
INVARIANT_SLACK = 2.0 ** -12


def assert_same_up_to_rounding(got, base, what=""):
    """|got - base| <= one bf16 spacing of the base value + INVARIANT_SLACK."""
    d = np.abs(got - base)
    excess = d - (bf16_spacing(base) + INVARIANT_SLACK)
    worst = float(excess.max()) if excess.size else -1.0
    assert worst <= 0, "%s: max diff %.3g, worst excess over one bf16 spacing %.3g" % (
        what, float(d.max()), worst)
    return float(d.max())


def assert_attn_close(got, ref, inp, max_abs=1e-2, mean_abs=1e-3):
    """Tolerance of the verify path vs fp64: every live element within
    attn_bound (max-abs 1e-2 wherever bf16 can hold it), mean-abs 1e-3;
    tail rows exactly zero."""
    live = int(inp.cu_qlens[-1])
    assert np.isfinite(got).all(), "non-finite output"
    mx, mn = attn_errors(got, ref, inp)
    err = np.abs(got[:live] - ref[:live])
    over = err - attn_bound(ref[:live], max_abs)
    worst = float(over.max()) if over.size else -1.0
    assert worst <= 0 and mn <= mean_abs, "max %.3g mean %.3g (worst excess over the bound %.3g)" % (
        mx, mn, worst)
    assert not got[live:].any(), "tail rows not zero"
    return mx, mn


class AcceptDev:
    def __init__(self, acc: W.AcceptInputs):
        self.acc = acc
        if acc.dtype == "bf16":
            self.logits = bf16_dev(acc.logits)
        else:
            self.logits = torch.from_numpy(acc.logits).to(DEV)
        self.cu = i32_dev(acc.cu_qlens)
        self.draft = i32_dev(acc.draft_tokens)
        B = acc.num_reqs
        self.a = torch.full((B,), -7, dtype=torch.int32, device=DEV)
        self.nxt = torch.full((B,), -7, dtype=torch.int32, device=DEV)
        self.ws = dsv.alloc_workspace(
            dsv.accept_workspace_bytes(acc.capacity, B, acc.vocab), DEV)

    def run(self, stream=None):
        dsv.accept(self.logits, self.cu, self.draft, self.a, self.nxt, workspace=self.ws,
                   stream=stream)

    def result(self):
        torch.cuda.synchronize()
        return self.a.cpu().numpy(), self.nxt.cpu().numpy()


class DvlDev:
    """A DvlInputs uploaded once; `run()` enqueues dvl_allocate_pack into
    buffers pre-filled with a poison value (so unwritten entries show)."""

    POISON = -123456

    def __init__(self, d: W.DvlInputs):
        self.d = d
        n_bs, w = d.tokens.shape
        m_bs = w * n_bs // 2
        self.logits = torch.from_numpy(np.ascontiguousarray(d.pred_logits)).to(DEV)
        self.num_live = i32_dev([d.n_live])
        self.tokens = i32_dev(d.tokens)
        self.positions = i32_dev(d.positions)
        self.kv_refs = i32_dev(d.kv_refs)
        full = lambda n: torch.full((n,), self.POISON, dtype=torch.int32, device=DEV)
        self.k = full(n_bs)
        self.cu = full(n_bs + 1)
        self.ptok, self.ppos, self.pref = full(m_bs), full(m_bs), full(m_bs)
        self.scores = torch.full((n_bs, w), float("nan"), dtype=torch.float32, device=DEV)

    def run(self, stream=None, scores=True):
        dsv.dvl_allocate_pack(self.logits, self.num_live, self.tokens, self.positions,
                              self.kv_refs, self.k, self.cu, self.ptok, self.ppos, self.pref,
                              self.scores if scores else None, stream=stream)

    def result(self):
        torch.cuda.synchronize()
        return dict(k=self.k.cpu().numpy(), offsets=self.cu.cpu().numpy(),
                    tokens=self.ptok.cpu().numpy(), positions=self.ppos.cpu().numpy(),
                    kv_refs=self.pref.cpu().numpy(), q=self.scores.cpu().numpy())


def gather_oracle_inputs(q_rows, kv_pool, page_row, ctx, k):
    """Host inputs of one request for the attention oracle: its q rows
    [k, Hq, D], its pages gathered from the device pool (renumbered 0..),
    a one-row page table, its context and offsets."""
    npg = -(-(int(ctx) + int(k)) // W.PAGE_SIZE)
    ids = torch.as_tensor(np.asarray(page_row[:npg], dtype=np.int64), device=kv_pool.device)
    as_bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return dict(q=as_bits(q_rows), cu_qlens=np.array([0, k], np.int32),
                kv_pages=as_bits(kv_pool[ids]),
                page_table=np.arange(npg, dtype=np.int32)[None, :],
                ctx_lens=np.array([ctx], np.int32))
