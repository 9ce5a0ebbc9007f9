"""GPU: stream-K shares longer than the page-id staging window (Eq. (16)
over the whole committed context).

The attention kernel stages the page ids of at most 512 pages (8192 keys) in
LDS at a time; a piece longer than that runs as several sub-pieces that
carry the online-softmax state across the restaging.  A share only gets that
long when the batch's work is large against the grid: here 64 requests with
contexts U[10000, 14000] and one or two verify rows over 8 KV heads (G = 1,
D = 128).  The KV pool (3.7 GB) and q are drawn on the device from a seeded
generator; sampled requests, among them ones with a piece above 8192 keys
that is whole and ones whose segment is cut between workgroups, are checked
against the fp64 oracle.
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, bf16_host, gather_oracle_inputs, i32_dev, say
except Exception:  # pragma: no cover
    pass

STAGE_KEYS = 512 * W.PAGE_SIZE  # keys whose page ids the kernel stages at a time
LEAD = 6 * 32                   # stream-K lead-in of virtual keys per segment
SKEW_PCT = 6                    # even workgroups' shares are this much larger, odd ones' smaller


def share_bounds(b, share):
    """[begin, end) of workgroup b's share in the virtual space, as the kernel
    lays them out: pairs of shares of share +- skew (whole 32-key blocks)."""
    skew = share * SKEW_PCT // 100 // 32 * 32
    begin = lambda w: w * share + (w & 1) * skew
    return begin(b), begin(b + 1)


def pieces_of(plan, B, hkv, seg_keys):
    """Key length of every (request, KV head, workgroup) piece, from the plan
    the kernel published: plan[i] = virtual prefix of request i, plan[B+1] =
    mean share.  Segment (i, g) occupies [plan[i]*hkv + g*segv, + segv) of
    the virtual space, its keys after a lead-in of LEAD."""
    share = int(plan[B + 1])
    total = int(plan[B]) * hkv
    bounds = []
    b = 0
    while True:
        lo, hi = share_bounds(b, share)
        if lo >= total:
            break
        bounds.append((lo, min(hi, total)))
        b += 1
    out = {}
    for i in range(B):
        segv = seg_keys[i] + LEAD
        for g in range(hkv):
            s0 = int(plan[i]) * hkv + g * segv
            k0, k1 = s0 + LEAD, s0 + segv
            out[(i, g)] = [min(k1, hi) - max(k0, lo) for lo, hi in bounds
                           if min(k1, hi) > max(k0, lo)]
    return share, out


def test_shares_longer_than_the_page_id_window():
    B, hq, hkv, d = 64, 8, 8, 128
    rng = np.random.default_rng(W.SEED_BASE + 800)
    ctx = rng.integers(10000, 14001, size=B).astype(np.int32)
    k = rng.integers(1, 3, size=B).astype(np.int32)
    keys = ctx.astype(np.int64) + k
    max_kv_len = int(keys.max())
    pmax = -(-max_kv_len // W.PAGE_SIZE)
    npg = -(-keys // W.PAGE_SIZE)
    num_pages = int(npg.sum()) + 4
    perm = rng.permutation(num_pages).astype(np.int32)
    pt = np.full((B, pmax), -1, np.int32)
    at = 0
    for i in range(B):
        pt[i, :npg[i]] = perm[at:at + npg[i]]
        at += npg[i]
    cu = W.cu_from_lengths(k)
    cap = int(cu[-1]) + 3
    say("long-shares", "B=%d ctx %d..%d, %d pages (%.2f GB of KV)"
        % (B, ctx.min(), ctx.max(), num_pages, num_pages * 2 * hkv * 16 * d * 2 / 1e9))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(W.SEED_BASE + 801)
    kv = torch.randn((num_pages, 2, hkv, W.PAGE_SIZE * d), generator=gen, device=DEV,
                     dtype=torch.bfloat16)
    q = torch.randn((cap, hq, d), generator=gen, device=DEV, dtype=torch.bfloat16)
    out = torch.full_like(q, float("nan"))
    cu_d, pt_d, ctx_d = i32_dev(cu), i32_dev(pt), i32_dev(ctx)
    dims = dsv.attn_dims(q, kv, pt_d, max_kv_len=max_kv_len, scale=1.0 / np.sqrt(d))
    ws = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(dims), DEV)
    dsv.verify_attn(q, cu_d, kv, pt_d, ctx_d, out, dims=dims, workspace=ws)
    torch.cuda.synchronize()
    plan = ws[:4 * (2 * B + 3)].view(torch.int32).cpu().numpy()
    seg_keys = (-(-keys // 32) * 32).astype(np.int64)
    assert int(plan[B]) == int((seg_keys + LEAD).sum())
    share, pieces = pieces_of(plan, B, hkv, seg_keys)
    long_whole = [i for i in range(B) if any(len(pieces[(i, g)]) == 1 and
                                             pieces[(i, g)][0] > STAGE_KEYS
                                             for g in range(hkv))]
    long_cut = [i for i in range(B) if any(len(pieces[(i, g)]) > 1 and
                                           max(pieces[(i, g)]) > STAGE_KEYS
                                           for g in range(hkv))]
    say("long-shares", "share %d keys; %d requests hold a whole piece over %d keys, "
        "%d a cut segment with such a piece" % (share, len(long_whole), STAGE_KEYS,
                                                len(long_cut)))
    assert share > STAGE_KEYS
    assert long_whole and long_cut
    mid = lambda xs: xs[len(xs) // 2]
    sample = sorted({long_whole[0], mid(long_whole), long_whole[-1], long_cut[0],
                     mid(long_cut), long_cut[-1], 0, B - 1})
    got_all = bf16_host(out)
    assert np.isfinite(got_all[:int(cu[-1])]).all()
    assert not got_all[int(cu[-1]):].any()
    for i in sample:
        o = int(cu[i])
        g = gather_oracle_inputs(q[o:o + int(k[i])], kv, pt[i], int(ctx[i]), int(k[i]))
        ref = oracle.verify_attn(g["q"], g["cu_qlens"], g["kv_pages"], g["page_table"],
                                 g["ctx_lens"], num_q_heads=hq, num_kv_heads=hkv,
                                 head_dim=d, page_size=W.PAGE_SIZE, scale=1.0 / np.sqrt(d))
        got = got_all[o:o + int(k[i])]
        err = np.abs(got - ref)
        say("long-shares", "request %d (ctx %d, k %d, pieces %s): max %.3g mean %.3g"
            % (i, ctx[i], k[i], [pieces[(i, gg)] for gg in range(2)], err.max(), err.mean()))
        assert err.max() <= 1e-2 and err.mean() <= 1e-3
