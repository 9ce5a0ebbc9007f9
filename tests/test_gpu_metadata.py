"""GPU: device metadata that breaks the contract of include/dsv.h.

dsv_validate_metadata reports each violated rule with its bit; verify_attn
never reads outside its buffers for such metadata, skips a request whose
offsets or lengths are out of range (its rows stay untouched), reads page 0
in place of an out-of-range page id, and leaves every other request exact
to the usual tolerance.  All violations are planted from the host; every
kernel runs to completion.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_37532_amd as dsv
import workloads as W

pytestmark = pytest.mark.gpu

try:
    from gpu_util import DEV, AttnDev, attn_errors, bf16_host, say
except Exception:  # pragma: no cover
    pass


def base_inputs():
    rng = np.random.default_rng(77)
    return W.make_attn_inputs(rng, ctx_lens=[100, 40, 300, 7], qlens=[3, 16, 5, 1],
                              capacity=30, num_q_heads=8, num_kv_heads=2, head_dim=128,
                              spare_pages=3, max_kv_len=512)


def validate(dev):
    err = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    dsv.validate_metadata(dev.cu, dev.ctx, dev.pt, dev.dims, err)
    torch.cuda.synchronize()
    return int(err.item())


def rows_of(inp, i):
    return slice(int(inp.cu_qlens[i]), int(inp.cu_qlens[i + 1]))


def test_validate_accepts_clean_metadata():
    inp = base_inputs()
    assert validate(AttnDev(inp)) == 0


@pytest.mark.parametrize("rule,bit", [("cu0", 1), ("decreasing", 1), ("qlen", 2),
                                      ("capacity", 4), ("ctx-neg", 8), ("ctx-long", 8),
                                      ("page", 16)])
def test_validate_flags_each_rule(rule, bit):
    inp = base_inputs()
    dev = AttnDev(inp)
    cu = inp.cu_qlens.copy()
    if rule == "cu0":
        cu[0] = 1
    elif rule == "decreasing":
        cu[2] = cu[1] - 1
    elif rule == "qlen":
        cu[2:] += 1                   # request 1: k = 17
        cu[-1] = min(cu[-1], inp.capacity)
    elif rule == "capacity":
        cu[-1] = inp.capacity + 1
    if rule in ("cu0", "decreasing", "qlen", "capacity"):
        dev.cu.copy_(torch.from_numpy(cu.astype(np.int32)))
    elif rule == "ctx-neg":
        dev.ctx[0] = -1
    elif rule == "ctx-long":
        dev.ctx[2] = inp.max_kv_len
    elif rule == "page":
        dev.pt[2, 1] = inp.num_pages
    got = validate(dev)
    say("validate", rule, "err word", got)
    assert got & bit, got


def test_out_of_range_page_id_is_isolated():
    inp = base_inputs()
    ref = oracle.verify_attn(inp.q, inp.cu_qlens, inp.kv_pages, inp.page_table,
                             inp.ctx_lens, **inp.oracle_kwargs())
    dev = AttnDev(inp)
    dev.pt[2, 3] = inp.num_pages + 1000   # inside request 2's keys
    dev.pt[0, 0] = -7
    assert validate(dev) & 16
    dev.run()
    got = dev.result()
    for i in (1, 3):                      # untouched requests stay exact
        r = rows_of(inp, i)
        err = np.abs(got[r] - ref[r])
        assert np.isfinite(got[r]).all() and err.max() <= 1e-2, (i, err.max())
    assert not got[int(inp.cu_qlens[-1]):].any()


def test_request_with_bad_lengths_is_skipped():
    inp = base_inputs()
    ref = oracle.verify_attn(inp.q, inp.cu_qlens, inp.kv_pages, inp.page_table,
                             inp.ctx_lens, **inp.oracle_kwargs())
    dev = AttnDev(inp, fill_out=7.0)
    dev.ctx[1] = inp.max_kv_len          # ctx + k > max_kv_len
    assert validate(dev) & 8
    dev.run()
    got = dev.result()
    assert (got[rows_of(inp, 1)] == 7.0).all(), "skipped request's rows were written"
    for i in (0, 2, 3):
        r = rows_of(inp, i)
        assert np.abs(got[r] - ref[r]).max() <= 1e-2, i
