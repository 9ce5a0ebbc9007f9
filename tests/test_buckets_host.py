"""Host logic of the multi-bucket capture set (Sec. III-D, Eqs. (14)-(15)),
no GPU: bucket selection, and the bucket capacity identity checked on the
allocator oracle's packed layout."""
import numpy as np
import pytest

import oracle
import paper_2609_37532_amd as dsv
import workloads as W


def test_select_bucket_is_the_smallest_that_fits():
    B = (1, 2, 4, 8, 16, 24, 32, 48, 64)
    for n in range(1, 65):
        b = dsv.select_bucket(B, n)
        assert b >= n and all(x < n for x in B if x < b)
    assert dsv.select_bucket([32, 8, 16], 9) == 16   # order of the set does not matter
    for bad in (0, 65):
        with pytest.raises(ValueError):
            dsv.select_bucket(B, bad)


@pytest.mark.parametrize("n_bs,n", [(8, 8), (8, 5), (32, 17), (32, 1)])
def test_bucket_capacity_with_sentinels(n_bs, n):
    # Eq. (15): live rows plus 8 per sentinel fill exactly 8 N_bs rows, and
    # the offsets of sentinels all sit at M_live
    d = W.make_dvl_inputs(np.random.default_rng(n_bs * 100 + n), n_bs=n_bs, n_live=n)
    res = oracle.dvl_allocate_pack(d.pred_logits, n, d.tokens, d.positions, d.kv_refs)
    m_live = int(res["offsets"][-1])
    assert m_live == 8 * n
    assert m_live + 8 * (n_bs - n) == 8 * n_bs == res["tokens"].shape[0]
    assert (res["offsets"][n:] == m_live).all() and (res["k"][n:] == 0).all()
