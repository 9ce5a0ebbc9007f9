"""The read-rate probe reads exactly the tiles it is given (through the C ABI).

Each workgroup's XOR of the 32-bit words it read is compared bit for bit
with a host XOR over the same visit range.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, say
except Exception:  # pragma: no cover
    pass

TILE_WORDS = 4096 // 4


def expected_sinks(words, order, grid):
    """Per workgroup: XOR over visits [b*per, (b+1)*per) of the tile words,
    ids outside the buffer contributing nothing."""
    tiles = words.reshape(-1, TILE_WORDS)
    tile_xor = np.bitwise_xor.reduce(tiles, axis=1)
    n = tiles.shape[0]
    visits = len(order)
    per = -(-visits // grid)
    out = np.zeros(grid, dtype=np.uint32)
    for b in range(grid):
        ids = order[min(visits, b * per):min(visits, (b + 1) * per)]
        ids = ids[(ids >= 0) & (ids < n)]
        out[b] = np.bitwise_xor.reduce(tile_xor[ids]) if len(ids) else 0
    return out


@pytest.mark.parametrize("name,n_tiles,visits,grid,bad", [
    ("permutation-512", 4096, 4096, 512, False),
    ("ragged-rounds", 1000, 997, 7, False),
    ("several-staging-chunks", 3000, 5000, 2, True),
    ("grid-above-visits", 64, 50, 300, True),
    ("one-workgroup", 257, 300, 1, True),
])
def test_probe_reads_the_given_tiles(name, n_tiles, visits, grid, bad):
    rng = np.random.default_rng(n_tiles + visits + grid)
    words = rng.integers(0, 2 ** 32, size=n_tiles * TILE_WORDS, dtype=np.uint32)
    if visits == n_tiles:
        order = rng.permutation(n_tiles).astype(np.int32)
    else:
        order = rng.integers(0, n_tiles, size=visits).astype(np.int32)  # with repeats
    if bad:  # ids outside the buffer read nothing
        at = rng.choice(visits, size=max(1, visits // 10), replace=False)
        order[at] = rng.choice(np.array([-1, n_tiles, n_tiles + 5, 2 ** 31 - 1],
                                        dtype=np.int32), size=len(at))
    say("probe", name, "tiles=%d visits=%d grid=%d" % (n_tiles, visits, grid))
    buf = torch.from_numpy(words.view(np.int32)).to(DEV)
    ord_d = torch.from_numpy(order).to(DEV)
    sink = torch.full((grid,), -1, dtype=torch.int32, device=DEV)
    dsv.read_probe(buf, ord_d, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, expected_sinks(words, order, grid))


def test_probe_rejects_bad_arguments():
    buf = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    order = torch.zeros(4, dtype=torch.int32, device=DEV)
    with pytest.raises(ValueError):
        dsv.read_probe(torch.zeros(4000, dtype=torch.uint8, device=DEV), order,
                       torch.zeros(1, dtype=torch.int32, device=DEV))
    with pytest.raises(dsv.DSVError):
        dsv.read_probe(buf, order, torch.zeros(0, dtype=torch.int32, device=DEV))
