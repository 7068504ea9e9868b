"""The read probe (a measurement aid: the signature kernel's access pattern
with nothing computed but an xor) reads every byte exactly once: its per-tile
checksums equal numpy's xor of each tile's 64-bit words, with short last
tiles."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")


@pytest.mark.parametrize("nbytes,tile", [(3 * 2 ** 20 + 3072, 0), (3 * 2 ** 20 + 3072, 1024),
                                         (1024, 1024), (1000 * 1024, 65536), (2 ** 22, 2 ** 24)])
def test_probe_checksums_match_numpy(nbytes, tile):
    print("CASE probe", nbytes, tile, flush=True)
    rng = np.random.default_rng(nbytes + tile)
    host = rng.integers(0, 2 ** 63, nbytes // 8, dtype=np.int64).view(np.uint64)
    buf = torch.from_numpy(host.view(np.uint8).copy()).to("cuda")
    cs = c3.read_probe(buf, tile)
    torch.cuda.synchronize()
    tb = tile or 256 * 1024
    want = [np.bitwise_xor.reduce(host[o // 8:(o + tb) // 8]) for o in range(0, nbytes, tb)]
    assert cs.cpu().numpy().view(np.uint64).tolist() == [int(x) for x in want]


def test_probe_argument_errors():
    buf = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    with pytest.raises(c3.C3Error):
        c3.read_probe(buf[:4000])              # not a multiple of 1024
    with pytest.raises(c3.C3Error):
        c3.read_probe(buf, tile_bytes=3000)    # not a power of two
    with pytest.raises(c3.C3Error):
        c3.read_probe(torch.zeros(4096 + 8, dtype=torch.uint8, device="cuda")[8:])  # misaligned
