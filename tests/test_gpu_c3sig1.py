"""The HIP signature path against C3SIG-1's frozen known-answer vectors
(``golden/c3sig1_vectors.txt``), through the C ABI: every chunk signature and
every per-tensor signature, at the default tile and at 1 KiB tiles (many
tiles per chunk), alone and with all vector tensors in one plan."""
import numpy as np
import pytest
import torch

from test_c3sig1_pins import _vectors, _tensor_bytes

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
TORCH = {0: torch.float32, 1: torch.bfloat16, 2: torch.float16, 3: torch.uint8}


def _device_tensor(t, device="cuda"):
    raw = torch.from_numpy(_tensor_bytes(t).copy())
    if raw.numel() == 0:
        return torch.empty(t["shape"], dtype=TORCH[t["dtype"]], device=device)
    return raw.view(TORCH[t["dtype"]]).reshape(t["shape"]).to(device)


@pytest.mark.parametrize("tile", [0, 1024])
def test_each_vector_tensor_alone(tile):
    chunks, tensors = _vectors()
    for t in tensors:
        print("CASE c3sig1", t["name"], tile, flush=True)
        x = _device_tensor(t)
        rec = c3.signature([[x], [x.clone()]], t["cb"], tile_bytes=tile)
        ts = c3.tensor_signature(rec, 1)
        torch.cuda.synchronize()
        g = c3.records_numpy(rec)
        want = [v for v in chunks if v["name"] == t["name"]]
        assert g.shape == (2, t["C"])
        for r in range(2):
            assert [int(s) for s in g["sig"][r]] == [v["sig"] for v in want], t["name"]
            assert [int(k) for k in g["chunk_in_tensor"][r]] == [v["k"] for v in want]
            assert int(ts[r, 0].cpu().numpy().view(np.uint64)) == t["tsig"], t["name"]


def test_all_vector_tensors_in_one_plan():
    chunks, tensors = _vectors()
    cbs = {t["cb"] for t in tensors}
    for cb in sorted(cbs):
        group = [t for t in tensors if t["cb"] == cb]
        print("CASE c3sig1 plan", cb, len(group), flush=True)
        xs = [_device_tensor(t) for t in group]
        rec = c3.signature([xs, [x.clone() for x in xs], [x.clone() for x in xs]], cb)
        ts = c3.tensor_signature(rec, len(group))
        torch.cuda.synchronize()
        g = c3.records_numpy(rec)
        want = [v["sig"] for t in group for v in chunks if v["name"] == t["name"]]
        for r in range(3):
            assert [int(s) for s in g["sig"][r]] == want
            got_t = ts[r].cpu().numpy().view(np.uint64).tolist()
            assert got_t == [t["tsig"] for t in group]
