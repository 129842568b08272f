"""The streaming-read probe reads exactly what its header states: each wave
of workgroup g XORs the 16-byte words of pieces w, w+4, ... of region g,
whichever load pattern it uses."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_32831_amd as uc  # noqa: E402


@pytest.mark.parametrize("pattern", [0, 1])
@pytest.mark.parametrize("pieces", [1, 6])
def test_read_probe_covers_its_regions(pattern, pieces):
    print("CASE read_probe pattern", pattern, "pieces", pieces, flush=True)
    unit = uc.uc_read_probe_unit()
    n_wg = unit // 4096
    rng = np.random.default_rng(7 + pieces)
    host = rng.integers(0, 2**32, size=pieces * unit // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.uint8).copy()).cuda()
    sink = torch.zeros(uc.uc_read_probe_sink_bytes(), dtype=torch.uint8, device="cuda")
    uc.uc_read_probe(buf, pattern, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32).reshape(n_wg, 4, 4)
    words = host.reshape(n_wg, pieces, 256, 4)
    for w in range(4):
        mine = words[:, w::4]  # pieces w, w+4, ... of every region
        exp = np.bitwise_xor.reduce(mine.reshape(n_wg, -1, 4), axis=1) if mine.shape[1] else \
            np.zeros((n_wg, 4), np.uint32)
        assert np.array_equal(got[:, w], exp), (pattern, pieces, w)
