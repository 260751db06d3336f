"""The page-pattern gather probe (bellman_probe_gather): it must read every
tile of the pool exactly once, whatever the tile size and wave count, which
the XOR of all the pool's words checks exactly."""
from __future__ import annotations

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

bl = pytest.importorskip("paper_2510_15330_amd")


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bl.library()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("waves", [0, 1, 3, 1000, 100000])
@pytest.mark.parametrize("tiles", [1, 2, 4096])
@pytest.mark.parametrize("tile_bytes", [2048, 4096, 8192])
def test_probe_reads_every_tile_once(tile_bytes, tiles, waves):
    rng = np.random.default_rng(tile_bytes + tiles + waves)
    host = rng.integers(0, 2**32, size=tiles * tile_bytes // 4, dtype=np.uint32)
    pool = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    print(f"probe tile_bytes={tile_bytes} tiles={tiles} waves={waves}", flush=True)
    bl.probe_gather(pool, tile_bytes, sink, max_waves=waves)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(host)
    assert np.uint32(sink.cpu().numpy().view(np.uint32)[0]) == want
