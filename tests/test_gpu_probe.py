"""The HBM streaming probe behind bench.py's ceiling: it runs on uneven splits of tiles and
granules over workgroups, writes exactly its destination range, and every written granule is
one of the source's (its contents are otherwise unspecified)."""
import numpy as np
import pytest
import torch

from paper_2607_20538_amd import codec as cg

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ntiles,ngran", [(1, 0), (1, 1), (7, 5), (13, 1000), (2000, 300001)])
def test_stream_probe_writes_its_range_from_the_source(ntiles, ngran):
    print(f"stream_probe ntiles={ntiles} ngran={ngran}", flush=True)
    g = torch.Generator().manual_seed(ntiles * 7919 + ngran)
    src = torch.randint(0, 256, (ntiles * 8192,), dtype=torch.uint8, generator=g).cuda()
    guard = 4096
    dst = torch.full((ngran * 16 + guard,), 0xA5, dtype=torch.uint8, device="cuda")
    cg.cg_stream_probe(src, ntiles * 8192, dst, ngran * 16)
    torch.cuda.synchronize()
    out = dst.cpu().numpy()
    assert (out[ngran * 16:] == 0xA5).all()
    if ngran:
        s = src.cpu().numpy().view(np.dtype((np.void, 16)))
        o = out[: ngran * 16].view(np.dtype((np.void, 16)))
        assert np.isin(o, s).all()
