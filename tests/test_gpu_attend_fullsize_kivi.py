"""Full-size parity of the fused decode-phase attention over KIVI-style caches: the KIVI
configuration (32 layers, batch 4, 8 KV heads with 4 query heads each, 32768 tokens, head_dim
128, bf16; Haar gauge g = 32; keys in 32-token groups with per-channel ranges, values in
64-channel blocks per token, 3 bits, the last 128 tokens kept in bf16) in the launch
configuration bench.py --workload attend_kivi times (every layer in one kv_attend call, device
row lengths, bf16 output) on the matrix-core attention kernel.  Every row holds the whole
history, so the last split of each row also scores the window's 128 raw positions.

Sampled outputs: for several (layer, batch row, KV head) slices the oracle attends, in binary64,
over the GPU cache's own rows of that slice (copied back), with the same queries and the
oracle's Haar gauge; tolerance as in test_gpu_attend.py plus the bf16 rounding of the output."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_dev, cache_slice

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["kivi"]
GRP = 4
SAMPLES = [(0, 0, 0), (9, 3, 5), (22, 1, 2), (31, 2, 7)]   # (layer, batch row, KV head)
ATT_TOL = 1e-4


def _oc():
    return O.Codec(backend=O.KIVI, bits=W.bits, block_c=64, key_tokens=W.key_tokens, val_channels=W.val_channels,
                   residual=W.residual)


@pytest.fixture(scope="module")
def full():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shp = cg.shape(W.L, W.H, W.d, W.g)
    codec = cg.Codec(cg.KIVI, W.bits, 64, W.key_tokens, W.val_channels, W.residual)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    caches = []
    for s in (0, 1):
        # one layer of the workload viewed with layer stride 0, as in the benchmark
        x1 = torch.from_numpy(synth.kv_tensor(W, s, L=1).view(np.int16)).view(torch.bfloat16).cuda()
        c = cg.Cache(codec, s, W.L, W.B, W.H, W.T, W.d)
        cg.kv_encode(s, x1.expand(W.L, W.B, W.H, W.T, W.d), Gd, shp, codec, c, err_flag=err)
        torch.cuda.synchronize()
        del x1
        caches.append(c)
    qh = synth.queries(W, W.H * GRP)
    q = bf16_dev(qh).reshape(W.L, W.B, W.H * GRP, 1, W.d)
    lens = torch.full((W.B,), W.T, dtype=torch.int32, device="cuda")
    o = torch.empty((W.L, W.B, W.H * GRP, 1, W.d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(16, cg.attend_workspace_bytes(shp, W.L, W.B, W.H * GRP, W.T)), dtype=torch.uint8,
                     device="cuda")
    scale = 1.0 / np.sqrt(W.d)
    cg.kv_attend(0, W.L, q, caches[0], caches[1], Gd, shp, codec, lens, scale, o, ws, err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return dict(caches=caches, qh=qh, o=o, scale=scale)


def test_sampled_rows_match_oracle(full):
    oc = _oc()
    G = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    o = full["o"].float().cpu().numpy()[:, :, :, 0]
    qf = (full["qh"].astype(np.uint32) << 16).view(np.float32)
    n = W.T
    for l, b, h in SAMPLES:
        kh = cache_slice(full["caches"][0], oc, 0, l, b, h)
        vh = cache_slice(full["caches"][1], oc, 1, l, b, h)
        Gs = np.ascontiguousarray(G[l:l + 1, :, h:h + 1])
        qs = np.ascontiguousarray(qf[l:l + 1, b:b + 1, h * GRP:(h + 1) * GRP])
        ref = O.attend(oc, Gs, kh, vh, qs, [n], full["scale"])[0, 0]
        Vh = O.kv_decode(oc, 1, Gs, vh, 0, n, lens=[n], out_bf16=False)
        vmax = float(np.abs(Vh).max())
        got = o[l, b, h * GRP:(h + 1) * GRP]
        tol = ATT_TOL * vmax + np.abs(ref) * 2.0 ** -8
        err = np.abs(got - ref)
        assert (err <= tol).all(), (l, b, h, float(err.max()))


def test_every_output_is_finite_and_nonzero(full):
    o = full["o"].float()
    assert torch.isfinite(o).all()
    assert (o.abs().amax(dim=-1) > 0).all()
