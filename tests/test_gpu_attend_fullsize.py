"""Full-size parity of the fused decode-phase attention: the rolling-decode configuration
(32 layers, batch 32, 8 KV heads with 4 query heads each, 32768-token history, head_dim 128,
bf16; Haar gauge g = 128; block-uniform 6-bit, block 64) in the launch configuration bench.py
times (every layer in one kv_attend call, device row lengths, bf16 output), with ragged row
lengths.

Sampled outputs: for several (layer, batch row, KV head) slices the oracle attends, in
binary64, over the GPU cache's own rows of that slice (copied back), with the same queries
and the oracle's Haar gauge; tolerance as in test_gpu_attend.py plus the bf16 rounding of the
output.  Every output: a convex combination of the decoded values has a norm of at most the
largest decoded value norm of its row, which the stored side information bounds (the gauge is
orthogonal: ||xhat_t|| = ||zhat_t|| <= sqrt(sum_k n max(|mn_k|, |mn_k + (2^b - 1) sc_k|)^2))."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_dev, to_cg

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["rolling"]
GRP = 4
SAMPLES = [(0, 0, 0), (7, 31, 3), (19, 12, 6), (31, 5, 7)]   # (layer, batch row, KV head)
ATT_TOL = 1e-4


@pytest.fixture(scope="module")
def full():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shp = cg.shape(W.L, W.H, W.d, W.g)
    codec = cg.Codec(cg.BLOCK_UNIFORM, W.bits, W.block_c)
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
    lens_h = [W.T - 1021 * b for b in range(W.B)]
    lens = torch.tensor(lens_h, dtype=torch.int32, device="cuda")
    o = torch.empty((W.L, W.B, W.H * GRP, 1, W.d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(16, cg.attend_workspace_bytes(shp, W.L, W.B, W.H * GRP, W.T)), dtype=torch.uint8,
                     device="cuda")
    scale = 1.0 / np.sqrt(W.d)
    cg.kv_attend(0, W.L, q, caches[0], caches[1], Gd, shp, codec, lens, scale, o, ws, err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return dict(shp=shp, codec=codec, caches=caches, qh=qh, lens=lens_h, o=o, scale=scale)


def _slice(cache, s, l, b, h, n):
    """Rows [0, n) of slice (l, b, h) of a GPU cache as a one-slice oracle-layout cache."""
    nc = W.d * W.bits // 8
    nbk = W.d // W.block_c
    sl = (l * W.B + b) * W.H + h
    codes = cache.codes[: W.L * W.B * W.H * W.T * nc].view(W.L * W.B * W.H, W.T, nc)
    side = cache.side[: W.L * W.B * W.H * W.T * nbk * 4].view(torch.int16).view(W.L * W.B * W.H, W.T, nbk, 2)
    c = codes[sl, :n].cpu().numpy().reshape(1, 1, 1, n, nc)
    sd = side[sl, :n].cpu().numpy().view(np.uint16).reshape(1, 1, 1, n, nbk, 2)
    return {"codes": np.ascontiguousarray(c), "side": np.ascontiguousarray(sd), "residual": None}


def test_sampled_rows_match_oracle(full):
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=W.bits, block_c=W.block_c)
    G = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    o = full["o"].float().cpu().numpy()[:, :, :, 0]
    qf = (full["qh"].astype(np.uint32) << 16).view(np.float32)
    for l, b, h in SAMPLES:
        n = full["lens"][b]
        kh = _slice(full["caches"][0], 0, l, b, h, n)
        vh = _slice(full["caches"][1], 1, l, b, h, n)
        Gs = np.ascontiguousarray(G[l:l + 1, :, h:h + 1])
        qs = np.ascontiguousarray(qf[l:l + 1, b:b + 1, h * GRP:(h + 1) * GRP])
        ref = O.attend(oc, Gs, kh, vh, qs, [n], full["scale"])[0, 0]
        Vh = O.kv_decode(oc, 1, Gs, vh, 0, n, out_bf16=False)
        vmax = float(np.abs(Vh).max())
        got = o[l, b, h * GRP:(h + 1) * GRP]
        tol = ATT_TOL * vmax + np.abs(ref) * 2.0 ** -8
        err = np.abs(got - ref)
        assert (err <= tol).all(), (l, b, h, float(err.max()))


def test_every_output_within_the_value_norm_bound(full):
    nbk = W.d // W.block_c
    qmax = float((1 << W.bits) - 1)
    vc = full["caches"][1]
    side = vc.side[: W.L * W.B * W.H * W.T * nbk * 4].view(torch.float16).view(W.L, W.B, W.H, W.T, nbk, 2).float()
    mn, sc = side[..., 0], side[..., 1]
    bound = torch.maximum(mn.abs(), (mn + qmax * sc).abs())                     # per-block max |zhat|
    tok = (bound.square().sum(dim=-1) * W.block_c).sqrt()                          # per-token bound
    t = torch.arange(W.T, device="cuda")
    lens = torch.tensor(full["lens"], device="cuda")
    tok = torch.where(t[None, None, None, :] < lens[None, :, None, None], tok, torch.zeros((), device="cuda"))
    row = tok.amax(dim=3).repeat_interleave(GRP, dim=2)                            # [L][B][Hq]
    on = full["o"].float()[:, :, :, 0].norm(dim=-1)
    assert torch.isfinite(full["o"].float()).all()
    assert (on <= row * (1 + 2.0 ** -7) + 1e-6).all()
