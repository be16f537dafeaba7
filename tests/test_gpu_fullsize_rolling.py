"""Full-size parity of the rolling step (section 4.4: each new KV token passes through gauge,
backend, decode and inverse gauge): B = 32 rows of a 32k-token compressed history, Llama-3-8B
KV shape (L = 32, H = 8, head_dim 128), block-uniform 6-bit with 64-channel blocks, Haar gauge
g = 128, in the launch configuration bench.py times (kv_encode of each whole history tensor, then
one kv_append_step over all 32 layers that decodes every row's history [0, pos[b]]).

Rows append at different positions (pos[b] = 32760 + 7 (b mod 4), overwriting a slot of the
history), so every row's history ends in a different ragged tile.  History input: synth's first
four batch rows of layer 0 repeated over the 32 rows, viewed with layer stride 0 (each layer's
own gauge makes its cache distinct); the histories are decoded one cache type at a time so that
one 69 GB bf16 history view is alive at once.

Checked on whole (layer, batch, head) slices: the GPU cache (history codes and the appended
token) against the oracle's encode of the same slice input followed by the oracle's append,
under the fused-encoder criteria; the decoded history rows [0, pos[b]] against the oracle's
decode of the GPU's cache rows (bf16 within an ulp); the rows after pos[b] untouched."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_slice_host, cache_slice, check_bf16_within_ulp, check_fused_codes

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["rolling"]
NB = 4                                      # distinct batch rows, repeated over W.B
T_HIST = W.T + 16                           # history tokens encoded (positions past pos[b] included)
T_CAP = W.T + 32
SLICES = [(0, 0, 0), (17, 13, 3), (31, 31, 7), (5, 6, 2)]   # (layer, batch, head)
SENTINEL = 0x40A0                           # bf16 5.0


def _pos():
    return np.array([W.T - 8 + 7 * (b % 4) for b in range(W.B)], dtype=np.int32)


@pytest.fixture(scope="module")
def rolled():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shp = cg.shape(W.L, W.H, W.d, W.g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    codec = cg.Codec(cg.BLOCK_UNIFORM, W.bits, W.block_c)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    caches, news = [], []
    for s in (0, 1):
        x = synth.kv_tensor(W, s, L=1, B=NB, T=T_HIST)
        x = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
        rows = x.repeat(1, W.B // NB, 1, 1, 1)                     # [1][B][H][T][d]
        del x
        X = rows.expand(W.L, W.B, W.H, T_HIST, W.d)                 # layer stride 0
        c = cg.Cache(codec, s, W.L, W.B, W.H, T_CAP, W.d)
        cg.kv_encode(s, X, Gd, shp, codec, c, err_flag=err)
        torch.cuda.synchronize()
        del X, rows
        caches.append(c)
        nt = synth.new_tokens(W, s, 0, L=W.L, B=W.B, H=W.H)        # [L][B][H][d]
        news.append(nt)
    torch.cuda.empty_cache()
    pos = _pos()
    pos_d = torch.from_numpy(pos).cuda()
    kn = torch.from_numpy(news[0].view(np.int16)).view(torch.bfloat16).cuda()[:, :, :, None, :]
    vn = torch.from_numpy(news[1].view(np.int16)).view(torch.bfloat16).cuda()[:, :, :, None, :]
    hist = torch.full((W.L, W.B, W.H, T_HIST, W.d), 5.0, dtype=torch.bfloat16, device="cuda")
    out = {"shp": shp, "Gd": Gd, "codec": codec, "caches": caches, "news": news, "pos": pos, "slices": {}}
    # the step appends both tokens and decodes one history per call; appending the same token at
    # the same position again re-encodes it identically
    for s in (0, 1):
        hist.fill_(5.0)
        cg.kv_append_step(0, W.L, kn, vn, pos_d, Gd, shp, codec, caches[0], caches[1],
                          hist if s == 0 else None, hist if s == 1 else None, err_flag=err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        out["slices"][s] = {(l, b, h): hist[l, b, h].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                            for l, b, h in SLICES}
    del hist
    torch.cuda.empty_cache()
    out["G_orc"] = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    yield out
    out.clear()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("s", [0, 1])
def test_rolling_step_full_size_matches_oracle(rolled, s):
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=W.bits, block_c=W.block_c)
    pos = rolled["pos"]
    cache = rolled["caches"][s]
    for l, b, h in SLICES:
        xs = bf16_slice_host(synth.kv_slice(W.data_seed, s, 0, b % NB, h, T_HIST, W.d, W.keys))[None, None, None]
        Gs = np.ascontiguousarray(rolled["G_orc"][l:l + 1, :, h:h + 1])
        orc, flags = O.kv_encode(oc, s, xs, Gs, T_cap=T_CAP)
        assert flags == 0
        new = np.ascontiguousarray(rolled["news"][s][l:l + 1, b:b + 1, h:h + 1])
        assert O.kv_append(oc, s, new, Gs, orc, [int(pos[b])]) == 0
        # z of the history with the appended token in its slot, for the tie check
        xz = xs.copy()
        xz[0, 0, 0, pos[b]] = new[0, 0, 0]
        zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, xz, Gs, T_cap=T_CAP)
        got = cache_slice(cache, oc, s, l, b, h)
        check_fused_codes(got, orc, zo["codes"], oc, s, W.d, T_HIST)
        n = int(pos[b]) + 1
        ref = O.kv_decode(oc, s, Gs, got, 0, n, out_bf16=False)
        y = rolled["slices"][s][(l, b, h)][None, None, None]
        check_bf16_within_ulp(ref, y[:, :, :, :n], W.g)
        assert (y[:, :, :, n:] == SENTINEL).all()
