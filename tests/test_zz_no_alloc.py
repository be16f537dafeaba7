"""kv_attend_noalloc (through the C ABI) against kv_attend on the same inputs: the same split plan
and kernels, with the split rows' partial results in the library's device scratch instead of a
caller workspace, so the outputs must agree bit for bit.  Two calls in a row, the second with a
smaller input (the scratch keeps the first call's partials), on the matrix-core attention kernel
(block-uniform; KIVI with 64-channel value blocks) and on the general kernel (KIVI with 32-channel
value blocks), with device row lengths and with the caches' host length."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


def _case(codec, L, B, H, grp, T, T_cap, g, seed):
    w = synth.Workload("noalloc", L=L, B=B, H=H, T=T, d=128, dtype="bf16", g=g, backend="bu", bits=4,
                       data_seed=seed)
    shp = cg.shape(L, H, 128, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=seed, G_host=None, G_dev=Gd)
    caches = []
    for s in (0, 1):
        X = torch.from_numpy(synth.kv_tensor(w, s).view(np.int16)).view(torch.bfloat16).cuda()
        c = cg.Cache(codec, s, L, B, H, T_cap, 128)
        cg.kv_encode(s, X, Gd, shp, codec, c)
        c.len = T
        caches.append(c)
    q = synth.queries(w, H * grp)
    qd = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).cuda().reshape(L, B, H * grp, 1, 128)
    torch.cuda.synchronize()
    return shp, Gd, caches, qd


def _both(shp, Gd, caches, qd, codec, lens, dtype):
    L, B, Hq = qd.shape[:3]
    kc, vc = caches
    outs = []
    for noalloc in (False, True):
        out = torch.full((L, B, Hq, 1, 128), float("nan"), dtype=dtype, device="cuda")
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        if noalloc:
            qv, ov, cs, kcs, vcs = cg.view(qd), cg.view(out), codec.struct(), kc.struct(), vc.struct()
            rc = cg.lib().kv_attend_noalloc(0, L, C.byref(qv), C.byref(kcs), C.byref(vcs), Gd.data_ptr(), shp,
                                            C.byref(cs), None if lens is None else lens.data_ptr(), 0.088,
                                            C.byref(ov), err.data_ptr(), None)
            assert rc == cg.CG_OK, cg.status_str(rc)
        else:
            nws = cg.attend_workspace_bytes(shp, L, B, Hq, kc.T_cap)
            ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
            cg.kv_attend(0, L, qd, kc, vc, Gd, shp, codec, lens, 0.088, out, ws, err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        outs.append(out)
    return outs


CALLS = [
    # codec, (L, B, H, grp, T, T_cap, g), device lengths
    (cg.Codec(cg.BLOCK_UNIFORM, 4, 64), (2, 1, 8, 4, 4096, 4096, 128), [4096]),
    (cg.Codec(cg.BLOCK_UNIFORM, 4, 64), (1, 2, 8, 4, 1000, 1024, 128), None),
    (cg.Codec(cg.KIVI, 3, 64, 32, 64, 128), (2, 1, 4, 4, 3000, 3072, 32), [2990]),
    (cg.Codec(cg.KIVI, 3, 64, 32, 32, 128), (1, 1, 4, 4, 700, 768, 32), None),
]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_noalloc_matches_kv_attend_on_consecutive_calls(dtype):
    for i, (codec, (L, B, H, grp, T, T_cap, g), lens) in enumerate(CALLS):
        shp, Gd, caches, qd = _case(codec, L, B, H, grp, T, T_cap, g, seed=0xA10C + i)
        assert cg.attend_workspace_bytes(shp, L, B, H * grp, T_cap) > 0      # split rows use the scratch
        ln = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
        ref, got = _both(shp, Gd, caches, qd, codec, ln, dtype)
        assert not bool(torch.isnan(ref.float()).any())
        assert torch.equal(ref, got), f"call {i}: max diff {(ref.float() - got.float()).abs().max().item()}"
