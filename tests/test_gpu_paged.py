"""GPU parity of paged caches (kv_attend_paged, kv_encode_paged, kv_append_paged): a page pool
whose batch dimension counts pages of P positions, and a device page table mapping each batch
row's logical pages to pool pages in a seeded random order.

  * attention over the pool equals the oracle's attention over the same rows held contiguously
    (the oracle's own encodings, scattered into the pages here), under the tolerance of
    tests/test_gpu_attend.py, on the matrix-core and the general kernel;
  * a table entry outside the pool flags CG_FLAG_POS_RANGE and leaves the other rows exact;
  * encoding and appending through the table write, byte for byte, what the contiguous entry
    points write on the general kernels (gathered back from the pages)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_dev, cache_to_dev, cache_to_host, to_cg, x_dev

pytestmark = pytest.mark.gpu

ATT_TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


@pytest.fixture(params=["fast", "generic"])
def kernels(request, monkeypatch):
    if request.param == "generic":
        monkeypatch.setenv("CG_KERNELS", "generic")
    else:
        monkeypatch.delenv("CG_KERNELS", raising=False)
    return request.param


def _gauge(kind, L, H, d, g, seed=23):
    G = O.gauge_make(kind, L, H, d, g, seed=seed)
    shp = cg.shape(L, H, d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_USER, shp, params=G, G_host=None, G_dev=Gd)
    return G, Gd, shp


def _table(B, max_pages, spare, seed):
    """Page table [B][max_pages] over a pool of B * max_pages + spare pages, in random order."""
    perm = np.random.default_rng(seed).permutation(B * max_pages + spare).astype(np.int32)
    return perm[: B * max_pages].reshape(B, max_pages), B * max_pages + spare


def _scatter(host, table, P, Bpool):
    """Contiguous rows [L][B][H][max_pages * P][...] -> pool pages [L][Bpool][H][P][...]."""
    out = {"residual": None}
    for key in ("codes", "side"):
        arr = host[key]
        if arr is None:
            out[key] = None
            continue
        pool = np.zeros((arr.shape[0], Bpool, arr.shape[2], P) + arr.shape[4:], dtype=arr.dtype)
        for b in range(table.shape[0]):
            for i in range(table.shape[1]):
                pool[:, table[b, i]] = arr[:, b, :, i * P:(i + 1) * P]
        out[key] = pool
    return out


def _gather(pool, table, P):
    out = {}
    for key in ("codes", "side"):
        arr = pool[key]
        if arr is None:
            out[key] = None
            continue
        rows = [np.concatenate([arr[:, table[b, i]] for i in range(table.shape[1])], axis=2)
                for b in range(table.shape[0])]
        out[key] = np.stack(rows, axis=1)
    return out


PAGED = [
    ("bu4-n64-g32", O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64), 32),
    ("bu6-n64-g128", O.Codec(backend=O.BLOCK_UNIFORM, bits=6, block_c=64), 128),
    ("bu3-n128-g64", O.Codec(backend=O.BLOCK_UNIFORM, bits=3, block_c=128), 64),
    ("pass", O.Codec(backend=O.PASSTHROUGH), 32),
]


@pytest.mark.parametrize("cid,oc,g", PAGED, ids=[c[0] for c in PAGED])
def test_paged_attention_matches_oracle(kernels, cid, oc, g):
    L, B, H, d, grp, P, maxp = 2, 4, 2, 128, 4, 64, 5
    lens = [300, 130, 64, 1]
    T = max(lens)
    w = synth.Workload("pg", L=L, B=B, H=H, T=T, d=d, dtype="bf16", g=g, backend="bu", bits=4, data_seed=0x9A6)
    K, V = synth.kv_tensor(w, 0), synth.kv_tensor(w, 1)
    G, Gd, shp = _gauge(O.GAUGE_HAAR, L, H, d, g)
    kh, _ = O.kv_encode(oc, 0, K, G, T_cap=maxp * P)
    vh, _ = O.kv_encode(oc, 1, V, G, T_cap=maxp * P)
    table, Bpool = _table(B, maxp, 3, seed=5)
    kd = cache_to_dev(_scatter(kh, table, P, Bpool), oc, 0, L, Bpool, H, P, d)
    vd = cache_to_dev(_scatter(vh, table, P, Bpool), oc, 1, L, Bpool, H, P, d)
    qh = synth.queries(w, H * grp)
    qf = (qh.astype(np.uint32) << 16).view(np.float32)
    scale = 1.0 / np.sqrt(d)
    ref = O.attend(oc, G, kh, vh, qf, lens, scale)
    Vh = O.kv_decode(oc, 1, G, vh, 0, T, lens=lens, out_bf16=False)

    pages = torch.from_numpy(table).cuda()
    pt = cg.page_table(pages, P)
    q = bf16_dev(qh).reshape(L, B, H * grp, 1, d)
    out = torch.full((L, B, H * grp, 1, d), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, cg.attend_paged_workspace_bytes(shp, L, B, H * grp, maxp, P)), dtype=torch.uint8,
                     device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ln = torch.tensor(lens, dtype=torch.int32, device="cuda")
    cg.kv_attend_paged(0, L, q, kd, vd, pt, Gd, shp, to_cg(oc), ln, scale, out, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    got = out.cpu().numpy()[:, :, :, 0]
    for b in range(B):
        vmax = np.abs(Vh[:, b, :, : lens[b]]).max()
        assert np.abs(got[:, b] - ref[:, b]).max() <= ATT_TOL * vmax, b

    # a page outside the pool: flagged, contributes nothing; the other rows unchanged
    bad = table.copy()
    bad[1, 0] = Bpool
    pages2 = torch.from_numpy(bad).cuda()
    err.zero_()
    out2 = torch.zeros_like(out)
    cg.kv_attend_paged(0, L, q, kd, vd, cg.page_table(pages2, P), Gd, shp, to_cg(oc), ln, scale, out2, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == cg.CG_FLAG_POS_RANGE
    o2 = out2.cpu().numpy()[:, :, :, 0]
    assert np.isfinite(o2).all()
    np.testing.assert_array_equal(o2[:, [0, 2, 3]], got[:, [0, 2, 3]])


@pytest.mark.parametrize("oc", [O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64), O.Codec(backend=O.PASSTHROUGH)],
                         ids=["bu4", "pass"])
def test_paged_encode_and_append_equal_contiguous(monkeypatch, oc):
    monkeypatch.setenv("CG_KERNELS", "generic")   # the contiguous reference on the same kernels
    L, B, H, d, P, maxp, T = 2, 3, 2, 128, 64, 4, 192
    w = synth.Workload("pg", L=L, B=B, H=H, T=T, d=d, dtype="bf16", g=32, backend="bu", bits=4, data_seed=0x9A7)
    G, Gd, shp = _gauge(O.GAUGE_HAAR, L, H, d, 32)
    table, Bpool = _table(B, maxp, 2, seed=6)
    pages = torch.from_numpy(table).cuda()
    pt = cg.page_table(pages, P)
    c = to_cg(oc)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        pool = cg.Cache(c, s, L, Bpool, H, P, d)
        cg.kv_encode_paged(s, x_dev(X), pt, Gd, shp, c, pool, 0, err)
        cont = cg.Cache(c, s, L, B, H, maxp * P, d)
        cg.kv_encode(s, x_dev(X), Gd, shp, c, cont, 0, err)
        torch.cuda.synchronize()
        got = _gather(cache_to_host(pool, oc, s), table, P)
        want = cache_to_host(cont, oc, s)
        for key in ("codes", "side"):
            if want[key] is not None:
                np.testing.assert_array_equal(got[key][:, :, :, :T], want[key][:, :, :, :T])
    # appends at positions 192 .. 194 (the fourth page of every row)
    kpool, vpool = cg.Cache(c, 0, L, Bpool, H, P, d), cg.Cache(c, 1, L, Bpool, H, P, d)
    kc, vc = cg.Cache(c, 0, L, B, H, maxp * P, d), cg.Cache(c, 1, L, B, H, maxp * P, d)
    pos = torch.full((B,), T, dtype=torch.int32, device="cuda")
    for step in range(3):
        kn = x_dev(synth.new_tokens(w, 0, step)).reshape(L, B, H, 1, d)
        vn = x_dev(synth.new_tokens(w, 1, step)).reshape(L, B, H, 1, d)
        cg.kv_append_paged(0, L, kn, vn, pos, pt, Gd, shp, c, kpool, vpool, err)
        cg.kv_append_step(0, L, kn, vn, pos, Gd, shp, c, kc, vc, err_flag=err)
        pos.add_(1)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for s, pool, cont in ((0, kpool, kc), (1, vpool, vc)):
        got = _gather(cache_to_host(pool, oc, s), table, P)
        want = cache_to_host(cont, oc, s)
        for key in ("codes", "side"):
            if want[key] is not None:
                np.testing.assert_array_equal(got[key][:, :, :, T:T + 3], want[key][:, :, :, T:T + 3])
    # an append past the table flags and writes nothing
    pos.fill_(maxp * P)
    cg.kv_append_paged(0, L, kn, vn, pos, pt, Gd, shp, c, kpool, vpool, err)
    torch.cuda.synchronize()
    assert int(err.item()) == cg.CG_FLAG_POS_RANGE
