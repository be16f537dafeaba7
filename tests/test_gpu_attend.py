"""GPU parity of the fused decode-phase attention (kv_attend, through the C ABI) against the
CPU oracle's attention over the decoded caches (oracle.attend: kv_decode in binary32, then
softmax(scale q Khat^T) Vhat in binary64).

The caches are the oracle's own encodings copied to the device, so the check isolates the
attention path.  Tolerance, per (layer, batch row, query head): |o - o_ref| <= 1e-4 max|Vhat|
over the row's positions.  Both sides compute every score from the same dequantised values;
the kernel's binary32 scores differ from the binary64 reference by a few units of 2^-24 of
sum |q'_c zhat_c| (the dot-product rounding, about 1e-6 of the score scale), which the softmax
turns into at most that much of 2 max|Vhat| in the output, plus the binary32 rounding of the
value sums; 1e-4 max|Vhat| leaves a margin of about 10x at |s| ~ 20.  bf16 outputs add one
bf16 rounding of the reference (2^-8 relative)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_dev, cache_to_dev, out_host, to_cg, x_f64

pytestmark = pytest.mark.gpu

ATT_TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


@pytest.fixture(params=["fast", "generic"])
def kernels(request, monkeypatch):
    """Run a case on the default dispatch and on the general kernel."""
    if request.param == "generic":
        monkeypatch.setenv("CG_KERNELS", "generic")
    else:
        monkeypatch.delenv("CG_KERNELS", raising=False)
    return request.param


def _encode_rows(oc, s, X, G, T_cap, lens):
    """The oracle's cache of a batch whose row b holds lens[b] tokens (rows encoded one by one,
    so that KIVI windows and staged tiles hold what a cache of that length holds)."""
    rows = [O.kv_encode(oc, s, np.ascontiguousarray(X[:, b:b + 1, :, : max(n, 1)]), G, T_cap=T_cap)[0]
            for b, n in enumerate(lens)]
    return {k: None if rows[0][k] is None else np.concatenate([r[k] for r in rows], axis=1) for k in rows[0]}


def _setup(oc, T, T_cap, L=1, B=2, H=2, d=128, g=32, grp=4, kind=O.GAUGE_HAAR, seed=0xA77, lens=None):
    w = synth.Workload("att", L=L, B=B, H=H, T=T, d=d, dtype="bf16", g=g, backend="bu", bits=4, data_seed=seed)
    K, V = synth.kv_tensor(w, 0), synth.kv_tensor(w, 1)
    G = O.gauge_make(kind, L, H, d, g, seed=seed + 1)
    shp = cg.shape(L, H, d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_USER, shp, params=G, G_host=None, G_dev=Gd)
    lens = [T] * B if lens is None else [min(n, T) for n in lens]
    kh = _encode_rows(oc, 0, K, G, T_cap, lens)
    vh = _encode_rows(oc, 1, V, G, T_cap, lens)
    kd = cache_to_dev(kh, oc, 0, L, B, H, T_cap, d, len_=T)
    vd = cache_to_dev(vh, oc, 1, L, B, H, T_cap, d, len_=T)
    q = synth.queries(w, H * grp)
    # the oracle takes the queries' values (bf16 values are exact in binary32)
    return dict(G=G, Gd=Gd, shp=shp, kh=kh, vh=vh, kd=kd, vd=vd, q=q, qf=x_f64(q).astype(np.float32), w=w)


def _attend_gpu(st, oc, lens, scale, out_dtype=torch.float32, lens_dev=True, l0=0, l1=None):
    q = st["q"]
    L_, B, Hq, d = q.shape
    l1 = L_ if l1 is None else l1
    qd = bf16_dev(q[l0:l1]).reshape(l1 - l0, B, Hq, 1, d)
    out = torch.full((l1 - l0, B, Hq, 1, d), float("nan"), dtype=out_dtype, device="cuda")
    ws_n = cg.attend_workspace_bytes(st["shp"], l1 - l0, B, Hq, st["kd"].T_cap)
    ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ln = torch.tensor(lens, dtype=torch.int32, device="cuda") if lens_dev else None
    cg.kv_attend(l0, l1, qd, st["kd"], st["vd"], st["Gd"], st["shp"], to_cg(oc), ln, scale, out, ws, err)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()[:, :, :, 0]
    return o, int(err.item())


def _check(got, ref, vh_max, bf16_out=False):
    assert np.isfinite(got).all()
    tol = np.broadcast_to(ATT_TOL * vh_max[..., None], ref.shape)
    if bf16_out:
        tol = tol + np.abs(ref) * 2.0 ** -8
    err = np.abs(got - ref)
    assert (err <= tol).all(), f"max err {err.max():.3e} (tolerance at argmax {tol.flat[err.argmax()]:.3e})"


def _vmax(st, oc, lens, grp):
    """max |Vhat| over each row's positions, per (layer, batch, query head)."""
    Tm = max(max(lens), 1)
    Vh = O.kv_decode(oc, 1, st["G"], st["vh"], 0, Tm, lens=lens, out_bf16=False)
    L_, B, H = Vh.shape[:3]
    m = np.zeros((L_, B, H * grp))
    for b in range(B):
        if lens[b]:
            m[:, b] = np.repeat(np.abs(Vh[:, b, :, : lens[b]]).max(axis=(2, 3)), grp, axis=1)
    return m


CASES = [
    # (id, codec, g, T, T_cap, lens)
    ("bu4-n32-g32", O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=32), 32, 300, 320, [300, 177]),
    ("bu6-n64-g128", O.Codec(backend=O.BLOCK_UNIFORM, bits=6, block_c=64), 128, 333, 352, [333, 64]),
    ("bu3-n64-g16", O.Codec(backend=O.BLOCK_UNIFORM, bits=3, block_c=64), 16, 257, 288, [257, 1]),
    ("bu2-n128-g64", O.Codec(backend=O.BLOCK_UNIFORM, bits=2, block_c=128), 64, 200, 224, [150, 200]),
    ("bu8-n64-g32", O.Codec(backend=O.BLOCK_UNIFORM, bits=8, block_c=64), 32, 100, 128, [100, 99]),
    ("kivi3", O.Codec(backend=O.KIVI, bits=3, key_tokens=32, val_channels=64, residual=64), 32, 300, 320, [300, 150]),
    # KIVI on the matrix cores at every width: rows wholly in the window (100, and 159 = window +
    # 31), a row with one key group, windows of 32 and 128 positions, two splits per row
    ("kivi2-g128", O.Codec(backend=O.KIVI, bits=2, key_tokens=32, val_channels=64, residual=128), 128, 420, 448,
     [420, 100]),
    ("kivi4-g16", O.Codec(backend=O.KIVI, bits=4, key_tokens=32, val_channels=64, residual=128), 16, 300, 320,
     [300, 161]),
    ("kivi6-g64", O.Codec(backend=O.KIVI, bits=6, key_tokens=32, val_channels=64, residual=32), 64, 260, 288, [260, 33]),
    ("kivi8-g32", O.Codec(backend=O.KIVI, bits=8, key_tokens=32, val_channels=64, residual=128), 32, 200, 224,
     [200, 159]),
    ("tile4-16", O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64, block_t=16), 128, 250, 256, [250, 200]),
    # tiles with 128-channel blocks (eight query heads per workgroup), a row shorter than one tile
    # (staged positions only) and a row ending on a tile boundary
    ("tile6-n128", O.Codec(backend=O.BLOCK_UNIFORM, bits=6, block_c=128, block_t=16), 128, 200, 224, [9, 192]),
    ("tile3-n64", O.Codec(backend=O.BLOCK_UNIFORM, bits=3, block_c=64, block_t=16), 128, 161, 192, [161, 47]),
    ("pass", O.Codec(backend=O.PASSTHROUGH), 32, 130, 160, [130, 77]),
]


@pytest.mark.parametrize("cid,oc,g,T,T_cap,lens", CASES, ids=[c[0] for c in CASES])
def test_attend_matches_oracle(kernels, cid, oc, g, T, T_cap, lens):
    st = _setup(oc, T, T_cap, g=g, lens=lens)
    scale = 1.0 / np.sqrt(128)
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale)
    assert err == 0
    _check(got, ref, _vmax(st, oc, lens, 4))


def test_attend_host_length_bf16_output_and_layer_range(kernels):
    """lens = NULL (every row holds the caches' len), bf16 output, a sub-range of layers."""
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64)
    st = _setup(oc, 190, 192, L=3, g=128)
    scale = 0.1
    lens = [190, 190]
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale, out_dtype=torch.bfloat16, lens_dev=False, l0=1, l1=3)
    assert err == 0
    _check(got, ref[1:3], _vmax(st, oc, lens, 4)[1:3], bf16_out=True)


@pytest.mark.parametrize("grp,d,g", [(1, 128, 32), (12, 128, 128), (2, 128, 8), (4, 64, 16), (8, 256, 64)])
def test_attend_head_groupings_and_dims(kernels, grp, d, g):
    """Multi-head (grp = 1), more query heads per KV head than one workgroup takes (12), and
    other head dimensions."""
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=32 if d == 64 else 64)
    st = _setup(oc, 97, 128, d=d, g=g, grp=grp, B=1)
    lens = [97]
    scale = 1.0 / np.sqrt(d)
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale)
    assert err == 0
    _check(got, ref, _vmax(st, oc, lens, grp))


def test_attend_split_rows_and_edges(kernels):
    """Long rows over few (layer, batch, head) rows are split over the positions and combined;
    a row with no positions gives zeros; a length beyond the capacity flags and gives zeros."""
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64)
    T = 2500
    lens = [2500, 0, 1, 1800]
    st = _setup(oc, T, 2560, B=4, H=1, g=128, lens=lens)
    assert cg.attend_workspace_bytes(st["shp"], 1, 4, 4, 2560) > 0
    scale = 1.0 / np.sqrt(128)
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale)
    assert err == 0
    _check(got, ref, _vmax(st, oc, lens, 4))
    assert (got[:, 1] == 0).all()
    got2, err2 = _attend_gpu(st, oc, [2500, 2561, 1, 1800], scale)
    assert err2 == cg.CG_FLAG_POS_RANGE
    assert (got2[:, 1] == 0).all()
    np.testing.assert_array_equal(got2[:, [0, 2, 3]], got[:, [0, 2, 3]])


@pytest.mark.parametrize("bits,n", [(4, 64), (8, 128)])
def test_attend_split_rows_over_tiles(kernels, bits, n):
    """Token-channel tiles on rows long enough to be split over positions: the staged positions
    of a row fall into its last split and are merged with the other splits' partial results."""
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=n, block_t=16)
    lens = [2500, 0, 13, 1811]
    st = _setup(oc, 2500, 2560, B=4, H=1, g=128, lens=lens)
    scale = 1.0 / np.sqrt(128)
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale)
    assert err == 0
    _check(got, ref, _vmax(st, oc, lens, 4))
    assert (got[:, 1] == 0).all()


@pytest.mark.parametrize("bits,win", [(3, 128), (4, 32)])
def test_attend_split_rows_over_kivi_caches(kernels, bits, win):
    """KIVI caches on rows long enough to be split over positions: key groups in every split,
    the window's raw positions in the last one; an empty row, a row inside the window, and 12
    query heads per KV head (three query chunks of the matrix-core kernel)."""
    oc = O.Codec(backend=O.KIVI, bits=bits, key_tokens=32, val_channels=64, residual=win)
    lens = [2500, 0, 13, 1811]
    st = _setup(oc, 2500, 2560, B=4, H=1, g=32, grp=12, lens=lens)
    scale = 1.0 / np.sqrt(128)
    ref = O.attend(oc, st["G"], st["kh"], st["vh"], st["qf"], lens, scale)
    got, err = _attend_gpu(st, oc, lens, scale)
    assert err == 0
    _check(got, ref, _vmax(st, oc, lens, 12))
    assert (got[:, 1] == 0).all()


def test_attend_error_free_cache_equals_attention_on_x(kernels):
    """Passthrough backend with the identity gauge: the fused path is plain attention over the
    bf16 cache (torch's, in float64 on the CPU)."""
    oc = O.Codec(backend=O.PASSTHROUGH)
    st = _setup(oc, 180, 192, kind=O.GAUGE_IDENTITY, g=128, B=1)
    scale = 1.0 / np.sqrt(128)
    got, _ = _attend_gpu(st, oc, [180], scale)
    K = torch.from_numpy(x_f64(synth.kv_tensor(st["w"], 0)))[0, 0]   # [H][T][d]
    V = torch.from_numpy(x_f64(synth.kv_tensor(st["w"], 1)))[0, 0]
    q = torch.from_numpy(x_f64(st["q"]))[0, 0]                       # [Hq][d]
    ref = torch.nn.functional.scaled_dot_product_attention(
        q[:, None, :], K.repeat_interleave(4, dim=0), V.repeat_interleave(4, dim=0), scale=scale)[:, 0]
    vmax = V.abs().amax(dim=(1, 2)).repeat_interleave(4).numpy()
    _check(got[0, 0], ref.numpy(), vmax)
