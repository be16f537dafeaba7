"""The fused-encoder criterion of tests/_parity.py on planted differences (CPU only): it accepts a
cache that differs from the oracle's only where a z within the gauge tolerance can move it, and
rejects the plausible kernel mistakes."""
import numpy as np
import pytest

import oracle as O
from paper_2607_20538_amd import synth

from _parity import check_fused_codes


def _case(bits=4, kind=O.GAUGE_HAAR):
    w = synth.Workload("crit", L=1, B=1, H=1, T=64, d=128, dtype="bf16", g=32, backend="bu", bits=bits,
                       data_seed=77)
    G = O.gauge_make(kind, 1, 1, 128, 32, seed=5)
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=64)
    X = synth.kv_tensor(w, 0)
    orc, _ = O.kv_encode(oc, 0, X, G, T_cap=64)
    zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), 0, X, G, T_cap=64)
    return oc, orc, zo["codes"]


def _copy(c):
    return {k: (None if v is None else v.copy()) for k, v in c.items()}


def test_identical_cache_passes():
    oc, orc, z = _case()
    assert check_fused_codes(_copy(orc), orc, z, oc, 0, 128, 64)["code_frac"] == 0.0


def test_minimum_moved_one_ulp_with_its_scale_passes():
    """The GPU's z lands just above a binary16 grid point the exact minimum lies just below: the
    minimum rounds one ulp higher and the scale follows from that minimum (can be two ulps off)."""
    oc, orc, z = _case()
    got = _copy(orc)
    t, k = 9, 1
    zb = z[0, 0, 0, t, 64 * k:64 * k + 64].astype(np.float32)
    mn_bits = int(orc["side"][0, 0, 0, t, k, 0])
    mn_new = mn_bits - 1 if mn_bits & 0x8000 else mn_bits + 1          # one ulp toward +inf
    mn_val = np.array([mn_new], dtype=np.uint16).view(np.float16).astype(np.float32)[0]
    s32 = np.float32((zb.max() - mn_val) / np.float32(15))
    h = np.float16(s32)
    if np.float32(h) < s32:
        h = np.nextafter(h, np.float16(np.inf))
    got["side"][0, 0, 0, t, k] = [mn_new, np.array([h]).view(np.uint16)[0]]
    check_fused_codes(got, orc, z, oc, 0, 128, 64)


@pytest.mark.parametrize("mistake", ["scale_3ulp", "min_2ulp", "code_off_by_one", "code_off_by_two",
                                     "swapped_blocks"])
def test_plausible_mistakes_fail(mistake):
    oc, orc, z = _case()
    got = _copy(orc)
    if mistake == "scale_3ulp":
        got["side"][0, 0, 0, 5, 0, 1] += 3
    elif mistake == "min_2ulp":
        got["side"][0, 0, 0, 5, 0, 0] += 2
    elif mistake == "code_off_by_one":
        got["codes"][0, 0, 0, 3, 0] ^= 0x01          # lowest code of the row moved by one, not at a tie
    elif mistake == "code_off_by_two":
        got["codes"][0, 0, 0, 3, 0] ^= 0x02
    else:
        got["side"][0, 0, 0, 7] = got["side"][0, 0, 0, 7, ::-1].copy()
    with pytest.raises(AssertionError):
        check_fused_codes(got, orc, z, oc, 0, 128, 64)
