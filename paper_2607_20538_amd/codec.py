"""ctypes binding of the codec library's C ABI (include/codec_gauge.h).

Argument marshalling only: every step of the codec runs in the HIP library.  Functions
carry the C names (gauge_make, kv_encode, kv_decode, kv_append_step, cache_bytes,
gauge_device_bytes) and accept torch tensors for device buffers; the stream defaults to
torch's current stream.  A missing library raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcodecgauge.so")

CG_OK, CG_ERR_ARG, CG_ERR_SHAPE, CG_ERR_ALIGN, CG_ERR_UNSUPPORTED, CG_ERR_NOT_ORTHOGONAL, CG_ERR_CAPACITY, \
    CG_ERR_DEVICE = range(8)
CG_FLAG_NONFINITE, CG_FLAG_SIDE_OVERFLOW, CG_FLAG_POS_RANGE = 1, 2, 4
GAUGE_IDENTITY, GAUGE_HAAR, GAUGE_DCT2, GAUGE_HADAMARD, GAUGE_EXPM, GAUGE_USER = range(6)
PASSTHROUGH, BLOCK_UNIFORM, KIVI, ZFP = 0, 1, 2, 3
DTYPE_BF16, DTYPE_F32 = 0, 1

EXPORTS = ["cg_status_str", "gauge_device_bytes", "gauge_make", "cache_bytes", "kv_encode", "kv_decode",
           "kv_append_step", "spectral_workspace_bytes", "kv_spectral_stats", "gauge_grad_workspace_bytes",
           "kv_gauge_grad", "attend_workspace_bytes", "kv_attend",
           "kv_attend_noalloc",
           "attend_paged_workspace_bytes", "kv_attend_paged", "kv_encode_paged", "kv_append_paged", "cg_selftest",
           "cg_stream_probe"]


class GaugeShape(C.Structure):
    _fields_ = [("L", C.c_int32), ("H", C.c_int32), ("d", C.c_int32), ("g", C.c_int32)]


class PageTable(C.Structure):
    _fields_ = [("pages", C.c_void_p), ("max_pages", C.c_int32), ("page_size", C.c_int32)]


class CodecStruct(C.Structure):
    _fields_ = [("backend", C.c_int32), ("bits", C.c_int32), ("block_c", C.c_int32), ("key_tokens", C.c_int32),
                ("val_channels", C.c_int32), ("residual", C.c_int32), ("block_t", C.c_int32)]


class KvView(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("dtype", C.c_int32), ("L", C.c_int32), ("B", C.c_int32), ("H", C.c_int32),
                ("T", C.c_int32), ("d", C.c_int32), ("stride_l", C.c_int64), ("stride_b", C.c_int64),
                ("stride_h", C.c_int64), ("stride_t", C.c_int64)]


class CacheStruct(C.Structure):
    _fields_ = [("codes", C.c_void_p), ("side", C.c_void_p), ("residual", C.c_void_p), ("L", C.c_int32),
                ("B", C.c_int32), ("H", C.c_int32), ("T_cap", C.c_int32), ("d", C.c_int32), ("len", C.c_int32)]


class CodecError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {status_str(status)} (status {status})")
        self.status = status


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2607_20538_amd/build.py")
        L = C.CDLL(LIB_PATH)
        p, i32, u64 = C.c_void_p, C.c_int32, C.c_uint64
        L.cg_status_str.argtypes = [i32]
        L.cg_status_str.restype = C.c_char_p
        L.gauge_device_bytes.argtypes = [GaugeShape]
        L.gauge_device_bytes.restype = C.c_size_t
        L.gauge_make.argtypes = [i32, GaugeShape, u64, p, p, p, p]
        L.gauge_make.restype = i32
        L.cache_bytes.argtypes = [C.POINTER(CodecStruct), i32, i32, i32, i32, i32, i32, p, p, p]
        L.cache_bytes.restype = i32
        L.kv_encode.argtypes = [i32, C.POINTER(KvView), p, GaugeShape, C.POINTER(CodecStruct),
                                C.POINTER(CacheStruct), i32, p, p]
        L.kv_encode.restype = i32
        L.kv_decode.argtypes = [i32, C.POINTER(CacheStruct), p, GaugeShape, C.POINTER(CodecStruct), p, i32,
                                C.POINTER(KvView), p, p]
        L.kv_decode.restype = i32
        L.kv_append_step.argtypes = [i32, i32, C.POINTER(KvView), C.POINTER(KvView), p, p, GaugeShape,
                                     C.POINTER(CodecStruct), C.POINTER(CacheStruct), C.POINTER(CacheStruct),
                                     C.POINTER(KvView), C.POINTER(KvView), p, p]
        L.kv_append_step.restype = i32
        L.spectral_workspace_bytes.argtypes = [GaugeShape, i32]
        L.spectral_workspace_bytes.restype = C.c_size_t
        L.kv_spectral_stats.argtypes = [i32, C.POINTER(KvView), p, GaugeShape, i32, C.c_float, p, p, p, p]
        L.kv_spectral_stats.restype = i32
        L.gauge_grad_workspace_bytes.argtypes = [GaugeShape, i32, i32, i32]
        L.gauge_grad_workspace_bytes.restype = C.c_size_t
        L.kv_gauge_grad.argtypes = [i32, C.POINTER(KvView), p, p, GaugeShape, i32, C.c_float, C.c_float, C.c_float, p,
                                    p, p, p]
        L.kv_gauge_grad.restype = i32
        L.attend_workspace_bytes.argtypes = [GaugeShape, i32, i32, i32, i32]
        L.attend_workspace_bytes.restype = C.c_size_t
        L.kv_attend.argtypes = [i32, i32, C.POINTER(KvView), C.POINTER(CacheStruct), C.POINTER(CacheStruct), p,
                                GaugeShape, C.POINTER(CodecStruct), p, C.c_float, C.POINTER(KvView), p, p, p]
        L.kv_attend.restype = i32
        L.kv_attend_noalloc.argtypes = [i32, i32, C.POINTER(KvView), C.POINTER(CacheStruct), C.POINTER(CacheStruct),
                                        p, GaugeShape, C.POINTER(CodecStruct), p, C.c_float, C.POINTER(KvView), p, p]
        L.kv_attend_noalloc.restype = i32
        L.attend_paged_workspace_bytes.argtypes = [GaugeShape, i32, i32, i32, i32, i32]
        L.attend_paged_workspace_bytes.restype = C.c_size_t
        L.kv_attend_paged.argtypes = [i32, i32, C.POINTER(KvView), C.POINTER(CacheStruct), C.POINTER(CacheStruct),
                                      C.POINTER(PageTable), p, GaugeShape, C.POINTER(CodecStruct), p, C.c_float,
                                      C.POINTER(KvView), p, p, p]
        L.kv_attend_paged.restype = i32
        L.kv_encode_paged.argtypes = [i32, C.POINTER(KvView), C.POINTER(PageTable), p, GaugeShape,
                                      C.POINTER(CodecStruct), C.POINTER(CacheStruct), i32, p, p]
        L.kv_encode_paged.restype = i32
        L.kv_append_paged.argtypes = [i32, i32, C.POINTER(KvView), C.POINTER(KvView), p, C.POINTER(PageTable), p,
                                      GaugeShape, C.POINTER(CodecStruct), C.POINTER(CacheStruct),
                                      C.POINTER(CacheStruct), p, p]
        L.kv_append_paged.restype = i32
        L.cg_selftest.argtypes = [i32, p, p]
        L.cg_selftest.restype = i32
        L.cg_stream_probe.argtypes = [p, C.c_int64, p, C.c_int64, p]
        L.cg_stream_probe.restype = i32
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().cg_status_str(int(status)).decode()


def _check(fn: str, rc: int):
    if rc != CG_OK:
        raise CodecError(fn, rc)


@dataclasses.dataclass(frozen=True)
class Codec:
    backend: int = BLOCK_UNIFORM
    bits: int = 4
    block_c: int = 64
    key_tokens: int = 32
    val_channels: int = 64
    residual: int = 128
    block_t: int = 1

    def struct(self) -> CodecStruct:
        return CodecStruct(self.backend, self.bits, self.block_c, self.key_tokens, self.val_channels, self.residual,
                           self.block_t)


def shape(L: int, H: int, d: int, g: int) -> GaugeShape:
    return GaugeShape(L, H, d, g)


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return int(stream)
    import torch

    if torch.cuda.is_available():
        return torch.cuda.current_stream().cuda_stream
    return None


def view(t) -> KvView:
    """cg_kv_view of a torch tensor [L][B][H][T][d] (bf16 or float32, channel stride 1)."""
    import torch

    if t.dim() != 5 or t.stride(4) != 1:
        raise ValueError("KV view needs a [L][B][H][T][d] tensor with unit channel stride")
    dt = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}[t.dtype]
    L_, B, H, T, d = t.shape
    s = t.stride()
    return KvView(t.data_ptr(), dt, L_, B, H, T, d, s[0], s[1], s[2], s[3])


# ------------------------------------------------------------------------------------------
# entry points
# ------------------------------------------------------------------------------------------

def gauge_device_bytes(shp: GaugeShape) -> int:
    return int(lib().gauge_device_bytes(shp))


def gauge_make(kind: int, shp: GaugeShape, seed: int = 0, params: np.ndarray | None = None, G_host=True,
               G_dev=None, stream=None):
    """Returns (G_host float32 [L][2][H][R][g][g] or None, G_dev)."""
    R = shp.d // shp.g
    host = np.zeros((shp.L, 2, shp.H, R, shp.g, shp.g), dtype=np.float32) if G_host is True else G_host
    par = None if params is None else np.ascontiguousarray(params, dtype=np.float32)
    rc = lib().gauge_make(kind, shp, seed, None if par is None else par.ctypes.data,
                          None if host is None else host.ctypes.data, _ptr(G_dev), _stream(stream))
    _check("gauge_make", rc)
    return host, G_dev


def alloc_gauge(shp: GaugeShape, device="cuda"):
    import torch

    return torch.empty(gauge_device_bytes(shp), dtype=torch.uint8, device=device)


def cache_bytes(codec: Codec, s: int, L: int, B: int, H: int, T_cap: int, d: int):
    c, sd, r = C.c_size_t(), C.c_size_t(), C.c_size_t()
    cs = codec.struct()
    rc = lib().cache_bytes(C.byref(cs), s, L, B, H, T_cap, d, C.addressof(c), C.addressof(sd), C.addressof(r))
    _check("cache_bytes", rc)
    return c.value, sd.value, r.value


class Cache:
    """Device buffers of one compressed K or V cache (flat uint8 tensors)."""

    def __init__(self, codec: Codec, s: int, L: int, B: int, H: int, T_cap: int, d: int, device="cuda"):
        import torch

        nc, ns, nr = cache_bytes(codec, s, L, B, H, T_cap, d)
        mk = lambda n: torch.zeros(max(n, 16), dtype=torch.uint8, device=device) if n else None
        self.codes, self.side, self.residual = mk(nc), mk(ns), mk(nr)
        self.nbytes = (nc, ns, nr)
        self.L, self.B, self.H, self.T_cap, self.d = L, B, H, T_cap, d
        self.len = 0

    def struct(self) -> CacheStruct:
        return CacheStruct(_ptr(self.codes), _ptr(self.side), _ptr(self.residual), self.L, self.B, self.H,
                           self.T_cap, self.d, self.len)


def kv_encode(s: int, X, G_dev, shp: GaugeShape, codec: Codec, cache: Cache, t0: int = 0, err_flag=None,
              stream=None):
    v, cs, ks = view(X), codec.struct(), cache.struct()
    rc = lib().kv_encode(s, C.byref(v), _ptr(G_dev), shp, C.byref(cs), C.byref(ks), t0, _ptr(err_flag),
                         _stream(stream))
    _check("kv_encode", rc)


def kv_decode(s: int, cache: Cache, G_dev, shp: GaugeShape, codec: Codec, t0: int, Xhat, err_flag=None,
              stream=None, lens=None):
    """lens: optional device int32 tensor [B] of per-row lengths (else every row holds cache.len)."""
    v, cs, ks = view(Xhat), codec.struct(), cache.struct()
    rc = lib().kv_decode(s, C.byref(ks), _ptr(G_dev), shp, C.byref(cs), _ptr(lens), t0, C.byref(v),
                         _ptr(err_flag), _stream(stream))
    _check("kv_decode", rc)


def cg_selftest(which: int, mismatches_dev, stream=None):
    """Adds the mismatch count of device self-test `which` to the uint64 device tensor."""
    rc = lib().cg_selftest(which, _ptr(mismatches_dev), _stream(stream))
    _check("cg_selftest", rc)


def cg_stream_probe(src, read_bytes: int, dst, write_bytes: int, stream=None):
    """Streams `read_bytes` of device tensor `src` and writes `write_bytes` into `dst` in one
    kernel (the HBM ceiling of that read / write mix; `dst` is left unspecified)."""
    if src.nbytes < read_bytes or (write_bytes and dst.nbytes < write_bytes):
        raise ValueError("cg_stream_probe: buffer smaller than the byte count")
    rc = lib().cg_stream_probe(_ptr(src), read_bytes, _ptr(dst), write_bytes, _stream(stream))
    _check("cg_stream_probe", rc)


def kv_append_step(l0: int, l1: int, k_new, v_new, pos, G_dev, shp: GaugeShape, codec: Codec, kc: Cache,
                   vc: Cache, k_hist=None, v_hist=None, err_flag=None, stream=None):
    kn, vn, cs, kcs, vcs = view(k_new), view(v_new), codec.struct(), kc.struct(), vc.struct()
    kh = None if k_hist is None else C.byref(view(k_hist))
    vh = None if v_hist is None else C.byref(view(v_hist))
    rc = lib().kv_append_step(l0, l1, C.byref(kn), C.byref(vn), _ptr(pos), _ptr(G_dev), shp, C.byref(cs),
                              C.byref(kcs), C.byref(vcs), kh, vh, _ptr(err_flag), _stream(stream))
    _check("kv_append_step", rc)


def spectral_workspace_bytes(shp: GaugeShape, block_t: int) -> int:
    return int(lib().spectral_workspace_bytes(shp, block_t))


def kv_spectral_stats(s: int, X, G_dev, shp: GaugeShape, block_t: int, tau: float, workspace, stats, energy=None,
                      stream=None):
    """Spectral statistics of G X (section 4.2) into the device float64 tensors stats [L][4] and,
    if given, energy [L][block_t][d]; workspace: device buffer of spectral_workspace_bytes."""
    v = view(X)
    rc = lib().kv_spectral_stats(s, C.byref(v), _ptr(G_dev), shp, block_t, tau, _ptr(workspace), _ptr(stats),
                                 _ptr(energy), _stream(stream))
    _check("kv_spectral_stats", rc)


def gauge_grad_workspace_bytes(shp: GaugeShape, B: int, T: int, block_t: int) -> int:
    return int(lib().gauge_grad_workspace_bytes(shp, B, T, block_t))


def kv_gauge_grad(s: int, X, A, G_dev, shp: GaugeShape, block_t: int, tau: float, lambda_f: float, lambda_r: float,
                  workspace, stats, grad, stream=None):
    """Gradient of the training objective (section 4.2) with respect to the generators A (device
    float32 [L][2][H][R][g][g], G = exp(A - A^T)) into the device float64 tensors grad
    [L][H][R][g][g] and stats [L][4]; workspace: device buffer of gauge_grad_workspace_bytes."""
    v = view(X)
    rc = lib().kv_gauge_grad(s, C.byref(v), _ptr(A), _ptr(G_dev), shp, block_t, tau, lambda_f, lambda_r,
                             _ptr(workspace), _ptr(stats), _ptr(grad), _stream(stream))
    _check("kv_gauge_grad", rc)


def attend_workspace_bytes(shp: GaugeShape, nl: int, B: int, Hq: int, T_cap: int) -> int:
    return int(lib().attend_workspace_bytes(shp, nl, B, Hq, T_cap))


def kv_attend(l0: int, l1: int, q, kc: Cache, vc: Cache, G_dev, shp: GaugeShape, codec: Codec, lens, scale: float,
              out, workspace=None, err_flag=None, stream=None):
    """Decode-phase attention of q [l1-l0][B][Hq][1][d] over the compressed caches into out (same
    shape); lens: device int32 [B] positions per row, or None for the caches' len."""
    qv, ov, cs, kcs, vcs = view(q), view(out), codec.struct(), kc.struct(), vc.struct()
    rc = lib().kv_attend(l0, l1, C.byref(qv), C.byref(kcs), C.byref(vcs), _ptr(G_dev), shp, C.byref(cs), _ptr(lens),
                         float(scale), C.byref(ov), _ptr(workspace), _ptr(err_flag), _stream(stream))
    _check("kv_attend", rc)


def kv_attend_noalloc(l0: int, l1: int, q, kc: Cache, vc: Cache, G_dev, shp: GaugeShape, codec: Codec, lens,
                      scale: float, out, err_flag=None, stream=None):
    """kv_attend without a workspace: split rows' partials go to the library's device scratch."""
    qv, ov, cs, kcs, vcs = view(q), view(out), codec.struct(), kc.struct(), vc.struct()
    rc = lib().kv_attend_noalloc(l0, l1, C.byref(qv), C.byref(kcs), C.byref(vcs), _ptr(G_dev), shp, C.byref(cs),
                                 _ptr(lens), float(scale), C.byref(ov), _ptr(err_flag), _stream(stream))
    _check("kv_attend_noalloc", rc)


def page_table(pages, page_size: int) -> PageTable:
    """cg_page_table of a device int32 tensor pages [B][max_pages]."""
    return PageTable(_ptr(pages), int(pages.shape[1]), int(page_size))


def attend_paged_workspace_bytes(shp: GaugeShape, nl: int, B: int, Hq: int, max_pages: int, page_size: int) -> int:
    return int(lib().attend_paged_workspace_bytes(shp, nl, B, Hq, max_pages, page_size))


def kv_attend_paged(l0: int, l1: int, q, kc: Cache, vc: Cache, pt: PageTable, G_dev, shp: GaugeShape, codec: Codec,
                    lens, scale: float, out, workspace=None, err_flag=None, stream=None):
    """kv_attend over page pools kc / vc (their B counts pages, T_cap = page size) through pt."""
    qv, ov, cs, kcs, vcs = view(q), view(out), codec.struct(), kc.struct(), vc.struct()
    rc = lib().kv_attend_paged(l0, l1, C.byref(qv), C.byref(kcs), C.byref(vcs), C.byref(pt), _ptr(G_dev), shp,
                               C.byref(cs), _ptr(lens), float(scale), C.byref(ov), _ptr(workspace), _ptr(err_flag),
                               _stream(stream))
    _check("kv_attend_paged", rc)


def kv_encode_paged(s: int, X, pt: PageTable, G_dev, shp: GaugeShape, codec: Codec, cache: Cache, t0: int = 0,
                    err_flag=None, stream=None):
    v, cs, ks = view(X), codec.struct(), cache.struct()
    rc = lib().kv_encode_paged(s, C.byref(v), C.byref(pt), _ptr(G_dev), shp, C.byref(cs), C.byref(ks), t0,
                               _ptr(err_flag), _stream(stream))
    _check("kv_encode_paged", rc)


def kv_append_paged(l0: int, l1: int, k_new, v_new, pos, pt: PageTable, G_dev, shp: GaugeShape, codec: Codec,
                    kc: Cache, vc: Cache, err_flag=None, stream=None):
    kn, vn, cs, kcs, vcs = view(k_new), view(v_new), codec.struct(), kc.struct(), vc.struct()
    rc = lib().kv_append_paged(l0, l1, C.byref(kn), C.byref(vn), _ptr(pos), C.byref(pt), _ptr(G_dev), shp,
                               C.byref(cs), C.byref(kcs), C.byref(vcs), _ptr(err_flag), _stream(stream))
    _check("kv_append_paged", rc)
