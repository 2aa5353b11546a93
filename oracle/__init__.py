"""fp64 CPU oracle for sparse absorbed-MLA partial attention and the LSE merge.

TEST INFRASTRUCTURE ONLY.  The tests, the smoke check and the benchmark's
CPU-baseline leg call it; the product path (the HIP library and its binding)
never imports it, and it imports nothing from the product.

The arithmetic lives in `oracle.c` (plain C, double precision, two-pass
softmax); this module only marshals numpy arrays through ctypes.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

KV_BF16 = 0
KV_E4M3FN = 1
DLAT = 512
DPE = 64
BLOCK = 64


def _load(path=None):
    global _lib
    if path is not None:
        lib = ctypes.CDLL(path)
    else:
        if _lib is not None:
            return _lib
        # (re)build when the library is missing or older than its source
        if (not os.path.exists(_build.LIB)
                or os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC)):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
    lib.oracle_partial.restype = i32
    lib.oracle_partial.argtypes = [i32, i32, i32, i64, i32, i32, vp, vp, i32, vp, vp, vp, vp,
                                   vp, vp, i32, i32, dbl, vp, vp, vp, vp, i32]
    lib.oracle_merge.restype = i32
    lib.oracle_merge.argtypes = [i32, i64, i32, vp, vp, vp, vp, i32]
    lib.oracle_bf16_to_f64.restype = dbl
    lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_e4m3fn_to_f64.restype = dbl
    lib.oracle_e4m3fn_to_f64.argtypes = [ctypes.c_uint8]
    if path is None:
        _lib = lib
    return lib


def default_threads():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def _ptr(a):
    return None if a is None else a.ctypes.data


def bf16_to_f64(bits):
    return _load().oracle_bf16_to_f64(int(bits))


def e4m3fn_to_f64(code):
    return _load().oracle_e4m3fn_to_f64(int(code))


def partial(q_lat, q_pe, ckv, kpe, table, sel, scale, ckv_scale=None, kpe_scale=None,
            n_threads=None, lib=None, tokens=False, stats=False):
    """Oracle partial attention.

    q_lat uint16 [R, Mq, H, 512] and q_pe uint16 [R, Mq, H, 64] hold bf16 bits;
    ckv [P, 64, 512] / kpe [P, 64, 64] hold bf16 bits (uint16) or e4m3fn codes
    (uint8, with float32 per-block scales ckv_scale / kpe_scale [P]);
    table int32 [R, NB]; sel int32 [R, K] (one selection per job) or
    [R, Mq, K] (one per query row); -1 = empty slot.  A slot names a logical
    block (all 64 tokens), or with tokens=True one logical token s (token
    s % 64 of logical block s // 64).
    Returns (out float64 [R, Mq, H, 512], lse float64 [R, Mq, H]); with
    stats=True also the largest score M and the denominator l = sum exp(s - M)
    of every row (float64 [R, Mq, H]; -inf and 0 for an empty row).
    """
    lib = lib or _load()
    q_lat = np.ascontiguousarray(q_lat, dtype=np.uint16)
    q_pe = np.ascontiguousarray(q_pe, dtype=np.uint16)
    R, Mq, H, dl = q_lat.shape
    assert dl == DLAT and q_pe.shape == (R, Mq, H, DPE)
    if ckv.dtype == np.uint16:
        kind = KV_BF16
        ckv = np.ascontiguousarray(ckv)
        kpe = np.ascontiguousarray(kpe, dtype=np.uint16)
        cs = ks = None
    else:
        kind = KV_E4M3FN
        ckv = np.ascontiguousarray(ckv, dtype=np.uint8)
        kpe = np.ascontiguousarray(kpe, dtype=np.uint8)
        cs = np.ascontiguousarray(ckv_scale, dtype=np.float32)
        ks = np.ascontiguousarray(kpe_scale, dtype=np.float32)
    P = ckv.shape[0]
    assert ckv.shape == (P, BLOCK, DLAT) and kpe.shape == (P, BLOCK, DPE)
    table = np.ascontiguousarray(table, dtype=np.int32)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    NB, K = table.shape[1], sel.shape[-1]
    per_row = sel.ndim == 3
    assert table.shape[0] == R and sel.shape[0] == R and (not per_row or sel.shape[1] == Mq)
    out = np.zeros((R, Mq, H, DLAT), np.float64)
    lse = np.zeros((R, Mq, H), np.float64)
    mx = np.zeros((R, Mq, H), np.float64) if stats else None
    den = np.zeros((R, Mq, H), np.float64) if stats else None
    rc = lib.oracle_partial(R, Mq, H, P, NB, K, _ptr(q_lat), _ptr(q_pe), kind, _ptr(ckv),
                            _ptr(kpe), _ptr(cs), _ptr(ks), _ptr(table), _ptr(sel),
                            int(per_row), int(bool(tokens)), float(scale), _ptr(out), _ptr(lse),
                            _ptr(mx), _ptr(den), int(n_threads or default_threads()))
    if rc != 0:
        raise ValueError("oracle_partial: invalid selected id or table entry")
    return (out, lse, mx, den) if stats else (out, lse)


def merge(parts_o, parts_lse, n_threads=None, lib=None):
    """Oracle merge of partials: parts_o [n, ..., dv], parts_lse [n, ...].

    Returns (out float64 [..., dv], lse float64 [...]).
    """
    lib = lib or _load()
    o = np.ascontiguousarray(parts_o, dtype=np.float64)
    lam = np.ascontiguousarray(parts_lse, dtype=np.float64)
    n = o.shape[0]
    dv = o.shape[-1]
    assert lam.shape == o.shape[:-1]
    n_rows = int(np.prod(lam.shape[1:], dtype=np.int64))
    out = np.zeros(o.shape[1:], np.float64)
    lse = np.zeros(lam.shape[1:], np.float64)
    rc = lib.oracle_merge(n, n_rows, dv, _ptr(o), _ptr(lam), _ptr(out), _ptr(lse),
                          int(n_threads or default_threads()))
    if rc != 0:
        raise ValueError("oracle_merge: invalid arguments")
    return out, lse
