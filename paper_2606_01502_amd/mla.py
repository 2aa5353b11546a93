"""Python binding of libmla_sparse.so (C ABI in include/mla_sparse.h).

Argument marshalling only: torch tensors are described to the library by
pointer, dtype, shape and strides, and the current HIP stream is passed
along.  Every step of the computation runs in the library's HIP kernels;
there is no fallback, and a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
import struct

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmla_sparse.so")

DLAT, DPE, BLOCK, MAX_PARTS = 512, 64, 64, 64

MLA_OK = 0
MLA_ERR_INVALID_ARGUMENT = -1
MLA_ERR_UNSUPPORTED = -2
MLA_ERR_HIP = -3
MLA_ERR_OUT_OF_MEMORY = -4

DTYPE_BF16, DTYPE_FP8_E4M3FN, DTYPE_FP32, DTYPE_INT32 = 1, 2, 3, 4

EXPORTS = ("mla_sparse_partial_attn", "mla_sparse_partial_attn_ex",
           "mla_sparse_partial_attn_tokens", "mla_merge_partials", "mla_merge_partials_ex",
           "mla_last_error", "mla_version", "mla_primitive_costs", "mla_fetch_gather",
           "mla_fetch_splice", "mla_sparse_partial_attn_noalloc")


class MlaError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 4), ("stride", ctypes.c_int64 * 4),
                ("block_scale", ctypes.c_void_p)]


class CostModel(ctypes.Structure):
    _fields_ = [("probe_us", ctypes.c_double), ("route_bw_gbs", ctypes.c_double),
                ("compute_us", ctypes.c_double), ("merge_us", ctypes.c_double),
                ("pull_bw_gbs", ctypes.c_double), ("splice_us", ctypes.c_double),
                ("prefill_us", ctypes.c_double), ("layers", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class CostCase(ctypes.Structure):
    _fields_ = [("mq", ctypes.c_int64), ("chunk_tokens", ctypes.c_int64),
                ("q_bytes", ctypes.c_int64), ("p_bytes", ctypes.c_int64),
                ("kv_bytes", ctypes.c_int64)]


class Cost(ctypes.Structure):
    _fields_ = [("route_us", ctypes.c_double), ("fetch_us", ctypes.c_double),
                ("local_us", ctypes.c_double), ("choice", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("wire_crossover_mq", ctypes.c_double),
                ("wire_saving", ctypes.c_double), ("congestion_bw_gbs", ctypes.c_double),
                ("splice_crossover_tokens", ctypes.c_double)]


PRIMITIVES = ("route", "fetch", "local")
# the constants the paper measured (Sections 4.3 and 5.1; c in [0.5, 1.5])
PAPER_COST_MODEL = dict(probe_us=16.0, route_bw_gbs=25.0, compute_us=0.0, merge_us=0.0,
                        pull_bw_gbs=25.0, splice_us=3000.0, prefill_us=1.0, layers=27)


class PartialOpts(ctypes.Structure):
    _fields_ = [("n_splits", ctypes.c_int32), ("row_tile", ctypes.c_int32),
                ("out_format", ctypes.c_int32), ("reserved", ctypes.c_int32 * 5)]


OUT_FP32, OUT_BF16_WIRE = 0, 1


_lib = None


def load(path: str = LIB_PATH):
    """Load the library (once) and declare its entry points."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(Tensor)
    PP = ctypes.POINTER(P)
    vp = ctypes.c_void_p
    lib.mla_sparse_partial_attn.restype = ctypes.c_int
    lib.mla_sparse_partial_attn.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, P, vp]
    lib.mla_sparse_partial_attn_ex.restype = ctypes.c_int
    lib.mla_sparse_partial_attn_ex.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, P,
                                               ctypes.POINTER(PartialOpts), vp]
    lib.mla_sparse_partial_attn_tokens.restype = ctypes.c_int
    lib.mla_sparse_partial_attn_tokens.argtypes = lib.mla_sparse_partial_attn_ex.argtypes
    lib.mla_sparse_partial_attn_noalloc.restype = ctypes.c_int
    lib.mla_sparse_partial_attn_noalloc.argtypes = lib.mla_sparse_partial_attn_ex.argtypes
    lib.mla_merge_partials.restype = ctypes.c_int
    lib.mla_merge_partials.argtypes = [PP, PP, ctypes.c_int32, P, vp]
    lib.mla_merge_partials_ex.restype = ctypes.c_int
    lib.mla_merge_partials_ex.argtypes = [PP, PP, ctypes.c_int32, P, P, vp]
    lib.mla_fetch_gather.restype = ctypes.c_int
    lib.mla_fetch_gather.argtypes = [P, P, P, P, P, P, vp]
    lib.mla_fetch_splice.restype = ctypes.c_int
    lib.mla_fetch_splice.argtypes = [P, P, P, P, P, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_float, ctypes.c_int32, vp]
    lib.mla_primitive_costs.restype = ctypes.c_int
    lib.mla_primitive_costs.argtypes = [ctypes.POINTER(CostModel), ctypes.POINTER(CostCase),
                                        ctypes.POINTER(Cost)]
    lib.mla_last_error.restype = ctypes.c_char_p
    lib.mla_last_error.argtypes = []
    lib.mla_version.restype = ctypes.c_int32
    lib.mla_version.argtypes = []
    if path == LIB_PATH:
        _lib = lib
    return lib


_TORCH_DTYPES = {
    torch.bfloat16: DTYPE_BF16,
    torch.float32: DTYPE_FP32,
    torch.int32: DTYPE_INT32,
    torch.uint8: DTYPE_FP8_E4M3FN,
    torch.float8_e4m3fn: DTYPE_FP8_E4M3FN,
}


# mla_tensor_t packed field by field: data, dtype, ndim, shape[4], stride[4],
# block_scale (88 bytes, no padding on x86-64)
_PACK = struct.Struct("=Qii4q4qQ")
assert _PACK.size == ctypes.sizeof(Tensor)
_PAD = ((), (0,), (0, 0), (0, 0, 0), (0, 0, 0, 0))


def describe(t: torch.Tensor | None, block_scale: torch.Tensor | None = None) -> Tensor | None:
    """mla_tensor_t for a torch tensor (uint8 tensors are fp8-e4m3fn codes)."""
    if t is None:
        return None
    shape, stride = t.shape, t.stride()
    nd = len(shape)
    if nd > 4:
        raise ValueError("at most 4 dims")
    bs = 0
    if block_scale is not None:
        if block_scale.dtype != torch.float32 or not block_scale.is_contiguous():
            raise ValueError("block_scale must be contiguous float32")
        bs = block_scale.data_ptr()
    pad = _PAD[4 - nd]
    return Tensor.from_buffer_copy(_PACK.pack(t.data_ptr() if t.numel() else 0,
                                              _TORCH_DTYPES.get(t.dtype, 0), nd, *shape, *pad,
                                              *stride, *pad, bs))


def _on_one_gpu(*tensors):
    """Raise ValueError unless every given tensor lives on one CUDA (HIP)
    device: the library reads and writes device memory only, and a host
    tensor's address handed to a kernel would fault."""
    devs = {t.device for t in tensors if t is not None}
    bad = [d for d in devs if d.type != "cuda"]
    if bad:
        raise ValueError(f"tensors must be on the GPU, got {bad[0]}")
    if len(devs) > 1:
        raise ValueError(f"tensors must be on one device, got {sorted(map(str, devs))}")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(lib, st):
    if st != MLA_OK:
        raise MlaError(st, lib.mla_last_error().decode())


def _ref(d):
    return ctypes.byref(d) if d is not None else None


class _Prepared:
    """One library call with its arguments fixed: the descriptors are built
    once and the tensors they point to are kept alive, so each call costs
    one foreign call (for serving loops that reuse static buffers)."""

    def __init__(self, fn, args, keep, result):
        self._fn, self._args, self._keep, self.result = fn, args, keep, result

    def __call__(self):
        st = self._fn(*self._args)
        if st != MLA_OK:
            raise MlaError(st, load().mla_last_error().decode())
        return self.result


def _partial_args(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids, scale,
                  out_lat, out_lse, ckv_scale, kpe_scale, n_splits, row_tile, stream, wire=False):
    R = chunk_block_table.shape[0]  # jobs; q may hold fewer rows (R_q dividing R)
    _, Mq, H, _ = q_lat.shape
    if out_lat is None:
        out_lat = torch.empty((R, Mq, H, DLAT), dtype=torch.bfloat16 if wire else torch.float32,
                              device=q_lat.device)
    if out_lse is None:
        out_lse = torch.empty((R, Mq, H, 2) if wire else (R, Mq, H), dtype=torch.float32,
                              device=q_lat.device)
    _on_one_gpu(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids, out_lat,
                out_lse, ckv_scale, kpe_scale)
    opts = PartialOpts()
    opts.n_splits = int(n_splits)
    opts.row_tile = int(row_tile)
    opts.out_format = OUT_BF16_WIRE if wire else OUT_FP32
    descs = (describe(q_lat), describe(q_pe), describe(ckv_pool, ckv_scale),
             describe(kpe_pool, kpe_scale), describe(chunk_block_table), describe(sel_block_ids))
    outs = (describe(out_lat), describe(out_lse))
    args = tuple(_ref(d) for d in descs) + (ctypes.c_float(scale),) + \
        tuple(_ref(d) for d in outs) + (ctypes.byref(opts), _stream(stream))
    keep = (descs, outs, opts, q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table,
            sel_block_ids, ckv_scale, kpe_scale)
    return args, keep, (out_lat, out_lse)


def _partial_fn(lib, tokens, no_alloc):
    if tokens and no_alloc:
        raise ValueError("the allocation-free entry point takes block selections only")
    if no_alloc:
        return lib.mla_sparse_partial_attn_noalloc
    return lib.mla_sparse_partial_attn_tokens if tokens else lib.mla_sparse_partial_attn_ex


def prepare_partial(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids, scale,
                    out_lat=None, out_lse=None, ckv_scale=None, kpe_scale=None, n_splits=0,
                    row_tile=0, stream=None, tokens=False, no_alloc=False, wire=False):
    """sparse_partial_attn with every argument fixed, the stream included
    (the current one when None); calling the result launches the work and
    returns (out_lat, out_lse)."""
    args, keep, result = _partial_args(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table,
                                       sel_block_ids, scale, out_lat, out_lse, ckv_scale,
                                       kpe_scale, n_splits, row_tile, stream, wire)
    lib = load()
    return _Prepared(_partial_fn(lib, tokens, no_alloc), args, keep, result)


def sparse_partial_attn(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids,
                        scale, out_lat=None, out_lse=None, ckv_scale=None, kpe_scale=None,
                        n_splits=0, row_tile=0, stream=None, tokens=False, no_alloc=False,
                        wire=False):
    """Partial attention of each job's Mq x H rows over its selected blocks,
    or with tokens=True over its selected single tokens (sel_block_ids then
    holds logical token ids, block * 64 + t).  no_alloc=True calls the
    allocation-free entry point (split-K partials in the library's static
    scratch array; block selections only).  wire=True asks for the bf16
    wire form of Section 3.2.

    Returns (out_lat fp32 [R, Mq, H, 512], out_lse fp32 [R, Mq, H]), or with
    wire=True (out_lat bf16 [R, Mq, H, 512], (m, l) pairs fp32 [R, Mq, H, 2]).
    """
    lib = load()
    args, _keep, result = _partial_args(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table,
                                        sel_block_ids, scale, out_lat, out_lse, ckv_scale,
                                        kpe_scale, n_splits, row_tile, stream, wire)
    _check(lib, _partial_fn(lib, tokens, no_alloc)(*args))
    return result


def fetch_gather(ckv_pool, kpe_pool, chunk_block_table, sel_token_ids, out_ckv=None,
                 out_kpe=None, stream=None):
    """FETCH's scattered gather: the selected tokens of every layer, in slot
    order, as contiguous bf16 [L, K, 512] / [L, K, 64] (zero rows for empty
    slots).  Pools are [L, P, 64, 512] / [L, P, 64, 64] bf16."""
    L = ckv_pool.shape[0]
    K = sel_token_ids.shape[0]
    if out_ckv is None:
        out_ckv = torch.empty((L, K, DLAT), dtype=torch.bfloat16, device=ckv_pool.device)
    if out_kpe is None:
        out_kpe = torch.empty((L, K, DPE), dtype=torch.bfloat16, device=ckv_pool.device)
    _on_one_gpu(ckv_pool, kpe_pool, chunk_block_table, sel_token_ids, out_ckv, out_kpe)
    lib = load()
    d = [describe(t) for t in (ckv_pool, kpe_pool, chunk_block_table, sel_token_ids, out_ckv,
                               out_kpe)]
    _check(lib, lib.mla_fetch_gather(*[_ref(x) for x in d], _stream(stream)))
    return out_ckv, out_kpe


def fetch_splice(chunk_ckv, chunk_kpe, ckv_pool, kpe_pool, block_table, dst_start, delta,
                 rope_base=10000.0, pairing=0, stream=None):
    """FETCH's splice: write the chunk [L, n, 512] / [L, n, 64] into the
    paged pools at positions dst_start .. dst_start + n - 1 of the sequence
    that block_table maps, its RoPE pairs turned by delta positions
    (pairing 0: dims (2i, 2i+1), 1: dims (i, i+32))."""
    _on_one_gpu(chunk_ckv, chunk_kpe, ckv_pool, kpe_pool, block_table)
    lib = load()
    d = [describe(t) for t in (chunk_ckv, chunk_kpe, ckv_pool, kpe_pool, block_table)]
    _check(lib, lib.mla_fetch_splice(*[_ref(x) for x in d], int(dst_start), int(delta),
                                     float(rope_base), int(pairing), _stream(stream)))


def primitive_costs(mq, chunk_tokens, q_bytes=1152, p_bytes=1032, kv_bytes=1152, **model):
    """ROUTE / FETCH / LOCAL costs of one (chunk, request) case from the
    closed-form model (host arithmetic in the library).  `model` overrides
    fields of PAPER_COST_MODEL.  Returns a dict of the mla_cost_t fields,
    with `choice` as a primitive name."""
    lib = load()
    m = CostModel(**{**PAPER_COST_MODEL, **model})
    c = CostCase(mq, chunk_tokens, q_bytes, p_bytes, kv_bytes)
    out = Cost()
    _check(lib, lib.mla_primitive_costs(ctypes.byref(m), ctypes.byref(c), ctypes.byref(out)))
    res = {f: getattr(out, f) for f, _ in Cost._fields_ if f != "reserved"}
    res["choice"] = PRIMITIVES[res["choice"]]
    return res


def _merge_args(parts_lat, parts_lse, out, out_lse, stream):
    n = len(parts_lat)
    if n != len(parts_lse):
        raise ValueError("parts_lat and parts_lse differ in length")
    want_lse = out_lse is not None
    if out is None:  # fp32 whatever form the parts take
        out = torch.empty(parts_lat[0].shape, dtype=torch.float32, device=parts_lat[0].device)
    if out_lse is True:
        out_lse = torch.empty(parts_lse[0].shape[:3], dtype=torch.float32,
                              device=parts_lse[0].device)
    _on_one_gpu(*parts_lat, *parts_lse, out, out_lse if want_lse else None)
    d_lat = [describe(t) for t in parts_lat]
    d_lse = [describe(t) for t in parts_lse]
    arr_lat = (ctypes.POINTER(Tensor) * max(n, 1))(*[ctypes.pointer(d) for d in d_lat])
    arr_lse = (ctypes.POINTER(Tensor) * max(n, 1))(*[ctypes.pointer(d) for d in d_lse])
    d_out = describe(out)
    d_out_lse = describe(out_lse) if want_lse else None
    args = (arr_lat, arr_lse, n, _ref(d_out), _ref(d_out_lse), _stream(stream))
    keep = (d_lat, d_lse, d_out, d_out_lse, list(parts_lat), list(parts_lse))
    return args, keep, ((out, out_lse) if want_lse else out)


def prepare_merge(parts_lat, parts_lse, out=None, out_lse=None, stream=None):
    """merge_partials with every argument fixed (see prepare_partial)."""
    args, keep, result = _merge_args(parts_lat, parts_lse, out, out_lse, stream)
    return _Prepared(load().mla_merge_partials_ex, args, keep, result)


def merge_partials(parts_lat, parts_lse, out=None, out_lse=None, stream=None):
    """LSE merge of partials (lists of [B, Mq, H, 512] / [B, Mq, H] fp32, or
    of wire-form parts: [B, Mq, H, 512] bf16 / [B, Mq, H, 2] (m, l) fp32).

    Returns out (and the merged lse when out_lse is given or requested by
    passing out_lse=True)."""
    lib = load()
    args, _keep, result = _merge_args(parts_lat, parts_lse, out, out_lse, stream)
    _check(lib, lib.mla_merge_partials_ex(*args))
    return result
