"""Seeded synthetic inputs for sparse absorbed-MLA partial attention.

This module only draws inputs.  It holds none of the attention arithmetic
and is shared by the GPU path's tests and benchmark and by the oracle's
tests, so both sides always consume the same bit patterns.

Shapes follow a DeepSeek-V3-class absorbed MLA layer: per head a 512-wide
latent part and a 64-wide decoupled-RoPE part (d_qk = 576, d_v = 512, the
dimensions of the paper's wire format, Section 3.2), 64-token cache blocks,
and a selection budget of 32 blocks = 2048 tokens, the V3.2 / GLM-5.1
top-2048 budget the paper's Section 5.4 names.

Recipe (all draws are PCG64 streams keyed by (seed, tensor tag, group), so a
tensor is the same whatever the thread count):
  * normals are float32 standard normals times sigma, rounded to bf16 by
    round-to-nearest-even;
  * a job's selection is drawn without replacement and sorted ascending;
  * the pool is scattered: logical block -> pool block goes through a
    seeded permutation of the pool;
  * fp8 caches are the same values quantised per 64-token block to OCP
    E4M3FN with scale absmax / 448 over the block's 576-wide entries (one
    scale for ckv and kpe; separate scales on request), round-to-nearest-even,
    saturating at +-448 (absmax 0 gives scale 1).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

DLAT = 512
DPE = 64
BLOCK = 64
SCALE = 1.0 / math.sqrt(192.0)  # 1/sqrt(128 + 64), the softmax scale of every config

# tensor tags of the PCG64 streams
_T_QLAT, _T_QPE, _T_CKV, _T_KPE, _T_CHUNK, _T_SEL, _T_PERM, _T_TABLE = range(1, 9)
_GROUP = 1 << 22  # elements per independent stream group


def _threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return 4


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32)


def normal_bf16(seed: int, tag: int, shape, sigma: float) -> np.ndarray:
    """bf16 bits of sigma * N(0, 1), drawn in independent stream groups."""
    n = int(np.prod(shape, dtype=np.int64))
    out = np.empty(n, np.uint16)
    groups = (n + _GROUP - 1) // _GROUP

    def work(g):
        lo = g * _GROUP
        hi = min(n, lo + _GROUP)
        rng = np.random.default_rng([seed, tag, g])
        x = rng.standard_normal(hi - lo, dtype=np.float32)
        if sigma != 1.0:
            x *= np.float32(sigma)
        out[lo:hi] = f32_to_bf16_bits(x)

    if groups <= 1:
        for g in range(groups):
            work(g)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(groups)))
    return out.reshape(shape)


# ---------------------------------------------------------------- fp8 E4M3FN
E4M3_MAX = 448.0


def quantize_e4m3fn(y: np.ndarray) -> np.ndarray:
    """float64 values -> OCP E4M3FN codes, round-to-nearest-even, saturating.

    E4M3FN: bias 7, normal exponents -6..8, 3 mantissa bits, subnormals
    m * 2^-9, largest finite 448 (code 0x7E), no infinities.
    """
    y = np.asarray(y, dtype=np.float64)
    sign = np.signbit(y).astype(np.uint8) << np.uint8(7)
    a = np.minimum(np.abs(y), E4M3_MAX)
    # Normal range [2^-6, 448]: round the float64 significand to 3 bits, ties
    # to even, on the bit pattern (a carry moves into the exponent); then
    # rebias the exponent from 1023 to 7.
    b = a.view(np.uint64)
    lsb = (b >> np.uint64(49)) & np.uint64(1)
    r = (b + np.uint64((1 << 48) - 1) + lsb) >> np.uint64(49)
    code_n = r.astype(np.int64) - ((1023 - 7) << 3)
    # Subnormal range: multiples of 2^-9 (rint ties to even; 8 * 2^-9 is the
    # smallest normal, code 8).
    code_s = np.rint(a * 512.0).astype(np.int64)
    code = np.where(a < 2.0 ** -6, code_s, code_n)
    return code.astype(np.uint8) | sign


def quantize_blocks_e4m3fn(*pools: np.ndarray):
    """Per-block fp8 quantisation of bf16 pools [P, 64, D_i] that share one
    scale per block: scale = float32(absmax / 448) over the block's values in
    all the given pools (1 when that absmax is 0), code = E4M3FN(value / scale).

    Returns (codes uint8 per pool..., scales float32 [P]).
    """
    P = pools[0].shape[0]
    codes = [np.empty(b.shape, np.uint8) for b in pools]
    scales = np.empty(P, np.float32)
    step = 16  # small chunks: temporaries of a few MB are reused from the heap

    def work(lo):
        hi = min(P, lo + step)
        xs = [bf16_bits_to_f32(b[lo:hi]) for b in pools]
        amax = np.max([np.abs(x).reshape(hi - lo, -1).max(axis=1) for x in xs], axis=0)
        s = (amax / np.float32(E4M3_MAX)).astype(np.float32)
        s[amax == 0] = np.float32(1.0)
        scales[lo:hi] = s
        for c, x in zip(codes, xs):
            c[lo:hi] = quantize_e4m3fn(x.astype(np.float64) / s.astype(np.float64)[:, None, None])

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(0, P, step)))
    return (*codes, scales)


# ------------------------------------------------------------------ workloads
@dataclass
class Workload:
    """One call's inputs as host arrays (bf16 as uint16 bits)."""
    name: str
    q_lat: np.ndarray            # uint16 [R, Mq, H, 512]
    q_pe: np.ndarray             # uint16 [R, Mq, H, 64]
    ckv: np.ndarray              # uint16 [P, 64, 512] (or uint8 codes)
    kpe: np.ndarray              # uint16 [P, 64, 64]  (or uint8 codes)
    table: np.ndarray            # int32  [R, NB]
    sel: np.ndarray              # int32  [R, K] (or [R, Mq, K])
    scale: float = SCALE
    ckv_scale: np.ndarray | None = None  # float32 [P] for fp8 pools
    kpe_scale: np.ndarray | None = None
    n_requests: int = 0          # routed requests the call serves
    merge_parts: int = 1         # partials merged per request (slot-major jobs)
    meta: dict = field(default_factory=dict)
    tokens: bool = False         # sel holds logical token ids (block * 64 + t)

    @property
    def shape(self):
        R, Mq, H, _ = self.q_lat.shape
        return dict(R=R, Mq=Mq, H=H, P=self.ckv.shape[0], NB=self.table.shape[1],
                    K=self.sel.shape[1])

    @property
    def fp8(self):
        return self.ckv.dtype == np.uint8

    def n_selected_blocks(self):
        """Blocks a job must read: its valid slots (one selection per job), or
        the distinct blocks its query rows select (a selection per row).  For
        token selections: the valid slots / 64 (a token is 1/64 of a block)."""
        if self.tokens:
            return (self.sel >= 0).sum() / BLOCK
        if self.sel.ndim == 3:
            return int(sum(np.unique(s[s >= 0]).size for s in self.sel))
        return int((self.sel >= 0).sum())

    def algorithmic_flops(self):
        R, Mq, H, _ = self.q_lat.shape
        per_slot = 1 if self.tokens else BLOCK
        if self.sel.ndim == 3:  # each query row attends its own slots
            return int((self.sel >= 0).sum()) * per_slot * H * 2 * (DLAT + DPE + DLAT)
        per_job = (self.sel >= 0).sum(axis=1).astype(np.int64) * per_slot
        return int((per_job * Mq * H).sum()) * 2 * (DLAT + DPE + DLAT)

    def kv_bytes(self):
        per_tok = (DLAT + DPE) * (1 if self.fp8 else 2)
        b = int(round(self.n_selected_blocks() * BLOCK * per_tok))
        if self.fp8:
            b += self.n_selected_blocks() * 8  # two fp32 scales per block
        return b

    def to_fp8(self, shared_scale=True):
        """The same values with E4M3FN caches and per-block absmax/448 scales:
        one scale per block for the whole 576-wide entries (the same array for
        ckv_scale and kpe_scale), or with shared_scale=False separate latent
        and RoPE scales."""
        if shared_scale:
            ckv, kpe, cs = quantize_blocks_e4m3fn(self.ckv, self.kpe)
            ks = cs
        else:
            ckv, cs = quantize_blocks_e4m3fn(self.ckv)
            kpe, ks = quantize_blocks_e4m3fn(self.kpe)
        return Workload(self.name + "-fp8", self.q_lat, self.q_pe, ckv, kpe, self.table,
                        self.sel, self.scale, cs, ks, self.n_requests, self.merge_parts,
                        dict(self.meta), self.tokens)


def _perm(seed, n):
    return np.random.default_rng([seed, _T_PERM]).permutation(n).astype(np.int32)


def _queries(seed, R, Mq, H, sigma=1.0):
    return (normal_bf16(seed, _T_QLAT, (R, Mq, H, DLAT), sigma),
            normal_bf16(seed, _T_QPE, (R, Mq, H, DPE), sigma))


def _pool(seed, P, sigma):
    return (normal_bf16(seed, _T_CKV, (P, BLOCK, DLAT), sigma),
            normal_bf16(seed, _T_KPE, (P, BLOCK, DPE), sigma))


def tiny(seed=1):
    """1 request, Mq=1, 16 heads, one 256-token chunk (4 blocks), all N(0,1);
    2 of the 4 blocks selected by seed, 2 empty slots."""
    q_lat, q_pe = _queries(seed, 1, 1, 16)
    ckv, kpe = _pool(seed, 4, 1.0)
    table = _perm(seed, 4)[None, :]
    ids = np.sort(np.random.default_rng([seed, _T_SEL]).choice(4, 2, replace=False))
    sel = np.array([[ids[0], ids[1], -1, -1]], np.int32)
    return Workload("tiny", q_lat, q_pe, ckv, kpe, table.astype(np.int32), sel,
                    n_requests=1, merge_parts=1)


def dsv3_one_request(seed=2):
    """Mq=1, 128 heads, q ~ N(0,1); one 4096-token chunk (64 blocks) ~ N(0,0.5);
    top-32 blocks uniform without replacement."""
    q_lat, q_pe = _queries(seed, 1, 1, 128)
    ckv, kpe = _pool(seed, 64, 0.5)
    table = _perm(seed, 64)[None, :]
    sel = np.sort(np.random.default_rng([seed, _T_SEL]).choice(64, 32, replace=False))
    return Workload("dsv3-one-request", q_lat, q_pe, ckv, kpe, table.astype(np.int32),
                    sel[None, :].astype(np.int32), n_requests=1, merge_parts=1)


def batched_merge(seed=3, n_requests=64, n_chunks=256, chunk_blocks=128, hits=4, topk=32):
    """64 requests, Mq=1, 128 heads, q ~ N(0,1); a pool of 256 chunks x 8192
    tokens ~ N(0,0.5); each request hits 4 distinct chunks and selects 32
    blocks per chunk.  Jobs are slot-major (job = hit * n_requests + request),
    so the partials of hit j of every request form one contiguous range for
    the merge."""
    q_req_lat, q_req_pe = _queries(seed, n_requests, 1, 128)
    P = n_chunks * chunk_blocks
    ckv, kpe = _pool(seed, P, 0.5)
    perm = _perm(seed, P).reshape(n_chunks, chunk_blocks)
    rng_c = np.random.default_rng([seed, _T_CHUNK])
    chunks = np.stack([rng_c.choice(n_chunks, hits, replace=False) for _ in range(n_requests)])
    rng_s = np.random.default_rng([seed, _T_SEL])
    R = hits * n_requests
    table = np.empty((R, chunk_blocks), np.int32)
    sel = np.empty((R, topk), np.int32)
    for j in range(hits):
        for b in range(n_requests):
            r = j * n_requests + b
            table[r] = perm[chunks[b, j]]
            sel[r] = np.sort(rng_s.choice(chunk_blocks, topk, replace=False))
    q_lat = np.ascontiguousarray(np.broadcast_to(q_req_lat[None], (hits,) + q_req_lat.shape)
                                 .reshape(R, 1, 128, DLAT))
    q_pe = np.ascontiguousarray(np.broadcast_to(q_req_pe[None], (hits,) + q_req_pe.shape)
                                .reshape(R, 1, 128, DPE))
    # (the q of job j * n_requests + b is request b's: the first n_requests
    # rows hold every distinct q, which a holder needs only once)
    return Workload("batched-merge", q_lat, q_pe, ckv, kpe, table, sel,
                    n_requests=n_requests, merge_parts=hits,
                    meta=dict(chunks=chunks, q_rows=n_requests))


def zipf_ids(rng, n, k, a=1.1):
    """k distinct positions in [0, n) by successive Zipf(a)-weighted draws
    without replacement, sorted."""
    w = (np.arange(1, n + 1, dtype=np.float64)) ** (-a)
    return np.sort(rng.choice(n, k, replace=False, p=w / w.sum()))


def few_head(seed=4, n_requests=16, mq=4, heads=16, chunk_blocks=512, topk=32):
    """16 requests, Mq=4, 16 heads (one TP share of 128), q ~ N(0,1); each
    request owns one 32768-token chunk (512 blocks) ~ N(0,1) and selects 32
    blocks drawn Zipf(1.1) over block position; the 4 rows share it."""
    q_lat, q_pe = _queries(seed, n_requests, mq, heads)
    P = n_requests * chunk_blocks
    ckv, kpe = _pool(seed, P, 1.0)
    table = _perm(seed, P).reshape(n_requests, chunk_blocks)
    rng_s = np.random.default_rng([seed, _T_SEL])
    sel = np.stack([zipf_ids(rng_s, chunk_blocks, topk) for _ in range(n_requests)])
    return Workload("few-head", q_lat, q_pe, ckv, kpe, table.astype(np.int32),
                    sel.astype(np.int32), n_requests=n_requests, merge_parts=1)


def dense_local(seed=5, n_requests=32, chunk_blocks=1024, fp8=False):
    """32 requests, Mq=1, 128 heads, q ~ N(0,1); each attends all 1024 blocks
    (65536 tokens) of its own chunk ~ N(0,0.5); optionally as an fp8 cache."""
    q_lat, q_pe = _queries(seed, n_requests, 1, 128)
    P = n_requests * chunk_blocks
    ckv, kpe = _pool(seed, P, 0.5)
    table = _perm(seed, P).reshape(n_requests, chunk_blocks)
    sel = np.broadcast_to(np.arange(chunk_blocks, dtype=np.int32), (n_requests, chunk_blocks))
    w = Workload("dense-local", q_lat, q_pe, ckv, kpe, table.astype(np.int32),
                 np.ascontiguousarray(sel), n_requests=n_requests, merge_parts=1)
    return w.to_fp8() if fp8 else w


def holder(n_req, heads, sparse=False, as_jobs=False, seed=7):
    """One holder chunk serving n_req routed requesters (Mq = 1, `heads`
    heads each; q ~ N(0,1), cache ~ N(0,0.5)): the holder-compute experiment
    of Section 6.3, on one GPU.
      dense:  a 2048-token chunk (32 blocks), every requester attends all of
              it (the paper's c_t = 2048 resident tokens);
      sparse: an 8192-token chunk (128 blocks), each requester selects 32
              blocks drawn Zipf(1.1) over positions, so hot blocks are shared.
    By default the requesters are the query rows of one job (a shared
    selection when dense, one selection per row when sparse) and the library
    reads each block once for all of them; as_jobs routes every requester as
    a job of its own on the same chunk (each reads its blocks itself)."""
    nb = 128 if sparse else 32
    q_lat, q_pe = _queries(seed, n_req, 1, heads)  # [n_req, 1, H, .]
    ckv, kpe = _pool(seed, 2 * nb, 0.5)
    perm = _perm(seed, 2 * nb)[:nb].astype(np.int32)  # the chunk's blocks, scattered in the pool
    if sparse:
        rs = np.random.default_rng([seed, _T_SEL])
        rows = np.stack([zipf_ids(rs, nb, 32) for _ in range(n_req)]).astype(np.int32)
    else:
        rows = np.tile(np.arange(nb, dtype=np.int32), (n_req, 1))
    name = f"holder-{'sparse' if sparse else 'dense'}-n{n_req}-h{heads}" + ("-jobs" if as_jobs else "")
    if as_jobs:
        return Workload(name, q_lat, q_pe, ckv, kpe, np.tile(perm, (n_req, 1)), rows,
                        n_requests=n_req, merge_parts=1)
    q_lat = np.ascontiguousarray(q_lat.reshape(1, n_req, heads, DLAT))
    q_pe = np.ascontiguousarray(q_pe.reshape(1, n_req, heads, DPE))
    sel = rows[:1] if not sparse else rows[None]
    return Workload(name, q_lat, q_pe, ckv, kpe, perm[None], np.ascontiguousarray(sel),
                    n_requests=n_req, merge_parts=1)


def selection(kind, n_req, k, corpus, heads=128, seed=8):
    """The selection-regime holder of Section 6.3 at a selection budget of k
    tokens: n_req requests (Mq = 1, `heads` heads, q ~ N(0,1)), each over a
    chunk of its own of `corpus` tokens (corpus / 64 blocks ~ N(0,0.5),
    scattered in the pool).
      tok:   the top-k as k single tokens drawn uniformly without replacement
             over the chunk, sorted (a token-level indexer, block = 1);
      blk:   k / 64 whole blocks drawn uniformly without replacement, sorted;
      dense: the first k / 64 blocks of the chunk, laid out contiguously in
             the pool (dense decode over k resident tokens, the matched-k
             reference of the sparse premium)."""
    assert k % BLOCK == 0 and corpus % BLOCK == 0 and k <= corpus
    nb = corpus // BLOCK
    q_lat, q_pe = _queries(seed, n_req, 1, heads)
    P = n_req * nb
    ckv, kpe = _pool(seed, P, 0.5)
    rs = np.random.default_rng([seed, _T_SEL])
    if kind == "dense":
        table = np.arange(P, dtype=np.int32).reshape(n_req, nb)
        sel = np.tile(np.arange(k // BLOCK, dtype=np.int32), (n_req, 1))
    else:
        table = _perm(seed, P).reshape(n_req, nb)
        n_ids = nb * BLOCK if kind == "tok" else nb
        m = k if kind == "tok" else k // BLOCK
        sel = np.stack([np.sort(rs.choice(n_ids, m, replace=False)) for _ in range(n_req)])
    name = f"select-{kind}-b{n_req}-k{k}-c{corpus}" + ("" if heads == 128 else f"-h{heads}")
    return Workload(name, q_lat, q_pe, ckv, kpe, table.astype(np.int32), sel.astype(np.int32),
                    n_requests=n_req, merge_parts=1, tokens=kind == "tok")


def fetch_inputs(name, seed=9):
    """FETCH-side workloads (Section 2.2), as a dict of host arrays:
      fetch-splice-c<n>-l<L>: a pulled chunk of n tokens x L layers (~ N(0,
        0.5), bf16) to splice into a requester's paged pools of 2n + 128
        tokens per layer, re-homed at position 37 (not block aligned) with
        the chunk moving by delta = 4096 positions;
      fetch-gather-k<k>-c<c>-l<L>: k tokens drawn uniformly without
        replacement over a c-token chunk of L layers, gathered into a
        contiguous payload.
    The paper's case is c = 2048 tokens of a 27-layer model."""
    parts = name.split("-")
    kind = parts[1]
    rng = np.random.default_rng([seed, _T_SEL])
    if kind == "splice":
        n, L = int(parts[2][1:]), int(parts[3][1:])
        nb = (2 * n + 127) // BLOCK + 2
        P = nb + 3
        chunk_ckv = normal_bf16(seed, _T_CKV, (L, n, DLAT), 0.5)
        chunk_kpe = normal_bf16(seed, _T_KPE, (L, n, DPE), 0.5)
        ckv = normal_bf16(seed + 1, _T_CKV, (L, P, BLOCK, DLAT), 0.5)
        kpe = normal_bf16(seed + 1, _T_KPE, (L, P, BLOCK, DPE), 0.5)
        table = _perm(seed, P)[:nb].astype(np.int32)
        return dict(kind=kind, name=name, chunk_ckv=chunk_ckv, chunk_kpe=chunk_kpe, ckv=ckv,
                    kpe=kpe, table=table, dst_start=37, delta=4096, n=n, L=L)
    k, c, L = int(parts[2][1:]), int(parts[3][1:]), int(parts[4][1:])
    nb = c // BLOCK
    ckv = normal_bf16(seed, _T_CKV, (L, nb, BLOCK, DLAT), 0.5)
    kpe = normal_bf16(seed, _T_KPE, (L, nb, BLOCK, DPE), 0.5)
    table = _perm(seed, nb).astype(np.int32)
    sel = np.sort(rng.choice(c, k, replace=False)).astype(np.int32)
    return dict(kind=kind, name=name, ckv=ckv, kpe=kpe, table=table, sel=sel, n=k, L=L)


CONFIGS = {
    "tiny": tiny,
    "dsv3-one-request": dsv3_one_request,
    "batched-merge": batched_merge,
    "few-head": few_head,
    "dense-local": dense_local,
    "dense-local-fp8": lambda seed=5: dense_local(seed, fp8=True),
}


def make(name, seed=None, **kw):
    """A named workload; `holder-{dense|sparse}-n{N}-h{H}[-jobs]` builds the
    holder experiment (see holder), `select-{tok|blk|dense}-b{B}-k{k}-c{c}[-h{H}]`
    the selection-budget experiment (see selection); a `-fp8` suffix on any of
    these gives the same values as an e4m3 cache (one scale per block)."""
    if name.endswith("-fp8") and name not in CONFIGS:
        w = make(name[:-4], seed, **kw).to_fp8()
        w.name = name
        return w
    if name.startswith("select-"):
        parts = name.split("-")
        kw.update(kind=parts[1], n_req=int(parts[2][1:]), k=int(parts[3][1:]),
                  corpus=int(parts[4][1:]))
        if len(parts) > 5:
            kw.update(heads=int(parts[5][1:]))
        return selection(**kw) if seed is None else selection(seed=seed, **kw)
    if name.startswith("holder-"):
        parts = name.split("-")
        kw.update(n_req=int(parts[2][1:]), heads=int(parts[3][1:]),
                  sparse=parts[1] == "sparse", as_jobs=parts[-1] == "jobs")
        return holder(**kw) if seed is None else holder(seed=seed, **kw)
    fn = CONFIGS[name]
    return fn(**kw) if seed is None else fn(seed=seed, **kw)


def _slot_ids(rs, NB, K, nv, allow_dup, pad_pattern, common=None, shared_frac=0.0):
    """K slots holding nv sorted ids (the rest -1).  With a common set, each
    id is taken from it with probability shared_frac (rows that overlap)."""
    if allow_dup:
        ids = rs.integers(0, NB, nv)
    else:
        ids = rs.choice(NB, nv, replace=False)
    if common is not None and nv:
        take = rs.random(nv) < shared_frac
        pick = rs.choice(common, nv, replace=True)
        ids = np.where(take, pick, ids)
        if not allow_dup:
            ids = np.unique(ids)
            extra = np.setdiff1d(np.arange(NB), ids)
            if ids.size < nv:
                ids = np.concatenate([ids, rs.choice(extra, nv - ids.size, replace=False)])
    ids = np.sort(ids)
    row = np.full(K, -1, np.int32)
    if pad_pattern == "interleaved" and nv < K:
        row[np.sort(rs.choice(K, nv, replace=False))] = ids
    else:
        row[:nv] = ids
    return row


def random_case(seed, R, Mq, H, P, NB, K, n_valid=None, sigma=1.0, allow_dup=False,
                pad_pattern="tail", per_row=False, shared_frac=0.5, tokens=False):
    """Small random case for tests: R jobs over a P-block pool, NB logical
    blocks per job, K slots of which n_valid[r] hold ids.  pad_pattern is
    'tail' (ids first), 'interleaved' (empty slots spread) or 'none'.
    per_row gives every query row its own selection, sel [R, Mq, K], drawing
    each id from a per-job common set with probability shared_frac so that
    rows overlap; n_valid may then be [R][Mq].  tokens draws logical token
    ids in [0, 64 NB) instead of block ids."""
    q_lat, q_pe = _queries(seed, R, Mq, H, sigma)
    ckv, kpe = _pool(seed, P, sigma)
    rng = np.random.default_rng([seed, _T_TABLE])
    table = np.stack([rng.choice(P, NB, replace=NB > P) for _ in range(R)]).astype(np.int32)
    rs = np.random.default_rng([seed, _T_SEL])
    n_ids = NB * BLOCK if tokens else NB

    def nvalid(r, i=None):
        if n_valid is None:
            return K
        v = n_valid[r] if np.ndim(n_valid) else n_valid
        return v[i] if (i is not None and np.ndim(v)) else v

    if per_row:
        sel = np.full((R, Mq, K), -1, np.int32)
        for r in range(R):
            common = rs.choice(n_ids, min(n_ids, K), replace=False)
            for i in range(Mq):
                sel[r, i] = _slot_ids(rs, n_ids, K, nvalid(r, i), allow_dup, pad_pattern,
                                      common, shared_frac)
    else:
        sel = np.full((R, K), -1, np.int32)
        for r in range(R):
            sel[r] = _slot_ids(rs, n_ids, K, nvalid(r), allow_dup, pad_pattern)
    return Workload(f"random-{seed}", q_lat, q_pe, ckv, kpe, table, sel,
                    n_requests=R, merge_parts=1, tokens=tokens)
