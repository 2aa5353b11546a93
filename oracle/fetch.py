"""FETCH-side operations, written out plainly (numpy, float64 where values
are computed).  TEST INFRASTRUCTURE ONLY: tests compare the library's
gather and splice kernels against these; the product path never imports
this module.

Section 2.2: FETCH pulls a chunk's latent cache, re-rotates its positional
part to the requester's offset when the chunk is re-homed at a new
contiguous position, and scatters it into the requester's paged pool;
under sparse selection the entries keep their canonical positions and the
only work left is the scattered gather of the selected set.

Readings (the paper gives no RoPE convention): the 64-wide RoPE part holds
32 rotation pairs; pair i turns at frequency theta_i = base^(-2i/64), and
its two elements are either dims (2i, 2i+1) ("interleaved") or dims
(i, i+32) ("half").  Moving a token from position p to p + delta multiplies
every pair (x, y) by the rotation through angle delta * theta_i:
(x, y) -> (x cos - y sin, x sin + y cos).  The latent part is not
positional and is copied unchanged.  Results are rounded to bf16 once, to
nearest even.
"""
import numpy as np

DLAT, DPE, BLOCK = 512, 64, 64
INTERLEAVED, HALF = 0, 1


def bf16_to_f64(bits):
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16(x):
    """float64 -> bf16 bits, round to nearest even, in one step: a bf16 has
    8 significant bits, so for 2^(e-1) <= |x| < 2^e its spacing is 2^(e-8);
    x / spacing is rounded to the nearest integer (ties to even) and scaled
    back, which float32 then holds exactly."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    ulp_exp = np.maximum(e - 8, -133)
    q = np.rint(np.ldexp(x, -ulp_exp))
    y = np.ldexp(q, ulp_exp).astype(np.float32)
    return (y.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def pair_index(pairing):
    """(first, second) element dims of the 32 rotation pairs."""
    i = np.arange(DPE // 2)
    if pairing == INTERLEAVED:
        return 2 * i, 2 * i + 1
    return i, i + DPE // 2


def frequencies(base):
    return base ** (-2.0 * np.arange(DPE // 2) / DPE)


def rotate(kpe_f64, delta, base, pairing):
    """Rotate RoPE rows [..., 64] (float64) by delta positions."""
    a, b = pair_index(pairing)
    ang = float(delta) * frequencies(base)
    c, s = np.cos(ang), np.sin(ang)
    x, y = kpe_f64[..., a], kpe_f64[..., b]
    out = np.empty_like(kpe_f64)
    out[..., a] = x * c - y * s
    out[..., b] = x * s + y * c
    return out


def gather(ckv_pool, kpe_pool, table, sel):
    """Copy of the selected tokens in slot order: for every slot j with
    s = sel[j], entry j holds token s % 64 of pool block table[s // 64],
    for each layer; an empty slot (-1), an id outside [0, 64 NB) or a table
    entry outside [0, P) gives a zero row.  Pools [L, P, 64, D], table
    [NB], sel [K]; returns (ckv [L, K, 512], kpe [L, K, 64])."""
    L, P = ckv_pool.shape[:2]
    K = len(sel)
    out_c = np.zeros((L, K, DLAT), ckv_pool.dtype)
    out_k = np.zeros((L, K, DPE), kpe_pool.dtype)
    for j, s in enumerate(int(v) for v in sel):
        if s < 0 or s >= len(table) * BLOCK:
            continue
        b, t = int(table[s // BLOCK]), s % BLOCK
        if not 0 <= b < P:
            continue
        for layer in range(L):
            out_c[layer, j] = ckv_pool[layer, b, t]
            out_k[layer, j] = kpe_pool[layer, b, t]
    return out_c, out_k


def splice(chunk_ckv, chunk_kpe, dst_ckv, dst_kpe, dst_table, dst_start, delta, base, pairing):
    """Scatter a pulled chunk (chunk_* [L, n, D], token t at the holder's
    position p_t) into copies of the paged pools dst_* [L, P, 64, D]:
    token t lands in slot dst_start + t of the requester's sequence, i.e.
    block dst_table[(dst_start + t) // 64], row (dst_start + t) % 64, with
    its RoPE part rotated by delta positions.  Returns the new pools."""
    ckv, kpe = dst_ckv.copy(), dst_kpe.copy()
    L, n = chunk_ckv.shape[:2]
    for layer in range(L):
        rot = f64_to_bf16(rotate(bf16_to_f64(chunk_kpe[layer]), delta, base, pairing))
        for t in range(n):
            slot = dst_start + t
            b, r = int(dst_table[slot // BLOCK]), slot % BLOCK
            ckv[layer, b, r] = chunk_ckv[layer, t]
            kpe[layer, b, r] = rot[t]
    return ckv, kpe
