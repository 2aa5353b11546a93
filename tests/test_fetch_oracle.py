"""The FETCH-side oracle (oracle/fetch.py) against facts outside itself:
the bf16 rounding against the workload generator's float32 rounding and
hand-made ties, the gather against a reshaped view of the chunk, the
splice's placement against the requester's logical sequence, and the
rotation against rotary position embedding applied from its definition
(complex rotation) at two positions.  CPU only."""
import numpy as np

from oracle import fetch as F
from paper_2606_01502_amd import workloads as W


def test_bf16_rounding():
    x = np.random.default_rng(0).standard_normal(50000).astype(np.float32) * np.float32(7)
    assert np.array_equal(F.f64_to_bf16(x.astype(np.float64)), W.f32_to_bf16_bits(x))
    # exact ties round to the even neighbour; just above a tie rounds up
    one = 1.0
    assert F.f64_to_bf16(np.array([one + 2.0 ** -8]))[0] == 0x3F80          # tie -> 1.0
    assert F.f64_to_bf16(np.array([one + 3 * 2.0 ** -8]))[0] == 0x3F82      # tie -> even
    assert F.f64_to_bf16(np.array([one + 2.0 ** -8 + 2.0 ** -40]))[0] == 0x3F81
    assert F.f64_to_bf16(np.array([-0.0]))[0] == 0x8000


def _pools(seed, L, P):
    rng = np.random.default_rng(seed)
    ckv = W.f32_to_bf16_bits(rng.standard_normal((L, P, 64, 512)).astype(np.float32))
    kpe = W.f32_to_bf16_bits(rng.standard_normal((L, P, 64, 64)).astype(np.float32))
    return ckv, kpe


def test_gather_whole_chunk_is_its_blocks():
    ckv, kpe = _pools(1, 2, 9)
    table = np.array([4, 0, 7], np.int32)
    sel = np.arange(3 * 64, dtype=np.int32)
    gc, gk = F.gather(ckv, kpe, table, sel)
    assert np.array_equal(gc, ckv[:, table].reshape(2, -1, 512))
    assert np.array_equal(gk, kpe[:, table].reshape(2, -1, 64))
    # slot order, duplicates repeat, empty and out-of-range slots are zero rows
    sel2 = np.array([130, -1, 5, 130, 3 * 64], np.int32)
    gc2, _ = F.gather(ckv, kpe, table, sel2)
    seq = ckv[:, table].reshape(2, -1, 512)
    assert np.array_equal(gc2[:, [0, 2, 3]], seq[:, [130, 5, 130]])
    assert not gc2[:, [1, 4]].any()


def test_splice_placement_and_identity():
    """delta = 0 copies bit for bit; token t lands at position dst_start + t
    of the requester's sequence (table order), across block boundaries;
    everything else in the pools is untouched."""
    ckv, kpe = _pools(2, 2, 6)
    chunk_c, chunk_k = _pools(3, 2, 2)
    chunk_c, chunk_k = chunk_c.reshape(2, 128, 512)[:, :100], chunk_k.reshape(2, 128, 64)[:, :100]
    table = np.array([5, 2, 0, 3], np.int32)
    nc, nk = F.splice(chunk_c, chunk_k, ckv, kpe, table, 37, 0, 10000.0, F.INTERLEAVED)
    seq_c = nc[:, table].reshape(2, -1, 512)
    seq_k = nk[:, table].reshape(2, -1, 64)
    assert np.array_equal(seq_c[:, 37:137], chunk_c)
    assert np.array_equal(seq_k[:, 37:137], chunk_k)
    old_c = ckv[:, table].reshape(2, -1, 512)
    assert np.array_equal(seq_c[:, :37], old_c[:, :37])
    assert np.array_equal(seq_c[:, 137:], old_c[:, 137:])
    untouched = [b for b in range(6) if b not in table]
    assert np.array_equal(nc[:, untouched], ckv[:, untouched])


def _rope_from_definition(x, pos, base, pairing):
    """Rotary embedding by its definition: pair i as the complex number
    x_a + i x_b, multiplied by exp(i * pos * base^(-i/32))."""
    a, b = F.pair_index(pairing)
    z = x[..., a] + 1j * x[..., b]
    theta = np.power(float(base), -np.arange(32) / 32.0)
    z = z * np.exp(1j * pos * theta)
    out = np.empty_like(x)
    out[..., a], out[..., b] = z.real, z.imag
    return out


def test_rotation_moves_rope_to_the_new_position():
    """A key embedded at position p and rotated by delta equals the key
    embedded at p + delta (within two bf16 roundings), for both pairings,
    forward and backward moves and a large offset."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((300, 64))
    for pairing in (F.INTERLEAVED, F.HALF):
        for p, delta, base in ((0, 5, 10000.0), (4096, -1000, 10000.0), (17, 131072, 50000.0)):
            at_p = F.f64_to_bf16(_rope_from_definition(x, p, base, pairing))
            moved = F.f64_to_bf16(F.rotate(F.bf16_to_f64(at_p), delta, base, pairing))
            want = _rope_from_definition(x, p + delta, base, pairing)
            # an input rounding error of a pair rotates into both of its
            # elements: bound each element by the pair's magnitude (two
            # roundings of relative size 2^-9 each, plus the rotation's own)
            a, b = F.pair_index(pairing)
            r = np.hypot(want[..., a], want[..., b])
            err = np.abs(F.bf16_to_f64(moved) - want)
            rel = np.maximum(err[..., a], err[..., b]) / r
            assert rel.max() < 2.0 ** -7, (pairing, p, delta, float(rel.max()))
    # the pairings differ: the same rotation on the other pairing moves other dims
    y = rng.standard_normal((4, 64))
    assert not np.allclose(F.rotate(y, 3, 10000.0, F.INTERLEAVED), F.rotate(y, 3, 10000.0, F.HALF))
