"""FETCH-side kernels against the oracle (oracle/fetch.py): the gather is
bit-exact, the splice copies latent rows bit for bit, leaves every other
pool row untouched, and turns RoPE pairs to within one bf16 unit at the
pair's magnitude (the kernel multiplies in fp32 with float cos/sin of a
double angle; the oracle rotates in double; both round once)."""
import numpy as np
import pytest
import torch

from oracle import fetch as F
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(
        G.device())


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(G.device())


def _pools(seed, L, P, sigma=1.0):
    return (W.normal_bf16(seed, 3, (L, P, 64, 512), sigma),
            W.normal_bf16(seed, 4, (L, P, 64, 64), sigma))


@pytest.mark.parametrize("k", [1, 63, 64, 65, 200])
def test_gather_matches_oracle_bit_for_bit(k):
    print(f"case: gather k={k}", flush=True)
    ckv, kpe = _pools(800 + k, 3, 20)
    table = np.random.default_rng(k).permutation(20)[:8].astype(np.int32)
    rng = np.random.default_rng(900 + k)
    sel = rng.integers(0, 8 * 64, k).astype(np.int32)
    sel[rng.random(k) < 0.2] = -1
    if k > 2:
        sel[1] = 8 * 64          # past the chunk
        sel[2] = -5              # negative, not -1
    tbl = table.copy()
    tbl[3] = 25                  # a table entry past the pool
    oc, ok = mla.fetch_gather(_bf16(ckv), _bf16(kpe), _i32(tbl), _i32(sel))
    torch.cuda.synchronize()
    rc, rk = F.gather(ckv, kpe, tbl, sel)
    assert np.array_equal(_bits(oc), rc) and np.array_equal(_bits(ok), rk)


def _check_splice(n, L, dst_start, delta, pairing, base, seed, bad_entry=False):
    P, nb = 24, 12
    ckv, kpe = _pools(seed, L, P)
    chunk_c = W.normal_bf16(seed, 5, (L, n, 512), 1.0)
    chunk_k = W.normal_bf16(seed, 6, (L, n, 64), 1.0)
    table = np.random.default_rng(seed).permutation(P)[:nb].astype(np.int32)
    if bad_entry:
        table[(dst_start + n // 2) // 64] = P + 7   # that block's tokens are skipped
    d_ckv, d_kpe = _bf16(ckv), _bf16(kpe)
    mla.fetch_splice(_bf16(chunk_c), _bf16(chunk_k), d_ckv, d_kpe, _i32(table), dst_start,
                     delta, base, pairing)
    torch.cuda.synchronize()
    got_c, got_k = _bits(d_ckv), _bits(d_kpe)
    ok_tbl = np.where((table >= 0) & (table < P), table, -1)
    safe = np.where(ok_tbl >= 0, ok_tbl, P)  # the oracle writes skipped tokens to a spare block
    ref_c, ref_k = F.splice(chunk_c, chunk_k, np.concatenate([ckv, ckv[:, :1]], 1),
                            np.concatenate([kpe, kpe[:, :1]], 1), safe, dst_start, delta, base,
                            pairing)
    ref_c, ref_k = ref_c[:, :P], ref_k[:, :P]
    assert np.array_equal(got_c, ref_c), "latent rows or placement differ"
    if delta == 0:
        assert np.array_equal(got_k, ref_k)
        return
    a, b = F.pair_index(pairing)
    g, r = F.bf16_to_f64(got_k), F.bf16_to_f64(ref_k)
    mag = np.maximum(np.abs(r[..., a]), np.abs(r[..., b]))
    unit = np.ldexp(1.0, np.frexp(mag)[1] - 8)  # a bf16 unit at the pair's magnitude
    err = np.maximum(np.abs(g - r)[..., a], np.abs(g - r)[..., b])
    assert np.all(err <= unit), float((err / unit).max())
    # rows the chunk does not cover are untouched, bit for bit
    changed = np.any(got_k != kpe, axis=-1) | np.any(got_c != ckv, axis=-1)
    assert changed.sum() <= L * n


@pytest.mark.parametrize("pairing", [0, 1])
@pytest.mark.parametrize("n,dst_start,delta", [(1, 0, 5), (63, 37, -1000), (64, 64, 0),
                                               (100, 37, 4096), (300, 5, 131072)])
def test_splice_matches_oracle(n, dst_start, delta, pairing):
    print(f"case: splice n={n} start={dst_start} delta={delta} pairing={pairing}", flush=True)
    _check_splice(n, 2, dst_start, delta, pairing, 10000.0, 810 + n)


def test_splice_other_base_and_skipped_block():
    print("case: splice base 50000, skipped block", flush=True)
    _check_splice(200, 3, 20, 777, 0, 50000.0, 830, bad_entry=True)


def test_splice_paper_chunk_27_layers():
    """A 2048-token chunk of a 27-layer model (the paper's splice case)."""
    print("case: splice 2048 x 27", flush=True)
    w = W.fetch_inputs("fetch-splice-c2048-l27")
    d_ckv, d_kpe = _bf16(w["ckv"]), _bf16(w["kpe"])
    mla.fetch_splice(_bf16(w["chunk_ckv"]), _bf16(w["chunk_kpe"]), d_ckv, d_kpe, _i32(w["table"]),
                     w["dst_start"], w["delta"])
    torch.cuda.synchronize()
    layers = [0, 13, 26]
    ref_c, ref_k = F.splice(w["chunk_ckv"][layers], w["chunk_kpe"][layers], w["ckv"][layers],
                            w["kpe"][layers], w["table"], w["dst_start"], w["delta"], 10000.0, 0)
    got_c, got_k = _bits(d_ckv)[layers], _bits(d_kpe)[layers]
    assert np.array_equal(got_c, ref_c)
    g, r = F.bf16_to_f64(got_k), F.bf16_to_f64(ref_k)
    a, b = F.pair_index(0)
    mag = np.maximum(np.abs(r[..., a]), np.abs(r[..., b]))
    unit = np.ldexp(1.0, np.frexp(mag)[1] - 8)
    err = np.maximum(np.abs(g - r)[..., a], np.abs(g - r)[..., b])
    assert np.all(err <= unit)


def test_splice_host_checks():
    ckv, kpe = _pools(840, 1, 4)
    chunk = _bf16(W.normal_bf16(840, 5, (1, 100, 512), 1.0))
    chunk_k = _bf16(W.normal_bf16(840, 6, (1, 100, 64), 1.0))
    table = _i32(np.arange(2))
    with pytest.raises(mla.MlaError) as e:  # 100 tokens from slot 40 overrun 2 blocks
        mla.fetch_splice(chunk, chunk_k, _bf16(ckv), _bf16(kpe), table, 40, 0)
    assert e.value.status == mla.MLA_ERR_INVALID_ARGUMENT
    with pytest.raises(mla.MlaError):
        mla.fetch_splice(chunk, chunk_k, _bf16(ckv), _bf16(kpe), table, 0, 0, pairing=2)
