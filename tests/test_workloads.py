"""Input generator: rounding, fp8 quantiser and the configs' structure. CPU only."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([1.00390625, 1.01171875, -1.00390625, 3.0e-39, 0.0, -0.0],
                                 np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits(x), ref)
    assert np.array_equal(W.bf16_bits_to_f32(ref), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_e4m3_roundtrip_every_code():
    lib = oracle._load()
    codes = [c for c in range(256) if (c & 0x7F) != 0x7F]
    vals = np.array([lib.oracle_e4m3fn_to_f64(c) for c in codes])
    assert np.array_equal(W.quantize_e4m3fn(vals), np.array(codes, np.uint8))


def test_e4m3_quantiser_matches_torch_in_range():
    rng = np.random.default_rng(1)
    y = np.concatenate([rng.uniform(-448, 448, 50000), rng.standard_normal(50000) * 0.01,
                        rng.standard_normal(50000)])
    # ties: midpoints between neighbouring codes
    lib = oracle._load()
    pos = np.array([lib.oracle_e4m3fn_to_f64(c) for c in range(0x7F)])
    y = np.concatenate([y, (pos[:-1] + pos[1:]) / 2, -(pos[:-1] + pos[1:]) / 2])
    ref = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(W.quantize_e4m3fn(y), ref)


def test_e4m3_saturates():
    q = W.quantize_e4m3fn(np.array([448.0, 500.0, 1e30, -1e30, -460.0]))
    assert list(q) == [0x7E, 0x7E, 0x7E, 0xFE, 0xFE]


def test_block_quantisation_scale_and_error():
    w = W.random_case(5, R=1, Mq=1, H=1, P=3, NB=3, K=1, sigma=0.5)
    ckv = w.ckv.copy()
    ckv[1] = 0  # all-zero block -> scale 1
    codes, scales = W.quantize_blocks_e4m3fn(ckv)
    lib = oracle._load()
    dec = np.vectorize(lib.oracle_e4m3fn_to_f64)(codes)
    x = W.bf16_bits_to_f32(ckv).astype(np.float64)
    for b in range(3):
        amax = np.abs(x[b]).max()
        assert scales[b] == (np.float32(amax / np.float32(448.0)) if amax else 1.0)
        rec = dec[b] * scales[b]
        # E4M3 has 3 mantissa bits: relative error <= 2^-4 for normals, and an
        # absolute error <= 2^-10 * scale in the subnormal range
        err = np.abs(rec - x[b])
        assert np.all(err <= np.maximum(np.abs(x[b]) * 2.0 ** -4, 2.0 ** -10 * scales[b]) + 1e-30)


def test_shared_block_scale_covers_both_pools():
    """One scale per block for the 576-wide entries: absmax over ckv and kpe."""
    w = W.random_case(6, R=1, Mq=1, H=1, P=4, NB=4, K=1, sigma=0.5)
    kpe = w.kpe.copy()
    kpe[2] = W.f32_to_bf16_bits(np.full((64, 64), 7.5, np.float32))  # kpe dominates block 2
    c_codes, k_codes, scales = W.quantize_blocks_e4m3fn(w.ckv, kpe)
    xc = W.bf16_bits_to_f32(w.ckv).astype(np.float64)
    xk = W.bf16_bits_to_f32(kpe).astype(np.float64)
    for b in range(4):
        amax = max(np.abs(xc[b]).max(), np.abs(xk[b]).max())
        assert scales[b] == np.float32(amax / np.float32(448.0))
    assert scales[2] == np.float32(7.5 / 448.0)
    only_c, s_c = W.quantize_blocks_e4m3fn(w.ckv)
    assert np.array_equal(c_codes[[0, 1, 3]], only_c[[0, 1, 3]]) or not np.array_equal(
        scales[[0, 1, 3]], s_c[[0, 1, 3]])
    f = w.to_fp8()
    assert f.kpe_scale is f.ckv_scale
    g = w.to_fp8(shared_scale=False)
    assert g.kpe_scale is not g.ckv_scale


def test_config_structure_small():
    t = W.tiny()
    assert t.q_lat.shape == (1, 1, 16, 512) and t.ckv.shape == (4, 64, 512)
    assert sorted(t.table[0]) == [0, 1, 2, 3]
    assert (t.sel[0] >= 0).sum() == 2 and list(t.sel[0, 2:]) == [-1, -1]
    d = W.dsv3_one_request()
    ids = d.sel[0]
    assert len(set(ids)) == 32 and np.all(np.diff(ids) > 0) and ids.max() < 64
    assert d.algorithmic_flops() == 128 * 2048 * 2176


def test_workload_is_deterministic():
    a = W.random_case(9, R=2, Mq=1, H=2, P=5, NB=4, K=3)
    b = W.random_case(9, R=2, Mq=1, H=2, P=5, NB=4, K=3)
    for k in ("q_lat", "q_pe", "ckv", "kpe", "table", "sel"):
        assert np.array_equal(getattr(a, k), getattr(b, k))


def test_normal_groups_independent_of_threads(monkeypatch):
    a = W.normal_bf16(3, 7, (3, W._GROUP // 2 + 5), 0.5)
    monkeypatch.setattr(W, "_threads", lambda: 1)
    b = W.normal_bf16(3, 7, (3, W._GROUP // 2 + 5), 0.5)
    assert np.array_equal(a, b)


@pytest.mark.slow
def test_few_head_zipf_selection():
    w = W.few_head()
    assert w.q_lat.shape == (16, 4, 16, 512) and w.table.shape == (16, 512)
    assert all(len(set(s)) == 32 and np.all(np.diff(s) > 0) for s in w.sel)
    # Zipf(1.1) favours low positions: far more ids below 64 than uniform (1/8)
    assert (w.sel < 64).mean() > 0.3
