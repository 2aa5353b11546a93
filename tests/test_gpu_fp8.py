"""fp8-e4m3 latent-cache path against the oracle on the dequantised values.

The cache pools hold OCP E4M3FN codes with fp32 scales per 64-token block:
one scale for the whole 576-wide entries (the same array passed for both
pools), or separate latent and RoPE scales (two arrays), which the library
handles on a path of its own.  The oracle decodes every code exactly and
multiplies by the block scale in fp64; the GPU path must meet the same bar as
bf16 (row-normwise 1e-2, lse 1e-3).
"""
import numpy as np
import pytest

import oracle
from paper_2606_01502_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _check(w, n_splits=0, what="", jobs=None, row_tile=0):
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale, n_splits=n_splits, row_tile=row_tile)
    if jobs is None:
        ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                      w.ckv_scale, w.kpe_scale)
    else:
        jobs = np.asarray(jobs)
        ref_o, ref_l = oracle.partial(w.q_lat[jobs], w.q_pe[jobs], w.ckv, w.kpe, w.table[jobs],
                                      w.sel[jobs], w.scale, w.ckv_scale, w.kpe_scale)
        out, lse = out[jobs], lse[jobs]
    return G.assert_parity(out, lse, ref_o, ref_l, what or w.name)


@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("n_splits", [0, 1, 3, 7])
def test_fp8_random_splits(n_splits, shared):
    print(f"case: fp8 random splits={n_splits} shared={shared}", flush=True)
    w = W.random_case(201, R=3, Mq=1, H=128, P=20, NB=9, K=7, sigma=0.5).to_fp8(shared)
    for rt in (64, 128):
        _check(w, n_splits, f"fp8 splits={n_splits} row_tile={rt}", row_tile=rt)


@pytest.mark.parametrize("mq,h", [(1, 1), (1, 16), (2, 40), (1, 64), (3, 64), (2, 128), (5, 31)])
def test_fp8_ragged_rows(mq, h):
    print(f"case: fp8 ragged mq={mq} h={h}", flush=True)
    w = W.random_case(202 + 1000 * mq + h, R=2, Mq=mq, H=h, P=12, NB=6, K=3, sigma=0.7)
    for rt in (64, 128):
        _check(w.to_fp8(), 0, f"ragged {mq}x{h} shared row_tile={rt}", row_tile=rt)
        _check(w.to_fp8(shared_scale=False), 0, f"ragged {mq}x{h} separate row_tile={rt}",
               row_tile=rt)


@pytest.mark.parametrize("shared", [True, False])
def test_fp8_padding_duplicates_empty(shared):
    print(f"case: fp8 padding shared={shared}", flush=True)
    w = W.random_case(203, R=4, Mq=1, H=32, P=10, NB=6, K=6, n_valid=[0, 1, 3, 6],
                      allow_dup=True, pad_pattern="interleaved").to_fp8(shared)
    for s in (0, 1, 2, 6):
        _check(w, s, f"fp8 padding splits={s}")


def _every_code_pool(seed, P):
    """Pools whose codes run through every finite E4M3FN code (0x7F and 0xFF
    are NaN and left out) in a seeded order, so each code meets every column
    and lane position over the pool."""
    finite = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    rng = np.random.default_rng([seed, 77])

    def fill(n):
        reps = -(-n // finite.size)
        return np.concatenate([rng.permutation(finite) for _ in range(reps)])[:n]

    ckv = fill(P * 64 * 512).reshape(P, 64, 512)
    kpe = fill(P * 64 * 64).reshape(P, 64, 64)
    return ckv, kpe


@pytest.mark.parametrize("ratio", [None, 1.0, 37.0, 1.0 / 53.0])
def test_fp8_every_code_and_scale_ratios(ratio):
    """All 254 finite codes, including +-448, the subnormals and -0, under
    per-block scales that differ from block to block; ratio None passes one
    scale array for both pools, otherwise the RoPE scales differ from the
    latent ones by about `ratio`."""
    print(f"case: fp8 every code ratio={ratio}", flush=True)
    P = 10
    base = W.random_case(204, R=2, Mq=1, H=128, P=P, NB=8, K=8, n_valid=[8, 5])
    ckv, kpe = _every_code_pool(204, P)
    rng = np.random.default_rng([204, 78])
    cs = (rng.uniform(0.3, 3.0, P) / 448.0).astype(np.float32)
    if ratio is None:
        ks = cs
    else:
        ks = (cs * np.float32(ratio) * rng.uniform(0.5, 2.0, P)).astype(np.float32)
    w = W.Workload("every-code", base.q_lat, base.q_pe, ckv, kpe, base.table, base.sel,
                   ckv_scale=cs, kpe_scale=ks)
    for s in (0, 1, 3):
        _check(w, s, f"every code ratio={ratio} splits={s}")


def test_fp8_zero_blocks():
    """Blocks that quantise to all-zero codes (scale 1 by the absmax rule)
    next to ordinary blocks."""
    print("case: fp8 zero blocks", flush=True)
    w = W.random_case(205, R=2, Mq=1, H=64, P=8, NB=8, K=6, sigma=0.5)
    w.ckv = w.ckv.copy()
    w.kpe = w.kpe.copy()
    w.ckv[[1, 4]] = 0
    w.kpe[[1, 4]] = 0
    w.kpe[6] = 0  # RoPE part zero, latent part not
    _check(w.to_fp8(), 0, "fp8 zero blocks shared")
    _check(w.to_fp8(shared_scale=False), 0, "fp8 zero blocks separate")


@pytest.mark.parametrize("shared", [True, False])
def test_fp8_many_slots(shared):
    print(f"case: fp8 many slots shared={shared}", flush=True)
    w = W.random_case(206, R=1, Mq=1, H=128, P=1200, NB=1100, K=1100, sigma=0.5).to_fp8(shared)
    for s in (1, 0):
        _check(w, s, f"fp8 many slots splits={s}")


def test_dense_local_fp8_config_sampled():
    """The dense-local workload with an fp8 cache at full size (32 jobs x 1024
    blocks x 128 heads): every job on the GPU, three jobs on the oracle; the
    fp8-vs-bf16 difference of the GPU results is printed, not gated."""
    print("case: dense-local-fp8 sampled", flush=True)
    wb = W.make("dense-local")
    w8 = wb.to_fp8()
    jobs = [0, 17, 31]
    _check(w8, 0, "dense-local-fp8", jobs=jobs)
    out8, lse8 = G.run_partial(G.upload(w8), w8.scale)
    outb, lseb = G.run_partial(G.upload(wb), wb.scale)
    print(f"fp8 vs bf16 cache: max row-rel {G.row_errors(out8, outb).max():.3g}, "
          f"max lse {np.abs(lse8 - lseb).max():.3g}", flush=True)
