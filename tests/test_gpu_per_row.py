"""Per-row selections (sel [R, Mq, K]): one holder serving several routed
requesters on one chunk, each query row with its own selected blocks
(Section 6.3).  The library loads the union of a row tile's selections once
and masks every row to its own multiset; the oracle attends each row's
multiset directly."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _check(w, n_splits=0, what="", row_tile=0):
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale, n_splits=n_splits, row_tile=row_tile)
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale)
    return G.assert_parity(out, lse, ref_o, ref_l, what or w.name)


@pytest.mark.parametrize("mq,h", [(4, 16), (8, 16), (3, 40), (2, 128), (64, 2), (70, 1),
                                  (5, 31), (1, 64)])
@pytest.mark.parametrize("row_tile", [0, 64, 128])
def test_per_row_layouts(mq, h, row_tile):
    """Row tiles of 128 rows spanning 8 query rows, tiles straddling query
    rows (H = 40, 31), one query row per tile (H = 128), 64 query rows per
    tile (H = 2), and H = 1, where a 128-row tile would span more query rows
    than a mask holds (the library takes 64-row tiles; forcing 128 fails)."""
    print(f"case: per-row mq={mq} h={h} row_tile={row_tile}", flush=True)
    w = W.random_case(600 + 100 * mq + h, R=2, Mq=mq, H=h, P=30, NB=12, K=6, sigma=0.7,
                      per_row=True, shared_frac=0.6)
    if h == 1 and mq > 64 and row_tile == 128:
        with pytest.raises(mla.MlaError) as e:
            _check(w, 0, row_tile=row_tile)
        assert e.value.status == mla.MLA_ERR_UNSUPPORTED
        return
    _check(w, 0, f"per-row {mq}x{h} row_tile={row_tile}", row_tile=row_tile)


@pytest.mark.parametrize("n_splits", [1, 2, 3, 7])
def test_per_row_splits_duplicates_padding(n_splits):
    """Duplicated ids within a row (counted twice for that row only),
    interleaved empty slots, a row with nothing selected, split-K."""
    print(f"case: per-row splits={n_splits}", flush=True)
    n_valid = [[7, 0, 3, 7], [1, 7, 5, 2]]
    w = W.random_case(650 + n_splits, R=2, Mq=4, H=16, P=20, NB=9, K=7, sigma=0.6,
                      n_valid=n_valid, allow_dup=True, pad_pattern="interleaved",
                      per_row=True, shared_frac=0.5)
    assert (w.sel[0, 1] == -1).all()
    for rt in (64, 128):
        _check(w, n_splits, f"per-row dup splits={n_splits} row_tile={rt}", row_tile=rt)


@pytest.mark.parametrize("n_splits", [0, 1, 5])
def test_per_row_long_selections_split_by_slot(n_splits):
    """Four query rows per 128-row tile selecting 300 blocks each: the tile's
    slots overflow one block list, so splits take slot ranges (the short
    selections above split by logical block instead); ids repeat across and
    within rows."""
    print(f"case: per-row long selections splits={n_splits}", flush=True)
    w = W.random_case(655 + n_splits, R=1, Mq=4, H=32, P=500, NB=400, K=300, sigma=0.5,
                      allow_dup=True, per_row=True, shared_frac=0.5)
    _check(w, n_splits, f"per-row K=300 splits={n_splits}")


def test_per_row_invalid_ids_are_skipped():
    print("case: per-row invalid ids", flush=True)
    w = W.random_case(660, R=2, Mq=3, H=16, P=10, NB=6, K=4, per_row=True)
    sel = w.sel.copy()
    sel[0, 1, 1] = 6           # >= NB
    sel[1, 2, 0] = -3          # negative, not -1
    table = w.table.copy()
    table[1, sel[1, 0, 2]] = 10  # >= P: every row selecting this id skips it
    bad = W.Workload("bad", w.q_lat, w.q_pe, w.ckv, w.kpe, table, sel)
    t = G.upload(bad)
    out, lse = G.run_partial(t, w.scale)
    clean = sel.copy()
    clean[0, 1, 1] = -1
    clean[1, 2, 0] = -1
    clean[1][sel[1] == sel[1, 0, 2]] = -1
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, table, clean, w.scale)
    G.assert_parity(out, lse, ref_o, ref_l, "per-row invalid ids")


def test_per_row_equal_rows_match_shared_selection():
    """All rows selecting the same blocks: the per-row form equals the
    shared-selection form (the union is that selection, every mask full)."""
    print("case: per-row equal rows", flush=True)
    w = W.random_case(670, R=3, Mq=8, H=16, P=40, NB=16, K=10, sigma=0.5, allow_dup=True)
    sel3 = np.ascontiguousarray(np.broadcast_to(w.sel[:, None, :], (3, 8, 10)))
    t = G.upload(w)
    out2, lse2 = G.run_partial(t, w.scale)
    out3, lse3 = G.run_partial(t, w.scale, sel=torch.from_numpy(sel3).to(G.device()))
    G.assert_parity(out3, lse3, out2, lse2, "per-row vs shared")


def test_per_row_many_requesters_sampled():
    """64 requesters x 16 heads on one 128-block chunk, each selecting 32
    blocks with heavy overlap (8 row tiles, unions of up to 128 blocks); the
    oracle checks 12 of the 64 requesters."""
    print("case: per-row 64 requesters", flush=True)
    w = W.random_case(680, R=1, Mq=64, H=16, P=400, NB=128, K=32, sigma=0.5, per_row=True,
                      shared_frac=0.7)
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale)
    rows = np.array([0, 1, 7, 8, 15, 20, 31, 32, 47, 50, 62, 63])
    ref_o, ref_l = oracle.partial(w.q_lat[:, rows], w.q_pe[:, rows], w.ckv, w.kpe, w.table,
                                  w.sel[:, rows], w.scale)
    G.assert_parity(out[:, rows], lse[:, rows], ref_o, ref_l, "per-row 64 requesters")


def _check8(w, n_splits=0, row_tile=0, what=""):
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale, n_splits=n_splits, row_tile=row_tile)
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                  w.ckv_scale, w.kpe_scale)
    return G.assert_parity(out, lse, ref_o, ref_l, what)


@pytest.mark.parametrize("row_tile", [64, 128])
@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("mq,h,k", [(8, 16, 6), (4, 32, 140), (3, 40, 9)])
def test_per_row_fp8(mq, h, k, shared, row_tile):
    """fp8 caches with a selection per query row: block splits (short
    selections) and slot-range splits (140 slots x 4 query rows of a
    128-row tile overflow the fp8 per-row list of 512), duplicates and
    padding, both scale layouts."""
    print(f"case: per-row fp8 {mq}x{h} K={k} shared={shared} row_tile={row_tile}", flush=True)
    w = W.random_case(690 + mq + h + k, R=2, Mq=mq, H=h, P=60, NB=50, K=k, sigma=0.7,
                      allow_dup=True, pad_pattern="interleaved", per_row=True, shared_frac=0.6)
    w8 = w.to_fp8(shared)
    for s_ in (0, 3):
        _check8(w8, s_, row_tile, f"per-row fp8 {mq}x{h} K={k} splits={s_}")


@pytest.mark.parametrize("kind", ["dense", "sparse"])
def test_holder_rows_match_jobs_and_oracle(kind):
    """The holder workload served as one job whose query rows are the
    requesters equals the same requesters routed as separate jobs, and both
    match the oracle on sampled requesters."""
    print(f"case: holder {kind} rows vs jobs", flush=True)
    n, h = 24, 16
    wr = W.make(f"holder-{kind}-n{n}-h{h}")
    wj = W.make(f"holder-{kind}-n{n}-h{h}-jobs")
    out_r, lse_r = G.run_partial(G.upload(wr), wr.scale)
    out_j, lse_j = G.run_partial(G.upload(wj), wj.scale)
    G.assert_parity(out_r.reshape(out_j.shape), lse_r.reshape(lse_j.shape), out_j, lse_j,
                    f"holder {kind} rows vs jobs")
    req = np.array([0, 5, 11, 23])
    ref_o, ref_l = oracle.partial(wj.q_lat[req], wj.q_pe[req], wj.ckv, wj.kpe, wj.table[req],
                                  wj.sel[req], wj.scale)
    G.assert_parity(out_r[0, req][:, None], lse_r[0, req][:, None], ref_o, ref_l,
                    f"holder {kind} vs oracle")
