"""The bf16 wire form of the partial (Section 3.2: 1032 bytes per row, a bf16
output row with the fp32 pair (m, l)) against the oracle, through the C ABI.

The wire form is the fp32 form rounded: out_lat must equal the fp32 call's
output rounded to nearest even bf16 bit for bit, on the same inputs and split
setting.  The pair must satisfy m + ln l = the fp32 call's lse, m must match
the oracle's largest score and l the oracle's denominator (relative to its
own m) at the log-sum-exp bar; an empty row is (-inf, 0) with a zero row.
Wire-form parts merge like fp32 parts: the merge of the wire partials of a
split selection matches the oracle's attention over the whole selection.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

# m and ln l each carry about the score error of the fp32 path; their sum is
# the fp32 call's lse up to a few fp32 roundings of the two formulas
PAIR_ABS_TOL = 1e-3
SUM_ABS_TOL = 1e-4


def _call(t, w, wire, n_splits=0, sel=None, row_tile=0):
    out, lse = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       t["sel"] if sel is None else sel, w.scale,
                                       ckv_scale=t["ckv_scale"], kpe_scale=t["kpe_scale"],
                                       n_splits=n_splits, row_tile=row_tile, tokens=w.tokens,
                                       wire=wire)
    torch.cuda.synchronize()
    return out, lse


def _check_wire(w, n_splits=0, row_tile=0, what=""):
    t = G.upload(w)
    o32, l32 = _call(t, w, False, n_splits, row_tile=row_tile)
    o16, ml = _call(t, w, True, n_splits, row_tile=row_tile)
    assert o16.dtype == torch.bfloat16 and tuple(ml.shape) == tuple(l32.shape) + (2,)
    # bit for bit the fp32 form rounded
    want = o32.to(torch.bfloat16)
    same = o16.view(torch.int16) == want.view(torch.int16)
    assert bool(same.all()), f"{what}: {int((~same).sum())} bf16 elements differ from the rounded fp32 form"
    o16 = o16.float().cpu().numpy().astype(np.float64)
    ml = ml.cpu().numpy().astype(np.float64)
    l32 = l32.cpu().numpy().astype(np.float64)
    m, l = ml[..., 0], ml[..., 1]
    ref_o, ref_lse, ref_m, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel,
                                                  w.scale, w.ckv_scale, w.kpe_scale,
                                                  tokens=w.tokens, stats=True)
    empty = ref_lse == -np.inf
    assert np.array_equal(m == -np.inf, empty), f"{what}: -inf pattern of m differs"
    assert np.all(l[empty] == 0.0) and np.all(o16[empty] == 0.0), f"{what}: empty rows must be (-inf, 0), 0"
    live = ~empty
    if live.any():
        # the pair is the lse split in two
        s_err = np.abs(m[live] + np.log(l[live]) - l32[live]).max()
        assert s_err <= SUM_ABS_TOL, f"{what}: m + ln l is {s_err:.3g} off the fp32 lse"
        m_err = np.abs(m[live] - ref_m[live]).max()
        assert m_err <= PAIR_ABS_TOL, f"{what}: m abs error {m_err:.3g}"
        # l is relative to the row's own largest score, so at least exp(0) = 1
        assert l[live].min() >= 1.0 - 1e-6, f"{what}: l below 1 ({l[live].min():.9g})"
        ll_err = np.abs(np.log(l[live]) - np.log(ref_l[live])).max()
        assert ll_err <= PAIR_ABS_TOL, f"{what}: ln l abs error {ll_err:.3g}"
    lse = np.where(live, m + np.log(np.where(live, l, 1.0)), -np.inf)
    G.assert_parity(o16, lse, ref_o, ref_lse, what)
    return o16, m, l


@pytest.mark.parametrize("n_splits", [0, 1, 3])
def test_wire_bf16_blocks(n_splits):
    print(f"case: wire bf16 splits={n_splits}", flush=True)
    w = W.random_case(301, R=4, Mq=2, H=40, P=24, NB=10, K=7, n_valid=[0, 1, 4, 7],
                      pad_pattern="interleaved")
    _check_wire(w, n_splits, what=f"wire bf16 splits={n_splits}")


@pytest.mark.parametrize("row_tile", [64, 128])
def test_wire_row_tiles(row_tile):
    print(f"case: wire row_tile={row_tile}", flush=True)
    w = W.random_case(302, R=2, Mq=1, H=128, P=16, NB=8, K=6)
    _check_wire(w, 0, row_tile=row_tile, what=f"wire row_tile={row_tile}")
    _check_wire(w, 2, row_tile=row_tile, what=f"wire row_tile={row_tile} splits=2")


@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("n_splits", [1, 3])
def test_wire_fp8(shared, n_splits):
    print(f"case: wire fp8 shared={shared} splits={n_splits}", flush=True)
    w = W.random_case(303, R=3, Mq=1, H=64, P=20, NB=9, K=6, n_valid=[6, 0, 3]).to_fp8(
        shared_scale=shared)
    _check_wire(w, n_splits, what=f"wire fp8 shared={shared} splits={n_splits}")


@pytest.mark.parametrize("n_splits", [1, 2])
def test_wire_per_row(n_splits):
    print(f"case: wire per-row splits={n_splits}", flush=True)
    w = W.random_case(304, R=2, Mq=4, H=16, P=24, NB=12, K=5, per_row=True,
                      n_valid=[[5, 0, 2, 5], [1, 5, 5, 3]])
    _check_wire(w, n_splits, what=f"wire per-row splits={n_splits}")


@pytest.mark.parametrize("n_splits", [1, 2])
def test_wire_tokens(n_splits):
    print(f"case: wire tokens splits={n_splits}", flush=True)
    w = W.random_case(305, R=2, Mq=1, H=32, P=16, NB=8, K=150, n_valid=[150, 0], tokens=True)
    _check_wire(w, n_splits, what=f"wire tokens splits={n_splits}")


def test_wire_dsv3_one_request_full_size():
    """The 128-head, 64-block request of the Section 6.3 decode point, whole."""
    print("case: wire dsv3-one-request", flush=True)
    _check_wire(W.make("dsv3-one-request"), 0, what="wire dsv3-one-request")


def _split_selection(w, n_parts):
    """n_parts disjoint selections whose union is w's selection: every job's
    slots dealt round robin, except job 0, whose whole selection is part 0's,
    so that its other parts are dead ((-inf, 0) pairs)."""
    parts = []
    for j in range(n_parts):
        s = np.full_like(w.sel, -1)
        s[1:, j::n_parts] = w.sel[1:, j::n_parts]
        if j == 0:
            s[0] = w.sel[0]
        parts.append(s)
    return parts


@pytest.mark.parametrize("n_parts", [2, 3, 8])
def test_wire_merge_against_oracle(n_parts):
    """Route + merge in the wire form: each part attends a disjoint share of
    the selection; the merge of the bf16 rows and (m, l) pairs must give the
    oracle's attention over the whole selection, and its lse."""
    print(f"case: wire merge parts={n_parts}", flush=True)
    w = W.random_case(306 + n_parts, R=3, Mq=2, H=24, P=40, NB=24, K=16)
    t = G.upload(w)
    dev = G.device()
    lats, pairs, lats32, lses32 = [], [], [], []
    for s in _split_selection(w, n_parts):
        sel = torch.from_numpy(s).to(dev)
        o16, ml = _call(t, w, True, 0, sel=sel)
        o32, l32 = _call(t, w, False, 0, sel=sel)
        lats.append(o16); pairs.append(ml); lats32.append(o32); lses32.append(l32)
    out, lse = mla.merge_partials(lats, pairs, out_lse=True)
    out32, lse32 = mla.merge_partials(lats32, lses32, out_lse=True)
    torch.cuda.synchronize()
    assert out.dtype == torch.float32
    ref_o, ref_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale)
    out = out.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    G.assert_parity(out, lse, ref_o, ref_lse, f"wire merge parts={n_parts}")
    # the merged lse depends only on the pairs: it matches the fp32 parts' merge
    assert np.abs(lse - lse32.cpu().numpy()).max() <= SUM_ABS_TOL
    # and the merged rows differ from the fp32 parts' merge by bf16 rounding only
    rel = G.row_errors(out, out32.cpu().numpy().astype(np.float64))
    assert rel.max() <= 2.0 ** -7, f"wire vs fp32 parts: {rel.max():.3g}"


def test_wire_rejections_write_nothing():
    """The wire form's own shape and dtype rules."""
    print("case: wire rejections", flush=True)
    w = W.random_case(310, R=2, Mq=1, H=16, P=8, NB=4, K=3)
    t = G.upload(w)
    dev = G.device()
    R, Mq, H = 2, 1, 16
    cases = [
        ("fp32 rows", torch.empty((R, Mq, H, 512), dtype=torch.float32, device=dev),
         torch.empty((R, Mq, H, 2), dtype=torch.float32, device=dev), "wrong dtype"),
        ("lse without pairs", torch.empty((R, Mq, H, 512), dtype=torch.bfloat16, device=dev),
         torch.empty((R, Mq, H), dtype=torch.float32, device=dev), "expected 4 dims"),
        ("three per row", torch.empty((R, Mq, H, 512), dtype=torch.bfloat16, device=dev),
         torch.empty((R, Mq, H, 3), dtype=torch.float32, device=dev), "(m, l) pairs"),
    ]
    for name, o, l, text in cases:
        o.view(torch.int16).fill_(0x5a5a) if o.dtype == torch.bfloat16 else o.fill_(7.0)
        l.fill_(7.0)
        o0, l0 = o.clone(), l.clone()
        with pytest.raises(mla.MlaError) as e:
            mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                    t["sel"], w.scale, out_lat=o, out_lse=l, wire=True)
        assert text in str(e.value), (name, str(e.value))
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16) if o.dtype == torch.bfloat16 else o,
                           o0.view(torch.int16) if o0.dtype == torch.bfloat16 else o0), name
        assert torch.equal(l, l0), name


@pytest.mark.parametrize("fp8", [False, True])
def test_wire_through_the_allocation_free_entry_point(fp8):
    """The wire form through mla_sparse_partial_attn_noalloc (split partials in
    the static scratch array, the largest score kept beside each split's lse)
    equals the allocating entry point's wire output bit for bit."""
    print(f"case: wire no-alloc fp8={fp8}", flush=True)
    w = W.random_case(311, R=3, Mq=2, H=24, P=20, NB=9, K=7, n_valid=[7, 0, 4])
    if fp8:
        w = w.to_fp8(shared_scale=False)
    t = G.upload(w)
    for n_splits in (1, 3):
        o_a, ml_a = _call(t, w, True, n_splits)
        o_n, ml_n = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                            t["sel"], w.scale, ckv_scale=t["ckv_scale"],
                                            kpe_scale=t["kpe_scale"], n_splits=n_splits,
                                            no_alloc=True, wire=True)
        torch.cuda.synchronize()
        assert torch.equal(o_a.view(torch.int16), o_n.view(torch.int16)), n_splits
        assert torch.equal(ml_a, ml_n), n_splits
