"""HIP path against the oracle, element by element, through the C ABI.

Small cases cover several tiles, ragged row counts, empty / padded /
duplicated / invalid selections and every split-K setting; the workload
configurations run at full size, compared on the rows the oracle can afford.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _oracle(w, jobs=None):
    if jobs is None:
        return oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                              w.ckv_scale, w.kpe_scale)
    jobs = np.asarray(jobs)
    return oracle.partial(w.q_lat[jobs], w.q_pe[jobs], w.ckv, w.kpe, w.table[jobs], w.sel[jobs],
                          w.scale, w.ckv_scale, w.kpe_scale)


def _check_case(w, n_splits=0, what="", row_tile=0):
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale, n_splits=n_splits, row_tile=row_tile)
    ref_o, ref_l = _oracle(w)
    return G.assert_parity(out, lse, ref_o, ref_l, what or w.name)


def test_tiny_config():
    print("case: tiny", flush=True)
    _check_case(W.tiny())


@pytest.mark.parametrize("n_splits", [0, 1, 2, 3, 7])
def test_small_random_all_splits(n_splits):
    print(f"case: random splits={n_splits}", flush=True)
    w = W.random_case(101, R=3, Mq=1, H=16, P=20, NB=9, K=7)
    _check_case(w, n_splits)


@pytest.mark.parametrize("row_tile", [0, 64, 128])
@pytest.mark.parametrize("mq,h", [(1, 1), (3, 7), (1, 64), (2, 40), (1, 128), (2, 128), (5, 31)])
def test_ragged_rows(mq, h, row_tile):
    """Row counts below, at and above the 64- and 128-row tiles, with the
    library's tile choice and each tile size forced."""
    print(f"case: ragged mq={mq} h={h} row_tile={row_tile}", flush=True)
    w = W.random_case(102 + mq * 1000 + h, R=2, Mq=mq, H=h, P=12, NB=6, K=3, sigma=0.7)
    _check_case(w, row_tile=row_tile)


def test_padding_duplicates_and_empty_jobs():
    print("case: padding", flush=True)
    w = W.random_case(103, R=4, Mq=3, H=32, P=10, NB=6, K=6, n_valid=[0, 1, 3, 6],
                      allow_dup=True, pad_pattern="interleaved")
    for s in (0, 1, 2, 6):
        for rt in (64, 128):
            _check_case(w, s, f"padding splits={s} row_tile={rt}", row_tile=rt)


def test_no_slots_at_all():
    print("case: K=0", flush=True)
    w = W.random_case(104, R=2, Mq=1, H=16, P=4, NB=4, K=1)
    w.sel = np.zeros((2, 0), np.int32)
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale)
    assert np.all(out == 0) and np.all(lse == -np.inf)


def test_invalid_ids_are_skipped():
    """Ids outside [0, NB) and table entries outside [0, P) count as empty
    slots (the header's documented behaviour)."""
    print("case: invalid ids", flush=True)
    w = W.random_case(105, R=2, Mq=1, H=16, P=8, NB=5, K=4)
    sel = w.sel.copy()
    sel[0, 1] = 5          # >= NB
    sel[1, 2] = -7         # negative, not -1
    table = w.table.copy()
    table[1, sel[1, 0]] = 8  # >= P
    w_bad = W.Workload("bad", w.q_lat, w.q_pe, w.ckv, w.kpe, table, sel)
    t = G.upload(w_bad)
    out, lse = G.run_partial(t, w.scale)
    clean = sel.copy()
    clean[0, 1] = -1
    clean[1, 2] = -1
    clean[1, 0] = -1
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, table, clean, w.scale)
    G.assert_parity(out, lse, ref_o, ref_l, "invalid ids")


def test_large_scale_near_one_hot():
    print("case: one-hot", flush=True)
    w = W.random_case(106, R=1, Mq=1, H=16, P=6, NB=4, K=4)
    w.scale = 2.0
    _check_case(w)


@pytest.mark.parametrize("scale", [-0.07, 0.0])
@pytest.mark.parametrize("kind", ["blocks", "tokens", "per_row", "fp8"])
def test_nonpositive_scale(kind, scale):
    """Any finite scale is allowed: a negative scale weights the lowest scores
    most, and a zero scale gives every selected token the same weight."""
    import dataclasses
    print(f"case: scale={scale} kind={kind}", flush=True)
    if kind == "tokens":
        w = W.random_case(111, R=2, Mq=1, H=64, P=40, NB=30, K=100, tokens=True)
    elif kind == "per_row":
        w = W.random_case(112, R=2, Mq=3, H=16, P=20, NB=9, K=5, per_row=True)
    else:
        w = W.random_case(113, R=2, Mq=2, H=40, P=20, NB=9, K=7, sigma=2.0)
        if kind == "fp8":
            w = w.to_fp8(False)
    w = dataclasses.replace(w, scale=scale)
    t = G.upload(w)
    for n_splits in (1, 3):
        out, lse = G.run_partial(t, w.scale, n_splits=n_splits, tokens=kind == "tokens")
        ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                      w.ckv_scale, w.kpe_scale, tokens=kind == "tokens")
        G.assert_parity(out, lse, ref_o, ref_l, f"{kind} scale={scale} splits={n_splits}")


def test_zero_query_gives_mean():
    print("case: zero query", flush=True)
    w = W.random_case(107, R=1, Mq=1, H=16, P=6, NB=4, K=3)
    w.q_lat = np.zeros_like(w.q_lat)
    w.q_pe = np.zeros_like(w.q_pe)
    _check_case(w)


def test_many_slots_split_limits():
    """More slots than one workgroup compacts at once (1024) and long splits."""
    print("case: many slots", flush=True)
    w = W.random_case(108, R=1, Mq=1, H=16, P=1500, NB=1400, K=1300, sigma=0.5)
    for s in (1, 2, 0):
        _check_case(w, s, f"many slots splits={s}")


@pytest.mark.parametrize("jobs,heads,n_splits", [(2, 16, 3), (16, 128, 2), (16, 128, 32)])
def test_split_workspace_formats(jobs, heads, n_splits):
    """Split rows below a megabyte (2 jobs x 16 rows x 3 splits, 192 KB as
    fp32) stay fp32; 8 MB (two splits of 16 x 128 rows) and 134 MB (thirty-
    two) are stored as scaled fp16.  All against the oracle on up to three
    jobs."""
    print(f"case: workspace format jobs={jobs} heads={heads} splits={n_splits}", flush=True)
    w = W.random_case(111, R=jobs, Mq=1, H=heads, P=80, NB=70, K=64, sigma=0.5)
    t = G.upload(w)
    out, lse = G.run_partial(t, w.scale, n_splits=n_splits)
    sample = [0, 7, 15] if jobs == 16 else [0, 1]
    ref_o, ref_l = _oracle(w, sample)
    G.assert_parity(out[sample], lse[sample], ref_o, ref_l, f"workspace splits={n_splits}")


def test_split_invariance_gpu_only():
    """Different split plans agree with each other within rounding."""
    print("case: split invariance", flush=True)
    w = W.random_case(109, R=2, Mq=1, H=128, P=40, NB=33, K=32, sigma=0.5)
    t = G.upload(w)
    outs = [G.run_partial(t, w.scale, n_splits=s, row_tile=rt) for rt in (128, 64)
            for s in (1, 2, 4, 32)]
    for o, l in outs[1:]:
        assert np.abs(l - outs[0][1]).max() < 1e-4
        assert G.row_errors(o, outs[0][0]).max() < 5e-3


def test_deterministic_run_to_run():
    print("case: determinism", flush=True)
    w = W.random_case(110, R=3, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    t = G.upload(w)
    a = G.run_partial(t, w.scale, n_splits=3)
    b = G.run_partial(t, w.scale, n_splits=3)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_dsv3_one_request_config():
    print("case: dsv3-one-request", flush=True)
    _check_case(W.dsv3_one_request())


def test_few_head_config_full():
    print("case: few-head full", flush=True)
    _check_case(W.few_head())


@pytest.mark.parametrize("n_splits", [1, 3])
@pytest.mark.parametrize("tokens", [False, True])
def test_strided_queries_and_outputs(n_splits, tokens):
    """q_lat / q_pe as views with padded strides on the R, Mq and H dims, and
    out_lat / out_lse written into views of larger buffers: the results equal
    those of contiguous tensors bit for bit, and nothing outside the views
    is written."""
    print(f"case: strided splits={n_splits} tokens={tokens}", flush=True)
    w = W.random_case(112, R=3, Mq=2, H=40, P=20, NB=9, K=100 if tokens else 6, sigma=0.7,
                      tokens=tokens)
    t = G.upload(w)
    dev = G.device()
    R, Mq, H = 3, 2, 40
    # queries inside larger buffers: padding on every outer dim
    big_l = torch.zeros((R + 1, Mq + 1, H + 3, 512 + 64), dtype=torch.bfloat16, device=dev)
    big_p = torch.zeros((R, Mq, H + 5, 64 + 32), dtype=torch.bfloat16, device=dev)
    ql = big_l[1:, :Mq, 2:2 + H, 64:576]
    qp = big_p[:, :, 3:3 + H, 16:80]
    ql.copy_(t["q_lat"])
    qp.copy_(t["q_pe"])
    out_big = torch.full((R, Mq, H + 2, 512 + 8), 7.0, dtype=torch.float32, device=dev)
    lse_big = torch.full((R, Mq + 1, H + 4), 7.0, dtype=torch.float32, device=dev)
    out_v = out_big[:, :, 1:1 + H, 4:516]
    lse_v = lse_big[:, 1:, 2:2 + H]
    mla.sparse_partial_attn(ql, qp, t["ckv"], t["kpe"], t["table"], t["sel"], w.scale, out_v,
                            lse_v, n_splits=n_splits, tokens=tokens)
    ref_o, ref_l = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                           t["sel"], w.scale, n_splits=n_splits, tokens=tokens)
    torch.cuda.synchronize()
    assert torch.equal(out_v, ref_o) and torch.equal(lse_v, ref_l)
    mask = torch.ones_like(out_big, dtype=torch.bool)
    mask[:, :, 1:1 + H, 4:516] = False
    assert bool((out_big[mask] == 7.0).all()), "a write landed outside out_lat's view"
    mask = torch.ones_like(lse_big, dtype=torch.bool)
    mask[:, 1:, 2:2 + H] = False
    assert bool((lse_big[mask] == 7.0).all()), "a write landed outside out_lse's view"
    o_or, l_or = _oracle(w) if not tokens else oracle.partial(
        w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, tokens=True)
    G.assert_parity(out_v.cpu().numpy().astype(np.float64), lse_v.cpu().numpy().astype(np.float64),
                    o_or, l_or, "strided")


def test_dense_local_bf16_config_sampled():
    """The dense-local workload with a bf16 cache at full size (32 jobs x 1024
    blocks x 128 heads, each job attending all 65,536 tokens of its chunk,
    the dense holder of Section 6.3): every job on the GPU with the library's
    plan (128-row tiles, long splits, the scaled-fp16 split workspace), three
    jobs on the oracle."""
    print("case: dense-local bf16 sampled", flush=True)
    w = W.make("dense-local")
    jobs = [0, 17, 31]
    out, lse = G.run_partial(G.upload(w), w.scale)
    ref_o, ref_l = _oracle(w, jobs)
    rel, lerr = G.assert_parity(out[jobs], lse[jobs], ref_o, ref_l, "dense-local bf16")
    print(f"dense-local bf16: max row-rel {rel:.3g}, max lse {lerr:.3g}", flush=True)


@pytest.mark.parametrize("mode", ["blocks", "tokens", "per_row"])
@pytest.mark.parametrize("n_splits", [0, 2])
def test_shared_q_rows(mode, n_splits):
    """q with R_q < R rows: job r reads q row r mod R_q (a request's q sent
    once for all its chunks).  Bit-identical to the same q replicated per job,
    and equal to the oracle on the replicated q."""
    print(f"case: shared q rows {mode} splits={n_splits}", flush=True)
    Rq, R = 2, 8
    w = W.random_case(120, R=R, Mq=2, H=16, P=30, NB=10, K=150 if mode == "tokens" else 6,
                      tokens=mode == "tokens", per_row=mode == "per_row")
    w.q_lat = np.ascontiguousarray(np.tile(w.q_lat[:Rq], (R // Rq, 1, 1, 1)))
    w.q_pe = np.ascontiguousarray(np.tile(w.q_pe[:Rq], (R // Rq, 1, 1, 1)))
    t = G.upload(w)
    full = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"], t["sel"],
                                   w.scale, n_splits=n_splits, tokens=w.tokens)
    shared = mla.sparse_partial_attn(t["q_lat"][:Rq], t["q_pe"][:Rq], t["ckv"], t["kpe"],
                                     t["table"], t["sel"], w.scale, n_splits=n_splits,
                                     tokens=w.tokens)
    torch.cuda.synchronize()
    assert torch.equal(full[0], shared[0]) and torch.equal(full[1], shared[1])
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                  tokens=w.tokens)
    G.assert_parity(shared[0].cpu().numpy().astype(np.float64),
                    shared[1].cpu().numpy().astype(np.float64), ref_o, ref_l,
                    f"shared q {mode} splits={n_splits}")


def test_shared_q_rows_must_divide_the_jobs():
    print("case: shared q rows that do not divide R", flush=True)
    w = W.random_case(121, R=6, Mq=1, H=16, P=10, NB=5, K=3)
    t = G.upload(w)
    for rq in (4, 5):
        with pytest.raises(mla.MlaError) as e:
            mla.sparse_partial_attn(t["q_lat"][:rq], t["q_pe"][:rq], t["ckv"], t["kpe"], t["table"],
                                    t["sel"], w.scale)
        assert e.value.status == mla.MLA_ERR_INVALID_ARGUMENT and "divide" in str(e.value)
