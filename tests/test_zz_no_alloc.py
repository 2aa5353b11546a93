"""The allocation-free entry point (mla_sparse_partial_attn_noalloc), for
callers that cannot allocate device memory: its split-K partials live in the
library's static scratch array.  Through the C ABI, against the allocating
entry point on the same inputs (the same kernels: equal bit for bit) and
against the oracle, on two calls in a row, the second smaller than the
first (the array keeps the first call's contents); then inside a captured
HIP graph on a stream that never made an allocating call."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _run(t, w, n_splits, row_tile, no_alloc):
    out, lse = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       t["sel"], w.scale, ckv_scale=t["ckv_scale"],
                                       kpe_scale=t["kpe_scale"], n_splits=n_splits,
                                       row_tile=row_tile, no_alloc=no_alloc)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("fp8", [False, True])
def test_no_alloc_matches_allocating_entry(fp8):
    print(f"case: no-alloc fp8={fp8}", flush=True)
    big = W.random_case(901, R=6, Mq=2, H=64, P=60, NB=40, K=24, sigma=0.6, allow_dup=True)
    small = W.random_case(902, R=2, Mq=1, H=128, P=20, NB=10, K=7, sigma=0.6)
    if fp8:
        big, small = big.to_fp8(shared_scale=False), small.to_fp8()
    for w, n_splits, rt in ((big, 5, 128), (small, 3, 64)):
        t = G.upload(w)
        o_a, l_a = _run(t, w, n_splits, rt, no_alloc=True)
        o_b, l_b = _run(t, w, n_splits, rt, no_alloc=False)
        assert torch.equal(o_a, o_b) and torch.equal(l_a, l_b), w.name
        ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                      w.ckv_scale, w.kpe_scale)
        G.assert_parity(o_a.cpu().numpy().astype(np.float64),
                        l_a.cpu().numpy().astype(np.float64), ref_o, ref_l, f"no-alloc {w.name}")


def test_no_alloc_rejects_beyond_scratch():
    """A call whose partials exceed the 64 MiB array is refused before
    anything is enqueued, with its outputs untouched."""
    print("case: no-alloc too large", flush=True)
    dev = G.device()
    R, H, K = 64, 128, 40
    q_lat = torch.zeros((R, 1, H, 512), dtype=torch.bfloat16, device=dev)
    q_pe = torch.zeros((R, 1, H, 64), dtype=torch.bfloat16, device=dev)
    ckv = torch.zeros((K, 64, 512), dtype=torch.bfloat16, device=dev)
    kpe = torch.zeros((K, 64, 64), dtype=torch.bfloat16, device=dev)
    table = torch.arange(K, dtype=torch.int32, device=dev).repeat(R, 1)
    sel = table.clone()
    out = torch.full((R, 1, H, 512), 7.25, dtype=torch.float32, device=dev)
    lse = torch.full((R, 1, H), 7.25, dtype=torch.float32, device=dev)
    with pytest.raises(mla.MlaError) as e:
        mla.sparse_partial_attn(q_lat, q_pe, ckv, kpe, table, sel, 0.1, out, lse, n_splits=40,
                                row_tile=128, no_alloc=True)
    assert e.value.status == mla.MLA_ERR_UNSUPPORTED and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.25).all()) and bool((lse == 7.25).all())


def test_no_alloc_under_graph_capture():
    """Captured on a fresh stream (no workspace of its own) the call needs no
    allocation; replays reproduce the eager result, with eager work between
    them."""
    print("case: no-alloc graph capture", flush=True)
    dev = G.device()
    w = W.random_case(903, R=3, Mq=1, H=128, P=30, NB=16, K=10, sigma=0.5)
    t = G.upload(w)
    out = torch.empty((3, 1, 128, 512), dtype=torch.float32, device=dev)
    lse = torch.empty((3, 1, 128), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()

    def call():
        mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"], t["sel"],
                                w.scale, out, lse, n_splits=4, no_alloc=True)

    with torch.cuda.stream(stream):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            call()
        call()
        stream.synchronize()
        ref = (out.clone(), lse.clone())
        for rep in range(3):
            out.fill_(float("nan"))
            stream.synchronize()
            g.replay()
            stream.synchronize()
            assert torch.equal(out, ref[0]) and torch.equal(lse, ref[1]), f"replay {rep}"
            call()
            stream.synchronize()
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale)
    G.assert_parity(ref[0].cpu().numpy().astype(np.float64), ref[1].cpu().numpy().astype(np.float64),
                    ref_o, ref_l, "no-alloc captured")
