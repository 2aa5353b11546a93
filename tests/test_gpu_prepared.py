"""Prepared calls (descriptors built once, stream fixed) give the same
results as the direct calls, also after the input buffers' contents change
between calls."""
import numpy as np
import pytest
import torch

from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def test_prepared_partial_and_merge_match_direct_calls():
    print("case: prepared calls", flush=True)
    w = W.random_case(501, R=4, Mq=2, H=64, P=30, NB=16, K=10, sigma=0.5)
    w2 = W.random_case(502, R=4, Mq=2, H=64, P=30, NB=16, K=10, sigma=0.5)
    t, t2 = G.upload(w), G.upload(w2)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        o, l = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       t["sel"], w.scale, n_splits=3)
        m, ml = mla.merge_partials([o[0:2], o[2:4]], [l[0:2], l[2:4]], out_lse=True)
        stream.synchronize()
        ref = [x.clone() for x in (o, l, m, ml)]
        po = torch.full_like(o, float("nan"))
        pl = torch.full_like(l, float("nan"))
        part = mla.prepare_partial(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                   t["sel"], w.scale, po, pl, n_splits=3, stream=stream)
        merge = mla.prepare_merge([po[0:2], po[2:4]], [pl[0:2], pl[2:4]], out_lse=True,
                                  stream=stream)
        for rep in range(2):
            part()
            pm, pml = merge()
            stream.synchronize()
            for a, b in zip((po, pl, pm, pml), ref):
                assert torch.equal(a, b), f"prepared call {rep} differs from the direct call"
        # new contents in the same buffers: the prepared call reads them
        for k in ("q_lat", "q_pe", "ckv", "kpe", "table", "sel"):
            t[k].copy_(t2[k])
        part()
        stream.synchronize()
        o2, l2 = mla.sparse_partial_attn(t2["q_lat"], t2["q_pe"], t2["ckv"], t2["kpe"],
                                         t2["table"], t2["sel"], w.scale, n_splits=3)
        stream.synchronize()
        assert torch.equal(po, o2) and torch.equal(pl, l2)
    torch.cuda.synchronize()
