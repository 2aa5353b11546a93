"""The library's calls captured in a HIP graph and replayed.

Serving loops capture a decode step once and replay it; the benchmark times
such replays.  Every replay must reproduce the eager result exactly (the
kernels are deterministic), also with other eager work on the same stream,
which shares the split-K workspace, between the replays.
"""
import numpy as np
import pytest
import torch

from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    print("case: graph replay", flush=True)
    w = W.random_case(401, R=4, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    other = W.random_case(402, R=4, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    t, t2 = G.upload(w), G.upload(other)
    dev = G.device()
    R, Mq, H = 4, 1, 128
    out = torch.empty((R, Mq, H, 512), dtype=torch.float32, device=dev)
    lse = torch.empty((R, Mq, H), dtype=torch.float32, device=dev)
    merged = torch.empty((2, Mq, H, 512), dtype=torch.float32, device=dev)
    mlse = torch.empty((2, Mq, H), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()

    def step(tt, n_splits):
        mla.sparse_partial_attn(tt["q_lat"], tt["q_pe"], tt["ckv"], tt["kpe"], tt["table"],
                                tt["sel"], w.scale, out, lse, n_splits=n_splits)
        mla.merge_partials([out[0:2], out[2:4]], [lse[0:2], lse[2:4]], out=merged,
                           out_lse=mlse)

    with torch.cuda.stream(stream):
        step(t, 3)  # eager, also sizes this stream's workspace
        stream.synchronize()
        ref = [x.clone() for x in (out, lse, merged, mlse)]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step(t, 3)
        for rep in range(3):
            for x in (out, lse, merged, mlse):
                x.fill_(float("nan"))
            stream.synchronize()
            g.replay()
            stream.synchronize()
            got = [x.clone() for x in (out, lse, merged, mlse)]
            for a, b in zip(got, ref):
                assert torch.equal(a, b), f"replay {rep} differs from the eager result"
            # eager work on the same stream between replays (other inputs,
            # same workspace), then a synchronisation
            step(t2, 3)
            stream.synchronize()
            assert not torch.equal(out, ref[0])
    torch.cuda.synchronize()
