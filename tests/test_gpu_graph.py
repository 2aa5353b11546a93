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


def test_graph_replay_tokens_fp8_and_fetch():
    """A captured step of the other entry points: an fp8 token-selection
    partial with a large split workspace (fp16 rows), an fp8 per-row partial,
    and the FETCH gather and splice.  Replays equal the eager results, with
    eager work of other sizes between them."""
    print("case: graph replay tokens / per-row / fetch", flush=True)
    w = W.make("select-tok-b16-k2048-c8192").to_fp8(shared_scale=False)
    pr = W.random_case(403, R=2, Mq=8, H=16, P=30, NB=20, K=8, per_row=True).to_fp8()
    t, tp = G.upload(w), G.upload(pr)
    f = W.fetch_inputs("fetch-splice-c300-l2")
    g_in = W.fetch_inputs("fetch-gather-k500-c4096-l2")
    dev = G.device()

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    R, H = 16, 128
    out = torch.empty((R, 1, H, 512), dtype=torch.float32, device=dev)
    lse = torch.empty((R, 1, H), dtype=torch.float32, device=dev)
    out_p = torch.empty((2, 8, 16, 512), dtype=torch.float32, device=dev)
    lse_p = torch.empty((2, 8, 16), dtype=torch.float32, device=dev)
    cc, ck = bf16(f["chunk_ckv"]), bf16(f["chunk_kpe"])
    pool_c, pool_k, ftable = bf16(f["ckv"]), bf16(f["kpe"]), i32(f["table"])
    pool_c0, pool_k0 = pool_c.clone(), pool_k.clone()
    gc, gk, gt, gs = bf16(g_in["ckv"]), bf16(g_in["kpe"]), i32(g_in["table"]), i32(g_in["sel"])
    oc = torch.empty((2, 500, 512), dtype=torch.bfloat16, device=dev)
    ok = torch.empty((2, 500, 64), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.Stream()

    def step():
        mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"], t["sel"],
                                w.scale, out, lse, ckv_scale=t["ckv_scale"],
                                kpe_scale=t["kpe_scale"], n_splits=16, tokens=True)
        mla.sparse_partial_attn(tp["q_lat"], tp["q_pe"], tp["ckv"], tp["kpe"], tp["table"],
                                tp["sel"], pr.scale, out_p, lse_p, ckv_scale=tp["ckv_scale"],
                                kpe_scale=tp["kpe_scale"], n_splits=3)
        mla.fetch_splice(cc, ck, pool_c, pool_k, ftable, f["dst_start"], f["delta"])
        mla.fetch_gather(gc, gk, gt, gs, oc, ok)

    outs = (out, lse, out_p, lse_p, pool_c, pool_k, oc, ok)
    with torch.cuda.stream(stream):
        step()  # eager: sizes the workspace (16 splits x 2048 rows: fp16 rows)
        stream.synchronize()
        ref = [x.clone() for x in outs]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        for rep in range(3):
            for x in (out, lse, out_p, lse_p):
                x.fill_(float("nan"))
            oc.zero_()
            pool_c.copy_(pool_c0)
            pool_k.copy_(pool_k0)
            stream.synchronize()
            g.replay()
            stream.synchronize()
            for a, b in zip(outs, ref):
                assert torch.equal(a, b), f"replay {rep} differs from the eager result"
            # eager work of another size on the same stream (another split plan)
            mla.sparse_partial_attn(t["q_lat"][:2], t["q_pe"][:2], t["ckv"], t["kpe"],
                                    t["table"][:2], t["sel"][:2], w.scale,
                                    ckv_scale=t["ckv_scale"], kpe_scale=t["kpe_scale"],
                                    n_splits=2, tokens=True)
            stream.synchronize()
    torch.cuda.synchronize()
