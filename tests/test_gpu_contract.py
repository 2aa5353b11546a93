"""The contract at its edges, on the GPU, through the C ABI.

- Rejected calls write nothing: the host-side rejections of
  tests/abi_cases.py with device tensors whose outputs hold a canary.
- Softmax scales up to the accepted bound 2^64 (and down to -2^64): the
  weights are one-hot and the result is the oracle's.
- fp8 caches whose latent scale is 0 (what an absmax/448 rule gives an
  all-zero latent block), or far below the RoPE scale, and RoPE scales of 0,
  on every selection path.
- The split-K workspace after graph capture: a graph captured before the
  workspace grew still replays correctly, and the workspace refuses to grow
  during capture.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import abi_cases as C
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _snapshot(a):
    return {k: (v.clone() if torch.is_tensor(v) else [x.clone() for x in v]
                if isinstance(v, list) else None) for k, v in a.items()}


def _unchanged(a, snap, what):
    torch.cuda.synchronize()
    for k, v in a.items():
        if torch.is_tensor(v):
            assert torch.equal(v, snap[k]), f"{what}: {k} was written"
        elif isinstance(v, list):
            for x, y in zip(v, snap[k]):
                assert torch.equal(x, y), f"{what}: a {k} part was written"


def _cases(kind):
    dev = G.device()
    return {"partial": C.partial_cases, "fp8": C.partial_cases_fp8, "merge": C.merge_cases}[kind](dev)


@pytest.mark.parametrize("kind", ["partial", "fp8", "merge"])
def test_rejected_calls_write_nothing(kind):
    print(f"case: rejected {kind} calls", flush=True)
    dev = G.device()
    for name, mutate, status, text in _cases(kind):
        a = C.merge_args(dev) if kind == "merge" else C.partial_args(dev, fp8=kind == "fp8")
        mutate(a)
        snap = _snapshot(a)
        st, msg = C.call_merge(a) if kind == "merge" else C.call_partial(a)
        assert st == status and text in msg, (name, st, msg)
        _unchanged(a, snap, name)  # outputs keep their canary, inputs their values


def _decode(a):
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _scores_and_values(w, r):
    """fp64 dot products q . k [Mq, H, T] of job r's selected tokens, and
    their value rows [T, 512], from the decoded bit patterns."""
    blocks = [w.table[r, s] for s in w.sel[r] if s >= 0]
    kl = _decode(w.ckv[blocks]).reshape(-1, 512)
    kp = _decode(w.kpe[blocks]).reshape(-1, 64)
    return _decode(w.q_lat[r]) @ kl.T + _decode(w.q_pe[r]) @ kp.T, kl


@pytest.mark.parametrize("scale", [1e18, 2.0 ** 64, -(2.0 ** 64), 2.0 ** 40])
def test_huge_scales_one_hot(scale):
    """At these scales the softmax is one-hot: each row's output is the ckv
    row of its highest-scoring token, lse = scale x that score.  Rows whose
    two best dot products lie closer than 0.05 (where fp32 accumulation may
    order them differently from fp64) are checked to hold one of the two
    candidate rows; the others must match the oracle."""
    print(f"case: scale {scale:g}", flush=True)
    w = W.random_case(811, R=2, Mq=1, H=128, P=16, NB=8, K=3)
    w.scale = float(np.float32(scale))
    t = G.upload(w)
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale)
    for rt in (64, 128):
        for ns in (0, 3):
            out, lse = G.run_partial(t, w.scale, n_splits=ns, row_tile=rt)
            assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
            clear_rows = 0
            for r in range(2):
                d, vals = _scores_and_values(w, r)
                d = d[0] * np.sign(w.scale)  # [H, T], larger is heavier
                order = np.argsort(d, axis=1)
                best, second = order[:, -1], order[:, -2]
                gap = d[np.arange(128), best] - d[np.arange(128), second]
                clear = gap >= 0.05
                rel = G.row_errors(out[r, 0][clear], ref_o[r, 0][clear])
                assert rel.max() <= G.OUT_REL_TOL, (scale, rt, ns, rel.max())
                lerr = np.abs(lse[r, 0][clear] - ref_l[r, 0][clear]) / np.abs(ref_l[r, 0][clear])
                assert lerr.max() <= 1e-5, (scale, rt, ns, lerr.max())
                for h in np.nonzero(~clear)[0]:
                    e = min(G.row_errors(out[r, 0, h][None], vals[best[h]][None]).max(),
                            G.row_errors(out[r, 0, h][None], vals[second[h]][None]).max())
                    assert e <= G.OUT_REL_TOL, (scale, rt, ns, h, e)
                clear_rows += int(clear.sum())
            assert clear_rows >= 0.9 * 2 * 128, clear_rows


def _zero_latent_scales(w8, shared):
    """fp8 workload with some selected blocks' scales set to 0 (shared: the
    whole entry; separate: the latent part of two blocks, the RoPE part of
    one, a latent scale of 1e-30 under a RoPE scale of 1 in another)."""
    cs = w8.ckv_scale.copy()
    ks = cs if shared else w8.kpe_scale.copy()
    sel = w8.sel if w8.sel.ndim == 2 else w8.sel[:, 0]
    picked = []
    for r in range(sel.shape[0]):
        for s in sel[r]:
            if s >= 0:
                b = int(w8.table[r, s // 64 if w8.tokens else s])
                if b not in picked:
                    picked.append(b)
    assert len(picked) >= 4, picked
    if shared:
        cs[picked[0]] = 0.0
        cs[picked[1]] = 0.0
    else:
        cs[picked[0]] = 0.0
        cs[picked[1]] = 0.0
        ks[picked[2]] = 0.0
        cs[picked[3]] = 1e-30
        ks[picked[3]] = 1.0
    w8.ckv_scale, w8.kpe_scale = cs, ks
    return w8


@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("path", ["blocks", "per-row", "tokens"])
def test_fp8_zero_latent_scale(path, shared):
    print(f"case: fp8 zero scales path={path} shared={shared}", flush=True)
    kw = dict(R=2, Mq=2, H=64, P=24, NB=10, K=6, sigma=0.6)
    if path == "per-row":
        w = W.random_case(821, per_row=True, shared_frac=0.6, **kw)
    elif path == "tokens":
        w = W.random_case(822, tokens=True, **{**kw, "K": 200})
    else:
        w = W.random_case(823, **kw)
    w8 = _zero_latent_scales(w.to_fp8(shared), shared)
    t = G.upload(w8)
    ref_o, ref_l = oracle.partial(w8.q_lat, w8.q_pe, w8.ckv, w8.kpe, w8.table, w8.sel, w8.scale,
                                  w8.ckv_scale, w8.kpe_scale, tokens=w8.tokens)
    for rt in (64, 128):
        for ns in (0, 2):
            out, lse = G.run_partial(t, w8.scale, n_splits=ns, row_tile=rt, tokens=w8.tokens)
            G.assert_parity(out, lse, ref_o, ref_l, f"fp8 zero scales {path} rt={rt} splits={ns}")


def _call(tt, w, out, lse, n_splits):
    mla.sparse_partial_attn(tt["q_lat"], tt["q_pe"], tt["ckv"], tt["kpe"], tt["table"], tt["sel"],
                            w.scale, out, lse, n_splits=n_splits)


def test_graph_replay_after_workspace_grows():
    """A graph captured while the stream's workspace was small replays
    correctly after a larger eager call on the same stream has replaced that
    workspace (the old buffer is kept, not freed)."""
    print("case: replay after workspace growth", flush=True)
    dev = G.device()
    ws = W.random_case(831, R=2, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    wb = W.random_case(832, R=12, Mq=1, H=128, P=60, NB=30, K=24, sigma=0.5)
    ts, tb = G.upload(ws), G.upload(wb)
    o_s = torch.empty((2, 1, 128, 512), dtype=torch.float32, device=dev)
    l_s = torch.empty((2, 1, 128), dtype=torch.float32, device=dev)
    o_b = torch.empty((12, 1, 128, 512), dtype=torch.float32, device=dev)
    l_b = torch.empty((12, 1, 128), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        _call(ts, ws, o_s, l_s, 3)  # sizes this stream's workspace for the small call
        stream.synchronize()
        ref_s = (o_s.clone(), l_s.clone())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            _call(ts, ws, o_s, l_s, 3)
        _call(tb, wb, o_b, l_b, 6)  # needs a larger workspace: a new buffer
        stream.synchronize()
        ref_b = (o_b.clone(), l_b.clone())
        for rep in range(3):
            o_s.fill_(float("nan"))
            l_s.fill_(float("nan"))
            stream.synchronize()
            g.replay()
            stream.synchronize()
            assert torch.equal(o_s, ref_s[0]) and torch.equal(l_s, ref_s[1]), f"replay {rep}"
            _call(tb, wb, o_b, l_b, 6)
            stream.synchronize()
            assert torch.equal(o_b, ref_b[0]) and torch.equal(l_b, ref_b[1])
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.partial(ws.q_lat, ws.q_pe, ws.ckv, ws.kpe, ws.table, ws.sel, ws.scale)
    G.assert_parity(ref_s[0].cpu().numpy().astype(np.float64),
                    ref_s[1].cpu().numpy().astype(np.float64), ref_o, ref_l, "small call")


def test_workspace_cannot_grow_during_capture():
    """On a stream whose workspace is too small, a captured split call is
    refused (nothing is allocated or enqueued); the same call made eagerly
    first can then be captured."""
    print("case: growth refused during capture", flush=True)
    dev = G.device()
    w = W.random_case(841, R=2, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    t = G.upload(w)
    out = torch.empty((2, 1, 128, 512), dtype=torch.float32, device=dev)
    lse = torch.empty((2, 1, 128), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()  # a new stream: no workspace yet
    with torch.cuda.stream(stream):
        g = torch.cuda.CUDAGraph()
        with pytest.raises(mla.MlaError) as e:
            with torch.cuda.graph(g, stream=stream):
                _call(t, w, out, lse, 3)
        assert e.value.status == mla.MLA_ERR_UNSUPPORTED and "capture" in str(e.value)
        _call(t, w, out, lse, 3)
        stream.synchronize()
        ref = (out.clone(), lse.clone())
        g2 = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g2, stream=stream):
            _call(t, w, out, lse, 3)
        out.zero_()
        stream.synchronize()
        g2.replay()
        stream.synchronize()
        assert torch.equal(out, ref[0]) and torch.equal(lse, ref[1])
    torch.cuda.synchronize()
