"""Pools larger than 4 GiB: the selected blocks sit past the 4 GiB byte
offset, so every pool address on the path needs 64-bit arithmetic (block,
token and scale indexing of the partial kernel in all its selection modes,
and the FETCH copies).  The values are those of a small random case, placed
into a large zero-filled device pool; the oracle runs on the small case."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fetch as F
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

GIB4 = 4 << 30


def _big_pools(w, p_big, at):
    """Device pools of p_big blocks holding w's pool blocks at indices `at`."""
    dev = G.device()
    fp8 = w.fp8
    dt = torch.uint8 if fp8 else torch.bfloat16
    ckv = torch.zeros((p_big, 64, 512), dtype=dt, device=dev)
    kpe = torch.zeros((p_big, 64, 64), dtype=dt, device=dev)
    idx = torch.from_numpy(at.astype(np.int64)).to(dev)
    small = G.upload(w)
    ckv[idx] = small["ckv"]
    kpe[idx] = small["kpe"]
    assert int(at.min()) * ckv[0].numel() * ckv.element_size() > GIB4
    scales = None
    if fp8:
        cs = torch.ones(p_big, dtype=torch.float32, device=dev)
        ks = torch.ones(p_big, dtype=torch.float32, device=dev)
        cs[idx] = small["ckv_scale"]
        ks[idx] = small["kpe_scale"]
        scales = (cs, ks if small["kpe_scale"] is not small["ckv_scale"] else cs)
    return small, ckv, kpe, scales


@pytest.mark.parametrize("mode", ["blocks", "tokens", "per_row", "fp8_blocks", "fp8_tokens"])
def test_partial_with_pool_past_4gib(mode):
    print(f"case: pool past 4 GiB, {mode}", flush=True)
    tokens = "tokens" in mode
    kw = dict(R=2, Mq=2 if mode == "per_row" else 1, H=64, P=10, NB=8,
              K=200 if tokens else 6, sigma=0.7, tokens=tokens, per_row=mode == "per_row")
    w = W.random_case(880, **kw)
    if mode.startswith("fp8"):
        w = w.to_fp8(shared_scale=False)
    elt = 1 if w.fp8 else 2
    p_big = (GIB4 // (64 * 512 * elt)) + 64
    at = np.arange(p_big - 10, p_big)  # the small pool's blocks, last in the big one
    small, ckv, kpe, scales = _big_pools(w, p_big, at)
    table = torch.from_numpy(at[w.table].astype(np.int32)).to(G.device())
    out, lse = mla.sparse_partial_attn(small["q_lat"], small["q_pe"], ckv, kpe, table,
                                       small["sel"], w.scale,
                                       ckv_scale=scales[0] if scales else None,
                                       kpe_scale=scales[1] if scales else None, tokens=tokens)
    torch.cuda.synchronize()
    del ckv, kpe, scales
    torch.cuda.empty_cache()
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                  w.ckv_scale, w.kpe_scale, tokens=tokens)
    G.assert_parity(out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64),
                    ref_o, ref_l, f"pool past 4 GiB ({mode})")


def test_fetch_with_pool_past_4gib():
    """Gather from, and splice into, blocks past the 4 GiB offset of a
    one-layer pool; the rest of the pool stays zero."""
    print("case: fetch past 4 GiB", flush=True)
    dev = G.device()
    p_big = GIB4 // (64 * 512 * 2) + 64
    at = np.arange(p_big - 6, p_big)
    rng = np.random.default_rng(881)
    small_c = W.normal_bf16(881, 3, (1, 6, 64, 512), 1.0)
    small_k = W.normal_bf16(881, 4, (1, 6, 64, 64), 1.0)

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    ckv = torch.zeros((1, p_big, 64, 512), dtype=torch.bfloat16, device=dev)
    kpe = torch.zeros((1, p_big, 64, 64), dtype=torch.bfloat16, device=dev)
    idx = torch.from_numpy(at).to(dev)
    ckv[0, idx] = bf16(small_c)[0]
    kpe[0, idx] = bf16(small_k)[0]
    table_small = rng.permutation(6).astype(np.int32)
    sel = rng.integers(0, 6 * 64, 300).astype(np.int32)
    table = torch.from_numpy(at[table_small].astype(np.int32)).to(dev)
    oc, ok = mla.fetch_gather(ckv, kpe, table, torch.from_numpy(sel).to(dev))
    torch.cuda.synchronize()
    rc, rk = F.gather(small_c, small_k, table_small, sel)
    assert np.array_equal(oc.view(torch.int16).cpu().numpy().view(np.uint16), rc)
    assert np.array_equal(ok.view(torch.int16).cpu().numpy().view(np.uint16), rk)
    # splice a 200-token chunk into the same high blocks, delta 0 (bit-exact)
    chunk_c = W.normal_bf16(882, 5, (1, 200, 512), 1.0)
    chunk_k = W.normal_bf16(882, 6, (1, 200, 64), 1.0)
    mla.fetch_splice(bf16(chunk_c), bf16(chunk_k), ckv, kpe, table, 50, 0)
    torch.cuda.synchronize()
    got_c = ckv[0, idx].view(torch.int16).cpu().numpy().view(np.uint16)[None]
    got_k = kpe[0, idx].view(torch.int16).cpu().numpy().view(np.uint16)[None]
    ref_c, ref_k = F.splice(chunk_c, chunk_k, small_c, small_k, table_small, 50, 0, 10000.0, 0)
    assert np.array_equal(got_c, ref_c) and np.array_equal(got_k, ref_k)
    assert float(ckv[0, :p_big - 6].float().abs().max()) == 0.0
