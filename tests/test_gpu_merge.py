"""mla_merge_partials against the oracle merge, and the route-and-merge
property end to end on the GPU: partials over disjoint parts of a selection,
merged, equal attention over the whole selection (Section 3.3)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _random_parts(seed, n, shape, dead_frac=0.2, nan_dead=True):
    """n partials of `shape` rows: o ~ N(0,1), lse ~ N(0, 4); a fraction of
    (part, row) pairs is dead (lse = -inf, o = NaN), and some rows are dead in
    every part."""
    rng = np.random.default_rng([seed, 91])
    o = rng.standard_normal((n,) + shape + (512,)).astype(np.float32)
    lam = (rng.standard_normal((n,) + shape) * 4.0).astype(np.float32)
    dead = rng.random((n,) + shape) < dead_frac
    flat = dead.reshape(n, -1)
    flat[:, ::7] = True  # every 7th row: no live part at all
    lam[dead] = -np.inf
    if nan_dead:
        o[dead] = np.nan
    return o, lam


def _gpu_merge(o, lam, strided=False):
    dev = G.device()
    n = o.shape[0]
    if strided:
        # parts as slices of one larger buffer, like jobs laid out part-major
        big_o = torch.from_numpy(np.concatenate([o, o[:1]], axis=0)).to(dev)
        big_l = torch.from_numpy(np.concatenate([lam, lam[:1]], axis=0)).to(dev)
        parts_o = [big_o[j] for j in range(n)]
        parts_l = [big_l[j] for j in range(n)]
    else:
        parts_o = [torch.from_numpy(o[j]).to(dev) for j in range(n)]
        parts_l = [torch.from_numpy(lam[j]).to(dev) for j in range(n)]
    out, lse = mla.merge_partials(parts_o, parts_l, out_lse=True)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("n", [1, 2, 4, 7, 64])
def test_merge_random_parts(n):
    print(f"case: merge n={n}", flush=True)
    o, lam = _random_parts(300 + n, n, (6, 2, 16))
    out, lse = _gpu_merge(o, lam)
    ref_o, ref_l = oracle.merge(o.astype(np.float64), lam.astype(np.float64))
    G.assert_parity(out, lse, ref_o, ref_l, f"merge n={n}")


def test_merge_strided_parts_and_large_rows():
    print("case: merge strided", flush=True)
    o, lam = _random_parts(310, 4, (64, 1, 128), dead_frac=0.05)
    out, lse = _gpu_merge(o, lam, strided=True)
    ref_o, ref_l = oracle.merge(o.astype(np.float64), lam.astype(np.float64))
    G.assert_parity(out, lse, ref_o, ref_l, "merge strided")


def test_merge_extreme_lse_spread():
    """Parts whose lse differ by hundreds: the small ones must vanish without
    overflow or NaN."""
    print("case: merge spread", flush=True)
    o, lam = _random_parts(311, 5, (3, 1, 16), dead_frac=0.0, nan_dead=False)
    lam[0] += 300.0
    lam[3] -= 300.0
    out, lse = _gpu_merge(o, lam)
    ref_o, ref_l = oracle.merge(o.astype(np.float64), lam.astype(np.float64))
    G.assert_parity(out, lse, ref_o, ref_l, "merge spread")


@pytest.mark.parametrize("m", [2, 3, 8])
def test_route_and_merge_equals_whole_selection(m):
    """Split each job's selected blocks over m holders (disjoint, scattered,
    some holders empty), run the partial per holder on the GPU, merge on the
    GPU: the result matches the oracle over the whole selection."""
    print(f"case: route+merge m={m}", flush=True)
    w = W.random_case(320 + m, R=3, Mq=2, H=64, P=40, NB=24, K=16, sigma=0.5)
    t = G.upload(w)
    rng = np.random.default_rng([320 + m, 5])
    owner = rng.integers(0, m, size=w.sel.shape)
    parts_o, parts_l = [], []
    for j in range(m):
        sel_j = np.where(owner == j, w.sel, -1).astype(np.int32)
        o, l = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       torch.from_numpy(sel_j).to(G.device()), w.scale)
        parts_o.append(o)
        parts_l.append(l)
    out, lse = mla.merge_partials(parts_o, parts_l, out_lse=True)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale)
    G.assert_parity(out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64),
                    ref_o, ref_l, f"route+merge m={m}")


def test_batched_merge_config_sampled():
    """The batched workload at full size: 256 partials on the GPU, merged into
    64 requests; the oracle checks eight requests end to end."""
    print("case: batched-merge sampled", flush=True)
    w = W.make("batched-merge")
    t = G.upload(w)
    out, lse = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       t["sel"], w.scale)
    n, parts = w.n_requests, w.merge_parts
    merged, mlse = mla.merge_partials([out[j * n:(j + 1) * n] for j in range(parts)],
                                      [lse[j * n:(j + 1) * n] for j in range(parts)], out_lse=True)
    torch.cuda.synchronize()
    reqs = np.array([0, 9, 21, 33, 40, 51, 62, 63])
    jobs = np.concatenate([j * n + reqs for j in range(parts)])
    po, pl = oracle.partial(w.q_lat[jobs], w.q_pe[jobs], w.ckv, w.kpe, w.table[jobs],
                            w.sel[jobs], w.scale)
    k = reqs.size
    ref_o, ref_l = oracle.merge(po.reshape(parts, k, *po.shape[1:]),
                                pl.reshape(parts, k, *pl.shape[1:]))
    G.assert_parity(out.cpu().numpy()[jobs].astype(np.float64),
                    lse.cpu().numpy()[jobs].astype(np.float64), po, pl, "batched partials")
    G.assert_parity(merged.cpu().numpy()[reqs].astype(np.float64),
                    mlse.cpu().numpy()[reqs].astype(np.float64), ref_o, ref_l, "batched merge")
