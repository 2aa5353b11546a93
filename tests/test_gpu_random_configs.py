"""Randomised configurations against the oracle: every combination of cache
type (bf16, fp8 with one or two scale arrays) and selection mode (blocks,
tokens, per-row blocks), with random job counts, rows, heads, slot counts,
padding, duplicates, split counts and row tiles, and every fourth draw again
with the wire-form output.  The draws are seeded, so each case is
reproducible from its index."""
import numpy as np
import pytest

import oracle
from paper_2606_01502_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

N_CASES = 72


def _draw(i):
    rng = np.random.default_rng([424242, i])
    cache = ("bf16", "fp8", "fp8s")[i % 3]
    mode = ("blocks", "tokens", "per_row")[(i // 3) % 3]
    R = int(rng.integers(1, 4))
    H = int(rng.choice([1, 7, 16, 31, 64, 128]))
    Mq = int(rng.integers(1, 4 if mode != "per_row" else 9))
    NB = int(rng.integers(2, 24))
    P = NB + int(rng.integers(0, 10))
    if mode == "tokens":
        K = int(rng.integers(1, 400))
    else:
        K = int(rng.integers(1, 3 * NB))
    n_valid = [int(rng.integers(0, K + 1)) for _ in range(R)]
    if mode == "per_row":
        n_valid = [[int(rng.integers(0, K + 1)) for _ in range(Mq)] for _ in range(R)]
    kw = dict(R=R, Mq=Mq, H=H, P=P, NB=NB, K=K, n_valid=n_valid,
              sigma=float(rng.uniform(0.3, 1.5)), allow_dup=bool(rng.integers(0, 2)),
              pad_pattern=str(rng.choice(["tail", "interleaved"])), tokens=mode == "tokens",
              per_row=mode == "per_row", shared_frac=float(rng.uniform(0, 1)))
    if not kw["allow_dup"]:
        cap = NB * 64 if mode == "tokens" else NB
        kw["K"] = min(K, cap)
        kw["n_valid"] = (np.minimum(np.asarray(n_valid), min(K, cap))).tolist()
    n_splits = int(rng.choice([0, 0, 1, 2, 3, 7]))
    rows = Mq * H
    row_tile = int(rng.choice([0, 64, 128])) if not (mode == "per_row" and H == 1) else 64
    return cache, mode, kw, n_splits, row_tile


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_config(i):
    cache, mode, kw, n_splits, row_tile = _draw(i)
    print(f"case {i}: {cache} {mode} {kw} splits={n_splits} row_tile={row_tile}", flush=True)
    w = W.random_case(9000 + i, **kw)
    if cache != "bf16":
        w = w.to_fp8(shared_scale=cache == "fp8")
    out, lse = G.run_partial(G.upload(w), w.scale, n_splits=n_splits, row_tile=row_tile,
                             tokens=w.tokens)
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                  w.ckv_scale, w.kpe_scale, tokens=w.tokens)
    G.assert_parity(out, lse, ref_o, ref_l, f"random case {i}")


@pytest.mark.parametrize("i", range(0, N_CASES, 4))
def test_random_config_wire(i):
    """The same draws with the output in Section 3.2's wire form: bf16 rows
    bit-exact against the fp32 form rounded, (m, l) against the oracle."""
    from tests.test_gpu_wire import _check_wire
    cache, mode, kw, n_splits, row_tile = _draw(i)
    print(f"case {i} wire: {cache} {mode} {kw} splits={n_splits} row_tile={row_tile}", flush=True)
    w = W.random_case(9000 + i, **kw)
    if cache != "bf16":
        w = w.to_fp8(shared_scale=cache == "fp8")
    _check_wire(w, n_splits, row_tile=row_tile, what=f"random case {i} wire")
