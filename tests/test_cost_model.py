"""The closed-form ROUTE / FETCH / LOCAL cost model.

The oracle (oracle/cost.py, the formulas written out from Sections 3.2,
4.2, 5.1, 5.2 and 8) is pinned to the numbers the paper prints; the
library's host-side `mla_primitive_costs` is then compared with the oracle
on random cases.  CPU only: the model is host arithmetic and needs no GPU.
"""
import math

import numpy as np
import pytest

from oracle import cost as C

Q, P = 1152, 1032          # Section 3.2: 576 x 2 and 512 x 2 + 2 x 4
PAPER = dict(probe_us=16.0, route_bw_gbs=25.0, compute_us=0.0, merge_us=0.0, pull_bw_gbs=25.0,
             splice_us=3000.0, prefill_us=1.0, layers=27)


# ------------------------------------------------------------ oracle pins
def test_wire_payload_sizes():
    """q = 1152 B and p = 1032 B per row, q + p = 2184 B (Section 3.2)."""
    assert C.query_row_bytes() == 1152
    assert C.partial_row_bytes() == 1032
    assert C.query_row_bytes() + C.partial_row_bytes() == 2184


def test_chunk_bytes():
    """A 2048-token chunk is 2.36 MB per layer and ~64 MB over 27 layers
    (Figure 2a); the routed row is ~1000x smaller."""
    one = 2048 * 1152
    assert round(one / 1e6, 2) == 2.36
    assert round(27 * one / 1e6, 1) == 63.7
    assert 900 < one / (Q + P) < 1100


def test_wire_crossover():
    """Section 5.2 / 5.4: the wire-byte break-even is ~1080 rows at c_t =
    2048 and ~270 at c_t = 512."""
    assert round(C.wire_crossover_mq(2048, 1152, Q, P), 1) == 1080.3
    assert round(C.wire_crossover_mq(512, 1152, Q, P), 1) == 270.1


def test_wire_saving_at_256_rows():
    """Section 5.2: at c_t = 2048 routing moves >= 76 % fewer bytes for
    Mq <= 256 (76 % at 256, more for smaller batches)."""
    assert round(100 * C.wire_saving(256, 2048, 1152, Q, P), 1) == 76.3
    assert all(C.wire_saving(m, 2048, 1152, Q, P) > 0.76 for m in (1, 16, 64, 255))
    assert C.wire_saving(1081, 2048, 1152, Q, P) < 0 < C.wire_saving(1080, 2048, 1152, Q, P)


def test_route_round_trip_fit():
    """Section 4.3's table: the model T_probe + Mq (q + p) / BW, with each
    row's measured probe and throughput, undershoots the measured full round
    trip at Mq = 1024 by the fixed ~9 us kernel turnaround the paper names,
    for every payload; at the real payload the model gives 105.5 us."""
    rows = [(900, 16.2, 62.8, 24.6), (2184, 15.9, 115.8, 24.7), (4368, 16.6, 207.7, 24.7),
            (8736, 16.1, 389.1, 24.7)]
    for payload, sig, full, bw in rows:
        model = C.t_route(sig, bw, 1024, payload, 0)
        assert 8.0 < full - model < 12.0, (payload, model, full)
    assert round(C.t_route(16.0, 25.0, 1024, Q, P), 1) == 105.5
    # the fit quality the paper quotes for the amortised regime (about 7 %
    # mean absolute percentage error at Mq >= 512)
    errs = [abs(full - C.t_route(sig, bw, 1024, pl, 0)) / full for pl, sig, full, bw in rows[1:]]
    assert np.mean(errs) < 0.07


def test_all_layer_pull_and_splice():
    """Section 5.1: FETCH is a ~2.5 ms all-layer pull of a 2 K-token chunk
    plus the ~3 ms splice."""
    pull = C.t_fetch(25.0, 27, 2048, 1152, 0.0)
    assert 2400 < pull < 2600
    assert round(C.t_fetch(25.0, 27, 2048, 1152, 3000.0) - pull) == 3000


def test_congestion_floor():
    """Section 8: routing loses to FETCH only below Mq (q + p) / T_splice,
    about 0.2 GB/s at Mq = 256, a ~125x degradation from 25 GB/s."""
    bw = C.congestion_bw_gbs(256, Q, P, 3000.0)
    assert round(bw, 3) == 0.186
    assert 120 < 25.0 / bw < 140


def test_splice_vs_reprefill_crossover():
    """Section 5.1: the flat splice undercuts re-prefill above c_t ~ 75-220
    tokens for c between 1.5 and 0.5 us per token and layer."""
    assert math.floor(C.splice_crossover_tokens(3000.0, 27, 1.5)) == 74
    assert math.floor(C.splice_crossover_tokens(3000.0, 27, 0.5)) == 222


def test_predicate_shape():
    """Section 5.1: ROUTE undercuts both others across chunk sizes at decode
    batches; it cedes only where Mq exceeds the chunk by a wide margin, and
    LOCAL wins for very small chunks against FETCH."""
    m = dict(PAPER)
    for ct in (64, 256, 2048, 16384, 65536):
        for mq in (1, 16, 256):
            r = C.costs(m, dict(mq=mq, chunk_tokens=ct, q_bytes=Q, p_bytes=P, kv_bytes=1152))
            assert r["choice"] == C.ROUTE, (ct, mq, r)
    # a huge query batch over a tiny chunk: re-prefill is cheaper than routing
    r = C.costs(m, dict(mq=200000, chunk_tokens=64, q_bytes=Q, p_bytes=P, kv_bytes=1152))
    assert r["choice"] == C.LOCAL
    # without routing, small chunks re-prefill and large ones fetch
    assert C.t_local(64, 27, 1.0) < C.t_fetch(25.0, 27, 64, 1152, 3000.0)
    assert C.t_local(4096, 27, 1.0) > C.t_fetch(25.0, 27, 4096, 1152, 3000.0)


# ------------------------------------------------------------ library vs oracle
def _lib_costs(model, case):
    from paper_2606_01502_amd import mla
    return mla.primitive_costs(case["mq"], case["chunk_tokens"], case["q_bytes"],
                               case["p_bytes"], case["kv_bytes"], **model)


def test_library_matches_oracle_on_random_cases():
    rng = np.random.default_rng(5)
    for _ in range(300):
        model = dict(probe_us=float(rng.uniform(0, 50)), route_bw_gbs=float(rng.uniform(0.1, 400)),
                     compute_us=float(rng.choice([0.0, rng.uniform(0, 60)])),
                     merge_us=float(rng.choice([0.0, rng.uniform(0, 25)])),
                     pull_bw_gbs=float(rng.uniform(0.1, 400)),
                     splice_us=float(rng.choice([0.0, rng.uniform(0, 5000)])),
                     prefill_us=float(rng.choice([0.0, rng.uniform(0.1, 2)])),
                     layers=int(rng.integers(1, 128)))
        case = dict(mq=int(rng.integers(0, 1 << 20)), chunk_tokens=int(rng.integers(1, 1 << 20)),
                    q_bytes=int(rng.integers(0, 9000)), p_bytes=int(rng.integers(0, 9000)),
                    kv_bytes=int(rng.integers(1, 9000)))
        got = _lib_costs(model, case)
        ref = C.costs(model, case)
        assert got["choice"] == ("route", "fetch", "local")[ref["choice"]], (model, case)
        for k in ("route_us", "fetch_us", "local_us", "wire_crossover_mq", "wire_saving",
                  "congestion_bw_gbs", "splice_crossover_tokens"):
            a, b = got[k], ref[k]
            assert (a == b) or abs(a - b) <= 1e-12 * max(abs(a), abs(b)), (k, a, b)


def test_library_paper_case():
    r = _lib_costs(PAPER, dict(mq=1024, chunk_tokens=2048, q_bytes=Q, p_bytes=P, kv_bytes=1152))
    assert round(r["route_us"], 1) == 105.5 and r["choice"] == "route"
    assert round(r["wire_crossover_mq"], 1) == 1080.3


@pytest.mark.parametrize("bad", [dict(route_bw_gbs=0.0), dict(pull_bw_gbs=-1.0),
                                 dict(probe_us=-1.0), dict(splice_us=math.inf),
                                 dict(layers=0), dict(prefill_us=math.nan)])
def test_library_rejects_bad_models(bad):
    from paper_2606_01502_amd import mla
    with pytest.raises(mla.MlaError) as e:
        mla.primitive_costs(16, 2048, **bad)
    assert e.value.status == mla.MLA_ERR_INVALID_ARGUMENT


def test_library_rejects_bad_cases():
    from paper_2606_01502_amd import mla
    for args in [(-1, 2048), (16, 0), (16, 2048, -1), (16, 2048, 1152, 1032, 0)]:
        with pytest.raises(mla.MlaError):
            mla.primitive_costs(*args)
