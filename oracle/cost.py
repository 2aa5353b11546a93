"""Cost model of the three redistribution primitives, written out from the
paper.  TEST INFRASTRUCTURE ONLY: the tests compare the library's
`mla_primitive_costs` against these formulas; nothing in the product path
imports this module.

Units: microseconds, GB/s (1e9 bytes per second), bytes.  A transfer of n
bytes at W GB/s takes n / (W * 1e3) microseconds.
"""
import math

ROUTE, FETCH, LOCAL = 0, 1, 2


def query_row_bytes(d_qk=576, elt=2):
    """q: one absorbed query row of d_qk elements (Section 3.2 wire format)."""
    return d_qk * elt


def partial_row_bytes(d_v=512, elt=2, n_stats=2, stat_bytes=4):
    """p: one output row of d_v elements plus the max logit and the softmax
    denominator (Section 3.2 wire format)."""
    return d_v * elt + n_stats * stat_bytes


def t_route(probe_us, bw_gbs, mq, q, p, compute_us=0.0, merge_us=0.0):
    """Q-routing (Section 4.2): T_probe(F) + Mq (q + p) / BW(F) + T_compute
    + T_merge."""
    return probe_us + mq * (q + p) / (bw_gbs * 1e3) + compute_us + merge_us


def t_fetch(pull_bw_gbs, layers, chunk_tokens, kv_bytes, splice_us):
    """FETCH (Section 4.2): T_pull + T_splice, the pull moving the whole
    chunk, c_t b_KV bytes per layer, for every layer (Section 5.1's
    all-layer pull)."""
    return layers * chunk_tokens * kv_bytes / (pull_bw_gbs * 1e3) + splice_us


def t_local(chunk_tokens, layers, prefill_us):
    """LOCAL (Section 5.1): a fresh prefill of the chunk, c_t L c."""
    return chunk_tokens * layers * prefill_us


def choose(route_us, fetch_us, local_us):
    """The predicate (Section 5.1): the argmin over the three; ties go to
    ROUTE, then FETCH."""
    best, who = route_us, ROUTE
    if fetch_us < best:
        best, who = fetch_us, FETCH
    if local_us < best:
        who = LOCAL
    return who


def wire_crossover_mq(chunk_tokens, kv_bytes, q, p):
    """Section 5.2: on wire bytes routing and pulling one layer of the chunk
    break even at Mq = c_t b_KV / (q + p)."""
    return chunk_tokens * kv_bytes / (q + p) if q + p > 0 else math.inf


def wire_saving(mq, chunk_tokens, kv_bytes, q, p):
    """The share of one layer's pull bytes that routing Mq rows does not move."""
    return 1.0 - mq * (q + p) / (chunk_tokens * kv_bytes)


def congestion_bw_gbs(mq, q, p, splice_us):
    """Section 8 (congestion): routing loses to FETCH's splice only once its
    effective throughput falls below Mq (q + p) / T_splice."""
    return mq * (q + p) / (splice_us * 1e3) if splice_us > 0 else math.inf


def splice_crossover_tokens(splice_us, layers, prefill_us):
    """Section 5.1: the flat splice undercuts re-prefill above
    c_t = T_splice / (L c)."""
    return splice_us / (layers * prefill_us) if prefill_us > 0 else math.inf


def costs(model, case):
    """All of the above for one case (dicts with the field names of the
    library's mla_cost_model_t and mla_cost_case_t)."""
    m, c = model, case
    q, p = c["q_bytes"], c["p_bytes"]
    r = t_route(m["probe_us"], m["route_bw_gbs"], c["mq"], q, p, m["compute_us"], m["merge_us"])
    f = t_fetch(m["pull_bw_gbs"], m["layers"], c["chunk_tokens"], c["kv_bytes"], m["splice_us"])
    lo = t_local(c["chunk_tokens"], m["layers"], m["prefill_us"])
    return dict(route_us=r, fetch_us=f, local_us=lo, choice=choose(r, f, lo),
                wire_crossover_mq=wire_crossover_mq(c["chunk_tokens"], c["kv_bytes"], q, p),
                wire_saving=wire_saving(c["mq"], c["chunk_tokens"], c["kv_bytes"], q, p),
                congestion_bw_gbs=congestion_bw_gbs(c["mq"], q, p, m["splice_us"]),
                splice_crossover_tokens=splice_crossover_tokens(m["splice_us"], m["layers"],
                                                                m["prefill_us"]))
