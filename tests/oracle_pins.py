"""Checks that pin the oracle to facts outside itself.

Each pin_* function takes an oracle library handle (the normal build, or a
deliberately broken copy in the mutation test) and raises AssertionError
when the oracle disagrees with:
  * brute force written independently (struct decoding, math.fsum dot
    products, mpmath exponentials, no max shift);
  * the dense special case computed by numpy/scipy library routines;
  * closed forms (identical keys, zero query, two token groups, one-hot);
  * invariants of the merge algebra (partition, commutativity,
    associativity, zero-weight identity, n = 1) stated in the paper's
    Sections 2.2 and 3.3;
  * torch's float8_e4m3fn codec and the E4M3FN format's anchor values.
"""
import math
import struct

import mpmath
import numpy as np
import scipy.special

import oracle
from paper_2606_01502_amd import workloads as W

DLAT, DPE, BLOCK = 512, 64, 64


# ------------------------------------------------------------ brute force
def _bf16_struct(bits):
    """bf16 bits -> float via struct (big-endian binary32 with a zero low half)."""
    b = int(bits)
    return struct.unpack(">f", bytes([b >> 8, b & 0xFF, 0, 0]))[0]


def _e4m3_anchor_table():
    """E4M3FN positive values listed binade by binade from the format's
    description: 8 subnormals k/8 * 2^-6, then for each exponent -6..8 the
    eight values (1 + k/8) * 2^e; the last one of exponent 8 is NaN."""
    vals = [mpmath.mpf(k) / 8 * mpmath.mpf(2) ** -6 for k in range(8)]
    for e in range(-6, 9):
        for k in range(8):
            vals.append((1 + mpmath.mpf(k) / 8) * mpmath.mpf(2) ** e)
    vals[-1] = None
    return vals


_E4M3 = _e4m3_anchor_table()


def _kv_value(w, which, b, t, d):
    if which == "ckv":
        arr, sc = w.ckv, w.ckv_scale
    else:
        arr, sc = w.kpe, w.kpe_scale
    if not w.fp8:
        return _bf16_struct(arr[b, t, d])
    c = int(arr[b, t, d])
    v = _E4M3[c & 0x7F]
    v = float(v) * float(sc[b])
    return -v if c & 0x80 else v


def brute_force(w, rows=None, stats=None):
    """Partial attention by the definition, without the max shift.
    Returns {(r, i, h): (out list, lse float)} for the requested rows; a dict
    given as stats receives {(r, i, h): (M, l)}, the largest score and
    sum exp(s - M) (Section 3.2's wire statistics), from the same scores."""
    R, Mq, H, _ = w.q_lat.shape
    mpmath.mp.dps = 40
    res = {}
    rows = rows or [(r, i, h) for r in range(R) for i in range(Mq) for h in range(H)]
    cache_v = {}
    for (r, i, h) in rows:
        toks = []
        for s in (w.sel[r, i] if w.sel.ndim == 3 else w.sel[r]):
            if s < 0:
                continue
            if w.tokens:  # one logical token: token s % 64 of logical block s // 64
                toks.append((int(w.table[r, s // BLOCK]), int(s % BLOCK)))
                continue
            b = int(w.table[r, s])
            toks.extend((b, t) for t in range(BLOCK))
        if not toks:
            res[(r, i, h)] = ([0.0] * DLAT, -math.inf)
            if stats is not None:
                stats[(r, i, h)] = (-math.inf, 0.0)
            continue
        ql = [_bf16_struct(x) for x in w.q_lat[r, i, h]]
        qp = [_bf16_struct(x) for x in w.q_pe[r, i, h]]
        weights = []
        scores = []
        for (b, t) in toks:
            key = (b, t)
            if key not in cache_v:
                cache_v[key] = ([_kv_value(w, "ckv", b, t, d) for d in range(DLAT)],
                                [_kv_value(w, "kpe", b, t, d) for d in range(DPE)])
            kv, kp = cache_v[key]
            dot = math.fsum([a * c for a, c in zip(ql, kv)] + [a * c for a, c in zip(qp, kp)])
            scores.append(mpmath.mpf(w.scale) * mpmath.mpf(dot))
            weights.append(mpmath.exp(scores[-1]))
        z = mpmath.fsum(weights)
        if stats is not None:
            m = max(scores)
            stats[(r, i, h)] = (float(m), float(mpmath.fsum(mpmath.exp(x - m) for x in scores)))
        lse = float(mpmath.log(z))
        pw = [float(x / z) for x in weights]
        out = [math.fsum(pw[k] * cache_v[toks[k]][0][d] for k in range(len(toks)))
               for d in range(DLAT)]
        res[(r, i, h)] = (out, lse)
    return res


def rel_err(a, b):
    """Row-normwise relative error max|a-b| / max|b| (floor 1e-300)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _check_rows(out, lse, ref, tol_out, tol_lse):
    for (r, i, h), (o_ref, l_ref) in ref.items():
        if l_ref == -math.inf:
            assert lse[r, i, h] == -math.inf, (r, i, h)
            assert np.all(out[r, i, h] == 0.0)
            continue
        assert abs(lse[r, i, h] - l_ref) <= tol_lse, (r, i, h, lse[r, i, h], l_ref)
        assert rel_err(out[r, i, h], o_ref) <= tol_out, (r, i, h, rel_err(out[r, i, h], o_ref))


def pin_bruteforce_tiny(lib):
    w = W.tiny()
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_multi(lib):
    """Several jobs, Mq > 1, duplicate ids, interleaved empty slots, and a
    job with nothing selected."""
    w = W.random_case(11, R=3, Mq=2, H=2, P=7, NB=5, K=4, n_valid=[3, 0, 4],
                      allow_dup=True, pad_pattern="interleaved")
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_fp8(lib):
    """Both scale layouts: one scale per block for the whole entry, and
    separate latent and RoPE scales (which tells the two scales apart)."""
    base = W.random_case(12, R=2, Mq=1, H=3, P=5, NB=5, K=3, sigma=0.7)
    for shared in (True, False):
        w = base.to_fp8(shared_scale=shared)
        if not shared:
            assert not np.array_equal(w.ckv_scale, w.kpe_scale)
        out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                  w.ckv_scale, w.kpe_scale, lib=lib)
        _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_per_row(lib):
    """A selection per query row (one holder serving several requesters on
    one chunk): overlapping rows, duplicates, interleaved empty slots, and a
    row with nothing selected."""
    w = W.random_case(13, R=2, Mq=3, H=2, P=9, NB=6, K=4, n_valid=[[3, 0, 4], [4, 2, 1]],
                      allow_dup=True, pad_pattern="interleaved", per_row=True)
    assert w.sel.ndim == 3 and not all(np.array_equal(w.sel[0, 0], w.sel[0, i]) for i in range(3))
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_negative_scale(lib):
    """Any finite scale is allowed: a negative one weights the lowest scores
    most.  Brute force on a case with spread scores."""
    import dataclasses
    w = dataclasses.replace(W.random_case(14, R=2, Mq=2, H=2, P=7, NB=5, K=3, sigma=1.5),
                            scale=-0.3)
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_wire_stats(lib):
    """The largest score M and the denominator l of every row (the two
    statistics Section 3.2 ships with the bf16 partial) against brute force,
    over block, fp8, per-row and token selections with empty rows."""
    cases = [W.tiny(),
             W.random_case(31, R=2, Mq=2, H=3, P=6, NB=4, K=3, n_valid=[0, 2]).to_fp8(False),
             W.random_case(32, R=1, Mq=3, H=2, P=5, NB=4, K=3, per_row=True,
                           n_valid=[[3, 0, 1]]),
             W.random_case(33, R=2, Mq=1, H=3, P=5, NB=3, K=40, tokens=True, n_valid=[40, 7])]
    for w in cases:
        st = {}
        brute_force(w, stats=st)
        out, lse, mx, den = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                           w.ckv_scale, w.kpe_scale, lib=lib, tokens=w.tokens,
                                           stats=True)
        for (r, i, h), (m_ref, l_ref) in st.items():
            if m_ref == -math.inf:
                assert mx[r, i, h] == -math.inf and den[r, i, h] == 0.0, (w.name, r, i, h)
                continue
            assert abs(mx[r, i, h] - m_ref) <= 1e-12 * max(1.0, abs(m_ref)), (w.name, r, i, h)
            assert abs(den[r, i, h] - l_ref) <= 1e-12 * l_ref and den[r, i, h] >= 1.0
            assert abs(lse[r, i, h] - (m_ref + math.log(l_ref))) <= 1e-12 * max(1.0, abs(m_ref))


def pin_per_row_is_one_job_per_row(lib):
    """Per-row selections equal the shared-selection form with every query
    row routed as a job of its own (Mq = 1) on the same chunk."""
    w = W.random_case(14, R=2, Mq=4, H=3, P=12, NB=8, K=5, allow_dup=True, per_row=True,
                      shared_frac=0.7)
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    R, Mq, H, _ = w.q_lat.shape
    q_lat = w.q_lat.reshape(R * Mq, 1, H, DLAT)
    q_pe = w.q_pe.reshape(R * Mq, 1, H, DPE)
    table = np.repeat(w.table, Mq, axis=0)
    sel = w.sel.reshape(R * Mq, -1)
    o2, l2 = oracle.partial(q_lat, q_pe, w.ckv, w.kpe, table, sel, w.scale, lib=lib)
    assert np.array_equal(out.reshape(o2.shape), o2) and np.array_equal(lse.reshape(l2.shape), l2)


def _partial(w, lib):
    return oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, w.ckv_scale,
                          w.kpe_scale, lib=lib, tokens=w.tokens)


def pin_bruteforce_tokens(lib):
    """Single-token selections (an indexer's top-k tokens): ids anywhere in
    the chunk, duplicates, interleaved empty slots, a job with nothing."""
    w = W.random_case(15, R=3, Mq=2, H=2, P=7, NB=3, K=24, n_valid=[24, 0, 9], allow_dup=True,
                      pad_pattern="interleaved", tokens=True)
    assert w.sel.max() >= 64 and (w.sel % 64 != 0).any()
    out, lse = _partial(w, lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_bruteforce_tokens_per_row(lib):
    """Token selections per query row."""
    w = W.random_case(16, R=1, Mq=3, H=2, P=6, NB=2, K=10, allow_dup=True, per_row=True,
                      tokens=True)
    out, lse = _partial(w, lib)
    _check_rows(out, lse, brute_force(w), 1e-12, 1e-12)


def pin_tokens_cover_blocks(lib):
    """Listing all 64 tokens of every selected block, in a shuffled order,
    equals selecting the blocks (the token path decodes block s // 64 and
    token s % 64)."""
    w = W.random_case(17, R=2, Mq=2, H=3, P=10, NB=6, K=3, sigma=0.7)
    out_b, lse_b = _partial(w, lib)
    rng = np.random.default_rng(17)
    tok = np.stack([rng.permutation((w.sel[r][:, None] * BLOCK + np.arange(BLOCK)).ravel())
                    for r in range(w.sel.shape[0])]).astype(np.int32)
    wt = W.Workload("tok", w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, tok, w.scale, tokens=True)
    out_t, lse_t = _partial(wt, lib)
    np.testing.assert_allclose(lse_t, lse_b, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out_t, out_b, rtol=1e-11, atol=1e-13)


def pin_single_token(lib):
    """One selected token: its value row comes back exactly and lse is its
    score; the same token twice adds ln 2 to lse."""
    w = W.random_case(18, R=1, Mq=1, H=3, P=5, NB=4, K=2)
    s_id = 2 * BLOCK + 37
    one = np.array([[s_id, -1]], np.int32)
    wt = W.Workload("one", w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, one, w.scale, tokens=True)
    out, lse = _partial(wt, lib)
    b = int(w.table[0, 2])
    ckv = W.bf16_bits_to_f32(w.ckv[b, 37]).astype(np.float64)
    kpe = W.bf16_bits_to_f32(w.kpe[b, 37]).astype(np.float64)
    for h in range(3):
        ql = W.bf16_bits_to_f32(w.q_lat[0, 0, h]).astype(np.float64)
        qp = W.bf16_bits_to_f32(w.q_pe[0, 0, h]).astype(np.float64)
        score = w.scale * math.fsum(list(ql * ckv) + list(qp * kpe))
        assert abs(lse[0, 0, h] - score) < 1e-12
        assert np.array_equal(out[0, 0, h], ckv)
    wt.sel = np.array([[s_id, s_id]], np.int32)
    out2, lse2 = _partial(wt, lib)
    np.testing.assert_allclose(lse2, lse + math.log(2), rtol=0, atol=1e-12)
    np.testing.assert_allclose(out2, out, rtol=1e-15, atol=0)


# ------------------------------------------------------------ library special case
def _dense_numpy(w, r):
    """Dense softmax attention over job r's selected tokens with numpy/scipy."""
    blocks = [int(w.table[r, s]) for s in w.sel[r] if s >= 0]
    ckv = W.bf16_bits_to_f32(w.ckv[blocks]).astype(np.float64).reshape(-1, DLAT)
    kpe = W.bf16_bits_to_f32(w.kpe[blocks]).astype(np.float64).reshape(-1, DPE)
    keys = np.concatenate([ckv, kpe], axis=1)                     # [T, 576]
    q = np.concatenate([W.bf16_bits_to_f32(w.q_lat[r]), W.bf16_bits_to_f32(w.q_pe[r])],
                       axis=-1).astype(np.float64).reshape(-1, DLAT + DPE)  # [Mq*H, 576]
    s = w.scale * (q @ keys.T)
    lse = scipy.special.logsumexp(s, axis=1)
    out = scipy.special.softmax(s, axis=1) @ ckv
    return out, lse


def pin_dense_equals_library(lib):
    w = W.random_case(21, R=2, Mq=2, H=4, P=9, NB=6, K=6, sigma=0.8)
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    for r in range(2):
        o_ref, l_ref = _dense_numpy(w, r)
        np.testing.assert_allclose(lse[r].reshape(-1), l_ref, rtol=0, atol=1e-12)
        for k in range(o_ref.shape[0]):
            assert rel_err(out[r].reshape(-1, DLAT)[k], o_ref[k]) <= 1e-12


# ------------------------------------------------------------ closed forms
def _single_block_case(seed, key_lat, key_pe, val_rows):
    """One job, one selected block whose 64 tokens have the given keys/values."""
    w = W.random_case(seed, R=1, Mq=1, H=3, P=2, NB=2, K=1)
    ckv = w.ckv.copy()
    kpe = w.kpe.copy()
    b = int(w.table[0, w.sel[0, 0]])
    ckv[b] = val_rows
    if key_lat is not None:
        ckv[b] = key_lat
    kpe[b] = key_pe
    return W.Workload("closed", w.q_lat, w.q_pe, ckv, kpe, w.table, w.sel, w.scale), b


def pin_identical_tokens(lib):
    """64 identical tokens: out = their value, lse = s + ln 64."""
    rng = np.random.default_rng(31)
    row = W.f32_to_bf16_bits(rng.standard_normal(DLAT).astype(np.float32))
    pe = W.f32_to_bf16_bits(rng.standard_normal(DPE).astype(np.float32))
    w, b = _single_block_case(31, None, np.broadcast_to(pe, (BLOCK, DPE)),
                              np.broadcast_to(row, (BLOCK, DLAT)))
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    v = W.bf16_bits_to_f32(row).astype(np.float64)
    for h in range(3):
        ql = W.bf16_bits_to_f32(w.q_lat[0, 0, h]).astype(np.float64)
        qp = W.bf16_bits_to_f32(w.q_pe[0, 0, h]).astype(np.float64)
        s = w.scale * (math.fsum(ql * v) + math.fsum(qp * W.bf16_bits_to_f32(pe)))
        assert abs(lse[0, 0, h] - (s + math.log(64))) <= 1e-12
        assert rel_err(out[0, 0, h], v) <= 1e-14


def pin_identical_keys_mean(lib):
    """Identical keys with distinct values: out = mean of the values."""
    rng = np.random.default_rng(32)
    w = W.random_case(32, R=1, Mq=1, H=2, P=3, NB=3, K=2)
    ckv = w.ckv.copy()
    kpe = w.kpe.copy()
    # zero the query's latent part so only the (identical) pe keys matter
    q_lat = np.zeros_like(w.q_lat)
    pe = W.f32_to_bf16_bits(rng.standard_normal(DPE).astype(np.float32))
    blocks = [int(w.table[0, s]) for s in w.sel[0]]
    for b in blocks:
        kpe[b] = pe
    w2 = W.Workload("keys", q_lat, w.q_pe, ckv, kpe, w.table, w.sel, w.scale)
    out, lse = oracle.partial(w2.q_lat, w2.q_pe, ckv, kpe, w.table, w.sel, w.scale, lib=lib)
    vals = W.bf16_bits_to_f32(ckv[blocks]).astype(np.float64).reshape(-1, DLAT)
    mean = vals.mean(axis=0)
    for h in range(2):
        qp = W.bf16_bits_to_f32(w.q_pe[0, 0, h]).astype(np.float64)
        s = w.scale * math.fsum(qp * W.bf16_bits_to_f32(pe))
        assert abs(lse[0, 0, h] - (s + math.log(vals.shape[0]))) <= 1e-12
        assert rel_err(out[0, 0, h], mean) <= 1e-13


def pin_zero_query(lib):
    """q = 0 (and, separately, scale = 0): out = mean of selected values,
    lse = ln(number of selected tokens)."""
    w = W.random_case(33, R=2, Mq=1, H=2, P=6, NB=4, K=3, n_valid=[3, 2])
    for q_lat, q_pe, scale in [(np.zeros_like(w.q_lat), np.zeros_like(w.q_pe), w.scale),
                               (w.q_lat, w.q_pe, 0.0)]:
        out, lse = oracle.partial(q_lat, q_pe, w.ckv, w.kpe, w.table, w.sel, scale, lib=lib)
        for r in range(2):
            blocks = [int(w.table[r, s]) for s in w.sel[r] if s >= 0]
            vals = W.bf16_bits_to_f32(w.ckv[blocks]).astype(np.float64).reshape(-1, DLAT)
            for h in range(2):
                assert abs(lse[r, 0, h] - math.log(vals.shape[0])) <= 1e-13
                assert rel_err(out[r, 0, h], vals.mean(axis=0)) <= 1e-13


def pin_two_groups(lib):
    """Two blocks, each of 64 identical tokens (keys kA, kB; values vA, vB):
    lse = logaddexp(sA, sB) + ln 64, out = sigmoid(sA - sB) vA + sigmoid(sB - sA) vB."""
    rng = np.random.default_rng(34)
    w = W.random_case(34, R=1, Mq=1, H=4, P=2, NB=2, K=2)
    ckv = w.ckv.copy()
    kpe = w.kpe.copy()
    rows = {}
    for s in range(2):
        b = int(w.table[0, w.sel[0, s]])
        v = W.f32_to_bf16_bits(rng.standard_normal(DLAT).astype(np.float32))
        p = W.f32_to_bf16_bits(rng.standard_normal(DPE).astype(np.float32))
        ckv[b] = v
        kpe[b] = p
        rows[s] = (W.bf16_bits_to_f32(v).astype(np.float64), W.bf16_bits_to_f32(p).astype(np.float64))
    out, lse = oracle.partial(w.q_lat, w.q_pe, ckv, kpe, w.table, w.sel, w.scale, lib=lib)
    for h in range(4):
        ql = W.bf16_bits_to_f32(w.q_lat[0, 0, h]).astype(np.float64)
        qp = W.bf16_bits_to_f32(w.q_pe[0, 0, h]).astype(np.float64)
        sA, sB = (w.scale * (math.fsum(ql * rows[s][0]) + math.fsum(qp * rows[s][1]))
                  for s in range(2))
        assert abs(lse[0, 0, h] - (np.logaddexp(sA, sB) + math.log(64))) <= 1e-12
        ref = scipy.special.expit(sA - sB) * rows[0][0] + scipy.special.expit(sB - sA) * rows[1][0]
        assert rel_err(out[0, 0, h], ref) <= 1e-12


def pin_one_hot(lib):
    """A huge scale makes the softmax one-hot: out = the top token's value and
    lse = the top score (gaps above 50 nats make the rest < 1e-21)."""
    w = W.random_case(35, R=1, Mq=1, H=3, P=3, NB=3, K=2)
    scale = 2000.0
    out, lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, scale, lib=lib)
    blocks = [int(w.table[0, s]) for s in w.sel[0]]
    ckv = W.bf16_bits_to_f32(w.ckv[blocks]).astype(np.float64).reshape(-1, DLAT)
    kpe = W.bf16_bits_to_f32(w.kpe[blocks]).astype(np.float64).reshape(-1, DPE)
    checked = 0
    for h in range(3):
        ql = W.bf16_bits_to_f32(w.q_lat[0, 0, h]).astype(np.float64)
        qp = W.bf16_bits_to_f32(w.q_pe[0, 0, h]).astype(np.float64)
        s = np.array([scale * (math.fsum(ql * ckv[k]) + math.fsum(qp * kpe[k]))
                      for k in range(ckv.shape[0])])
        top = np.argsort(s)[::-1]
        if s[top[0]] - s[top[1]] < 50:
            continue
        checked += 1
        assert abs(lse[0, 0, h] - s[top[0]]) <= 1e-9 * abs(s[top[0]])
        assert rel_err(out[0, 0, h], ckv[top[0]]) <= 1e-14
    assert checked >= 1


def pin_empty_and_duplicates(lib):
    """An empty selection gives (0, -inf); a block listed twice counts twice
    (same out, lse + ln 2); slot order does not matter."""
    w = W.random_case(36, R=1, Mq=1, H=2, P=4, NB=4, K=3)
    base_out, base_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table,
                                        w.sel[:, :1], w.scale, lib=lib)
    dup = np.array([[w.sel[0, 0], -1, w.sel[0, 0]]], np.int32)
    d_out, d_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, dup, w.scale, lib=lib)
    np.testing.assert_allclose(d_lse, base_lse + math.log(2), rtol=0, atol=1e-12)
    np.testing.assert_allclose(d_out, base_out, rtol=1e-13, atol=1e-15)
    empty = np.full((1, 3), -1, np.int32)
    e_out, e_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, empty, w.scale, lib=lib)
    assert np.all(e_lse == -np.inf) and np.all(e_out == 0.0)
    f_out, f_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, lib=lib)
    r_out, r_lse = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel[:, ::-1],
                                  w.scale, lib=lib)
    np.testing.assert_allclose(r_lse, f_lse, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r_out, f_out, rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------ merge algebra
def pin_merge_partition(lib):
    """Partials of any split of a selection, merged, equal the partial of the
    whole selection (Section 3.3: M-way scattered subsets reproduce the whole
    set); empty parts included."""
    w = W.random_case(41, R=1, Mq=2, H=3, P=12, NB=10, K=8)
    full_o, full_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale,
                                    lib=lib)
    rng = np.random.default_rng(41)
    for M in (1, 2, 3, 5, 8):
        owner = rng.integers(0, M, w.sel.shape[1])
        po, pl = [], []
        for m in range(M):
            sel = np.where(owner == m, w.sel[0], -1)[None, :].astype(np.int32)
            o, l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, sel, w.scale, lib=lib)
            po.append(o)
            pl.append(l)
        mo, ml = oracle.merge(np.stack(po), np.stack(pl), lib=lib)
        np.testing.assert_allclose(ml, full_l, rtol=0, atol=1e-12)
        for idx in np.ndindex(full_l.shape):
            assert rel_err(mo[idx], full_o[idx]) <= 1e-12


def _random_parts(seed, n, rows=5, dv=16):
    rng = np.random.default_rng(seed)
    o = rng.standard_normal((n, rows, dv))
    lam = rng.standard_normal((n, rows)) * 3
    return o, lam


def pin_merge_algebra(lib):
    """Commutativity, associativity, n = 1 identity, lse = logsumexp(lses),
    out = softmax(lses)-weighted sum of the parts."""
    o, lam = _random_parts(42, 4)
    mo, ml = oracle.merge(o, lam, lib=lib)
    np.testing.assert_allclose(ml, scipy.special.logsumexp(lam, axis=0), rtol=0, atol=1e-13)
    wts = scipy.special.softmax(lam, axis=0)
    np.testing.assert_allclose(mo, np.einsum("nr,nrd->rd", wts, o), rtol=1e-13, atol=1e-14)
    perm = [2, 0, 3, 1]
    po, pl = oracle.merge(o[perm], lam[perm], lib=lib)
    np.testing.assert_allclose(po, mo, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(pl, ml, rtol=0, atol=1e-13)
    ab_o, ab_l = oracle.merge(o[:2], lam[:2], lib=lib)
    cd_o, cd_l = oracle.merge(o[2:], lam[2:], lib=lib)
    t_o, t_l = oracle.merge(np.stack([ab_o, cd_o]), np.stack([ab_l, cd_l]), lib=lib)
    np.testing.assert_allclose(t_o, mo, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(t_l, ml, rtol=0, atol=1e-13)
    one_o, one_l = oracle.merge(o[:1], lam[:1], lib=lib)
    assert np.array_equal(one_o, o[0]) and np.array_equal(one_l, lam[0])


def pin_merge_zero_weight(lib):
    """A part with lse = -inf is skipped even when its output is NaN; all
    parts -inf gives (0, -inf) (Section 3.3: zero-weight identity)."""
    o, lam = _random_parts(43, 3)
    ref_o, ref_l = oracle.merge(o, lam, lib=lib)
    o2 = np.concatenate([o[:1], np.full_like(o[:1], np.nan), o[1:]])
    lam2 = np.concatenate([lam[:1], np.full_like(lam[:1], -np.inf), lam[1:]])
    z_o, z_l = oracle.merge(o2, lam2, lib=lib)
    np.testing.assert_allclose(z_o, ref_o, rtol=1e-15, atol=0)
    np.testing.assert_allclose(z_l, ref_l, rtol=1e-15, atol=0)
    n_o, n_l = oracle.merge(np.full_like(o, np.nan), np.full_like(lam, -np.inf), lib=lib)
    assert np.all(n_o == 0.0) and np.all(n_l == -np.inf)


# ------------------------------------------------------------ codecs
def pin_bf16_decode(lib):
    for bits in list(range(0, 0x7F80, 97)) + [0x3F80, 0xC000, 0x0001, 0x7F7F, 0x8000, 0x4049]:
        for sgn in (0, 0x8000):
            b = bits | sgn
            assert lib.oracle_bf16_to_f64(b) == _bf16_struct(b), hex(b)
    assert lib.oracle_bf16_to_f64(0x3F80) == 1.0
    assert lib.oracle_bf16_to_f64(0xC040) == -3.0


def pin_e4m3_decode(lib):
    import torch
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    for c in range(256):
        v = lib.oracle_e4m3fn_to_f64(c)
        if c & 0x7F == 0x7F:
            assert math.isnan(v) and math.isnan(ref[c])
            continue
        a = _E4M3[c & 0x7F]
        assert v == ref[c], (hex(c), v, ref[c])
        assert abs(v) == float(a), (hex(c), v)
        assert math.copysign(1.0, v) == (-1.0 if c & 0x80 else 1.0)
    assert lib.oracle_e4m3fn_to_f64(0x7E) == 448.0
    assert lib.oracle_e4m3fn_to_f64(0x01) == 2.0 ** -9
    assert lib.oracle_e4m3fn_to_f64(0x08) == 2.0 ** -6
    assert lib.oracle_e4m3fn_to_f64(0x38) == 1.0


ALL_PINS = [pin_bf16_decode, pin_e4m3_decode, pin_bruteforce_tiny, pin_bruteforce_multi,
            pin_bruteforce_per_row, pin_per_row_is_one_job_per_row, pin_bruteforce_tokens,
            pin_bruteforce_tokens_per_row, pin_tokens_cover_blocks, pin_single_token,
            pin_bruteforce_fp8, pin_dense_equals_library, pin_identical_tokens,
            pin_identical_keys_mean, pin_zero_query, pin_two_groups, pin_one_hot,
            pin_empty_and_duplicates, pin_merge_partition, pin_merge_algebra,
            pin_merge_zero_weight, pin_bruteforce_negative_scale, pin_bruteforce_wire_stats]
