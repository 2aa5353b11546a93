"""Token selections (an indexer's top-k single tokens, Section 6.3's
selection budgets) against the oracle: ids anywhere in the chunk, ragged
counts that leave a partly filled last group of 64, duplicates, empty and
invalid slots, every split and tile setting, and top-2048 over a 32K-token
chunk at 128 heads sampled at full size."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01502_amd import mla, workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _ref(w, jobs=None):
    if jobs is None:
        return oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, w.table, w.sel, w.scale, tokens=True)
    j = np.asarray(jobs)
    return oracle.partial(w.q_lat[j], w.q_pe[j], w.ckv, w.kpe, w.table[j], w.sel[j], w.scale,
                          tokens=True)


def _check(w, n_splits=0, row_tile=0, what=""):
    out, lse = G.run_partial(G.upload(w), w.scale, n_splits=n_splits, row_tile=row_tile,
                             tokens=True)
    ref_o, ref_l = _ref(w)
    return G.assert_parity(out, lse, ref_o, ref_l, what or w.name)


@pytest.mark.parametrize("row_tile", [0, 64, 128])
@pytest.mark.parametrize("n_splits", [0, 1, 2, 5])
def test_tokens_random_splits(n_splits, row_tile):
    print(f"case: tokens splits={n_splits} row_tile={row_tile}", flush=True)
    w = W.random_case(701, R=3, Mq=1, H=128, P=30, NB=12, K=300, sigma=0.6, allow_dup=True,
                      tokens=True)
    _check(w, n_splits, row_tile, f"tokens splits={n_splits} row_tile={row_tile}")


@pytest.mark.parametrize("k", [1, 37, 63, 64, 65, 127, 129, 1000, 1025])
def test_tokens_ragged_counts(k):
    """Listed-token counts around multiples of 64 (the last group is partly
    fill) and past one list (1024 slots per split)."""
    print(f"case: tokens k={k}", flush=True)
    nb = max(2, -(-k // 64) + 3)
    w = W.random_case(710 + k, R=2, Mq=2, H=16, P=nb + 5, NB=nb, K=k, sigma=0.8,
                      allow_dup=k > 64 * nb // 2, tokens=True)
    _check(w, what=f"tokens k={k}")


def test_tokens_padding_duplicates_empty():
    print("case: tokens padding", flush=True)
    w = W.random_case(720, R=4, Mq=1, H=32, P=12, NB=8, K=200, n_valid=[0, 1, 70, 200],
                      allow_dup=True, pad_pattern="interleaved", tokens=True)
    for s in (0, 1, 3):
        _check(w, s, what=f"tokens padding splits={s}")


def test_tokens_invalid_ids_are_skipped():
    print("case: tokens invalid ids", flush=True)
    w = W.random_case(730, R=2, Mq=1, H=16, P=9, NB=5, K=90, tokens=True)
    sel = w.sel.copy()
    sel[0, 3] = 5 * 64            # >= 64 NB
    sel[1, 10] = -9               # negative, not -1
    table = w.table.copy()
    table[1, sel[1, 20] // 64] = 9  # >= P: every token of that block is skipped
    bad = W.Workload("bad", w.q_lat, w.q_pe, w.ckv, w.kpe, table, sel, w.scale, tokens=True)
    out, lse = G.run_partial(G.upload(bad), w.scale, tokens=True)
    clean = sel.copy()
    clean[0, 3] = -1
    clean[1, 10] = -1
    clean[1][(sel[1] >= 0) & (sel[1] // 64 == sel[1, 20] // 64)] = -1
    ref_o, ref_l = oracle.partial(w.q_lat, w.q_pe, w.ckv, w.kpe, table, clean, w.scale,
                                  tokens=True)
    G.assert_parity(out, lse, ref_o, ref_l, "tokens invalid ids")


def test_tokens_listing_whole_blocks_equals_block_selection():
    """Every token of the selected blocks, shuffled, against the block
    selection of the same blocks, both on the GPU."""
    print("case: tokens vs blocks", flush=True)
    w = W.random_case(740, R=3, Mq=1, H=128, P=40, NB=20, K=12, sigma=0.5)
    rng = np.random.default_rng(740)
    tok = np.stack([rng.permutation((w.sel[r][:, None] * 64 + np.arange(64)).ravel())
                    for r in range(3)]).astype(np.int32)
    t = G.upload(w)
    out_b, lse_b = G.run_partial(t, w.scale)
    out_t, lse_t = G.run_partial(t, w.scale, sel=torch.from_numpy(tok).to(G.device()),
                                 tokens=True)
    G.assert_parity(out_t, lse_t, out_b, lse_b, "tokens vs blocks")


def test_tokens_top2048_of_32k_sampled():
    """The selection budget of DeepSeek-V3.2 / GLM-5.1 (top-2048 tokens) over
    a 32K-token chunk, 128 heads, 8 requests; the oracle checks 2."""
    print("case: tokens top-2048 of 32K", flush=True)
    w = W.make("select-tok-b8-k2048-c32768")
    out, lse = G.run_partial(G.upload(w), w.scale, tokens=True)
    jobs = [0, 5]
    ref_o, ref_l = _ref(w, jobs)
    G.assert_parity(out[jobs], lse[jobs], ref_o, ref_l, "top-2048 of 32K")


def _check8(w, n_splits=0, row_tile=0, what="", jobs=None):
    out, lse = G.run_partial(G.upload(w), w.scale, n_splits=n_splits, row_tile=row_tile,
                             tokens=True)
    j = np.arange(w.sel.shape[0]) if jobs is None else np.asarray(jobs)
    ref_o, ref_l = oracle.partial(w.q_lat[j], w.q_pe[j], w.ckv, w.kpe, w.table[j], w.sel[j],
                                  w.scale, w.ckv_scale, w.kpe_scale, tokens=True)
    return G.assert_parity(out[j], lse[j], ref_o, ref_l, what or w.name)


def _fp8_tokens(seed, shared, **kw):
    """A token case whose pool blocks have distinct fp8 scales (each block's
    values drawn at its own magnitude), so every listed token carries its
    own block's scale."""
    w = W.random_case(seed, tokens=True, **kw)
    P = w.ckv.shape[0]
    mag = np.random.default_rng(seed).uniform(0.2, 3.0, P).astype(np.float32)
    for name in ("ckv", "kpe"):
        x = W.bf16_bits_to_f32(getattr(w, name)) * mag[:, None, None]
        setattr(w, name, W.f32_to_bf16_bits(x))
    return w.to_fp8(shared)


@pytest.mark.parametrize("row_tile", [64, 128])
@pytest.mark.parametrize("n_splits", [0, 1, 3])
@pytest.mark.parametrize("shared", [True, False])
def test_tokens_fp8(shared, n_splits, row_tile):
    print(f"case: fp8 tokens shared={shared} splits={n_splits} row_tile={row_tile}", flush=True)
    w = _fp8_tokens(760, shared, R=3, Mq=1, H=128, P=30, NB=12, K=300, sigma=0.6,
                    allow_dup=True)
    assert len(np.unique(w.ckv_scale)) > 20
    _check8(w, n_splits, row_tile, f"fp8 tokens shared={shared} splits={n_splits}")


@pytest.mark.parametrize("k", [1, 63, 65, 1025])
@pytest.mark.parametrize("shared", [True, False])
def test_tokens_fp8_ragged_and_padding(k, shared):
    print(f"case: fp8 tokens k={k} shared={shared}", flush=True)
    nb = max(2, -(-k // 64) + 3)
    w = _fp8_tokens(770 + k, shared, R=2, Mq=2, H=16, P=nb + 5, NB=nb, K=k, sigma=0.8,
                    allow_dup=True, pad_pattern="interleaved", n_valid=[k, max(0, k - 7)])
    _check8(w, what=f"fp8 tokens k={k}")


def test_tokens_fp8_top2048_of_32k_sampled():
    print("case: fp8 tokens top-2048 of 32K", flush=True)
    w = W.make("select-tok-b8-k2048-c32768").to_fp8(shared_scale=False)
    _check8(w, jobs=[1, 6], what="fp8 top-2048 of 32K")


def test_tokens_reject_per_row():
    w = W.random_case(750, R=1, Mq=2, H=16, P=8, NB=4, K=10, tokens=True)
    t = G.upload(w)
    sel3 = torch.zeros((1, 2, 10), dtype=torch.int32, device=G.device())
    with pytest.raises(mla.MlaError) as e:
        mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"], sel3,
                                w.scale, tokens=True)
    assert e.value.status == mla.MLA_ERR_INVALID_ARGUMENT
