"""Shared helpers of the GPU tests: upload a workload, run the HIP path through
the C ABI, and compare it with the oracle at the parity bar.

Parity bar (bf16 inputs, fp32 accumulation): every output row within a
row-normwise relative error of 1e-2, max_d |gpu - ref| / max_d |ref|, and
every log-sum-exp within 1e-3 absolute; -inf must match exactly.
"""
import numpy as np
import torch

from paper_2606_01502_amd import mla

OUT_REL_TOL = 1e-2
LSE_ABS_TOL = 1e-3


def device():
    return torch.device("cuda:0")


def upload(w):
    """Workload host arrays -> device tensors (bf16 bits reinterpreted)."""
    dev = device()

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    t = dict(q_lat=bf16(w.q_lat), q_pe=bf16(w.q_pe),
             table=torch.from_numpy(np.ascontiguousarray(w.table)).to(dev),
             sel=torch.from_numpy(np.ascontiguousarray(w.sel)).to(dev))
    if w.fp8:
        t["ckv"] = torch.from_numpy(np.ascontiguousarray(w.ckv)).to(dev)
        t["kpe"] = torch.from_numpy(np.ascontiguousarray(w.kpe)).to(dev)
        t["ckv_scale"] = torch.from_numpy(np.ascontiguousarray(w.ckv_scale)).to(dev)
        # one array for both pools selects the library's shared-scale path
        t["kpe_scale"] = (t["ckv_scale"] if w.kpe_scale is w.ckv_scale else
                          torch.from_numpy(np.ascontiguousarray(w.kpe_scale)).to(dev))
    else:
        t["ckv"] = bf16(w.ckv)
        t["kpe"] = bf16(w.kpe)
        t["ckv_scale"] = t["kpe_scale"] = None
    return t


def run_partial(t, scale, n_splits=0, sel=None, row_tile=0, tokens=False):
    out, lse = mla.sparse_partial_attn(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                       t["sel"] if sel is None else sel, scale,
                                       ckv_scale=t["ckv_scale"], kpe_scale=t["kpe_scale"],
                                       n_splits=n_splits, row_tile=row_tile, tokens=tokens)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def row_errors(out, ref):
    """Row-normwise relative errors of [..., 512] arrays."""
    o = out.reshape(-1, out.shape[-1])
    r = ref.reshape(-1, ref.shape[-1])
    num = np.abs(o - r).max(axis=1)
    den = np.maximum(np.abs(r).max(axis=1), 1e-30)
    zero = np.abs(r).max(axis=1) == 0
    rel = np.where(zero, num, num / den)
    return rel


def assert_parity(out, lse, ref_out, ref_lse, what=""):
    assert np.all(np.isfinite(out)), f"{what}: non-finite output"
    ninf_ref = ref_lse == -np.inf
    assert np.array_equal(lse == -np.inf, ninf_ref), f"{what}: -inf pattern of lse differs"
    live = ~ninf_ref
    if live.any():
        err = np.abs(lse[live] - ref_lse[live]).max()
        assert err <= LSE_ABS_TOL, f"{what}: lse abs error {err:.3g}"
    if ninf_ref.any():
        assert np.all(out[ninf_ref] == 0.0), f"{what}: empty rows must be 0"
    rel = row_errors(out, ref_out)
    assert rel.max() <= OUT_REL_TOL, f"{what}: row-relative error {rel.max():.3g} at row {rel.argmax()}"
    return rel.max(), (np.abs(lse[live] - ref_lse[live]).max() if live.any() else 0.0)
