"""Host-side rejections of the C ABI (CPU only): every call in
tests/abi_cases.py must return its status and name the problem in
mla_last_error() before anything is launched.  The same cases run on the GPU
with canary-filled outputs in test_gpu_abi_canary.py."""
import pytest
import torch

from paper_2606_01502_amd import mla
from tests import abi_cases as C

CPU = torch.device("cpu")


def _ids(cases):
    return [c[0] for c in cases]


@pytest.mark.parametrize("case", C.partial_cases(CPU), ids=_ids(C.partial_cases(CPU)))
def test_partial_rejects(case):
    name, mutate, status, text = case
    a = C.partial_args(CPU)
    mutate(a)
    st, msg = C.call_partial(a)
    assert st == status, (name, st, msg)
    assert text in msg, (name, msg)


@pytest.mark.parametrize("case", C.partial_cases_fp8(CPU), ids=_ids(C.partial_cases_fp8(CPU)))
def test_partial_fp8_rejects(case):
    name, mutate, status, text = case
    a = C.partial_args(CPU, fp8=True)
    mutate(a)
    st, msg = C.call_partial(a)
    assert st == status, (name, st, msg)
    assert text in msg, (name, msg)


@pytest.mark.parametrize("case", C.merge_cases(CPU), ids=_ids(C.merge_cases(CPU)))
def test_merge_rejects(case):
    name, mutate, status, text = case
    a = C.merge_args(CPU)
    mutate(a)
    st, msg = C.call_merge(a)
    assert st == status, (name, st, msg)
    assert text in msg, (name, msg)


def test_error_text_cleared_by_next_call():
    """mla_last_error() describes the last non-OK status of the thread; a
    later call starts from an empty text."""
    lib = mla.load()
    a = C.partial_args(CPU)
    a["scale"] = float("nan")
    st, msg = C.call_partial(a)
    assert st != mla.MLA_OK and msg
    m = C.merge_args(CPU)
    m["n"] = 0
    st2, msg2 = C.call_merge(m)
    assert st2 != mla.MLA_OK and "n_parts" in msg2 and "scale" not in msg2
    assert lib.mla_last_error().decode() == msg2


def test_wrappers_refuse_host_tensors():
    """The Python binding refuses host tensors before calling the library: a
    host address handed to a kernel would fault the GPU."""
    a = C.partial_args(CPU)
    with pytest.raises(ValueError, match="GPU"):
        mla.sparse_partial_attn(a["q_lat"], a["q_pe"], a["ckv"], a["kpe"], a["table"], a["sel"],
                                0.1)
    m = C.merge_args(CPU)
    with pytest.raises(ValueError, match="GPU"):
        mla.merge_partials(m["lat"], m["lse"])
