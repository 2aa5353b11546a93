"""The C-ABI library loads and exports every entry point the header declares.
CPU only: no entry point that launches work is called here."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mla_sparse.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:mla_status_t|const char\*|int32_t)\s+(mla_\w+)\(",
                                 text, re.M)))


def test_header_declares_the_entry_points():
    from paper_2606_01502_amd import mla
    assert set(_declared()) == set(mla.EXPORTS)


def test_library_exports_every_declared_symbol():
    from paper_2606_01502_amd import mla
    lib = ctypes.CDLL(mla.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name


def test_version_and_error_string_without_gpu():
    from paper_2606_01502_amd import mla
    lib = mla.load()
    with open(os.path.join(ROOT, "include", "mla_sparse.h")) as f:
        want = int(re.search(r"#define MLA_SPARSE_VERSION (\d+)", f.read()).group(1))
    assert lib.mla_version() == want == 4
    assert lib.mla_last_error() == b""


def test_descriptor_layout_matches_header():
    from paper_2606_01502_amd import mla
    # void* + 2 x int32 + 4 x int64 + 4 x int64 + pointer
    assert ctypes.sizeof(mla.Tensor) == 8 + 8 + 32 + 32 + 8
    assert ctypes.sizeof(mla.PartialOpts) == 32


def _describe_fieldwise(t, block_scale=None):
    from paper_2606_01502_amd import mla
    d = mla.Tensor()
    d.data = t.data_ptr() if t.numel() else None
    d.dtype = mla._TORCH_DTYPES.get(t.dtype, 0)
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.stride[i] = t.stride(i)
    if block_scale is not None:
        d.block_scale = block_scale.data_ptr()
    return d


def test_packed_descriptor_equals_fieldwise():
    """describe() packs the struct in one go; it must give the same bytes as
    setting each field of mla_tensor_t."""
    import torch
    from paper_2606_01502_amd import mla
    base = torch.arange(4 * 6 * 5 * 8, dtype=torch.float32).reshape(4, 6, 5, 8)
    scale = torch.ones(7, dtype=torch.float32)
    cases = [(base, None), (base[1:3, ::2, :, 3:], None), (base.transpose(0, 2), None),
             (torch.zeros(3, 64, 512, dtype=torch.uint8), scale),
             (torch.zeros(5, 7, dtype=torch.int32), None), (torch.zeros(9, dtype=torch.bfloat16), None),
             (torch.zeros(0, 4, dtype=torch.float32), None), (torch.zeros((), dtype=torch.float32), None)]
    for t, bs in cases:
        assert bytes(mla.describe(t, bs)) == bytes(_describe_fieldwise(t, bs)), (t.shape, t.stride())


def _cpu_call(sel_shape, fp8=False, R=2, Mq=3, H=16, P=8, NB=5, row_tile=0, tokens=False,
              scale=0.1):
    """Call the partial entry point on host tensors through ctypes: only the
    host-side checks run (each of these calls must fail before anything is
    launched)."""
    import torch
    from tests import abi_cases as C
    a = C.partial_args(torch.device("cpu"), fp8=fp8, R=R, Mq=Mq, H=H, P=P, NB=NB)
    a["sel"] = torch.zeros(sel_shape, dtype=torch.int32)
    a["opts"].row_tile = row_tile
    a["tokens"] = tokens
    a["scale"] = scale
    return C.call_partial(a)


def test_per_row_selection_host_checks():
    from paper_2606_01502_amd import mla
    st, msg = _cpu_call((2, 4, 3))  # Mq mismatch
    assert st == mla.MLA_ERR_INVALID_ARGUMENT and "[R, Mq, K]" in msg
    st, msg = _cpu_call((3, 3))  # R mismatch
    assert st == mla.MLA_ERR_INVALID_ARGUMENT
    st, msg = _cpu_call((2, 3, 3), NB=40000)  # per-row counters would not fit in LDS
    assert st == mla.MLA_ERR_UNSUPPORTED and "NB" in msg
    st, msg = _cpu_call((2, 3, 3, 1))  # 4-d selection
    assert st == mla.MLA_ERR_INVALID_ARGUMENT
    # a 128-row tile of H = 1 spans 128 query rows, more than a row mask holds
    st, msg = _cpu_call((2, 70, 3), Mq=70, H=1, row_tile=128)
    assert st == mla.MLA_ERR_UNSUPPORTED and "128-row" in msg


def test_token_selection_host_checks():
    from paper_2606_01502_amd import mla
    st, msg = _cpu_call((2, 3, 3), tokens=True)  # no per-row token selections
    assert st == mla.MLA_ERR_INVALID_ARGUMENT and "sel_token_ids" in msg
    st, msg = _cpu_call((3, 3), tokens=True)  # R mismatch
    assert st == mla.MLA_ERR_INVALID_ARGUMENT


def test_row_tile_option_checked():
    from paper_2606_01502_amd import mla
    for bad in (96, -64, 1, 256):
        st, msg = _cpu_call((2, 3), row_tile=bad)
        assert st == mla.MLA_ERR_INVALID_ARGUMENT and "row_tile" in msg


def test_scale_must_be_finite_and_bounded():
    """The last host check before planning and launch: shapes here are valid,
    so only the scale stops these calls (negative and zero scales are
    allowed and computed; see the GPU parity tests)."""
    import torch
    from paper_2606_01502_amd import mla
    if torch.cuda.is_available():
        pytest.skip("host-check test: its tensors live in host memory")
    for bad in (float("inf"), float("-inf"), float("nan"), 2.0 ** 64 * (1 + 2.0 ** -23), -(2.0 ** 70)):
        for kw in ({}, {"tokens": True}, {"fp8": True}):
            st, msg = _cpu_call((2, 3), scale=bad, **kw)
            assert st == mla.MLA_ERR_INVALID_ARGUMENT and "scale" in msg, (bad, kw, msg)
