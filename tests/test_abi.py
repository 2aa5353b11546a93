"""The C-ABI library loads and exports every entry point the header declares.
CPU only: no entry point that launches work is called here."""
import ctypes
import os
import re

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
    assert lib.mla_version() == 1
    assert lib.mla_last_error() == b""


def test_descriptor_layout_matches_header():
    from paper_2606_01502_amd import mla
    # void* + 2 x int32 + 4 x int64 + 4 x int64 + pointer
    assert ctypes.sizeof(mla.Tensor) == 8 + 8 + 32 + 32 + 8
    assert ctypes.sizeof(mla.PartialOpts) == 32
