"""The committed rocprofv3 summaries under profiles/ are consistent with
themselves: the counter summaries name existing sources, their traffic is
their scaled FETCH_SIZE and WRITE_SIZE, their matrix-core FLOP are the MOPS
counter times 512, and the bench reads them back as stored.  (Whether a
summary is current for the kernel source is the bench's check: it reports no
traffic for a summary taken from other code.)
"""
import glob
import json
import os

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COUNTERS = sorted(glob.glob(os.path.join(ROOT, "profiles", "*_counters.json")))
MFMA = sorted(glob.glob(os.path.join(ROOT, "profiles", "*_mfma.json")))


def _load(path):
    with open(path) as f:
        return json.load(f)


def test_there_are_summaries():
    assert COUNTERS and MFMA


@pytest.mark.parametrize("path", COUNTERS, ids=os.path.basename)
def test_traffic_summary_is_self_consistent(path):
    d = _load(path)
    sources = d.get("sources") or [d["source"]]
    for s in sources:
        assert os.path.exists(os.path.join(ROOT, s)), s
    # the copy calibration: 512 MiB moved each way, FETCH_SIZE counts it twice
    ref = d["copy_reference"]
    assert ref["bytes"] == 512 << 20
    assert abs(d["fetch_scale"] - ref["bytes"] / 1024 / ref["fetch_size_kib"]) < 1e-9
    assert abs(d["write_scale"] - ref["bytes"] / 1024 / ref["write_size_kib"]) < 1e-9
    assert 1.9 < d["fetch_scale"] < 2.1 and 0.95 < d["write_scale"] < 1.05
    t = (d["fetch_size_kib_per_dispatch"] * d["fetch_scale"]
         + d["write_size_kib_per_dispatch"] * d["write_scale"]) * 1024
    assert abs(t - d["traffic_bytes"]) <= 1.0
    assert d["traffic_bytes"] > 0
    md = path.replace("_counters.json", ".md")
    if os.path.basename(md).startswith(("partial_kernel", "gather_kernel", "splice_kernel")):
        assert os.path.exists(md), md


@pytest.mark.parametrize("path", MFMA, ids=os.path.basename)
def test_mfma_summary_is_self_consistent(path):
    d = _load(path)
    assert d["counter"] == "SQ_INSTS_VALU_MFMA_MOPS_BF16"
    assert d["flop_per_dispatch"] == d["mops_bf16_per_dispatch"] * 512
    for s in d["sources"]:
        assert os.path.exists(os.path.join(ROOT, s)), s


def test_bench_reads_the_summaries_back():
    """Where a summary matches the current source, the bench reports exactly
    its figure; otherwise it reports none."""
    for path in COUNTERS:
        d = _load(path)
        name = os.path.basename(path)[:-len("_counters.json")]
        kernel = next(k for k in ("partial_kernel", "merge_kernel", "gather_kernel", "splice_kernel")
                      if name.startswith(k))
        workload = name[len(kernel) + 1:]
        got = bench.counted_traffic(workload, 0, kernel)
        fresh = bench.sources_fingerprint(d.get("sources") or [d["source"]]) == \
            d.get("source_code_fingerprint")
        assert got == (d["traffic_bytes"] if fresh else None), name
    for path in MFMA:
        d = _load(path)
        workload = os.path.basename(path)[len("partial_kernel_"):-len("_mfma.json")]
        fresh = bench.sources_fingerprint(d["sources"]) == d.get("source_code_fingerprint")
        assert bench.counted_flop(workload, 0) == (d["flop_per_dispatch"] if fresh else None)
