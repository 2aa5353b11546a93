"""Calls from several host threads on one stream.  Split jobs go through the
library's per-stream workspace (partial kernel, then combine); each call must
queue both kernels without another call's partial kernel between them, also
while the workspace grows.  Every thread's results must equal, bit for bit,
the same call made alone."""
import threading

import numpy as np
import pytest
import torch

from paper_2606_01502_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def test_threads_share_one_stream():
    print("case: 4 threads x 12 split calls on the default stream", flush=True)
    cases = []
    for i in range(4):
        # different job counts give different workspace sizes
        w = W.random_case(900 + i, R=2 + 2 * i, Mq=2, H=32, P=24, NB=12, K=10, sigma=0.8)
        cases.append((w, G.upload(w)))
    alone = [G.run_partial(t, w.scale, n_splits=5) for w, t in cases]
    errors = []

    def worker(i):
        try:
            w, t = cases[i]
            for it in range(12):
                out, lse = G.run_partial(t, w.scale, n_splits=5)
                if not (np.array_equal(out, alone[i][0]) and
                        np.array_equal(lse, alone[i][1], equal_nan=True)):
                    errors.append(f"thread {i} call {it}: result differs from the lone call")
                    return
        except Exception as e:  # reported below, with the thread
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=100)
    torch.cuda.synchronize()
    assert not any(th.is_alive() for th in threads), "a thread did not finish"
    assert not errors, errors
