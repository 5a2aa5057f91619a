"""Host-side rules of the benchmark (CPU): the KV copies it rotates keep both
each call's cache bytes and each draft's gathered rows out of the 256 MB
Infinity Cache, so that its figures are HBM figures."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_27735_amd.workloads import CONFIGS, make_config  # noqa: E402

MIB = 1 << 20


@pytest.mark.parametrize("n", sorted(CONFIGS))
def test_rotation_keeps_cache_and_gathers_cold(n):
    w = make_config(n)
    kv_bytes = w.k.size * 2 * 2          # K and V, bf16
    draft = bench.algorithmic_bytes(w, out_bytes=2)[0]["draft"]
    c = bench.kv_copies(w, kv_bytes)
    assert 2 <= c <= 256
    # between two uses of one copy, the other copies' bytes (and their
    # drafts' gathered rows) exceed 512 MiB, unless the cap of 256 copies
    # binds first
    assert (c - 1) * kv_bytes > 512 * MIB
    assert (c - 1) * draft > 512 * MIB or c == 256


def test_algorithmic_bytes_of_the_32k_workload():
    """Verify: K and V once (8 heads x 32768 keys x 256 B each), the scores
    and the query / output rows; draft: the gathered K and V rows and their
    indices; select: the scores and the index list."""
    w = make_config(2)
    nb, n_idx = bench.algorithmic_bytes(w, out_bytes=2)
    assert nb["verify"] == 8 * 32768 * 128 * 2 * 2 + 8 * 32768 * 4 + 7 * 32 * 128 * 2 * 2
    assert n_idx == [2048]
    assert nb["draft"] == 8 * 2048 * (128 * 2 * 2 + 4) + 32 * 128 * 4
    assert nb["select"] == 8 * 32768 * 4 + 8 * 2048 * 4 + 4
