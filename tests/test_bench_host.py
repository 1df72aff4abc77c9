"""Host-side pieces of bench.py: the pair and table-row counts behind the dQ/dK roofline
and the refusal of more than one GPU (no device needed)."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
torch = pytest.importorskip("torch")
import bench  # noqa: E402


@pytest.mark.parametrize("bh,nq,nk,m,tau,t", [(3, 50, 57, 4, 3, 2), (1, 1, 1, 1, 1, 0), (2, 200, 130, 7, 8, 1),
                                              (2, 300, 310, 3, 2, 32)])
def test_bucket_work_matches_brute_force(bh, nq, nk, m, tau, t):
    g = np.random.default_rng(bh + nq + m)
    # high bits above tau are set at random: only the low tau bits are a code
    q = g.integers(0, 2**15, (bh, nq, m)).astype(np.int16)
    k = g.integers(0, 2**15, (bh, nk, m)).astype(np.int16)
    mask = (1 << tau) - 1
    pairs = pair_form = table_rows = 0
    for b in range(bh):
        for h in range(m):
            for c in range(1 << tau):
                bq = int(((q[b, :, h] & mask) == c).sum())
                bk = int(((k[b, :, h] & mask) == c).sum())
                pairs += bq * bk
                if bq * bk > t * (bq + bk):
                    table_rows += bq + bk
                else:
                    pair_form += bq * bk
    brute = sum(int(((q[b, :, h, None] & mask) == (k[b, None, :, h] & mask)).sum()) for b in range(bh) for h in range(m))
    assert pairs == brute
    assert bench.bucket_work(torch.from_numpy(q), torch.from_numpy(k), tau, t) == (pairs, pair_form, table_rows)


def test_identical_codes_give_all_pairs_per_bucket():
    # every row in bucket 0: n_q * n_k pairs per (head, hash), in the table form when
    # 600 > t * 50
    q = torch.zeros((2, 30, 5), dtype=torch.int16)
    k = torch.zeros((2, 20, 5), dtype=torch.int16)
    assert bench.bucket_work(q, k, 8, 32) == (2 * 5 * 30 * 20, 2 * 5 * 30 * 20, 0)
    assert bench.bucket_work(q, k, 8, 11) == (2 * 5 * 30 * 20, 0, 2 * 5 * 50)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_bucket_load_by_hand():
    # tau = 2 (4 buckets), one head, one hash: queries fill bucket 1 with 20 rows and
    # bucket 3 with 4; keys put all 24 rows in bucket 0
    q = torch.tensor([1] * 20 + [3] * 4, dtype=torch.int16).reshape(1, 24, 1)
    k = torch.zeros((1, 24, 1), dtype=torch.int16)
    load = bench.bucket_load(q, k, 2)
    assert load["queries"]["mean_rows"] == 6.0
    assert load["queries"]["max_rows"] == 20 and load["queries"]["max_over_mean"] == round(20 / 6, 2)
    assert load["queries"]["row_share_by_bucket_rows"]["<=16"] == round(4 / 24, 4)
    assert load["queries"]["row_share_by_bucket_rows"]["<=64"] == round(20 / 24, 4)
    assert load["keys"]["max_rows"] == 24 and load["keys"]["row_share_by_bucket_rows"]["<=64"] == 1.0
    # every row is counted once, whatever the high bits above tau hold
    g = np.random.default_rng(3)
    r = torch.from_numpy(g.integers(0, 2**15, (3, 500, 7)).astype(np.int16))
    shares = bench.bucket_load(r, r, 5)["queries"]["row_share_by_bucket_rows"]
    assert abs(sum(shares.values()) - 1.0) < 1e-3
