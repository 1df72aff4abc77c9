"""gfx950 facts the backward kernels rely on, checked on the device.

* fp16 subnormal inputs of the 16x16x32 f16 MFMA are multiplied exactly: the low halves of the
  hi/lo splits of dY, V, Q and K are often subnormal, and a flush would drop them.
* `ds_read_b64_tr_b16` distributes its 16-bit elements as the pair kernel's transposed reads assume.

The probe is built by `__graft_entry__.build()` (or `python tests/hw/hw_facts.py --build`).
"""
from __future__ import annotations

import os
import sys

import pytest

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "hw"))
import hw_facts  # noqa: E402


@pytest.mark.gpu
def test_mfma_subnormals_and_transpose_read_layout():
    res = hw_facts.run(checks_only=True)
    print(res.stdout, flush=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "check fp16 subnormal products exact in MFMA: yes" in res.stdout
    assert "check ds_read_b64_tr_b16 lane layout as documented: yes" in res.stdout
