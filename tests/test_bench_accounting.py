"""The bench's algorithmic work per launch (op_plan), which the roofline
fractions divide by, against counts derived by hand for the production
retrieval shape (16 requests x 65,536 candidates; IKBO linear 2048 + 512 ->
1024 ReLU -> 256; history 2048 x 1024 per request, 8 heads x 128):

- layer 1: 2 N K_c D + 2 R K_r D FLOPs; x_cand, output, both weights and
  x_req once: 2 (N K_c + N D + (K_r + K_c) D + R K_r) bytes;
- layer 2: 2 N 1024 256 FLOPs; 2 (N 1024 + N 256 + 1024 256) bytes;
- K/V projection: 2 (R L) 1024 2048 FLOPs; S, W and [K | V] once;
- attention: 4 d H sum_r n_r L_r FLOPs (QK^T and PV); Q, O and K/V once.
"""

from types import SimpleNamespace

import numpy as np
import pytest

import bench

R, PER, L = 16, 65536, 2048
N = R * PER


@pytest.fixture(scope="module")
def plan5():
    w = SimpleNamespace(config_id=5, n_req=R, n_cand=N,
                        cand_offsets=np.arange(R + 1) * PER, kv_offsets=np.arange(R + 1) * L)
    return {name: (flops, byts, bound) for name, flops, byts, bound in bench.op_plan(w)}


def test_production_retrieval_counts(plan5):
    assert plan5["ikbo_linear_l1"][:2] == (2 * N * 512 * 1024 + 2 * R * 2048 * 1024,
                                           2 * (N * 512 + N * 1024 + 2560 * 1024 + R * 2048))
    assert plan5["linear_l2"][:2] == (2 * N * 1024 * 256, 2 * (N * 1024 + N * 256 + 1024 * 256))
    assert plan5["kv_projection"][:2] == (2 * R * L * 1024 * 2048,
                                          2 * (R * L * 1024 + 2048 * 1024 + R * L * 2048))
    assert plan5["dca_attention"][:2] == (4 * 128 * 8 * N * L,
                                          2 * (2 * N * 8 * 128 + 2 * R * L * 8 * 128))


def test_production_retrieval_bounds(plan5):
    # Arithmetic intensity against the bf16 ridge (2.5 PFLOP/s / 8 TB/s ~ 312 FLOP/B).
    ridge = bench.PEAK_BF16_TFLOPS * 1e12 / (bench.PEAK_HBM_GBS * 1e9)
    for name, (flops, byts, bound) in plan5.items():
        assert bound == ("mfma" if flops / byts > ridge else "hbm"), name
