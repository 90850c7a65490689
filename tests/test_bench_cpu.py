"""Host-side checks of bench.py's work model (no GPU)."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads.configs import make_config  # noqa: E402


@pytest.fixture(scope="module")
def w2():
    return make_config(2)


def test_boxes_view_counts_the_boxes_nodes(w2):
    v = bench.boxes_view(w2, 1234)
    assert (v.n_dst, v.n_src) == (1234, 1234)
    assert (v.d, v.H1, v.H2, v.layers) == (w2.d, w2.H1, w2.H2, w2.layers)
    assert (w2.n_dst, w2.n_src) == (8192, 8192)   # the workload itself is unchanged


def test_inference_work_model_runs_on_the_view(w2):
    v = bench.boxes_view(w2, 2000)
    work = bench.work_model(v, 50000, 2000, True, n_dst=2000)
    work.update(bench.agg_work(v, 50000, 2000, True))
    assert {"edge_mlp", "outer_fwd", "gemm_fwd", "dz"} <= set(work)
    for fl, by in work.values():
        assert fl >= 0 and by > 0


def test_dz_bytes_of_the_feature_gradient_form():
    """d = 128, h = 256 (bf16): U_i and g_i once per destination; per edge the
    source index, h_j, z, z's mask bits, and the da2 and m_e rows written."""
    class S:   # the shape alone decides the formula: a stand-in with the workload-5 shape
        d, H1, H2, D, de, dtype = 128, 256, 256, 3, 8, "bf16"
        n_dst = 1000
    E = 24000
    fl, by = bench.agg_work(S, E, 1100)["dz"]
    assert by == 1000 * (256 * 128 + 128) * 2 + E * (4 + 256 + 512 + 32 + 512 + 256)
    assert fl == 2 * E * (128 * 256 * 2) + 2 * 1000 * 128 * 128
