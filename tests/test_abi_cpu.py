"""The C ABI library loads and exports every declared entry point (no GPU needed)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dsmpnn.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dsmp_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    import paper_2402_15106_amd as dm
    if not os.path.exists(dm.LIB_PATH):
        pytest.fail("libdsmpnn.so is not built; run __graft_entry__.build()")
    return dm.load_library()


def test_every_declared_symbol_is_exported_and_bound(lib):
    import paper_2402_15106_amd as dm
    names = _declared()
    assert len(names) >= 16
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(dm.EXPORTED) == names


def test_version(lib):
    assert lib.dsmp_version() == 10000


def test_host_side_queries(lib):
    import paper_2402_15106_amd as dm
    nb = ctypes.c_size_t()
    assert lib.dsmp_sample_workspace(1000, ctypes.byref(nb)) == dm.OK and nb.value > 0
    assert lib.dsmp_sample_workspace(-1, ctypes.byref(nb)) == dm.INVALID_ARG
    q = dm._lib.GraphQuery(0, 1000, 900, 2, 0.1, 0, 0, 0)
    assert lib.dsmp_radius_graph_workspace(ctypes.byref(q), ctypes.byref(nb)) == dm.OK and nb.value > 0
    for (dtype, d, h1, h2) in [(dm.F32, 32, 64, 64), (dm.BF16, 64, 128, 128), (dm.BF16, 128, 256, 256)]:
        desc = dm.layer_desc(3, d, h1, h2, dtype)
        assert lib.dsmp_nnconv_packed_bytes(ctypes.byref(desc), ctypes.byref(nb)) == dm.OK
        assert nb.value % 256 == 0 and nb.value >= 3 * d * d * h2 * (2 if dtype == dm.BF16 else 4)
        g = dm._lib.CGraph(100, 120, 5000, 0, 0, 0, 0, 0)
        s, f, b = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        assert lib.dsmp_nnconv_workspace(ctypes.byref(desc), ctypes.byref(g), ctypes.byref(s),
                                         ctypes.byref(f), ctypes.byref(b)) == dm.OK
        esz = 2 if dtype == dm.BF16 else 4
        # z and z1 per edge, plus the per-destination sums of the aggregate form
        assert s.value >= 5000 * (h1 + h2) * esz + 100 * (h2 + 1) * d * esz
    assert lib.dsmp_set_edge_algorithm(None, dm.EDGE_AGGREGATE) == dm.INVALID_ARG


def test_unsupported_and_invalid_descriptors(lib):
    import paper_2402_15106_amd as dm
    nb = ctypes.c_size_t()
    bad = [dm.layer_desc(2, 48, 128, 128, dm.BF16), dm.layer_desc(2, 128, 256, 256, dm.F32),
           dm.layer_desc(2, 64, 128, 64, dm.BF16)]
    for desc in bad:
        assert lib.dsmp_nnconv_packed_bytes(ctypes.byref(desc), ctypes.byref(nb)) == dm.UNSUPPORTED
    assert lib.dsmp_nnconv_packed_bytes(ctypes.byref(dm.layer_desc(4, 64, 128, 128, dm.BF16)),
                                        ctypes.byref(nb)) == dm.INVALID_ARG
    assert lib.dsmp_nnconv_packed_bytes(ctypes.byref(dm.layer_desc(2, 64, 128, 128, 7)),
                                        ctypes.byref(nb)) == dm.INVALID_ARG


def test_null_handle_is_rejected(lib):
    import paper_2402_15106_amd as dm
    assert lib.dsmp_sample_nodes(None, 10, 5, 0, None, None, 0) == dm.INVALID_ARG
    assert lib.dsmp_set_stream(None, None) == dm.INVALID_ARG
    assert lib.dsmp_last_error(None) == b""
    assert lib.dsmp_create(None, 0) == dm.INVALID_ARG


def test_hop_loop_host_side_queries(lib):
    import paper_2402_15106_amd as dm
    sb, wb = ctypes.c_size_t(), ctypes.c_size_t()
    desc = dm.MlpDesc(3, 64, 32)
    assert lib.dsmp_mlp_workspace(ctypes.byref(desc), 1000, ctypes.byref(sb), ctypes.byref(wb)) == dm.OK
    assert sb.value >= 2 * 1000 * 64 * 4 and wb.value >= 2 * 1000 * 64 * 4
    assert lib.dsmp_mlp_workspace(ctypes.byref(dm.MlpDesc(3, 6, 32)), 10, ctypes.byref(sb),
                                  ctypes.byref(wb)) == dm.UNSUPPORTED          # hidden width not a multiple of 4
    assert lib.dsmp_mlp_workspace(ctypes.byref(desc), -1, ctypes.byref(sb), ctypes.byref(wb)) == dm.INVALID_ARG
    assert lib.dsmp_masked_mse_workspace(5000, ctypes.byref(sb)) == dm.OK and sb.value >= 20 * 8
    assert lib.dsmp_masked_mse_workspace(-1, ctypes.byref(sb)) == dm.INVALID_ARG
    assert lib.dsmp_mlp_forward(None, ctypes.byref(desc), None, None, 0, None, None, None, 0) == dm.INVALID_ARG
