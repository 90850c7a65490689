"""GPU check of the allocation-free sampling entry point against
dsmp_sample_nodes: two calls in a row, the second smaller, bit for bit, and
the size limit rejected on the host."""

import numpy as np
import pytest

from tests.helpers import announce, gpu_lib

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    return gpu_lib()


def test_noalloc_sampling_matches_workspace_sampling(env):
    dm, lib, torch = env
    for M, s, seed in ((1000003, 12345, 77), (65536, 8192, 4002), (4096, 4096, 5), (1 << 24, 3, 9)):
        announce("noalloc sampling", M, s, seed)
        want = lib.dsmp_sample_nodes(M, s, seed)
        got = torch.full((s,), -1, dtype=torch.int32, device="cuda")
        lib.dsmp_sample_nodes_noalloc(M, s, seed, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), (M, s)
        assert np.all(np.diff(got.cpu().numpy()) > 0)


def test_noalloc_sampling_rejects_oversize(env):
    dm, lib, torch = env
    out = torch.empty(4, dtype=torch.int32, device="cuda")
    with pytest.raises(dm.DsmpError) as e:
        lib.dsmp_sample_nodes_noalloc((1 << 24) + 1, 4, 1, out)
    assert e.value.status == dm.UNSUPPORTED
