"""The allocation-free index hash (ams_index_hash_noalloc) against the workspace entry point
(ams_index_hash) and the reference, bit for bit, on two calls in a row -- the second with a
smaller input -- plus its size limit."""
import ctypes as C

import numpy as np
import pytest

import oracle.index as X

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_noalloc_matches_workspace_entry_point():
    import torch
    from paper_2508_10259_amd import capi
    lib = capi.load()
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(77)
    for n, s in ((131072 * 64 - 5, 64), (100_003, 4096)):  # the first fills the scratch to its last segment
        host = rng.integers(0, 256, size=n, dtype=np.uint8)
        data = torch.from_numpy(host).cuda()
        k = -(-n // s)
        ws = torch.empty(k, dtype=torch.int64, device="cuda")
        out_ws = torch.zeros(1, dtype=torch.int64, device="cuda")
        out_na = torch.zeros(1, dtype=torch.int64, device="cuda")
        capi.check(lib.ams_index_hash(data.data_ptr(), n, s, ws.data_ptr(), k * 8, out_ws.data_ptr(), stream),
                   "ams_index_hash")
        capi.check(lib.ams_index_hash_noalloc(data.data_ptr(), n, s, out_na.data_ptr(), stream),
                   "ams_index_hash_noalloc")
        torch.cuda.synchronize()
        a = int(out_ws.item()) & 0xFFFFFFFFFFFFFFFF
        b = int(out_na.item()) & 0xFFFFFFFFFFFFFFFF
        assert a == b
        assert b == X.two_phase_hash(host.tobytes(), s)


def test_noalloc_rejects_more_segments_than_its_scratch():
    import torch
    from paper_2508_10259_amd import capi
    lib = capi.load()
    data = torch.empty(131072 * 16 + 16, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    st = lib.ams_index_hash_noalloc(data.data_ptr(), data.numel(), 16, out.data_ptr(), None)
    assert st == capi.AMS_EINVAL
    assert b"scratch" in lib.ams_last_error()
    torch.cuda.synchronize()
    assert int(out.item()) == 0  # nothing was enqueued
