"""The two-phase hash (Algorithm 1) on the GPU through the C ABI against the reference,
bit for bit: segment hashes and the final index value, over ragged sizes, every segment
size regime (one partial 16-byte chunk, right-aligned short segments, multi-block segments)
and the full packed prefix of the 7B batch-64 workload (157 MB)."""
import numpy as np
import pytest

import oracle.index as X
from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _gpu_hash(data: bytes, s: int):
    import torch
    from paper_2508_10259_amd.runtime import index_hash
    t = torch.from_numpy(np.frombuffer(data, dtype=np.uint8).copy()).cuda()
    out, ws = index_hash(t, s)
    torch.cuda.synchronize()
    u = lambda x: [int(v) & 0xFFFFFFFFFFFFFFFF for v in x.cpu().numpy().tolist()]
    return u(out)[0], u(ws)


CASES = [(1, 16), (15, 16), (16, 16), (17, 16), (100, 64), (4095, 4096), (4096, 4096), (4097, 4096),
         (12345, 4096), (8192 * 3 + 10, 8192), (65536 * 3 + 7, 65536), (300001, 48), (2 * 65536, 65536)]


@pytest.mark.parametrize("n,s", CASES)
def test_index_hash_matches_reference(n, s):
    data = np.random.default_rng(n + s).integers(0, 256, size=n, dtype=np.uint8).tobytes()
    H, segs = _gpu_hash(data, s)
    ref = X.segment_hashes(data, s)
    assert segs == ref
    assert H == X.two_phase_hash(data, s)


def test_index_hash_full_7b_batch64_inputs():
    """The serialised inputs of the 7B batch-64 workload's first epoch -- each row's bf16 patch
    embeddings (about 18,000 tokens x 8 KB in all) followed by its instruction ids (int32) --
    in 4 KB segments: every segment hash and the final value equal the reference's."""
    from paper_2508_10259_amd import workload as W
    wl = W.WORKLOADS["7b-b64-ragged"]
    data = b"".join(pr.patches.tobytes() + pr.text_ids.astype("<i4").tobytes() for pr in W.make_prefixes(wl, 0, 0))
    log(f"index hash over {len(data) / 1e6:.1f} MB")
    H, segs = _gpu_hash(data, 4096)
    ref = X.segment_hashes(data, 4096)
    assert len(segs) == len(ref) and segs == ref
    assert H == X.hash_func2(ref, len(data))
