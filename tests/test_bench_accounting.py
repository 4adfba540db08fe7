"""The work bench.py divides its times by -- the algorithmic bytes of a step, the FLOPs of
a build, the FLOPs of an extension -- against closed forms written here from the model
shapes alone: matmul parameters n_layers (4 d^2 + 3 d F), K/V bytes per token n_layers * 2 d
* 2 bytes, causal query-key pairs L (L + 1) / 2, and the per-unit figures they give for the
12-layer and 7B workloads (3.09 GB and 78.6 GB per step, 0.917 and 3.75 TFLOP per build)."""
import numpy as np

import bench
from paper_2508_10259_amd import workload as W


def _shape(name):
    wl = W.WORKLOADS[name]
    s = wl.spec
    return wl, s, s.n_layers, s.d_model, s.d_ffn


def test_matmul_params():
    for name, want in (("mid-b8", 201_326_592), ("7b-b1", 6_476_005_376)):
        wl, s, L, d, F = _shape(name)
        assert L * (4 * d * d + 3 * d * F) == want == s.matmul_params


def test_step_bytes():
    """A step with no new tokens: A - 1 passes each read every weight once (bf16) and row b's
    K/V for keys 0 .. L_b + j - 1 and write its new key/value; A evaluations of the 256 bin
    rows of the head."""
    for name, gb in (("mid-b8", 3.09), ("7b-b1", 78.6), ("7b-chunk56-b16", 1002.7)):
        wl, s, L, d, F = _shape(name)
        B, A, Lb = wl.batch, wl.n_actions, sum(wl.prefix)
        kv_tok = L * 2 * d * 2
        passes = A - 1
        weights = passes * 2 * L * (4 * d * d + 3 * d * F)
        kv_read = kv_tok * B * (passes * Lb + passes * (passes + 1) // 2)
        kv_write = kv_tok * B * passes
        head = A * 256 * d * 2
        want = weights + kv_read + kv_write + head
        got = bench.step_bytes(s, np.full(B, Lb), A)
        assert got == want, name
        assert abs(got / 1e9 - gb) < 0.05 * max(1.0, gb / 100), (name, got)


def test_build_flops():
    """2 P_mm FLOPs per prefix token plus 4 d n_layers per causal query-key pair."""
    for name, tf in (("mid-b8", 0.917), ("7b-b1", 3.75), ("7b-chunk56-b16", 125.85)):
        wl, s, L, d, F = _shape(name)
        B, Lb = wl.batch, sum(wl.prefix)
        want = 2 * L * (4 * d * d + 3 * d * F) * B * Lb + 4 * d * L * B * (Lb * (Lb + 1) // 2)
        got = bench.build_flops(s, np.full(B, Lb))
        assert got == want, name
        assert abs(got / 1e12 - tf) < 0.005 * tf + 0.001, (name, got)
    # ragged rows add up row by row
    wl, s, L, d, F = _shape("7b-b64-ragged")
    lens = np.array([200, 333, 400])
    assert bench.build_flops(s, lens) == sum(bench.build_flops(s, np.array([x])) for x in lens)


def test_shared_build_flops():
    """A row that attaches k shared prefix pages computes positions 64 k .. L - 1 only: the FLOPs of
    its build are those of the whole row less those of a row of 64 k tokens; the first positions
    are read from the page table (the leading run of pages an earlier row of the build holds)."""
    wl, s, L, d, F = _shape("7b-b64-ragged")
    lens = [300, 250, 130, 200]
    pt = np.array([[0, 1, 2, 3, 4],
                   [0, 1, 5, 6, 7],   # attaches pages 0, 1
                   [0, 8, 9, 10, 11],  # attaches page 0 only (page 8 is its own)
                   [12, 1, 13, 14, 15]])  # page 0 differs: nothing attached, though page 1 repeats
    starts = bench.shared_starts(pt, lens)
    assert starts == [0, 128, 64, 0]
    # at most floor((L - 1) / 64) pages are attached: the row's last position is always computed
    assert bench.shared_starts(np.array([[0, 1, 2], [0, 1, 2]]), [192, 128]) == [0, 64]
    got = bench.build_flops(s, lens, starts)
    want = sum(bench.build_flops(s, [l]) - bench.build_flops(s, [k]) for l, k in zip(lens, starts))
    assert got == want
    assert bench.build_flops(s, lens, [0] * 4) == bench.build_flops(s, lens)


def test_extension_flops():
    """Appending n tokens to a row of L committed tokens: 2 P_mm FLOPs per new token, and new token
    i attends to L + i + 1 keys (4 d n_layers FLOPs per query-key pair).  The 7B batch-64 step
    (16 tokens per row on rows of about 468) is 13.5 TFLOP."""
    wl, s, L, d, F = _shape("7b-b64-ragged")
    P = L * (4 * d * d + 3 * d * F)
    for Lb, n in ((0, 5), (300, 16), (17, 1)):
        pairs = sum(Lb + i + 1 for i in range(n))
        assert bench.extension_flops(s, [Lb], [n]) == 2 * P * n + 4 * d * L * pairs
    assert bench.extension_flops(s, [300, 10], [0, 0]) == 0
    got = bench.extension_flops(s, [460] * 64, [16] * 64)
    assert abs(got / 1e12 - 13.5) < 0.1, got
    # prefix + extension pairs = the pairs of building the longer prefix
    assert bench.extension_flops(s, [40], [9]) + bench.build_flops(s, [40]) == bench.build_flops(s, [49])


def test_phase_summary():
    hbm = bench.phase_summary([(0.5, 2e12), (0.5, 2e12)], "hbm", 8000.0)
    assert hbm["achieved"] == 4000.0 and hbm["frac"] == 0.5 and hbm["bytes_per_launch"] == 2e12
    assert hbm["avg_launch_us"] == 5e5 and hbm["launches"] == 2
    mf = bench.phase_summary([(2.0, 2.5e15)], "mfma", 2500.0)
    assert mf["achieved"] == 1250.0 and mf["frac"] == 0.5
    assert bench.phase_summary([], "hbm", 8000.0) is None


def test_decode_kernel_names():
    mid, s7 = W.MODELS["mid"], W.MODELS["7b"]
    assert bench.decode_kernel_name(mid, 8, 7, True).startswith("k_decode_fused<64>")
    assert bench.decode_kernel_name(s7, 1, 7, True).startswith("k_decode_fused<128>")
    assert "k_gemm_wide<1,2>" in bench.decode_kernel_name(s7, 16, 56, False)
    assert "k_gemm_wide<4,2>" in bench.decode_kernel_name(s7, 64, 7, False)
