"""The work bench.py divides its times by -- the algorithmic bytes of a step, the FLOPs of
a build, the bytes of the gate|up launch -- against closed forms written here from the model
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


def test_gate_up_launch_bytes():
    """Weights [2F, d] in fp16 once, the input rows as fp16 pairs, and the gated output as fp16
    pairs where the kernel writes it (up to 8 rows; the wide kernel leaves it to its reduction)."""
    wl, s, L, d, F = _shape("7b-b1")
    for B, out in ((1, True), (8, True), (16, False), (64, False)):
        want = 2 * F * d * 2 + B * d * 4 + (B * F * 4 if out else 0)
        assert bench.gu_launch_bytes(s, B) == want, B


def test_roofline_kernel_names():
    mid, s7 = W.MODELS["mid"], W.MODELS["7b"]
    assert bench.roofline_kernel_name(mid, 7, 8, True).startswith("k_decode_fused<64>")
    assert bench.roofline_kernel_name(s7, 7, 1, True).startswith("k_decode_fused<128>")
    assert bench.roofline_kernel_name(s7, 56, 16, False).startswith("k_gemm_wide<1,2>")
    assert bench.roofline_kernel_name(s7, 7, 64, False).startswith("k_gemm_wide<4,2>")
