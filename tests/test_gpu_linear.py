"""tri_linear (C = A B^T on the layer's GEMM kernels) on the GPU, through the
C ABI, against the oracle's projection in float64.

Every output element must be the bf16 rounding of the exact product or an
adjacent bf16 value, with at most 1% of the elements one ulp off (fp32
accumulation over K moves a value across a rounding boundary now and then).
The shapes reach each GEMM path: the short-batch split-K planes (M <= 128),
the mid-size 128-row tiles with three LDS stages (row blocks past M skipped),
the 128 x 256 tiles that fill one round, the 256 x 256 tiles (a final
round a quarter to a half full as 128-row halves of its tiles), and the tail split with uneven K splits (long K).  The
largest shapes are checked on sampled rows.
"""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import to_device_bf16, to_host_f64
from synth import bf16_to_f32, normal_bf16
from test_gpu_layer import assert_rounded

pytestmark = pytest.mark.gpu

SHAPES = [
    (1, 256, 512),        # one row: skinny planes
    (25, 1024, 2048),     # skinny, 64-row tile, split K
    (128, 4608, 3584),    # skinny at its row limit (the q/k/v shape)
    (130, 640, 576),      # mid-size tiles, 2 valid rows in the last M-tile
    (544, 3584, 18944),   # long K: 256 x 256 tail split, uneven K splits
    (1000, 768, 1024),    # mid-size tiles, 104 valid rows in the last M-tile
    (4096, 4096, 1024),   # 256 x 256 tiles, one full round
    (4096, 2048, 4096),   # 128 x 256 tiles, one round of 256
    (3000, 2048, 1024),   # 128 x 256 tiles, 56 valid rows in the last M-tile
    (6144, 4096, 256),    # 1.5 rounds of 256 x 256: the last 128 tiles as 128-row halves
    (5944, 4096, 256),    # same, the last M-tile's second half empty
    (5120, 4096, 512),    # 64 tail tiles (a four-way split at short K) as 128-row halves
]


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_linear_against_oracle(M, N, K):
    import torch
    a_bits = normal_bf16(11, 1, (M, K), std=1.0)
    b_bits = normal_bf16(11, 2, (N, K), std=0.05)
    a, b = to_device_bf16(a_bits), to_device_bf16(b_bits)
    c = T.linear(a, b)
    torch.cuda.synchronize()
    rows = np.arange(M) if M * N * K <= 2 ** 33 else np.unique(
        np.r_[0, 1, 127, 128, 255, 256, 511, 512, M // 2, M - 2, M - 1].clip(0, M - 1))
    a64 = bf16_to_f32(a_bits).astype(np.float64)[rows]
    b64 = bf16_to_f32(b_bits).astype(np.float64)
    exact = oracle.project(a64, b64)
    got = to_host_f64(c)[rows]
    assert_rounded(got, exact, f"linear {M}x{N}x{K}")


def test_linear_twice_bit_identical_and_stream_ordered():
    """Two calls on one stream, the second reading the first's output: the
    results are deterministic and ordered (no reduction depends on timing)."""
    import torch
    M, N, K = 300, 1024, 1024
    a = to_device_bf16(normal_bf16(12, 1, (M, K)))
    b = to_device_bf16(normal_bf16(12, 2, (N, K), std=0.03))
    c1 = T.linear(a, b)
    c2 = T.linear(a, b)
    d = T.linear(c1, b[:, :N].contiguous())     # K = N: chained on the same stream
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    exact = oracle.project(to_host_f64(c1), to_host_f64(b))
    assert_rounded(to_host_f64(d), exact, "linear chained")
