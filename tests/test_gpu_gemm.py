"""GPU parity of focus_gemm against a float64 matrix product of the same bf16
inputs (a plain NumPy matmul is the definition).  Tolerance: f32 output
rel-L2 <= 1e-5 and max-abs <= 1e-4 * sqrt(k); bf16 output adds the output
rounding (relative 2^-9): rel-L2 <= 5e-3.  Cases: ragged M (tails of the
128-row and 256-row tiles), several N and K tiles (K = 64 and 192 take the
128 x 128 tile, multiples of 128 the 256 x 256 one), gathered rows, alpha, leading dimensions larger than the row,
and the projection shapes of an Evo-2-scale layer (d = 4096)."""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, rel_l2, to64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("m,n,k", [(1, 128, 64), (127, 128, 64), (129, 256, 128), (300, 384, 192),
                                   (300, 512, 256), (256, 256, 128), (256, 256, 64), (1000, 512, 1024), (4096, 1024, 4096)])
@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_gemm_matches_float64(m, n, k, out_dtype):
    announce(f"gemm m={m} n={n} k={k} out={out_dtype}")
    a = fw.randn((m, k), "bf16", m + k, DEV)
    b = fw.randn((k, n), "bf16", n + 7, DEV)
    od = torch.float32 if out_dtype == "f32" else torch.bfloat16
    c = F.focus_gemm(a, b, out_dtype=od, alpha=0.5)
    torch.cuda.synchronize()
    ref = 0.5 * (to64(a) @ to64(b))
    got = to64(c)
    r = rel_l2(got, ref)
    if out_dtype == "f32":
        assert r <= 1e-5 and np.abs(got - ref).max() <= 1e-4 * np.sqrt(k), r
    else:
        assert r <= 5e-3, r


def test_gemm_gathered_rows_and_strides():
    announce("gemm gather / strides")
    rows, k, n = 500, 256, 256
    big = fw.randn((rows, k + 64), "bf16", 3, DEV)
    a = big[:, :k]                                  # lda = k + 64
    b = fw.randn((k, n + 128), "bf16", 4, DEV)[:, :n]
    idx = np.random.default_rng(0).integers(0, rows, 333)
    out = torch.zeros(333, n + 128, dtype=torch.float32, device=DEV)[:, :n]
    F.focus_gemm(a, b, out=out, a_rows=idx)
    torch.cuda.synchronize()
    ref = to64(a)[idx] @ to64(b)
    assert rel_l2(to64(out), ref) <= 1e-5


def test_gemm_rejects_unsupported_shapes():
    a = torch.zeros(10, 100, dtype=torch.bfloat16, device=DEV)
    b = torch.zeros(100, 128, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(F.FocusError):
        F.focus_gemm(a, b)                          # k not a multiple of 64
