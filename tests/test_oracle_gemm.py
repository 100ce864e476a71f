"""Pins for the oracle's GEMM, consumer sum and RMSNorm.

GEMM: against numpy's float64 matmul (an independent BLAS routine), a
pure-Python brute force on tiny inputs, the identity-operand case (products by
1 and sums with 0 are exact, so C = B bit for bit) and a closed form.
Consumer: the sum of two fp16 values against numpy's float16 addition (IEEE
correctly rounded). RMSNorm: against torch's float64 rms_norm and closed
forms (constant rows, bias = -x).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads


def _rand(shape, seed, dtype="fp16", scale=1.0):
    rng = np.random.default_rng(seed)
    return workloads.to_bits(rng.uniform(-1, 1, shape) * scale, dtype)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("shape", [(64, 48, 80), (128, 64, 256), (7, 5, 3)])
def test_gemm_matches_numpy_float64(dtype, shape):
    M, N, K = shape
    A = _rand((M, K), 1, dtype)
    W = _rand((N, K), 2, dtype, 1 / math.sqrt(K))
    got = oracle.gemm_exact(A, W, dtype)
    ref = oracle.decode(A, dtype) @ oracle.decode(W, dtype).T
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_gemm_bruteforce_tiny():
    M, N, K = 3, 4, 5
    A = _rand((M, K), 3)
    W = _rand((N, K), 4)
    a = A.view(np.float16).astype(float)
    w = W.view(np.float16).astype(float)
    ref = np.zeros((M, N))
    for i in range(M):
        for n in range(N):
            s = 0.0
            for k in range(K):
                s += a[i, k] * w[n, k]
            ref[i, n] = s
    np.testing.assert_array_equal(oracle.gemm_exact(A, W, "fp16"), ref)
    np.testing.assert_array_equal(oracle.gemm_exact_bits_path(A, W, "fp16"), ref)


def test_gemm_identity_operand_is_exact():
    K = N = 64
    A = workloads.to_bits(np.eye(K), "fp16")
    B = _rand((K, N), 5)                  # logical [K, N]
    W = np.ascontiguousarray(B.T)
    C = oracle.gemm_ref(A, W, "fp16")
    np.testing.assert_array_equal(C, B)


def test_gemm_closed_form_ones():
    M, N, K = 8, 8, 96
    A = workloads.to_bits(np.ones((M, K)), "fp16")
    W = workloads.to_bits(np.ones((N, K)), "fp16")
    np.testing.assert_array_equal(oracle.gemm_exact(A, W, "fp16"), np.full((M, N), float(K)))


def test_gemm_row_subset_matches_full():
    A = _rand((32, 40), 6)
    W = _rand((24, 40), 7)
    full = oracle.gemm_exact(A, W, "fp16")
    rows = np.array([3, 17, 31])
    sub = oracle.gemm_exact(A, W, "fp16", rows=rows, cols=(5, 19))
    np.testing.assert_array_equal(sub, full[rows][:, 5:19])


def test_add_matches_numpy_float16():
    a = _rand(100_000, 8)
    b = _rand(100_000, 9)
    ref = (a.view(np.float16) + b.view(np.float16)).view(np.uint16)
    np.testing.assert_array_equal(oracle.add_rne(a, b, "fp16"), ref)


def test_add_bf16_matches_torch():
    a = _rand(50_000, 10, "bf16")
    b = _rand(50_000, 11, "bf16")
    ta = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    tb = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16)
    # torch adds bf16 in float32 and rounds once; float32 holds the exact sum
    # of two bf16 values of these magnitudes, so this is correctly rounded.
    ref = (ta.float() + tb.float()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.add_rne(a, b, "bf16"), ref)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_rmsnorm_matches_torch_float64(dtype):
    rows, n = 16, 512
    x = _rand((rows, n), 12, dtype, 3.0)
    bias = _rand(n, 13, dtype, 0.1)
    gamma = workloads.to_bits(np.random.default_rng(14).uniform(0.5, 1.5, n), dtype)
    eps = 1e-6
    h = torch.from_numpy(oracle.decode(x, dtype) + oracle.decode(bias, dtype))
    ref = torch.nn.functional.rms_norm(h, (n,), weight=torch.from_numpy(oracle.decode(gamma, dtype)), eps=eps)
    ref_bits = oracle.encode(ref.numpy(), dtype)
    got = oracle.rmsnorm(x, dtype, bias=bias, gamma=gamma, eps=eps)
    # same math in fp64 (different summation order): at most one ulp apart,
    # and almost always identical
    diff = np.abs(got.astype(np.int32) - ref_bits.astype(np.int32))
    assert diff.max() <= 1
    assert (diff == 0).mean() > 0.999


def test_rmsnorm_closed_forms():
    n = 256
    for c in (0.5, -3.0, 1e-3):
        x = workloads.to_bits(np.full((1, n), c), "fp16")
        cv = float(oracle.decode(x, "fp16")[0, 0])
        y = oracle.rmsnorm(x, "fp16", eps=1e-6)
        expect = oracle.encode(np.array([cv / math.sqrt(cv * cv + 1e-6)]), "fp16")[0]
        assert np.all(y == expect)
    x = _rand((4, n), 15)
    neg = (x ^ np.uint16(0x8000)).astype(np.uint16)[0]      # bias = -x (row 0)
    y = oracle.rmsnorm(x[:1], "fp16", bias=neg, eps=1e-6)
    assert np.all(oracle.decode(y, "fp16") == 0.0)


def test_rmsnorm_unit_mean_square():
    x = _rand((8, 1024), 16, "fp16", 2.0)
    y = oracle.decode(oracle.rmsnorm(x, "fp16", eps=1e-6), "fp16")
    ms = (y * y).mean(axis=1)
    np.testing.assert_allclose(ms, 1.0, rtol=2e-3)
