"""GPU: the matrix-core GEMMs through the C ABI (dex_debug_gemm): the
skinny-M decode kernel (M <= 64) and the M-tiled prompt kernel (M > 64).

Parity with a float64 reference of the same bf16/fp32 inputs, batch
invariance (a row's bits do not depend on M or on the other rows), and
determinism.  Shapes span several tiles, a ragged last tile and ragged K."""
import ctypes

import numpy as np
import pytest

from synth import gen
from tests.gpu_common import torch_cuda

pytestmark = pytest.mark.gpu


def _gemm(torch, dtype, Wt, xt, M):
    from paper_2606_29223_amd import dexlib
    lib = dexlib.load()
    N, K = Wt.shape
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    st = lib.dex_debug_gemm(dtype, Wt.data_ptr(), N, K, xt.data_ptr(), M, y.data_ptr(),
                            torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _inputs(torch, dtype, N, K, M, seed):
    if dtype == 1:
        W = gen.uniform(seed, N * K, 0.05, bf16=True).reshape(N, K)
        x = gen.uniform(seed + 1, M * K, 1.0, bf16=True).reshape(M, K)
        Wt = torch.from_numpy(W.view(np.int16)).cuda()
        xt = torch.from_numpy(x.view(np.int16)).cuda()
        W64, x64 = gen.bf16_bits_to_f32(W).astype(np.float64), gen.bf16_bits_to_f32(x).astype(np.float64)
    else:
        W = gen.uniform(seed, N * K, 0.05).reshape(N, K)
        x = gen.uniform(seed + 1, M * K, 1.0).reshape(M, K)
        Wt, xt = torch.from_numpy(W).cuda(), torch.from_numpy(x).cuda()
        W64, x64 = W.astype(np.float64), x.astype(np.float64)
    return Wt, xt, W64, x64


@pytest.mark.parametrize("dtype,N,K", [(1, 784, 768), (1, 2048, 4096), (1, 96, 14336), (0, 344, 128),
                                       (0, 128, 344), (0, 52, 36)])
def test_gemm_matches_float64(dtype, N, K):
    torch = torch_cuda()
    for M in (1, 5, 16, 23, 64):
        Wt, xt, W64, x64 = _inputs(torch, dtype, N, K, M, 100 + N + M)
        y = _gemm(torch, dtype, Wt, xt, M)
        ref = x64 @ W64.T
        err = np.abs(y - ref).max()
        scale = np.sqrt(K) * 0.05
        assert err <= 2e-5 * scale + 1e-6, (M, err)


@pytest.mark.parametrize("N,K,M", [(784, 768, 65), (2048, 4096, 300), (96, 14336, 129), (6144, 4096, 1000)])
def test_tiled_prefill_gemm_matches_float64(N, K, M):
    """The M-tiled prompt GEMM (M > 64): ragged M against the 128-row
    workgroup tile, tile counts that leave a workgroup partly idle, long K."""
    torch = torch_cuda()
    Wt, xt, W64, x64 = _inputs(torch, 1, N, K, M, 300 + N + M)
    y = _gemm(torch, 1, Wt, xt, M)
    ref = x64 @ W64.T
    err = np.abs(y - ref).max()
    assert err <= 2e-5 * np.sqrt(K) * 0.05 + 1e-6, err
    # deterministic run to run
    assert np.array_equal(y.view(np.uint32), _gemm(torch, 1, Wt, xt, M).view(np.uint32))


@pytest.mark.parametrize("N,K,M", [(6144, 4096, 2100), (2064, 14336, 3000), (1552, 776, 4000)])
def test_large_prefill_gemm_matches_the_small_tiles(N, K, M):
    """A grid of 96 or more 256 x 256 workgroups (here 216, 108 and 112, with
    ragged last blocks in M and N, and a last k-step only a quarter inside
    K = 776) takes the LDS-staged kernel.  It feeds
    every MFMA tile the same operands in the same k-step order as the
    128 x 128 kernel, which 500-row launches of the same rows take (at most
    48 such workgroups), so each row's bits are equal; and float64 parity
    on rows at the workgroup edges and in the ragged last block."""
    torch = torch_cuda()
    Wt, xt, W64, x64 = _inputs(torch, 1, N, K, M, 500 + N)
    big = _gemm(torch, 1, Wt, xt, M)
    rows = [0, 1, 255, 256, 1023, M - 257, M - 256, M - 1] + list(np.random.default_rng(N).integers(0, M, 8))
    ref = x64[rows] @ W64.T
    err = np.abs(big[rows] - ref).max()
    assert err <= 2e-5 * np.sqrt(K) * 0.05 + 1e-6, err
    for lo, hi in ((0, 500), (M - 500, M)):
        small = _gemm(torch, 1, Wt, xt[lo:hi].contiguous(), hi - lo)
        assert np.array_equal(small.view(np.uint32), big[lo:hi].view(np.uint32)), (lo, hi)
    assert np.array_equal(big.view(np.uint32), _gemm(torch, 1, Wt, xt, M).view(np.uint32))


@pytest.mark.parametrize("dtype", [1, 0])
def test_gemm_batch_invariance_and_determinism(dtype):
    torch = torch_cuda()
    N, K = (1040, 4096) if dtype == 1 else (344, 344)
    Wt, xt, _, _ = _inputs(torch, dtype, N, K, 64, 7)
    full = _gemm(torch, dtype, Wt, xt, 64)
    again = _gemm(torch, dtype, Wt, xt, 64)
    assert np.array_equal(full.view(np.uint32), again.view(np.uint32))
    for M in (1, 2, 3, 4, 7, 16, 17, 32, 33, 48):
        y = _gemm(torch, dtype, Wt, xt[:M].contiguous(), M)
        assert np.array_equal(y.view(np.uint32), full[:M].view(np.uint32)), M
    # a row's bits do not depend on its position or on its neighbours
    perm = torch.randperm(64, generator=torch.Generator().manual_seed(0))
    yp = _gemm(torch, dtype, Wt, xt[perm.cuda()].contiguous(), 64)
    assert np.array_equal(yp.view(np.uint32), full[perm.numpy()].view(np.uint32))
    one = _gemm(torch, dtype, Wt, xt[37:38].contiguous(), 1)
    assert np.array_equal(one.view(np.uint32), full[37:38].view(np.uint32))


def test_copy_kernel():
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    lib = dexlib.load()
    a = torch.arange(1 << 20, dtype=torch.int32, device="cuda")
    b = torch.zeros_like(a)
    assert lib.dex_debug_copy(b.data_ptr(), a.data_ptr(), a.numel() * 4, None) == 0
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("dtype", [1, 0])
def test_weight_row_bits_do_not_depend_on_its_tile(dtype):
    """A weight row's outputs have the same bits whatever the other rows of
    its 16-row tile hold (zeros, other rows, the row itself moved to another
    tile and position): the matrix cores give each output element its own
    row's dot product.  (With the activation-row independence above, this is
    what lets the workgroup tiling of a GEMM change without changing a
    bit.)"""
    torch = torch_cuda()
    N, K = 64, 4096 if dtype == 1 else 344
    for M in (1, 7, 16):
        Wt, xt, _, _ = _inputs(torch, dtype, N, K, M, 500 + M)
        y = _gemm(torch, dtype, Wt, xt, M)
        rng = np.random.default_rng(M)
        perm = rng.permutation(N)
        y_perm = _gemm(torch, dtype, Wt[torch.from_numpy(perm).cuda()].contiguous(), xt, M)
        assert np.array_equal(y_perm.view(np.uint32), y[:, perm].view(np.uint32))
        keep = np.zeros(N, dtype=bool)
        keep[rng.choice(N, size=N // 3, replace=False)] = True
        Wz = Wt.clone()
        Wz[torch.from_numpy(~keep).cuda()] = 0
        y_z = _gemm(torch, dtype, Wz, xt, M)
        assert np.array_equal(y_z[:, keep].view(np.uint32), y[:, keep].view(np.uint32))
