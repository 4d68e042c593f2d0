"""Maximum sizes on the GPU: a decode weight above 4 GB (the decode kernel
addresses weights with 64-bit offsets), its repack round trip, and a prefill
weight just below the prefill kernel's 4 GB offset limit; sampled outputs
against the oracle.  The weights are seeded draws made on the device (too
large to draw and ship from the host in a test); the oracle receives the
sampled rows copied back, never a value computed by the library."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_bits, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.empty_cache()


def device_weight(N, K, seed):
    """bf16 [N, K] ~ N(0, 0.02^2), drawn on the device by torch's seeded generator."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn((N, K), generator=g, device="cuda", dtype=torch.float32) * synth.W_SIGMA).to(torch.bfloat16)


def sampled_check(A_bits, W_dev, C, n_samples, seed, what):
    """Compare C at random (m, n) with the oracle on the same A and the sampled weight rows."""
    import torch
    M, N = C.shape
    rng = np.random.default_rng(seed)
    ms = rng.integers(0, M, n_samples)
    ns = rng.integers(0, N, n_samples)
    rows = np.unique(ns)
    W_rows = host_bits(W_dev[torch.from_numpy(rows).cuda()])
    where = {int(r): i for i, r in enumerate(rows)}
    y_ref = oracle.gemm_f64_points(A_bits, W_rows, ms, np.array([where[int(n)] for n in ns]))
    got = C.float()[torch.from_numpy(ms).cuda(), torch.from_numpy(ns).cuda()].cpu().numpy()
    parity(got, y_ref, what)


def test_decode_weight_above_4GB():
    import torch
    M, N, K = 8, 131072, 32768          # 8 GiB of bf16 weights
    banner(f"large decode M={M} N={N} K={K}")
    W = device_weight(N, K, seed=71)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    A = synth.normal_bf16((M, K), seed=72)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), Wt, C, M, N, K, tl.layout(), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    sampled_check(A, W, C, 512, 73, "decode tile-major > 4 GB")
    # the last rows and columns are where 32-bit offsets would wrap
    tail = torch.arange(N - 64, N, device="cuda")
    y_ref = oracle.gemm_f64(A, host_bits(W[tail]))
    parity(C[:, N - 64:].cpu().numpy(), y_ref, "last 64 columns")
    C2 = torch.empty_like(C)
    tl.tl_gemm(dev_bf16(A), W, C2, M, N, K, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), tl.TL_FETCH_NATIVE)
    torch.cuda.synchronize()
    sampled_check(A, W, C2, 512, 74, "decode row-major > 4 GB")
    del C2
    # round trip and Eq. 2 placement of sampled elements
    back = torch.empty_like(W)
    tl.tl_unpack(Wt, back, N, K, 2, 4096, 32)
    assert torch.equal(back, W)
    del back
    rng = np.random.default_rng(75)
    rs, cs = rng.integers(0, N, 2048), rng.integers(0, K, 2048)
    rs[:8], cs[:8] = N - 1, K - 1 - np.arange(8)
    offs = np.array([oracle.tm_offset(int(r), int(c), K, 2, 4096, 32) // 2 for r, c in zip(rs, cs)])
    got = Wt.view(-1)[torch.from_numpy(offs).cuda()].view(torch.int16).cpu().numpy()
    want = W[torch.from_numpy(rs).cuda(), torch.from_numpy(cs).cuda()].view(torch.int16).cpu().numpy()
    assert np.array_equal(got, want)


def test_prefill_weight_just_below_4GB():
    import torch
    M, N, K = 256, 131072, 16320        # 2 * N * K = 4,278,190,080 < 2^32
    banner(f"large prefill M={M} N={N} K={K}")
    assert 2 * N * K < (1 << 32) <= 2 * N * (K + 64)
    W = device_weight(N, K, seed=81)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    A = synth.normal_bf16((M, K), seed=82)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), Wt, C, M, N, K, tl.layout(), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    sampled_check(A, W, C, 1024, 83, "prefill just below 4 GB")
    tail = torch.arange(N - 32, N, device="cuda")
    parity(C[:, N - 32:].cpu().numpy(), oracle.gemm_f64(A, host_bits(W[tail])), "last 32 columns")
