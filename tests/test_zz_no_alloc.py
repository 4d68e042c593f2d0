"""tl_gemm_noalloc: the split-K partials in the library's static device
scratch instead of a per-stream workspace.  Two calls in a row (the second on
a smaller input, so it runs over what the first left in the scratch) must
equal tl_gemm's results on the same inputs bit for bit -- same plan, same
kernels, same fixed-order reduce -- and the fp64 oracle within the gate.
Covered plans: the streaming decode kernel with K splits, the LDS-staged
decode kernel with K splits, an FP8 weight with K splits, prefill without
scratch, prefill whose columns all run with a K split (medium M), and prefill
whose remaining columns run with a K split.  Errors: partials beyond the scratch, and the per-stream tally."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, dev_u8, host_f32, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def _bf16_case(M, N, K, seed):
    import torch
    A = synth.normal_bf16((M, K), seed=seed)
    W = synth.normal_bf16((N, K), seed=seed + 1, sigma=synth.W_SIGMA)
    Wd = dev_bf16(W)
    Wt = torch.empty_like(Wd)
    tl.tl_repack(Wd, Wt, N, K, 2, 4096, 32)
    return A, W, dev_bf16(A), Wt


def _both(A, Wt, M, N, K, d):
    """(tl_gemm's C, tl_gemm_noalloc's C) on the same inputs, outputs poisoned first."""
    import torch
    dt = torch.bfloat16 if d.out_dtype == tl.TL_OUT_BF16 else torch.float32
    C_ref = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    C_na = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    tl.tl_gemm(A, Wt, C_ref, M, N, K, d, tl.TL_FETCH_BLOCK)
    tl.tl_gemm_noalloc(A, Wt, C_na, M, N, K, d, tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    return C_ref, C_na


# (first call, second smaller call): M, N, K, split_k (0 = the library's plan)
CASES = [
    ("streaming decode, split-K", (8, 10240, 8192, 0), (5, 2048, 4096, 3)),
    ("LDS-staged decode, split-K", (32, 10240, 8192, 0), (20, 4096, 4096, 0)),
    ("LDS-staged decode with four M tiles, split-K", (64, 10240, 8192, 0), (40, 8192, 2048, 0)),
    ("prefill (no scratch), then split-K decode", (256, 1024, 512, 0), (3, 1024, 2048, 4)),
    ("prefill with K split over all columns, then split-K decode", (256, 1024, 2048, 0), (3, 1024, 2048, 4)),
    ("prefill with K-split remaining columns, then split-K decode", (2000, 10240, 2048, 0), (6, 4096, 4096, 2)),
]


@pytest.mark.parametrize("what,first,second", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_tl_gemm(what, first, second):
    for call, (M, N, K, S) in (("first", first), ("second", second)):
        d = tl.layout(split_k=S)
        plan = tl.tl_gemm_plan(M, N, K, d)
        banner(f"noalloc {what}, {call} call: M={M} N={N} K={K} plan={plan}")
        assert plan["workspace_bytes"] <= tl.TL_NOALLOC_SCRATCH_BYTES
        A_bits, W_bits, A, Wt = _bf16_case(M, N, K, seed=700 + M + N)
        C_ref, C_na = _both(A, Wt, M, N, K, d)
        assert np.array_equal(host_f32(C_na), host_f32(C_ref)), f"{what} {call}: differs from tl_gemm"
        parity(host_f32(C_na), oracle.gemm_f64(A_bits, W_bits), f"{what} {call}")
    # the plans the test names really use the scratch where they say so
    first_plan = tl.tl_gemm_plan(*first[:3], tl.layout(split_k=first[3]))
    assert (first_plan["workspace_bytes"] == 0) == ("no scratch" in what), first_plan


def test_noalloc_fp8_split_k_twice():
    import torch
    d = tl.layout(elem_bytes=1, G=4096, block_rows=64, split_k=4)
    for M, N, K in ((16, 4096, 8192), (7, 1024, 2048)):
        banner(f"noalloc fp8 split-K M={M} N={N} K={K}")
        A = synth.normal_bf16((M, K), seed=800 + M)
        W8, _ = synth.fp8_weights((N, K), seed=801 + M)
        W = dev_u8(W8)
        Wt = torch.empty_like(W)
        tl.tl_repack(W, Wt, N, K, 1, 4096, 64)
        C_ref, C_na = _both(dev_bf16(A), Wt, M, N, K, d)
        assert np.array_equal(host_f32(C_na), host_f32(C_ref))
        parity(host_f32(C_na), oracle.gemm_w8_f64(A, W8), f"fp8 M={M}")


def test_noalloc_bf16_out_twice():
    for M, N, K in ((24, 8192, 16384), (9, 2048, 4096)):
        d = tl.layout(split_k=4, out_dtype=tl.TL_OUT_BF16)
        banner(f"noalloc bf16 out split-K M={M} N={N} K={K}")
        _, _, A, Wt = _bf16_case(M, N, K, seed=900 + M)
        C_ref, C_na = _both(A, Wt, M, N, K, d)
        import torch
        assert torch.equal(C_na.view(torch.int16), C_ref.view(torch.int16))


def test_noalloc_rejections():
    """Partials beyond TL_NOALLOC_SCRATCH_BYTES -> TL_ESCRATCH; TL_FETCH_COUNT
    -> TL_EUNSUPPORTED; both before anything is enqueued (small buffers
    suffice: nothing is read or written)."""
    import torch
    banner("noalloc rejections")
    A = torch.zeros(64 * 16, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(64 * 16, dtype=torch.bfloat16, device="cuda")
    C = torch.zeros(64 * 16, dtype=torch.float32, device="cuda")
    d = tl.layout(split_k=16)
    M, N, K = 64, 32768, 65536                 # 16 splits x 64 x 32768 fp32 = 128 MiB of partials
    assert tl.tl_gemm_plan(M, N, K, d)["workspace_bytes"] > tl.TL_NOALLOC_SCRATCH_BYTES
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_noalloc(A, W, C, M, N, K, d, tl.TL_FETCH_BLOCK)
    assert e.value.status == tl.TL_ESCRATCH
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_noalloc(A, W, C, 8, 64, 64, tl.layout(), tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    assert e.value.status == tl.TL_EUNSUPPORTED
    torch.cuda.synchronize()
