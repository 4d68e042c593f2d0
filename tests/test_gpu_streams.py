"""Library state per (device, stream): split-K calls from several host threads,
each on its own stream with its own workspace, run concurrently and give the
results of the same calls made alone; tl_release frees that state and the
next call re-creates it."""
import threading

import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_f32, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def _case(i):
    M, N, K = [(8, 1024, 4096), (32, 8192, 8192), (1, 512, 8192), (17, 2048, 4096)][i % 4]
    A = synth.normal_bf16((M, K), seed=500 + i)
    W = synth.normal_bf16((N, K), seed=600 + i, sigma=synth.W_SIGMA)
    return M, N, K, A, W


def test_threads_on_separate_streams():
    import torch
    banner("split-K calls from 4 host threads on 4 streams")
    cases = [_case(i) for i in range(4)]
    dev = []
    for (M, N, K, A, W) in cases:
        Wd = dev_bf16(W)
        Wt = torch.empty_like(Wd)
        tl.tl_repack(Wd, Wt, N, K, 2, 4096, 32)
        dev.append((dev_bf16(A), Wt))
    torch.cuda.synchronize()
    want = [oracle.gemm_f64(A, W) for (_, _, _, A, W) in cases]
    outs = [None] * 4
    errors = []

    def worker(i):
        try:
            M, N, K, _, _ = cases[i]
            A, Wt = dev[i]
            s = torch.cuda.Stream()
            C = torch.empty((M, N), dtype=torch.float32, device="cuda")
            with torch.cuda.stream(s):
                for _ in range(20):                     # repeated: the workspace is reused on its stream
                    tl.tl_gemm(A, Wt, C, M, N, K, tl.layout(split_k=4), tl.TL_FETCH_BLOCK, stream=s)
            s.synchronize()
            outs[i] = host_f32(C)
        except Exception as e:                          # reported on the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i in range(4):
        parity(outs[i], want[i], f"thread {i}")


def test_release_then_reuse():
    import torch
    banner("tl_release, then a split-K call re-creates the state")
    M, N, K, A, W = _case(0)
    Wd = dev_bf16(W)
    Wt = torch.empty_like(Wd)
    tl.tl_repack(Wd, Wt, N, K, 2, 4096, 32)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), Wt, C, M, N, K, tl.layout(split_k=4), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    first = host_f32(C)
    tl.tl_release()
    C2 = torch.empty_like(C)
    tl.tl_gemm(dev_bf16(A), Wt, C2, M, N, K, tl.layout(split_k=4), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    assert np.array_equal(host_f32(C2), first)
    parity(first, oracle.gemm_f64(A, W), "after release")


def test_graph_replay_after_workspace_growth():
    """A graph captured while the stream's split-K workspace was small keeps
    working after a later eager call grows the workspace: the old buffer is
    retired, not freed, so the graph's kernels still write valid memory.
    Every replay (with eager split-K work on the grown workspace between the
    replays) equals the eager result of the captured call."""
    import torch
    banner("capture split-K on a small workspace, grow it eagerly, replay")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        tl.tl_release()                                   # start from no state on any stream
        small = _case(0)                                  # M=8, N=1024, K=4096: 128 KiB of partials
        big = _case(1)                                    # M=32, N=8192, K=8192: 4 MiB at split_k 4
        dev = []
        for (M, N, K, A, W) in (small, big):
            Wd = dev_bf16(W)
            Wt = torch.empty_like(Wd)
            tl.tl_repack(Wd, Wt, N, K, 2, 4096, 32)
            dev.append((dev_bf16(A), Wt, torch.zeros((M, N), dtype=torch.float32, device="cuda")))
        d = tl.layout(split_k=4)
        (Ms, Ns, Ks, As, Ws), (Mb, Nb, Kb, Ab, Wb) = small, big
        (A0, W0, C0), (A1, W1, C1) = dev
        tl.tl_gemm(A0, W0, C0, Ms, Ns, Ks, d, tl.TL_FETCH_BLOCK)      # creates the small workspace
        side.synchronize()
        eager_small = C0.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            tl.tl_gemm(A0, W0, C0, Ms, Ns, Ks, d, tl.TL_FETCH_BLOCK)
        assert tl.tl_gemm_plan(Mb, Nb, Kb, d)["workspace_bytes"] > (1 << 20)
        tl.tl_gemm(A1, W1, C1, Mb, Nb, Kb, d, tl.TL_FETCH_BLOCK)      # grows the workspace
        side.synchronize()
        eager_big = C1.clone()
        for rep in range(4):
            C0.fill_(float("nan"))
            side.synchronize()
            g.replay()
            side.synchronize()
            assert torch.equal(C0, eager_small), f"replay {rep}"
            tl.tl_gemm(A1, W1, C1, Mb, Nb, Kb, d, tl.TL_FETCH_BLOCK)  # eager work on the new workspace
            side.synchronize()
            assert torch.equal(C1, eager_big), f"eager call after replay {rep}"
        del g
    parity(host_f32(eager_small), oracle.gemm_f64(As, Ws), "captured call")
    parity(host_f32(eager_big), oracle.gemm_f64(Ab, Wb), "growing call")


def test_prefill_ksplit_on_separate_streams():
    """The prefill plan whose columns past the whole rounds split K (fp32
    partials in the calling stream's workspace, then the split-order reduce):
    three host threads, each on its own stream, run it repeatedly at the same
    time; every result equals the call made alone bit for bit (fp32 and bf16
    out), and that result meets the oracle."""
    import torch
    M, N, K = 2000, 12288, 1024
    banner("prefill K-split plan from 3 host threads on 3 streams")
    A = synth.normal_bf16((M, K), seed=700)
    W = synth.normal_bf16((N, K), seed=701, sigma=synth.W_SIGMA)
    Ad = dev_bf16(A)
    Wd = dev_bf16(W)
    Wt = torch.empty_like(Wd)
    tl.tl_repack(Wd, Wt, N, K, 2, 4096, 32)
    y_ref = oracle.gemm_f64(A, W)
    for out, dt in ((tl.TL_OUT_F32, torch.float32), (tl.TL_OUT_BF16, torch.bfloat16)):
        d = tl.layout(out_dtype=out)
        plan = tl.tl_gemm_plan(M, N, K, d)
        assert plan["split_k"] == 2 and plan["workspace_bytes"] > 0, plan
        alone = torch.empty((M, N), dtype=dt, device="cuda")
        tl.tl_gemm(Ad, Wt, alone, M, N, K, d, tl.TL_FETCH_BLOCK)
        torch.cuda.synchronize()
        alone = alone.view(torch.int16 if out == tl.TL_OUT_BF16 else torch.int32).cpu().numpy()
        if out == tl.TL_OUT_F32:
            parity(alone.view(np.float32), y_ref, "K-split plan alone")
        outs = [None] * 3
        errors = []

        def worker(i):
            try:
                s = torch.cuda.Stream()
                C = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
                with torch.cuda.stream(s):
                    for _ in range(5):
                        tl.tl_gemm(Ad, Wt, C, M, N, K, d, tl.TL_FETCH_BLOCK, stream=s)
                s.synchronize()
                outs[i] = C.view(torch.int16 if out == tl.TL_OUT_BF16 else torch.int32).cpu().numpy()
            except Exception as e:                      # reported on the main thread
                errors.append(e)

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(3)]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        assert not errors, errors
        for i in range(3):
            assert np.array_equal(outs[i], alone), (out, i)
