"""GPU parity of tl_gemm_grouped (one launch over a stack of expert weights)
against the CPU oracle's grouped GEMM, through the C ABI: the full
Qwen-3-30B-A3B-shaped expert set under the seeded top-8 routing, and the
edge cases of the group tables (empty groups, groups larger than the M tile,
identity rows, ids and offsets outside range, which the kernel clamps)."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_bits, host_f32, parity, parity_bf16_out

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def stacked_tile_major(Ws, G=4096, br=32):
    """Upload row-major expert weights and repack each into one stacked buffer."""
    import torch
    N, K = Ws[0].shape
    stack = torch.empty((len(Ws), N, K), dtype=torch.bfloat16, device="cuda")
    for e, W in enumerate(Ws):
        tl.tl_repack(dev_bf16(W), stack[e], N, K, 2, G, br)
    return stack


def run_grouped(A_bits, ids, offsets, Ws, max_rows, desc=None, total_rows=None, fetch=tl.TL_FETCH_BLOCK,
                stack=None):
    import torch
    desc = desc or tl.layout()
    E = len(Ws)
    N, K = Ws[0].shape
    T = int(offsets[-1]) if total_rows is None else total_rows
    stack = stacked_tile_major(Ws, desc.G, desc.block_rows) if stack is None else stack
    A = dev_bf16(A_bits)
    C = torch.full((max(T, 1), N), float("nan"), dtype=torch.float32, device="cuda")
    d_ids = None if ids is None else dev_i32(ids)
    tl.tl_gemm_grouped(A, A_bits.shape[0], d_ids, dev_i32(offsets), E, T, max_rows, stack, N * K * 2, C,
                       N, K, desc, fetch)
    torch.cuda.synchronize()
    return C[:T]


@pytest.mark.parametrize("proj", ["gate_up", "down"])
def test_qwen_moe_experts_full(proj):
    """All 128 experts, 64 tokens, top-8: 512 rows, every row against the oracle."""
    routing = synth.moe_routing()
    offsets, ids = synth.moe_tables(routing)
    max_rows = int(np.diff(offsets).max())
    if proj == "gate_up":
        N, K = synth.QWEN_GATE_UP
        A = synth.normal_bf16((synth.QWEN_TOKENS, K), seed=synth.QWEN_SEED_HIDDEN)
        seeds = [synth.qwen_gate_up_seed(e) for e in range(synth.QWEN_EXPERTS)]
        tok = ids
    else:
        N, K = synth.QWEN_DOWN
        A = synth.normal_bf16((int(offsets[-1]), K), seed=synth.QWEN_SEED_DOWN_IN)
        seeds = [synth.qwen_down_seed(e) for e in range(synth.QWEN_EXPERTS)]
        tok = None                                   # row r of the down input is row r
    banner(f"grouped moe {proj}: E=128 rows={offsets[-1]} max_rows={max_rows} N={N} K={K}")
    Ws = [synth.normal_bf16((N, K), seed=s, sigma=synth.W_SIGMA) for s in seeds]
    C = run_grouped(A, tok, offsets, Ws, max_rows)
    parity(host_f32(C), oracle.grouped_gemm_f64(A, tok, offsets, Ws), f"grouped {proj}")


@pytest.mark.parametrize("max_rows", [16, 32, 64])
def test_grouped_edge_groups(max_rows):
    """Empty first, middle and last groups; a 40-row group (several passes when
    the M tile is 16 or 32 rows); ids that repeat across groups."""
    N, K = 256, 512
    counts = [0, 3, 40, 0, 1, 17, 0]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    rng = np.random.default_rng(7)
    ids = rng.integers(0, 24, size=T).astype(np.int32)
    A = synth.normal_bf16((24, K), seed=8)
    Ws = [synth.normal_bf16((N, K), seed=60 + e, sigma=synth.W_SIGMA) for e in range(len(counts))]
    banner(f"grouped edges max_rows={max_rows} T={T}")
    C = run_grouped(A, ids, offsets, Ws, max_rows)
    parity(host_f32(C), oracle.grouped_gemm_f64(A, ids, offsets, Ws), f"edges max_rows={max_rows}")


def test_grouped_small_integers_exact_and_identity_rows():
    N, K = 128, 1024
    counts = [5, 0, 12, 33]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    A = synth.small_int_bf16((T, K), seed=11)
    Ws = [synth.small_int_bf16((N, K), seed=70 + e) for e in range(len(counts))]
    banner(f"grouped small integers identity T={T}")
    C = run_grouped(A, None, offsets, Ws, 16)
    assert np.array_equal(host_f32(C).astype(np.float64), oracle.grouped_gemm_f64(A, None, offsets, Ws))


def test_grouped_row_major_weights():
    """Plain row-major expert weights (no repack), native fetch."""
    import torch
    N, K = 192, 256
    counts = [2, 7, 0, 4]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    ids = np.arange(T, dtype=np.int32)[::-1].copy()
    A = synth.normal_bf16((T, K), seed=12)
    Ws = [synth.normal_bf16((N, K), seed=80 + e, sigma=synth.W_SIGMA) for e in range(len(counts))]
    stack = torch.stack([dev_bf16(W) for W in Ws]).contiguous()
    banner("grouped row-major weights")
    C = run_grouped(A, ids, offsets, Ws, 8, desc=tl.layout(kind=tl.TL_LAYOUT_NK_ROW),
                    fetch=tl.TL_FETCH_NATIVE, stack=stack)
    parity(host_f32(C), oracle.grouped_gemm_f64(A, ids, offsets, Ws), "grouped row-major")


def test_grouped_out_of_range_ids_and_offsets_are_clamped():
    """Token ids outside [0, a_rows) read zeros; offsets past total_rows are
    clamped, so the rows past it are neither computed nor written."""
    import torch
    N, K = 64, 256
    offsets = np.array([0, 4, 9, 14], dtype=np.int32)        # last group claims rows up to 14
    T = 11                                                      # but C has 11 rows
    ids = np.array([0, 1, -3, 2, 5, 99, 3, 4, 6, 7, 2], dtype=np.int32)
    A = synth.normal_bf16((8, K), seed=13)
    Ws = [synth.normal_bf16((N, K), seed=90 + e, sigma=synth.W_SIGMA) for e in range(3)]
    banner("grouped clamped ids / offsets")
    stack = stacked_tile_major(Ws)
    Cbig = torch.full((T + 5, N), float("nan"), dtype=torch.float32, device="cuda")
    tl.tl_gemm_grouped(dev_bf16(A), 8, dev_i32(ids), dev_i32(offsets), 3, T, 8, stack, N * K * 2, Cbig,
                       N, K, tl.layout(), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    got = host_f32(Cbig)
    assert np.all(np.isnan(got[T:])), "rows past total_rows were written"
    A_ext = np.concatenate([A, np.zeros((1, K), dtype=np.uint16)])   # row 8 = zeros
    ids_ext = np.where((ids >= 0) & (ids < 8), ids, 8)
    clamped = np.minimum(offsets, T)
    want = oracle.grouped_gemm_f64(A_ext, ids_ext, clamped, Ws)
    parity(got[:T], want, "clamped")
    assert np.all(got[2] == 0.0) and np.all(got[5] == 0.0)


def test_grouped_fetch_counter():
    """The tally equals the weight bytes streamed: once per non-empty group and
    M-tile pass."""
    N, K = 256, 512
    counts = [3, 0, 20, 1]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    A = synth.normal_bf16((T, K), seed=14)
    Ws = [synth.normal_bf16((N, K), seed=100 + e, sigma=synth.W_SIGMA) for e in range(4)]
    banner("grouped fetch counter")
    tl.tl_fetch_counter_read()
    C = run_grouped(A, None, offsets, Ws, 16, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    passes = sum(-(-c // 16) for c in counts)
    assert got == passes * N * K * 2
    parity(host_f32(C), oracle.grouped_gemm_f64(A, None, offsets, Ws), "counted")


def test_grouped_graph_replay():
    import torch
    N, K = 512, 1024
    routing = synth.moe_routing(M=16, E=8, topk=2, seed=3)
    offsets, ids = synth.moe_tables(routing, E=8)
    T = int(offsets[-1])
    A = synth.normal_bf16((16, K), seed=15)
    Ws = [synth.normal_bf16((N, K), seed=110 + e, sigma=synth.W_SIGMA) for e in range(8)]
    banner("grouped graph replay")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        stack = stacked_tile_major(Ws)
        dA, dids, doff = dev_bf16(A), dev_i32(ids), dev_i32(offsets)
        C = torch.zeros((T, N), dtype=torch.float32, device="cuda")
        args = (dA, 16, dids, doff, 8, T, int(np.diff(offsets).max()), stack, N * K * 2, C, N, K, tl.layout(),
                tl.TL_FETCH_BLOCK)
        tl.tl_gemm_grouped(*args)
        side.synchronize()
        eager = C.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            tl.tl_gemm_grouped(*args)
        for rep in range(4):
            C.fill_(float("nan"))
            side.synchronize()
            g.replay()
            side.synchronize()
            assert torch.equal(C, eager), f"replay {rep}"
    parity(host_f32(eager), oracle.grouped_gemm_f64(A, ids, offsets, Ws), "graph")


# ---------------------------------------------------------------------------
# Gated expert activation fused into the gate+up projection
# ---------------------------------------------------------------------------

def run_swiglu(A_bits, ids, offsets, Ws, max_rows, desc=None, fetch=tl.TL_FETCH_BLOCK, stack=None):
    """Ws: stacked [2I, K] gate+up weights per group -> H [T, I] from tl_gemm_grouped_swiglu."""
    import torch
    desc = desc or tl.layout()
    E = len(Ws)
    I2, K = Ws[0].shape
    I = I2 // 2
    T = int(offsets[-1])
    stride = tl.tl_tile_bytes(I2, K, 2, desc.G, desc.block_rows) if desc.kind == tl.TL_LAYOUT_TILE else I2 * K * 2
    if stack is None:
        stack = torch.empty((E * stride // 2,), dtype=torch.bfloat16, device="cuda")
        for e, W in enumerate(Ws):
            seg = stack[e * stride // 2:(e + 1) * stride // 2]
            if desc.kind == tl.TL_LAYOUT_TILE:
                tl.tl_repack(dev_bf16(W), seg, I2, K, 2, desc.G, desc.block_rows)
            else:
                seg.copy_(dev_bf16(W).view(-1))
    out_dt = torch.bfloat16 if desc.out_dtype == tl.TL_OUT_BF16 else torch.float32
    H = torch.full((max(T, 1), I), float("nan"), dtype=out_dt, device="cuda")
    d_ids = None if ids is None else dev_i32(ids)
    tl.tl_gemm_grouped_swiglu(dev_bf16(A_bits), A_bits.shape[0], d_ids, dev_i32(offsets), E, T, max_rows, stack,
                              stride, H, I, K, desc, fetch)
    torch.cuda.synchronize()
    return H[:T]


def test_swiglu_qwen_moe_experts_full():
    """All 128 Qwen experts' gate+up [1536, 2048] as gate [768] + up [768]:
    the fused activation of every routed row against the oracle."""
    routing = synth.moe_routing()
    offsets, ids = synth.moe_tables(routing)
    max_rows = int(np.diff(offsets).max())
    N2, K = synth.QWEN_GATE_UP
    A = synth.normal_bf16((synth.QWEN_TOKENS, K), seed=synth.QWEN_SEED_HIDDEN)
    Ws = [synth.normal_bf16((N2, K), seed=synth.qwen_gate_up_seed(e), sigma=synth.W_SIGMA)
          for e in range(synth.QWEN_EXPERTS)]
    banner(f"grouped swiglu qwen: E=128 rows={offsets[-1]} I={N2 // 2} K={K}")
    H = run_swiglu(A, ids, offsets, Ws, max_rows)
    parity(host_f32(H), oracle.grouped_swiglu_f64(A, ids, offsets, Ws), "swiglu qwen")
    Hb = run_swiglu(A, ids, offsets, Ws, max_rows, desc=tl.layout(out_dtype=tl.TL_OUT_BF16))
    parity_bf16_out(host_bits(Hb), oracle.grouped_swiglu_f64(A, ids, offsets, Ws), "swiglu qwen bf16")


@pytest.mark.parametrize("max_rows", [16, 64])
@pytest.mark.parametrize("G,br", [(4096, 32), (4096, 16), (1024, 8)])
def test_swiglu_edge_groups_and_memory_tiles(max_rows, G, br):
    """Empty groups, a 40-row group (passes of the M tile), repeated ids,
    memory tiles of 32, 16 and 8 rows, a K that is not a multiple of 64."""
    I, K = 96, 520
    counts = [0, 3, 40, 0, 1, 17, 0]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    ids = np.random.default_rng(9).integers(0, 24, size=T).astype(np.int32)
    A = synth.normal_bf16((24, K), seed=10)
    Ws = [synth.normal_bf16((2 * I, K), seed=120 + e, sigma=synth.W_SIGMA * 10) for e in range(len(counts))]
    banner(f"grouped swiglu edges max_rows={max_rows} G={G} br={br}")
    H = run_swiglu(A, ids, offsets, Ws, max_rows, desc=tl.layout(G=G, block_rows=br))
    parity(host_f32(H), oracle.grouped_swiglu_f64(A, ids, offsets, Ws), f"swiglu G={G} br={br}")


def test_swiglu_row_major_and_rejections():
    import torch
    I, K = 64, 256
    counts = [2, 5, 0, 3]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    T = int(offsets[-1])
    A = synth.normal_bf16((T, K), seed=16)
    Ws = [synth.normal_bf16((2 * I, K), seed=130 + e, sigma=synth.W_SIGMA * 10) for e in range(len(counts))]
    banner("grouped swiglu row-major")
    H = run_swiglu(A, None, offsets, Ws, 8, desc=tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch=tl.TL_FETCH_NATIVE)
    parity(host_f32(H), oracle.grouped_swiglu_f64(A, None, offsets, Ws), "swiglu row-major")
    stack = torch.zeros((4, 2 * 64, K), dtype=torch.bfloat16, device="cuda")   # as large as the calls describe
    Hs = torch.zeros((T, 64), dtype=torch.float32, device="cuda")
    for kw, status in ((dict(I=48), tl.TL_EUNSUPPORTED),                               # I % 32
                       (dict(desc=tl.layout(block_rows=64)), tl.TL_EUNSUPPORTED)):     # 64-row memory tiles
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_grouped_swiglu(dev_bf16(A), T, None, dev_i32(offsets), 4, T, 8, stack, 2 * 64 * K * 2, Hs,
                                      kw.get("I", 64), K, kw.get("desc", tl.layout()), tl.TL_FETCH_BLOCK)
        assert e.value.status == status


def test_swiglu_graph_replay():
    import torch
    I, K = 128, 1024
    routing = synth.moe_routing(M=16, E=8, topk=2, seed=4)
    offsets, ids = synth.moe_tables(routing, E=8)
    T = int(offsets[-1])
    A = synth.normal_bf16((16, K), seed=17)
    Ws = [synth.normal_bf16((2 * I, K), seed=140 + e, sigma=synth.W_SIGMA) for e in range(8)]
    banner("grouped swiglu graph replay")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        stack = torch.empty((8, 2 * I, K), dtype=torch.bfloat16, device="cuda")
        for e, W in enumerate(Ws):
            tl.tl_repack(dev_bf16(W), stack[e], 2 * I, K, 2, 4096, 32)
        dA, dids, doff = dev_bf16(A), dev_i32(ids), dev_i32(offsets)
        H = torch.zeros((T, I), dtype=torch.float32, device="cuda")
        args = (dA, 16, dids, doff, 8, T, int(np.diff(offsets).max()), stack, 2 * I * K * 2, H, I, K, tl.layout(),
                tl.TL_FETCH_BLOCK)
        tl.tl_gemm_grouped_swiglu(*args)
        side.synchronize()
        eager = H.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            tl.tl_gemm_grouped_swiglu(*args)
        for rep in range(4):
            H.fill_(float("nan"))
            side.synchronize()
            g.replay()
            side.synchronize()
            assert torch.equal(H, eager), f"replay {rep}"
    parity(host_f32(eager), oracle.grouped_swiglu_f64(A, ids, offsets, Ws), "swiglu graph")
