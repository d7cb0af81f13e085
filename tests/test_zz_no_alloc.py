"""resbm_encode_bwd_noalloc (the library's fixed device-resident scratch instead
of a caller workspace) against resbm_encode_bwd on the same inputs.

Both run the same kernels in the same order on the same partial-sum layout, so
every output must agree bit for bit.  Calls follow each other on one device
with a smaller input second (the scratch keeps the previous call's contents),
the headline shape is checked once, a HIP graph of the call is replayed, and
a call beyond the scratch's size is rejected before any work.
"""
import pytest
import torch

from gpu_helpers import lib, say
from paper_2604_11947_amd import inputs as I
from paper_2604_11947_amd import resbm as R

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20   # RESBM_NOALLOC_SCRATCH_BYTES in include/resbm.h


def case(T, n, r, seed, gx_mode):
    d = I.make_inputs(T, n, r, "student_t3", seed)
    g = {k: d[k].cuda() for k in ("z", "W_e")}
    g["a"] = (0.5 * I.make_bf16(T, r, seed + 1).float()).cuda()
    g["g_b"] = I.make_bf16(T, r, seed + 2, std=0.1).cuda()
    g["gx0"] = I.make_bf16(T, n, seed + 3, std=0.1).cuda()
    g["dW0"] = torch.randn(n, r, generator=torch.Generator().manual_seed(seed)).cuda()
    return g


def run(L, g, T, n, r, gx_mode, accumulate, noalloc):
    bf = torch.bfloat16
    g_z = torch.full((T, n), float("nan"), dtype=bf, device="cuda")
    g_x = {"separate": g["gx0"].clone(), "fused": g_z, "none": None}[gx_mode]
    dW = g["dW0"].clone() if accumulate else torch.full((n, r), float("nan"), device="cuda")
    if noalloc:
        L.encode_bwd_noalloc(g["z"], g["W_e"], g["a"], g["g_b"], g_z, dW, g_x=g_x, accumulate=accumulate)
    else:
        L.encode_bwd(g["z"], g["W_e"], g["a"], g["g_b"], g_z, dW, g_x=g_x, accumulate=accumulate)
    torch.cuda.synchronize()
    return g_z, dW, g_x


def same(a, b, name):
    assert a.shape == b.shape, name
    assert torch.equal(a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32),
                       b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)), f"{name} differs"


def compare(L, T, n, r, seed, gx_mode, accumulate):
    say(f"noalloc encode_bwd T={T} n={n} r={r} g_x={gx_mode} accumulate={accumulate}")
    g = case(T, n, r, seed, gx_mode)
    got = run(L, g, T, n, r, gx_mode, accumulate, noalloc=True)
    ref = run(L, g, T, n, r, gx_mode, accumulate, noalloc=False)
    same(got[0], ref[0], "g_z")
    same(got[1], ref[1], "dW_e")
    if gx_mode == "separate":
        same(got[2], ref[2], "g_x")
    assert not bool(torch.isnan(got[0].float()).any()), "g_z not fully written"


def test_noalloc_two_calls_second_smaller():
    L = lib()
    compare(L, 3000, 512, 40, 31, "separate", False)
    compare(L, 777, 256, 16, 32, "fused", True)


def test_noalloc_headline_shape():
    L = lib()
    compare(L, 16384, 4096, 32, 33, "none", False)
    compare(L, 1000, 4096, 32, 34, "separate", True)


def test_noalloc_graph_replay():
    """Captured in a HIP graph (after one eager call on the device) and replayed
    with eager work between the replays: every replay equals the eager result."""
    L = lib()
    T, n, r = 2048, 1024, 64
    say(f"noalloc encode_bwd graph replay T={T} n={n} r={r}")
    g = case(T, n, r, 35, "none")
    ref = run(L, g, T, n, r, "none", False, noalloc=True)
    g_z = torch.empty(T, n, dtype=torch.bfloat16, device="cuda")
    dW = torch.empty(n, r, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            L.encode_bwd_noalloc(g["z"], g["W_e"], g["a"], g["g_b"], g_z, dW)
    torch.cuda.synchronize()
    for rep in range(3):
        g_z.fill_(0.0)
        dW.fill_(float("nan"))
        run(L, case(600, 256, 8, 36 + rep, "fused"), 600, 256, 8, "fused", False, noalloc=True)
        graph.replay()
        torch.cuda.synchronize()
        same(g_z, ref[0], f"replay {rep}: g_z")
        same(dW, ref[1], f"replay {rep}: dW_e")


def test_noalloc_rejects_beyond_scratch():
    """n = 65536, r = 256 needs more than the fixed scratch: rejected by host
    validation before any HIP call (the addresses are never dereferenced)."""
    L = lib()
    T, n, r = 16384, 65536, 256
    need = L.workspace_bytes(T, n, r)
    assert need > SCRATCH_BYTES
    A = 0x10000000000
    st = L.cdll.resbm_encode_bwd_noalloc(T, n, r, R.ACT_SILU, A, n, 2 * A, 3 * A, 4 * A, 5 * A, n, None, 0,
                                         6 * A, 0, None)
    assert st == R.E_WORKSPACE
