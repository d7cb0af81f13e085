"""The four boundary ops captured in one HIP graph replay exactly like eager launches.

The graph is replayed several times with unrelated eager work (the outputs
overwritten) and synchronizations in between; every replay must reproduce the
eager outputs bit for bit (the kernels add every partial sum in a fixed order,
so results do not depend on scheduling).
"""
import pytest
import torch

from gpu_helpers import lib, say
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [(1000, 512, 32), (333, 320, 40)], ids=["T1000_n512_r32", "T333_n320_r40"])
def test_graph_replay_matches_eager(shape):
    T, n, r = shape
    say(f"graph replay T={T} n={n} r={r}")
    L = lib()
    d = I.make_inputs(T, n, r, "normal", 3)
    g = {k: d[k].cuda() for k in ("x_attn", "z", "W_e", "W_d", "g_zt", "g_id")}
    io = L.io_dtype
    out = {
        "b": torch.empty(T, r, dtype=io, device="cuda"), "a": torch.empty(T, r, device="cuda"),
        "zt": torch.empty(T, n, dtype=io, device="cuda"), "gb": torch.empty(T, r, dtype=io, device="cuda"),
        "gz": torch.empty(T, n, dtype=io, device="cuda"), "dWd": torch.empty(r, n, device="cuda"),
        "dWe": torch.empty(n, r, device="cuda"),
    }
    ws = L.workspace(T, n, r, "cuda")

    def step():
        L.encode_fwd(g["x_attn"], g["z"], g["W_e"], out["b"], out["a"], ws=ws)
        L.decode_fwd(out["b"], g["W_d"], out["zt"], ws=ws)
        L.decode_bwd(out["b"], g["W_d"], g["g_zt"], g["g_id"], out["gb"], out["dWd"], ws=ws)
        L.encode_bwd(g["z"], g["W_e"], out["a"], out["gb"], out["gz"], out["dWe"], ws=ws)

    step()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan"))          # eager work between replays
        ws.fill_(0x5A)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert torch.equal(v.view(torch.uint8), ref[k].view(torch.uint8)), f"replay {rep}: {k} differs"
