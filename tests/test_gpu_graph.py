"""winograd_conv2d captured in a HIP graph (what ``bench.py --graph`` replays).

Each path is captured once and replayed several times, with eager work of the
program (the same convolution launched directly, a fill of the output) and a
synchronisation between replays; every replay must equal the eager result bit
for bit.  The kernels are deterministic, so any difference would come from
the capture (a node that does not replay like its eager launch).
"""
import pytest
import torch

from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

CASES = [
    # path, plan, m, dtype, (N, H, W, C, K)
    ("separate", WL.F4_LINEAR, 4, "f32", (2, 22, 19, 40, 48)),
    ("fused", WL.F4_A2P1, 4, "bf16", (2, 30, 26, 32, 40)),
    ("fused_input", WL.F4_A2P1, 4, "bf16", (2, 30, 26, 3, 64)),
]
TD = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@pytest.mark.parametrize("path,spec,m,dtype,shape", CASES, ids=[c[0] for c in CASES])
def test_graph_replays_match_eager(path, spec, m, dtype, shape):
    from paper_1905_05233_amd.winograd import Plan
    Nn, H, W, C, K = shape
    print(f"[graph] {path} {spec} m={m} {dtype} {shape}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(11)
    x = torch.randn(Nn, H, W, C, device="cuda", generator=g).abs().to(TD[dtype])
    w = (torch.randn(K, 3, 3, C, device="cuda", generator=g) * 0.1).to(TD[dtype])
    p = Plan(spec, m=m, dtype=dtype, path=path)
    try:
        y_eager = torch.empty(Nn, H, W, K, dtype=TD[dtype], device="cuda")
        y_graph = torch.empty_like(y_eager)
        eager = p.bind_call(x, w, y_eager)
        eager()
        torch.cuda.synchronize()
        ref = y_eager.clone()

        captured = p.bind_call(x, w, y_graph)   # same plan, same bound workspace
        captured()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            captured()
        for r in range(3):
            y_graph.fill_(float("nan"))
            y_eager.zero_()
            eager()
            torch.cuda.synchronize()
            assert torch.equal(y_eager, ref)
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(y_graph, ref), f"replay {r} differs from the eager result"
        del graph
    finally:
        p.close()
