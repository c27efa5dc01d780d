"""winograd_conv2d_static, the entry point that allocates nothing (its
workspace is the library's per-GPU device array), against winograd_conv2d
with a bound workspace: the same plan, path and kernels, so the outputs are
equal bit for bit.  Two calls in a row per case, the second on a smaller
layer (the array keeps the first call's contents), on the separate and the
fused path; a layer whose workspace exceeds the array is rejected before
anything is launched."""
import pytest
import torch

from gpu_helpers import to_dev
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

CASES = [
    (WL.F4_LINEAR, 4, "f32", "separate", (8, 56, 56, 128, 128), (1, 13, 11, 24, 40)),   # 60 MB: the array's largest use
    (WL.F4_A2P1, 4, "bf16", "fused", (4, 56, 56, 64, 64), (1, 20, 18, 40, 52)),
    (WL.F6_TWO_QUAD, 6, "f16", "separate", (2, 28, 28, 96, 80), (1, 9, 7, 5, 3)),
]


def _layer(shape, dtype, seed):
    N, H, W, C, K = shape
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=seed)
    return to_dev(x, dtype), to_dev(w, dtype)


@pytest.mark.parametrize("spec,m,dtype,path,big,small", CASES, ids=[f"{c[2]}-{c[3]}" for c in CASES])
def test_static_workspace_matches_bound_workspace(spec, m, dtype, path, big, small):
    from paper_1905_05233_amd.winograd import Plan
    p = Plan(spec, m=m, dtype=dtype, path=path)
    for i, shape in enumerate((big, small)):
        N, H, W, C, K = shape
        print(f"[no-alloc] {spec} {dtype} {path} call {i} shape {shape}", flush=True)
        assert p.conv_path(N, H, W, C, K) == path
        assert p.workspace_bytes(N, H, W, C, K) <= 64 << 20
        x, w = _layer(shape, dtype, seed=i + C)
        y_ref = p.conv2d(x, w)
        y = torch.empty_like(y_ref)
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        p.conv2d_static(x, w, y)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        assert torch.equal(y, y_ref)


def test_static_workspace_rejects_large_layers():
    from paper_1905_05233_amd._native import WinogradError
    from paper_1905_05233_amd.winograd import Plan
    p = Plan(WL.F6_TWO_QUAD, m=6, dtype="bf16")
    shape = (16, 28, 28, 256, 256)                     # alpha' = 10: 74.5 MB of workspace
    assert p.workspace_bytes(*shape) > 64 << 20
    x, w = _layer(shape, "bf16", seed=1)
    y = torch.zeros((16, 28, 28, 256), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(WinogradError, match="WORKSPACE"):
        p.conv2d_static(x, w, y)
    torch.cuda.synchronize()
    assert bool((y == 0).all())                        # nothing ran
