"""The VGG-16-shaped stack (thirteen 3x3 layers, N = 32, fp16 and bf16, ReLU
and 2x2 max-pooling between stages, the most accurate candidate plan per
layer) at full size on the GPU.

Every layer is checked on its own GPU input:
  * the transforms at the full batch (the launch conv2d makes, including
    the instance whose workgroups walk several tiles on the large layers):
    U, and V of two images (one per layer in turn, and the last image of the
    batch), equal to the oracle's bit for bit;
  * those two images' outputs element by element within ``pair_bound`` of the
    oracle's same-algorithm result (about one unit in the last place of y),
    and their rel-L2 error against float64 direct convolution at most
    min(2 x the oracle's, 5e-2).
The stack must also run deterministically and stay finite.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_against_oracle, stages_on_device_layout, to_np
from oracle import conv as OC
from oracle import plan as OP

pytestmark = pytest.mark.gpu

CAP = 5e-2


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_vgg_stack_parity(dtype):
    from paper_1905_05233_amd.vgg import VggStack
    N = 32
    stack = VggStack(dtype)
    print(f"[vgg] {dtype} plans: " + "; ".join(stack.summary()), flush=True)
    x = stack.input(N)
    out, trace = stack.forward(x, keep=True)
    out2 = stack.forward(x)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    assert bool(torch.isfinite(out.float()).all())
    for li, (L, (xi, yi)) in enumerate(zip(stack.layers, trace)):
        spec, p = L["spec"], L["plan"]
        op = OP.build_plan(spec.moduli, n_o=spec.m, inner=spec.inner)
        hw, C, K = L["hw"], L["C"], L["K"]
        w = to_np(L["w"]).astype(np.float32)
        Ug, Vg = p.kernel_input_transform(L["w"], xi)
        per = (-(-hw // spec.m)) ** 2                     # tiles per image
        Ug = to_np(Ug)[:, :, :C]
        for n0 in sorted({li % N, N - 1}):
            xa = to_np(xi[n0:n0 + 1])
            ya = to_np(yi[n0:n0 + 1]).astype(np.float64)
            st = OC.winograd_emulated_stages(xa, w, op, dtype)
            Uo, Vo = stages_on_device_layout(st)
            assert np.array_equal(Ug, Uo), (li, "U")
            assert np.array_equal(to_np(Vg[:, n0 * per:(n0 + 1) * per, :C]), Vo), (li, n0, "V")
            check_against_oracle(ya, st, op, dtype, hw, hw, label=f"layer {li} image {n0}")
            y64 = OC.direct_f64(xa, w)
            e_gpu, e_or = OC.rel_l2(ya, y64), OC.rel_l2(st["y"], y64)
            print(f"[vgg] layer {li} {hw}x{hw} {C}->{K} {{{spec.moduli}}} path {p.conv_path(N, hw, hw, C, K)}: "
                  f"image {n0} err {e_gpu:.2e} (oracle {e_or:.2e})", flush=True)
            assert e_gpu <= min(2 * e_or, CAP), (li, n0, e_gpu, e_or)
        del Vg
