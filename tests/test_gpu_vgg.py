"""The VGG-16-shaped stack (thirteen 3x3 layers, N = 32, fp16 and bf16, ReLU
and 2x2 max-pooling between stages, the most accurate candidate plan per
layer) at full size on the GPU.

Every layer is checked on its own GPU input:
  * one whole image per layer (a different image for each layer) against the
    oracle: rel-L2 against float64 direct convolution at most twice the
    oracle's same-algorithm, same-dtype error, and element by element within
    twice the a-priori rounding bound of the oracle's result;
  * whole output tiles sampled across the other images, tile rows, tile
    columns and all output channels against the float64 convolution, within
    the a-priori rounding bound of each tile.
The stack must also run deterministically and stay finite.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import elementwise_bound, sampled_tile_check, to_np
from oracle import conv as OC
from oracle import plan as OP

pytestmark = pytest.mark.gpu


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
    rng = np.random.default_rng(123)
    for li, (L, (xi, yi)) in enumerate(zip(stack.layers, trace)):
        spec = L["spec"]
        op = OP.build_plan(spec.moduli, n_o=spec.m, inner=spec.inner)
        w = to_np(L["w"]).astype(np.float32)
        # one whole image through the oracle
        n0 = li % N
        xa = to_np(xi[n0:n0 + 1])
        ya = to_np(yi[n0:n0 + 1]).astype(np.float64)
        y64 = OC.direct_f64(xa, w)
        yo = OC.winograd_emulated(xa, w, op, dtype)
        e_gpu, e_or = OC.rel_l2(ya, y64), OC.rel_l2(yo, y64)
        assert e_gpu <= 2 * e_or, (li, e_gpu, e_or)
        bound = elementwise_bound(xa, w, op, dtype, y64)
        assert np.all(np.abs(ya - yo) <= 2 * bound)
        # sampled tiles of other images, all output channels
        th = -(-L["hw"] // spec.m)
        tiles = [(int(rng.integers(N)), int(rng.integers(th)), int(rng.integers(th))) for _ in range(4)]
        tiles.append((N - 1, th - 1, th - 1))                      # the ragged corner
        worst = 0.0
        for n, ty, tx in tiles:
            xn = to_np(xi[n:n + 1]).astype(np.float64)
            yn = to_np(yi[n:n + 1]).astype(np.float64)
            worst = max(worst, sampled_tile_check(xn, w.astype(np.float64), yn, op, dtype, [(0, ty, tx)]))
        print(f"[vgg] layer {li} {L['hw']}x{L['hw']} {L['C']}->{L['K']} {{{spec.moduli}}}: "
              f"image {n0} err {e_gpu:.2e} (oracle {e_or:.2e}); sampled tiles error/bound {worst:.3f}", flush=True)
