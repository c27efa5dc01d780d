"""The VGG-16-shaped stack of thirteen 3x3 convolutions on the library.

The paper's CNN experiments (Section 3.2, Tables 2 and 3) run VGG-16; here the stack has VGG-16's
layer shapes with seeded random weights (N(0, 2/(9C)), seed 1 + layer) and a
seeded half-normal input, and each layer uses the Winograd plan chosen for it
from a candidate list (most accurate by default, see ``search.best_plan``).
Between layers: ReLU, and 2x2 stride-2 max-pooling after the last layer of
each stage.  The convolutions run through the library's kernels; the ReLU and
pooling between them are plain tensor operations on the device (they are not
part of the Winograd path and are excluded from the timed convolutions).
"""
import numpy as np
import torch

from . import search
from .winograd import Plan
from .workloads import VGG16_LAYERS, VGG_CANDIDATES, vgg_input, vgg_layer_weights

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def relu_pool(y, pool):
    """ReLU, then 2x2/2 max-pooling on NHWC if ``pool``."""
    y = torch.relu(y)
    if pool:
        N, H, W, C = y.shape
        y = y.view(N, H // 2, 2, W // 2, 2, C).amax(dim=(2, 4))
    return y.contiguous()


class VggStack:
    """Thirteen conv layers with their weights resident on the device."""

    def __init__(self, dtype="bf16", plans=None, policy="accuracy", cap=None, device="cuda"):
        self.dtype = dtype
        self.tdt = TORCH_DTYPES[dtype]
        self.layers = []
        for i, (hw, C, K, pool) in enumerate(VGG16_LAYERS):
            w = torch.from_numpy(vgg_layer_weights(i, C, K)).to(device).to(self.tdt)
            if plans is not None:
                spec = plans[i]
            else:
                spec, _ = search.best_plan(hw, hw, C, K, dtype, VGG_CANDIDATES, policy=policy, cap=cap)
            plan = Plan(spec.moduli, m=spec.m, dtype=dtype, inner=spec.inner)
            self.layers.append({"hw": hw, "C": C, "K": K, "pool": pool, "w": w, "spec": spec, "plan": plan})

    def input(self, N, seed=0, device="cuda"):
        return torch.from_numpy(vgg_input(N, seed)).to(device).to(self.tdt)

    def direct_flops(self, N):
        return sum(2 * N * L["hw"] * L["hw"] * L["C"] * L["K"] * 9 for L in self.layers)

    def forward(self, x, keep=False):
        """Run the stack; with ``keep`` also return every layer's (input, raw conv output)."""
        trace = []
        for L in self.layers:
            y = L["plan"].conv2d(x, L["w"])
            if keep:
                trace.append((x, y))
            x = relu_pool(y, L["pool"])
        return (x, trace) if keep else x

    def timed_forward(self, x):
        """One pass with HIP events around each convolution; returns (output, conv ms per layer)."""
        ev = []
        stream = torch.cuda.current_stream()
        for L in self.layers:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            y = L["plan"].conv2d(x, L["w"])
            e1.record(stream)
            ev.append((e0, e1))
            x = relu_pool(y, L["pool"])
        torch.cuda.synchronize()
        return x, [a.elapsed_time(b) for a, b in ev]

    def summary(self):
        return [f"{L['hw']}x{L['hw']} {L['C']}->{L['K']}: {{{L['spec'].moduli}}} m={L['spec'].m}"
                for L in self.layers]
