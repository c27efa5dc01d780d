"""The VGG-16-shaped stack of thirteen 3x3 convolutions on the library.

The paper's CNN experiments (Section 3.2, Tables 2 and 3) run VGG-16; here
the stack has VGG-16's layer shapes with seeded random weights (N(0, 2/(9C)),
seed 1 + layer) and a seeded half-normal input.  Each layer's Winograd plan
is chosen from a candidate list on that layer's own input: the first images
of the batch are run through the stack once, and at every layer the most
accurate candidate against float64 direct convolution of those images is
kept (``search.best_plan``).  Between layers: ReLU, and 2x2 stride-2
max-pooling after the last layer of each stage.  The convolutions, and the
ReLU and pooling between them, run in the library's kernels (the ReLU and
pooling are not part of the Winograd path and are timed apart from the
convolutions).
"""
import torch

from . import search
from .layer_ops import relu_pool as _relu_pool
from .winograd import Plan
from .workloads import VGG16_LAYERS, VGG_CANDIDATES, vgg_input, vgg_layer_weights

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def relu_pool(y, pool):
    """ReLU, then 2x2/2 max-pooling on NHWC if ``pool`` (one HIP kernel)."""
    return _relu_pool(y, pool)


class VggStack:
    """Thirteen conv layers with their weights resident on the device."""

    def __init__(self, dtype="bf16", plans=None, policy="accuracy", cap=None, device="cuda", calib_images=2,
                 candidates=VGG_CANDIDATES):
        self.dtype = dtype
        self.tdt = TORCH_DTYPES[dtype]
        self.layers = []
        for i, (hw, C, K, pool) in enumerate(VGG16_LAYERS):
            w = torch.from_numpy(vgg_layer_weights(i, C, K)).to(device).to(self.tdt)
            self.layers.append({"hw": hw, "C": C, "K": K, "pool": pool, "w": w})
        if plans is not None:
            for L, spec in zip(self.layers, plans):
                L["spec"], L["search"] = spec, []
                L["plan"] = Plan(spec.moduli, m=spec.m, dtype=dtype, inner=spec.inner)
            return
        # choose each layer's plan on the first images of its real input
        x = self.input(calib_images, device=device)
        for L in self.layers:
            spec, rows = search.best_plan(x, L["w"], candidates, policy=policy, cap=cap)
            L["spec"], L["search"] = spec, rows
            L["plan"] = Plan(spec.moduli, m=spec.m, dtype=dtype, inner=spec.inner)
            x = relu_pool(L["plan"].conv2d(x, L["w"]), L["pool"])

    def share_workspace(self, N):
        """Bind one device workspace, sized for the largest layer at batch N,
        to every layer's plan.  The layers run one after another on one
        stream, so they can share it; the next layer's transforms then write
        where the previous layer's fused kernel read (a pass of the stack at
        N = 32 in bf16: 1.89 against 1.92-1.96 ms with a workspace per layer)."""
        if getattr(self, "_shared_n", None) == N:
            return
        need = max(L["plan"].workspace_bytes(N, L["hw"], L["hw"], L["C"], L["K"]) for L in self.layers)
        ws = torch.empty(need, dtype=torch.uint8, device=self.layers[0]["w"].device)
        for L in self.layers:
            L["plan"].bind_workspace(ws)
        self._shared_n = N

    def input(self, N, seed=0, device="cuda"):
        return torch.from_numpy(vgg_input(N, seed)).to(device).to(self.tdt)

    def direct_flops(self, N):
        return sum(2 * N * L["hw"] * L["hw"] * L["C"] * L["K"] * 9 for L in self.layers)

    def forward(self, x, keep=False):
        """Run the stack; with ``keep`` also return every layer's (input, raw conv output)."""
        trace = []
        self.share_workspace(x.shape[0])
        for L in self.layers:
            y = L["plan"].conv2d(x, L["w"])
            if keep:
                trace.append((x, y))
            x = relu_pool(y, L["pool"])
        return (x, trace) if keep else x

    def timed_forward(self, x, flush=None, lead=None):
        """One pass with HIP events around each convolution; returns (output,
        conv ms per layer).  With ``flush`` (a large device buffer) the buffer
        is overwritten before each convolution, outside its events, so that
        each layer starts with its data out of the caches.  With ``lead`` (a
        device buffer) the buffer is overwritten once before the first
        convolution, outside its events: the GPU is then still busy while the
        host enqueues that convolution, so its events time the GPU's work
        rather than the host's launch latency (the later convolutions are
        enqueued while earlier work runs)."""
        ev = []
        stream = torch.cuda.current_stream()
        self.share_workspace(x.shape[0])
        if lead is not None and flush is None:
            lead.fill_(1)
        for L in self.layers:
            if flush is not None:
                flush.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            y = L["plan"].conv2d(x, L["w"])
            e1.record(stream)
            ev.append((e0, e1))
            x = relu_pool(y, L["pool"])
        torch.cuda.synchronize()
        return x, [a.elapsed_time(b) for a, b in ev]

    def timed_pass(self, x, reps):
        """Average ms of a whole pass (convolutions, ReLU and pooling) over
        ``reps`` back-to-back passes, HIP events around them."""
        stream = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            self.forward(x)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def summary(self):
        return [f"{L['hw']}x{L['hw']} {L['C']}->{L['K']}: {{{L['spec'].moduli}}} m={L['spec'].m}"
                for L in self.layers]
