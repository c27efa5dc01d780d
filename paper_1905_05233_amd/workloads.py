"""Seeded synthetic workloads shared by the tests, the bench and the CPU oracle.

This module holds no arithmetic of the method: it only names the layer shapes,
the modulus sets and the value distributions, and draws the inputs.  Values
are drawn in float64 from ``numpy.random.Generator(PCG64(seed))`` -- the input
x first (NHWC order), then the weights w ([K][3][3][C] order) -- and stored as
float32, the data as it would sit in memory before the storage dtype is
chosen.  Each consumer rounds float32 to fp16/bf16 itself.

Distributions (CNN-layer-shaped data):
  * ``uniform``:    x ~ U[-1, 1]
  * ``halfnormal``: x ~ |N(0, 1)|  (post-ReLU activations)
  * ``normal_clip1``: x and the weights ~ N(0, 1) restricted to (-1, 1)
    (values redrawn until they fall inside; the random data of the error
    study of Section 3.1)
  * weights otherwise N(0, 2 / (9 C))  (He initialisation of a 3x3xC filter)
"""
from dataclasses import dataclass, field

import numpy as np

# modulus sets, written as the plan spec strings the library parses
F2_LINEAR = "0,1,-1,inf"
F4_LINEAR = "0,1,-1,1/2,-1/2,inf"
F4_A2P1 = "0,1,-1,a^2+1,inf"
F6_LINEAR = "0,-1,1,-1/2,2,1/2,-2,inf"
F6_TWO_QUAD = "0,-1,1,a^2+1,a^2-2,inf"
F6_ONE_A2P1 = "0,-1,1,-1/2,2,a^2+1,inf"
INNER_DEFAULT = "0,-1,inf"


@dataclass(frozen=True)
class PlanSpec:
    moduli: str
    m: int
    inner: str = INNER_DEFAULT


@dataclass
class Workload:
    name: str
    N: int
    H: int
    W: int
    C: int
    K: int
    dtype: str
    plans: tuple
    x_dist: str
    seed: int = 0
    cap: float = 5e-2
    note: str = ""

    def draw(self):
        return draw_inputs(self.N, self.H, self.W, self.C, self.K, self.x_dist, self.seed)

    @property
    def direct_flops(self):
        """Direct-convolution flop count 2 N H W C K 9 (the throughput numerator)."""
        return 2 * self.N * self.H * self.W * self.C * self.K * 9


def _normal_in_unit(rng, shape):
    """N(0, 1) values restricted to (-1, 1) by redrawing those outside."""
    v = rng.standard_normal(size=shape)
    bad = np.abs(v) >= 1.0
    while np.any(bad):
        v[bad] = rng.standard_normal(size=int(np.sum(bad)))
        bad = np.abs(v) >= 1.0
    return v


def draw_inputs(N, H, W, C, K, x_dist, seed, w_seed=None):
    """x [N][H][W][C] and w [K][3][3][C] as float32 arrays.

    With ``w_seed`` the weights come from their own generator (stacked layers).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    if x_dist == "uniform":
        x = rng.uniform(-1.0, 1.0, size=(N, H, W, C))
    elif x_dist == "halfnormal":
        x = np.abs(rng.standard_normal(size=(N, H, W, C)))
    elif x_dist == "ternary":
        x = rng.integers(-1, 2, size=(N, H, W, C)).astype(np.float64)
    elif x_dist == "int2":
        x = rng.integers(-2, 3, size=(N, H, W, C)).astype(np.float64)
    elif x_dist == "normal_clip1":
        x = _normal_in_unit(rng, (N, H, W, C))
    else:
        raise ValueError(f"unknown distribution {x_dist!r}")
    wrng = rng if w_seed is None else np.random.Generator(np.random.PCG64(w_seed))
    if x_dist in ("ternary", "int2"):
        lo, hi = (-1, 2) if x_dist == "ternary" else (-2, 3)
        w = wrng.integers(lo, hi, size=(K, 3, 3, C)).astype(np.float64)
    elif x_dist == "normal_clip1":
        w = _normal_in_unit(wrng, (K, 3, 3, C))
    else:
        w = wrng.standard_normal(size=(K, 3, 3, C)) * np.sqrt(2.0 / (9.0 * C))
    return x.astype(np.float32), w.astype(np.float32)


CONFIGS = {
    "cfg1": Workload("cfg1", N=1, H=16, W=16, C=8, K=8, dtype="f32",
                     plans=(PlanSpec(F2_LINEAR, 2),), x_dist="uniform", cap=1e-5,
                     note="F(2x2,3x3) linear points, fp32"),
    "cfg2": Workload("cfg2", N=8, H=56, W=56, C=128, K=128, dtype="f32",
                     plans=(PlanSpec(F4_LINEAR, 4),), x_dist="halfnormal", cap=1e-4,
                     note="F(4x4,3x3) linear points, fp32"),
    "cfg3": Workload("cfg3", N=1, H=16, W=16, C=8, K=8, dtype="f16",
                     plans=(PlanSpec(F4_LINEAR, 4), PlanSpec(F4_A2P1, 4)), x_dist="uniform",
                     note="F(4x4,3x3) linear vs {0,1,-1,a^2+1,inf}, fp16"),
    "cfg4": Workload("cfg4", N=16, H=28, W=28, C=256, K=256, dtype="bf16",
                     plans=(PlanSpec(F6_LINEAR, 6), PlanSpec(F6_TWO_QUAD, 6)), x_dist="halfnormal",
                     note="F(6x6,3x3) linear vs {0,-1,1,a^2+1,a^2-2,inf}, bf16"),
}

# VGG-16's thirteen 3x3 convolutions: (H = W, C, K); 2x2 max-pool after the
# layers marked True.  conv1_1 takes the 3-channel image.
VGG16_LAYERS = (
    (224, 3, 64, False), (224, 64, 64, True),
    (112, 64, 128, False), (112, 128, 128, True),
    (56, 128, 256, False), (56, 256, 256, False), (56, 256, 256, True),
    (28, 256, 512, False), (28, 512, 512, False), (28, 512, 512, True),
    (14, 512, 512, False), (14, 512, 512, False), (14, 512, 512, True),
)

# candidate plans for the VGG-16 stack (best accuracy per layer is chosen)
VGG_CANDIDATES = (
    PlanSpec(F4_LINEAR, 4), PlanSpec(F4_A2P1, 4),
    PlanSpec(F6_LINEAR, 6), PlanSpec(F6_TWO_QUAD, 6), PlanSpec(F6_ONE_A2P1, 6),
)


def vgg_layer_weights(layer, C, K):
    """Weights of VGG-16 layer ``layer`` (0-based): seed 1 + layer, N(0, 2/(9C))."""
    rng = np.random.Generator(np.random.PCG64(1 + layer))
    return (rng.standard_normal(size=(K, 3, 3, C)) * np.sqrt(2.0 / (9.0 * C))).astype(np.float32)


def vgg_input(N, seed=0):
    rng = np.random.Generator(np.random.PCG64(seed))
    return np.abs(rng.standard_normal(size=(N, 224, 224, 3))).astype(np.float32)
