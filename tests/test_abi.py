"""C-ABI library on the CPU: it loads, exports every symbol the header
declares, builds plans whose exact matrices and fp32 tables equal the oracle's
bit for bit, and rejects invalid input with the documented status codes.
No kernel is launched here."""
import ctypes
import os
import re
from fractions import Fraction

import numpy as np
import pytest

from conftest import ROOT, load_golden
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import _native as N
from paper_1905_05233_amd import workloads as WL
from paper_1905_05233_amd.winograd import Plan

HEADER = os.path.join(ROOT, "include", "winograd_crt.h")

PLAN_SETS = [
    (WL.F2_LINEAR, 2, "0,-1,inf"), (WL.F4_LINEAR, 4, "0,-1,inf"), (WL.F4_A2P1, 4, "0,-1,inf"),
    (WL.F6_LINEAR, 6, "0,-1,inf"), (WL.F6_TWO_QUAD, 6, "0,-1,inf"), (WL.F6_ONE_A2P1, 6, "0,-1,inf"),
    ("0,a^2+1,inf", 2, "0,1,inf"), ("0,a^2+a+1,inf", 2, "0,1,inf"), ("0,a^2-2,inf", 2, "0,-1,inf"),
    ("a^2+1,a^2+a+1", 2, "0,-1,inf"), ("a^2+1,a^2+a+1,a^2-a+1", 4, "0,-1,inf"),
    ("0,a^3+2", 2, "0,-1,1,-2,inf"), ("0,1,-1,2,-2,inf", 4, "0,-1,inf"),
    ("0,-1,1,-1/2,2,1/2,-2,a^2+1,inf", 8, "0,-1,inf"),
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,a^2+1,inf", 10, "0,-1,inf"),
    ("0,1,-1,1/2,-1/2,2,-2,1/4,-4,4,-1/4,a^2+1,inf", 12, "0,-1,inf"),
    ("0,-1,a^3+2,inf", 4, "0,-1,1,-2,inf"), ("0,1,-1,1/2,-1/2,2", 4, "0,-1,inf"),
]


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\**\s*(winograd_\w+)\s*\(", text, re.M)))


def test_library_loads_and_exports_every_symbol():
    lib = N.lib()
    names = header_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("spec,m,inner", PLAN_SETS)
def test_plan_exact_parity_with_oracle(spec, m, inner):
    ref = OP.build_plan(spec, n_o=m, inner=inner)
    p = Plan(spec, m=m, dtype="f32", inner=inner)
    assert p.alpha == ref.alpha and p.tile_in == ref.tile_in
    assert p.matrix("G") == ref.G
    assert p.matrix("A") == ref.A
    assert p.matrix("B") == ref.B
    assert p.ratio == ref.ratio
    for which, mat in (("G", ref.G), ("A", ref.A), ("B", ref.B)):
        ours = np.array(p.matrix_f32(which), dtype=np.float32)
        want = np.array([[OF.fraction_to_f32(v) for v in row] for row in mat], dtype=np.float32)
        assert np.array_equal(ours.view(np.uint32), want.view(np.uint32)), which


@pytest.mark.parametrize("spec,m,inner", PLAN_SETS[::2])
def test_factors_in_g_plan_parity_with_oracle(spec, m, inner):
    """winograd_plan_create_ex with WG_FACTORS_IN_G: exact matrices and fp32
    tables equal the oracle's factors="G" construction."""
    ref = OP.build_plan(spec, n_o=m, inner=inner, factors="G")
    p = Plan(spec, m=m, dtype="f32", inner=inner, factors="G")
    for which, mat in (("G", ref.G), ("A", ref.A), ("B", ref.B)):
        assert p.matrix(which) == mat
        ours = np.array(p.matrix_f32(which), dtype=np.float32)
        want = np.array([[OF.fraction_to_f32(v) for v in row] for row in mat], dtype=np.float32)
        assert np.array_equal(ours.view(np.uint32), want.view(np.uint32)), which


@pytest.mark.parametrize("spec,m,inner", PLAN_SETS[1::2])
@pytest.mark.parametrize("factors", ["B", "G"])
def test_scaled_plan_parity_with_oracle(spec, m, inner, factors):
    """WG_SCALE_ROWS_L1: exact matrices and fp32 tables equal the oracle's
    scaling="l1" construction (with either CRT factor placement)."""
    ref = OP.build_plan(spec, n_o=m, inner=inner, factors=factors, scaling="l1")
    p = Plan(spec, m=m, dtype="f32", inner=inner, factors=factors, scaling="l1")
    assert p.builtin == -1 or factors == "B"
    for which, mat in (("G", ref.G), ("A", ref.A), ("B", ref.B)):
        assert p.matrix(which) == mat
        ours = np.array(p.matrix_f32(which), dtype=np.float32)
        want = np.array([[OF.fraction_to_f32(v) for v in row] for row in mat], dtype=np.float32)
        assert np.array_equal(ours.view(np.uint32), want.view(np.uint32)), which


def test_unknown_scaling_rejected():
    lib = N.lib()
    bad = N.WgPlanOptions(0, 0, 0, 5)
    h = ctypes.c_void_p()
    assert lib.winograd_plan_create_ex(WL.F4_LINEAR.encode(), b"", 4, 3, 0, ctypes.byref(bad), ctypes.byref(h)) == 1
    assert not h.value
    with pytest.raises(ValueError):
        Plan(WL.F4_LINEAR, m=4, scaling="l2")


def test_create_ex_defaults_and_errors():
    lib = N.lib()
    h = ctypes.c_void_p()
    # NULL options = the paper's placement
    assert lib.winograd_plan_create_ex(WL.F4_LINEAR.encode(), b"", 4, 3, 0, None, ctypes.byref(h)) == 0
    p = Plan(WL.F4_LINEAR, m=4)
    buf = (N.WgRational * (p.alpha * 3))()
    assert lib.winograd_plan_matrix(h, b"G", buf, len(buf)) == 0
    assert [[Fraction(buf[i * 3 + j].num, buf[i * 3 + j].den) for j in range(3)] for i in range(p.alpha)] == \
        p.matrix("G")
    lib.winograd_plan_destroy(h)
    bad = N.WgPlanOptions(7)
    h2 = ctypes.c_void_p()
    assert lib.winograd_plan_create_ex(WL.F4_LINEAR.encode(), b"", 4, 3, 0, ctypes.byref(bad), ctypes.byref(h2)) == 1
    assert not h2.value
    with pytest.raises(ValueError):
        Plan(WL.F4_LINEAR, m=4, factors="A")


def test_struct_entry_matches_string_entry():
    p1 = Plan(WL.F6_TWO_QUAD, m=6, dtype="bf16")
    mods = [[0, 1], [1, 1], [-1, 1], [1, 0, 1], [-2, 0, 1], None]
    p2 = Plan.from_moduli(mods, m=6, dtype="bf16", inner_points=[0, -1], inner_inf=True)
    for w in "GAB":
        assert p1.matrix(w) == p2.matrix(w)


def test_non_monic_moduli_are_normalised():
    p1 = Plan("0,1,-1,a^2+1,inf", m=4)
    p2 = Plan.from_moduli([[0, 2], [-3, 3], [1, 1], [2, 0, 2], None], m=4)
    for w in "GAB":
        assert p1.matrix(w) == p2.matrix(w)


def test_worked_example_through_the_library():
    """Section 2.2's printed G^W and (at b=0, c=1) B^W, via the C ABI."""
    from conftest import frac_matrix
    gold = load_golden("worked_example_sec2_2.json")
    for b, c in [(0, 1), (1, 1), (0, -2)]:
        p = Plan.from_moduli([[0, 1], [c, b, 1], None], m=2, inner_points=[0, 1], inner_inf=True)
        env = {"b": Fraction(b), "c": Fraction(c)}
        assert p.matrix("G") == frac_matrix(gold["general"]["G_W"], env)
    p = Plan("0,a^2+1,inf", m=2, inner="0,1,inf")
    assert p.matrix("B") == frac_matrix(gold["b0c1"]["B_W"], {"b": Fraction(0), "c": Fraction(1)})


@pytest.mark.parametrize("spec,m,inner,code", [
    ("0,1,inf", 4, "", 2),                        # degree sum
    ("0,1,-1,a^2+1,a^2+1,inf", 6, "", 3),         # not coprime
    ("0,0,1,-1,1/2,inf", 4, "", 3),               # repeated point
    ("0,1,-1,a^2-1,inf", 4, "", 4),               # reducible
    ("0,1,-1,a^2-4a+4,inf", 4, "", 4),            # reducible (double root)
    ("0,1,x,inf", 2, "", 1),                      # parse error
    ("0,1,-1,1/0,inf", 4, "", 1),                 # zero denominator
    ("0,a^2+1,inf", 2, "0,inf", 1),               # too few inner points
    ("0,a^2+1,inf", 2, "0,0,inf", 1),             # repeated inner point
    ("0,1,inf,-1,inf", 2, "", 1),                 # infinity twice
    ("0,1,-1,99999999999999999999,inf", 2, "", 6),  # out of int64
])
def test_invalid_plans_rejected(spec, m, inner, code):
    with pytest.raises(N.WinogradError) as ei:
        Plan(spec, m=m, inner=inner)
    assert ei.value.status == code
    assert str(ei.value)


def test_unsupported_shapes_rejected():
    with pytest.raises(N.WinogradError) as ei:
        Plan("0,1,-1,inf", m=2, r=5)
    assert ei.value.status == 5
    pts = ",".join(str(i) for i in range(-8, 8))      # m = 15 -> tile 17 > 16
    with pytest.raises(N.WinogradError) as ei:
        Plan(pts + ",inf", m=15)
    assert ei.value.status == 5
    with pytest.raises(ValueError):
        Plan("0,1,-1,inf", m=2, dtype="f64")


def test_exact_overflow_is_reported():
    """Points whose Lagrange denominators leave int64 must raise, not wrap."""
    big = [str(Fraction(1, 3 ** k)) for k in range(1, 11)]
    with pytest.raises(N.WinogradError) as ei:
        Plan(",".join(["0"] + big) + ",inf", m=10)
    assert ei.value.status in (6,)


def test_conv_chunks_and_chunked_workspace():
    """The fused path runs a batch whose V exceeds 160 MiB in balanced chunks
    of images (winograd_conv_chunks), with a workspace of U and one chunk's
    V; other layers run in one launch pair."""
    p = Plan(WL.F4_A2P1, m=4, dtype="bf16")
    v_img = 49 * 56 * 56 * 64 * 2                         # 224x224x64, F(4x4), alpha' = 7
    per = (160 << 20) // v_img                            # 8 images within the budget
    assert per == 8
    assert p.conv_chunks(32, 224, 224, 64, 64) == (4, 8)
    assert p.conv_chunks(9, 224, 224, 64, 64) == (2, 5)   # 5 + 4
    assert p.conv_chunks(8, 224, 224, 64, 64) == (1, 8)
    assert p.conv_chunks(32, 112, 112, 128, 128) == (2, 16)
    u = -(-49 * 64 * 64 * 2 // 256) * 256
    for n, chunk in ((32, 8), (9, 5), (8, 8)):
        v = -(-49 * chunk * 56 * 56 * 64 * 2 // 256) * 256
        assert p.workspace_bytes(n, 224, 224, 64, 64) == u + v
    ps = Plan(WL.F4_A2P1, m=4, dtype="bf16", path="separate")
    assert ps.conv_chunks(32, 224, 224, 64, 64) == (1, 32)
    assert p.conv_path(32, 28, 28, 512, 512) == "separate"            # 1024-byte rows
    assert p.conv_chunks(32, 28, 28, 512, 512) == (1, 32)
    assert p.conv_path(32, 28, 28, 256, 512) == "fused"               # 512-byte rows, 2^19 pairs and more
    assert p.conv_path(8, 28, 28, 256, 512) == "separate"


def test_conv_path_option_and_workspace():
    """WG_PATH_SEPARATE / WG_PATH_FUSED / WG_PATH_AUTO: the resolved path and
    the workspace (the fused path needs no M), and the errors."""
    Nn, H, W, C, K = 2, 20, 20, 16, 24
    ps = Plan(WL.F4_LINEAR, m=4, path="separate")
    pf = Plan(WL.F4_LINEAR, m=4, path="fused")
    pa = Plan(WL.F4_LINEAR, m=4)
    assert ps.conv_path(Nn, H, W, C, K) == "separate"
    assert pf.conv_path(Nn, H, W, C, K) == "fused"
    assert pa.conv_path(Nn, H, W, C, K) in ("separate", "fused")
    T, a2, Kp = Nn * 5 * 5, 36, 24
    m_bytes = -(-a2 * T * Kp * 4 // 256) * 256
    assert ps.workspace_bytes(Nn, H, W, C, K) - pf.workspace_bytes(Nn, H, W, C, K) == m_bytes
    # input tile 10 (m = 8): no fused kernel; asking for it is an error, auto takes the separate path
    spec8 = "0,-1,1,-1/2,2,1/2,-2,a^2+1,inf"
    big = Plan(spec8, m=8, path="fused")
    for call in (big.conv_path, big.workspace_bytes):
        with pytest.raises(N.WinogradError) as ei:
            call(Nn, H, W, C, K)
        assert ei.value.status == 5
    assert Plan(spec8, m=8).conv_path(Nn, H, W, C, K) == "separate"
    lib = N.lib()
    h = ctypes.c_void_p()
    bad = N.WgPlanOptions(0, 9)
    assert lib.winograd_plan_create_ex(WL.F4_LINEAR.encode(), b"", 4, 3, 0, ctypes.byref(bad), ctypes.byref(h)) == 1
    assert not h.value
    with pytest.raises(ValueError):
        Plan(WL.F4_LINEAR, m=4, path="fast")


def test_fused_input_path_rule():
    """WG_PATH_FUSED_INPUT (the input transform inside the fused kernel) is taken
    only when asked for, on channel rows of at most 32 bytes, more than 32
    output channels and alpha'^2 x 32 V rows within 48 KB; it needs neither V
    nor M in the workspace."""
    vgg0 = (32, 224, 224, 3, 64)
    ok = [(WL.F4_A2P1, 4, "bf16"), (WL.F4_A2P1, 4, "f16"), (WL.F6_LINEAR, 6, "bf16"), (WL.F4_LINEAR, 4, "f32")]
    for spec, m, dt in ok:
        assert Plan(spec, m=m, dtype=dt, path="fused_input").conv_path(*vgg0) == "fused_input"
        assert Plan(spec, m=m, dtype=dt).conv_path(*vgg0) == "fused"          # never chosen automatically
    no = [(WL.F4_A2P1, 4, "f32", vgg0),                       # 32-byte rows, alpha' 7: 49 KB of V rows
          (WL.F6_TWO_QUAD, 6, "bf16", vgg0),                  # alpha' 10: 50 KB
          (WL.F4_A2P1, 4, "bf16", (32, 224, 224, 3, 32)),     # K <= 32
          (WL.F4_A2P1, 4, "bf16", (32, 224, 224, 24, 64))]    # 48-byte rows
    for spec, m, dt, shape in no:
        with pytest.raises(N.WinogradError) as ei:
            Plan(spec, m=m, dtype=dt, path="fused_input").conv_path(*shape)
        assert ei.value.status == 5
    pf, pi = Plan(WL.F4_A2P1, m=4, dtype="bf16", path="fused"), Plan(WL.F4_A2P1, m=4, dtype="bf16", path="fused_input")
    Nn, H, W, C, K = 1, 9, 9, 3, 40
    T = Nn * 3 * 3
    v_bytes = -(-49 * T * 8 * 2 // 256) * 256
    assert pf.workspace_bytes(Nn, H, W, C, K) - pi.workspace_bytes(Nn, H, W, C, K) == v_bytes


def test_workspace_bytes_and_errors():
    p = Plan(WL.F4_LINEAR, m=4, dtype="f32", path="separate")
    Nn, H, W, C, K = 8, 56, 56, 128, 128
    T = Nn * 14 * 14
    need = p.workspace_bytes(Nn, H, W, C, K)
    a2 = 36
    assert need >= a2 * (K * C * 4 + T * C * 4 + T * K * 4)
    assert need <= a2 * (K * C * 4 + T * C * 4 + T * K * 4) + 3 * 256
    with pytest.raises(N.WinogradError) as ei:
        p.workspace_bytes(0, H, W, C, K)
    assert ei.value.status == 1
    lib = N.lib()
    fake = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: the call fails before any launch
    x = N.WgTensor(fake, Nn, H, W, C)
    w = N.WgTensor(fake, K, 3, 3, C)
    y = N.WgTensor(fake, Nn, H, W, K)
    st = lib.winograd_conv2d(p._h, ctypes.byref(x), ctypes.byref(w), ctypes.byref(y), None)
    assert st == 7 and b"workspace" in lib.winograd_last_error()
    bad = N.WgTensor(ctypes.c_void_p((1 << 20) + 4), Nn, H, W, C)
    assert lib.winograd_conv2d(p._h, ctypes.byref(bad), ctypes.byref(w), ctypes.byref(y), None) == 1
    wrong = N.WgTensor(fake, K, 3, 3, C + 1)
    assert lib.winograd_conv2d(p._h, ctypes.byref(x), ctypes.byref(wrong), ctypes.byref(y), None) == 1
    assert lib.winograd_conv2d(None, ctypes.byref(x), ctypes.byref(w), ctypes.byref(y), None) == 1
    assert lib.winograd_plan_set_workspace(p._h, ctypes.c_void_p((1 << 20) + 16), 4096) == 1


def test_unsupported_kernel_shape_reported_at_launch():
    """A valid plan whose (tile, alpha') has no compiled kernel fails cleanly."""
    p = Plan("a^2+1,a^2-2,inf", m=3)     # tile 5 with alpha' 7: no compiled transform kernels
    assert (p.tile_in, p.alpha) == (5, 7)
    lib = N.lib()
    fake = ctypes.c_void_p(1 << 20)
    x = N.WgTensor(fake, 1, 8, 8, 4)
    assert lib.winograd_input_transform(p._h, ctypes.byref(x), fake, None) == 5


def test_contraction_row_limit_reported_before_launch():
    """Channel rows too long for the kernels' 32-bit offsets (128 rows of
    36 MB here) fail with WG_ERR_HIP before anything is launched; the pointers
    are never dereferenced."""
    p = Plan(WL.F4_LINEAR, m=4, dtype="f32", path="separate")
    lib = N.lib()
    fake = ctypes.c_void_p(1 << 20)
    st = lib.winograd_contract(p._h, fake, fake, fake, 1, 9_000_000, 1, None)
    assert st == 8 and b"contraction" in lib.winograd_last_error()


def test_geometry_helpers():
    p = Plan(WL.F6_LINEAR, m=6, dtype="bf16")
    g = p.geometry(16, 28, 28, 256, 256)
    assert g["T"] == 16 * 5 * 5 and g["Cp"] == 256
    assert OC.tile_counts(28, 28, 6) == (5, 5)


def test_builtin_plans_identified():
    """The plans of the workloads run on the constant-coefficient transform
    kernels; any other table (other points, inner points, factor placement)
    and the generic option keep the run-time tables."""
    expect = [(WL.F2_LINEAR, 2), (WL.F4_LINEAR, 4), (WL.F4_A2P1, 4), (WL.F6_LINEAR, 6), (WL.F6_TWO_QUAD, 6),
              (WL.F6_ONE_A2P1, 6)]
    for i, (spec, m) in enumerate(expect):
        for dt in ("f32", "bf16"):
            assert Plan(spec, m=m, dtype=dt).builtin == i
        assert Plan(spec, m=m, generic_transforms=True).builtin == -1
        assert Plan(spec, m=m, factors="G").builtin == -1
    assert Plan("0,1,-1,2,-2,inf", m=4).builtin == -1
    assert Plan(WL.F4_A2P1, m=4, inner="0,1,inf").builtin == -1
    assert Plan("0,a^2+1,inf", m=2).builtin == -1
    lib = N.lib()
    h = ctypes.c_void_p()
    bad = N.WgPlanOptions(0, 0, 2)
    assert lib.winograd_plan_create_ex(WL.F4_LINEAR.encode(), b"", 4, 3, 0, ctypes.byref(bad), ctypes.byref(h)) == 1
