"""ctypes declarations for ``libwinograd_crt.so`` (the C ABI in
``include/winograd_crt.h``).  Marshalling only: no arithmetic happens here."""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwinograd_crt.so")

WG_OK = 0
STATUS_NAMES = {
    0: "WG_OK", 1: "WG_ERR_ARG", 2: "WG_ERR_DEGREE_SUM", 3: "WG_ERR_NOT_COPRIME", 4: "WG_ERR_REDUCIBLE",
    5: "WG_ERR_UNSUPPORTED", 6: "WG_ERR_OVERFLOW", 7: "WG_ERR_WORKSPACE", 8: "WG_ERR_HIP", 9: "WG_ERR_INTERNAL",
}
DTYPE_CODES = {"f32": 0, "f16": 1, "bf16": 2}
SQ_SUMS_DOUBLES = 514   # WG_SQ_SUMS_DOUBLES


class WgRational(ctypes.Structure):
    _fields_ = [("num", ctypes.c_int64), ("den", ctypes.c_int64)]


class WgModulus(ctypes.Structure):
    _fields_ = [("degree", ctypes.c_int), ("coef", WgRational * 4)]


class WgPolySet(ctypes.Structure):
    _fields_ = [("n_mod", ctypes.c_int), ("mods", ctypes.POINTER(WgModulus)), ("n_inner", ctypes.c_int),
                ("inner_pts", ctypes.POINTER(WgRational)), ("inner_inf", ctypes.c_int)]


class WgPlanOptions(ctypes.Structure):
    _fields_ = [("factors", ctypes.c_int), ("path", ctypes.c_int), ("generic_transforms", ctypes.c_int),
                ("scaling", ctypes.c_int), ("channel_sum", ctypes.c_int)]


FACTOR_CODES = {"B": 0, "G": 1}
SCALING_CODES = {"none": 0, "l1": 1}
CHANNEL_SUM_CODES = {"mfma": 0, "pairwise": 1}
PATH_CODES = {"auto": 0, "separate": 1, "fused": 2, "fused_input": 3}
PATH_NAMES = {v: k for k, v in PATH_CODES.items()}


class WgTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n", ctypes.c_int64), ("h", ctypes.c_int64),
                ("w", ctypes.c_int64), ("c", ctypes.c_int64)]


class WinogradError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def lib():
    """Load the native library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"native library {LIB_PATH} is missing; build it with "
                           "`python -m paper_1905_05233_amd.build_native`")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    sz = ctypes.c_size_t
    plan_p = ctypes.POINTER(ctypes.c_void_p)
    sigs = {
        "winograd_plan_create": (ctypes.c_int, [ctypes.POINTER(WgPolySet), ctypes.c_int, ctypes.c_int,
                                                ctypes.c_int, plan_p]),
        "winograd_plan_create_str": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int, ctypes.c_int,
                                                    ctypes.c_int, plan_p]),
        "winograd_plan_create_ex": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int, ctypes.c_int,
                                                   ctypes.c_int, ctypes.POINTER(WgPlanOptions), plan_p]),
        "winograd_plan_destroy": (None, [P]),
        "winograd_plan_alpha": (ctypes.c_int, [P]),
        "winograd_plan_builtin": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_int)]),
        "winograd_plan_info": (ctypes.c_int, [P] + [ctypes.POINTER(ctypes.c_int)] * 5),
        "winograd_plan_matrix": (ctypes.c_int, [P, ctypes.c_char, ctypes.POINTER(WgRational), sz]),
        "winograd_plan_matrix_f32": (ctypes.c_int, [P, ctypes.c_char, ctypes.POINTER(ctypes.c_float), sz]),
        "winograd_plan_ratio": (ctypes.c_int, [P, ctypes.POINTER(i64), ctypes.POINTER(i64)]),
        "winograd_workspace_bytes": (ctypes.c_int, [P, i64, i64, i64, i64, i64, ctypes.POINTER(sz)]),
        "winograd_plan_set_workspace": (ctypes.c_int, [P, P, sz]),
        "winograd_conv_path": (ctypes.c_int, [P, i64, i64, i64, i64, i64, ctypes.POINTER(ctypes.c_int)]),
        "winograd_conv_chunks": (ctypes.c_int, [P, i64, i64, i64, i64, i64, ctypes.POINTER(i64), ctypes.POINTER(i64)]),
        "winograd_conv2d": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), ctypes.POINTER(WgTensor),
                                           ctypes.POINTER(WgTensor), P]),
        "winograd_workspace_bytes_1d": (ctypes.c_int, [P, i64, i64, i64, i64, ctypes.POINTER(sz)]),
        "winograd_conv1d": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), ctypes.POINTER(WgTensor),
                                           ctypes.POINTER(WgTensor), P]),
        "winograd_conv2d_static": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), ctypes.POINTER(WgTensor),
                                                  ctypes.POINTER(WgTensor), P]),
        "winograd_kernel_transform": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), P, P]),
        "winograd_input_transform": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), P, P]),
        "winograd_kernel_input_transform": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), ctypes.POINTER(WgTensor),
                                                           P, P, P]),
        "winograd_contract": (ctypes.c_int, [P, P, P, P, i64, i64, i64, P]),
        "winograd_output_transform": (ctypes.c_int, [P, P, ctypes.POINTER(WgTensor), P]),
        "winograd_contract_output": (ctypes.c_int, [P, P, P, i64, ctypes.POINTER(WgTensor), P]),
        "winograd_input_contract_output": (ctypes.c_int, [P, ctypes.POINTER(WgTensor), P, ctypes.POINTER(WgTensor),
                                                          P]),
        "winograd_relu_pool": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(WgTensor), ctypes.POINTER(WgTensor),
                                              ctypes.c_int, P]),
        "winograd_direct_conv_f64": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(WgTensor),
                                                    ctypes.POINTER(WgTensor), P, P]),
        "winograd_sq_error_sums": (ctypes.c_int, [ctypes.c_int, P, P, i64, P, P]),
        "winograd_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def check(status):
    if status != WG_OK:
        msg = lib().winograd_last_error()
        raise WinogradError(status, msg.decode() if msg else "")
