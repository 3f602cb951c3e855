"""ctypes view of include/iso.h (argument marshalling only; all work runs in libiso.so)."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# ISO_LIB_PATH selects another build of the same library (the host-sanitized one of build.py)
LIB_PATH = os.environ.get("ISO_LIB_PATH") or os.path.join(HERE, "libiso.so")
MAX_K = 8

OK, ERR_INVALID_ARG, ERR_ALIGNMENT, ERR_WORKSPACE, ERR_NONFINITE, ERR_HIP, ERR_UNSUPPORTED, ERR_INTERNAL = range(8)
F32, BF16 = 0, 1
MERGE_TA, MERGE_TIES, MERGE_RAM = 0, 1, 2
UPDATE_APPLY, UPDATE_FUSED, UPDATE_SPECTRAL, UPDATE_ORTHO = 0, 1, 2, 3
(OP_TOPK, OP_SIGN, OP_MERGE, OP_UPDATE_APPLY, OP_UPDATE_FUSED, OP_UPDATE_FUSED_SELECT, OP_UPDATE_SPECTRAL,
 OP_BLOCKDIAG, OP_UPDATE_ORTHO) = range(9)

SYMBOLS = ["iso_workspace_size", "iso_topk_mask", "iso_sign_elect", "iso_merge", "iso_update",
           "iso_blockdiag_project", "iso_blockdiag_project_factors", "iso_workspace_size_tsv", "iso_k_from_density", "iso_read_device_status",
           "iso_read_fallback_count", "iso_profile_begin", "iso_profile_end", "iso_profile_flops", "iso_status_string",
           "iso_workspace_size_optimizer", "iso_optimizer_step", "iso_optimizer_step_muon", "iso_spectral_diagnostics",
           "iso_spectrum_interpolate", "iso_transport_ratios", "iso_spectral_error", "iso_update_noalloc"]


class IsoTensor(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("deltas", ctypes.c_void_p * MAX_K), ("out", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("k", ctypes.c_int64),
                ("select_group", ctypes.c_int32)]


class IsoFactors(ctypes.Structure):
    _fields_ = [("u", ctypes.c_void_p), ("s", ctypes.c_void_p), ("v", ctypes.c_void_p)]


class IsoFrame(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("u", "v", "sigma", "m_u", "v_u", "m_v", "v_v", "grad", "w_out")] + \
        [("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("rank", ctypes.c_int64)]


class IsoAdamW(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double), ("step", ctypes.c_int64)]


class IsoMuon(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("momentum", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("nesterov", ctypes.c_int32)]


class IsoSelectDesc(ctypes.Structure):
    _fields_ = [("t_key", ctypes.c_uint32), ("key_max", ctypes.c_uint32), ("n_above", ctypes.c_int64),
                ("tie_quota", ctypes.c_int64), ("tie_cutoff", ctypes.c_int64)]


class IsoUpdateArgs(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("merge", ctypes.c_int), ("lambda_", ctypes.c_double),
                ("eps_act", ctypes.c_double), ("desc", ctypes.c_void_p), ("tau_in", ctypes.c_void_p),
                ("sign_out", ctypes.c_void_p), ("rho_keep", ctypes.c_double), ("ridge", ctypes.c_double),
                ("c_min", ctypes.c_double), ("c_max", ctypes.c_double), ("coef_out", ctypes.c_void_p)]


_lib = None


def load():
    """Load libiso.so; raises if it has not been built (there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, I, Z, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_double
    T = ctypes.POINTER(IsoTensor)
    L.iso_workspace_size.argtypes = [I, T, I, I, I]
    L.iso_workspace_size.restype = Z
    L.iso_topk_mask.argtypes = [T, I, I, I, P, P, P, Z, P]
    L.iso_sign_elect.argtypes = [T, I, I, I, P, P, P, Z, P]
    L.iso_merge.argtypes = [T, I, I, I, I, P, D, D, P, P, Z, P]
    L.iso_update.argtypes = [T, I, I, I, ctypes.POINTER(IsoUpdateArgs), P, Z, P]
    L.iso_update_noalloc.argtypes = [T, I, I, I, ctypes.POINTER(IsoUpdateArgs), ctypes.POINTER(ctypes.c_void_p), P]
    L.iso_blockdiag_project.argtypes = [T, I, I, I, I, D, P, P, Z, P]
    L.iso_blockdiag_project_factors.argtypes = [T, I, I, I, I, D, ctypes.POINTER(IsoFactors), P, P, Z, P]
    L.iso_workspace_size_tsv.argtypes = [T, I, I, I, I]
    L.iso_workspace_size_tsv.restype = Z
    L.iso_k_from_density.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
    L.iso_k_from_density.restype = ctypes.c_int64
    L.iso_read_device_status.argtypes = [P, P]
    L.iso_read_fallback_count.argtypes = [P, P, ctypes.POINTER(ctypes.c_int32)]
    L.iso_profile_begin.argtypes = []
    L.iso_profile_end.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]
    L.iso_profile_flops.argtypes = [ctypes.POINTER(ctypes.c_double)]
    L.iso_workspace_size_optimizer.argtypes = [ctypes.POINTER(IsoFrame), I]
    L.iso_workspace_size_optimizer.restype = Z
    L.iso_optimizer_step.argtypes = [ctypes.POINTER(IsoFrame), I, I, ctypes.POINTER(IsoAdamW), P, Z, P]
    L.iso_optimizer_step_muon.argtypes = [ctypes.POINTER(IsoFrame), I, I, ctypes.POINTER(IsoMuon), P, Z, P]
    L.iso_spectral_diagnostics.argtypes = [T, I, I, P, P, Z, P]
    L.iso_spectrum_interpolate.argtypes = [T, I, I, D, P, Z, P]
    L.iso_spectral_error.argtypes = [T, I, I, I, P, P, Z, P]
    L.iso_transport_ratios.argtypes = [T, I, I, ctypes.POINTER(ctypes.c_double), I, P, P, Z, P]
    L.iso_status_string.argtypes = [I]
    L.iso_status_string.restype = ctypes.c_char_p
    for fn in ("iso_topk_mask", "iso_sign_elect", "iso_merge", "iso_update", "iso_update_noalloc",
               "iso_blockdiag_project",
               "iso_blockdiag_project_factors", "iso_optimizer_step", "iso_optimizer_step_muon",
               "iso_spectral_diagnostics",
               "iso_spectrum_interpolate", "iso_transport_ratios", "iso_spectral_error",
               "iso_read_device_status", "iso_read_fallback_count", "iso_profile_begin", "iso_profile_end",
               "iso_profile_flops"):
        getattr(L, fn).restype = I
    _lib = L
    return L
