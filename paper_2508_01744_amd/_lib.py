"""ctypes binding of libagft.so: argument marshalling only.

The names mirror include/agft.h and include/agft_sim.h.  Loading fails loudly
when the library has not been built: there is no other implementation to
fall back to.
"""
import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libagft.so")

AGFT_OK = 0
AGFT_E_INVAL = -1
AGFT_E_UNSUPPORTED = -2
AGFT_E_STATE = -3
AGFT_E_HIP = -4
AGFT_ADOPT_STATE = 0x1

_i32, _u32, _f32, _i64, _sz, _vp = (ctypes.c_int32, ctypes.c_uint32, ctypes.c_float,
                                    ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p)


class agft_config(ctypes.Structure):
    _fields_ = [("B", _i32), ("K", _i32), ("d", _i32), ("lambda_", _f32), ("alpha0", _f32),
                ("alpha_sched", _i32), ("prune_rule", _i32), ("prune_period", _i32),
                ("prune_sticky", _i32), ("flags", _u32),
                ("ext_rounds", _i32), ("ext_min_n", _i32), ("ext_thr", _f32),
                ("hist_after", _i32), ("hist_min_n", _i32), ("hist_kappa", _f32),
                ("hist_min_arms", _i32), ("cascade_k", _i32),
                ("exploit", _i32), ("ph_delta", _f32), ("ph_lambda", _f32),
                ("ph_window", _i32), ("ph_min_rounds", _i32),
                ("refine", _i32), ("refine_period", _i32), ("refine_stride", _i32),
                ("refine_half", _i32), ("refine_mature", _i32), ("refine_min_n", _i32)]


class agft_state_view(ctypes.Structure):
    _fields_ = [("t", _i64), ("pending", _i32), ("B", _i32), ("K", _i32), ("d", _i32),
                ("chunks", _i32), ("block_arms", _i32), ("tail_floats", _i32),
                ("mask_words", _i32), ("arms", _vp), ("mask", _vp),
                ("inst", _vp), ("inst_words", _i32), ("stats", _vp), ("theta", _vp)]


class agft_env_config(ctypes.Structure):
    _fields_ = [("B", _i32), ("K", _i32), ("d", _i32), ("T", _i32),
                ("P0", _f32), ("c", _f32), ("l0", _f32), ("a", _f32), ("b", _f32),
                ("lat_min", _f32), ("f_lo", _f32), ("f_hi", _f32), ("f_init", _f32),
                ("tpot_div", _f32), ("drift", _f32),
                ("svc_lo", _i32), ("svc_hi", _i32), ("svc_init", _i32),
                ("q_cap", _i32), ("run_cap", _i32),
                ("mu", _f32 * 7), ("sd", _f32 * 7)]


class agft_launch_shape(ctypes.Structure):
    _fields_ = [("waves", _i32), ("simd_waves", _i32), ("tail_floats", _i32), ("early_update", _i32),
                ("cu_workgroups", _i32)]


ABI_VERSION = 6   # AGFT_ABI_VERSION of the agft_config layout declared here

EXPORTED = ["agft_state_bytes", "agft_create", "agft_step", "agft_get_state", "agft_export",
            "agft_set_stream", "agft_destroy", "agft_strerror", "agft_abi_version", "agft_launch_shape_for",
            "agft_env_state_bytes", "agft_env_reset", "agft_env_step", "agft_sim_step"]

_lib = None


class AgftError(RuntimeError):
    def __init__(self, fn, code):
        msg = _lib.agft_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{fn} failed: {msg} ({code})")
        self.code = code


def _declare(lib):
    cfgp = ctypes.POINTER(agft_config)
    envp = ctypes.POINTER(agft_env_config)
    lib.agft_state_bytes.restype = _sz
    lib.agft_state_bytes.argtypes = [cfgp]
    lib.agft_create.restype = ctypes.c_int
    lib.agft_create.argtypes = [cfgp, _vp, _sz, _vp, ctypes.POINTER(_vp)]
    lib.agft_step.restype = ctypes.c_int
    lib.agft_step.argtypes = [_vp, _vp, _vp, _vp, _vp]
    lib.agft_get_state.restype = ctypes.c_int
    lib.agft_get_state.argtypes = [_vp, ctypes.POINTER(agft_state_view)]
    lib.agft_export.restype = ctypes.c_int
    lib.agft_export.argtypes = [_vp, _vp, _vp]
    lib.agft_set_stream.restype = ctypes.c_int
    lib.agft_set_stream.argtypes = [_vp, _vp]
    lib.agft_destroy.restype = ctypes.c_int
    lib.agft_destroy.argtypes = [_vp]
    lib.agft_strerror.restype = ctypes.c_char_p
    lib.agft_strerror.argtypes = [ctypes.c_int]
    lib.agft_abi_version.restype = ctypes.c_int
    lib.agft_abi_version.argtypes = []
    lib.agft_launch_shape_for.restype = ctypes.c_int
    lib.agft_launch_shape_for.argtypes = [cfgp, ctypes.POINTER(agft_launch_shape)]
    lib.agft_env_state_bytes.restype = _sz
    lib.agft_env_state_bytes.argtypes = [envp]
    lib.agft_env_reset.restype = ctypes.c_int
    lib.agft_env_reset.argtypes = [envp, _vp, _sz, _vp, _vp, _vp, _vp]
    lib.agft_env_step.restype = ctypes.c_int
    lib.agft_env_step.argtypes = [envp, _vp, _sz, _i32, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.agft_sim_step.restype = ctypes.c_int
    lib.agft_sim_step.argtypes = [_vp, envp, _vp, _sz, _vp, _vp, _vp, _vp, _vp, _vp]
    return lib


def lib():
    """The loaded libagft.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2508_01744_amd._build` (hipcc, gfx950)")
        handle = _declare(ctypes.CDLL(LIB_PATH))
        if handle.agft_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {handle.agft_abi_version()}, these "
                               f"bindings expect {ABI_VERSION}: rebuild it")
        _lib = handle
    return _lib


def check(fn, code):
    if code != AGFT_OK:
        raise AgftError(fn, code)
    return code


# Same names as the C ABI.

def agft_state_bytes(cfg):
    return lib().agft_state_bytes(ctypes.byref(cfg))


def agft_create(cfg, d_state, nbytes, stream):
    h = _vp()
    code = lib().agft_create(ctypes.byref(cfg), d_state, nbytes, stream, ctypes.byref(h))
    return code, h


def agft_step(h, d_ctx, d_reward, d_action, d_scores):
    return lib().agft_step(h, d_ctx, d_reward, d_action, d_scores)


def agft_get_state(h):
    view = agft_state_view()
    code = lib().agft_get_state(h, ctypes.byref(view))
    return code, view


def agft_export(h, d_theta, d_ainv):
    return lib().agft_export(h, d_theta, d_ainv)


def agft_set_stream(h, stream):
    return lib().agft_set_stream(h, stream)


def agft_destroy(h):
    return lib().agft_destroy(h)


def agft_strerror(code):
    return lib().agft_strerror(code).decode()


def agft_abi_version():
    return lib().agft_abi_version()


def agft_launch_shape_for(cfg):
    shape = agft_launch_shape()
    code = lib().agft_launch_shape_for(ctypes.byref(cfg), ctypes.byref(shape))
    return code, shape


def agft_env_state_bytes(cfg):
    return lib().agft_env_state_bytes(ctypes.byref(cfg))


def agft_env_reset(cfg, d_env, nbytes, d_arrivals, d_noise, d_ctx, stream):
    return lib().agft_env_reset(ctypes.byref(cfg), d_env, nbytes, d_arrivals, d_noise, d_ctx, stream)


def agft_env_step(cfg, d_env, nbytes, t, d_action, d_arrivals, d_noise, d_reward, d_ctx, stream):
    return lib().agft_env_step(ctypes.byref(cfg), d_env, nbytes, t, d_action, d_arrivals, d_noise,
                               d_reward, d_ctx, stream)


def agft_sim_step(h, env_cfg, d_env, env_nbytes, d_arrivals, d_noise, d_ctx, d_reward, d_action, d_scores):
    return lib().agft_sim_step(h, ctypes.byref(env_cfg), d_env, env_nbytes, d_arrivals, d_noise, d_ctx,
                               d_reward, d_action, d_scores)
