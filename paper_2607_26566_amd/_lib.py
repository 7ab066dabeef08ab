"""ctypes declarations of ``libt2i_dit.so`` (``include/t2i_dit.h``, ``include/t2i_ops.h``).

Argument marshalling only.  Loading fails loudly when the library has not been
built: there is no fallback implementation of any step.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libt2i_dit.so")

T2I_OK = 0
T2I_F32, T2I_BF16 = 0, 1
T2I_ARCH_CROSS_DIT, T2I_ARCH_MMDIT = 0, 1
T2I_CACHE_ACCUMULATE, T2I_CACHE_PER_STEP = 0, 1
T2I_EPI_STORE, T2I_EPI_GELU, T2I_EPI_SILU, T2I_EPI_RESID, T2I_EPI_RESID_GATED = range(5)
T2I_MAX_SEQ, T2I_MAX_REQ = 64, 32

KERNEL_CLASSES = ["gemm_qkv", "attn_self", "gemm_o", "gemm_xq", "attn_cross", "gemm_xo",
                  "ln_mod", "gemm_fc1", "gemm_fc2", "embed", "final", "cache"]

STATUS_NAMES = {0: "T2I_OK", 1: "T2I_ERR_INVALID_ARG", 2: "T2I_ERR_SHAPE",
                3: "T2I_ERR_UNSUPPORTED", 4: "T2I_ERR_WORKSPACE",
                5: "T2I_ERR_OUT_OF_MEMORY", 6: "T2I_ERR_DEVICE"}

i32, u32, i64, f32, f64, u8 = C.c_int32, C.c_uint32, C.c_int64, C.c_float, C.c_double, C.c_uint8
vp, sz = C.c_void_p, C.c_size_t


class t2i_dit_config(C.Structure):
    _fields_ = [("struct_size", u32), ("arch", i32), ("dtype", i32),
                ("latent_channels", i32), ("patch", i32), ("hidden", i32), ("heads", i32),
                ("head_dim", i32), ("depth", i32), ("mlp_hidden", i32), ("text_dim", i32),
                ("text_tokens", i32), ("freq_dim", i32), ("max_tokens", i32),
                ("max_requests", i32), ("max_steps", i32), ("ln_eps", f32), ("t_scale", f32)]


class t2i_control(C.Structure):
    _fields_ = [("struct_size", u32), ("n", i32), ("blocks", C.POINTER(i32)),
                ("residuals", C.POINTER(vp)), ("ready", C.POINTER(vp))]


class t2i_step_args(C.Structure):
    _fields_ = [("struct_size", u32), ("n_req", i32), ("lat_h", C.POINTER(i32)),
                ("lat_w", C.POINTER(i32)), ("t", C.POINTER(f64)), ("t_next", C.POINTER(f64)),
                ("latents", vp), ("prompt_embeds", vp), ("guidance", f32), ("noise_pred", vp),
                ("n_blocks", i32), ("hidden_out", vp), ("skip", C.POINTER(u8)),
                ("cache_state", vp), ("cache_state_bytes", sz), ("control_outputs", vp)]


class t2i_cache_args(C.Structure):
    _fields_ = [("struct_size", u32), ("n_req", i32), ("lat_h", C.POINTER(i32)),
                ("lat_w", C.POINTER(i32)), ("t", C.POINTER(f64)), ("latents", vp),
                ("step", i32), ("n_steps", i32), ("tau", f64), ("mode", i32),
                ("branches", i32), ("cache_state", vp), ("cache_state_bytes", sz),
                ("rel_l1", C.POINTER(f64)), ("skip", C.POINTER(u8))]


class t2i_sample_args(C.Structure):
    _fields_ = [("struct_size", u32), ("n_req", i32), ("lat_h", C.POINTER(i32)),
                ("lat_w", C.POINTER(i32)), ("n_steps", i32), ("start_step", i32),
                ("timesteps", C.POINTER(f64)), ("latents", vp), ("prompt_embeds", vp),
                ("guidance", f32), ("cache_tau", f64), ("cache_mode", i32),
                ("cache_state", vp), ("cache_state_bytes", sz),
                ("skip_log", C.POINTER(u8)), ("rel_l1_log", C.POINTER(f64))]


# name -> (restype, argtypes); every symbol the two headers declare
SIGNATURES = {
    "t2i_dit_weight_count": (sz, [C.POINTER(t2i_dit_config)]),
    "t2i_dit_weight_desc": (i32, [C.POINTER(t2i_dit_config), sz, C.c_char_p,
                                  C.POINTER(i64), C.POINTER(i32)]),
    "t2i_dit_workspace_bytes": (sz, [C.POINTER(t2i_dit_config)]),
    "t2i_cache_state_bytes": (sz, [C.POINTER(t2i_dit_config), i32, C.POINTER(i32), i32]),
    "t2i_dit_init": (i32, [C.POINTER(t2i_dit_config), C.POINTER(vp), vp, sz, vp,
                           C.POINTER(vp)]),
    "t2i_dit_init_static": (i32, [C.POINTER(t2i_dit_config), C.POINTER(vp), vp, C.POINTER(vp)]),
    "t2i_dit_rebind_weights": (i32, [vp, C.POINTER(vp), vp]),
    "t2i_dit_block_layout": (sz, [C.POINTER(t2i_dit_config), C.POINTER(i32), C.POINTER(i32),
                                  C.POINTER(sz)]),
    "t2i_dit_host_tier": (i32, [vp, vp, vp, sz]),
    "t2i_dit_evict": (i32, [vp, i32]),
    "t2i_dit_load_async": (i32, [vp, vp, C.POINTER(i32)]),
    "t2i_dit_block_state": (i32, [vp, C.POINTER(i32)]),
    "t2i_first_layers": (i32, [i32, f64, f64]),
    "t2i_dit_step": (i32, [vp, C.POINTER(t2i_step_args), vp]),
    "t2i_cache_check": (i32, [vp, C.POINTER(t2i_cache_args), vp]),
    "t2i_dit_sample": (i32, [vp, C.POINTER(t2i_sample_args), vp]),
    "t2i_dit_destroy": (None, [vp]),
    "t2i_dit_profile": (i32, [vp, u32]),
    "t2i_dit_profile_read": (i32, [vp, i32, C.POINTER(f64), C.POINTER(i64)]),
    "t2i_status_str": (C.c_char_p, [i32]),
    "t2i_last_error": (C.c_char_p, [vp]),
    "t2i_op_linear": (i32, [i32, i32, i32, i32, i32, vp, i32, vp, i32, vp, vp, i32, vp, i32,
                            vp, vp, vp]),
    "t2i_op_attention": (i32, [i32, i32, i32, i32, C.POINTER(i32), C.POINTER(i32),
                               C.POINTER(i32), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32),
                               vp, i32, vp, i32, vp, i32, vp, i32, vp]),
    "t2i_op_cross_attention": (i32, [i32, i32, i32, i32, C.POINTER(i32), C.POINTER(i32),
                                     C.POINTER(i32), C.POINTER(i32), vp, i32, vp, i32, vp, i32,
                                     vp, i32, vp]),
    "t2i_op_linear_cross_attention": (i32, [i32, i32, i32, i32, C.POINTER(i32), C.POINTER(i32),
                                            C.POINTER(i32), C.POINTER(i32), i32, vp, i32, vp,
                                            i32, vp, vp, i32, vp, i32, vp, i32, vp, i32, vp]),
    "t2i_op_ln_modulate": (i32, [i32, i32, i32, vp, vp, vp, f32, vp, vp]),
    "t2i_op_dma_read": (i32, [vp, sz, vp, vp]),
    "t2i_op_lora_merge_batch": (i32, [i32, i32, i32, i32, i32, f32, C.POINTER(vp), i32,
                                      C.POINTER(vp), C.POINTER(vp), vp]),
    "t2i_op_lora_merge": (i32, [i32, i32, i32, i32, f32, vp, i32, vp, vp, vp]),
    "t2i_sched_create": (i32, [f64, C.POINTER(vp)]),
    "t2i_sched_destroy": (None, [vp]),
    "t2i_sched_submit": (i32, [vp, i32, C.c_int64, f64, f64, f64]),
    "t2i_sched_schedule": (i32, [vp, f64, C.POINTER(i32), C.POINTER(C.c_int64), C.POINTER(i32),
                                 C.POINTER(f64)]),
    "t2i_sched_complete": (i32, [vp, C.c_int64, f64]),
    "t2i_sched_vtime": (i32, [vp, i32, C.POINTER(f64)]),
    "t2i_ops_last_error": (C.c_char_p, []),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load the library (once).  Raises if it is missing: build it first."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is not built; run `python -m paper_2607_26566_amd.build` "
            "(the HIP library is the only implementation of the denoising step)")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class T2IError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def check(status: int, handle=None):
    if status != T2I_OK:
        lib = load()
        msg = (lib.t2i_last_error(handle) if handle else lib.t2i_ops_last_error()) or b""
        raise T2IError(status, msg.decode())
