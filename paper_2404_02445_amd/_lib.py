"""ctypes declarations of include/mopar.h and the loader of libmopar.so.

Argument marshalling only: every computation happens in the library.  The
library must have been built (``paper_2404_02445_amd.build``); a missing
library is an error, never a fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmopar.so")

c_i32, c_i64, c_f32, c_f64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_void_p

MOPAR_OK, MOPAR_E_ARG, MOPAR_E_SHAPE, MOPAR_E_DTYPE, MOPAR_E_UNSUPPORTED = 0, 1, 2, 3, 4
MOPAR_E_INFEASIBLE, MOPAR_E_WORKSPACE, MOPAR_E_HIP = 5, 6, 7
MOPAR_F32, MOPAR_BF16, MOPAR_I32 = 0, 1, 2
OP_CONV, OP_LINEAR, OP_MAXPOOL, OP_AVGPOOL, OP_LAYERNORM = 1, 2, 3, 4, 5
OP_ATTENTION, OP_EMBED_BERT, OP_EMBED, OP_LSTM = 6, 7, 8, 9
ACT = {"none": 0, "relu": 1, "gelu": 2}
CODEC_RAW, CODEC_AE = 0, 1
# MOPAR_STATIC_WORKSPACE_BYTES of include/mopar.h: the static workspace of mopar_model_forward_static
STATIC_WORKSPACE_BYTES = 64 << 20
STATUS_NAMES = {0: "OK", 1: "E_ARG", 2: "E_SHAPE", 3: "E_DTYPE", 4: "E_UNSUPPORTED", 5: "E_INFEASIBLE",
                6: "E_WORKSPACE", 7: "E_HIP"}


class LayerProfile(ctypes.Structure):
    _fields_ = [("mem_bytes", c_f64), ("time_s", c_f64), ("out_bytes", c_f64), ("rd_width", c_i32),
                ("reserved", c_i32)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("n_slices", c_i32), ("k_max", c_i32), ("allowed_cut", ctypes.POINTER(ctypes.c_uint8)),
                ("elim_tau", c_f64), ("c_m", c_f64), ("c_n", c_f64), ("bw_Bps", c_f64),
                ("ratio", ctypes.POINTER(c_f64)), ("lambda_bytes", c_f64), ("tp_table", ctypes.POINTER(c_f64)),
                ("ta_table", ctypes.POINTER(c_f64)), ("k_override", ctypes.POINTER(c_i32)),
                ("uniform", c_i32), ("reserved", c_i32)]


class Plan(ctypes.Structure):
    _fields_ = [("n_layers", c_i32), ("n_slices", c_i32), ("slice_end", ctypes.POINTER(c_i32)),
                ("k", ctypes.POINTER(c_i32)), ("cost", c_f64), ("t_tau", c_f64), ("t_unsplit", c_f64),
                ("latency_ok", c_i32), ("reserved", c_i32)]


class TensorDesc(ctypes.Structure):
    _fields_ = [("dtype", c_i32), ("rank", c_i32), ("dims", c_i64 * 4)]


class Op(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("act", c_i32), ("layer", c_i32), ("branch", c_i32), ("pos", c_i32),
                ("rd", c_i32), ("in0", c_i32), ("in1", c_i32), ("out", c_i32), ("kh", c_i32), ("kw", c_i32),
                ("stride", c_i32), ("pad", c_i32), ("heads", c_i32), ("n_out", c_i32), ("out_off", c_i32),
                ("eps", c_f32), ("scale", c_f32), ("rows", c_i64 * 3), ("w", c_i64), ("b", c_i64),
                ("w2", c_i64), ("w3", c_i64), ("w4", c_i64), ("w5", c_i64)]


class ModelDesc(ctypes.Structure):
    _fields_ = [("dtype", c_i32), ("n_tensors", c_i32), ("tensors", ctypes.POINTER(TensorDesc)),
                ("n_ops", c_i32), ("ops", ctypes.POINTER(Op)), ("n_layers", c_i32), ("input", c_i32),
                ("output", c_i32)]


class Codec(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("c", c_i32), ("c_code", c_i32), ("reserved", c_i32), ("w_enc", c_vp),
                ("b_enc", c_vp), ("w_dec", c_vp), ("b_dec", c_vp)]


# every exported symbol of include/mopar.h, with its signature
SIGNATURES = {
    "mopar_subslice_range": (c_i32, [c_i32, c_i32, c_i32, ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]),
    "mopar_plan_slices": (c_i32, [ctypes.POINTER(LayerProfile), c_i32, ctypes.POINTER(PlanOpts), ctypes.POINTER(Plan)]),
    "mopar_model_create": (c_i32, [ctypes.POINTER(ModelDesc), c_vp, ctypes.c_size_t, ctypes.POINTER(c_vp)]),
    "mopar_model_destroy": (None, [c_vp]),
    "mopar_model_profile": (c_i32, [c_vp, ctypes.POINTER(LayerProfile)]),
    "mopar_model_workspace_bytes": (c_i32, [c_vp, ctypes.POINTER(Plan), ctypes.POINTER(ctypes.c_size_t)]),
    "mopar_slice_forward": (c_i32, [c_vp, ctypes.POINTER(Plan), c_i32, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "mopar_boundary_code_bytes": (c_i32, [ctypes.POINTER(Codec), ctypes.POINTER(TensorDesc),
                                          ctypes.POINTER(ctypes.c_size_t)]),
    "mopar_boundary_encode": (c_i32, [ctypes.POINTER(Codec), ctypes.POINTER(TensorDesc), c_vp, c_vp, c_vp]),
    "mopar_boundary_decode": (c_i32, [ctypes.POINTER(Codec), ctypes.POINTER(TensorDesc), c_vp, c_vp, c_vp]),
    "mopar_model_forward": (c_i32, [c_vp, ctypes.POINTER(Plan), ctypes.POINTER(Codec), c_vp, c_vp,
                                    ctypes.POINTER(c_vp), c_vp, ctypes.c_size_t, c_vp]),
    "mopar_model_forward_static": (c_i32, [c_vp, ctypes.POINTER(Plan), ctypes.POINTER(Codec), c_vp, c_vp,
                                           ctypes.POINTER(c_vp), c_vp]),
    "mopar_pipeline_workspace_bytes": (c_i32, [c_vp, ctypes.POINTER(Plan), c_i32, ctypes.POINTER(ctypes.c_size_t)]),
    "mopar_pipeline_create": (c_i32, [c_vp, ctypes.POINTER(Plan), ctypes.POINTER(Codec), c_i32, c_i32,
                                      ctypes.POINTER(c_vp), c_vp, ctypes.c_size_t, ctypes.POINTER(c_vp),
                                      ctypes.POINTER(c_vp)]),
    "mopar_pipeline_submit": (c_i32, [c_vp, c_vp, c_vp]),
    "mopar_pipeline_use_graphs": (c_i32, [c_vp, c_i32]),
    "mopar_pipeline_destroy": (None, [c_vp]),
    "mopar_model_set_timing": (c_i32, [c_vp, c_i32]),
    "mopar_model_timing_slots": (c_i32, [c_vp, ctypes.POINTER(c_i32)]),
    "mopar_model_op_times": (c_i32, [c_vp, ctypes.POINTER(c_f32), c_i32]),
    "mopar_model_profile_dominant": (c_i32, [c_vp, c_f64, ctypes.POINTER(LayerProfile)]),
    "mopar_model_cut_tensors": (c_i32, [c_vp, c_i32, ctypes.POINTER(c_i32), c_i32, ctypes.POINTER(c_i32)]),
    "mopar_model_measure": (c_i32, [c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp,
                                    ctypes.POINTER(c_f64)]),
    "mopar_last_error": (ctypes.c_char_p, []),
    "mopar_version": (ctypes.c_char_p, []),
}

_lib = None


class MoparError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib():
    """Load libmopar.so (built in-tree).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2404_02445_amd.build` "
                               "(there is no non-HIP fallback)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status):
    if status != MOPAR_OK:
        raise MoparError(status, lib().mopar_last_error().decode())
    return status
