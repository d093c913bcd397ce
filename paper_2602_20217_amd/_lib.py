"""ctypes binding of libknapspec.so: the structures of include/knapspec.h and the
entry points under the same names.  Argument marshalling only; every step of
the decode path runs in the library's HIP kernels.  Importing this module loads
the library and fails loudly when it has not been built."""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# KNAPSPEC_LIB selects another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("KNAPSPEC_LIB") or os.path.join(HERE, "libknapspec.so")

KS_OK, KS_EINVAL, KS_ENOMEM, KS_ECAPACITY, KS_ESTATE, KS_EHIP = 0, -1, -2, -3, -4, -5
KS_F32, KS_BF16 = 0, 1
KS_QUANT_PAPER_MIN, KS_QUANT_BINS = 0, 1
KS_MAX_SUBLAYERS = 256

STATUS_NAMES = {0: "KS_OK", -1: "KS_EINVAL", -2: "KS_ENOMEM", -3: "KS_ECAPACITY",
                -4: "KS_ESTATE", -5: "KS_EHIP"}


class ModelDesc(C.Structure):
    _fields_ = [("L", C.c_int), ("d", C.c_int), ("hq", C.c_int), ("hkv", C.c_int),
                ("hd", C.c_int), ("ffn", C.c_int), ("vocab", C.c_int), ("n_max", C.c_int),
                ("qk_norm", C.c_int), ("dtype", C.c_int), ("eps", C.c_float),
                ("rope_theta", C.c_double)]


class Limits(C.Structure):
    _fields_ = [("gamma_max", C.c_int), ("m_rounds", C.c_int), ("cap_max", C.c_int),
                ("prefill_chunk", C.c_int)]


_VPP = C.POINTER(C.c_void_p)


class Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("lm_head", C.c_void_p), ("final_norm", C.c_void_p),
                ("attn_norm", _VPP), ("wqkv", _VPP), ("wo", _VPP), ("q_norm", _VPP),
                ("k_norm", _VPP), ("mlp_norm", _VPP), ("w_gate_up", _VPP), ("w_down", _VPP)]


class SelectParams(C.Structure):
    _fields_ = [("c1", C.c_double), ("c2", C.c_double), ("c3", C.c_double),
                ("quant_mode", C.c_int), ("bins", C.c_int), ("tau", C.c_float),
                ("prune_half", C.c_int), ("D", C.c_int), ("t_head", C.c_double)]


class Selection(C.Structure):
    _fields_ = [("exec", C.c_uint8 * KS_MAX_SUBLAYERS), ("j_star", C.c_int),
                ("gamma_star", C.c_int), ("C", C.c_int), ("w_attn", C.c_int), ("w_mlp", C.c_int),
                ("n_rows", C.c_int), ("n_cells", C.c_int), ("tpt_star", C.c_double),
                ("alpha_hat", C.c_double), ("delta", C.c_double), ("iv_rounds", C.c_int),
                ("iv_drafted", C.c_int), ("iv_accepted", C.c_int), ("iv_tokens", C.c_int),
                ("iv_ms", C.c_double)]


class SelectionDebug(C.Structure):
    _fields_ = [("J_cap", C.c_int), ("bits", C.POINTER(C.c_uint8)),
                ("reach", C.POINTER(C.c_uint8)), ("sig_e", C.POINTER(C.c_double)),
                ("sig_s", C.POINTER(C.c_double)), ("n_match", C.POINTER(C.c_int))]


KS_GAMMA_FIXED, KS_GAMMA_SELECTED = 0, 1


class DraftPolicy(C.Structure):
    _fields_ = [("tau_conf", C.c_float), ("gamma_source", C.c_int)]


KS_SAMPLE_KMAX = 128


class Sampling(C.Structure):
    _fields_ = [("temperature", C.c_float), ("top_k", C.c_int), ("top_p", C.c_float),
                ("seed", C.c_uint64)]


class GenStats(C.Structure):
    _fields_ = [("n_rounds", C.c_int), ("n_selections", C.c_int), ("n_drafted", C.c_int),
                ("n_accepted", C.c_int), ("ms_total", C.c_double), ("ms_select", C.c_double),
                ("ms_prefill", C.c_double)]


KS_KC_NAMES = ("embed", "norm", "gemm_qkv", "qkv_post", "attn", "combine", "gemm_o",
               "gemm_gate_up", "gemm_down", "gemm_head", "argmax", "other")
KS_KC_COUNT = len(KS_KC_NAMES)


class KernelProfile(C.Structure):
    _fields_ = [("ms", C.c_double * KS_KC_COUNT), ("launches", C.c_int * KS_KC_COUNT),
                ("ms_step", C.c_double), ("steps", C.c_int)]


class KsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _load():
    # PyTorch ships its own HIP runtime (same SONAME as the system one).  Loading
    # torch first makes the dynamic loader bind the library to that runtime, so
    # device pointers and streams from torch are valid in the library's calls;
    # loading the library first would bring a second HIP runtime into the process.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2602_20217_amd.build` (hipcc, gfx950)")
    return C.CDLL(LIB_PATH)


lib = _load()

_P = C.c_void_p
_I = C.c_int
_SIG = {
    "ks_last_error": (C.c_char_p, []),
    "ks_kv_cache_bytes": (C.c_size_t, [C.POINTER(ModelDesc)]),
    "ks_workspace_bytes": (C.c_size_t, [C.POINTER(ModelDesc), C.POINTER(Limits)]),
    "ks_pack_matrix": (_I, [_P, _P, _I, _I, _I, _P]),
    "ks_pack_gate_up": (_I, [_P, _P, _P, _I, _I, _I, _P]),
    "ks_pack_qkv": (_I, [_P, _P, _I, _I, _I, _I, _I, _P]),
    "ks_create": (_I, [C.POINTER(ModelDesc), C.POINTER(Limits), C.POINTER(Weights), _P,
                       C.c_size_t, _P, C.c_size_t, _P, C.POINTER(_P)]),
    "ks_destroy": (_I, [_P]),
    "ks_prefill": (_I, [_P, _P, _I, C.POINTER(C.c_int32)]),
    "ks_set_context": (_I, [_P, _I, C.c_int32]),
    "ks_draft_step": (_I, [_P, _P, C.POINTER(C.c_int32), C.POINTER(C.c_float)]),
    "ks_verify": (_I, [_P, _P, _I, _P, C.POINTER(C.c_int)]),
    "ks_hidden_cos": (_I, [_P, _P, _I, _I, _I, _P, _P]),
    "ks_knapsack_select": (_I, [_P, C.POINTER(SelectParams), C.POINTER(Selection),
                                C.POINTER(SelectionDebug)]),
    "ks_generate": (_I, [_P, _P, _I, _I, _I, _I, C.POINTER(SelectParams), _P,
                         C.POINTER(GenStats), C.POINTER(Selection), _I]),
    "ks_decode": (_I, [_P, _I, _I, _I, C.POINTER(SelectParams), _P, C.POINTER(GenStats),
                       C.POINTER(Selection), _I]),
    "ks_set_draft_policy": (_I, [_P, C.POINTER(DraftPolicy)]),
    "ks_set_sampling": (_I, [_P, C.POINTER(Sampling)]),
    "ks_sample_workspace_bytes": (C.c_size_t, [_I, _I, _I]),
    "ks_sample_filter": (_I, [_P, _I, _I, _I, C.POINTER(Sampling), _I, _I, _P, _P, _P, _P, _P,
                              _P, C.c_size_t, _P]),
    "ks_sample_filter_noalloc": (_I, [_P, _I, _I, _I, C.POINTER(Sampling), _I, _I, _P, _P, _P,
                                      _P, _P, _P]),
    "ks_spec_accept": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, C.c_uint64, _I, _P, _P]),
    "ks_sample_uniforms": (_I, [C.c_uint64, _P, _I, _I, _P, _P]),
    "ks_profile_decode": (_I, [_P, _P, _I, _I, C.POINTER(KernelProfile)]),
    "ks_time_launches": (_I, [_P, _P]),
    "ks_sublayer_apply": (_I, [_P, _I, _P, _P, _P, _I, _I]),
    "ks_head_rows": (_I, [_P, _P, _I, _P, _P, _P]),
    "ks_knapsack_quantize": (_I, [_P, _P, _I, _I, _I, _P, _P]),
    "ks_knapsack_batch": (_I, [_P, _P, _I, _I, _I, _I, _P, _P, _P]),
    "ks_knapsack_backtrack": (_I, [_P, _P, _I, _I, _I, _P, _P, _P, _P]),
    "ks_knapsack_batch_select": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "ks_stream_read": (_I, [_P, C.c_size_t, _P, _P]),
}
EXPORTS = tuple(_SIG)

for _name, (_res, _args) in _SIG.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def last_error() -> str:
    return lib.ks_last_error().decode()


def check(status: int):
    if status != KS_OK:
        raise KsError(status, last_error())
    return status


def _wrap(name):
    f = getattr(lib, name)

    def call(*args):
        return check(f(*args))

    call.__name__ = name
    return call


# the same names as the C ABI; status-returning calls raise KsError on failure
ks_pack_matrix = _wrap("ks_pack_matrix")
ks_pack_gate_up = _wrap("ks_pack_gate_up")
ks_pack_qkv = _wrap("ks_pack_qkv")
ks_create = _wrap("ks_create")
ks_destroy = _wrap("ks_destroy")
ks_prefill = _wrap("ks_prefill")
ks_set_context = _wrap("ks_set_context")
ks_draft_step = _wrap("ks_draft_step")
ks_verify = _wrap("ks_verify")
ks_hidden_cos = _wrap("ks_hidden_cos")
ks_knapsack_select = _wrap("ks_knapsack_select")
ks_generate = _wrap("ks_generate")
ks_decode = _wrap("ks_decode")
ks_set_draft_policy = _wrap("ks_set_draft_policy")
ks_set_sampling = _wrap("ks_set_sampling")
ks_sample_filter = _wrap("ks_sample_filter")
ks_sample_filter_noalloc = _wrap("ks_sample_filter_noalloc")
ks_spec_accept = _wrap("ks_spec_accept")
ks_sample_uniforms = _wrap("ks_sample_uniforms")
ks_sample_workspace_bytes = lib.ks_sample_workspace_bytes
ks_profile_decode = _wrap("ks_profile_decode")
ks_time_launches = _wrap("ks_time_launches")
ks_sublayer_apply = _wrap("ks_sublayer_apply")
ks_head_rows = _wrap("ks_head_rows")
ks_knapsack_quantize = _wrap("ks_knapsack_quantize")
ks_knapsack_batch = _wrap("ks_knapsack_batch")
ks_knapsack_backtrack = _wrap("ks_knapsack_backtrack")
ks_knapsack_batch_select = _wrap("ks_knapsack_batch_select")
ks_stream_read = _wrap("ks_stream_read")
ks_kv_cache_bytes = lib.ks_kv_cache_bytes
ks_workspace_bytes = lib.ks_workspace_bytes
