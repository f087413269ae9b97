"""ctypes binding of libfeatfix.so: the C ABI of include/featfix.h under the same names.

Argument marshalling only -- every step of the denoising path runs in the library's
HIP kernels.  Device buffers are passed as integer addresses (e.g. torch's
``tensor.data_ptr()``) and streams as integer HIP stream handles (0 = default stream).
Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfeatfix.so")

FF_OK, FF_E_NULL, FF_E_SHAPE, FF_E_DTYPE, FF_E_RANGE, FF_E_STATE, FF_E_WORKSPACE, FF_E_HIP, \
    FF_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6, -7, -8
FF_DIT, FF_MMDIT_DOUBLE, FF_MMDIT_SINGLE = 0, 1, 2
FF_ABI_VERSION = 3          # the struct layouts below; must equal the library's
FF_F32, FF_BF16 = 0, 1
FF_VANILLA, FF_DRAFT, FF_VERIFY, FF_FEATFIX, FF_EXACT_ONLY = 0, 1, 2, 3, 4
FF_TOKENS_PARTIAL, FF_CHANNELS_PARTIAL, FF_RECOMPUTE = 5, 6, 7
FF_FWD_DRAFT, FF_FWD_EXACT, FF_FWD_TOKENS, FF_FWD_CHANNELS = 0, 1, 2, 3
FF_RESIDUAL, FF_OUTPUT = 0, 1
FF_STEP_REFRESH, FF_STEP_CACHED = 0, 1
FF_ACT_EXACT, FF_ACT_DRAFT, FF_ACT_SITE, FF_ACT_RECOMPUTE = 0, 1, 2, 3
FF_MAX_K, FF_MAX_SLOTS, FF_TEMB_DIM = 3, 8, 256
FF_NOALLOC_VERIFY_MAX_B = 16

# every symbol include/featfix.h declares
EXPORTED = ("ff_abi_version", "ff_last_error", "ff_plan_build", "ff_plan_destroy", "ff_plan_export",
            "ff_cache_bytes", "ff_workspace_bytes", "ff_block_exact", "ff_cache_update",
            "ff_draft_forecast", "ff_verify_replace", "ff_verify_replace_noalloc", "ff_ctx_create", "ff_ctx_destroy",
            "ff_ctx_reset", "ff_get_counts", "ff_ctx_step_kinds", "ff_denoise_step", "ff_ctx_trace", "ff_hist_sum_bytes", "ff_ctx_hist_sums", "ff_cond_cache_bytes", "ff_ctx_cond_cache", "ff_rel_l1",
            "ff_ctx_profile", "ff_ctx_profile_read")
PROF_CLASSES = ("gemm", "attn", "norm", "gemv", "draft", "verify", "cache", "other")


class ff_model_desc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("kinds", C.POINTER(C.c_int32)),
                ("C", C.c_int32), ("H", C.c_int32), ("d", C.c_int32), ("mlp_hidden", C.c_int32),
                ("n_img", C.c_int32), ("n_txt", C.c_int32), ("B", C.c_int32),
                ("lat_c", C.c_int32), ("lat_f", C.c_int32), ("lat_h", C.c_int32), ("lat_w", C.c_int32),
                ("pt", C.c_int32), ("ph", C.c_int32), ("pw", C.c_int32),
                ("dtype", C.c_int32), ("ln_eps", C.c_float), ("rope_axes", C.c_int32 * 3), ("rope_theta", C.c_float),
                ("cfg_pairs", C.c_int32), ("cfg_scale", C.c_float)]


_STREAM_FIELDS = ("mod_w", "mod_b", "qkv_w", "qkv_b", "o_w", "o_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b",
                  "lin1_w", "lin1_b", "lin2_w", "lin2_b", "q_g", "k_g")


class ff_stream_weights(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in _STREAM_FIELDS]


class ff_layer_weights(C.Structure):
    _fields_ = [("s", ff_stream_weights * 2)]


_GLOBAL_FIELDS = ("t1_w", "t1_b", "t2_w", "t2_b", "pe_w", "pe_b", "fmod_w", "fmod_b", "f_w", "f_b")


class ff_global_weights(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in _GLOBAL_FIELDS]


class ff_sched_desc(C.Structure):
    _fields_ = [("T", C.c_int32), ("R", C.c_int32), ("K", C.c_int32), ("S", C.c_int32),
                ("eps", C.c_float), ("mode", C.c_int32), ("feature_mode", C.c_int32), ("tau", C.c_float),
                ("part_stride", C.c_int32)]


class ff_counts(C.Structure):
    _fields_ = [("n_full_refresh", C.c_int64), ("n_paid_checks", C.c_int64), ("n_forwarded", C.c_int64),
                ("n_recomputed", C.c_int64)]

    def as_dict(self):
        return {"n_full_refresh": self.n_full_refresh, "n_paid_checks": self.n_paid_checks,
                "n_forwarded": self.n_forwarded, "n_recomputed": self.n_recomputed}


class ff_prof_stat(C.Structure):
    _fields_ = [("launches", C.c_int64), ("ms", C.c_double), ("flops", C.c_double), ("bytes", C.c_double)]


class FFError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"featfix error {status}: {msg}")
        self.status = status


_lib = None


def lib():
    """The loaded library (raises if it has not been built: there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_27842_amd.build`")
        L = C.CDLL(LIB_PATH)
        vp, i32, sz, f32 = C.c_void_p, C.c_int32, C.c_size_t, C.c_float
        P = C.POINTER
        sig = {
            "ff_abi_version": (i32, []),
            "ff_last_error": (C.c_char_p, []),
            "ff_plan_build": (i32, [P(ff_sched_desc), i32, P(C.c_uint8), P(vp)]),
            "ff_plan_destroy": (None, [vp]),
            "ff_plan_export": (i32, [vp, P(i32), P(i32), P(i32), P(i32), P(i32), P(i32), P(C.c_float),
                                     P(ff_counts)]),
            "ff_cache_bytes": (sz, [P(ff_model_desc), i32]),
            "ff_workspace_bytes": (sz, [P(ff_model_desc)]),
            "ff_block_exact": (i32, [P(ff_model_desc), i32, P(ff_layer_weights), vp, vp, vp, vp, sz, vp]),
            "ff_cache_update": (i32, [P(ff_model_desc), vp, i32, i32, i32, vp, vp, i32, vp]),
            "ff_draft_forecast": (i32, [P(ff_model_desc), vp, i32, i32, i32, P(i32), P(C.c_float), vp, vp, vp]),
            "ff_verify_replace": (i32, [P(ff_model_desc), vp, i32, i32, i32, P(i32), P(C.c_float), vp, vp, vp,
                                        i32, i32, f32, vp, vp, sz, vp]),
            "ff_verify_replace_noalloc": (i32, [P(ff_model_desc), vp, i32, i32, i32, P(i32), P(C.c_float), vp, vp,
                                                vp, i32, i32, f32, vp, vp]),
            "ff_ctx_create": (i32, [P(ff_model_desc), P(ff_layer_weights), P(ff_global_weights), vp, vp, sz,
                                    vp, sz, P(vp)]),
            "ff_ctx_destroy": (None, [vp]),
            "ff_ctx_reset": (i32, [vp]),
            "ff_get_counts": (i32, [vp, P(ff_counts)]),
            "ff_ctx_step_kinds": (i32, [vp, P(i32)]),
            "ff_ctx_trace": (i32, [vp, vp, sz]),
            "ff_hist_sum_bytes": (sz, [P(ff_model_desc), vp]),
            "ff_ctx_hist_sums": (i32, [vp, vp, sz]),
            "ff_cond_cache_bytes": (sz, [P(ff_model_desc), vp]),
            "ff_ctx_cond_cache": (i32, [vp, vp, sz]),
            "ff_rel_l1": (i32, [P(ff_model_desc), vp, vp, f32, vp, vp, sz, vp]),
            "ff_denoise_step": (i32, [vp, i32, vp, vp, vp, vp, vp]),
            "ff_ctx_profile": (i32, [vp, i32]),
            "ff_ctx_profile_read": (i32, [vp, P(ff_prof_stat)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        if L.ff_abi_version() != FF_ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {L.ff_abi_version()}, the binding expects "
                               f"{FF_ABI_VERSION}: rebuild it")
        _lib = L
    return _lib


def check(status):
    if status != FF_OK:
        raise FFError(status, lib().ff_last_error().decode())
    return status


def _i32arr(vals):
    vals = list(vals)
    return (C.c_int32 * max(1, len(vals)))(*vals)


def _f32arr(vals):
    vals = list(vals)
    return (C.c_float * max(1, len(vals)))(*vals)


# ------------------------------------------------------------------ thin wrappers (same names)

def ff_abi_version():
    return lib().ff_abi_version()


def ff_last_error():
    return lib().ff_last_error().decode()


def ff_plan_build(sched, n_layers, site_mask):
    """sched: ff_sched_desc; site_mask: uint8 sequence/array [T*L] (step-major). Returns a handle."""
    import numpy as np
    m = np.ascontiguousarray(np.asarray(site_mask, dtype=np.uint8).reshape(-1))
    out = C.c_void_p()
    check(lib().ff_plan_build(C.byref(sched), n_layers, m.ctypes.data_as(C.POINTER(C.c_uint8)), C.byref(out)))
    return out


def ff_plan_destroy(plan):
    lib().ff_plan_destroy(plan)


def ff_plan_export(plan, T, L, K):
    """Returns the plan's decisions as numpy arrays (and counts as a dict)."""
    import numpy as np
    a = {"step_kind": np.zeros(T, np.int32), "refresh_ord": np.zeros(T, np.int32), "k_eff": np.zeros(T, np.int32),
         "read_slots": np.zeros((T, K + 1), np.int32), "write_slot": np.zeros(T, np.int32),
         "action": np.zeros((T, L), np.int32), "coeffs": np.zeros((T, K + 1), np.float32)}
    cnt = ff_counts()
    ip = lambda x: x.ctypes.data_as(C.POINTER(C.c_int32))
    check(lib().ff_plan_export(plan, ip(a["step_kind"]), ip(a["refresh_ord"]), ip(a["k_eff"]), ip(a["read_slots"]),
                               ip(a["write_slot"]), ip(a["action"]),
                               a["coeffs"].ctypes.data_as(C.POINTER(C.c_float)), C.byref(cnt)))
    a["counts"] = cnt.as_dict()
    return a


def ff_cache_bytes(model, n_slots):
    return lib().ff_cache_bytes(C.byref(model), n_slots)


def ff_workspace_bytes(model):
    return lib().ff_workspace_bytes(C.byref(model))


def ff_block_exact(model, layer, weights, c_t, u, h, ws, ws_bytes, stream=0):
    return check(lib().ff_block_exact(C.byref(model), layer, C.byref(weights), c_t, u, h, ws, ws_bytes, stream))


def ff_cache_update(model, cache, n_slots, layer, slot, u, h, feature_mode=FF_RESIDUAL, stream=0):
    return check(lib().ff_cache_update(C.byref(model), cache, n_slots, layer, slot, u, h, feature_mode, stream))


def ff_draft_forecast(model, cache, n_slots, layer, k_eff, slots, coeffs, u, h_d, stream=0):
    return check(lib().ff_draft_forecast(C.byref(model), cache, n_slots, layer, k_eff, _i32arr(slots),
                                         _f32arr(coeffs), u, h_d, stream))


def ff_verify_replace(model, cache, n_slots, layer, k_eff, slots, coeffs, u, h_f, h_out, forward, eps,
                      rel_l1, ws, ws_bytes, stream=0, stride=1):
    """forward: FF_FWD_DRAFT / FF_FWD_EXACT / FF_FWD_TOKENS / FF_FWD_CHANNELS (a bool is
    read as exact (True) or draft (False)); stride for the partial kinds."""
    return check(lib().ff_verify_replace(C.byref(model), cache, n_slots, layer, k_eff, _i32arr(slots),
                                         _f32arr(coeffs), u, h_f, h_out, int(forward), int(stride), eps, rel_l1,
                                         ws, ws_bytes, stream))


def ff_verify_replace_noalloc(model, cache, n_slots, layer, k_eff, slots, coeffs, u, h_f, h_out, forward, eps,
                              rel_l1, stream=0, stride=1):
    """ff_verify_replace without a workspace (partial sums in the library's own device
    array; B <= FF_NOALLOC_VERIFY_MAX_B)."""
    return check(lib().ff_verify_replace_noalloc(C.byref(model), cache, n_slots, layer, k_eff, _i32arr(slots),
                                                 _f32arr(coeffs), u, h_f, h_out, int(forward), int(stride), eps,
                                                 rel_l1, stream))


def ff_ctx_create(model, layer_weights, global_weights, plan, cache, cache_bytes, ws, ws_bytes):
    out = C.c_void_p()
    check(lib().ff_ctx_create(C.byref(model), layer_weights, C.byref(global_weights), plan, cache, cache_bytes,
                              ws, ws_bytes, C.byref(out)))
    return out


def ff_ctx_destroy(ctx):
    lib().ff_ctx_destroy(ctx)


def ff_ctx_reset(ctx):
    return check(lib().ff_ctx_reset(ctx))


def ff_get_counts(ctx):
    cnt = ff_counts()
    check(lib().ff_get_counts(ctx, C.byref(cnt)))
    return cnt.as_dict()


def ff_ctx_step_kinds(ctx, T):
    """Realised step kinds [T] (FF_STEP_REFRESH / FF_STEP_CACHED, -1 for steps not run)."""
    out = (C.c_int32 * T)()
    check(lib().ff_ctx_step_kinds(ctx, out))
    return np.array(out[:], dtype=np.int32)


def ff_ctx_trace(ctx, buf, nbytes):
    return check(lib().ff_ctx_trace(ctx, buf, nbytes))


def ff_hist_sum_bytes(model, plan):
    return lib().ff_hist_sum_bytes(C.byref(model), plan)


def ff_ctx_hist_sums(ctx, buf, nbytes):
    return check(lib().ff_ctx_hist_sums(ctx, buf, nbytes))


def ff_cond_cache_bytes(model, plan):
    return lib().ff_cond_cache_bytes(C.byref(model), plan)


def ff_ctx_cond_cache(ctx, buf, nbytes):
    return check(lib().ff_ctx_cond_cache(ctx, buf, nbytes))


def ff_rel_l1(model, a, b, eps, rel, ws, ws_bytes, stream=0):
    return check(lib().ff_rel_l1(C.byref(model), a, b, eps, rel, ws, ws_bytes, stream))


def ff_denoise_step(ctx, step, x, cond, txt, audit, stream=0):
    return check(lib().ff_denoise_step(ctx, step, x, cond, txt, audit, stream))


def ff_ctx_profile(ctx, enable):
    return check(lib().ff_ctx_profile(ctx, int(enable)))


def ff_ctx_profile_read(ctx):
    """Per kernel class: {class: dict(launches, ms, flops, bytes)} (synchronises the events)."""
    out = (ff_prof_stat * len(PROF_CLASSES))()
    check(lib().ff_ctx_profile_read(ctx, out))
    return {n: {"launches": o.launches, "ms": o.ms, "flops": o.flops, "bytes": o.bytes}
            for n, o in zip(PROF_CLASSES, out)}
