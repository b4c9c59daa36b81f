"""ctypes binding of libtasp (include/tasp.h). Argument marshalling only: every step of the decode
path runs in the library's HIP kernels. Device memory and streams come from PyTorch.

The functions keep the C names (``tasp_compile_plan`` ...). ``TaspError`` is raised for any
non-zero status, with the library's thread-local message. Loading fails loudly when the library
has not been built: there is no other implementation behind these names.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# TASP_LIB selects another build of the same library (the host-sanitizer build of the tests)
LIB_PATH = os.environ.get("TASP_LIB") or os.path.join(HERE, "libtasp.so")

TASP_OK = 0
STATUS = {0: "TASP_OK", -1: "TASP_ERR_INVALID_ARG", -2: "TASP_ERR_SHAPE", -3: "TASP_ERR_MASK",
          -4: "TASP_ERR_WORKSPACE", -5: "TASP_ERR_POS_RANGE", -6: "TASP_ERR_CACHE_PLAN_MISMATCH",
          -7: "TASP_ERR_HIP", -8: "TASP_ERR_UNSUPPORTED", -9: "TASP_ERR_INTERNAL"}
IDX_Q, IDX_KV, IDX_QKVSLOT, IDX_FFN = 0, 1, 2, 3
PANEL_QKV, PANEL_O, PANEL_GATE, PANEL_UP, PANEL_DOWN = 0, 1, 2, 3, 4
KERNEL_KINDS = {0: "qkv_gemv", 1: "attention", 2: "o_gemv", 3: "gateup_gemv", 4: "down_gemv",
                5: "lmhead_gemv", 6: "operand_prep", 7: "rope_append"}
# the same stages in a prefill, where the projections are GEMMs over the prompt's tokens
PREFILL_KINDS = {k: v.replace("_gemv", "_gemm") for k, v in KERNEL_KINDS.items()}

EXPORTS = ["tasp_plan_workspace_bytes", "tasp_compile_plan", "tasp_plan_counts",
           "tasp_plan_indices", "tasp_plan_panel", "tasp_plan_ledger", "tasp_plan_destroy",
           "tasp_shared_plan_workspace_bytes", "tasp_compile_shared_plan",
           "tasp_kv_bind", "tasp_decode_step", "tasp_prefill", "tasp_prefill_last", "tasp_prefill_timed",
           "tasp_generate",
           "tasp_decode_step_timed",
           "tasp_profile_stage", "tasp_mask_workspace_bytes", "tasp_build_mask",
           "tasp_router_workspace_bytes", "tasp_route", "tasp_route_noalloc", "tasp_serve_turn", "tasp_copy_probe",
           "tasp_status_string", "tasp_last_error"]


class TaspError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class tasp_model_desc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ffn", C.c_int32),
                ("vocab", C.c_int32), ("max_batch", C.c_int32), ("max_seq", C.c_int32),
                ("max_prefill", C.c_int32), ("rms_eps", C.c_float), ("reserved0", C.c_float),
                ("rope_theta", C.c_double)]


class tasp_qmat(C.Structure):
    _fields_ = [("w", C.c_void_p), ("scale", C.c_void_p)]


class tasp_layer(C.Structure):
    _fields_ = [("wq", tasp_qmat), ("wk", tasp_qmat), ("wv", tasp_qmat), ("wo", tasp_qmat),
                ("wg", tasp_qmat), ("wu", tasp_qmat), ("wd", tasp_qmat),
                ("attn_norm", C.c_void_p), ("ffn_norm", C.c_void_p)]


class tasp_store(C.Structure):
    _fields_ = [("layers", C.POINTER(tasp_layer)), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p)]


class tasp_gqmat(C.Structure):
    _fields_ = [("w", C.c_void_p), ("scale", C.c_void_p)]


class tasp_glayer(C.Structure):
    _fields_ = [("wqkv", tasp_gqmat), ("wo", tasp_gqmat), ("wg", tasp_gqmat), ("wu", tasp_gqmat),
                ("wd", tasp_gqmat), ("attn_norm", C.c_void_p), ("ffn_norm", C.c_void_p)]


class tasp_gstore(C.Structure):
    _fields_ = [("layers", C.POINTER(tasp_glayer)), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p)]


class tasp_mask(C.Structure):
    _fields_ = [("q_keep", C.c_void_p), ("kv_keep", C.c_void_p), ("ffn_keep", C.c_void_p)]


class tasp_kv_cache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("batch", C.c_int32),
                ("max_seq", C.c_int32), ("plan_sig", C.c_uint64)]


class tasp_router(C.Structure):
    _fields_ = [("n_bins", C.c_int32), ("proj_dim", C.c_int32), ("hidden1", C.c_int32),
                ("hidden2", C.c_int32), ("n_tasks", C.c_int32), ("temperature", C.c_float),
                ("tau", C.c_float), ("proj", C.c_void_p), ("w1", C.c_void_p), ("b1", C.c_void_p),
                ("w2", C.c_void_p), ("b2", C.c_void_p), ("w3", C.c_void_p), ("b3", C.c_void_p)]


ROUTER_SCALARS = 11

_lib = None


def load(path: str = LIB_PATH):
    """Load libtasp.so once; raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libtasp.so not found at {path}: build it with "
                          "`python -m paper_2609_29499_amd.build` (or __graft_entry__.build())")
    lib = C.CDLL(path)
    P, I32, U64, SZ = C.c_void_p, C.c_int32, C.c_uint64, C.c_size_t
    sig = {
        "tasp_plan_workspace_bytes": [C.POINTER(tasp_model_desc), C.POINTER(tasp_mask), C.POINTER(SZ)],
        "tasp_compile_plan": [C.POINTER(tasp_model_desc), C.POINTER(tasp_store), C.POINTER(tasp_mask),
                              P, SZ, P, C.POINTER(P)],
        "tasp_shared_plan_workspace_bytes": [C.POINTER(tasp_model_desc), C.POINTER(SZ), C.POINTER(SZ)],
        "tasp_compile_shared_plan": [C.POINTER(tasp_model_desc), C.POINTER(tasp_gstore),
                                     C.POINTER(tasp_mask), P, SZ, P, SZ, P, C.POINTER(P)],
        "tasp_plan_counts": [P, I32, C.POINTER(I32), C.POINTER(I32), C.POINTER(I32)],
        "tasp_plan_indices": [P, I32, I32, C.POINTER(I32), I32, C.POINTER(I32)],
        "tasp_plan_panel": [P, I32, I32, C.POINTER(P), C.POINTER(P), C.POINTER(C.c_int64),
                            C.POINTER(C.c_int64), C.POINTER(C.c_int64)],
        "tasp_plan_ledger": [P, C.POINTER(C.c_double), C.POINTER(U64), C.POINTER(U64), C.POINTER(U64)],
        "tasp_plan_destroy": [P],
        "tasp_kv_bind": [P, C.POINTER(tasp_kv_cache)],
        "tasp_decode_step": [P, P, C.POINTER(tasp_kv_cache), I32, P, P],
        "tasp_prefill": [P, P, I32, C.POINTER(tasp_kv_cache), I32, P, P],
        "tasp_prefill_last": [P, P, I32, C.POINTER(tasp_kv_cache), I32, P, P],
        "tasp_generate": [P, P, P, P, I32, I32, C.POINTER(tasp_kv_cache), P, P, P, P],
        "tasp_prefill_timed": [P, P, I32, C.POINTER(tasp_kv_cache), I32, P, P, C.POINTER(C.c_float),
                               C.POINTER(I32), I32, C.POINTER(I32)],
        "tasp_decode_step_timed": [P, P, C.POINTER(tasp_kv_cache), I32, P, P, C.POINTER(C.c_float),
                                   C.POINTER(I32), I32, C.POINTER(I32)],
        "tasp_profile_stage": [C.POINTER(P), C.POINTER(tasp_kv_cache), I32, I32, I32, I32, I32, P,
                               C.POINTER(C.c_float)],
        "tasp_mask_workspace_bytes": [C.POINTER(tasp_model_desc), I32, C.POINTER(SZ)],
        "tasp_build_mask": [C.POINTER(tasp_model_desc), P, P, I32, C.c_double, P, SZ, P, P, P,
                            C.POINTER(U64), P],
        "tasp_router_workspace_bytes": [C.POINTER(tasp_router), I32, C.POINTER(SZ)],
        "tasp_route": [C.POINTER(tasp_router), P, I32, P, I32, P, P, SZ, P, P, P, P],
        "tasp_route_noalloc": [C.POINTER(tasp_router), P, I32, P, I32, P, P, P, P, P],
        "tasp_serve_turn": [C.POINTER(tasp_router), C.POINTER(P), P, P, I32, P, P, P, P, I32, I32,
                            I32, C.POINTER(tasp_kv_cache), P, P, P, P, SZ, C.POINTER(I32),
                            C.POINTER(I32), P],
        "tasp_copy_probe": [P, P, SZ, P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int32
    lib.tasp_status_string.argtypes = [C.c_int32]
    lib.tasp_status_string.restype = C.c_char_p
    lib.tasp_last_error.argtypes = []
    lib.tasp_last_error.restype = C.c_char_p
    _lib = lib
    return lib


def _check(status):
    if status != TASP_OK:
        raise TaspError(status, _lib.tasp_last_error().decode())
    return status


# ----------------------------------------------------------------------- same-name wrappers

def tasp_plan_workspace_bytes(desc, mask):
    n = C.c_size_t()
    _check(load().tasp_plan_workspace_bytes(C.byref(desc), mask, C.byref(n)))
    return n.value


def tasp_compile_plan(desc, store, mask, workspace_ptr, workspace_bytes, stream):
    plan = C.c_void_p()
    _check(load().tasp_compile_plan(C.byref(desc), C.byref(store), mask, workspace_ptr,
                                    workspace_bytes, stream, C.byref(plan)))
    return plan


def tasp_shared_plan_workspace_bytes(desc):
    """(plan_bytes, scratch_bytes)."""
    n, m = C.c_size_t(), C.c_size_t()
    _check(load().tasp_shared_plan_workspace_bytes(C.byref(desc), C.byref(n), C.byref(m)))
    return n.value, m.value


def tasp_compile_shared_plan(desc, store, mask, workspace_ptr, workspace_bytes, scratch_ptr,
                             scratch_bytes, stream):
    out = C.c_void_p()
    _check(load().tasp_compile_shared_plan(C.byref(desc), C.byref(store), mask, workspace_ptr,
                                           workspace_bytes, scratch_ptr, scratch_bytes, stream,
                                           C.byref(out)))
    return out


def tasp_plan_counts(plan, layer):
    a, b, c = C.c_int32(), C.c_int32(), C.c_int32()
    _check(load().tasp_plan_counts(plan, layer, C.byref(a), C.byref(b), C.byref(c)))
    return a.value, b.value, c.value


def tasp_plan_indices(plan, layer, which):
    n = C.c_int32()
    _check(load().tasp_plan_indices(plan, layer, which, None, 0, C.byref(n)))
    buf = (C.c_int32 * max(n.value, 1))()
    _check(load().tasp_plan_indices(plan, layer, which, buf, n.value, C.byref(n)))
    return list(buf[:n.value])


def tasp_plan_panel(plan, layer, which):
    w, s = C.c_void_p(), C.c_void_p()
    rows, cols, ld = C.c_int64(), C.c_int64(), C.c_int64()
    _check(load().tasp_plan_panel(plan, layer, which, C.byref(w), C.byref(s), C.byref(rows),
                                  C.byref(cols), C.byref(ld)))
    return w.value, s.value, rows.value, cols.value, ld.value


def tasp_plan_ledger(plan):
    r, wb, sb, sg = C.c_double(), C.c_uint64(), C.c_uint64(), C.c_uint64()
    _check(load().tasp_plan_ledger(plan, C.byref(r), C.byref(wb), C.byref(sb), C.byref(sg)))
    return r.value, wb.value, sb.value, sg.value


def tasp_plan_destroy(plan):
    _check(load().tasp_plan_destroy(plan))


def tasp_kv_bind(plan, cache):
    _check(load().tasp_kv_bind(plan, C.byref(cache)))


def tasp_decode_step(plan, x_ptr, cache, pos, out_ptr, stream):
    _check(load().tasp_decode_step(plan, x_ptr, C.byref(cache), pos, out_ptr, stream))


def tasp_prefill(plan, x_ptr, T, cache, pos0, out_ptr, stream):
    _check(load().tasp_prefill(plan, x_ptr, T, C.byref(cache), pos0, out_ptr, stream))


def tasp_prefill_last(plan, x_ptr, T, cache, pos0, out_ptr, stream):
    _check(load().tasp_prefill_last(plan, x_ptr, T, C.byref(cache), pos0, out_ptr, stream))


def tasp_generate(plan, embed_ptr, scale_ptr, prompt_ptr, T, n_new, cache, out_ids_ptr, x_ptr,
                  logits_ptr, stream):
    _check(load().tasp_generate(plan, embed_ptr, scale_ptr, prompt_ptr, T, n_new, C.byref(cache),
                                out_ids_ptr, x_ptr, logits_ptr, stream))


def tasp_prefill_timed(plan, x_ptr, T, cache, pos0, out_ptr, stream, cap=4096):
    ms = (C.c_float * cap)()
    kinds = (C.c_int32 * cap)()
    n = C.c_int32()
    _check(load().tasp_prefill_timed(plan, x_ptr, T, C.byref(cache), pos0, out_ptr, stream, ms,
                                     kinds, cap, C.byref(n)))
    return [(PREFILL_KINDS[kinds[i]], ms[i]) for i in range(n.value)]


def tasp_decode_step_timed(plan, x_ptr, cache, pos, out_ptr, stream, cap=4096):
    ms = (C.c_float * cap)()
    kinds = (C.c_int32 * cap)()
    n = C.c_int32()
    _check(load().tasp_decode_step_timed(plan, x_ptr, C.byref(cache), pos, out_ptr, stream, ms,
                                         kinds, cap, C.byref(n)))
    return [(KERNEL_KINDS[kinds[i]], ms[i]) for i in range(n.value)]


def tasp_profile_stage(plans, caches, layer, kind, pos, reps, stream):
    """``caches``: tasp_kv_cache structs, one per plan."""
    arr = (C.c_void_p * len(plans))(*[p.value if isinstance(p, C.c_void_p) else p for p in plans])
    carr = (tasp_kv_cache * len(caches))(*caches)
    ms = C.c_float()
    _check(load().tasp_profile_stage(arr, carr, len(plans), layer, kind, pos, reps, stream,
                                     C.byref(ms)))
    return ms.value


def tasp_mask_workspace_bytes(desc, granule):
    n = C.c_size_t()
    _check(load().tasp_mask_workspace_bytes(C.byref(desc), granule, C.byref(n)))
    return n.value


def tasp_build_mask(desc, head_scores_ptr, chan_scores_ptr, granule, target, ws_ptr, ws_bytes,
                    q_ptr, kv_ptr, f_ptr, stream):
    spent = C.c_uint64()
    _check(load().tasp_build_mask(C.byref(desc), head_scores_ptr, chan_scores_ptr, granule, target,
                                  ws_ptr, ws_bytes, q_ptr, kv_ptr, f_ptr, C.byref(spent), stream))
    return spent.value


def tasp_router_workspace_bytes(router, n_prompts):
    n = C.c_size_t()
    _check(load().tasp_router_workspace_bytes(C.byref(router), n_prompts, C.byref(n)))
    return n.value


def tasp_route(router, text_ptr, n_text, offsets_ptr, n_prompts, logprob_ptr, ws_ptr, ws_bytes,
               feats_ptr, probs_ptr, choice_ptr, stream):
    _check(load().tasp_route(C.byref(router), text_ptr, n_text, offsets_ptr, n_prompts,
                             logprob_ptr, ws_ptr, ws_bytes, feats_ptr, probs_ptr, choice_ptr,
                             stream))


def tasp_route_noalloc(router, text_ptr, n_text, offsets_ptr, n_prompts, logprob_ptr, feats_ptr,
                       probs_ptr, choice_ptr, stream):
    _check(load().tasp_route_noalloc(C.byref(router), text_ptr, n_text, offsets_ptr, n_prompts,
                                     logprob_ptr, feats_ptr, probs_ptr, choice_ptr, stream))


def tasp_serve_turn(router, task_plans, dense_plan, text_ptr, n_text, logprob_ptr, embed_ptr,
                    scale_ptr, prompt_ptr, T, n_cached, n_new, cache, out_ids_ptr, x_ptr,
                    logits_ptr, ws_ptr, ws_bytes, stream):
    """Returns (choice, reused)."""
    arr = (C.c_void_p * len(task_plans))(
        *[p.value if isinstance(p, C.c_void_p) else p for p in task_plans])
    chosen, reused = C.c_int32(), C.c_int32()
    _check(load().tasp_serve_turn(C.byref(router), arr, dense_plan, text_ptr, n_text, logprob_ptr,
                                  embed_ptr, scale_ptr, prompt_ptr, T, n_cached, n_new,
                                  C.byref(cache), out_ids_ptr, x_ptr, logits_ptr, ws_ptr, ws_bytes,
                                  C.byref(chosen), C.byref(reused), stream))
    return chosen.value, reused.value


def tasp_copy_probe(dst_ptr, src_ptr, nbytes, stream):
    _check(load().tasp_copy_probe(dst_ptr, src_ptr, nbytes, stream))
