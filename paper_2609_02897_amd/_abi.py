"""ctypes mirror of include/asv.h and the loader of libasv.so (argument marshalling only)."""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libasv.so")

ASV_OK, ASV_EINVAL, ASV_EWORKSPACE, ASV_EHIP, ASV_ESCRATCH = 0, -1, -2, -3, -4
STATIC_SCRATCH_BYTES = 32 << 20   # ASV_STATIC_SCRATCH_BYTES
W_ROW_MAJOR, W_PACKED = 0, 1     # asv_verify_args.w_lm_layout
RS_BAD_ROOT, RS_BAD_PARENT, RS_BAD_TOKEN, RS_BAD_OFFSETS, RS_BAD_TAU = 1, 2, 4, 16, 32
RS_MASK_SMALL, RS_BAD_PATH = 64, 128
DS_BAD_SHAPE, DS_OVERFLOW = 1, 2
HIST_WINDOW = 16
TOPK_MAX, POOL_MAX = 4, 256

# Every entry point include/asv.h declares.
EXPORTS = ("asv_version", "asv_status_string", "asv_last_error", "asv_workspace_bytes",
           "asv_tree_policy", "asv_state_init", "asv_verify", "asv_draft_workspace_bytes",
           "asv_draft_step", "asv_draft_prune", "asv_tree_meta", "asv_commit",
           "asv_packed_lm_head_bytes", "asv_pack_lm_head", "asv_packed_draft_head_bytes",
           "asv_pack_draft_head", "asv_verify_tuned", "asv_draft_step_tuned",
           "asv_verify_noalloc", "asv_k1_plan")


class AsvReqState(ctypes.Structure):
    _fields_ = [("rar", ctypes.c_float), ("hist", ctypes.c_float * HIST_WINDOW),
                ("hist_head", ctypes.c_int32), ("hist_count", ctypes.c_int32),
                ("zero_streak", ctypes.c_int32), ("breaker", ctypes.c_int32),
                ("steps", ctypes.c_int32), ("hist_mean", ctypes.c_float),
                ("draft_conf", ctypes.c_float), ("dcs", ctypes.c_float),
                ("shape", ctypes.c_int32 * 3)]


class AsvParams(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("rar0", ctypes.c_float),
                ("breaker_n", ctypes.c_int32), ("max_promotions", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("dcs_divisor", ctypes.c_float), ("shape_lo", ctypes.c_int32 * 3),
                ("shape_hi", ctypes.c_int32 * 3), ("shape_start", ctypes.c_int32 * 3)]


_P = ctypes.c_void_p


class AsvVerifyArgs(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("H", ctypes.c_int32),
                ("V", ctypes.c_int32),
                ("hidden", _P), ("w_lm", _P), ("draft_tok", _P), ("parent", _P),
                ("req_offsets", _P), ("tau", _P), ("draft_logits", _P),
                ("row_max", _P), ("row_lse", _P), ("row_argmax", _P),
                ("drafted_logit", _P), ("accept", _P),
                ("accepted_len", _P), ("bonus_token", _P), ("accepted_path", _P),
                ("draft_conf", _P), ("state", _P), ("req_status", _P),
                ("params", AsvParams), ("w_lm_layout", ctypes.c_int32)]


class AsvTuning(ctypes.Structure):
    _fields_ = [("begin_event", _P), ("end_event", _P), ("tile_rows", ctypes.c_int32)]


class AsvK1Launch(ctypes.Structure):
    _fields_ = [("tile_rows", ctypes.c_int32), ("slab0", ctypes.c_int32),
                ("n_slabs", ctypes.c_int32), ("row_tiles", ctypes.c_int32),
                ("k_loop", ctypes.c_int32), ("stream_w", ctypes.c_int32),
                ("blk_slabs", ctypes.c_int32), ("blk_rows", ctypes.c_int32)]


class AsvDraftTree(ctypes.Structure):
    _fields_ = [("nsteps", ctypes.c_int32), ("topk", ctypes.c_int32), ("ndt", ctypes.c_int32),
                ("steps", ctypes.c_int32), ("n_pool", ctypes.c_int32),
                ("n_front", ctypes.c_int32), ("status", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("front", ctypes.c_int32 * TOPK_MAX),
                ("front_score", ctypes.c_float * TOPK_MAX), ("tok", ctypes.c_int32 * POOL_MAX),
                ("par", ctypes.c_int32 * POOL_MAX), ("score", ctypes.c_float * POOL_MAX)]


class AsvDraftArgs(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("V", ctypes.c_int32),
                ("step", ctypes.c_int32), ("hidden", _P), ("w_draft", _P), ("vocab_map", _P),
                ("state", _P), ("shape", ctypes.c_int32 * 3), ("tree", _P), ("topk_id", _P),
                ("topk_logp", _P), ("row_lse", _P), ("front_tok", _P), ("draft_conf", _P),
                ("w_draft_layout", ctypes.c_int32)]


class AsvCommitArgs(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("req_offsets", _P),
                ("draft_tok", _P), ("accepted_len", _P), ("accepted_path", _P),
                ("bonus_token", _P), ("commit_off", _P), ("commit_tok", _P),
                ("commit_row", _P), ("row_src", _P), ("row_dst", _P),
                ("row_bytes", ctypes.c_int64), ("req_status", _P)]


assert ctypes.sizeof(AsvReqState) == 112
assert ctypes.sizeof(AsvDraftTree) == 3136


class LibraryMissing(RuntimeError):
    pass


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libasv.so (built in-tree by ``__graft_entry__.build()``); raise if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise LibraryMissing(
            f"{path} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
    # torch wheels bundle their own HIP runtime (same soname, libamdhip64.so.7). Importing torch
    # first makes the dynamic loader bind libasv to that already-loaded runtime, so torch's
    # allocations, streams and events and libasv's launches share one HIP context; a second
    # runtime in the same process would not see the GPU.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    lib.asv_version.restype = ctypes.c_int
    lib.asv_version.argtypes = []
    lib.asv_status_string.restype = ctypes.c_char_p
    lib.asv_status_string.argtypes = [ctypes.c_int]
    lib.asv_last_error.restype = ctypes.c_char_p
    lib.asv_last_error.argtypes = []
    lib.asv_workspace_bytes.restype = ctypes.c_int
    lib.asv_workspace_bytes.argtypes = [ctypes.c_int32] * 4 + [ctypes.POINTER(ctypes.c_uint64)]
    lib.asv_tree_policy.restype = ctypes.c_int
    lib.asv_tree_policy.argtypes = [_P, _P, ctypes.c_int32, ctypes.POINTER(AsvParams), _P]
    lib.asv_state_init.restype = ctypes.c_int
    lib.asv_state_init.argtypes = [_P, ctypes.c_int32, ctypes.POINTER(AsvParams), _P]
    lib.asv_verify.restype = ctypes.c_int
    lib.asv_verify.argtypes = [ctypes.POINTER(AsvVerifyArgs), _P, ctypes.c_uint64, _P]
    lib.asv_draft_workspace_bytes.restype = ctypes.c_int
    lib.asv_draft_workspace_bytes.argtypes = [ctypes.c_int32] * 3 + [
        ctypes.POINTER(ctypes.c_uint64)]
    lib.asv_draft_step.restype = ctypes.c_int
    lib.asv_draft_step.argtypes = [ctypes.POINTER(AsvDraftArgs), _P, ctypes.c_uint64, _P]
    lib.asv_verify_noalloc.restype = ctypes.c_int
    lib.asv_verify_noalloc.argtypes = [ctypes.POINTER(AsvVerifyArgs), _P]
    lib.asv_verify_tuned.restype = ctypes.c_int
    lib.asv_verify_tuned.argtypes = [ctypes.POINTER(AsvVerifyArgs), ctypes.POINTER(AsvTuning),
                                     _P, ctypes.c_uint64, _P]
    lib.asv_k1_plan.restype = ctypes.c_int
    lib.asv_k1_plan.argtypes = [ctypes.c_int32] * 4 + [ctypes.POINTER(AsvK1Launch),
                                                       ctypes.POINTER(ctypes.c_int32)]
    lib.asv_draft_step_tuned.restype = ctypes.c_int
    lib.asv_draft_step_tuned.argtypes = [ctypes.POINTER(AsvDraftArgs),
                                         ctypes.POINTER(AsvTuning), _P, ctypes.c_uint64, _P]
    lib.asv_draft_prune.restype = ctypes.c_int
    lib.asv_draft_prune.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_int32, _P, _P, _P, _P, _P]
    lib.asv_tree_meta.restype = ctypes.c_int
    lib.asv_tree_meta.argtypes = [_P, _P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int32,
                                  _P, _P, _P, _P]
    lib.asv_commit.restype = ctypes.c_int
    lib.asv_commit.argtypes = [ctypes.POINTER(AsvCommitArgs), _P]
    for f in (lib.asv_packed_lm_head_bytes, lib.asv_packed_draft_head_bytes):
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_uint64)]
    for f in (lib.asv_pack_lm_head, lib.asv_pack_draft_head):
        f.restype = ctypes.c_int
        f.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_uint64, _P]
    _lib = lib
    return lib
