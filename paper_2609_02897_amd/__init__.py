"""AdaptiveSpec verification on MI355X (gfx950): Python binding of libasv.

The computation happens in the HIP kernels behind the C ABI of ``include/asv.h``; this module
only checks tensor types, allocates outputs and the workspace with torch, and passes raw
device pointers and torch's current HIP stream through ctypes. There is no CPU fallback: if
``libasv.so`` is not built, or a tensor is not on a GPU, the call raises.
"""

from __future__ import annotations

import ctypes
from typing import NamedTuple, Optional

from ._abi import (  # noqa: F401
    ASV_EHIP, ASV_EINVAL, ASV_ESCRATCH, ASV_EWORKSPACE, ASV_OK, DS_BAD_SHAPE, DS_OVERFLOW,
    EXPORTS, LIB_PATH, POOL_MAX, RS_BAD_OFFSETS, RS_BAD_PARENT, RS_BAD_PATH, RS_BAD_ROOT,
    RS_BAD_TAU, RS_BAD_TOKEN, RS_MASK_SMALL, STATIC_SCRATCH_BYTES, TOPK_MAX, W_PACKED,
    W_ROW_MAJOR, AsvCommitArgs, AsvDraftArgs, AsvDraftTree, AsvParams, AsvReqState, AsvTuning,
    AsvVerifyArgs, LibraryMissing, load)

STATE_BYTES = ctypes.sizeof(AsvReqState)
TREE_BYTES = ctypes.sizeof(AsvDraftTree)


class VerifyOut(NamedTuple):
    row_max: "torch.Tensor"          # f32 [N]
    row_lse: "torch.Tensor"          # f32 [N]
    row_argmax: "torch.Tensor"       # i32 [N]
    drafted_logit: "torch.Tensor"    # f32 [N]
    accept: "torch.Tensor"           # u8 [N]
    accepted_len: "torch.Tensor"     # i32 [B]
    bonus_token: "torch.Tensor"      # i32 [B]
    accepted_path: "torch.Tensor"    # i32 [N]
    draft_conf: Optional["torch.Tensor"]  # f32 [B] or None
    req_status: "torch.Tensor"       # i32 [B]


class AsvError(RuntimeError):
    def __init__(self, code: int):
        lib = load()
        msg = lib.asv_status_string(code).decode()
        detail = lib.asv_last_error().decode() if code in (ASV_EHIP, ASV_ESCRATCH) else ""
        super().__init__(f"libasv returned {code}: {msg}" + (f" [{detail}]" if detail else ""))
        self.code = code


def make_params(alpha: float = 0.3, rar0: float = 1.0, breaker_n: int = 5,
                max_promotions: int = -1, temperature: float = 1.0, dcs_divisor: float = 0.5,
                shape_lo=(3, 4, 4), shape_hi=(7, 1, 8), shape_start=(3, 4, 4)) -> AsvParams:
    """Policy parameters; defaults are the paper's (EMA alpha 0.3, breaker after 5 steps,
    margin at temperature 1, DCS divisor 0.5, tree shapes (3,4,4) <-> (7,1,8))."""
    tri = ctypes.c_int32 * 3
    return AsvParams(alpha, rar0, breaker_n, max_promotions, temperature, dcs_divisor,
                     tri(*shape_lo), tri(*shape_hi), tri(*shape_start))


def _check(code: int):
    if code != ASV_OK:
        raise AsvError(code)


def _stream_handle(device) -> int:
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def workspace_bytes(B: int, N: int, H: int, V: int) -> int:
    out = ctypes.c_uint64(0)
    _check(load().asv_workspace_bytes(B, N, H, V, ctypes.byref(out)))
    return int(out.value)


def alloc_workspace(B: int, N: int, H: int, V: int, device):
    """A workspace tensor for asv_verify (torch allocations are 256-byte aligned)."""
    import torch
    n = max(workspace_bytes(B, N, H, V), 256)
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def tree_policy(state, conf=None, params: Optional[AsvParams] = None):
    """``asv_tree_policy``: the Draft Confidence Score and tree shape of every request, from a
    fresh draft confidence ``conf`` (f32 [B], optional) and the state's RAR (in place)."""
    import torch
    B = state.shape[0]
    _need(state, "state", torch.uint8, (B, STATE_BYTES))
    if conf is not None:
        _need(conf, "conf", torch.float32, (B,))
    p = params or make_params()
    _check(load().asv_tree_policy(_ptr(conf), _ptr(state), B, ctypes.byref(p),
                                  _stream_handle(state.device)))
    return state


def state_init(B: int, params: Optional[AsvParams] = None, device="cuda"):
    """Per-request policy state, one 112-byte ``asv_req_state`` per row of a [B, 112] u8
    tensor."""
    import torch
    p = params or make_params()
    st = torch.empty((B, STATE_BYTES), dtype=torch.uint8, device=device)
    _check(load().asv_state_init(_ptr(st), B, ctypes.byref(p), _stream_handle(st.device)))
    return st


def alloc_outputs(B: int, N: int, device, with_conf: bool) -> VerifyOut:
    import torch
    f32, i32 = torch.float32, torch.int32
    return VerifyOut(
        torch.empty(N, dtype=f32, device=device), torch.empty(N, dtype=f32, device=device),
        torch.empty(N, dtype=i32, device=device), torch.empty(N, dtype=f32, device=device),
        torch.empty(N, dtype=torch.uint8, device=device),
        torch.empty(B, dtype=i32, device=device), torch.empty(B, dtype=i32, device=device),
        torch.empty(N, dtype=i32, device=device),
        torch.empty(B, dtype=f32, device=device) if with_conf else None,
        torch.empty(B, dtype=i32, device=device))


def _verify_out_spec(B: int, N: int, with_conf: bool) -> dict:
    import torch
    f32, i32 = torch.float32, torch.int32
    return dict(row_max=(f32, (N,)), row_lse=(f32, (N,)), row_argmax=(i32, (N,)),
                drafted_logit=(f32, (N,)), accept=(torch.uint8, (N,)),
                accepted_len=(i32, (B,)), bonus_token=(i32, (B,)), accepted_path=(i32, (N,)),
                draft_conf=(f32, (B,)) if with_conf else None, req_status=(i32, (B,)))


def _need_out(out, spec: dict, device):
    """Caller-supplied output buffers: every field of the dtype and shape these sizes need,
    contiguous and on the inputs' device (the kernels write exactly that many elements)."""
    for name, want in spec.items():
        t = getattr(out, name)
        if want is None:
            continue
        _need(t, f"out.{name}", *want)
        if t.device != device:
            raise ValueError(f"out.{name}: on {t.device}, the inputs are on {device}")


def _need_workspace(ws, need: int, device):
    import torch
    if not isinstance(ws, torch.Tensor) or ws.device != device or not ws.is_contiguous():
        raise ValueError("workspace: a contiguous tensor on the inputs' device")
    if ws.dtype != torch.uint8 or ws.numel() < need or ws.data_ptr() % 256:
        raise ValueError(f"workspace: a 256-byte aligned uint8 tensor of >= {need} bytes")


def _need(t, name, dtype, shape):
    import torch
    if t is None or not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be on a GPU (no CPU path exists)")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def _same_device(device, **tensors):
    """Every given tensor (None skipped) on `device`: the kernels run on one GPU and take raw
    pointers, so an input on another GPU would be read through a foreign address."""
    for name, t in tensors.items():
        if t is not None and t.device != device:
            raise ValueError(f"{name}: on {t.device}, the hidden states are on {device}")


class PackedLmHead(NamedTuple):
    """An LM-head weight in a packed tile layout: ``kind`` "target" (``asv_pack_lm_head``,
    [256 rows][64 columns] tiles, for ``verify``) or "draft" (``asv_pack_draft_head``, [64][64]
    tiles, for ``draft_step``). Tiles are stored 64-column block major, zero rows past V."""
    data: "torch.Tensor"             # bf16, flat, packed_*_bytes(V, H) / 2 values
    V: int
    H: int
    kind: str


def packed_lm_head_bytes(V: int, H: int, kind: str = "target") -> int:
    out = ctypes.c_uint64()
    lib = load()
    f = lib.asv_packed_lm_head_bytes if kind == "target" else lib.asv_packed_draft_head_bytes
    _check(f(V, H, ctypes.byref(out)))
    return out.value


def _pack(w, kind: str) -> PackedLmHead:
    import torch
    V, H = w.shape
    _need(w, "weight", torch.bfloat16, (V, H))
    n = packed_lm_head_bytes(V, H, kind)
    data = torch.empty(n // 2, dtype=torch.bfloat16, device=w.device)
    lib = load()
    f = lib.asv_pack_lm_head if kind == "target" else lib.asv_pack_draft_head
    _check(f(w.data_ptr(), V, H, data.data_ptr(), n, _stream_handle(w.device)))
    return PackedLmHead(data, V, H, kind)


def pack_lm_head(w_lm) -> PackedLmHead:
    """The packed copy of a bf16 [V, H] target LM-head weight (``asv_pack_lm_head`` on torch's
    current stream). ``verify`` takes it in place of the row-major weight, with bit-identical
    results."""
    return _pack(w_lm, "target")


def pack_draft_head(w_draft) -> PackedLmHead:
    """The packed copy of a bf16 [V, H] draft LM-head weight (``asv_pack_draft_head``).
    ``draft_step`` takes it in place of the row-major weight, with bit-identical results."""
    return _pack(w_draft, "draft")


def _weight(w, kind: str, name: str, H: int):
    """(pointer, V, layout) of a row-major [V, H] weight or its packed copy of this kind."""
    import torch
    if isinstance(w, PackedLmHead):
        if w.kind != kind:
            raise ValueError(f"{name}: packed for the {w.kind} LM head, not the {kind}")
        if w.H != H:
            raise ValueError(f"{name}: packed for H = {w.H}, the hidden states have H = {H}")
        _need(w.data, f"{name}.data", torch.bfloat16,
              (packed_lm_head_bytes(w.V, H, kind) // 2,))
        return w.data.data_ptr(), w.V, W_PACKED
    V = w.shape[0] if isinstance(w, torch.Tensor) and w.dim() == 2 else -1
    _need(w, name, torch.bfloat16, (V, H))
    return w.data_ptr(), V, W_ROW_MAJOR


def verify(hidden, w_lm, draft_tok, parent, req_offsets, tau, draft_logits=None, state=None,
           params: Optional[AsvParams] = None, out: Optional[VerifyOut] = None,
           workspace=None, k1_events=None, k1_tile: int = 0,
           noalloc: bool = False) -> VerifyOut:
    """One verification step through ``asv_verify`` on torch's current stream.

    hidden bf16 [N, H]; w_lm bf16 [V, H] or its ``PackedLmHead``; draft_tok, parent int32 [N];
    req_offsets int32 [B+1]; tau float32 [B]; draft_logits float32 [N, V] or None; state u8
    [B, 112] (in/out) or None. ``out`` and ``workspace`` may be passed to reuse buffers
    (checked against these sizes). Measurement and tuning go through ``asv_verify_tuned``:
    ``k1_events`` is an optional pair of raw hipEvent_t handles set to the start and end of
    the LM-head kernel's launches, and ``k1_tile`` forces the LM-head tile (64, 128, 192 or 256 tree rows); 0 lets the
    library pick it. Without either, the product entry point ``asv_verify`` is called.
    ``noalloc`` calls ``asv_verify_noalloc`` instead, whose workspace is the library's static
    device scratch (no workspace tensor; pass ``out`` to allocate nothing at all here either).
    """
    import torch
    if noalloc and (workspace is not None or k1_events is not None or k1_tile):
        raise ValueError("noalloc takes no workspace, events or forced tile")
    N, H = hidden.shape
    B = req_offsets.shape[0] - 1
    _need(hidden, "hidden", torch.bfloat16, (N, H))
    w_ptr, V, layout = _weight(w_lm, "target", "w_lm", H)
    _need(draft_tok, "draft_tok", torch.int32, (N,))
    _need(parent, "parent", torch.int32, (N,))
    _need(req_offsets, "req_offsets", torch.int32, (B + 1,))
    _need(tau, "tau", torch.float32, (B,))
    if draft_logits is not None:
        _need(draft_logits, "draft_logits", torch.float32, (N, V))
    if state is not None:
        _need(state, "state", torch.uint8, (B, STATE_BYTES))
    dev = hidden.device
    _same_device(dev, w_lm=w_lm.data if isinstance(w_lm, PackedLmHead) else w_lm,
                 draft_tok=draft_tok, parent=parent, req_offsets=req_offsets, tau=tau,
                 draft_logits=draft_logits, state=state)
    if out is None:
        out = alloc_outputs(B, N, dev, draft_logits is not None)
    else:
        _need_out(out, _verify_out_spec(B, N, out.draft_conf is not None), dev)
    if noalloc:
        pass
    elif workspace is None:
        workspace = alloc_workspace(B, N, H, V, dev)
    else:
        _need_workspace(workspace, workspace_bytes(B, N, H, V), dev)
    a = AsvVerifyArgs()
    a.B, a.N, a.H, a.V = B, N, H, V
    a.hidden, a.w_lm, a.w_lm_layout = hidden.data_ptr(), w_ptr, layout
    a.draft_tok, a.parent = draft_tok.data_ptr(), parent.data_ptr()
    a.req_offsets, a.tau = req_offsets.data_ptr(), tau.data_ptr()
    a.draft_logits = _ptr(draft_logits)
    a.row_max, a.row_lse, a.row_argmax = (out.row_max.data_ptr(), out.row_lse.data_ptr(),
                                          out.row_argmax.data_ptr())
    a.drafted_logit, a.accept = out.drafted_logit.data_ptr(), out.accept.data_ptr()
    a.accepted_len, a.bonus_token = out.accepted_len.data_ptr(), out.bonus_token.data_ptr()
    a.accepted_path = out.accepted_path.data_ptr()
    a.draft_conf = _ptr(out.draft_conf)
    a.state = _ptr(state)
    a.req_status = out.req_status.data_ptr()
    a.params = params or make_params()
    lib = load()
    if noalloc:
        _check(lib.asv_verify_noalloc(ctypes.byref(a), _stream_handle(dev)))
    elif k1_events is None and not k1_tile:
        _check(lib.asv_verify(ctypes.byref(a), workspace.data_ptr(), workspace.numel(),
                              _stream_handle(dev)))
    else:
        tu = _tuning(k1_events, k1_tile)
        _check(lib.asv_verify_tuned(ctypes.byref(a), ctypes.byref(tu), workspace.data_ptr(),
                                    workspace.numel(), _stream_handle(dev)))
    return out


def k1_plan(N: int, V: int, cus: int, tile_rows: int = 0) -> list:
    """The LM-head launches ``verify`` enqueues for N tree rows and V vocabulary ids on a GPU
    with ``cus`` compute units (``k1_tile`` = tile_rows; 0 = the library's choice), as dicts
    in launch order. Host computation only (``asv_k1_plan``)."""
    lib = load()
    out = (_abi.AsvK1Launch * 2)()
    n = ctypes.c_int32(0)
    _check(lib.asv_k1_plan(N, V, cus, tile_rows, out, ctypes.byref(n)))
    return [{f: getattr(out[i], f) for f, _ in _abi.AsvK1Launch._fields_}
            for i in range(n.value)]


def _tuning(events=None, tile_rows: int = 0) -> AsvTuning:
    tu = AsvTuning()
    if events is not None:
        tu.begin_event, tu.end_event = events
    tu.tile_rows = tile_rows
    return tu


def state_fields(state) -> list:
    """Decode a [B, 112] u8 state tensor (copied to the host) into AsvReqState structs."""
    raw = state.detach().cpu().contiguous().numpy().tobytes()
    return [AsvReqState.from_buffer_copy(raw[i * STATE_BYTES:(i + 1) * STATE_BYTES])
            for i in range(state.shape[0])]


# ----------------------------------------------------------------------------- draft side

class DraftOut(NamedTuple):
    topk_id: "torch.Tensor"          # i32 [4B, 4]
    topk_logp: "torch.Tensor"        # f32 [4B, 4]
    row_lse: "torch.Tensor"          # f32 [4B]
    front_tok: "torch.Tensor"        # i32 [B, 4]
    draft_conf: Optional["torch.Tensor"]  # f32 [B] or None


def draft_workspace_bytes(B: int, H: int, V: int) -> int:
    out = ctypes.c_uint64(0)
    _check(load().asv_draft_workspace_bytes(B, H, V, ctypes.byref(out)))
    return int(out.value)


def alloc_draft_trees(B: int, device="cuda"):
    """Storage for B growing draft trees (``asv_draft_tree``, 3136 bytes each); asv_draft_step
    initialises them at step 0."""
    import torch
    return torch.empty((B, TREE_BYTES), dtype=torch.uint8, device=device)


def draft_step(hidden, w_draft, trees, step: int, state=None, shape=None, vocab_map=None,
               with_conf: bool = False, out: Optional[DraftOut] = None, workspace=None,
               events=None) -> DraftOut:
    """One draft step through ``asv_draft_step`` on torch's current stream.

    hidden bf16 [4B, H] (row 4b + j = frontier slot j of request b); w_draft bf16 [V, H] or its
    ``PackedLmHead`` from ``pack_draft_head``;
    trees u8 [B, 3136] (in/out); state u8 [B, 112] supplies each tree's shape at step 0, else
    ``shape`` = (nsteps, topk, ndt) for all; vocab_map int32 [V] or None.
    """
    import torch
    R, H = hidden.shape
    B = trees.shape[0]
    if R != TOPK_MAX * B:
        raise ValueError(f"hidden: expected {TOPK_MAX * B} rows (4 per request), got {R}")
    _need(hidden, "hidden", torch.bfloat16, (R, H))
    w_ptr, V, layout = _weight(w_draft, "draft", "w_draft", H)
    _need(trees, "trees", torch.uint8, (B, TREE_BYTES))
    if vocab_map is not None:
        _need(vocab_map, "vocab_map", torch.int32, (V,))
    if state is not None:
        _need(state, "state", torch.uint8, (B, STATE_BYTES))
    dev = hidden.device
    _same_device(dev, w_draft=w_draft.data if isinstance(w_draft, PackedLmHead) else w_draft,
                 trees=trees, vocab_map=vocab_map, state=state)
    if out is None:
        out = DraftOut(torch.empty((R, TOPK_MAX), dtype=torch.int32, device=dev),
                       torch.empty((R, TOPK_MAX), dtype=torch.float32, device=dev),
                       torch.empty(R, dtype=torch.float32, device=dev),
                       torch.empty((B, TOPK_MAX), dtype=torch.int32, device=dev),
                       torch.empty(B, dtype=torch.float32, device=dev) if with_conf else None)
    else:
        f32, i32 = torch.float32, torch.int32
        _need_out(out, dict(topk_id=(i32, (R, TOPK_MAX)), topk_logp=(f32, (R, TOPK_MAX)),
                            row_lse=(f32, (R,)), front_tok=(i32, (B, TOPK_MAX)),
                            draft_conf=(f32, (B,)) if out.draft_conf is not None else None),
                  dev)
    if workspace is None:
        workspace = torch.empty(max(draft_workspace_bytes(B, H, V), 256), dtype=torch.uint8,
                                device=dev)
    else:
        _need_workspace(workspace, draft_workspace_bytes(B, H, V), dev)
    a = AsvDraftArgs()
    a.B, a.H, a.V, a.step = B, H, V, step
    a.hidden, a.w_draft, a.w_draft_layout = hidden.data_ptr(), w_ptr, layout
    a.vocab_map, a.state = _ptr(vocab_map), _ptr(state)
    a.shape = (ctypes.c_int32 * 3)(*(shape or (1, 1, 1)))
    a.tree = trees.data_ptr()
    a.topk_id, a.topk_logp = out.topk_id.data_ptr(), out.topk_logp.data_ptr()
    a.row_lse, a.front_tok = out.row_lse.data_ptr(), out.front_tok.data_ptr()
    a.draft_conf = _ptr(out.draft_conf)
    lib = load()
    if events is None:
        _check(lib.asv_draft_step(ctypes.byref(a), workspace.data_ptr(), workspace.numel(),
                                  _stream_handle(dev)))
    else:
        tu = _tuning(events)
        _check(lib.asv_draft_step_tuned(ctypes.byref(a), ctypes.byref(tu), workspace.data_ptr(),
                                        workspace.numel(), _stream_handle(dev)))
    return out


def draft_prune(trees, n_cap: int, root_tok=None):
    """``asv_draft_prune``: (parent [n_cap], draft_tok [n_cap], req_offsets [B+1], req_status
    [B]) in the layout asv_verify reads; rows past req_offsets[B] are untouched."""
    import torch
    B = trees.shape[0]
    _need(trees, "trees", torch.uint8, (B, TREE_BYTES))
    if root_tok is not None:
        _need(root_tok, "root_tok", torch.int32, (B,))
    dev = trees.device
    parent = torch.empty(max(n_cap, 1), dtype=torch.int32, device=dev)
    tok = torch.empty(max(n_cap, 1), dtype=torch.int32, device=dev)
    off = torch.empty(B + 1, dtype=torch.int32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    _check(load().asv_draft_prune(trees.data_ptr(), B, _ptr(root_tok), n_cap,
                                  parent.data_ptr(), tok.data_ptr(), off.data_ptr(),
                                  status.data_ptr(), _stream_handle(dev)))
    return parent, tok, off, status


def draft_tree_fields(trees) -> list:
    """Decode a [B, 3136] u8 tree tensor (copied to the host) into AsvDraftTree structs."""
    raw = trees.detach().cpu().contiguous().numpy().tobytes()
    return [AsvDraftTree.from_buffer_copy(raw[i * TREE_BYTES:(i + 1) * TREE_BYTES])
            for i in range(trees.shape[0])]


# ----------------------------------------------------------------------------- around the target

def tree_meta(parent, req_offsets, pos_base=None, mask_words: int = 0):
    """``asv_tree_meta``: (pos [N], mask [N, mask_words] u32 as int32 or None, req_status [B])."""
    import torch
    N = parent.shape[0]
    B = req_offsets.shape[0] - 1
    _need(parent, "parent", torch.int32, (N,))
    _need(req_offsets, "req_offsets", torch.int32, (B + 1,))
    if pos_base is not None:
        _need(pos_base, "pos_base", torch.int32, (B,))
    dev = parent.device
    pos = torch.empty(N, dtype=torch.int32, device=dev)
    mask = (torch.empty((N, mask_words), dtype=torch.int32, device=dev) if mask_words > 0
            else None)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    _check(load().asv_tree_meta(parent.data_ptr(), req_offsets.data_ptr(), B, N,
                                _ptr(pos_base), mask_words, pos.data_ptr(), _ptr(mask),
                                status.data_ptr(), _stream_handle(dev)))
    return pos, mask, status


def commit(req_offsets, draft_tok, accepted_len, accepted_path, bonus_token, row_src=None):
    """``asv_commit``: (commit_off [B+1], commit_tok [N], commit_row [N], row_dst or None,
    req_status [B]). row_src: any contiguous [N, ...] tensor whose rows are a multiple of 4
    bytes; its kept rows are gathered into row_dst (same shape)."""
    import torch
    N = draft_tok.shape[0]
    B = req_offsets.shape[0] - 1
    _need(req_offsets, "req_offsets", torch.int32, (B + 1,))
    _need(draft_tok, "draft_tok", torch.int32, (N,))
    _need(accepted_len, "accepted_len", torch.int32, (B,))
    _need(accepted_path, "accepted_path", torch.int32, (N,))
    _need(bonus_token, "bonus_token", torch.int32, (B,))
    dev = draft_tok.device
    c_off = torch.empty(B + 1, dtype=torch.int32, device=dev)
    c_tok = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    c_row = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    dst = None
    a = AsvCommitArgs()
    a.B, a.N = B, N
    a.req_offsets, a.draft_tok = req_offsets.data_ptr(), draft_tok.data_ptr()
    a.accepted_len, a.accepted_path = accepted_len.data_ptr(), accepted_path.data_ptr()
    a.bonus_token = bonus_token.data_ptr()
    a.commit_off, a.commit_tok, a.commit_row = c_off.data_ptr(), c_tok.data_ptr(), c_row.data_ptr()
    if row_src is not None:
        if row_src.device.type != "cuda" or not row_src.is_contiguous() or row_src.shape[0] != N:
            raise ValueError("row_src: a contiguous GPU tensor with N rows")
        dst = torch.empty_like(row_src)
        a.row_src, a.row_dst = row_src.data_ptr(), dst.data_ptr()
        a.row_bytes = row_src[0].numel() * row_src.element_size() if N else 4
    a.req_status = status.data_ptr()
    _check(load().asv_commit(ctypes.byref(a), _stream_handle(dev)))
    return c_off, c_tok, c_row, dst, status
