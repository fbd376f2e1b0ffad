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
    ASV_EHIP, ASV_EINVAL, ASV_EWORKSPACE, ASV_OK, EXPORTS, LIB_PATH, RS_BAD_OFFSETS,
    RS_BAD_PARENT, RS_BAD_ROOT, RS_BAD_TAU, RS_BAD_TOKEN, AsvParams, AsvReqState,
    AsvVerifyArgs, LibraryMissing, load)

STATE_BYTES = ctypes.sizeof(AsvReqState)


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
        detail = lib.asv_last_error().decode() if code == ASV_EHIP else ""
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


def verify(hidden, w_lm, draft_tok, parent, req_offsets, tau, draft_logits=None, state=None,
           params: Optional[AsvParams] = None, out: Optional[VerifyOut] = None,
           workspace=None, k1_events=None) -> VerifyOut:
    """One verification step through ``asv_verify`` on torch's current stream.

    hidden bf16 [N, H]; w_lm bf16 [V, H]; draft_tok, parent int32 [N]; req_offsets int32
    [B+1]; tau float32 [B]; draft_logits float32 [N, V] or None; state u8 [B, 112] (in/out) or
    None. ``out`` and ``workspace`` may be passed to reuse buffers. ``k1_events`` is an
    optional pair of raw hipEvent_t handles recorded around the LM-head kernel.
    """
    import torch
    N, H = hidden.shape
    V = w_lm.shape[0]
    B = req_offsets.shape[0] - 1
    _need(hidden, "hidden", torch.bfloat16, (N, H))
    _need(w_lm, "w_lm", torch.bfloat16, (V, H))
    _need(draft_tok, "draft_tok", torch.int32, (N,))
    _need(parent, "parent", torch.int32, (N,))
    _need(req_offsets, "req_offsets", torch.int32, (B + 1,))
    _need(tau, "tau", torch.float32, (B,))
    if draft_logits is not None:
        _need(draft_logits, "draft_logits", torch.float32, (N, V))
    if state is not None:
        _need(state, "state", torch.uint8, (B, STATE_BYTES))
    dev = hidden.device
    if out is None:
        out = alloc_outputs(B, N, dev, draft_logits is not None)
    if workspace is None:
        workspace = alloc_workspace(B, N, H, V, dev)
    a = AsvVerifyArgs()
    a.B, a.N, a.H, a.V = B, N, H, V
    a.hidden, a.w_lm = hidden.data_ptr(), w_lm.data_ptr()
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
    if k1_events is not None:
        a.k1_begin_event, a.k1_end_event = k1_events
    _check(load().asv_verify(ctypes.byref(a), workspace.data_ptr(), workspace.numel(),
                             _stream_handle(dev)))
    return out


def state_fields(state) -> list:
    """Decode a [B, 96] u8 state tensor (copied to the host) into AsvReqState structs."""
    raw = state.detach().cpu().contiguous().numpy().tobytes()
    return [AsvReqState.from_buffer_copy(raw[i * STATE_BYTES:(i + 1) * STATE_BYTES])
            for i in range(state.shape[0])]
