"""The C-ABI library: it loads, exports every entry point of include/asv.h, and rejects bad
arguments on the host before touching the GPU (these calls run without a GPU)."""

import ctypes
import os
import re

import pytest

import paper_2609_02897_amd as asv
from paper_2609_02897_amd import _abi, _build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not _build.is_built():
        _build.build_library()
    return asv.load()


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "asv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(asv_[a-z0-9_]+)\s*\(", src)))


def test_header_matches_binding():
    assert _declared_functions() == sorted(_abi.EXPORTS)


def test_exports(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status(lib):
    assert lib.asv_version() == 160
    for code in (0, -1, -2, -3, -4, 7):
        assert lib.asv_status_string(code)


def test_struct_layouts():
    assert ctypes.sizeof(_abi.AsvReqState) == 112
    assert ctypes.sizeof(_abi.AsvParams) == 60
    # 4 ints, 18 pointers, params (60 B), the layout int
    assert ctypes.sizeof(_abi.AsvVerifyArgs) == 16 + 18 * 8 + 60 + 4
    assert ctypes.sizeof(_abi.AsvDraftTree) == 64 + 3 * 4 * 256
    # 4 ints, 4 pointers, 3 ints (+4 padding), 6 pointers, 1 int (+4 padding)
    assert ctypes.sizeof(_abi.AsvDraftArgs) == 16 + 4 * 8 + 16 + 6 * 8 + 8
    # 2 event pointers, the tile int (+4 padding)
    assert ctypes.sizeof(_abi.AsvTuning) == 2 * 8 + 8
    # 2 ints, 10 pointers, an int64, a pointer
    assert ctypes.sizeof(_abi.AsvCommitArgs) == 8 + 10 * 8 + 8 + 8


def test_param_and_policy_checks_on_host(lib):
    """Invalid parameters are rejected before anything is enqueued (no GPU needed)."""
    state = ctypes.c_void_p(0x1000)      # never dereferenced: the call must fail first
    good = asv.make_params()
    assert lib.asv_tree_policy(None, None, 0, ctypes.byref(good), None) == asv.ASV_OK
    assert lib.asv_tree_policy(None, None, 3, ctypes.byref(good), None) == asv.ASV_EINVAL
    assert lib.asv_tree_policy(None, state, -1, ctypes.byref(good), None) == asv.ASV_EINVAL
    for bad in (asv.make_params(dcs_divisor=0.0), asv.make_params(dcs_divisor=-1.0),
                asv.make_params(dcs_divisor=float("nan")),
                asv.make_params(dcs_divisor=float("inf")),
                asv.make_params(shape_lo=(0, 4, 4)), asv.make_params(shape_hi=(7, 0, 8)),
                asv.make_params(shape_start=(3, 4, -1)), asv.make_params(alpha=0.0),
                asv.make_params(breaker_n=0), asv.make_params(max_promotions=-2),
                asv.make_params(temperature=0.0), asv.make_params(temperature=float("inf"))):
        assert lib.asv_tree_policy(None, state, 4, ctypes.byref(bad), None) == asv.ASV_EINVAL
        assert lib.asv_state_init(state, 4, ctypes.byref(bad), None) == asv.ASV_EINVAL


def test_workspace_bytes(lib):
    out = ctypes.c_uint64(0)
    assert lib.asv_workspace_bytes(1, 60, 4096, 128256, ctypes.byref(out)) == 0
    S = (128256 + 255) // 256
    assert out.value >= 3 * 60 * S * 4
    assert out.value % 256 == 0
    assert lib.asv_workspace_bytes(0, 0, 64, 10, ctypes.byref(out)) == 0
    for bad in [(1, 0, 64, 10), (2, 1, 64, 10), (1, 4, 100, 10), (1, 4, 64, 0),
                (-1, 4, 64, 10), (1, 4, (1 << 20) + 64, 10),
                (1, 1 << 30, 64, 10), (1, 4, 64, 1 << 30),      # indices past 2^30
                (1, 1 << 24, 64, 1 << 23)]:                        # 2^33 LM-head workgroups
        assert lib.asv_workspace_bytes(*bad, ctypes.byref(out)) == asv.ASV_EINVAL, bad
    # the largest accepted workgroup count: ceil(V / 256) * ceil(N / 64) just below 2^31
    assert lib.asv_workspace_bytes(1, 64 * 1023, 64, 256 * (((1 << 31) - 1) // 1023),
                                   ctypes.byref(out)) == 0
    assert lib.asv_workspace_bytes(1, 4, 64, 10, None) == asv.ASV_EINVAL


def test_verify_rejects_on_host(lib):
    """Every rejection below happens before any HIP call, so it runs without a GPU."""
    a = _abi.AsvVerifyArgs()
    assert lib.asv_verify(None, None, 0, None) == asv.ASV_EINVAL
    a.B, a.N, a.H, a.V = 1, 4, 100, 10          # H not a multiple of 64
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.H = 64                                    # null pointers
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    fake = 0x100000
    for f, _ in _abi.AsvVerifyArgs._fields_[4:]:
        if f not in ("params", "draft_logits", "draft_conf", "state", "w_lm_layout"):
            setattr(a, f, fake)
    a.params = asv.make_params()
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EWORKSPACE
    tu = _abi.AsvTuning()
    assert lib.asv_verify_tuned(ctypes.byref(a), None, None, 0, None) == asv.ASV_EWORKSPACE
    for rows in (0, 64, 128, 192, 256):             # a forced LM-head tile is accepted
        tu.tile_rows = rows
        assert lib.asv_verify_tuned(ctypes.byref(a), ctypes.byref(tu), None, 0,
                                    None) == asv.ASV_EWORKSPACE
    for rows in (-1, 1, 100, 512):                  # a value that names no tile is not
        tu.tile_rows = rows
        assert lib.asv_verify_tuned(ctypes.byref(a), ctypes.byref(tu), None, 0,
                                    None) == asv.ASV_EINVAL
    for layout in (asv.W_ROW_MAJOR, asv.W_PACKED):  # both weight layouts are accepted
        a.w_lm_layout = layout
        assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EWORKSPACE
    for layout in (-1, 2, 7):
        a.w_lm_layout = layout
        assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.w_lm_layout = asv.W_ROW_MAJOR
    a.params = asv.make_params(alpha=0.0)
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.params = asv.make_params(breaker_n=0)
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.params = asv.make_params(max_promotions=-2)
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.params = asv.make_params()
    a.hidden = fake + 2                         # misaligned bf16 rows
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.hidden = fake
    need = ctypes.c_uint64(0)
    lib.asv_workspace_bytes(1, 4, 64, 10, ctypes.byref(need))
    assert lib.asv_verify(ctypes.byref(a), ctypes.c_void_p(fake + 64), need.value,
                          None) == asv.ASV_EWORKSPACE          # misaligned workspace
    assert lib.asv_verify(ctypes.byref(a), ctypes.c_void_p(fake), need.value - 1,
                          None) == asv.ASV_EWORKSPACE          # too small
    a.B, a.N = 0, 0                              # empty batch: nothing to do
    assert lib.asv_verify(ctypes.byref(a), None, 0, None) == asv.ASV_OK


def test_verify_noalloc_rejects_on_host(lib):
    """asv_verify_noalloc refuses sizes beyond its static scratch (and bad sizes) before any
    HIP call; an empty batch is a no-op."""
    a = _abi.AsvVerifyArgs()
    assert lib.asv_verify_noalloc(None, None) == asv.ASV_EINVAL
    assert lib.asv_verify_noalloc(ctypes.byref(a), None) == asv.ASV_EINVAL     # H = 0
    a.B, a.N, a.H, a.V = 1, 8192, 64, 151936
    need = ctypes.c_uint64(0)
    assert lib.asv_workspace_bytes(a.B, a.N, a.H, a.V, ctypes.byref(need)) == asv.ASV_OK
    assert need.value > asv.STATIC_SCRATCH_BYTES
    assert lib.asv_verify_noalloc(ctypes.byref(a), None) == asv.ASV_ESCRATCH
    assert b"static scratch" in lib.asv_last_error()
    assert b"static scratch" in lib.asv_status_string(asv.ASV_ESCRATCH)
    a.B, a.N = 0, 0
    assert lib.asv_verify_noalloc(ctypes.byref(a), None) == asv.ASV_OK


def test_packed_lm_head_sizes_and_rejections(lib):
    """The packed weight holds ceil(V / 256) slabs of 256 rows; bad arguments are rejected
    before anything is enqueued."""
    out = ctypes.c_uint64(0)
    for V, H in ((128256, 4096), (151936, 4096), (1, 64), (256, 64), (257, 128)):
        assert lib.asv_packed_lm_head_bytes(V, H, ctypes.byref(out)) == asv.ASV_OK
        assert out.value == -(-V // 256) * 256 * H * 2
    assert lib.asv_packed_lm_head_bytes(128256, 16384, ctypes.byref(out)) == asv.ASV_OK
    assert out.value == 501 * 256 * 16384 * 2                 # 3.9 GiB: the largest kind
    for V, H in ((0, 64), (-1, 64), (10, 0), (10, 100), (10, 1 << 21),
                 (2048 * 256, 4096), (1 << 20, 4096)):      # 4 GiB and more
        assert lib.asv_packed_lm_head_bytes(V, H, ctypes.byref(out)) == asv.ASV_EINVAL
    assert lib.asv_packed_lm_head_bytes(10, 64, None) == asv.ASV_EINVAL
    V, H = 300, 64
    need = 2 * 256 * H * 2
    w, p = 0x100000, 0x100000 + (1 << 20)
    pk = lib.asv_pack_lm_head
    assert pk(None, V, H, p, need, None) == asv.ASV_EINVAL
    assert pk(w, V, H, None, need, None) == asv.ASV_EINVAL
    assert pk(w + 2, V, H, p, need, None) == asv.ASV_EINVAL        # misaligned weight
    assert pk(w, V, H, p + 8, need, None) == asv.ASV_EINVAL        # misaligned output
    assert pk(w, V, H, p, need - 1, None) == asv.ASV_EINVAL        # output too small
    assert pk(w, V, 100, p, need, None) == asv.ASV_EINVAL          # H not a multiple of 64
    assert pk(w, 0, H, p, need, None) == asv.ASV_EINVAL
    assert pk(w, V, H, w + V * H * 2 - 16, need, None) == asv.ASV_EINVAL   # overlap
    assert pk(p + need - 16, V, H, p, need, None) == asv.ASV_EINVAL        # overlap


def test_packed_draft_head_sizes_and_rejections(lib):
    """The packed draft weight holds V rounded up to a multiple of 128 rows; bad arguments and
    bad layouts are rejected before anything is enqueued."""
    out = ctypes.c_uint64(0)
    for V, H in ((32000, 4096), (4, 64), (128, 64), (129, 128), (777, 128)):
        assert lib.asv_packed_draft_head_bytes(V, H, ctypes.byref(out)) == asv.ASV_OK
        assert out.value == -(-V // 128) * 128 * H * 2
    for V, H in ((3, 64), (0, 64), (10, 100), (1 << 19, 4096)):
        assert lib.asv_packed_draft_head_bytes(V, H, ctypes.byref(out)) == asv.ASV_EINVAL
    V, H = 300, 64
    need = 384 * H * 2
    w, p = 0x100000, 0x100000 + (1 << 20)
    pk = lib.asv_pack_draft_head
    assert pk(None, V, H, p, need, None) == asv.ASV_EINVAL
    assert pk(w, V, H, p, need - 1, None) == asv.ASV_EINVAL
    assert pk(w, 3, H, p, need, None) == asv.ASV_EINVAL
    assert pk(w, V, H, w + 64, need, None) == asv.ASV_EINVAL              # overlap
    a = _abi.AsvDraftArgs()
    a.B, a.H, a.V = 1, 64, 300
    for layout in (-1, 2):
        a.w_draft_layout = layout
        assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL
    a.B = 0                                   # an empty batch with a valid layout is a no-op
    for layout in (asv.W_ROW_MAJOR, asv.W_PACKED):
        a.w_draft_layout = layout
        assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_OK


def test_state_init_rejects(lib):
    p = asv.make_params()
    assert lib.asv_state_init(None, 3, ctypes.byref(p), None) == asv.ASV_EINVAL
    assert lib.asv_state_init(None, 0, ctypes.byref(p), None) == asv.ASV_OK


def test_microbench_library_exports_and_checks():
    """The measurement-only library exports what include/asv_microbench.h declares and rejects
    bad arguments before launching."""
    if not _build.is_built(_build.MICROBENCH_OUT):
        _build.build_microbench()
    asv.load()      # binds the HIP runtime the process already uses
    mb = ctypes.CDLL(_build.MICROBENCH_OUT)
    src = open(os.path.join(ROOT, "include", "asv_microbench.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(asvb_[a-z0-9_]+)\s*\(", src)))
    assert names == ["asvb_lds_read", "asvb_mfma_loop", "asvb_stream_read",
                     "asvb_stream_read_nt"]
    for n in names:
        assert hasattr(mb, n), n
    for f in (mb.asvb_stream_read, mb.asvb_stream_read_nt):
        f.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int32,
                      ctypes.c_void_p]
    mb.asvb_mfma_loop.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_void_p]
    p = ctypes.c_void_p(0x1000)
    assert mb.asvb_stream_read(None, 64, p, 4, None) == -1
    assert mb.asvb_stream_read(p, 65, p, 4, None) == -1           # not a multiple of 16
    assert mb.asvb_stream_read(ctypes.c_void_p(0x1004), 64, p, 4, None) == -1
    assert mb.asvb_stream_read(p, 64, p, 0, None) == -1
    for bad in ((None, 64, p, 4), (p, 65, p, 4), (ctypes.c_void_p(0x1004), 64, p, 4),
                (p, 64, p, 0), (p, 64, None, 4)):
        assert mb.asvb_stream_read_nt(*bad, None) == -1
    assert mb.asvb_mfma_loop(None, 4, 4, None) == -1
    assert mb.asvb_mfma_loop(p, 0, 4, None) == -1
    mb.asvb_lds_read.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                 ctypes.c_int32, ctypes.c_void_p]
    for bad in ((None, 4, p, 4), (p, 0, p, 4), (p, 4, None, 4), (p, 4, p, 0)):
        assert mb.asvb_lds_read(*bad, None) == -1


def test_draft_and_tree_entry_points_reject_on_host(lib):
    """asv_draft_*, asv_tree_meta and asv_commit reject bad arguments before any HIP call."""
    out = ctypes.c_uint64(0)
    assert lib.asv_draft_workspace_bytes(2, 4096, 32000, ctypes.byref(out)) == 0
    S = (32000 + 63) // 64                         # 8 draft rows use 64-wide vocabulary slabs
    assert out.value >= 8 * S * (4 + 4 + 1) * 4 and out.value % 256 == 0
    for bad in [(-1, 64, 10), (1, 100, 10), (1, 64, 3), (1, 0, 10), (1, 64, 1 << 30),
                (1 << 20, 64, 1 << 29)]:                          # 2^32 draft workgroups
        assert lib.asv_draft_workspace_bytes(*bad, ctypes.byref(out)) == asv.ASV_EINVAL, bad
    assert lib.asv_draft_workspace_bytes(1, 64, (1 << 30) - 1, ctypes.byref(out)) == 0
    a = _abi.AsvDraftArgs()
    a.B, a.H, a.V, a.step = 0, 64, 10, 0
    assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_OK       # empty batch
    a.B = 1
    assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL   # null pointers
    fake = 0x100000
    for f in ("hidden", "w_draft", "tree", "topk_id", "topk_logp", "row_lse", "front_tok"):
        setattr(a, f, fake)
    for shape in [(0, 1, 1), (1, 5, 4), (1, 1, 0), (17, 4, 8)]:   # the last overflows the pool
        a.shape = (ctypes.c_int32 * 3)(*shape)
        assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL, shape
    a.shape = (ctypes.c_int32 * 3)(3, 4, 4)
    assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EWORKSPACE
    a.hidden = fake + 2
    assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL   # misaligned
    a.hidden = fake
    tu = _abi.AsvTuning()
    assert lib.asv_draft_step_tuned(ctypes.byref(a), ctypes.byref(tu), None, 0,
                                    None) == asv.ASV_EWORKSPACE
    tu.tile_rows = 64                              # the draft LM head takes no forced tile
    assert lib.asv_draft_step_tuned(ctypes.byref(a), ctypes.byref(tu), None, 0,
                                    None) == asv.ASV_EINVAL
    a.hidden, a.step = fake, -1
    assert lib.asv_draft_step(ctypes.byref(a), None, 0, None) == asv.ASV_EINVAL

    p = ctypes.c_void_p(fake)
    assert lib.asv_draft_prune(None, 0, None, 0, None, None, None, None, None) == asv.ASV_OK
    assert lib.asv_draft_prune(p, -1, None, 0, p, p, p, p, None) == asv.ASV_EINVAL
    assert lib.asv_draft_prune(p, 1, None, -1, p, p, p, p, None) == asv.ASV_EINVAL
    assert lib.asv_draft_prune(p, 1, None, 4, None, p, p, p, None) == asv.ASV_EINVAL

    assert lib.asv_tree_meta(None, None, 0, 0, None, 0, None, None, None, None) == asv.ASV_OK
    assert lib.asv_tree_meta(p, p, 2, 1, None, 0, p, None, p, None) == asv.ASV_EINVAL  # N < B
    assert lib.asv_tree_meta(p, p, 1, 4, None, 0, p, p, p, None) == asv.ASV_EINVAL  # 0 words
    assert lib.asv_tree_meta(None, p, 1, 4, None, 1, p, p, p, None) == asv.ASV_EINVAL

    c = _abi.AsvCommitArgs()
    assert lib.asv_commit(ctypes.byref(c), None) == asv.ASV_OK                      # B = N = 0
    c.B, c.N = 1, 4
    assert lib.asv_commit(ctypes.byref(c), None) == asv.ASV_EINVAL                  # nulls
    for f in ("req_offsets", "draft_tok", "accepted_len", "accepted_path", "bonus_token",
              "commit_off", "commit_tok", "commit_row", "req_status"):
        setattr(c, f, fake)
    c.row_src, c.row_dst, c.row_bytes = fake, fake, 6                               # not % 4
    assert lib.asv_commit(ctypes.byref(c), None) == asv.ASV_EINVAL
    c.row_bytes, c.row_dst = 8, None
    assert lib.asv_commit(ctypes.byref(c), None) == asv.ASV_EINVAL
    c.row_dst, c.row_src = fake, fake + 2                                           # misaligned
    assert lib.asv_commit(ctypes.byref(c), None) == asv.ASV_EINVAL


def test_inputs_on_another_device_are_rejected():
    """The binding refuses inputs that sit on another device than the hidden states (the
    kernels would read them through a foreign address); None entries are skipped."""
    torch = pytest.importorskip("torch")
    dev = torch.device("cuda", 0)
    with pytest.raises(ValueError, match="w_lm"):
        asv._same_device(dev, w_lm=torch.empty(2, device="meta"))
    with pytest.raises(ValueError, match="tau"):
        asv._same_device(dev, parent=None, tau=torch.empty(2, device="meta"))
    asv._same_device(dev, state=None)
