"""Throughput of the AdaptiveSpec verification hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1|3] [--no-cpu] \
                    [--secondary 3|none] [--no-draft] | --reference | --copy-calibration MIB

A step is one asv_verify call (LM-head kernel over every tree row with the per-slab
reductions and drafted-logit gather, then the fused slab merge + margin rule + tree walk +
policy-state update) on one batch of
seeded synthetic inputs already resident in HBM. The headline workload is the Llama-3.1-8B
shaped batch-1 verify (H=4096, V=128256, one 60-node EAGLE-style tree, kappa=0.3); the
32x64-node batch (2048 rows) is measured after it as the MFMA-bound point. Prints one JSON
line: verified tree nodes per second, the LM-head kernel's roofline fraction (its duration
from HIP events that carry its dispatches' start and end times, in a second timed pass) and
the CPU oracle's throughput on a
bounded sample of the same workload. The JSON line also carries the draft step that precedes
verification (``draft``: the draft LM head reduced to each row's top-4, and one tree-growth
step) on the EAGLE-3-shaped draft head at batch 1 and 32, with its kernel's roofline.
"""

from __future__ import annotations

import argparse
import ctypes
import hashlib
import re
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 flop/clk)
TABLES = os.path.join(ROOT, "tests", "golden")
TRAFFIC = os.path.join(ROOT, "profiles", "k1_traffic.json")
# the kernels and the host code that picks their tiles
K1_SOURCES = [os.path.join(ROOT, "paper_2609_02897_amd", "csrc", f)
              for f in ("k_lmhead.h", "k_common.h", "asv_api.hip")]
K5_SOURCES = [os.path.join(ROOT, "paper_2609_02897_amd", "csrc", f)
              for f in ("k_draft.h", "k_lmhead.h", "k_common.h", "asv_api.hip")]


def _code_text(path) -> str:
    """The C++ source with comments removed and whitespace collapsed: what the kernel is made
    of, so that a comment edit does not disown the counters taken on the same code."""
    src = open(path, encoding="utf-8").read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def _sha(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        h.update(_code_text(p).encode())
    return h.hexdigest()[:16]


def k1_source_sha() -> str:
    return _sha(K1_SOURCES)


def k5_source_sha() -> str:
    return _sha(K5_SOURCES)


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime torch loaded (same soname)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                 ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(ev)) == 0
        return ev.value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value

    def destroy(self, ev: int):
        self.hip.hipEventDestroy(ev)

    def record(self, ev: int, stream: int):
        assert self.hip.hipEventRecord(ctypes.c_void_p(ev), ctypes.c_void_p(stream)) == 0


def load_workload(cfg: int, step: int = 0):
    from workloads import CONFIGS, make_workload
    w = make_workload(cfg, step)
    path = os.path.join(TABLES, f"oracle_cfg{cfg}.npz")
    with np.load(path, allow_pickle=False) as t:
        w.draft_tok = t[f"draft_tok_s{step}"].astype(np.int32)
        assert t[f"sha_hidden_s{step}"] == hashlib.sha256(w.hidden.tobytes()).hexdigest(), \
            "seeded hidden states differ from the ones the oracle tables were made for"
    return w, CONFIGS[cfg]


def to_device(w, W, dev):
    import torch

    def t(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    return dict(hidden=t(w.hidden.view(np.int16)).view(torch.bfloat16),
                w_lm=t(W.view(np.int16)).view(torch.bfloat16),
                draft_tok=t(w.draft_tok), parent=t(w.parent), req_offsets=t(w.req_offsets),
                tau=t(w.tau),
                draft_logits=None if w.draft_logits is None else t(w.draft_logits))


def _per_call_us(fn, reps: int) -> float:
    import torch
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    return 1e6 * (time.perf_counter() - t0) / reps


def measure(cfg: int, steps: int, warmup: int, dev, hip: HipEvents, tau=None,
            layout: str = "packed", before_warmup=None):
    """Time asv_verify on configuration `cfg`. With layout "packed" the LM-head weight is
    packed once (asv_pack_lm_head, as at model load; timed alone as pack_ms) and the row-major
    copy freed before anything is timed; "row-major" passes the [V, H] weight as it is.
    ``before_warmup`` runs once the inputs are resident, right before the warm-up steps."""
    import torch
    import paper_2609_02897_amd as asv
    w, c = load_workload(cfg)
    if tau is not None:
        w.tau[:] = np.float32(tau)
    W = w.weights()
    d = to_device(w, W, dev)
    pack_ms = None
    if layout == "packed":
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        packed = asv.pack_lm_head(d["w_lm"])
        torch.cuda.synchronize()
        pack_ms = 1e3 * (time.perf_counter() - t0)
        d["w_lm"] = packed
        torch.cuda.empty_cache()
    out = asv.alloc_outputs(w.B, w.N, dev, d["draft_logits"] is not None)
    ws = asv.alloc_workspace(w.B, w.N, w.H, w.V, dev)
    state = asv.state_init(w.B, device=dev)
    evs = [(hip.create(), hip.create()) for _ in range(steps)]

    def step(k1=None):
        asv.verify(d["hidden"], d["w_lm"], d["draft_tok"], d["parent"], d["req_offsets"],
                   d["tau"], d["draft_logits"], state=state, out=out, workspace=ws,
                   k1_events=k1)

    if before_warmup is not None:
        before_warmup()
    for _ in range(warmup):
        step()
    # Timed region 1: the throughput. Nothing but the verify calls is enqueued.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    # Timed region 2: the same steps with HIP events set to the start of the LM-head kernel's
    # first launch and the end of its last, on the stream it runs on (the library passes them
    # to hipExtLaunchKernelGGL; this region is kept out of the throughput).
    torch.cuda.synchronize()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    k1_ms = [hip.elapsed_ms(a, b) for a, b in evs]
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    status = out.req_status.cpu().numpy()
    assert np.all(status == 0), status
    # The steps on either side of the target forward on the same trees: tree-attention metadata
    # (positions and ancestor masks) and the commit of this step's accepted paths with a gather
    # of their hidden rows. Both are latency-bound; host-inclusive wall clock per call.
    words = (int(np.diff(w.req_offsets).max()) + 31) // 32
    base = torch.zeros(w.B, dtype=torch.int32, device=dev)
    around = dict(
        tree_meta_us_per_call=round(_per_call_us(
            lambda: asv.tree_meta(d["parent"], d["req_offsets"], base, words), steps), 2),
        commit_us_per_call=round(_per_call_us(
            lambda: asv.commit(d["req_offsets"], d["draft_tok"], out.accepted_len,
                               out.accepted_path, out.bonus_token, d["hidden"]), steps), 2),
        note="host-inclusive wall clock per call; kernel durations in profiles/")
    k1_avg = float(np.mean(k1_ms))
    nodes = w.N * steps
    bytes_alg = 2 * w.V * w.H + 2 * w.N * w.H
    flops_alg = 2 * w.N * w.V * w.H
    res = dict(cfg=cfg, name=c["name"], N=w.N, B=w.B, H=w.H, V=w.V, layout=layout,
               pack_ms=pack_ms, tau=float(w.tau[0]), value=nodes / dt,
               ms_per_step=1e3 * dt / steps,
               k1_avg_ms=k1_avg, k1_min_ms=float(np.min(k1_ms)),
               k1_share=k1_avg * steps / (1e3 * dt),
               hbm_gbs=bytes_alg / (k1_avg * 1e-3) / 1e9,
               mfma_tflops=flops_alg / (k1_avg * 1e-3) / 1e12,
               bytes_alg=bytes_alg, flops_alg=flops_alg,
               accepted_len=out.accepted_len.cpu().numpy().tolist()[:4],
               mean_accepted_len=float(out.accepted_len.float().mean().cpu()), around=around)
    del d, out, ws
    torch.cuda.empty_cache()
    return res, w, W


def _microbench_lib():
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_02897_amd", "libasv_microbench.so"))
    for f in (lib.asvb_stream_read, lib.asvb_stream_read_nt):
        f.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int32,
                      ctypes.c_void_p]
    return lib


def measure_draft(name: str, steps: int, warmup: int, dev, hip: HipEvents, cpu: bool,
                  layout: str = "packed") -> dict:
    """One draft step (asv_draft_step: the draft LM head with its top-4 epilogue, then the slab
    merge and one tree-growth step) on the EAGLE-3-shaped draft head (H=4096, 32000 draft ids),
    trees of the wide end of the paper's range (3,4,4): four draft rows per request.

    Throughput: back-to-back steps. The draft LM head (262 MB) fits the 256 MB last-level cache
    about whole, which back-to-back launches would read from; in a decode loop the draft
    model's other weights evict it between steps, so the kernel's roofline uses launches that
    each follow a clean 1 GiB read, timed with HIP events around the kernel on its stream."""
    import torch
    import paper_2609_02897_amd as asv
    from workloads import make_draft_workload
    dw = make_draft_workload(name)
    W, x, vmap = dw.weights(), dw.hidden(0), dw.vocab_map()

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    wd = t(W.view(np.int16)).view(torch.bfloat16)
    if layout == "packed":          # once, as at model load; the row-major copy is freed
        wd = asv.pack_draft_head(wd)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    xd = t(x.view(np.int16)).view(torch.bfloat16)
    vm = t(vmap)
    B, R = dw.B, 4 * dw.B
    shape = (3, 4, 4)
    trees = asv.alloc_draft_trees(B, dev)
    ws = torch.empty(max(asv.draft_workspace_bytes(B, dw.H, dw.V), 256), dtype=torch.uint8,
                     device=dev)
    out = asv.draft_step(xd, wd, trees, 0, shape=shape, vocab_map=vm, workspace=ws,
                         with_conf=True)

    def step(i, ev=None):
        asv.draft_step(xd, wd, trees, i % shape[0], shape=shape, vocab_map=vm, out=out,
                       workspace=ws, events=ev)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    # cold launches: a clean read of 1 GiB before each, outside the event window
    mb = _microbench_lib()
    flush = torch.ones((1 << 30) // 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(1 << 16, dtype=torch.int32, device=dev)
    handle = torch.cuda.current_stream(dev).cuda_stream
    reps = 50
    evs = [(hip.create(), hip.create()) for _ in range(reps)]
    for i in range(reps):
        assert mb.asvb_stream_read(flush.data_ptr(), 1 << 30, sink.data_ptr(), 1024,
                                   handle) == 0
        step(i, evs[i])
    torch.cuda.synchronize()
    k_ms = [hip.elapsed_ms(a, b) for a, b in evs]
    # the achievable ceiling for this launch: a streaming read of the same number of bytes
    # after the same flush, best of the plain and the non-temporal read at two grid sizes
    n_rd = (2 * dw.V * dw.H) // 16 * 16
    rd = torch.ones(n_rd // 4, dtype=torch.int32, device=dev)
    rd_ms = []
    for read, grid in ((mb.asvb_stream_read, 1024), (mb.asvb_stream_read, 2048),
                       (mb.asvb_stream_read_nt, 512), (mb.asvb_stream_read_nt, 1024)):
        t_ms = []
        for i in range(20):
            assert mb.asvb_stream_read(flush.data_ptr(), 1 << 30, sink.data_ptr(), 1024,
                                       handle) == 0
            a, b = evs[i]
            hip.record(a, handle)
            assert read(rd.data_ptr(), n_rd, sink.data_ptr(), grid, handle) == 0
            hip.record(b, handle)
            torch.cuda.synchronize()
            t_ms.append(hip.elapsed_ms(a, b))
        rd_ms.append(float(np.mean(t_ms)))
    read_gbs = n_rd / (min(rd_ms) * 1e-3) / 1e9
    del rd
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    del flush
    # pruning the grown trees into the verification layout (host-inclusive, per call)
    for i in range(shape[0]):
        step(i)
    prune_us = _per_call_us(lambda: asv.draft_prune(trees, B * shape[2]), steps)
    k_avg = float(np.mean(k_ms))
    S = (dw.V + (64 if R <= 64 else 128) - 1) // (64 if R <= 64 else 128)
    bytes_alg = 2 * dw.V * dw.H + 2 * R * dw.H + R * S * 36
    flops_alg = 2 * R * dw.V * dw.H
    res = dict(workload=name, requests=B, rows=R, H=dw.H, V=dw.V, tree_shape=list(shape),
               w_layout=layout,
               us_per_step=round(1e6 * dt / steps, 2),
               draft_steps_per_s=round(steps / dt, 1),
               prune_us_per_call=round(prune_us, 2),
               roofline=dict(bound="hbm", kernel="k_draft_partial",
                             k_avg_us_cold=round(1e3 * k_avg, 2),
                             achieved=round(bytes_alg / (k_avg * 1e-3) / 1e9, 1),
                             peak=HBM_PEAK_GBS, unit="GB/s",
                             frac=round(bytes_alg / (k_avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                             measured_peak=round(read_gbs, 1),
                             frac_of_measured=round(bytes_alg / (k_avg * 1e-3) / 1e9 / read_gbs,
                                                    4),
                             bytes_alg=bytes_alg, flops_alg=flops_alg,
                             traffic=measured_draft_traffic(name)))
    if cpu:
        import oracle
        w64 = oracle.widen_weights(W)
        x64 = oracle.widen_bf16(x)
        n, t0 = 0, time.perf_counter()
        while n < 3 or time.perf_counter() - t0 < 3.0:
            oracle.draft_topk(x64, w64, 4, vmap)
            n += 1
        res["cpu_oracle_us_per_step"] = round(1e6 * (time.perf_counter() - t0) / n, 1)
    del wd, xd, ws, out, trees
    torch.cuda.empty_cache()
    return res


def roofline(r: dict, ceilings: dict = None) -> dict:
    """Roofline of K1 against the published peak; with ``ceilings`` (measured_ceilings) also
    against the peak a microbenchmark reaches on this GPU."""
    bound_hbm = r["bytes_alg"] / (HBM_PEAK_GBS * 1e9) >= r["flops_alg"] / (BF16_PEAK_TFLOPS * 1e12)
    if bound_hbm:
        ro = dict(bound="hbm", achieved=round(r["hbm_gbs"], 1), peak=HBM_PEAK_GBS, unit="GB/s",
                  frac=round(r["hbm_gbs"] / HBM_PEAK_GBS, 4))
        measured = (ceilings or {}).get("stream_read_gbps")
    else:
        ro = dict(bound="mfma", achieved=round(r["mfma_tflops"], 1), peak=BF16_PEAK_TFLOPS,
                  unit="TFLOP/s", frac=round(r["mfma_tflops"] / BF16_PEAK_TFLOPS, 4))
        measured = (ceilings or {}).get("mfma_bf16_tflops")
    if measured:
        ro["measured_peak"] = measured
        ro["frac_of_measured"] = round(ro["achieved"] / measured, 4)
    ro["kernel"] = "k_lmhead_partial"
    ro["k1_avg_us"] = round(1e3 * r["k1_avg_ms"], 2)
    ro["traffic"] = measured_traffic(r["cfg"])
    return ro


def other_bound(r: dict) -> dict:
    """K1 against the roofline that does not bind at this row count (both fractions are asked
    for where the row count sits near the ridge)."""
    return dict(hbm_frac=round(r["hbm_gbs"] / HBM_PEAK_GBS, 4),
                mfma_frac=round(r["mfma_tflops"] / BF16_PEAK_TFLOPS, 4))


def measured_traffic(cfg: int):
    """HBM bytes per K1 launch from the committed rocprofv3 counter summary, if it was taken
    on the current K1 source; otherwise None."""
    if not os.path.exists(TRAFFIC):
        return None
    with open(TRAFFIC) as f:
        t = json.load(f)
    e = t.get(f"cfg{cfg}")
    if not e or t.get("k1_source_sha") != k1_source_sha():
        return None
    return e.get("bytes_per_launch")


def measured_draft_traffic(name: str):
    """The same for the draft LM-head kernel, keyed by draft workload."""
    if not os.path.exists(TRAFFIC):
        return None
    with open(TRAFFIC) as f:
        t = json.load(f)
    e = t.get(name)
    if not e or t.get("k5_source_sha") != k5_source_sha():
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(w, W, budget_s: float = 12.0, requests: int = 0) -> dict:
    """The float64 oracle on the same step, repeated until about ``budget_s`` of CPU work. With
    ``requests`` > 0 only the first that many requests of the batch (their rows, trees and
    thresholds) make up the sample, for workloads whose full step takes the oracle longer."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    B = w.B if requests <= 0 else min(requests, w.B)
    n_rows = int(w.req_offsets[B])
    args = (w.hidden[:n_rows], w.draft_tok[:n_rows], w.parent[:n_rows], w.req_offsets[:B + 1],
            w.tau[:B], None if w.draft_logits is None else w.draft_logits[:n_rows])
    w64 = oracle.widen_weights(W)
    n, t0 = 0, time.perf_counter()
    while True:
        oracle.verify(w64, *args)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    what = (f"{n} full verify steps of the workload ({n_rows} rows each)" if B == w.B else
            f"{n} verify steps of the first {B} of its {w.B} requests ({n_rows} of "
            f"{w.N} rows)")
    return dict(value=round(n_rows * n / dt, 2), unit="nodes/s", cores=int(threads),
                kind="oracle",
                sample=f"{what}; float64 logits via BLAS, weights pre-widened outside the "
                       f"timing; {dt:.1f} s")


def measured_ceilings(dev) -> dict:
    """Achievable peaks on this GPU from the microbenchmark library (include/asv_microbench.h):
    a streaming read of 2 GiB (larger than the 256 MB last-level cache), the best of the plain
    and the non-temporal read at two grid sizes each, and a register-only bf16 MFMA loop on
    every SIMD. Timed with HIP events on the stream the kernels are launched on."""
    import torch
    torch.cuda.init()
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_02897_amd", "libasv_microbench.so"))
    for f in (lib.asvb_stream_read, lib.asvb_stream_read_nt):
        f.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int32,
                      ctypes.c_void_p]
    lib.asvb_mfma_loop.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p]
    stream = torch.cuda.current_stream(dev)
    handle = stream.cuda_stream

    def timed(launch, reps):
        for _ in range(3):
            assert launch() == 0
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            assert launch() == 0
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    nbytes = 2 << 30
    buf = torch.full((nbytes // 4,), 0x01020304, dtype=torch.int32, device=dev)
    sink = torch.zeros(1 << 16, dtype=torch.int32, device=dev)
    best = 0.0
    for read, grid in ((lib.asvb_stream_read, 1024), (lib.asvb_stream_read, 2048),
                       (lib.asvb_stream_read_nt, 512), (lib.asvb_stream_read_nt, 1024)):
        sec = timed(lambda: read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, handle), 10)
        best = max(best, nbytes / sec / 1e9)
    del buf
    grid, iters = 256, 16384
    fsink = torch.zeros(grid * 256, dtype=torch.float32, device=dev)
    sec = timed(lambda: lib.asvb_mfma_loop(fsink.data_ptr(), iters, grid, handle), 5)
    tflops = grid * 4 * iters * 8 * 32768 / sec / 1e12
    return {"stream_read_gbps": round(best, 1), "mfma_bf16_tflops": round(tflops, 1)}


def lds_probe_patterns() -> list:
    """Lane patterns for the LDS read probe (asvb_lds_read): the 16-byte LDS unit each lane of a
    wave reads with one ds_read_b128. Bit-selection patterns put lane l on bank group
    (four lane bits of l) at a distinct address; the fragment patterns are the LM-head tiles'
    staged operand reads (128-byte rows, logical chunk c of row r at c ^ f(r)) for both MFMA
    shapes, with the current swizzle f(r) = (r >> 1) & 7 and the earlier
    f(r) = (r & 7) ^ ((r >> 3) & 1)."""
    import itertools
    pats = [("linear", list(range(64))), ("one_bank_group", [16 * l for l in range(64)])]
    for bits in itertools.combinations(range(6), 4):
        g = [sum(((l >> b) & 1) << i for i, b in enumerate(bits)) for l in range(64)]
        pats.append(("group_from_lane_bits_" + "".join(map(str, bits)),
                     [16 * l + g[l] for l in range(64)]))
    swz = {"current": lambda r: (r >> 1) & 7, "earlier": lambda r: (r & 7) ^ ((r >> 3) & 1)}
    for name, f in swz.items():
        for s in range(2):       # 16x16x32: lane l reads row l % 16, chunk 4 s + l / 16
            pats.append((f"mfma16x16x32_{name}_swizzle_step{s}",
                         [(l % 16) * 8 + ((4 * s + l // 16) ^ f(l % 16)) for l in range(64)]))
        for s in range(4):       # 32x32x16: lane l reads row l % 32, chunk 2 s + l / 32
            pats.append((f"mfma32x32x16_{name}_swizzle_step{s}",
                         [(l % 32) * 8 + ((2 * s + l // 32) ^ f(l % 32)) for l in range(64)]))
    assert all(len(u) == 64 and 0 <= min(u) and max(u) < 1024 for _, u in pats)
    return pats


def vendor_reference() -> dict:
    """Context for the roofline fractions: the vendor bf16 GEMM computing only the [N, V]
    logits of the four verify shapes (no reductions, gather or walk), and the copy bandwidth."""
    import torch
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    H = 4096
    out = {}

    def timed(fn, reps):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps

    for V, rows in ((128256, (60, 2048)), (151936, (378, 3048))):
        W = (torch.randn(V, H, device=dev, generator=g) * 0.02).to(torch.bfloat16)
        for N in rows:
            X = torch.randn(N, H, device=dev, generator=g).to(torch.bfloat16)
            sec = timed(lambda: torch.matmul(X, W.t()), 50 if N < 1000 else 20)
            out[f"hipblaslt_logits_n{N}_v{V}_us"] = round(sec * 1e6, 1)
            out[f"hipblaslt_logits_n{N}_v{V}_tflops"] = round(2 * N * V * H / sec / 1e12, 1)
        del W
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    sec = timed(lambda: dst.copy_(src), 20)
    out["d2d_copy_1gib_read_plus_write_gbps"] = round(2 * (1 << 30) / sec / 1e9, 1)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", type=int, default=1)
    ap.add_argument("--secondary", default="3")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-row-major", action="store_true",
                    help="skip the headline step on the row-major [V, H] weight (reported "
                         "under row_major beside the packed product path)")
    ap.add_argument("--no-draft", action="store_true",
                    help="skip the draft-step measurement (the step before verification)")
    ap.add_argument("--others", default="2,4",
                    help="further verify workloads reported under other_configs ('none' to "
                         "skip); configuration 4 is timed at each of its thresholds")
    ap.add_argument("--reference", action="store_true",
                    help="only time the vendor references on the bench shapes and exit: "
                         "torch.matmul (hipBLASLt) of the logits alone, and a 1 GiB "
                         "device-to-device copy")
    ap.add_argument("--w-layout", choices=("packed", "row-major"), default="packed",
                    help="layout of the target and draft LM-head weights in every workload: "
                         "packed once by asv_pack_lm_head / asv_pack_draft_head before timing "
                         "(default), or row-major [V, H]; both give bit-identical results")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (the "
                         "reference dispatch for scaling HBM traffic counters) and exit")
    ap.add_argument("--read-calibration", type=int, default=0, metavar="MIB",
                    help="only stream-read a buffer of MIB MiB five times back to back (the "
                         "microbenchmark read; a buffer smaller than the last-level cache is "
                         "read from it after the first pass) and exit: shows which traffic "
                         "counters see last-level-cache hits")
    ap.add_argument("--lds-probe", action="store_true",
                    help="only run the LDS read-pattern probe (one asvb_lds_read dispatch per "
                         "lane pattern, in the printed order, for SQ_LDS_BANK_CONFLICT counters) "
                         "and exit")
    args = ap.parse_args()
    if args.lds_probe:
        import torch
        mb = _microbench_lib()
        mb.asvb_lds_read.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_int32, ctypes.c_void_p]
        stream = torch.cuda.current_stream()
        handle = stream.cuda_stream
        grid, iters = 1024, 4096
        sink = torch.zeros(grid * 256, dtype=torch.int32, device="cuda:0")
        rows = []
        for name, units in lds_probe_patterns():
            u = torch.tensor(units, dtype=torch.int32, device="cuda:0")
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            assert mb.asvb_lds_read(u.data_ptr(), iters, sink.data_ptr(), grid, handle) == 0
            b.record(stream)
            b.synchronize()
            rows.append({"pattern": name, "us": round(a.elapsed_time(b) * 1e3, 1)})
        print(json.dumps({"lds_probe": rows, "grid": grid, "iters": iters,
                          "reads_per_dispatch": grid * 4 * iters}))
        return
    if args.read_calibration:
        import torch
        n = args.read_calibration << 20
        buf = torch.ones(n // 4, dtype=torch.int32, device="cuda:0")
        sink = torch.zeros(1 << 16, dtype=torch.int32, device="cuda:0")
        mb = _microbench_lib()
        handle = torch.cuda.current_stream().cuda_stream
        for _ in range(5):
            assert mb.asvb_stream_read(buf.data_ptr(), n, sink.data_ptr(), 1024, handle) == 0
        torch.cuda.synchronize()
        print(json.dumps({"read_calibration_bytes": n, "dispatches": 5}))
        return
    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "dispatches": 5}))
        return
    if args.reference:
        import torch
        ref = vendor_reference()
        ref.update(measured_ceilings(torch.device("cuda:0")))
        print(json.dumps(ref))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only: the verification path "
                          "runs on a single MI355X (multi-GPU sharding is design-only)"}))
        sys.exit(2)
    import torch
    import paper_2609_02897_amd as asv
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    asv.load()
    dev = torch.device("cuda:0")
    hip = HipEvents()
    # The achievable peaks are measured once the headline's inputs are resident, right before
    # its warm-up: seconds of streaming reads and MFMA loops, which also leave the GPU's memory
    # and shader clocks in the working state of a serving loop (the first ~100 steps after an
    # idle host phase read about 6% slower).
    ceilings = {}

    def take_ceilings():
        try:
            ceilings.update(measured_ceilings(dev))
            print(f"# measured ceilings: {ceilings}", file=sys.stderr, flush=True)
        except OSError as e:      # microbenchmark library not built: published peaks only
            print(f"# measured ceilings unavailable: {e}", file=sys.stderr, flush=True)

    r, w, W = measure(args.config, args.steps, args.warmup, dev, hip, layout=args.w_layout,
                      before_warmup=take_ceilings)
    ceilings = ceilings or None
    print(f"# cfg{r['cfg']} {r['name']}: {r['ms_per_step']*1e3:.1f} us/step, "
          f"K1 {r['k1_avg_ms']*1e3:.1f} us, {r['hbm_gbs']:.0f} GB/s, "
          f"{r['mfma_tflops']:.0f} TFLOP/s", file=sys.stderr, flush=True)
    line = {
        "metric": "verified tree nodes/sec (fused LM-head+margin accept); % HBM/MFMA roofline",
        "value": round(r["value"], 1), "unit": "nodes/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded bf16 W~N(0,0.02), hidden~N(0,1), EAGLE-style trees)",
        "config": {"workload": r["name"], "H": r["H"], "V": r["V"], "rows": r["N"],
                   "requests": r["B"], "tau": r["tau"], "w_layout": r["layout"],
                   "parallelism": "single GPU"},
        "roofline": None,
        "around_target_forward": r["around"],
    }
    if r["pack_ms"] is not None:
        line["w_pack_ms_once"] = round(r["pack_ms"], 3)
    if args.secondary != "none" and int(args.secondary) != args.config:
        del w, W
        r2, _, _ = measure(int(args.secondary), args.steps, args.warmup, dev, hip,
                           layout=args.w_layout)
        print(f"# cfg{r2['cfg']} {r2['name']}: {r2['ms_per_step']*1e3:.1f} us/step, "
              f"K1 {r2['k1_avg_ms']*1e3:.1f} us, {r2['mfma_tflops']:.0f} TFLOP/s",
              file=sys.stderr, flush=True)
        line["secondary"] = {"workload": r2["name"], "rows": r2["N"], "requests": r2["B"],
                             "value": round(r2["value"], 1), "unit": "nodes/s",
                             "ms_per_step": round(r2["ms_per_step"], 4),
                             "around_target_forward": r2["around"]}
        w, _ = load_workload(args.config)
        W = w.weights()
    line["roofline"] = roofline(r, ceilings)
    if "secondary" in line:
        line["secondary"]["roofline"] = roofline(r2, ceilings)
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(w, W)
    del w, W
    if args.w_layout == "packed" and not args.no_row_major:
        # the boundary's own input: the same headline step on the row-major [V, H] weight
        rr, _, _ = measure(args.config, args.steps, args.warmup, dev, hip, layout="row-major")
        print(f"# cfg{rr['cfg']} row-major weight: {rr['ms_per_step']*1e3:.1f} us/step, "
              f"K1 {rr['k1_avg_ms']*1e3:.1f} us", file=sys.stderr, flush=True)
        line["row_major"] = {"workload": rr["name"], "w_layout": "row-major",
                             "value": round(rr["value"], 1), "unit": "nodes/s",
                             "ms_per_step": round(rr["ms_per_step"], 4),
                             "roofline": roofline(rr, ceilings)}
    if args.others != "none":
        from workloads import CONFIGS
        line["other_configs"] = []
        for cfg in (int(x) for x in args.others.split(",")):
            for i, tau in enumerate(CONFIGS[cfg]["taus"] if cfg == 4 else (None,)):
                ro, wo, Wo = measure(cfg, args.steps, args.warmup, dev, hip, tau,
                                     layout=args.w_layout)
                print(f"# cfg{cfg} {ro['name']} tau={ro['tau']:.2f}: "
                      f"{ro['ms_per_step']*1e3:.1f} us/step, K1 {ro['k1_avg_ms']*1e3:.1f} us",
                      file=sys.stderr, flush=True)
                entry = {
                    "workload": ro["name"], "rows": ro["N"], "requests": ro["B"],
                    "tau": round(ro["tau"], 4), "value": round(ro["value"], 1),
                    "unit": "nodes/s", "ms_per_step": round(ro["ms_per_step"], 4),
                    "mean_accepted_len": round(ro["mean_accepted_len"], 3),
                    "roofline": roofline(ro, ceilings),
                    "roofline_other_bound": other_bound(ro)}
                if cfg == 4 and i == 0 and not args.no_cpu:
                    # the largest workload: the oracle on a bounded sample of its requests
                    entry["cpu_baseline"] = cpu_baseline(wo, Wo, budget_s=10.0, requests=8)
                del wo, Wo
                line["other_configs"].append(entry)
    if not args.no_draft:
        line["draft"] = [measure_draft(n, args.steps, args.warmup, dev, hip, not args.no_cpu,
                                       args.w_layout)
                         for n in ("llama31_8b_draft_b1", "llama31_8b_draft_b32")]
        for d in line["draft"]:
            print(f"# draft {d['workload']}: {d['us_per_step']} us/step, K5 cold "
                  f"{d['roofline']['k_avg_us_cold']} us, {d['roofline']['achieved']} GB/s",
                  file=sys.stderr, flush=True)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
