"""Write the oracle tables of the full-size synthetic configurations (run on the CPU).

For every configuration 1-4 (and every decode step of configuration 2) this computes, with
the float64 oracle only, each row's target top-8 (to turn the seeded draft choices into
drafted token ids), max, argmax, log-sum-exp and top-2 gap, and each node's drafted logit.
The GPU tests compare against these values, recompute a sample of rows live, and the bench
reads the drafted tokens. Input fingerprints guard against generator drift.

    python tests/golden/make_oracle_tables.py [cfg ...]
"""

from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from workloads import CONFIGS, make_workload, resolve_drafts  # noqa: E402


def table_path(cfg: int) -> str:
    return os.path.join(HERE, f"oracle_cfg{cfg}.npz")


def sha(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def one_step(w, w64, row_chunk=256):
    N = w.N
    x64 = oracle.widen_bf16(w.hidden)
    M, L, gap = np.empty(N), np.empty(N), np.empty(N)
    a = np.empty(N, dtype=np.int64)
    top8 = np.empty((N, 8), dtype=np.int32)
    g = np.full(N, np.nan)
    tok = np.full(N, -1, dtype=np.int32)
    for r0 in range(0, N, row_chunk):
        z = oracle.logits(x64[r0:r0 + row_chunk], w64)
        n = len(z)
        M[r0:r0 + n], a[r0:r0 + n], L[r0:r0 + n], gap[r0:r0 + n] = oracle.row_stats(z)
        top8[r0:r0 + n] = oracle.row_top8(z)
        # children whose parent row is in this slice: resolve the drafted token, read g
        kids = np.nonzero((w.parent >= r0) & (w.parent < r0 + n))[0]
        tok[kids] = resolve_drafts(w.kind[kids], w.rank[kids], w.uid[kids],
                                   w.parent[kids] - r0, top8[r0:r0 + n])
        g[kids] = z[w.parent[kids] - r0, tok[kids]]
    return dict(draft_tok=tok, row_max=M, row_lse=L, row_argmax=a.astype(np.int32),
                row_gap=gap, drafted_logit=g,
                sha_hidden=sha(w.hidden), sha_parent=sha(w.parent),
                sha_offsets=sha(w.req_offsets),
                sha_choice=sha(np.concatenate([w.kind.astype(np.int32), w.rank, w.uid])))


def make(cfg: int):
    c = CONFIGS[cfg]
    t0 = time.time()
    w0 = make_workload(cfg, 0)
    W = w0.weights()
    w64 = oracle.widen_weights(W)
    out = {"sha_w": sha(W), "steps": np.int32(c["steps"])}
    for step in range(c["steps"]):
        w = w0 if step == 0 else make_workload(cfg, step)
        res = one_step(w, w64)
        for k, v in res.items():
            out[f"{k}_s{step}"] = v
        print(f"cfg{cfg} step {step}: N={w.N} ({time.time() - t0:.1f}s)", flush=True)
    np.savez_compressed(table_path(cfg), **out)
    print(f"wrote {table_path(cfg)}", flush=True)


if __name__ == "__main__":
    cfgs = [int(x) for x in sys.argv[1:]] or [1, 3, 4, 2]
    for cfg in cfgs:
        make(cfg)
