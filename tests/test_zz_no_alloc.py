"""asv_verify_noalloc (the workspace taken from the library's static device scratch) against
asv_verify with a caller-allocated workspace, through the C ABI: two calls in a row on one GPU,
the second with a smaller batch, so the second runs on what the first left in the scratch.
Every output and the policy state must be bit for bit those of asv_verify; the oracle checks
the noalloc outputs as well."""

import numpy as np
import pytest

import oracle
from harness import compare, device_inputs, reference, resolve_with_oracle, to_host
from workloads import build_tree, custom_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def asv():
    import paper_2609_02897_amd as m
    m.load()
    return m


def _workload(kind, n_req, H, V, seed):
    rng = np.random.default_rng(seed)
    trees = [build_tree(kind, rng, b) for b in range(n_req)]
    return custom_workload(f"noalloc_{kind}", H, V, trees, 0.2, seed=seed, w_std=0.09,
                           draft_logits=True)


def test_noalloc_matches_verify_two_calls(asv, dev):
    import torch
    cases = [_workload("adaptive", 9, 192, 2500, 3),      # 9 requests, several row tiles
             _workload("eagle60", 1, 128, 1300, 4)]       # then a smaller batch
    for i, w in enumerate(cases):
        print(f"noalloc call {i}: B={w.B} N={w.N} H={w.H} V={w.V}", flush=True)
        W = w.weights()
        w64 = oracle.widen_weights(W)
        resolve_with_oracle(w, w64)
        d = device_inputs(w, W, dev)
        st_a = asv.state_init(w.B, asv.make_params(), device=dev)
        st_b = st_a.clone()
        args = (d["hidden"], d["w_lm"], d["draft_tok"], d["parent"], d["req_offsets"],
                d["tau"], d["draft_logits"])
        out_a = asv.alloc_outputs(w.B, w.N, dev, True)
        asv.verify(*args, state=st_a, out=out_a, noalloc=True)
        out_b = asv.verify(*args, state=st_b)
        torch.cuda.synchronize()
        got = to_host(out_a)
        base = to_host(out_b)
        nonroot = w.parent >= 0                 # drafted_logit is unspecified at roots
        for k, v in base.items():
            sel = nonroot if k == "drafted_logit" else slice(None)
            assert np.array_equal(got[k][sel], v[sel], equal_nan=True), (i, k)
        assert torch.equal(st_a, st_b), i
        compare(w, reference(w, w64), got)


def test_noalloc_rejects_over_the_scratch(asv, dev):
    """Sizes whose workspace exceeds the static scratch are refused before any launch."""
    import torch
    B, N, H, V = 1, 8192, 64, 151936
    assert asv.workspace_bytes(B, N, H, V) > asv.STATIC_SCRATCH_BYTES
    e = dict(hidden=torch.zeros((N, H), dtype=torch.bfloat16, device=dev),
             w_lm=torch.zeros((V, H), dtype=torch.bfloat16, device=dev),
             draft_tok=torch.zeros(N, dtype=torch.int32, device=dev),
             parent=torch.arange(-1, N - 1, dtype=torch.int32, device=dev),
             req_offsets=torch.tensor([0, N], dtype=torch.int32, device=dev),
             tau=torch.full((1,), 0.3, dtype=torch.float32, device=dev))
    with pytest.raises(asv.AsvError) as err:
        asv.verify(**e, noalloc=True)
    assert err.value.code == asv.ASV_ESCRATCH
