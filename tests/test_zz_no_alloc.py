"""smallkv_step_noalloc, the whole step for callers that cannot allocate
(it runs on the library's static per-GPU scratch instead of a caller
workspace), against smallkv_step with a caller workspace: two calls in a row
on one GPU, the second over a smaller input, every output bit-identical to
the workspace call's (the same kernels run on the same inputs)."""
import dataclasses

import pytest
import torch

from paper_2508_02751_amd import smallkv as S
from paper_2508_02751_amd import workloads as W
from paper_2508_02751_amd.pipeline import prepare_step

pytestmark = pytest.mark.gpu
DEV = "cuda"


def results(ps):
    """Every output of the step, logits restricted to the tokens written."""
    b = ps.buf
    n = ps.batch.seq_len.to(torch.int64).cpu()
    out = {"logits": [b.logits[i, :, : int(n[i])].clone() for i in range(n.numel())]}
    for f in dataclasses.fields(b):
        t = getattr(b, f.name)
        if f.name not in ("ws", "logits", "acc_score") and t is not None:
            out[f.name] = t.clone()
    return out


def same(a, b, what):
    for k in a:
        xs, ys = (a[k], b[k]) if k == "logits" else ([a[k]], [b[k]])
        for x, y in zip(xs, ys):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"{what}: {k} differs"


def noalloc_vs_workspace(w):
    x = W.make_step_inputs(w, DEV)
    print(f"[no-alloc] {w.name}", flush=True)
    ref = prepare_step(x)
    ref.run()                                   # smallkv_step, caller workspace
    torch.cuda.synchronize()
    want = results(ref)
    got = prepare_step(x)                       # fresh intermediates and outputs
    S.smallkv_step_noalloc(got.desc)            # no workspace argument
    torch.cuda.synchronize()
    same(want, results(got), w.name)
    return want, got


def test_noalloc_step_matches_the_workspace_step_twice_second_smaller():
    big, small = W.WORKLOADS[2], W.WORKLOADS[1]     # N = 8192 bf16, then N = 512 fp32
    assert small.n_cap * small.batch < big.n_cap * big.batch
    noalloc_vs_workspace(big)
    noalloc_vs_workspace(small)


def test_noalloc_step_repeats_and_keeps_no_stale_state():
    """A bigger call between two identical small calls leaves the scratch
    holding its own records; the second small call is unchanged by them."""
    w = dataclasses.replace(W.WORKLOADS[2], wid=111, n_ctx=3000, ragged_min=700, batch=3)
    first, ps = noalloc_vs_workspace(w)
    noalloc_vs_workspace(W.WORKLOADS[2])
    S.smallkv_step_noalloc(ps.desc)
    torch.cuda.synchronize()
    same(first, results(ps), "repeat after a larger call")
