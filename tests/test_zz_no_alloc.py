"""qcf_probe_scores_select_noalloc (the selector call on the library's fixed device scratch
array) against qcf_probe_scores_select with a caller workspace: the same scores and the same
recomputation rows bit for bit, on two calls in a row, the second on a smaller input (the
scratch then holds the first call's values), also when the scores accumulate over a
second critical layer."""
import sys

import numpy as np
import pytest
import torch

from paper_2606_05875_amd import qcf
from paper_2606_05875_amd.step import FusionStep
from paper_2606_05875_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _select(step, noalloc, accumulate):
    """One selector call on the step's inputs into fresh outputs; returns (scores, R, R_pos)."""
    p = step.plan
    scores = step.scores.clone()
    R = step.R_idx_init.clone()
    R_pos = step.R_pos_init.clone()
    args = (scores, step.q_u, step.k, step.cu_q, step.cu_kv, step.ctx_len, p.max_q, p.max_ctx,
            step.scale, R, step.sel_start, step.sel_len, step.seg_k, step.out_start, step.sel_req,
            p.max_sel)
    if noalloc:
        qcf.qcf_probe_scores_select_noalloc(*args, out_pos=R_pos, accumulate=accumulate)
    else:
        ws = torch.empty(max(qcf.qcf_probe_scores_workspace_size(step.w.batch, p.max_q, p.max_ctx,
                                                                  step.w.n_q_heads, step.w.n_kv_heads,
                                                                  step.w.head_dim), 1),
                         dtype=torch.uint8, device=scores.device)
        qcf.qcf_probe_scores_select(*args, out_pos=R_pos, accumulate=accumulate, workspace=ws)
    torch.cuda.synchronize()
    return scores.cpu().numpy(), R.cpu().numpy(), R_pos.cpu().numpy()


@pytest.mark.parametrize("accumulate", [False, True])
def test_noalloc_selector_matches_workspace_call(accumulate):
    # a large call (c4: 32 768-token context, 64/8 heads) and then a smaller ragged batch
    for name, kw in (("c4", {}),
                     ("c2", dict(chunk_lens=[[300, 212], [64], [129, 1, 511, 40]], q_lens=[5, 64, 17],
                                 anchors_per_chunk=3))):
        w = make_workload(name, **kw)
        say(name, "rows", w.n_rows, "requests", w.batch, "accumulate", accumulate)
        step = FusionStep(w)
        step.run()              # fills the probe queries and the re-positioned keys
        torch.cuda.synchronize()
        want = _select(step, noalloc=False, accumulate=accumulate)
        got = _select(step, noalloc=True, accumulate=accumulate)
        for x, y, what in zip(got, want, ("scores", "R", "R_pos")):
            np.testing.assert_array_equal(x, y, err_msg=f"{name} {what}")
        assert np.all(got[1] >= 0)
