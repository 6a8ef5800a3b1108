"""Host-side layout of the fusion step (runs without a GPU): selection budgets, the slots of
the recomputed rows and the probe buffer, per chunk and in global mode."""
import numpy as np
import pytest

from paper_2606_05875_amd.step import FusionPlan
from paper_2606_05875_amd.workloads import make_workload


def _layouts():
    return [make_workload("c2", chunk_lens=[[300, 212], [64], [129, 1, 511, 40]], q_lens=[5, 64, 17],
                          anchors_per_chunk=3, dtype="f32"),
            make_workload("c2", chunk_lens=[[100, 37, 1, 333]], q_lens=[1], anchors_per_chunk=4,
                          dtype="f32")]


@pytest.mark.parametrize("selection", ["chunk", "global"])
@pytest.mark.parametrize("rho_bp", [0, 2500, 3000, 10000])
def test_plan_layout(selection, rho_bp):
    for w in _layouts():
        p = FusionPlan.build(w, rho_bp, selection)
        if selection == "chunk":
            segs = [(int(w.seg_start[s]), int(w.seg_len[s]), int(w.seg_req[s])) for s in range(w.n_chunks)]
        else:
            segs = [(int(w.cu_kv[b]), int(w.ctx_len[b]), b) for b in range(w.batch) if w.ctx_len[b] > 0]
        assert len(p.seg_k) == len(segs) == len(p.sel_start) == len(p.out_start) == len(p.pos_base)
        for i, (a, n, b) in enumerate(segs):
            assert (p.sel_start[i], p.sel_len[i]) == (a, n)
            assert p.seg_k[i] == (rho_bp * n) // 10000                    # floor(rho n), integer arithmetic
            assert p.pos_base[i] == w.cu_kv[b]
        # per request: [P_b ; U_b] slots, P slots filled by the selection in segment order
        for b in range(w.batch):
            mine = [i for i, s in enumerate(segs) if s[2] == b]
            assert p.n_P[b] == sum(int(p.seg_k[i]) for i in mine)
            assert p.cu_R[b + 1] - p.cu_R[b] == p.n_P[b] + w.q_lens[b]
            at = int(p.cu_R[b])
            for i in mine:
                assert p.out_start[i] == at
                at += int(p.seg_k[i])
            qs = slice(int(p.cu_R[b] + p.n_P[b]), int(p.cu_R[b + 1]))
            N = int(w.ctx_len[b])
            np.testing.assert_array_equal(p.R_pos_init[qs], np.arange(N, N + w.q_lens[b]))
            np.testing.assert_array_equal(p.R_idx_init[qs], w.cu_kv[b] + np.arange(N, N + w.q_lens[b]))
            assert np.all(p.R_idx_init[int(p.cu_R[b]):qs.start] == -1)
        assert p.max_sel == max((n for _, n, _ in segs), default=0)


def test_global_and_chunk_budgets_differ_by_less_than_the_chunk_count():
    """sum_i floor(rho n_i) <= floor(rho N) < sum_i floor(rho n_i) + (number of chunks)."""
    for w in _layouts():
        c = FusionPlan.build(w, 3000, "chunk")
        g = FusionPlan.build(w, 3000, "global")
        for b in range(w.batch):
            chunks = int(np.sum(w.seg_req == b))
            assert c.n_P[b] <= g.n_P[b] < c.n_P[b] + max(chunks, 1)


def test_unknown_selection_mode():
    with pytest.raises(ValueError):
        FusionPlan.build(_layouts()[0], 3000, "per-token")
