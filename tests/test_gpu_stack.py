"""The multi-layer stack (c3): libqcf's per-layer path against the float64 oracle.

The stack's glue (RMSNorm, projections, residual) is torch on the GPU side and
float64 in the oracle; every hot-path step runs in libqcf.  The float32 case
is compared element by element; the bf16 cases check what holds at any size
(score mass, selection counts, untouched cache rows, determinism) and, for
the reduced shape, the oracle's selection and states within bf16 tolerances.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import stack as S
from paper_2606_05875_amd import qcf
from paper_2606_05875_amd.stack import FusionStack
from paper_2606_05875_amd.workloads import make_stack_workload

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def cut_margin(scores, sw, rho_bp):
    """Smallest relative gap between the k-th and (k+1)-th score of any chunk."""
    m = np.inf
    for s in range(sw.n_chunks):
        a, n = int(sw.seg_start[s]), int(sw.seg_len[s])
        k = (rho_bp * n) // 10000
        if 0 < k < n:
            srt = np.sort(scores[a:a + n])[::-1]
            m = min(m, (srt[k - 1] - srt[k]) / max(abs(srt[k - 1]), 1e-30))
    return m


@pytest.mark.parametrize("layout", [dict(), dict(chunk_lens=[[40, 24, 17], [33]], q_lens=[6, 5])])
def test_stack_f32_matches_oracle(layout):
    sw = make_stack_workload("c3_small", **layout)
    say("stack f32", sw.chunk_lens, sw.q_lens)
    want = S.stack_fusion(sw)
    assert cut_margin(want["scores"], sw, sw.rho_bp) > 1e-4
    st = FusionStack(sw)
    st.run()
    got = st.results()
    np.testing.assert_allclose(got["scores"], want["scores"], rtol=1e-4, atol=1e-6)
    for b in range(sw.batch):
        np.testing.assert_array_equal(got["P"][b], want["P"][b])
        np.testing.assert_allclose(got["h_probe"][b], want["h_probe"][b], rtol=2e-4, atol=2e-4)
        np.testing.assert_allclose(got["h_R"][b], want["h_R"][b], rtol=2e-4, atol=2e-4)
    # the fused cache of every layer (context rows, query rows) against the oracle's
    rows = np.concatenate([np.arange(sw.cu_kv[b], sw.cu_kv[b + 1]) for b in range(sw.batch)])
    for l in range(sw.n_layers):
        np.testing.assert_allclose(got["k_fuse"][l][rows], want["k_fuse"][l][rows], rtol=2e-4, atol=2e-4)
        np.testing.assert_allclose(got["v_fuse"][l][rows], want["v_fuse"][l][rows], rtol=2e-4, atol=2e-4)


def bf16_properties(sw, st, got):
    """What holds at any size: score mass, counts, untouched rows, determinism."""
    for b in range(sw.batch):
        a, N = int(sw.cu_kv[b]), int(sw.ctx_len[b])
        tot = got["scores"][a:a + N].sum()
        want = len(sw.critical_layers) * sw.n_q_heads * sw.q_lens[b]
        assert abs(tot - want) < 2e-3 * want, (tot, want)
        segs = np.nonzero(sw.seg_req == b)[0]
        assert got["P"][b].size == sum((sw.rho_bp * int(sw.seg_len[s])) // 10000 for s in segs)
        assert np.all(np.diff(got["P"][b]) > 0)
    # context rows outside R hold the re-positioned PIC entry of their layer, bit for bit
    R = np.zeros(sw.n_rows, bool)
    R[got["R"]] = True
    keep = np.zeros(sw.n_rows, bool)
    for s in range(sw.n_chunks):
        keep[sw.seg_start[s]:sw.seg_start[s] + sw.seg_len[s]] = True
    keep &= ~R
    kt = torch.from_numpy(keep).cuda()
    for l in (0, max(sw.critical_layers), sw.n_layers - 1):
        kr = torch.empty_like(st.k_pic[l])
        vr = torch.empty_like(st.v_pic[l])
        qcf.qcf_rerope(kr, st.k_pic[l], st.seg_start, st.seg_len, st.seg_delta, st.plan.max_seg,
                       sw.rope_theta, v_out=vr, v_in=st.v_pic[l])
        assert torch.equal(st.k_req[l][kt], kr[kt]) and torch.equal(st.v_req[l][kt], vr[kt])
    for h in got["h_R"]:
        assert np.all(np.isfinite(h))
    # a second run gives the same bits
    st.run()
    again = st.results()
    np.testing.assert_array_equal(again["scores"], got["scores"])
    np.testing.assert_array_equal(again["R"], got["R"])
    for x, y in zip(again["h_R"], got["h_R"]):
        np.testing.assert_array_equal(x, y)


def test_stack_bf16_small_against_oracle():
    sw = make_stack_workload("c3_small", dtype="bf16", chunk_lens=[[96, 64, 80, 33], [70]], q_lens=[12, 9])
    say("stack bf16 small", sw.chunk_lens, sw.q_lens)
    want = S.stack_fusion(sw)
    st = FusionStack(sw)
    st.run()
    got = st.results()
    bf16_properties(sw, st, got)
    # scores within bf16 error of the oracle; selections agree except inside the
    # band where bf16 rounding can swap neighbours
    np.testing.assert_allclose(got["scores"], want["scores"], rtol=3e-2, atol=3e-3)
    for b in range(sw.batch):
        inter = np.intersect1d(got["P"][b], want["P"][b]).size
        assert inter >= 0.9 * want["P"][b].size, (inter, want["P"][b].size)
        if np.array_equal(got["P"][b], want["P"][b]):
            np.testing.assert_allclose(got["h_R"][b], want["h_R"][b], rtol=0.1, atol=0.1)


def test_stack_c3_full_size_properties():
    # the 36-layer, 20x512-chunk, 4096-wide stack at its real size (no oracle
    # run: properties that hold at any size)
    sw = make_stack_workload("c3")
    say("stack c3 full", sw.n_layers, sw.n_rows, sw.d_model)
    st = FusionStack(sw)
    st.run()
    got = st.results()
    bf16_properties(sw, st, got)


def test_stack_full_view_selector_matches_oracle():
    # the full-view reference selector: every context token an anchor, every layer scores
    from paper_2606_05875_amd.workloads import full_view
    sw = full_view(make_stack_workload("c3_small", chunk_lens=[[40, 24, 17], [33]], q_lens=[6, 5]))
    say("stack full view f32", sw.chunk_lens, sw.critical_layers)
    want = S.stack_fusion(sw)
    assert cut_margin(want["scores"], sw, sw.rho_bp) > 1e-4
    st = FusionStack(sw)
    st.run()
    got = st.results()
    np.testing.assert_allclose(got["scores"], want["scores"], rtol=1e-4, atol=1e-6)
    for b in range(sw.batch):
        np.testing.assert_array_equal(got["P"][b], want["P"][b])
        np.testing.assert_allclose(got["h_probe"][b], want["h_probe"][b], rtol=2e-4, atol=2e-4)
        np.testing.assert_allclose(got["h_R"][b], want["h_R"][b], rtol=2e-4, atol=2e-4)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stack_host_pipeline_is_bit_identical(dtype):
    # PIC caches streamed layer by layer from pinned host memory through two
    # staging slots give exactly the device-resident run's results
    from paper_2606_05875_amd.stack import HostPicPipeline
    sw = make_stack_workload("c3_small", dtype=dtype, chunk_lens=[[40, 24, 17], [33]], q_lens=[6, 5])
    say("stack host pipeline", dtype)
    st = FusionStack(sw)
    st.run()
    want = st.results()
    pipe = HostPicPipeline(st)
    pipe.free_device_pic()
    st.scores.zero_()
    st.run(pipe.begin())
    got = st.results()
    np.testing.assert_array_equal(got["scores"], want["scores"])
    np.testing.assert_array_equal(got["R"], want["R"])
    for x, y in zip(got["h_R"], want["h_R"]):
        np.testing.assert_array_equal(x, y)
    for x, y in zip(got["h_probe"], want["h_probe"]):
        np.testing.assert_array_equal(x, y)
    for l in range(sw.n_layers):
        np.testing.assert_array_equal(got["k_fuse"][l], want["k_fuse"][l])
    # and again, reusing the pipeline
    st.run(pipe.begin())
    again = st.results()
    for x, y in zip(again["h_R"], want["h_R"]):
        np.testing.assert_array_equal(x, y)


def test_knorm_anchors_match_oracle():
    from paper_2606_05875_amd.anchors import anchors_knorm
    sw = make_stack_workload("c3_small", chunk_lens=[[40, 24, 17], [33]], q_lens=[6, 5])
    say("knorm anchors", sw.chunk_lens)
    K, V = S.build_pic(sw)
    want = S.anchors_knorm(K, sw.seg_start, sw.seg_len, 1500)
    st = FusionStack(sw)
    st.build_pic()
    got = anchors_knorm(st.k_pic, sw.seg_start, sw.seg_len, 1500)
    for g, w_ in zip(got, want):
        np.testing.assert_array_equal(g, w_)
    # the shared-input view with those anchors runs and matches the oracle's selection
    import dataclasses
    sv = dataclasses.replace(sw, anchor_local=[np.asarray(a, np.int32) for a in want])
    st2 = FusionStack(sv, share=st)
    st2.run()
    ref = S.stack_fusion(sv, pic=(K, V))
    got2 = st2.results()
    for b in range(sw.batch):
        np.testing.assert_array_equal(got2["P"][b], ref["P"][b])
