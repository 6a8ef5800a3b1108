"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value comes from
a closed form, an independent formulation (complex rotation, a pure-Python
sort), a library routine the oracle does not use (torch SDPA / softmax in
float64), an invariant, or a special case the paper names (recomputation
ratio 0 = direct PIC reuse, ratio 1 = full prefill; Experiments, Metrics).
A few tests plant a mistake in a copy of an oracle function and check that
the pin catches it.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from hypothesis import given, settings, strategies as st

import oracle
from oracle import qcfuse as Q
from paper_2606_05875_amd.workloads import make_workload, round_to_bf16

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


# ---------------------------------------------------------------- helpers
def rope_complex(x, pos, theta):
    """Independent rotary formulation: z_j = x_j + i x_{j+d/2}, z_j * exp(i pos omega_j)."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    omega = np.array([theta ** (-(2.0 * j) / d) for j in range(h)])
    z = x[..., :h] + 1j * x[..., h:]
    ang = np.asarray(pos, np.float64)[..., None, None] * omega
    z = z * np.exp(1j * ang)
    return np.concatenate([z.real, z.imag], axis=-1)


def sdpa(q, k, v, mask=None, causal=False):
    """torch SDPA in float64 on the CPU; q [R,Hq,d], k/v [n,Hkv,d] -> [R,Hq,d]."""
    qt = torch.from_numpy(np.asarray(q, np.float64)).permute(1, 0, 2)[None]
    kt = torch.from_numpy(np.asarray(k, np.float64)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.asarray(v, np.float64)).permute(1, 0, 2)[None]
    m = None if mask is None else torch.from_numpy(mask)
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, is_causal=causal, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        [0.0, -0.0, 1.0, -2.5, 3.0e38, 1e-40, -1e-42]]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(Q.round_bf16(x.astype(np.float64)), want)


def test_bf16_ties_and_double_rounding():
    # ties go to the even 8-bit significand
    assert Q.round_bf16(1 + 2 ** -8) == 1.0
    assert Q.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6
    assert Q.round_bf16(1.5 * 2 ** -133) == 2 ** -132
    # a float64 value just above a tie rounds up (float32 first would lose it)
    assert Q.round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7


def test_generator_bf16_round_matches_torch():
    x = np.random.default_rng(1).standard_normal(5000).astype(np.float32)
    np.testing.assert_array_equal(round_to_bf16(x),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


# ---------------------------------------------------------------- rotary embedding
def test_rope_closed_form_d4():
    # d = 4, theta = 100: omega = (1, 0.1); position 1 turns pair 0 by 1 rad, pair 1 by 0.1 rad
    e0 = Q.rope(np.array([[[1.0, 0, 0, 0]]]), np.array([1]), 100.0)[0, 0]
    e1 = Q.rope(np.array([[[0, 1.0, 0, 0]]]), np.array([1]), 100.0)[0, 0]
    e2 = Q.rope(np.array([[[0, 0, 1.0, 0]]]), np.array([1]), 100.0)[0, 0]
    np.testing.assert_allclose(e0, [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    np.testing.assert_allclose(e1, [0, math.cos(0.1), 0, math.sin(0.1)], atol=1e-15)
    np.testing.assert_allclose(e2, [-math.sin(1), 0, math.cos(1), 0], atol=1e-15)


@pytest.mark.parametrize("d,theta", [(64, 1e4), (128, 5e5), (128, 1e6)])
def test_rope_matches_complex_rotation(d, theta):
    rng = np.random.default_rng(d)
    x = rng.standard_normal((50, 3, d))
    pos = rng.integers(0, 40000, 50)
    np.testing.assert_allclose(Q.rope(x, pos, theta), rope_complex(x, pos, theta), atol=1e-12)


def test_rope_group_properties():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((20, 2, 128))
    r = rng.integers(0, 1024, 20)
    o = rng.integers(0, 32000, 20)
    np.testing.assert_allclose(Q.rope(Q.rope(x, r, 5e5), o, 5e5), Q.rope(x, r + o, 5e5), atol=1e-11)
    np.testing.assert_allclose(np.linalg.norm(Q.rope(x, o, 5e5), axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_array_equal(Q.rope(x, np.zeros(20, int), 5e5), x)
    # logits depend only on relative position
    q, k = rng.standard_normal((1, 1, 128)), rng.standard_normal((1, 1, 128))
    a = np.sum(Q.rope(q, [700], 5e5) * Q.rope(k, [123], 5e5))
    b = np.sum(Q.rope(q, [700 + 9999], 5e5) * Q.rope(k, [123 + 9999], 5e5))
    assert abs(a - b) < 1e-10


def test_rope_pin_catches_planted_sign_error():
    def bad_rope(x, pos, theta):
        x = np.asarray(x, np.float64)
        h = x.shape[-1] // 2
        a = Q.rope_angles(pos, x.shape[-1], theta)[..., None, :]
        c, s = np.cos(a), np.sin(a)
        x1, x2 = x[..., :h], x[..., h:]
        return np.concatenate([x1 * c + x2 * s, x1 * s + x2 * c], axis=-1)   # wrong sign
    x = np.random.default_rng(3).standard_normal((5, 1, 64))
    pos = np.arange(5) * 7
    assert not np.allclose(bad_rope(x, pos, 1e4), rope_complex(x, pos, 1e4), atol=1e-6)


def test_rerope_is_rotation_to_request_position():
    # a stored key is its raw vector rotated at the chunk-local position r;
    # after re-positioning by offset o it equals the raw vector rotated at o + r
    rng = np.random.default_rng(4)
    raw = rng.standard_normal((300, 2, 64))
    seg_start, seg_len, seg_delta = np.array([0, 100, 180]), np.array([100, 80, 120]), np.array([0, 100, 180])
    local = np.concatenate([np.arange(n) for n in seg_len])
    stored = rope_complex(raw, local, 1e4)
    out = Q.rerope(stored, seg_start, seg_len, seg_delta, 1e4, "f32")
    want = rope_complex(raw, np.arange(300), 1e4).astype(np.float32)
    np.testing.assert_allclose(out, want, atol=2e-6)
    # offset 0 leaves the chunk untouched
    out0 = Q.rerope(stored, seg_start[:1], seg_len[:1], np.array([0]), 1e4, "f32")
    np.testing.assert_array_equal(out0[:100], stored[:100].astype(np.float32))


# ---------------------------------------------------------------- attention
@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 64), (4, 4, 32), (16, 2, 128)])
def test_attention_causal_matches_sdpa(hq, hkv, d):
    rng = np.random.default_rng(hq * d)
    n = 97
    q, k, v = rng.standard_normal((n, hq, d)), rng.standard_normal((n, hkv, d)), rng.standard_normal((n, hkv, d))
    pos = np.arange(n)
    got = Q.attention(q, pos, k, v, pos, 1 / math.sqrt(d), hkv)
    np.testing.assert_allclose(got, sdpa(q, k, v, causal=True), atol=1e-12)


def test_attention_explicit_positions_matches_masked_sdpa():
    rng = np.random.default_rng(5)
    hq, hkv, d = 8, 2, 64
    kpos = np.sort(rng.choice(500, 60, replace=False))
    qpos = rng.integers(0, 520, 25)
    q, k, v = rng.standard_normal((25, hq, d)), rng.standard_normal((60, hkv, d)), rng.standard_normal((60, hkv, d))
    qpos[0] = kpos[0]                           # sees exactly one key
    got = Q.attention(q, qpos, k, v, kpos, 0.125, hkv)
    mask = kpos[None, :] <= qpos[:, None]
    vis = mask.any(1)
    np.testing.assert_allclose(got[vis], sdpa(q[vis], k, v, mask=mask[vis]), atol=1e-12)
    np.testing.assert_allclose(got[0], np.repeat(v[0], hq // hkv, axis=0), atol=1e-14)   # one key -> its value
    assert np.all(got[~vis] == 0)


def test_attention_identical_keys_average_values():
    rng = np.random.default_rng(6)
    k = np.repeat(rng.standard_normal((1, 1, 16)), 10, axis=0)
    v = rng.standard_normal((10, 1, 16))
    q = rng.standard_normal((10, 2, 16))
    got = Q.attention(q, np.arange(10), k, v, np.arange(10), 0.25, 1)
    for r in range(10):
        np.testing.assert_allclose(got[r, 0], v[:r + 1, 0].mean(0), atol=1e-14)


def test_attention_pin_catches_dropped_scale():
    rng = np.random.default_rng(7)
    q, k, v = rng.standard_normal((9, 2, 16)), rng.standard_normal((9, 1, 16)), rng.standard_normal((9, 1, 16))
    wrong = Q.attention(q, np.arange(9), k, v, np.arange(9), 1.0, 1)
    assert not np.allclose(wrong, sdpa(q, k, v, causal=True), atol=1e-6)


# ---------------------------------------------------------------- scores
def test_scores_sum_and_torch_softmax():
    rng = np.random.default_rng(8)
    nq, hq, hkv, d, N = 7, 8, 2, 32, 123
    q, k = rng.standard_normal((nq, hq, d)) * 3, rng.standard_normal((N, hkv, d))
    got = Q.critical_scores(q, k, 1 / math.sqrt(d), hkv)
    assert abs(got.sum() - nq * hq) < 1e-10                       # each (h, i) distributes mass 1
    qt = torch.from_numpy(q).permute(1, 0, 2)                      # [hq, nq, d]
    kt = torch.from_numpy(k).permute(1, 2, 0).repeat_interleave(hq // hkv, 0)   # [hq, d, N]
    want = torch.softmax(qt @ kt / math.sqrt(d), dim=-1).sum(dim=(0, 1)).numpy()
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_scores_special_cases():
    rng = np.random.default_rng(9)
    q = rng.standard_normal((5, 4, 16))
    same = np.repeat(rng.standard_normal((1, 2, 16)), 40, axis=0)
    np.testing.assert_allclose(Q.critical_scores(q, same, 0.25, 2), np.full(40, 5 * 4 / 40), atol=1e-13)
    np.testing.assert_allclose(Q.critical_scores(q, same[:1], 0.25, 2), [20.0], atol=1e-13)
    # one key aligned with every query direction, others orthogonal -> it takes (almost) all mass
    k = np.zeros((30, 2, 16)); k[:, :, 1] = 1.0; k[17, :, 0] = 1.0
    qq = np.zeros((5, 4, 16)); qq[..., 0] = 1000.0
    got = Q.critical_scores(qq, k, 1.0, 2)
    assert abs(got[17] - 20.0) < 1e-9 and got.sum() == pytest.approx(20.0)


def test_scores_pin_catches_wrong_softmax_axis():
    rng = np.random.default_rng(10)
    q, k = rng.standard_normal((6, 4, 16)), rng.standard_normal((50, 2, 16))
    logits = np.einsum("ihd,thd->hit", q, np.repeat(k, 2, axis=1)) * 0.25
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)                   # softmax over query tokens: a planted mistake
    wrong = p.sum(axis=(0, 1))
    assert abs(wrong.sum() - 6 * 4) > 1.0          # the mass invariant of the real pin fails


# ---------------------------------------------------------------- selection
def brute_topk(s, k):
    return sorted(sorted(range(len(s)), key=lambda t: (-(s[t] + 0.0), t))[:k])


@settings(max_examples=300, deadline=None)
@given(st.lists(st.sampled_from([0.0, -0.0, 0.25, 0.5, 1.0, 3.0, 1e-30, 7.5]) | st.floats(0, 10, allow_nan=False),
                min_size=0, max_size=80), st.integers(0, 10000))
def test_topk_matches_brute_force(vals, rho_bp):
    s = np.array(vals, np.float64)
    k = Q.per_chunk_k(s.size, rho_bp)
    assert list(Q.select_topk(s, k)) == brute_topk(list(s), k)


def test_per_chunk_counts_and_endpoints():
    assert Q.per_chunk_k(512, 3000) == 153 and Q.per_chunk_k(1024, 3000) == 307
    assert Q.per_chunk_k(128, 3000) == 38 and Q.per_chunk_k(777, 2000) == 155
    s = np.random.default_rng(11).random(300)
    starts, lens = np.array([0, 100, 250]), np.array([100, 150, 50])
    assert Q.select_per_chunk(s, starts, lens, 0).size == 0
    np.testing.assert_array_equal(Q.select_per_chunk(s, starts, lens, 10000), np.arange(300))
    got = Q.select_per_chunk(s, starts, lens, 3000)
    assert got.size == 30 + 45 + 15 and np.all(np.diff(got) > 0)
    # one segment covering everything is the global top-k of eq. critical_mask
    np.testing.assert_array_equal(Q.select_per_chunk(s, [0], [300], 2500), brute_topk(list(s), 75))


def test_global_selection_mode():
    """selection="global" takes floor(rho N_b) rows over each request's whole context (eq.
    critical_mask as written): a brute-force stable sort of the request's scores; with one
    chunk per request it is the per-chunk selection."""
    w = make_workload("c2", chunk_lens=[[100, 37, 60], [80]], q_lens=[5, 3], anchors_per_chunk=3,
                      dtype="f32")
    o = Q.fusion_step(w, rho_bp=2500, selection="global")
    c = Q.fusion_step(w, rho_bp=2500)
    for b in range(w.batch):
        base, N = int(w.cu_kv[b]), int(w.ctx_len[b])
        sc = list(o["scores"][base:base + N])
        want = np.array(brute_topk(sc, (2500 * N) // 10000)) + base
        np.testing.assert_array_equal(o["P"][b], want)
    assert o["P"][0].size == (2500 * 197) // 10000 == 49              # 25 + 9 + 15 = 49 per chunk too
    np.testing.assert_array_equal(o["P"][1], c["P"][1])                # a one-chunk request
    np.testing.assert_array_equal(o["scores"], c["scores"])            # selection does not touch scores


# ---------------------------------------------------------------- the fusion step
def _full_prefill(w):
    """Dense causal attention of every row over fresh rotated K/V (independent formulation)."""
    outs = {}
    d = w.head_dim
    for b in range(w.batch):
        base, T = int(w.cu_kv[b]), int(w.cu_kv[b + 1] - w.cu_kv[b])
        pos = np.arange(T)
        rd = (lambda x: np.asarray(x, np.float32).astype(np.float64)) if w.dtype == "f32" else Q.round_bf16
        q = rd(rope_complex(w.q_new[base:base + T], pos, w.rope_theta))
        k = rd(rope_complex(w.k_new[base:base + T], pos, w.rope_theta))
        v = np.asarray(w.v_new[base:base + T], np.float64)
        outs[b] = sdpa(q, k, v, causal=True)
    return outs


def test_ratio_one_is_full_prefill():
    w = make_workload("c1")
    r = Q.fusion_step(w, rho_bp=10000)
    full = _full_prefill(w)[0]
    R = r["R"][0]
    assert R.size == w.n_rows                       # every context row plus the query
    got = np.stack([r["o"][int(t)] for t in R])
    np.testing.assert_allclose(got, full.astype(np.float32), atol=2e-6)


def test_ratio_zero_is_direct_reuse():
    w = make_workload("c1")
    r = Q.fusion_step(w, rho_bp=0)
    N = int(w.ctx_len[0])
    assert r["P"][0].size == 0
    np.testing.assert_array_equal(r["k_fuse"][:N], r["k_rerope"][:N])
    np.testing.assert_array_equal(r["v_fuse"][:N], w.v_pic[:N])
    # the query rows attend over the re-positioned PIC cache plus their own fresh K/V
    T = w.n_rows
    pos = np.arange(N, T)
    q = rope_complex(w.q_new[N:], pos, w.rope_theta).astype(np.float32)
    kq = rope_complex(w.k_new[N:], pos, w.rope_theta).astype(np.float32)
    k = np.concatenate([r["k_rerope"][:N], kq])
    v = np.concatenate([w.v_pic[:N], w.v_new[N:]])
    mask = np.arange(T)[None, :] <= pos[:, None]
    want = sdpa(q, k, v, mask=mask)
    got = np.stack([r["o"][int(t)] for t in range(N, T)])
    np.testing.assert_allclose(got, want, atol=2e-6)


def test_fused_cache_rows():
    w = make_workload("c1")
    r = Q.fusion_step(w)
    R = set(int(t) for t in r["R"][0])
    N = int(w.ctx_len[0])
    keep = np.array([t for t in range(N) if t not in R])
    np.testing.assert_array_equal(r["k_fuse"][keep], r["k_rerope"][keep])
    np.testing.assert_array_equal(r["v_fuse"][keep], w.v_pic[keep])
    for t in R:
        np.testing.assert_allclose(r["k_fuse"][t], rope_complex(w.k_new[t:t + 1], [t], w.rope_theta)[0].astype(np.float32), atol=1e-6)
        np.testing.assert_array_equal(r["v_fuse"][t], w.v_new[t])


def _near_tie_swap(w, r):
    """P with one selected row of the chunk with the smallest cut gap exchanged for the
    best unselected row of that chunk (a near-tied alternative selection)."""
    best = None
    for s in range(w.n_chunks):
        a, n = int(w.seg_start[s]), int(w.seg_len[s])
        sel = [int(t) for t in r["P"][0] if a <= t < a + n]
        rest = [t for t in range(a, a + n) if t not in sel]
        if not sel or not rest:
            continue
        x = min(sel, key=lambda t: (r["scores"][t], -t))          # the last one taken
        y = max(rest, key=lambda t: (r["scores"][t], -t))         # the first one left out
        gap = r["scores"][x] - r["scores"][y]
        if best is None or gap < best[0]:
            best = (gap, x, y)
    _, x, y = best
    return np.sort(np.array([t for t in r["P"][0] if t != x] + [y], np.int64)), x, y


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_given_selection_is_the_definition_on_that_selection(dtype):
    # an alternative selection (one near-tied row swapped) handed to the oracle: the fused
    # cache and every recomputed row's output must be what the definitions give for that
    # selection, built here by hand (complex rotation, torch SDPA in float64)
    w = make_workload("c1", dtype=dtype)
    own = Q.fusion_step(w)
    P, x, y = _near_tie_swap(w, own)
    r = Q.fusion_step(w, P=[P])
    np.testing.assert_array_equal(r["P_select"][0], own["P"][0])     # its own selection is kept
    np.testing.assert_array_equal(r["P"][0], P)
    N, T = int(w.ctx_len[0]), w.n_rows
    rd = (lambda a: np.asarray(a, np.float32).astype(np.float64)) if dtype == "f32" else Q.round_bf16
    pos = np.arange(T)
    local = np.concatenate([np.arange(n) for n in w.seg_len] + [np.zeros(T - N, int)])
    delta = np.concatenate([np.full(n, o) for n, o in zip(w.seg_len, w.seg_delta)] + [np.zeros(T - N, int)])
    # stored keys are rotated at their local positions: one more rotation by the offset
    k_pic = rd(rope_complex(w.k_pic, delta, w.rope_theta))
    k_pic[N:] = 0.0
    R = np.concatenate([P, np.arange(N, T)])
    fused_k = k_pic.copy()
    fused_v = np.array(w.v_pic, np.float64)
    fused_k[R] = rd(rope_complex(w.k_new[R], R, w.rope_theta))
    fused_v[R] = w.v_new[R]
    np.testing.assert_allclose(r["k_fuse"], fused_k, atol=2e-6 if dtype == "f32" else 1e-2)
    np.testing.assert_array_equal(r["v_fuse"], fused_v)
    assert not np.array_equal(r["k_fuse"][x], own["k_fuse"][x])     # x went back to its PIC entry
    q = rd(rope_complex(w.q_new[R], R, w.rope_theta))
    want = sdpa(q, fused_k, fused_v, mask=pos[None, :] <= R[:, None])
    got = np.stack([r["o"][int(t)] for t in R])
    tol = 2e-6 if dtype == "f32" else 1.6e-2
    np.testing.assert_allclose(got, want, atol=tol)
    # rows after y see y's fresh key: their outputs differ from those on the own selection
    later = [t for t in R if t > y and t in own["o"]]
    assert any(not np.array_equal(r["o"][t], own["o"][t]) for t in later)


def test_attention_rows_subset_equals_full_run():
    # evaluating only some rows gives those rows' outputs of the full evaluation, bit for bit
    w = make_workload("c1")
    full = Q.fusion_step(w)
    R = full["R"][0]
    some = R[::7]
    part = Q.fusion_step(w, attn_rows=some)
    assert sorted(part["o"]) == sorted(int(t) for t in some)
    for t in some:
        np.testing.assert_array_equal(part["o"][int(t)], full["o"][int(t)])


def test_anchor_probe_endpoints():
    # all positions as anchors: the probe is the query's attention over the full
    # re-positioned context (the full-view probe); no anchors: query-only probing
    base = make_workload("c1")
    N, T = int(base.ctx_len[0]), base.n_rows
    for anchors in (128, 0):
        w = make_workload("c1", anchors_per_chunk=anchors)
        r = Q.fusion_step(w)
        pos = np.arange(N, T)
        q = rope_complex(w.q_new[N:], pos, w.rope_theta).astype(np.float32)
        kq = rope_complex(w.k_new[N:], pos, w.rope_theta).astype(np.float32)
        if anchors:
            k = np.concatenate([r["k_rerope"][:N], kq]); v = np.concatenate([w.v_pic[:N], w.v_new[N:]])
            kp = np.arange(T)
        else:
            k, v, kp = kq, w.v_new[N:], pos
        want = sdpa(q, k, v, mask=kp[None, :] <= pos[:, None])
        np.testing.assert_allclose(r["o_probe"][0], want, atol=2e-6)


def test_scores_step_invariant_and_recall():
    for name in ("c1", "c2"):
        w = make_workload(name)
        r = Q.fusion_step(w, attn_rows=np.arange(int(w.ctx_len[0]), w.n_rows))
        assert abs(r["scores"].sum() - w.n_q_heads * sum(w.q_lens)) < 1e-6 * w.n_rows
        assert Q.recall(np.concatenate(r["P"]), w.evidence_rows) == 1.0


def test_generator_is_deterministic_and_exact():
    a, b = make_workload("c2"), make_workload("c2")
    for f in ("k_pic", "v_pic", "q_new", "k_new", "v_new"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
        x = getattr(a, f)
        np.testing.assert_array_equal(round_to_bf16(x), x)
    c5 = make_workload("c5")
    assert c5.batch == 16 and 8 * 16 <= c5.n_chunks <= 16 * 16
    assert np.all((c5.seg_len >= 256) & (c5.seg_len <= 1024))
    assert all(16 <= n <= 128 for n in c5.q_lens)


# ---------------------------------------------------------------- the multi-layer stack (c3)
from oracle import stack as S  # noqa: E402
from paper_2606_05875_amd.workloads import make_stack_workload  # noqa: E402


def torch_forward(sw, rows, n_layers=None):
    """Independent causal forward of rows (positions 0..n-1): torch float64, SDPA with
    repeated KV heads, complex rotary.  Returns per-layer rotated q and k, v, final h."""
    d, hq, hkv = sw.head_dim, sw.n_q_heads, sw.n_kv_heads
    n = len(rows)
    pos = np.arange(n)
    h = torch.tensor(np.asarray(sw.embed[rows], np.float64))
    qs, ks, vs = [], [], []
    for l in range(sw.n_layers if n_layers is None else n_layers):
        x = h / torch.sqrt((h * h).mean(-1, keepdim=True) + sw.rms_eps)
        t = lambda w: x @ torch.tensor(np.asarray(w[l], np.float64))
        q = torch.tensor(rope_complex(t(sw.wq).view(n, hq, d).numpy(), pos, sw.rope_theta))
        k = torch.tensor(rope_complex(t(sw.wk).view(n, hkv, d).numpy(), pos, sw.rope_theta))
        v = t(sw.wv).view(n, hkv, d)
        qs.append(q.numpy())
        ks.append(k.numpy())
        vs.append(v.numpy())
        kk = k.repeat_interleave(hq // hkv, dim=1).transpose(0, 1)
        vv = v.repeat_interleave(hq // hkv, dim=1).transpose(0, 1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), kk, vv, is_causal=True)
        h = h + o.transpose(0, 1).reshape(n, hq * d) @ torch.tensor(np.asarray(sw.wo[l], np.float64))
    return qs, ks, vs, h.numpy()


def small_stack(**kw):
    base = dict(overrides=dict(n_layers=4, critical_layers=(1, 2)))
    base.update(kw)
    return make_stack_workload("c3_small", **base)


def test_stack_ratio_one_is_full_forward():
    # every context row recomputed: each request's rows must come out of the
    # stack exactly as a plain causal forward of the request (paper: ratio 1 = full prefill)
    sw = small_stack(chunk_lens=[[40, 24], [33]], q_lens=[6, 5])
    res = S.stack_fusion(sw, rho_bp=10000)
    for b in range(sw.batch):
        rows = np.arange(sw.cu_kv[b], sw.cu_kv[b + 1])
        assert np.array_equal(res["R"][b], rows)
        _, ks, vs, h = torch_forward(sw, rows)
        np.testing.assert_allclose(res["h_R"][b], h, rtol=2e-5, atol=2e-5)
        for l in range(sw.n_layers):
            np.testing.assert_allclose(res["k_fuse"][l][rows], ks[l], rtol=2e-5, atol=2e-5)
            np.testing.assert_allclose(res["v_fuse"][l][rows], vs[l], rtol=2e-5, atol=2e-5)


def test_stack_ratio_zero_single_chunk_is_exact_reuse():
    # one chunk stored alone at positions 0..n-1 is exactly the prefix of the
    # request, so reusing it (ratio 0) gives the query rows the full forward's states
    sw = small_stack(chunk_lens=[[57]], q_lens=[7])
    res = S.stack_fusion(sw, rho_bp=0)
    rows = np.arange(sw.cu_kv[0], sw.cu_kv[1])
    assert res["P"][0].size == 0
    _, _, _, h = torch_forward(sw, rows)
    np.testing.assert_allclose(res["h_R"][0], h[57:], rtol=2e-5, atol=2e-5)


def test_stack_probe_with_every_token_as_anchor():
    # with every context token an anchor of a single chunk, the query probe is
    # the full forward of the request's query rows up to the last critical
    # layer, and the scores are the full-view softmax masses at the critical layers
    sw = small_stack(chunk_lens=[[45]], q_lens=[6], anchors_per_chunk=45)
    assert sw.anchor_local[0].size == 45
    res = S.stack_fusion(sw)
    rows = np.arange(sw.cu_kv[0], sw.cu_kv[1])
    lmax = max(sw.critical_layers)
    qs, ks, _, h = torch_forward(sw, rows, n_layers=lmax + 1)
    np.testing.assert_allclose(res["h_probe"][0], h[45:], rtol=2e-5, atol=2e-5)
    want = np.zeros(45)
    for l in sw.critical_layers:
        g = sw.n_q_heads // sw.n_kv_heads
        for hh in range(sw.n_q_heads):
            lg = torch.tensor(qs[l][45:, hh] @ ks[l][:45, hh // g].T) / math.sqrt(sw.head_dim)
            want += torch.softmax(lg, dim=1).sum(0).numpy()
    np.testing.assert_allclose(res["scores"][:45], want, rtol=1e-4, atol=1e-6)


def test_stack_scores_sum_to_softmax_count():
    # each (layer, head, query row) softmax over the context sums to 1
    sw = small_stack(chunk_lens=[[40, 24], [33]], q_lens=[6, 5])
    res = S.stack_fusion(sw)
    for b in range(sw.batch):
        a, N = int(sw.cu_kv[b]), int(sw.ctx_len[b])
        tot = res["scores"][a:a + N].sum()
        assert abs(tot - len(sw.critical_layers) * sw.n_q_heads * sw.q_lens[b]) < 1e-9 * tot
        counts = [(3000 * n) // 10000 for n in sw.chunk_lens[b]]
        assert res["P"][b].size == sum(counts)


def test_stack_pin_catches_probe_position_error():
    # a planted mistake (query rows rotated at 0..n_q-1 instead of N..N+n_q-1 in
    # the probe) must fail the all-anchors pin
    sw = small_stack(chunk_lens=[[45]], q_lens=[6], anchors_per_chunk=45)
    orig = S.block_qkv

    def bad(sw_, l, h, pos):
        if len(pos) == 6 and pos[0] == 45:
            pos = pos - 45
        return orig(sw_, l, h, pos)

    S.block_qkv = bad
    try:
        res = S.stack_fusion(sw)
    finally:
        S.block_qkv = orig
    rows = np.arange(sw.cu_kv[0], sw.cu_kv[1])
    _, _, _, h = torch_forward(sw, rows, n_layers=max(sw.critical_layers) + 1)
    assert not np.allclose(res["h_probe"][0], h[45:], rtol=2e-5, atol=2e-5)


def test_anchor_rules():
    # eq. anchor_set: ceil(r_a n) positions per chunk; Sink = the first ones; Knorm = the
    # smallest mean key norms, checked against a plain sort of hand-made norms
    assert [S.anchor_count(n, 1000) for n in (1, 9, 10, 11, 512)] == [1, 1, 1, 2, 52]
    assert all(S.anchor_count(n, ra) == math.ceil(ra * n / 10000) for n in range(1, 70) for ra in (1, 333, 5000))
    sk = S.anchors_sink([10, 3], 2500)
    assert [list(x) for x in sk] == [[0, 1, 2], [0]]
    rng = np.random.default_rng(5)
    L, T, H, d = 3, 14, 2, 4
    K = [rng.standard_normal((T, H, d)) for _ in range(L)]
    K[1][3] *= 0.01          # a near-zero key -> chosen first
    got = S.anchors_knorm(K, [0, 9], [9, 5], 3000)
    mean_norm = [np.mean([np.sqrt((K[l][t] ** 2).sum(-1)).mean() for l in range(L)]) for t in range(T)]
    want0 = sorted(sorted(range(9), key=lambda t: (mean_norm[t], t))[:3])
    want1 = sorted(sorted(range(5), key=lambda t: (mean_norm[9 + t], t))[:2])
    assert list(got[0]) == want0 and 3 in want0
    assert list(got[1]) == want1
