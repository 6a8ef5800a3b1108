"""Parity helpers shared by the GPU tests: tolerances and the step comparison.

Tolerances
  bf16 tensors (attention outputs, K/V): max-abs <= 2e-2 and relative L2 <= 1e-2.
  fp32 tensors: max-abs <= 1e-4 and relative L2 <= 1e-5 (float32 arithmetic
    against float64: a few hundred accumulated roundings of 6e-8 each).
  scores (always float32 on the GPU): |d| <= 1e-4 + 1e-3 * |I|.
  selection: equal counts per chunk; a row may differ only if the oracle's
    scores of every swapped pair differ by less than 1e-3 (sum units).
"""
import numpy as np

TOL = {"bf16": dict(max_abs=2e-2, rel_l2=1e-2), "f32": dict(max_abs=1e-4, rel_l2=1e-5)}
GAP = 1e-3


def rel_l2(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def assert_close(got, want, dtype, what):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.size == 0:
        return
    t = TOL[dtype]
    mx = float(np.max(np.abs(got - want)))
    rl = rel_l2(got, want)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert mx <= t["max_abs"] and rl <= t["rel_l2"], f"{what}: max-abs {mx:.3g}, rel-L2 {rl:.3g}"
    return mx, rl


def assert_ulp(got, want, dtype, what, rel_slack=2.0 ** -20, steps=1):
    """Each element within ``steps`` storage-dtype steps of the correctly rounded value
    (plus a float32 cancellation slack relative to the tensor's largest value)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.size == 0:
        return
    bits = 8 if dtype == "bf16" else 24
    step = np.ldexp(1.0, np.frexp(np.abs(want))[1] - bits)
    slack = rel_slack * float(np.max(np.abs(want)))
    bad = np.abs(got - want) > np.maximum(steps * step * 1.0001, slack)
    assert not bad.any(), f"{what}: {bad.sum()} elements more than {steps} step(s) off"


def assert_scores(got, want, what="scores"):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    bad = np.abs(got - want) > 1e-4 + 1e-3 * np.abs(want)
    assert not bad.any(), f"{what}: {bad.sum()} entries off, worst {np.max(np.abs(got - want)):.3g}"


def selection_segments(w, selection="chunk"):
    """(first row, length) of every selection segment: the chunks, or each request's context."""
    if selection == "global":
        return [(int(w.cu_kv[b]), int(w.ctx_len[b])) for b in range(w.batch) if w.ctx_len[b] > 0]
    return [(int(w.seg_start[s]), int(w.seg_len[s])) for s in range(w.n_chunks)]


def check_selection(w, P_gpu, scores_orc, P_orc, selection="chunk"):
    """Per selection segment: same count; swapped rows only across near-ties (gap < 1e-3)."""
    Pg = np.sort(np.concatenate(P_gpu)) if len(P_gpu) else np.zeros(0, int)
    Po = np.sort(np.concatenate(P_orc)) if len(P_orc) else np.zeros(0, int)
    swaps = 0
    for s, (a, n) in enumerate(selection_segments(w, selection)):
        g = Pg[(Pg >= a) & (Pg < a + n)]
        o = Po[(Po >= a) & (Po < a + n)]
        assert g.size == o.size, f"chunk {s}: {g.size} selected, oracle {o.size}"
        assert np.all(np.diff(g) > 0)
        xg = np.setdiff1d(g, o)
        xo = np.setdiff1d(o, g)
        if xg.size:
            gap = np.abs(scores_orc[xg][:, None] - scores_orc[xo][None, :]).max()
            assert gap < GAP, f"chunk {s}: swapped rows with score gap {gap:.3g}"
            swaps += xg.size
    return swaps


def tile_sample(w, g, seed=0, qv_per_tile=256):
    """Cache rows of R to compare on large configs: in every row tile of the GPU attention
    (per request, qv_per_tile / G consecutive rows of [P_b ; U_b]) one seeded row and the
    tile's last valid row, plus each request's first row."""
    G = w.n_q_heads // w.n_kv_heads
    rpt = max(1, qv_per_tile // G)
    rng = np.random.default_rng(seed)
    pick = []
    for b in range(w.batch):
        a, e = int(g["cu_R"][b]), int(g["cu_R"][b + 1])
        if e == a:
            continue
        pick.append(a)
        for t0 in range(a, e, rpt):
            t1 = min(e, t0 + rpt)
            pick += [int(rng.integers(t0, t1)), t1 - 1]
    return np.unique(np.asarray(g["R"])[np.unique(pick)])


def oracle_for(w, g, rho_bp=None, selection="chunk", sampled=False, seed=0):
    """The oracle's step on the GPU's selection P (teacher forcing; check_step first checks
    P against the oracle's own selection), on every row of R or on a tile sample."""
    import oracle
    rows = tile_sample(w, g, seed) if sampled else None
    return oracle.fusion_step(w, rho_bp=rho_bp, attn_rows=rows, selection=selection, P=g["P"])


def check_step(w, g, o, selection="chunk"):
    """Compare a GPU step (``FusionStep.results()``) with the oracle's ``fusion_step`` run on
    the GPU's selection (``oracle_for``).

    The GPU's P must pass the selection check against the oracle's own selection
    (``P_select``) and scores; everything downstream is then compared with what the
    definitions give for the GPU's P."""
    dt = w.dtype
    report = {}
    # scores of the context rows
    ctx = np.zeros(w.n_rows, bool)
    for s in range(w.n_chunks):
        ctx[w.seg_start[s]:w.seg_start[s] + w.seg_len[s]] = True
    assert_scores(g["scores"][ctx], o["scores"][ctx])
    # selection against the oracle's own, then the oracle must have run on the GPU's P
    report["swaps"] = check_selection(w, g["P"], o["scores"], o["P_select"], selection)
    for b in range(w.batch):
        np.testing.assert_array_equal(o["P"][b], g["P"][b])
        # R layout: per request, P ascending then the query rows
        Rg = g["R"][g["cu_R"][b]:g["cu_R"][b + 1]]
        np.testing.assert_array_equal(Rg, o["R"][b])
    # fused cache: fresh K/V on R, the re-positioned PIC entry elsewhere
    report["k"] = assert_close(g["k_fuse"], o["k_fuse"], dt, "fused K")
    assert_ulp(g["k_fuse"], o["k_fuse"], dt, "fused K")
    np.testing.assert_array_equal(g["v_fuse"], o["v_fuse"])
    # probe outputs
    report["o_probe"] = assert_close(np.concatenate(g["o_probe_list"]), np.concatenate(o["o_probe"]), dt,
                                     "probe output")
    # attention outputs on every row the oracle evaluated (all of R, or a tile sample)
    rows = [i for i, r in enumerate(g["R"]) if int(r) in o["o"]]
    assert len(rows) == len(o["o"]), "oracle rows missing from the GPU's R"
    assert rows, "no attention rows to compare"
    got = g["o"][rows]
    want = np.stack([o["o"][int(g["R"][i])] for i in rows])
    report["o"] = assert_close(got, want, dt, "attention output")
    report["o_rows"] = len(rows)
    return report
