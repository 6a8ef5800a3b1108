"""Teacher-forced per-layer parity of the multi-layer stack against the oracle.

At every traced layer the oracle takes that layer's GPU inputs -- the hidden
states entering the layer and the per-chunk caches the GPU built offline --
and applies the layer's definitions.  Each stage is compared on its own, so a
difference in one stage is not carried into the next:

  projections (oracle.stack.block_proj on the GPU's hidden states): q, k, v
      within 2 storage steps taken at max(|x|, the token row's RMS), relative
      L2 <= 1e-2;
  rotation (oracle.qcfuse.rope of the GPU's own stored projections): q and k
      within one storage step;
  cache rows outside R: the oracle's re-positioning of the GPU's stored chunk
      keys within one storage step, values bit for bit (eq. pic_online);
  fused cache rows R: the GPU's fresh K/V (eq. fuse_cache), checked above;
  attention (oracle.qcfuse.attention on the GPU's rotated q and fused cache):
      2e-2 max-abs (two storage steps where |o| >= 4, since one step there is
      already 0.031) and 1e-2 relative L2 per sampled row (Section 2.1.3);
  residual (oracle.stack.residual on the GPU's hidden states and attention
      output): one storage step at max(|x|, row RMS), relative L2 <= 1e-2.

The selector: at every critical layer the oracle scores the context keys it
re-positioned from the GPU's stored caches with the GPU's rotated probe
queries (eq. single_layer_importance), sums over the critical layers (eq.
critical_layer_importance) and selects per chunk (eq. critical_mask); the
GPU's scores must match per element and its selection must pass the
near-tie rule.  The probe layers are checked like the recompute layers
(block, probe attention over [anchors ; query rows], residual).

Why steps and not 2e-2 for K and hidden states: the projected keys and hidden
states of the stack reach |x| ~ 4-8, where one bfloat16 step is 0.03-0.06; a
float32-accumulated product can land on the other side of a rounding
boundary than the float64 one, so one step is the closest bound a bfloat16
result can meet.  Where |x| < 4 one step is below 2e-2.
"""
import numpy as np

from oracle import qcfuse as Q
from oracle import stack as S
from parity import assert_scores, check_selection, rel_l2


def f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _row_rms(want):
    """Per-token RMS of a [rows, ...] tensor, broadcast back to its shape."""
    w = want.reshape(want.shape[0], -1)
    r = np.sqrt(np.mean(w * w, axis=1))
    return r.reshape((-1,) + (1,) * (want.ndim - 1))


def steps_close(got, want, dtype, what, steps, report, floor=None):
    """Each element within ``steps`` bfloat16 steps taken at max(|want|, floor)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.size:
        mag = np.abs(want) if floor is None else np.maximum(np.abs(want), floor)
        step = np.ldexp(1.0, np.frexp(mag)[1] - 8)
        slack = 2.0 ** -20 * float(np.max(np.abs(want)))
        lim = np.maximum(steps * step * 1.0001, slack)
        bad = np.abs(got - want) > lim
        if bad.any():
            i = np.unravel_index(np.argmax(np.abs(got - want) / lim), got.shape)
            raise AssertionError(f"{what}: {bad.sum()} elements more than {steps} step(s) off; worst at {i}: "
                                 f"got {got[i]!r} want {want[i]!r} magnitude {mag[i]!r}")
    rl = rel_l2(got, want)
    assert rl <= 1e-2, f"{what}: rel-L2 {rl:.3g}"
    report[what] = (float(np.max(np.abs(got - want))) if got.size else 0.0, rl)


def projected_close(got, want, dtype, what, report):
    """A projection output (x W, stored in bfloat16): 2 steps at max(|want|, the token row's
    RMS).  The two sides differ in the float sum and occasionally by one step in the normed
    input; an element that cancels to a small value keeps an error at the scale of its
    terms, which the row's RMS measures."""
    steps_close(got, want, dtype, what, 2, report, floor=_row_rms(np.asarray(want, np.float64)))


def attention_close(got, want, what, report):
    """Attention outputs (bfloat16): 2e-2 max-abs, except that where |want| >= 4 one bfloat16
    step is itself 2^-5 = 0.031 and the bound is two steps of |want|; relative L2 <= 1e-2."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    step = np.ldexp(1.0, np.frexp(np.abs(want))[1] - 8)
    lim = np.maximum(2e-2, 2.0 * step * 1.0001)
    err = np.abs(got - want)
    if (err > lim).any():
        i = np.unravel_index(np.argmax(err / lim), got.shape)
        raise AssertionError(f"{what}: {(err > lim).sum()} elements off; worst at {i}: got {got[i]!r} "
                             f"want {want[i]!r}")
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    rl = rel_l2(got, want)
    assert rl <= 1e-2, f"{what}: rel-L2 {rl:.3g}"
    report[what] = (float(err.max()) if err.size else 0.0, rl)


def rope_close(got, raw, pos, theta, what, report):
    """The GPU's rotation of its own projection: one storage step of the oracle's rotation of
    the same stored values (plus a float32 slack for near-cancelling pairs)."""
    want = Q.round_storage(Q.rope(raw, pos, theta), "bf16")
    steps_close(got, want, "bf16", what, 1, report)


def sample_R(sw, res, rows_per_tile, seed):
    """Indices into R: per request its first slot, and per row tile of the GPU attention a
    seeded slot and the tile's last slot."""
    rng = np.random.default_rng(seed)
    pick = []
    for b in range(sw.batch):
        a, e = int(res["cu_R"][b]), int(res["cu_R"][b + 1])
        if e == a:
            continue
        pick.append(a)
        for t0 in range(a, e, rows_per_tile):
            t1 = min(e, t0 + rows_per_tile)
            pick += [int(rng.integers(t0, t1)), t1 - 1]
    return np.unique(pick)


def check_stack(sw, st, res, layers, seed=0, pic_layers=(), pic_chunks=()):
    """Compare the traced layers of a FusionStack run (``st.trace`` covering the critical
    layers, ``layers`` and ``pic_layers``) with the oracle, teacher forced.  ``res`` is
    ``st.results()``.  Returns a report of (max-abs, rel-L2) per compared tensor."""
    dt = sw.dtype
    assert dt == "bf16", "storage-step bounds are for bfloat16 results"
    d, hq, hkv = sw.head_dim, sw.n_q_heads, sw.n_kv_heads
    scale = 1.0 / np.sqrt(d)
    theta = sw.rope_theta
    p = st.plan
    rep = {}
    T = sw.n_rows
    ctx = np.zeros(T, bool)
    for s in range(sw.n_chunks):
        ctx[sw.seg_start[s]:sw.seg_start[s] + sw.seg_len[s]] = True
    krep_cache = {}

    def krep(l):
        if l not in krep_cache:
            krep_cache[l] = Q.rerope(f64(st.k_pic[l]), sw.seg_start, sw.seg_len, sw.seg_delta, theta, dt)
        return krep_cache[l]

    # ---- selector: scores from the GPU's probe queries at every critical layer
    scores = np.zeros(T)
    for l in sw.critical_layers:
        qu = f64(st.tr_sel[l]["q"])
        K = krep(l)
        for b in range(sw.batch):
            base, N = int(sw.cu_kv[b]), int(sw.ctx_len[b])
            scores[base:base + N] += Q.critical_scores(qu[sw.cu_q[b]:sw.cu_q[b + 1]], K[base:base + N],
                                                       scale, hkv)
    assert_scores(res["scores"][ctx], scores[ctx], "stack scores")
    P_orc = [Q.select_per_chunk(scores, sw.seg_start[sw.seg_req == b], sw.seg_len[sw.seg_req == b],
                                st.rho_bp) for b in range(sw.batch)]
    rep["swaps"] = check_selection(sw, res["P"], scores, P_orc)

    # ---- probe layers
    upos = p.u_pos.astype(np.int64)
    for l in sorted(set(st.tr_sel)):
        tr = st.tr_sel[l]
        h = f64(tr["h"])
        qo, ko, vo = S.block_proj(sw, l, h)
        qraw, kraw = f64(tr["q_raw"]), f64(tr["k_raw"])
        qg, kp, vp, og = f64(tr["q"]), f64(tr["k_probe"]), f64(tr["v_probe"]), f64(tr["o"])
        qs = p.query_slot.astype(np.int64)
        projected_close(qraw, qo, dt, f"probe q projection L{l}", rep)
        projected_close(kraw, ko, dt, f"probe k projection L{l}", rep)
        projected_close(vp[qs], vo, dt, f"probe query v L{l}", rep)
        rope_close(qg, qraw, upos, theta, f"probe q rotation L{l}", rep)
        rope_close(kp[qs], kraw, upos, theta, f"probe k rotation L{l}", rep)
        an = np.nonzero(p.probe_src >= 0)[0]
        src = p.probe_src[an].astype(np.int64)
        steps_close(kp[an], krep(l)[src], dt, f"probe anchor k L{l}", 1, rep)
        np.testing.assert_array_equal(vp[an], f64(st.v_pic[l])[src])
        want = np.zeros_like(og)
        for b in range(sw.batch):
            a0, a1 = int(p.cu_probe[b]), int(p.cu_probe[b + 1])
            u0, u1 = int(sw.cu_q[b]), int(sw.cu_q[b + 1])
            want[u0:u1] = Q.round_storage(Q.attention(qg[u0:u1], upos[u0:u1], kp[a0:a1], vp[a0:a1],
                                                      p.probe_pos[a0:a1], scale, hkv), dt)
        attention_close(og, want, f"probe attention L{l}", rep)
        hw = S.residual(sw, l, h, og)
        steps_close(f64(tr["h_out"]), hw, dt, f"probe residual L{l}", 1, rep, floor=_row_rms(hw))

    # ---- recompute layers
    R = np.asarray(res["R"], np.int64)
    Rpos = f64(st.R_pos).astype(np.int64)
    inR = np.zeros(T, bool)
    inR[R] = True
    G = hq // hkv
    sample = sample_R(sw, res, max(1, 256 // G), seed)
    for l in layers:
        tr = st.tr_rec[l]
        h = f64(tr["h"])
        qo, ko, vo = S.block_proj(sw, l, h)
        qraw, kraw = f64(tr["q_raw"]), f64(tr["k_raw"])
        qg, og = f64(tr["q"]), f64(tr["o"])
        kg, vg = f64(st.k_req[l]), f64(st.v_req[l])
        projected_close(qraw, qo, dt, f"q projection L{l}", rep)
        projected_close(kraw, ko, dt, f"k projection L{l}", rep)
        projected_close(vg[R], vo, dt, f"fused V rows R L{l}", rep)
        rope_close(qg, qraw, Rpos, theta, f"q rotation L{l}", rep)
        rope_close(kg[R], kraw, Rpos, theta, f"fused K rows R (rotation) L{l}", rep)
        keep = ctx & ~inR
        steps_close(kg[keep], krep(l)[keep], dt, f"fused K other rows L{l}", 1, rep)
        np.testing.assert_array_equal(vg[keep], f64(st.v_pic[l])[keep])
        got, want = [], []
        for b in range(sw.batch):
            base, n_b = int(sw.cu_kv[b]), int(sw.cu_kv[b + 1] - sw.cu_kv[b])
            idx = sample[(sample >= res["cu_R"][b]) & (sample < res["cu_R"][b + 1])]
            if idx.size == 0:
                continue
            o = Q.attention(qg[idx], Rpos[idx], kg[base:base + n_b], vg[base:base + n_b], np.arange(n_b),
                            scale, hkv)
            got.append(og[idx])
            want.append(Q.round_storage(o, dt))
        attention_close(np.concatenate(got), np.concatenate(want), f"attention L{l}", rep)
        hw = S.residual(sw, l, h, og)
        steps_close(f64(tr["h_out"]), hw, dt, f"residual L{l}", 1, rep, floor=_row_rms(hw))

    # ---- offline chunk pass (the stored caches themselves) on some chunks
    for l in pic_layers:
        tr = st.tr_pic[l]
        rows_all = np.concatenate([np.arange(a, a + n) for a, n in zip(sw.seg_start, sw.seg_len)])
        local_all = np.concatenate([np.arange(n) for n in sw.seg_len])
        h_all, q_all, o_all, ho_all = f64(tr["h"]), f64(tr["q"]), f64(tr["o"]), f64(tr["h_out"])
        kpic, vpic = f64(st.k_pic[l]), f64(st.v_pic[l])
        for s in pic_chunks:
            a, n = int(sw.seg_start[s]), int(sw.seg_len[s])
            sel = np.nonzero((rows_all >= a) & (rows_all < a + n))[0]
            pos = local_all[sel]
            qo, ko, vo = S.block_proj(sw, l, h_all[sel])
            qraw, kraw = f64(tr["q_raw"])[sel], f64(tr["k_raw"])[sel]
            projected_close(qraw, qo, dt, f"chunk {s} q projection L{l}", rep)
            projected_close(kraw, ko, dt, f"chunk {s} k projection L{l}", rep)
            projected_close(vpic[a:a + n], vo, dt, f"chunk {s} stored V L{l}", rep)
            rope_close(q_all[sel], qraw, pos, theta, f"chunk {s} q rotation L{l}", rep)
            rope_close(kpic[a:a + n], kraw, pos, theta, f"chunk {s} stored K (rotation) L{l}", rep)
            pick = np.unique(np.concatenate([[0, n - 1], np.random.default_rng(seed + s).integers(0, n, 32)]))
            o = Q.attention(q_all[sel][pick], pos[pick], kpic[a:a + n], vpic[a:a + n], np.arange(n), scale, hkv)
            attention_close(o_all[sel][pick], Q.round_storage(o, dt), f"chunk {s} attention L{l}", rep)
            hw = S.residual(sw, l, h_all[sel], o_all[sel])
            steps_close(ho_all[sel], hw, dt, f"chunk {s} residual L{l}", 1, rep, floor=_row_rms(hw))
    return rep
