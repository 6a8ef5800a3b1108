"""CPU oracle for one layer of the QCFuse cache-fusion step.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check of the graft entry
point and the CPU-baseline leg of the benchmark may import or run this module;
the product path never does.  It shares no code with the HIP library and
imports nothing from the package except through the arrays the tests pass in.

Every function is the plain definition from the paper, written out in NumPy
with float64 arithmetic (no tiling, no fusion, no reordering of the math).
Where a tensor is *stored* by a BF16 serving stack (the re-positioned cache,
the rotated fresh keys and queries, the attention outputs) the result is
rounded once to the storage dtype, exactly like the paper's BF16 stack stores
it (Experiments, Implementation); everything in between stays float64.

Readings of the paper that the code takes (the paper is silent or loose):
  * rotary embedding: rotate-half pairs (j, j + d/2), omega_j = theta^(-2j/d),
    no frequency scaling; angles in float64;
  * the stored chunk key is already rotated at its chunk-local position, so
    re-positioning rotates it by the chunk's request offset (Section 2.1.2,
    eq. pic_online);
  * the per-layer attention mass Attn^l(Q, K_C) is a softmax over the
    request's N context keys only, summed (not averaged) over query tokens
    and heads (Section 3.2.1, eq. importance; Section 3.4.2);
  * selection is per chunk with k_i = floor(rho * n_i) (rho in basis points,
    integer arithmetic); larger score first, equal scores to the lower index,
    output ascending (eq. critical_mask applied per chunk);
  * the user-query rows are always recomputed, sit after the context at
    positions N..N+n_q-1 and are not counted in rho (Section 2.1.1);
  * attention of a recomputed row at position p sees every key whose position
    is <= p, itself included, over the fused cache after all of the layer's
    fresh K/V are written (Section 2.1.3, eq. fuse_cache);
  * softmax scale 1/sqrt(d); no extra norms, capping or biases.
No function here is "parity unpinned": each has a pin in the CPU test suite
(closed forms, invariants, brute force or an independent library routine).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "round_storage", "round_bf16", "rope_angles", "rope", "rerope", "per_chunk_k",
    "attention", "critical_scores", "select_topk", "select_per_chunk",
    "fusion_step", "recall",
]


# ---------------------------------------------------------------------------
# storage rounding
# ---------------------------------------------------------------------------
def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to even.

    bfloat16 keeps float32's exponent range: normal numbers down to 2^-126,
    below that a fixed spacing of 2^-133.
    """
    x = np.asarray(x, np.float64)
    _, e = np.frexp(x)                       # x = m * 2^e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)                  # 0.5 * 2^-125 = 2^-126, smallest normal
    spacing = np.ldexp(1.0, e - 8)
    return np.round(x / spacing) * spacing   # np.round rounds half to even


def round_storage(x, dtype):
    """Round to the storage dtype ("bf16" or "f32"); returns float64."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# rotary position embedding  (Section 2.1.2: position remapping of rotary keys)
# ---------------------------------------------------------------------------
def rope_angles(pos, d, theta):
    """Angle pos * omega_j for j < d/2, omega_j = theta^(-2j/d), float64."""
    j = np.arange(d // 2, dtype=np.float64)
    omega = np.power(np.float64(theta), -2.0 * j / d)
    return np.asarray(pos, np.float64)[..., None] * omega


def rope(x, pos, theta):
    """Rotate x[..., H, d] by position pos[...] (one position per row, shared by heads).

    Pairs (x_j, x_{j+d/2}) turn by angle pos*omega_j:
    (x_j cos a - x_{j+d/2} sin a, x_j sin a + x_{j+d/2} cos a).
    """
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    a = rope_angles(pos, d, theta)[..., None, :]          # broadcast over heads
    c, s = np.cos(a), np.sin(a)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def rerope(k_pic, seg_start, seg_len, seg_delta, theta, dtype):
    """Pi_i of eq. pic_online for the keys: rotate each chunk's stored keys by its offset.

    Stored keys are encoded at chunk-local positions 0..n_i-1; rotary rotations
    compose, so moving chunk i to request offset o_i is one more rotation by o_i.
    Rows outside every chunk are copied unchanged.  Returns float64 values
    exact in the storage dtype.
    """
    out = np.array(k_pic, np.float64, copy=True)
    for s in range(len(seg_start)):
        a, n, o = int(seg_start[s]), int(seg_len[s]), int(seg_delta[s])
        if n == 0:
            continue
        out[a:a + n] = round_storage(rope(out[a:a + n], np.full(n, o), theta), dtype)
    return out


# ---------------------------------------------------------------------------
# attention with explicit key positions  (Section 2.1.3 causal rule; eq. anchor_query_state)
# ---------------------------------------------------------------------------
def attention(q, qpos, k, v, kpos, scale, n_kv_heads, rows_per_pass=16):
    """softmax(q k^T * scale) v per query row and head, over keys with kpos <= qpos.

    q [R, H_q, d]; k, v [n, H_kv, d]; kpos ascending.  Query head h reads KV
    head h // (H_q / H_kv) (grouped-query attention).  A row that sees no key
    returns zeros.  Returns float64 [R, H_q, d].

    The rows are taken a few at a time (``rows_per_pass``) only to bound the
    memory of the logit matrix; every row's softmax runs over all of its
    visible keys at once, with the invisible ones masked out.
    """
    q = np.asarray(q, np.float64)
    qpos = np.asarray(qpos)
    kpos = np.asarray(kpos)
    assert np.all(np.diff(kpos) >= 0), "key positions must be ascending"
    assert k.shape[1] == n_kv_heads and q.shape[1] % n_kv_heads == 0
    R, hq, d = q.shape
    g = hq // n_kv_heads
    kh = np.ascontiguousarray(np.asarray(k, np.float64).transpose(1, 0, 2))   # [H_kv, n, d]
    vh = np.ascontiguousarray(np.asarray(v, np.float64).transpose(1, 0, 2))   # [H_kv, n, d]
    out = np.zeros(q.shape, np.float64)
    for r0 in range(0, R, rows_per_pass):
        rows = np.arange(r0, min(R, r0 + rows_per_pass))
        nvis = np.searchsorted(kpos, qpos[rows], side="right")    # row i sees keys 0..nvis[i]-1
        m = int(nvis.max())
        if m == 0:
            continue
        # [H_kv, rows * g, d] @ [H_kv, d, m]: the logits of every (row, head) pair
        qb = q[rows].reshape(rows.size, n_kv_heads, g, d).transpose(1, 0, 2, 3).reshape(n_kv_heads, -1, d)
        s = np.matmul(qb, kh[:, :m].transpose(0, 2, 1))
        s *= scale
        hidden = np.repeat(np.arange(m)[None, :] >= nvis[:, None], g, axis=0)   # [rows * g, m]
        if hidden.any():
            s[:, hidden] = -np.inf
        mx = s.max(axis=-1, keepdims=True)
        s -= np.where(np.isfinite(mx), mx, 0.0)
        np.exp(s, out=s)                                               # exp(-inf) = 0
        den = s.sum(axis=-1, keepdims=True)
        np.divide(s, den, out=s, where=den > 0)
        o = np.matmul(s, vh[:, :m])                                    # [H_kv, rows * g, d]
        out[rows] = o.reshape(n_kv_heads, rows.size, g, d).transpose(1, 0, 2, 3).reshape(rows.size, hq, d)
    return out


# ---------------------------------------------------------------------------
# critical-layer importance  (eq. single_layer_importance, eq. critical_layer_importance)
# ---------------------------------------------------------------------------
def critical_scores(q_u, k_ctx, scale, n_kv_heads):
    """I(t) = sum over query tokens i and heads h of softmax_t(q_{h,i} . k_{g(h),t} * scale).

    q_u [n_q, H_q, d] are the (rotated) user-query states, k_ctx [N, H_kv, d]
    the request's context keys at their original positions.  The softmax runs
    over the N context keys.  Returns float64 [N].  Summing this over the
    critical layers gives eq. critical_layer_importance.
    """
    q_u = np.asarray(q_u, np.float64)
    k_ctx = np.asarray(k_ctx, np.float64)
    nq, hq, d = q_u.shape
    N = k_ctx.shape[0]
    g = hq // n_kv_heads
    out = np.zeros(N, np.float64)
    if N == 0 or nq == 0:
        return out
    for h in range(hq):
        logits = (q_u[:, h, :] @ k_ctx[:, h // g, :].T) * scale      # [n_q, N]
        logits -= logits.max(axis=1, keepdims=True)
        p = np.exp(logits)
        p /= p.sum(axis=1, keepdims=True)
        out += p.sum(axis=0)
    return out


# ---------------------------------------------------------------------------
# selection  (eq. critical_mask, applied per chunk)
# ---------------------------------------------------------------------------
def per_chunk_k(n, rho_bp):
    """k_i = floor(rho * n_i) with rho in basis points (integer arithmetic)."""
    return (int(rho_bp) * int(n)) // 10000


def select_topk(scores, k):
    """Positions of the k largest scores; equal scores go to the lower index; ascending."""
    scores = np.asarray(scores, np.float64)
    assert np.all(np.isfinite(scores))
    s = np.where(scores == 0.0, 0.0, scores)                 # -0 and +0 are equal
    order = np.lexsort((np.arange(s.size), -s))              # by -score, then index
    return np.sort(order[:k]).astype(np.int64)


def select_per_chunk(scores_rows, seg_start, seg_len, rho_bp):
    """Per-chunk top-k over a score vector indexed by cache row; returns sorted rows."""
    out = []
    for s in range(len(seg_start)):
        a, n = int(seg_start[s]), int(seg_len[s])
        k = per_chunk_k(n, rho_bp)
        out.append(a + select_topk(scores_rows[a:a + n], k))
    return np.concatenate(out) if out else np.zeros(0, np.int64)


# ---------------------------------------------------------------------------
# one layer of the fusion step
# ---------------------------------------------------------------------------
def fusion_step(w, rho_bp=None, attn_rows=None, selection="chunk", P=None):
    """Run one layer's QCFuse fusion step on workload ``w`` (see the package's workloads).

    Steps, per request b:
      1. re-position every chunk's stored keys (eq. pic_online);
      2. rotate the user-query rows' fresh q/k at positions N_b + i;
      3. anchor cache KV^A = re-positioned cache at rows o_i + A_i, keeping their
         request positions (eq. anchor_cache), probe attention of the query
         rows over [KV^A ; query K/V] (eq. anchor_query_state);
      4. scores I(t) of the context tokens (eq. single_layer_importance);
      5. top-k of the scores (eq. critical_mask): per chunk, k_i = floor(rho n_i)
         (``selection="chunk"``), or over the request's whole context, k = floor(rho N_b)
         as the equation is written (``selection="global"``);
      6. R = P + query rows: rotate the fresh q/k of R at their positions and
         write the fresh K/V into the cache rows R (eq. fuse_cache);
      7. causal attention of R over the fused cache (Section 2.1.3).

    ``P``: None, or the recomputed context rows to use instead of the
    selection of step 5 (one ascending array of cache rows per request).  The
    selection of step 5 is still computed and returned as ``P_select``; steps 6
    and 7 follow ``P``.  Where scores tie within rounding, several selections
    are correct; a caller that has accepted another selection against
    ``P_select`` and ``scores`` gets here the fused cache and the attention
    that the definitions give for that selection.
    ``attn_rows``: None (every row of R) or the cache rows (a subset of R)
    whose attention output is evaluated, for large configurations.
    Returns a dict of float64 / integer arrays; ``o`` maps a cache row to its
    attention output [H_q, d].
    """
    dt = w.dtype
    d, hq, hkv = w.head_dim, w.n_q_heads, w.n_kv_heads
    theta = w.rope_theta
    scale = 1.0 / np.sqrt(d)
    rho_bp = w.rho_bp if rho_bp is None else int(rho_bp)
    T = w.n_rows
    if selection not in ("chunk", "global"):
        raise ValueError(f"selection must be 'chunk' or 'global', not {selection!r}")

    K = rerope(w.k_pic, w.seg_start, w.seg_len, w.seg_delta, theta, dt)
    k_rerope = K.copy()
    V = np.array(w.v_pic, np.float64, copy=True)
    scores = np.zeros(T, np.float64)
    res = dict(k_rerope=k_rerope, o_probe=[], q_u=[], P=[], P_select=[], R=[], R_pos=[], o={})

    def fresh_row(rows, pos):
        """The recomputed rows' q and k rotated at their positions, and their v."""
        qr = round_storage(rope(w.q_new[rows], pos, theta), dt)
        kr = round_storage(rope(w.k_new[rows], pos, theta), dt)
        return qr, kr, np.asarray(w.v_new[rows], np.float64)

    for b in range(w.batch):
        base, N, nq = int(w.cu_kv[b]), int(w.ctx_len[b]), int(w.q_lens[b])
        urows = np.arange(base + N, base + N + nq)
        upos = np.arange(N, N + nq)
        qU, kU, vU = fresh_row(urows, upos)
        # anchor cache with request positions, then the probe over [KV^A ; query K/V]
        segs = np.nonzero(w.seg_req == b)[0]
        arows = (np.concatenate([w.seg_start[s] + w.anchor_local[s] for s in segs])
                 if segs.size else np.zeros(0, np.int64))
        kp = np.concatenate([K[arows], kU])
        vp = np.concatenate([V[arows], vU])
        ppos = np.concatenate([arows - base, upos])
        res["o_probe"].append(round_storage(attention(qU, upos, kp, vp, ppos, scale, hkv), dt))
        res["q_u"].append(qU)
        # scores over the request's context keys (re-positioned PIC keys), then the selection
        scores[base:base + N] = critical_scores(qU, K[base:base + N], scale, hkv)
        if selection == "global":
            sel = [(base, N)]
        else:
            sel = [(int(w.seg_start[s]), int(w.seg_len[s])) for s in segs]
        P_sel = select_per_chunk(scores, [a for a, _ in sel], [n for _, n in sel], rho_bp)
        P_b = P_sel if P is None else np.asarray(P[b], np.int64)
        assert np.all(np.diff(P_b) > 0) and np.all((P_b >= base) & (P_b < base + N))
        res["P_select"].append(P_sel)
        res["P"].append(P_b)
        R = np.concatenate([P_b, urows])
        res["R"].append(R)
        res["R_pos"].append(R - base)

    # fused cache: every recomputed row holds its fresh K/V (eq. fuse_cache)
    for b in range(w.batch):
        base = int(w.cu_kv[b])
        R = res["R"][b]
        _, kR, vR = fresh_row(R, R - base)
        K[R] = kR
        V[R] = vR

    # attention of R (or of the requested rows of R) over the fused cache
    want = None if attn_rows is None else set(int(r) for r in np.asarray(attn_rows).ravel())
    for b in range(w.batch):
        base, n_b = int(w.cu_kv[b]), int(w.cu_kv[b + 1] - w.cu_kv[b])
        R = res["R"][b]
        rows = R if want is None else np.array([r for r in R if int(r) in want], np.int64)
        if rows.size == 0:
            continue
        qr, _, _ = fresh_row(rows, rows - base)
        o = round_storage(attention(qr, rows - base, K[base:base + n_b], V[base:base + n_b],
                                    np.arange(n_b), scale, hkv), dt)
        for i, r in enumerate(rows):
            res["o"][int(r)] = o[i]
    if want is not None:
        inR = set(int(r) for b in range(w.batch) for r in res["R"][b])
        assert want <= inR, "attn_rows must be recomputed rows"

    res["scores"] = scores
    res["k_fuse"] = K
    res["v_fuse"] = V
    return res


def recall(P_rows, evidence_rows):
    """|P intersect E| / |E| (eq. profile_recall_at10 with planted evidence as E)."""
    E = np.asarray(evidence_rows)
    if E.size == 0:
        return 1.0
    return float(np.isin(E, np.asarray(P_rows)).sum()) / E.size
