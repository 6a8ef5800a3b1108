"""CPU oracle for a multi-layer QCFuse request (the c3 stack configuration).

TEST INFRASTRUCTURE ONLY, like ``oracle.qcfuse``: only the tests, the smoke
check of the graft entry point and the CPU-baseline leg of the benchmark may
import or run it.  It builds on the single-layer definitions of
``oracle.qcfuse`` and shares nothing with the HIP library.

The stack is a sequence of attention blocks; for layer l and hidden states h:
    x = RMSNorm(h)                      (no gain, eps from the workload)
    q = rope(x Wq_l, pos), k = rope(x Wk_l, pos), v = x Wv_l
    o = causal GQA attention of q over the layer's keys/values
    h <- h + o Wo_l
QCFuse on such a stack (Section 3.5 with the critical-layer selector of
Section 3.4.2):
  * offline, each chunk runs through the stack alone at positions 0..n_i-1;
    its per-layer K/V is the chunk's PIC cache (Section 2.1.2, eq. pic_offline);
  * online, the user-query rows run through layers 0..max(L*) attending only
    to [anchor cache ; themselves] (eq. anchor_query_state), where the anchor
    cache of layer l is the re-positioned PIC rows of the anchors (eq.
    anchor_cache); at each critical layer l in L* their rotated queries score
    the context keys of that layer's re-positioned cache, summed over L*
    (eq. critical_layer_importance);
  * one per-chunk top-k selection P (eq. critical_mask per chunk) drives the
    recomputation of every layer: rows R = P + query rows start from their
    input embeddings, and at each layer their fresh K/V replace the
    re-positioned PIC entries (eq. fuse_cache) before they attend causally
    over that layer's fused cache (Section 2.1.3).
Readings (the paper fixes none of them for a synthetic stack): attention-only
blocks without an MLP, RMSNorm without a learned gain, residual in the
storage dtype.  Where the GPU stores a tensor in the storage dtype (normed
input, projections, rotated q/k, attention output, hidden state) the oracle
rounds it once to that dtype; the arithmetic in between is float64.  The
output projection and the residual sum form one stored tensor (the product
is added into the hidden state before it is rounded).
"""
from __future__ import annotations

import numpy as np

from .qcfuse import (attention, critical_scores, round_storage, rope, select_per_chunk, select_topk)

__all__ = ["rms_norm", "block_proj", "block_qkv", "full_forward", "build_pic", "stack_fusion", "anchor_count",
           "anchors_sink", "anchors_knorm"]


def rms_norm(h, eps):
    """h / sqrt(mean(h^2) + eps) per row (float64)."""
    h = np.asarray(h, np.float64)
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def block_proj(sw, l, h):
    """Un-rotated q [n, H_q, d], k and v [n, H_kv, d] of layer l for hidden states h:
    RMSNorm(h) and the three products, each stored in the storage dtype."""
    dt, d = sw.dtype, sw.head_dim
    n = h.shape[0]
    x = round_storage(rms_norm(h, sw.rms_eps), dt)
    q = round_storage(x @ np.asarray(sw.wq[l], np.float64), dt).reshape(n, sw.n_q_heads, d)
    k = round_storage(x @ np.asarray(sw.wk[l], np.float64), dt).reshape(n, sw.n_kv_heads, d)
    v = round_storage(x @ np.asarray(sw.wv[l], np.float64), dt).reshape(n, sw.n_kv_heads, d)
    return q, k, v


def block_qkv(sw, l, h, pos):
    """Rotated q [n, H_q, d], rotated k and v [n, H_kv, d] of layer l for hidden states h."""
    dt = sw.dtype
    q, k, v = block_proj(sw, l, h)
    q = round_storage(rope(q, pos, sw.rope_theta), dt)
    k = round_storage(rope(k, pos, sw.rope_theta), dt)
    return q, k, v


def residual(sw, l, h, o):
    """h + o Wo_l, stored once in the storage dtype (the product and the sum are one
    step, as a projection that adds into its output does it)."""
    y = o.reshape(o.shape[0], -1) @ np.asarray(sw.wo[l], np.float64)
    return round_storage(np.asarray(h, np.float64) + y, sw.dtype)


def full_forward(sw, h0, pos):
    """Plain causal forward of one token sequence through every layer.

    h0 [n, d_model] input states, pos [n] ascending positions.  Returns the
    per-layer rotated keys and values (lists of [n, H_kv, d]) and the final
    hidden states [n, d_model].
    """
    scale = 1.0 / np.sqrt(sw.head_dim)
    h = round_storage(h0, sw.dtype)
    ks, vs = [], []
    for l in range(sw.n_layers):
        q, k, v = block_qkv(sw, l, h, pos)
        ks.append(k)
        vs.append(v)
        o = round_storage(attention(q, pos, k, v, pos, scale, sw.n_kv_heads), sw.dtype)
        h = residual(sw, l, h, o)
    return ks, vs, h


def build_pic(sw):
    """Per-layer PIC caches [T, H_kv, d] (zero on query rows): every chunk alone at 0..n_i-1."""
    T, hkv, d = sw.n_rows, sw.n_kv_heads, sw.head_dim
    K = [np.zeros((T, hkv, d)) for _ in range(sw.n_layers)]
    V = [np.zeros((T, hkv, d)) for _ in range(sw.n_layers)]
    for s in range(sw.n_chunks):
        a, n = int(sw.seg_start[s]), int(sw.seg_len[s])
        ks, vs, _ = full_forward(sw, sw.embed[a:a + n], np.arange(n))
        for l in range(sw.n_layers):
            K[l][a:a + n] = ks[l]
            V[l][a:a + n] = vs[l]
    return K, V


def _reposition(sw, K_pic_l, b):
    """Request b's context keys of one layer moved to their request positions (eq. pic_online)."""
    out = {}
    for s in np.nonzero(sw.seg_req == b)[0]:
        a, n, o = int(sw.seg_start[s]), int(sw.seg_len[s]), int(sw.seg_delta[s])
        out[a] = round_storage(rope(K_pic_l[a:a + n], np.full(n, o), sw.rope_theta), sw.dtype)
    return out


def stack_fusion(sw, rho_bp=None, pic=None):
    """QCFuse over the whole stack for every request of ``sw``.

    Returns a dict with, per request: the accumulated scores of the context
    rows, P, R ([P ascending ; query rows]), the final hidden states of R and
    the query probe's last output; and per layer the fused caches.
    """
    dt = sw.dtype
    scale = 1.0 / np.sqrt(sw.head_dim)
    rho_bp = sw.rho_bp if rho_bp is None else int(rho_bp)
    K_pic, V_pic = pic if pic is not None else build_pic(sw)
    L, T = sw.n_layers, sw.n_rows
    lmax = max(sw.critical_layers)
    res = dict(scores=np.zeros(T), P=[], R=[], h_R=[], o_probe=[], h_probe=[],
               k_fuse=[np.zeros_like(K_pic[0]) for _ in range(L)],
               v_fuse=[np.zeros_like(V_pic[0]) for _ in range(L)])
    for b in range(sw.batch):
        base, N, nq = int(sw.cu_kv[b]), int(sw.ctx_len[b]), int(sw.q_lens[b])
        n_b = N + nq
        urows = np.arange(base + N, base + n_b)
        upos = np.arange(N, n_b)
        segs = np.nonzero(sw.seg_req == b)[0]
        arows = (np.concatenate([sw.seg_start[s] + sw.anchor_local[s] for s in segs])
                 if segs.size else np.zeros(0, np.int64))
        apos = arows - base
        # per-layer request caches: re-positioned PIC (values stitched)
        Kreq, Vreq = [], []
        for l in range(L):
            Kl = np.zeros((n_b, sw.n_kv_heads, sw.head_dim))
            Vl = np.zeros_like(Kl)
            for a, kr in _reposition(sw, K_pic[l], b).items():
                Kl[a - base:a - base + kr.shape[0]] = kr
            Vl[:N] = V_pic[l][base:base + N]
            Kreq.append(Kl)
            Vreq.append(Vl)
        # query probe over [anchor cache ; query], scores at the critical layers
        hU = round_storage(sw.embed[urows], dt)
        scores = np.zeros(N)
        o_probe = np.zeros((nq, sw.n_q_heads, sw.head_dim))
        for l in range(lmax + 1):
            qU, kU, vU = block_qkv(sw, l, hU, upos)
            kp = np.concatenate([Kreq[l][apos], kU])
            vp = np.concatenate([Vreq[l][apos], vU])
            o_probe = round_storage(attention(qU, upos, kp, vp, np.concatenate([apos, upos]),
                                              scale, sw.n_kv_heads), dt)
            if l in sw.critical_layers:
                scores += critical_scores(qU, Kreq[l][:N], scale, sw.n_kv_heads)
            hU = residual(sw, l, hU, o_probe)
        res["scores"][base:base + N] = scores
        # one selection for every layer
        srows = np.zeros(T)
        srows[base:base + N] = scores
        P = select_per_chunk(srows, sw.seg_start[segs], sw.seg_len[segs], rho_bp)
        R = np.concatenate([P, urows])
        Rpos = R - base
        # recompute R through every layer over the fused caches
        hR = round_storage(sw.embed[R], dt)
        kpos = np.arange(n_b)
        for l in range(L):
            qR, kR, vR = block_qkv(sw, l, hR, Rpos)
            Kf, Vf = Kreq[l].copy(), Vreq[l].copy()
            Kf[Rpos] = kR
            Vf[Rpos] = vR
            oR = round_storage(attention(qR, Rpos, Kf, Vf, kpos, scale, sw.n_kv_heads), dt)
            hR = residual(sw, l, hR, oR)
            res["k_fuse"][l][base:base + n_b] = Kf
            res["v_fuse"][l][base:base + n_b] = Vf
        res["P"].append(P)
        res["R"].append(R)
        res["h_R"].append(hR)
        res["o_probe"].append(o_probe)
        res["h_probe"].append(hU)
    return res


# ---------------------------------------------------------------------------
# offline anchor sets  (Section 3.3.1, eq. anchor_set)
# ---------------------------------------------------------------------------
def anchor_count(n, ra_bp):
    """ceil(r_a * n) with r_a in basis points (integer arithmetic)."""
    return (int(ra_bp) * int(n) + 9999) // 10000


def anchors_sink(seg_len, ra_bp):
    """Sink rule: the first ceil(r_a n_i) positions of every chunk."""
    return [np.arange(anchor_count(n, ra_bp), dtype=np.int64) for n in seg_len]


def anchors_knorm(K_pic, seg_start, seg_len, ra_bp):
    """Knorm rule: per chunk, the ceil(r_a n_i) positions whose stored keys have the
    smallest L2 norm (mean over layers and KV heads of the per-head norm); equal
    scores to the lower position, output ascending."""
    norms = np.mean([np.linalg.norm(np.asarray(k, np.float64), axis=-1).mean(axis=-1) for k in K_pic], axis=0)
    out = []
    for a, n in zip(seg_start, seg_len):
        a, n = int(a), int(n)
        out.append(select_topk(-norms[a:a + n], anchor_count(n, ra_bp)))
    return out
