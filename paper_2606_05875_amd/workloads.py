"""Seeded synthetic workloads for one layer of the cache-fusion step.

This module only draws random tensors, lays out the packed variable-length
buffers and rounds every input once to its storage dtype.  It holds none of the
method's arithmetic (no rotation, no softmax, no selection, no counts derived
from the recomputation ratio): both the HIP path and the CPU oracle receive the
very same arrays from here and do that work themselves.

Workload shapes follow the paper's evaluation setting (retrieved chunks of a
few hundred tokens, a user query appended after the context, GQA attention of
7B-70B class models; Experiments section, Implementation / Datasets).  The
paper's datasets and trained weights are not available, so the values are
synthetic:

* stored chunk keys/values are i.i.d. N(0, 1)/sqrt(d) (isotropic);
* a fraction of context tokens is "evidence": its stored key is
  0.8*u_g + 0.6*eps with u_g a unit direction per KV head g and eps a unit
  Gaussian direction; the user-query rows carry beta*(0.8*u_g + 0.6*eps')
  with beta = 6.25*sqrt(d), so an evidence logit is about +4 while background
  logits have a standard deviation of about 0.55-0.78;
* u_g lives on the slowest rotary pairs (the last d/16 pairs of the
  rotate-half layout, whose rotation over the whole request stays below a few
  tenths of a radian), so the planted alignment survives re-positioning
  without this module applying any rotation;
* fresh (recomputed) projections are i.i.d.: keys/values N(0, 1)/sqrt(d),
  context-row queries N(0, 1)*sqrt(d) (unit-std logits);
* anchor positions are drawn uniformly without replacement inside each chunk
  (the paper's default anchor rule needs the language model).

Row layout (packed, token-major): request b owns cache rows
[cu_kv[b], cu_kv[b+1]); its N_b context tokens come first, in chunk order,
followed by its n_q,b user-query rows.  Query rows of the stored cache are
zero; the fusion step writes them.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["CONFIGS", "Workload", "make_workload", "round_to_bf16", "config_names", "STACK_CONFIGS",
           "StackWorkload", "make_stack_workload", "full_view"]


# ---------------------------------------------------------------------------
# configurations
# ---------------------------------------------------------------------------
# index: position of the config in the seeded RNG key; evidence: how planted
# evidence is spread.  rho_bp is the recomputation ratio in basis points.
CONFIGS = {
    "c1": dict(index=1, dtype="f32", chunks=[128] * 4, n_q=32, n_q_heads=8,
               n_kv_heads=2, head_dim=64, rope_theta=1.0e4, anchors=8,
               rho_bp=3000, evidence=("uniform_count", 51),
               desc="tiny fp32 layer: 4x128 chunks + 32-token query, 8/2/64"),
    "c2": dict(index=2, dtype="bf16", chunks=[512] * 10, n_q=64, n_q_heads=32,
               n_kv_heads=8, head_dim=128, rope_theta=5.0e5, anchors=16,
               rho_bp=3000, evidence=("chunks", 2, 256),
               desc="Llama-3-8B-shaped layer: 10x512 chunks + 64-token query, 32/8/128"),
    "c4": dict(index=4, dtype="bf16", chunks=[1024] * 32, n_q=128, n_q_heads=64,
               n_kv_heads=8, head_dim=128, rope_theta=5.0e5, anchors=32,
               rho_bp=3000, evidence=("chunks", 4, 983),
               desc="70B-GQA-shaped long-context layer: 32x1024 chunks + 128-token query, 64/8/128"),
    "c5": dict(index=5, dtype="bf16", ragged=dict(batch=16, chunks=(8, 16), chunk_len=(256, 1024),
                                                 n_q=(16, 128)),
               n_q_heads=32, n_kv_heads=8, head_dim=128, rope_theta=5.0e5, anchors=16,
               rho_bp=2000, evidence=("request_fraction_bp", 500),
               desc="ragged serving batch: 16 requests x U[8,16] chunks x U[256,1024] tokens, "
                    "U[16,128]-token queries, 32/8/128"),
}


def config_names():
    return list(CONFIGS)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round a float array to the nearest bfloat16 value (ties to even).

    Returns float32 values that are exactly representable in bfloat16.  Input
    preparation only: every tensor handed to either side is rounded once here.
    """
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    bits = a32.view(np.uint32).astype(np.uint64)
    bias = ((bits >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)
    out = ((bits + bias) & np.uint64(0xFFFF0000)).astype(np.uint32)
    return out.view(np.float32).reshape(a32.shape)


@dataclass
class Workload:
    """One layer's inputs for a batch of requests (host arrays).

    Integer layout arrays are int32; tensors are float32 holding values that
    are exact in ``dtype``.
    """

    name: str
    dtype: str                 # "f32" or "bf16": storage dtype of every tensor
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    rho_bp: int                # recomputation ratio in basis points
    anchors_per_chunk: int
    chunk_lens: list           # per request: list of chunk lengths
    q_lens: list               # per request: user-query length
    # packed layout
    cu_kv: np.ndarray          # [B+1] first cache row of each request
    ctx_len: np.ndarray        # [B] context tokens N_b
    cu_q: np.ndarray           # [B+1] prefix sums of q_lens
    seg_start: np.ndarray      # [n_chunks] first cache row of each chunk
    seg_len: np.ndarray        # [n_chunks] chunk length
    seg_req: np.ndarray        # [n_chunks] request of each chunk
    seg_delta: np.ndarray      # [n_chunks] request position of the chunk's first token
    anchor_local: list         # per chunk: sorted chunk-local anchor positions (int32)
    evidence_rows: np.ndarray  # sorted cache rows of planted evidence tokens
    # tensors
    k_pic: np.ndarray          # [T, H_kv, d] stored chunk keys (chunk-local rotation)
    v_pic: np.ndarray          # [T, H_kv, d] stored chunk values
    q_new: np.ndarray          # [T, H_q, d] fresh queries, before rotation
    k_new: np.ndarray          # [T, H_kv, d] fresh keys, before rotation
    v_new: np.ndarray          # [T, H_kv, d] fresh values
    meta: dict = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return len(self.q_lens)

    @property
    def n_rows(self) -> int:
        return int(self.cu_kv[-1])

    @property
    def n_chunks(self) -> int:
        return int(self.seg_start.shape[0])

    def query_rows(self, b: int) -> np.ndarray:
        """Cache rows of request b's user-query tokens."""
        s = int(self.cu_kv[b]) + int(self.ctx_len[b])
        return np.arange(s, s + int(self.q_lens[b]), dtype=np.int32)

    def anchor_rows(self) -> np.ndarray:
        """Cache rows of all anchors, chunk by chunk (so request by request)."""
        parts = [self.seg_start[i] + self.anchor_local[i] for i in range(self.n_chunks)]
        return np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)


def _layout(cfg, rng):
    if "ragged" in cfg:
        r = cfg["ragged"]
        chunk_lens, q_lens = [], []
        for _ in range(r["batch"]):
            m = int(rng.integers(r["chunks"][0], r["chunks"][1], endpoint=True))
            lens = rng.integers(r["chunk_len"][0], r["chunk_len"][1], endpoint=True, size=m)
            nq = int(rng.integers(r["n_q"][0], r["n_q"][1], endpoint=True))
            chunk_lens.append([int(x) for x in lens])
            q_lens.append(nq)
        return chunk_lens, q_lens
    return [list(cfg["chunks"])], [int(cfg["n_q"])]


def _slow_pair_direction(rng, d, n):
    """n unit vectors supported on the last d/16 rotary pairs (coords j and j+d/2)."""
    half = d // 2
    npair = max(d // 16, 1)
    coords = np.concatenate([np.arange(half - npair, half), np.arange(d - npair, d)])
    u = np.zeros((n, d), np.float64)
    u[:, coords] = rng.standard_normal((n, coords.size))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    return u


def _unit_rows(rng, shape):
    e = rng.standard_normal(shape)
    return e / np.linalg.norm(e, axis=-1, keepdims=True)


def make_workload(name: str, seed: int = 0, rho_bp: int | None = None,
                  chunk_lens=None, q_lens=None, anchors_per_chunk: int | None = None,
                  dtype: str | None = None, overrides: dict | None = None) -> Workload:
    """Draw one config's workload.

    ``chunk_lens``/``q_lens`` replace the config's request layout (used by the
    edge-case tests: ragged tails, single chunks, one-token queries);
    ``overrides`` replaces head counts / head_dim / theta.
    Draw order (fixed): layout, evidence placement, evidence directions,
    stored K, stored V, evidence noise, fresh Q, fresh K, fresh V, anchors.
    """
    cfg = dict(CONFIGS[name])
    if overrides:
        cfg.update(overrides)
    rng = np.random.default_rng([seed, cfg["index"]])
    if chunk_lens is None:
        chunk_lens, q_lens_l = _layout(cfg, rng)
    else:
        q_lens_l = list(q_lens)
    if q_lens is not None:
        q_lens_l = list(q_lens)
    chunk_lens = [list(map(int, c)) for c in chunk_lens]
    hq, hkv, d = int(cfg["n_q_heads"]), int(cfg["n_kv_heads"]), int(cfg["head_dim"])
    dt = dtype or cfg["dtype"]
    n_anchor = int(cfg["anchors"] if anchors_per_chunk is None else anchors_per_chunk)

    B = len(q_lens_l)
    ctx = np.array([sum(c) for c in chunk_lens], np.int64)
    rows = ctx + np.array(q_lens_l, np.int64)
    cu_kv = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(q_lens_l)]).astype(np.int32)
    seg_start, seg_len, seg_req, seg_delta = [], [], [], []
    for b in range(B):
        off = 0
        for n in chunk_lens[b]:
            seg_start.append(int(cu_kv[b]) + off)
            seg_len.append(n)
            seg_req.append(b)
            seg_delta.append(off)
            off += n
    seg_start = np.array(seg_start, np.int32)
    seg_len = np.array(seg_len, np.int32)
    seg_req = np.array(seg_req, np.int32)
    seg_delta = np.array(seg_delta, np.int32)
    T = int(cu_kv[-1])

    # -- evidence placement ------------------------------------------------
    ev = []
    kind = cfg["evidence"][0]
    for b in range(B):
        segs = np.nonzero(seg_req == b)[0]
        if kind == "uniform_count":
            cnt = min(int(cfg["evidence"][1]), int(ctx[b]))
            loc = rng.choice(int(ctx[b]), size=cnt, replace=False)
            ev.append(int(cu_kv[b]) + loc)
        elif kind == "request_fraction_bp":
            cnt = int(ctx[b]) * int(cfg["evidence"][1]) // 10000
            loc = rng.choice(int(ctx[b]), size=cnt, replace=False)
            ev.append(int(cu_kv[b]) + loc)
        elif kind == "chunks":
            nch = min(int(cfg["evidence"][1]), segs.size)
            total = int(cfg["evidence"][2])
            pick = np.sort(rng.choice(segs, size=nch, replace=False))
            per = [total // nch + (1 if i < total % nch else 0) for i in range(nch)]
            for s, cnt in zip(pick, per):
                cnt = min(cnt, int(seg_len[s]))
                loc = rng.choice(int(seg_len[s]), size=cnt, replace=False)
                ev.append(int(seg_start[s]) + loc)
        else:
            raise ValueError(kind)
    evidence_rows = np.sort(np.concatenate(ev)).astype(np.int32) if ev else np.zeros(0, np.int32)
    u = _slow_pair_direction(rng, d, hkv)                     # [H_kv, d]

    # -- stored chunk caches ------------------------------------------------
    is_ctx = np.zeros(T, bool)
    for s in range(seg_start.size):
        is_ctx[seg_start[s]:seg_start[s] + seg_len[s]] = True
    inv = 1.0 / np.sqrt(d)
    k_pic = rng.standard_normal((T, hkv, d), dtype=np.float32) * np.float32(inv)
    v_pic = rng.standard_normal((T, hkv, d), dtype=np.float32) * np.float32(inv)
    k_pic[~is_ctx] = 0.0
    v_pic[~is_ctx] = 0.0
    if evidence_rows.size:
        eps = _unit_rows(rng, (evidence_rows.size, hkv, d))
        k_pic[evidence_rows] = (0.8 * u[None] + 0.6 * eps).astype(np.float32)

    # -- fresh projections ----------------------------------------------------
    q_new = rng.standard_normal((T, hq, d), dtype=np.float32) * np.float32(np.sqrt(d))
    beta = 6.25 * np.sqrt(d)
    grp = hq // hkv
    qrows = np.concatenate([np.arange(cu_kv[b] + ctx[b], cu_kv[b + 1]) for b in range(B)])
    if qrows.size:
        eps_q = _unit_rows(rng, (qrows.size, hq, d))
        ug = np.repeat(u, grp, axis=0)                          # head h -> u_{h // grp}
        q_new[qrows] = (beta * (0.8 * ug[None] + 0.6 * eps_q)).astype(np.float32)
    k_new = rng.standard_normal((T, hkv, d), dtype=np.float32) * np.float32(inv)
    v_new = rng.standard_normal((T, hkv, d), dtype=np.float32) * np.float32(inv)

    # -- anchors --------------------------------------------------------------
    anchor_local = []
    for s in range(seg_start.size):
        a = min(n_anchor, int(seg_len[s]))
        anchor_local.append(np.sort(rng.choice(int(seg_len[s]), size=a, replace=False)).astype(np.int32))

    if dt == "bf16":
        k_pic, v_pic, q_new, k_new, v_new = (round_to_bf16(x) for x in (k_pic, v_pic, q_new, k_new, v_new))
    elif dt != "f32":
        raise ValueError(dt)

    return Workload(
        name=name, dtype=dt, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
        rope_theta=float(cfg["rope_theta"]),
        rho_bp=int(cfg["rho_bp"] if rho_bp is None else rho_bp),
        anchors_per_chunk=n_anchor, chunk_lens=chunk_lens, q_lens=q_lens_l,
        cu_kv=cu_kv, ctx_len=ctx.astype(np.int32), cu_q=cu_q,
        seg_start=seg_start, seg_len=seg_len, seg_req=seg_req, seg_delta=seg_delta,
        anchor_local=anchor_local, evidence_rows=evidence_rows,
        k_pic=k_pic, v_pic=v_pic, q_new=q_new, k_new=k_new, v_new=v_new,
        meta=dict(seed=seed, desc=cfg.get("desc", "")),
    )


# ---------------------------------------------------------------------------
# multi-layer stack (the c3 configuration)
# ---------------------------------------------------------------------------
# A stack of attention blocks (RMSNorm, Wq/Wk/Wv, rotary, causal GQA attention,
# Wo, residual) with random weights.  The selector scores at the critical
# layers and one selection drives the recomputation of every layer.  Weights
# are N(0, sigma^2) with sigma = 0.02 * sqrt(4096 / d_model), so a reduced
# shape keeps the logit statistics of the 4096-wide stack; embeddings are
# N(0, 1).  Anchors are drawn uniformly inside each chunk.
STACK_CONFIGS = {
    "c3": dict(index=3, dtype="bf16", chunks=[512] * 20, n_q=64, n_layers=36, d_model=4096,
               n_q_heads=32, n_kv_heads=8, head_dim=128, rope_theta=1.0e6, anchors=52,
               critical_layers=(2, 12, 24), rho_bp=3000,
               desc="Qwen3-8B-shaped 36-layer stack: 20x512 chunks + 64-token query, 32/8/128, "
                    "critical layers 2, 12, 24"),
    # the same structure at a size the float64 oracle runs in seconds
    "c3_small": dict(index=31, dtype="f32", chunks=[96, 64, 80, 33], n_q=12, n_layers=6,
                     d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, rope_theta=1.0e6,
                     anchors=6, critical_layers=(1, 3), rho_bp=3000,
                     desc="reduced c3-shaped stack: 6 layers, 4 chunks, 12-token query, 4/2/64"),
}


@dataclass
class StackWorkload:
    """Inputs of a multi-layer request batch (host arrays, float32 values exact in dtype)."""

    name: str
    dtype: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    rho_bp: int
    critical_layers: tuple
    rms_eps: float
    chunk_lens: list
    q_lens: list
    cu_kv: np.ndarray
    ctx_len: np.ndarray
    cu_q: np.ndarray
    seg_start: np.ndarray
    seg_len: np.ndarray
    seg_req: np.ndarray
    seg_delta: np.ndarray
    anchor_local: list
    embed: np.ndarray        # [T, d_model] input hidden state of every token
    wq: np.ndarray           # [L, d_model, H_q*d]
    wk: np.ndarray           # [L, d_model, H_kv*d]
    wv: np.ndarray           # [L, d_model, H_kv*d]
    wo: np.ndarray           # [L, H_q*d, d_model]
    meta: dict = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return len(self.q_lens)

    @property
    def n_rows(self) -> int:
        return int(self.cu_kv[-1])

    @property
    def n_chunks(self) -> int:
        return int(self.seg_start.shape[0])


def make_stack_workload(name: str = "c3", seed: int = 0, rho_bp: int | None = None,
                        chunk_lens=None, q_lens=None, anchors_per_chunk: int | None = None,
                        dtype: str | None = None, overrides: dict | None = None,
                        evidence: tuple | None = None) -> StackWorkload:
    """Draw a stack config's inputs.  Draw order (fixed): anchors, embeddings, then per
    layer Wq, Wk, Wv, Wo; then, with ``evidence``, the planted evidence.

    ``evidence = (n_chunks, count)`` plants answer-bearing tokens for a recall profile
    (a mechanism demonstration, the paper's span-labelled datasets being absent): ``count``
    context positions spread over ``n_chunks`` drawn chunks get the embedding of a drawn
    user-query token plus 10% noise, and in every layer the key projection of each KV head
    is the query projection of the group's first query head, so a query token's first
    head matches its own duplicates ("matching heads").  The positions are returned in
    ``meta["evidence_rows"]``."""
    cfg = dict(STACK_CONFIGS[name])
    if overrides:
        cfg.update(overrides)
    rng = np.random.default_rng([seed, cfg["index"]])
    chunk_lens = [list(map(int, c)) for c in (chunk_lens or [cfg["chunks"]])]
    q_lens_l = list(q_lens) if q_lens is not None else [int(cfg["n_q"])] * len(chunk_lens)
    hq, hkv, d = int(cfg["n_q_heads"]), int(cfg["n_kv_heads"]), int(cfg["head_dim"])
    dm, L = int(cfg["d_model"]), int(cfg["n_layers"])
    dt = dtype or cfg["dtype"]
    n_anchor = int(cfg["anchors"] if anchors_per_chunk is None else anchors_per_chunk)
    B = len(q_lens_l)
    ctx = np.array([sum(c) for c in chunk_lens], np.int64)
    rows = ctx + np.array(q_lens_l, np.int64)
    cu_kv = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(q_lens_l)]).astype(np.int32)
    seg_start, seg_len, seg_req, seg_delta = [], [], [], []
    for b in range(B):
        off = 0
        for n in chunk_lens[b]:
            seg_start.append(int(cu_kv[b]) + off)
            seg_len.append(n)
            seg_req.append(b)
            seg_delta.append(off)
            off += n
    seg_start, seg_len = np.array(seg_start, np.int32), np.array(seg_len, np.int32)
    seg_req, seg_delta = np.array(seg_req, np.int32), np.array(seg_delta, np.int32)
    anchor_local = []
    for s in range(seg_start.size):
        a = min(n_anchor, int(seg_len[s]))
        anchor_local.append(np.sort(rng.choice(int(seg_len[s]), size=a, replace=False)).astype(np.int32))
    T = int(cu_kv[-1])
    sigma = np.float32(0.02 * np.sqrt(4096.0 / dm))
    embed = rng.standard_normal((T, dm), dtype=np.float32)
    wq = np.empty((L, dm, hq * d), np.float32)
    wk = np.empty((L, dm, hkv * d), np.float32)
    wv = np.empty((L, dm, hkv * d), np.float32)
    wo = np.empty((L, hq * d, dm), np.float32)
    if dt not in ("bf16", "f32"):
        raise ValueError(dt)
    rnd = round_to_bf16 if dt == "bf16" else (lambda x: x)
    for l in range(L):   # rounded layer by layer (the full stack is several GB)
        wq[l] = rnd(rng.standard_normal((dm, hq * d), dtype=np.float32) * sigma)
        wk[l] = rnd(rng.standard_normal((dm, hkv * d), dtype=np.float32) * sigma)
        wv[l] = rnd(rng.standard_normal((dm, hkv * d), dtype=np.float32) * sigma)
        wo[l] = rnd(rng.standard_normal((hq * d, dm), dtype=np.float32) * sigma)
    ev_rows = np.zeros(0, np.int32)
    if evidence is not None:
        n_ev_chunks, count = int(evidence[0]), int(evidence[1])
        grp = hq // hkv
        for l in range(L):
            for g in range(hkv):
                wk[l][:, g * d:(g + 1) * d] = wq[l][:, g * grp * d:(g * grp + 1) * d]
        ev = []
        for b in range(B):
            segs = np.nonzero(seg_req == b)[0]
            pick = np.sort(rng.choice(segs, size=min(n_ev_chunks, segs.size), replace=False))
            per = [count // pick.size + (1 if i < count % pick.size else 0) for i in range(pick.size)]
            qrows = np.arange(cu_kv[b] + ctx[b], cu_kv[b + 1])
            for s_, cnt in zip(pick, per):
                loc = rng.choice(int(seg_len[s_]), size=min(cnt, int(seg_len[s_])), replace=False)
                rows_e = int(seg_start[s_]) + loc
                src = rng.choice(qrows, size=rows_e.size)
                embed[rows_e] = embed[src] + 0.1 * rng.standard_normal((rows_e.size, dm), dtype=np.float32)
                ev.append(rows_e)
        ev_rows = np.sort(np.concatenate(ev)).astype(np.int32)
    embed = rnd(embed)
    return StackWorkload(
        name=name, dtype=dt, n_layers=L, d_model=dm, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
        rope_theta=float(cfg["rope_theta"]), rho_bp=int(cfg["rho_bp"] if rho_bp is None else rho_bp),
        critical_layers=tuple(int(x) for x in cfg["critical_layers"]), rms_eps=1e-6,
        chunk_lens=chunk_lens, q_lens=q_lens_l, cu_kv=cu_kv, ctx_len=ctx.astype(np.int32),
        cu_q=cu_q, seg_start=seg_start, seg_len=seg_len, seg_req=seg_req, seg_delta=seg_delta,
        anchor_local=anchor_local, embed=embed, wq=wq, wk=wk, wv=wv, wo=wo,
        meta=dict(seed=seed, desc=cfg.get("desc", ""), evidence_rows=ev_rows))


def full_view(sw: StackWorkload) -> StackWorkload:
    """The same request batch seen by the full-view reference selector (Section 3.2.2):
    every context token is an anchor (the probe reads the complete stitched cache) and every
    layer scores (the full layer set).  Layout only; nothing is recomputed here."""
    import dataclasses
    return dataclasses.replace(
        sw, anchor_local=[np.arange(int(n), dtype=np.int32) for n in sw.seg_len],
        critical_layers=tuple(range(sw.n_layers)),
        meta=dict(sw.meta, view="full"))
