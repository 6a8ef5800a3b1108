"""One layer's QCFuse fusion step on the GPU, as a stream-ordered chain of libqcf calls.

The host only lays out index arrays whose sizes it already knows (chunk
offsets, per-chunk selection budgets k_i = floor(rho * n_i), the slots of the
recomputed rows, the probe buffer layout); they are computed once per batch
layout and uploaded before the step.  Every step of the path itself --
re-positioning, anchor gather, probe attention, scores, selection, scatter,
attention -- runs in the library's kernels, with no device-to-host
synchronisation inside the step.

Sequence of one step (Section 3.5, selective token localization followed by
one layer of cache fusion):
  1. qcf_assemble        stored chunk caches -> request cache (keys re-positioned,
                         values stitched, eq. pic_online); user-query rows rotated
                         at N+i into the cache and q_u; probe buffer
                         [KV^A ; query K/V] (eq. anchor_cache)
  2. qcf_sparse_prefill_attn  query probe over the anchor cache (eq. anchor_query_state)
  3. qcf_probe_scores    I(t) over the context keys (eq. single_layer_importance)
  4. qcf_select_topk     per-chunk top-k -> P (eq. critical_mask)
  5. qcf_scatter_kv      rows R = P + query: rotate fresh q/k, write fresh K/V (eq. fuse_cache)
  6. qcf_sparse_prefill_attn  causal attention of R over the fused cache (Section 2.1.3)
Step 1 can also run as qcf_rerope + qcf_scatter_kv + two qcf_gather_rows.

Fused flow (``fused=True``): the scores read the stored chunk keys and
re-position them in registers (qcf_probe_scores_pic with a qcf_rope_table
table of the chunk offsets), so they no longer wait for the request cache.
The main stream runs qcf_assemble for the query rows and the probe buffer
only, then scores -> select -> scatter -> attention; a second stream builds
the rotation table, re-positions the context into the request cache
(qcf_rerope, needed from the scatter on) and runs the anchor probe.  Results
are bit-identical to the default flow; on one layer of 10 x 512-token chunks
the default flow is the faster one (re-positioning the context inside
qcf_assemble costs a few microseconds, less than the fused scores' extra
rotation work and the cross-stream synchronisation).

Every libqcf call of a stage is validated and marshalled once per FusionStep
(qcf.prepare) and replayed by later steps, so a step's host cost is little
more than the launches themselves.
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass

import numpy as np
import torch

from . import qcf

__all__ = ["FusionPlan", "FusionStep"]


@dataclass
class FusionPlan:
    """Host-side layout of one layer's step for a batch (sizes only, no scores)."""

    seg_k: np.ndarray        # [n_sel] selection budget of each selection segment
    out_start: np.ndarray    # [n_sel] first slot of each segment's selection in R
    cu_R: np.ndarray         # [B+1] recomputed-row slots per request: [P_b ; U_b]
    n_P: np.ndarray          # [B] |P_b|
    R_idx_init: np.ndarray   # [|R|] cache rows; query-row slots filled, P slots -1
    R_pos_init: np.ndarray   # [|R|] positions; query-row slots filled
    pos_base: np.ndarray     # [n_sel] first cache row of the segment's request
    sel_req: np.ndarray      # [n_sel] request of each selection segment
    u_idx: np.ndarray        # [n_q] cache rows of all query tokens
    u_pos: np.ndarray        # [n_q] positions N_b + i
    probe_idx: np.ndarray    # [n_probe] cache rows held by the probe buffer
    probe_pos: np.ndarray    # [n_probe] request positions of those rows
    probe_src: np.ndarray    # [n_probe] stored-chunk row of an anchor slot, -1 for a query slot
    probe_delta: np.ndarray  # [n_probe] chunk offset of an anchor slot (0 for a query slot)
    query_slot: np.ndarray   # [n_q] probe slot of each query token
    cu_probe: np.ndarray     # [B+1]
    max_q: int
    max_ctx: int
    max_R: int
    max_probe: int
    max_seg: int
    # selection segments (per chunk, or one per request in global mode)
    sel_start: np.ndarray    # [n_sel] first cache row
    sel_len: np.ndarray      # [n_sel]
    max_sel: int

    @staticmethod
    def build(w, rho_bp: int, selection: str = "chunk") -> "FusionPlan":
        """``selection``: "chunk" (k_i = floor(rho n_i) per chunk) or "global" (one
        floor(rho N_b) over each request's whole context, eq. critical_mask as written)."""
        B = w.batch
        if selection == "chunk":
            sel_start, sel_len, sel_req = w.seg_start, w.seg_len, w.seg_req
        elif selection == "global":
            has = np.asarray(w.ctx_len) > 0
            sel_start = np.asarray(w.cu_kv[:-1])[has]
            sel_len = np.asarray(w.ctx_len)[has]
            sel_req = np.nonzero(has)[0]
        else:
            raise ValueError(f"selection must be 'chunk' or 'global', not {selection!r}")
        n_sel = len(sel_start)
        seg_k = (int(rho_bp) * np.asarray(sel_len, np.int64)) // 10000
        n_P = np.zeros(B, np.int64)
        for s in range(n_sel):
            n_P[sel_req[s]] += seg_k[s]
        q_lens = np.array(w.q_lens, np.int64)
        cu_R = np.concatenate([[0], np.cumsum(n_P + q_lens)])
        out_start = np.zeros(n_sel, np.int64)
        fill = cu_R[:-1].copy()
        for s in range(n_sel):
            out_start[s] = fill[sel_req[s]]
            fill[sel_req[s]] += seg_k[s]
        R_idx = np.full(int(cu_R[-1]), -1, np.int64)
        R_pos = np.full(int(cu_R[-1]), -1, np.int64)
        u_idx, u_pos, probe_idx, probe_pos, cu_probe = [], [], [], [], [0]
        probe_src, probe_delta, query_slot = [], [], []
        for b in range(B):
            base, N, nq = int(w.cu_kv[b]), int(w.ctx_len[b]), int(w.q_lens[b])
            rows = np.arange(base + N, base + N + nq)
            pos = np.arange(N, N + nq)
            s0 = int(cu_R[b] + n_P[b])
            R_idx[s0:s0 + nq] = rows
            R_pos[s0:s0 + nq] = pos
            u_idx.append(rows)
            u_pos.append(pos)
            segs = np.nonzero(w.seg_req == b)[0]
            arows = [w.seg_start[s] + w.anchor_local[s] for s in segs]
            adelta = [np.full(len(w.anchor_local[s]), w.seg_delta[s]) for s in segs]
            arows = np.concatenate(arows) if arows else np.zeros(0, np.int64)
            adelta = np.concatenate(adelta) if adelta else np.zeros(0, np.int64)
            probe_idx += [arows, rows]
            probe_pos += [arows - base, pos]
            probe_src += [arows, np.full(nq, -1)]
            probe_delta += [adelta, np.zeros(nq)]
            query_slot.append(cu_probe[-1] + arows.size + np.arange(nq))
            cu_probe.append(cu_probe[-1] + arows.size + nq)
        cat = lambda xs: np.concatenate(xs).astype(np.int32) if xs else np.zeros(0, np.int32)
        pos_base = np.asarray(w.cu_kv)[np.asarray(sel_req, np.int64)].astype(np.int32)
        return FusionPlan(
            seg_k=seg_k.astype(np.int32), out_start=out_start.astype(np.int32),
            cu_R=cu_R.astype(np.int32), n_P=n_P, R_idx_init=R_idx.astype(np.int32),
            R_pos_init=R_pos.astype(np.int32), pos_base=pos_base,
            sel_req=np.asarray(sel_req, np.int32), u_idx=cat(u_idx),
            u_pos=cat(u_pos), probe_idx=cat(probe_idx), probe_pos=cat(probe_pos),
            probe_src=cat(probe_src), probe_delta=cat(probe_delta), query_slot=cat(query_slot),
            cu_probe=np.array(cu_probe, np.int32), max_q=int(max(w.q_lens) if B else 0),
            max_ctx=int(w.ctx_len.max() if B else 0),
            max_R=int(np.diff(cu_R).max() if B else 0),
            max_probe=int(np.diff(cu_probe).max() if B else 0),
            max_seg=int(w.seg_len.max() if w.n_chunks else 0),
            sel_start=np.asarray(sel_start, np.int32), sel_len=np.asarray(sel_len, np.int32),
            max_sel=int(max(sel_len) if n_sel else 0))


def kv_buffer(rows, hkv, d, dtype, device, zero=False):
    """[rows, hkv, d] K/V buffer whose rows are qcf_recommended_row_stride elements apart."""
    stride = qcf.qcf_recommended_row_stride(hkv, d)
    alloc = torch.zeros if zero else torch.empty
    return alloc((rows, stride), dtype=dtype, device=device)[:, :hkv * d].view(rows, hkv, d)


class FusionStep:
    """Device buffers and the call chain of one layer's fusion step for workload ``w``.

    ``run()`` enqueues the stages on the current stream.  The stored
    chunk caches (``k_pic``, ``v_pic``) are never modified: re-positioning
    writes the request cache (``k``, ``v``), which then receives the recomputed
    rows, so ``run()`` can be repeated with identical results.
    """

    def __init__(self, w, rho_bp: int | None = None, device="cuda", fused: bool = False,
                 selection: str = "chunk", fused_select: bool = True, rot_in_attn: bool = True):
        """``rot_in_attn`` (bf16): the recomputed rows' queries are rotated inside the
        attention (qcf_sparse_prefill_attn_rope, reading q_new through R_idx) and the scatter
        writes K/V only; otherwise the scatter writes rotated queries q_R for the attention."""
        self.w = w
        self.fused = bool(fused)
        # scores and selection through qcf_probe_scores_select (one launch less) or the two calls
        self.fused_select = bool(fused_select)
        self.selection = selection
        self.rho_bp = w.rho_bp if rho_bp is None else int(rho_bp)
        self.plan = p = FusionPlan.build(w, self.rho_bp, selection)
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.dtype = dt
        self.rot_in_attn = bool(rot_in_attn) and dt == torch.bfloat16
        dev = torch.device(device)
        self.device = dev
        T, hq, hkv, d = w.n_rows, w.n_q_heads, w.n_kv_heads, w.head_dim
        self.scale = 1.0 / math.sqrt(d)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
        # inputs
        self.k_pic = f(w.k_pic)
        self.v_pic = f(w.v_pic)
        self.q_new = f(w.q_new)
        self.k_new = f(w.k_new)
        self.v_new = f(w.v_new)
        # layout (int32)
        self.seg_start, self.seg_len, self.seg_delta = t(w.seg_start), t(w.seg_len), t(w.seg_delta)
        self.seg_k, self.out_start, self.pos_base = t(p.seg_k), t(p.out_start), t(p.pos_base)
        self.sel_start, self.sel_len, self.sel_req = t(p.sel_start), t(p.sel_len), t(p.sel_req)
        self.cu_kv, self.ctx_len, self.cu_q = t(w.cu_kv), t(w.ctx_len), t(w.cu_q)
        self.cu_R, self.cu_probe = t(p.cu_R), t(p.cu_probe)
        self.u_idx, self.u_pos = t(p.u_idx), t(p.u_pos)
        self.probe_idx, self.probe_pos = t(p.probe_idx), t(p.probe_pos)
        self.probe_src, self.probe_delta = t(p.probe_src), t(p.probe_delta)
        self.query_slot = t(p.query_slot)
        self.R_idx_init, self.R_pos_init = t(p.R_idx_init), t(p.R_pos_init)
        # working state and outputs; the caches the attention and score kernels read (the
        # request cache and the probe buffer) get the library's padded row stride
        self.k = kv_buffer(T, hkv, d, dt, dev, zero=True)
        self.v = kv_buffer(T, hkv, d, dt, dev, zero=True)
        self.R_idx = self.R_idx_init.clone()
        self.R_pos = self.R_pos_init.clone()
        nU, nR, nP = p.u_idx.size, p.R_idx_init.size, p.probe_idx.size
        self.q_u = torch.empty((nU, hq, d), dtype=dt, device=dev)
        self.q_R = None if self.rot_in_attn else torch.empty((nR, hq, d), dtype=dt, device=dev)
        self.k_probe = kv_buffer(nP, hkv, d, dt, dev)
        self.v_probe = kv_buffer(nP, hkv, d, dt, dev)
        self.o_probe = torch.empty((nU, hq, d), dtype=dt, device=dev)
        self.o = torch.empty((nR, hq, d), dtype=dt, device=dev)
        self.scores = torch.zeros(T, dtype=torch.float32, device=dev)
        nws = qcf.qcf_probe_scores_workspace_size(w.batch, p.max_q, p.max_ctx, hq, hkv, d)
        self.ws_scores = torch.empty(max(nws, 256), dtype=torch.uint8, device=dev)
        self.max_kv = int(np.diff(w.cu_kv).max()) if w.batch else 0
        nwa = qcf.qcf_sparse_prefill_attn_workspace_size(w.batch, p.max_R, max(self.max_kv, 1), hq,
                                                         hkv, d, dt)
        self.ws_attn = torch.empty(max(nwa, 256), dtype=torch.uint8, device=dev)
        nwp = qcf.qcf_sparse_prefill_attn_workspace_size(w.batch, p.max_q, max(p.max_probe, 1), hq,
                                                         hkv, d, dt)
        self.ws_probe = torch.empty(max(nwp, 256), dtype=torch.uint8, device=dev)
        # (cos, sin) of every request position, for the attention's query rotation
        self.pos_table = (qcf.rope_position_table(max(self.max_kv, 1), d, w.rope_theta, dev)
                          if self.rot_in_attn else None)
        # the anchor probe depends only on the assembled buffers and nothing later in the
        # step reads its output, so it runs on a second stream (default priority) beside
        # the score -> select -> scatter chain and is joined at the end of the step
        self.side = torch.cuda.Stream(device=dev)
        self.ev_assembled = torch.cuda.Event()
        self.ev_probed = torch.cuda.Event()
        # fused flow: one rotation per chunk offset, and each context row's table row
        key_rot = np.zeros(T, np.int32)
        for s in range(w.n_chunks):
            a, n = int(w.seg_start[s]), int(w.seg_len[s])
            key_rot[a:a + n] = s
        self.key_rot = t(key_rot)
        self.rope_table = torch.empty((max(w.n_chunks, 1), d // 2, 2), dtype=torch.float32, device=dev)
        self.no_seg = torch.zeros(0, dtype=torch.int32, device=dev)
        self.ev_start = torch.cuda.Event()
        # each stage's libqcf call is validated and marshalled once, then replayed
        self._prep = {}
        self._stream = None                       # raw handle of the stream to launch on (None: current)
        self._side_h = ctypes.c_void_p(self.side.cuda_stream)
        self.ev_table = torch.cuda.Event()
        self.ev_context = torch.cuda.Event()

    # -- stages ---------------------------------------------------------------
    def _call(self, key, fn, *args, **kw):
        p = self._prep.get(key)
        if p is None:
            p = self._prep[key] = qcf.prepare(fn, *args, **kw)
        p(self._stream)

    def stage_assemble(self):
        """Request cache (chunks re-positioned, values stitched), query rows, probe buffer."""
        w, p = self.w, self.plan
        self._call("assemble", qcf.qcf_assemble, self.k, self.v, self.k_pic, self.v_pic,
                   self.seg_start, self.seg_len, self.seg_delta, p.max_seg, self.q_new, self.k_new,
                   self.v_new, self.u_idx, self.u_pos, self.q_u, self.k_probe, self.v_probe,
                   self.probe_src, self.probe_delta, w.rope_theta, query_src=self.u_idx,
                   query_slot=self.query_slot)

    def stage_query_assemble(self):
        """Query rows (cache rows, q_u) and the probe buffer; the context is left alone."""
        w = self.w
        self._call("query_assemble", qcf.qcf_assemble, self.k, self.v, self.k_pic, self.v_pic,
                   self.no_seg, self.no_seg, self.no_seg, 0, self.q_new, self.k_new, self.v_new,
                   self.u_idx, self.u_pos, self.q_u, self.k_probe, self.v_probe, self.probe_src,
                   self.probe_delta, w.rope_theta, query_src=self.u_idx, query_slot=self.query_slot)

    def stage_rope_table(self):
        if self.w.n_chunks:
            self._call("rope_table", qcf.qcf_rope_table, self.rope_table, self.seg_delta,
                       self.w.rope_theta)

    def stage_scores_pic(self, accumulate=False):
        p = self.plan
        self._call(("scores_pic", accumulate), qcf.qcf_probe_scores_pic, self.scores, self.q_u,
                   self.k_pic, self.key_rot, self.rope_table, self.cu_q, self.cu_kv, self.ctx_len,
                   p.max_q, p.max_ctx, self.scale, accumulate=accumulate, workspace=self.ws_scores)

    # the same work as three separate calls (kept for the stage-by-stage tests)
    def stage_rerope(self):
        w, p = self.w, self.plan
        self._call("rerope", qcf.qcf_rerope, self.k, self.k_pic, self.seg_start, self.seg_len,
                   self.seg_delta, p.max_seg, w.rope_theta, v_out=self.v, v_in=self.v_pic)

    def stage_query_rows(self):
        self._call("query_rows", qcf.qcf_scatter_kv, self.k, self.v, self.k_new, self.v_new,
                   self.u_idx, self.u_pos, self.w.rope_theta, q_new=self.q_new, q_out=self.q_u,
                   src_idx=self.u_idx)

    def stage_anchor_gather(self):
        self._call("gather_k", qcf.qcf_gather_rows, self.k_probe, self.k, self.probe_idx)
        self._call("gather_v", qcf.qcf_gather_rows, self.v_probe, self.v, self.probe_idx)

    def stage_probe_attn(self):
        p = self.plan
        self._call("probe_attn", qcf.qcf_sparse_prefill_attn, self.o_probe, self.q_u, self.u_pos,
                   self.cu_q, self.k_probe, self.v_probe, self.cu_probe, p.max_q, p.max_probe,
                   self.scale, kv_pos=self.probe_pos, workspace=self.ws_probe)

    def stage_scores(self, accumulate=False):
        p = self.plan
        self._call(("scores", accumulate), qcf.qcf_probe_scores, self.scores, self.q_u, self.k,
                   self.cu_q, self.cu_kv, self.ctx_len, p.max_q, p.max_ctx, self.scale,
                   accumulate=accumulate, workspace=self.ws_scores)

    def stage_scores_select(self, accumulate=False):
        """Scores and the selection in one call (the last score pass and the selection share a
        launch); results identical to stage_scores then stage_select."""
        p = self.plan
        self._call(("scores_select", accumulate), qcf.qcf_probe_scores_select, self.scores,
                   self.q_u, self.k, self.cu_q, self.cu_kv, self.ctx_len, p.max_q, p.max_ctx,
                   self.scale, self.R_idx, self.sel_start, self.sel_len, self.seg_k,
                   self.out_start, self.sel_req, p.max_sel, out_pos=self.R_pos,
                   accumulate=accumulate, workspace=self.ws_scores)

    def stage_select(self):
        p = self.plan
        self._call("select", qcf.qcf_select_topk, self.R_idx, self.scores, self.sel_start,
                   self.sel_len, self.seg_k, self.out_start, p.max_sel, out_pos=self.R_pos,
                   pos_base=self.pos_base)

    def stage_scatter(self):
        if self.rot_in_attn:
            self._call("scatter", qcf.qcf_scatter_kv, self.k, self.v, self.k_new, self.v_new,
                       self.R_idx, self.R_pos, self.w.rope_theta, src_idx=self.R_idx)
        else:
            self._call("scatter", qcf.qcf_scatter_kv, self.k, self.v, self.k_new, self.v_new,
                       self.R_idx, self.R_pos, self.w.rope_theta, q_new=self.q_new, q_out=self.q_R,
                       src_idx=self.R_idx)

    def stage_attn(self):
        p = self.plan
        if self.rot_in_attn:
            self._call("attn", qcf.qcf_sparse_prefill_attn_rope, self.o, self.q_new, self.R_pos,
                       self.cu_R, self.k, self.v, self.cu_kv, p.max_R, self.max_kv, self.scale,
                       self.pos_table, q_src=self.R_idx, workspace=self.ws_attn)
        else:
            self._call("attn", qcf.qcf_sparse_prefill_attn, self.o, self.q_R, self.R_pos, self.cu_R,
                       self.k, self.v, self.cu_kv, p.max_R, self.max_kv, self.scale,
                       workspace=self.ws_attn)

    STAGES = ("assemble", "probe_attn", "scores_select", "scatter", "attn")
    STAGES_FUSED = ("rope_table", "rerope", "query_assemble", "probe_attn", "scores_pic", "select",
                    "scatter", "attn")

    def run_front_fused(self):
        """Fused flow up to the recomputed-row attention (the probe joins in join())."""
        main = torch.cuda.current_stream(self.device)
        side, main_h = self.side, ctypes.c_void_p(main.cuda_stream)
        try:
            # the side stream rewrites the request cache: not before the previous step's
            # work on the main stream
            self.ev_start.record(main)
            side.wait_event(self.ev_start)
            self._stream = self._side_h
            self.stage_rope_table()
            self.ev_table.record(side)
            self.stage_rerope()
            self.ev_context.record(side)
            self._stream = main_h
            self.stage_query_assemble()
            self.ev_assembled.record(main)
            side.wait_event(self.ev_assembled)
            self._stream = self._side_h
            self.stage_probe_attn()
            self.ev_probed.record(side)
            self._stream = main_h
            main.wait_event(self.ev_table)
            self.stage_scores_pic()
            self.stage_select()
            main.wait_event(self.ev_context)
            self.stage_scatter()
        finally:
            self._stream = None

    def run_front(self, separate_assembly=False, overlap=True):
        """Everything before the recomputed-row attention; the probe forks to the side stream."""
        if self.fused and not separate_assembly and overlap:
            return self.run_front_fused()
        if separate_assembly:
            self.stage_rerope()
            self.stage_query_rows()
            self.stage_anchor_gather()
        else:
            self.stage_assemble()
        if overlap:
            main = torch.cuda.current_stream(self.device)
            self.ev_assembled.record(main)
            self.side.wait_event(self.ev_assembled)
            self._stream = self._side_h
            try:
                self.stage_probe_attn()
            finally:
                self._stream = None
            self.ev_probed.record(self.side)
        else:
            self.stage_probe_attn()
        if self.fused_select:
            self.stage_scores_select()
        else:
            self.stage_scores()
            self.stage_select()
        self.stage_scatter()

    def join(self, overlap=True):
        """Make the current stream wait for the probe (before anything reuses its buffers)."""
        if overlap:
            torch.cuda.current_stream(self.device).wait_event(self.ev_probed)

    def run(self, separate_assembly=False, overlap=True):
        self.run_front(separate_assembly, overlap)
        self.stage_attn()
        self.join(overlap)

    # -- results on the host ----------------------------------------------------
    def results(self):
        torch.cuda.synchronize()
        c = lambda x: x.float().cpu().numpy().astype(np.float64)
        p = self.plan
        R = self.R_idx.cpu().numpy()
        Rp = self.R_pos.cpu().numpy()
        P = [R[p.cu_R[b]:p.cu_R[b] + p.n_P[b]] for b in range(self.w.batch)]
        op = c(self.o_probe)
        cq = self.w.cu_q
        return dict(k_fuse=c(self.k), v_fuse=c(self.v), scores=self.scores.double().cpu().numpy(),
                    R=R, R_pos=Rp, P=P, cu_R=p.cu_R, o=c(self.o), o_probe=op,
                    o_probe_list=[op[cq[b]:cq[b + 1]] for b in range(self.w.batch)],
                    q_u=c(self.q_u), **({} if self.rot_in_attn else dict(q_R=c(self.q_R))))
