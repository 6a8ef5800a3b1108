"""QCFuse over a multi-layer attention stack on the GPU (the c3 configuration).

The hot-path steps of every layer run in libqcf (re-positioning, the probe
buffer and query-row rotation, probe attention, critical-layer scores, the
per-chunk top-k, the fresh-row scatter and the recomputed-row attention).  The
stack's own glue -- RMSNorm, the Wq/Wk/Wv/Wo projections and the residual --
is plain torch (library GEMMs); it only produces each layer's inputs.

Flow (Section 3.5 with the critical-layer selector of Section 3.4.2):
  offline  each chunk runs through the stack alone at positions 0..n_i-1 and
           its per-layer K/V becomes the chunk's PIC cache (all chunks of a
           layer as one batch of independent sequences);
  probe    layers 0..max(L*): qcf_assemble rotates the query rows' fresh q/k
           at N + i and fills the probe buffer [anchors ; query] (anchors
           re-positioned straight from the stored chunks); the query rows
           attend over it; at a critical layer the same launch also
           re-positions the layer's chunks into the request cache and
           qcf_probe_scores adds the layer's importance to the scores;
  select   one qcf_select_topk -> P; R = [P ; query rows] per request;
  recompute every layer: re-position (layers that were not scored), scatter
           R's fresh K/V (q rotated alongside), attend R over the fused cache.
No device-to-host synchronisation happens inside ``run()``.
"""
from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

from . import qcf
from .step import FusionPlan, kv_buffer

__all__ = ["FusionStack", "HostPicPipeline"]


class FusionStack:
    def __init__(self, sw, rho_bp: int | None = None, device="cuda", share: "FusionStack | None" = None):
        """``share``: another FusionStack of the same weights and chunks whose uploaded
        inputs and PIC caches are reused (another anchor view, critical-layer set or ratio)."""
        self.sw = sw
        self.rho_bp = sw.rho_bp if rho_bp is None else int(rho_bp)
        self.plan = p = FusionPlan.build(sw, self.rho_bp)
        dt = torch.bfloat16 if sw.dtype == "bf16" else torch.float32
        self.dtype = dt
        dev = torch.device(device)
        self.device = dev
        T, hq, hkv, d, L = sw.n_rows, sw.n_q_heads, sw.n_kv_heads, sw.head_dim, sw.n_layers
        self.scale = 1.0 / math.sqrt(d)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
        if share is not None:
            self.embed, self.wqkv, self.wo = share.embed, share.wqkv, share.wo
        else:
            self.embed = f(sw.embed)
            # W_q | W_k | W_v side by side: one product per layer gives q, k and v
            self.wqkv = torch.cat([f(sw.wq), f(sw.wk), f(sw.wv)], dim=2)
            self.wo = f(sw.wo)
        # layout
        self.seg_start, self.seg_len, self.seg_delta = t(sw.seg_start), t(sw.seg_len), t(sw.seg_delta)
        self.seg_k, self.out_start, self.pos_base = t(p.seg_k), t(p.out_start), t(p.pos_base)
        self.cu_kv, self.ctx_len, self.cu_q = t(sw.cu_kv), t(sw.ctx_len), t(sw.cu_q)
        self.cu_R, self.cu_probe = t(p.cu_R), t(p.cu_probe)
        self.u_idx, self.u_pos = t(p.u_idx), t(p.u_pos)
        self.probe_pos, self.probe_src = t(p.probe_pos), t(p.probe_src)
        self.probe_delta, self.query_slot = t(p.probe_delta), t(p.query_slot)
        self.R_idx_init, self.R_pos_init = t(p.R_idx_init), t(p.R_pos_init)
        self.u_src = t(np.arange(p.u_idx.size, dtype=np.int32))
        # offline PIC layout: every chunk a sequence of its own, keys at rows seg_start..
        self.ctx_rows = t(np.concatenate([np.arange(a, a + n) for a, n in zip(sw.seg_start, sw.seg_len)])
                          .astype(np.int32) if sw.n_chunks else np.zeros(0, np.int32))
        self.ctx_local = t(np.concatenate([np.arange(n) for n in sw.seg_len]).astype(np.int32)
                           if sw.n_chunks else np.zeros(0, np.int32))
        self.cu_chunk_rows = t(np.concatenate([[0], np.cumsum(sw.seg_len)]).astype(np.int32))
        self.cu_chunk_kv = t(np.concatenate([sw.seg_start, [T]]).astype(np.int32))
        self.max_chunk_kv = int(np.diff(np.concatenate([sw.seg_start, [T]])).max()) if sw.n_chunks else 1
        # caches: PIC and the per-layer request caches (padded rows, see kv_buffer)
        if share is not None:
            self.k_pic, self.v_pic = share.k_pic, share.v_pic
            self.k_req, self.v_req = share.k_req, share.v_req
        else:
            self.k_pic = [kv_buffer(T, hkv, d, dt, dev, zero=True) for _ in range(L)]
            self.v_pic = [kv_buffer(T, hkv, d, dt, dev, zero=True) for _ in range(L)]
            self.k_req = [kv_buffer(T, hkv, d, dt, dev, zero=True) for _ in range(L)]
            self.v_req = [kv_buffer(T, hkv, d, dt, dev, zero=True) for _ in range(L)]
        nU, nR, nP = p.u_idx.size, p.R_idx_init.size, p.probe_idx.size
        self.k_probe = kv_buffer(nP, hkv, d, dt, dev)
        self.v_probe = kv_buffer(nP, hkv, d, dt, dev)
        self.q_u = torch.empty((nU, hq, d), dtype=dt, device=dev)
        self.o_probe = torch.empty((nU, hq, d), dtype=dt, device=dev)
        self.scores = torch.zeros(T, dtype=torch.float32, device=dev)
        self.R_idx = self.R_idx_init.clone()
        self.R_pos = self.R_pos_init.clone()
        # bf16: the recompute's attention rotates the queries itself (table of every position)
        self.pos_table = (qcf.rope_position_table(max(self.max_kv_rows(sw), 1), d, sw.rope_theta, dev)
                          if dt == torch.bfloat16 else None)
        self.q_R = torch.empty((nR, hq, d), dtype=dt, device=dev) if self.pos_table is None else None
        self.o_R = torch.empty((nR, hq, d), dtype=dt, device=dev)
        self.max_kv = int(np.diff(sw.cu_kv).max()) if sw.batch else 1
        nws = qcf.qcf_probe_scores_workspace_size(sw.batch, p.max_q, p.max_ctx, hq, hkv, d)
        self.ws_scores = torch.empty(max(nws, 256), dtype=torch.uint8, device=dev)
        wa = lambda b, r, kv: qcf.qcf_sparse_prefill_attn_workspace_size(b, r, max(kv, 1), hq, hkv, d, dt)
        self.ws_attn = torch.empty(max(wa(sw.batch, p.max_R, self.max_kv),
                                       wa(sw.n_chunks, int(sw.seg_len.max()) if sw.n_chunks else 1,
                                          self.max_chunk_kv),
                                       wa(sw.batch, p.max_q, p.max_probe), 256),
                                   dtype=torch.uint8, device=dev)
        self.pic_built = share.pic_built if share is not None else False
        self.no_seg = torch.zeros(0, dtype=torch.int32, device=dev)
        # layers whose per-layer inputs and outputs are kept (device copies) for inspection:
        # tr_pic[l] (offline chunk pass), tr_sel[l] (query probe), tr_rec[l] (recompute)
        self.trace: set = set()
        self.tr_pic, self.tr_sel, self.tr_rec = {}, {}, {}

    @staticmethod
    def max_kv_rows(sw):
        return int(np.diff(sw.cu_kv).max()) if sw.batch else 1

    # -- glue: RMSNorm, projections, residual (torch) ---------------------------
    def _qkv(self, l, h):
        sw = self.sw
        n = h.shape[0]
        # float32 statistics inside the kernel, one rounding of the normed row to the storage dtype
        x = F.rms_norm(h, (h.shape[-1],), eps=sw.rms_eps)
        y = x @ self.wqkv[l]
        nq, nkv = sw.n_q_heads * sw.head_dim, sw.n_kv_heads * sw.head_dim
        q = y[:, :nq].reshape(n, sw.n_q_heads, sw.head_dim)
        k = y[:, nq:nq + nkv].reshape(n, sw.n_kv_heads, sw.head_dim)
        v = y[:, nq + nkv:].reshape(n, sw.n_kv_heads, sw.head_dim)
        return q.contiguous(), k.contiguous(), v.contiguous()

    def _residual(self, l, h, o):
        return torch.addmm(h, o.reshape(o.shape[0], -1), self.wo[l])

    # -- offline: PIC caches --------------------------------------------------
    def build_pic(self):
        """Each chunk alone through the stack at positions 0..n_i-1 (all chunks as one batch)."""
        sw = self.sw
        n = int(self.ctx_rows.numel())
        h = self.embed.index_select(0, self.ctx_rows.long())
        q_rot = torch.empty((n, sw.n_q_heads, sw.head_dim), dtype=self.dtype, device=self.device)
        o = torch.empty_like(q_rot)
        for l in range(sw.n_layers):
            q, k, v = self._qkv(l, h)
            qcf.qcf_scatter_kv(self.k_pic[l], self.v_pic[l], k, v, self.ctx_rows, self.ctx_local,
                               sw.rope_theta, q_new=q, q_out=q_rot)
            qcf.qcf_sparse_prefill_attn(o, q_rot, self.ctx_local, self.cu_chunk_rows, self.k_pic[l],
                                        self.v_pic[l], self.cu_chunk_kv,
                                        int(sw.seg_len.max()), self.max_chunk_kv, self.scale,
                                        workspace=self.ws_attn)
            h_in = h
            h = self._residual(l, h, o)
            if l in self.trace:
                self.tr_pic[l] = dict(h=h_in.clone(), q_raw=q.clone(), k_raw=k.clone(), q=q_rot.clone(),
                                      o=o.clone(), h_out=h.clone())
        self.pic_built = True

    # -- where the stored chunk caches come from ---------------------------------
    class _Resident:
        """Every layer's PIC cache stays in device memory."""

        def __init__(self, st):
            self.st = st

        def get(self, l, full):
            return self.st.k_pic[l], self.st.v_pic[l], self.st.probe_src

        def release(self, l):
            pass

    # -- online ---------------------------------------------------------------
    def run(self, src=None):
        self.select(src)
        self.recompute(src)

    def select(self, src=None):
        """Query probe up to the last critical layer, scores, one per-chunk top-k."""
        sw, p = self.sw, self.plan
        if not self.pic_built:
            self.build_pic()
        src = src or self._Resident(self)
        lmax = max(sw.critical_layers)
        # query probe over [anchor cache ; query] up to the last critical layer
        hU = self.embed.index_select(0, self.u_idx.long())
        first = True
        for l in range(lmax + 1):
            q, k, v = self._qkv(l, hU)
            # the whole context is re-positioned here only where it is scored; other
            # layers get the probe buffer and query rows now and their chunks in recompute()
            crit = l in sw.critical_layers
            segs = (self.seg_start, self.seg_len, self.seg_delta) if crit else (self.no_seg,) * 3
            kp, vp, psrc = src.get(l, full=crit)
            qcf.qcf_assemble(self.k_req[l], self.v_req[l], kp, vp, *segs,
                             p.max_seg if crit else 0, q, k, v, self.u_idx, self.u_pos,
                             self.q_u, self.k_probe, self.v_probe, psrc, self.probe_delta,
                             sw.rope_theta, query_src=self.u_src, query_slot=self.query_slot)
            src.release(l)
            qcf.qcf_sparse_prefill_attn(self.o_probe, self.q_u, self.u_pos, self.cu_q, self.k_probe,
                                        self.v_probe, self.cu_probe, p.max_q, p.max_probe, self.scale,
                                        kv_pos=self.probe_pos, workspace=self.ws_attn)
            if l in sw.critical_layers:
                qcf.qcf_probe_scores(self.scores, self.q_u, self.k_req[l], self.cu_q, self.cu_kv,
                                     self.ctx_len, p.max_q, p.max_ctx, self.scale,
                                     accumulate=not first, workspace=self.ws_scores)
                first = False
            h_in = hU
            hU = self._residual(l, hU, self.o_probe)
            if l in self.trace:
                self.tr_sel[l] = dict(h=h_in.clone(), q_raw=q.clone(), k_raw=k.clone(), q=self.q_u.clone(),
                                      k_probe=self.k_probe.clone(), v_probe=self.v_probe.clone(),
                                      o=self.o_probe.clone(), h_out=hU.clone())
        self.h_probe = hU
        # one selection for every layer
        self.R_idx.copy_(self.R_idx_init)
        self.R_pos.copy_(self.R_pos_init)
        qcf.qcf_select_topk(self.R_idx, self.scores, self.seg_start, self.seg_len, self.seg_k,
                            self.out_start, p.max_seg, out_pos=self.R_pos, pos_base=self.pos_base)

    def recompute(self, src=None):
        """R through every layer over the fused caches (after select())."""
        sw, p = self.sw, self.plan
        src = src or self._Resident(self)
        L = sw.n_layers
        hR = self.embed.index_select(0, self.R_idx.long())
        for l in range(L):
            if l not in sw.critical_layers:
                kp, vp, _ = src.get(l, full=True)
                qcf.qcf_rerope(self.k_req[l], kp, self.seg_start, self.seg_len, self.seg_delta,
                               p.max_seg, sw.rope_theta, v_out=self.v_req[l], v_in=vp)
                src.release(l)
            q, k, v = self._qkv(l, hR)
            if self.pos_table is not None:
                # fresh K/V into the cache; the attention rotates the queries itself
                qcf.qcf_scatter_kv(self.k_req[l], self.v_req[l], k, v, self.R_idx, self.R_pos,
                                   sw.rope_theta)
                qcf.qcf_sparse_prefill_attn_rope(self.o_R, q, self.R_pos, self.cu_R, self.k_req[l],
                                                 self.v_req[l], self.cu_kv, p.max_R, self.max_kv,
                                                 self.scale, self.pos_table, workspace=self.ws_attn)
            else:
                qcf.qcf_scatter_kv(self.k_req[l], self.v_req[l], k, v, self.R_idx, self.R_pos,
                                   sw.rope_theta, q_new=q, q_out=self.q_R)
                qcf.qcf_sparse_prefill_attn(self.o_R, self.q_R, self.R_pos, self.cu_R, self.k_req[l],
                                            self.v_req[l], self.cu_kv, p.max_R, self.max_kv, self.scale,
                                            workspace=self.ws_attn)
            h_in = hR
            hR = self._residual(l, hR, self.o_R)
            if l in self.trace:
                q_rot = self.q_R
                if self.pos_table is not None:
                    # the rotated queries are not stored by this flow: the scatter forms them
                    # for the record (the same K/V rows are written again)
                    q_rot = torch.empty_like(q)
                    qcf.qcf_scatter_kv(self.k_req[l], self.v_req[l], k, v, self.R_idx, self.R_pos,
                                       sw.rope_theta, q_new=q, q_out=q_rot)
                self.tr_rec[l] = dict(h=h_in.clone(), q_raw=q.clone(), k_raw=k.clone(), q=q_rot.clone(),
                                      o=self.o_R.clone(), h_out=hR.clone())
        self.h_R = hR

    def results(self, caches: bool = True):
        """Host copies of the outputs; ``caches=False`` leaves out the per-layer fused caches."""
        torch.cuda.synchronize()
        c = lambda x: x.float().cpu().numpy().astype(np.float64)
        p = self.plan
        R = self.R_idx.cpu().numpy()
        hR = c(self.h_R)
        hP = c(self.h_probe)
        cq = self.sw.cu_q
        out = dict(scores=self.scores.double().cpu().numpy(), R=R, cu_R=p.cu_R,
                   P=[R[p.cu_R[b]:p.cu_R[b] + p.n_P[b]] for b in range(self.sw.batch)],
                   h_R=[hR[p.cu_R[b]:p.cu_R[b + 1]] for b in range(self.sw.batch)],
                   h_probe=[hP[cq[b]:cq[b + 1]] for b in range(self.sw.batch)])
        if caches:
            out.update(k_fuse=[c(k) for k in self.k_req], v_fuse=[c(v) for v in self.v_req])
        return out


class HostPicPipeline:
    """Layer-wise pipelining of the stored chunk caches from pinned host memory
    (Section 3.5: the caches of later layers load while earlier layers compute).

    The PIC caches are moved to pinned host memory, every layer's full cache
    and, separately, the compact block of its anchor rows in probe-buffer
    order.  A copy stream (default priority) fills device staging slots (three
    by default) in
    the order the compute asks for them: during selection each probe layer
    needs only its anchor block (a critical layer its full cache, which is
    re-positioned there), during the recompute every layer not re-positioned
    during selection needs its full cache.  The compute stream waits for a
    slot's copy before its first use and frees the slot right after the launch
    that reads it (assemble or re-position), so the next copy into it overlaps
    the rest of that layer and the following one.  Results are bit-identical to
    the device-resident run (same kernels, same values).
    """

    def __init__(self, st: FusionStack, slots: int = 3):
        sw, p = st.sw, st.plan
        self.st = st
        self.n_slots = max(2, int(slots))
        dev, dt = st.device, st.dtype
        T, hkv, d = sw.n_rows, sw.n_kv_heads, sw.head_dim
        if not st.pic_built:
            st.build_pic()
        anchor_slots = np.nonzero(p.probe_src >= 0)[0]
        a_rows = torch.from_numpy(p.probe_src[anchor_slots].astype(np.int64)).to(dev)
        self.k_host, self.v_host, self.ka_host, self.va_host = [], [], [], []
        for l in range(sw.n_layers):
            for lst, x in ((self.k_host, st.k_pic[l]), (self.v_host, st.v_pic[l])):
                h = torch.empty((T, hkv, d), dtype=dt, pin_memory=True)
                h.copy_(x)
                lst.append(h)
            for lst, x in ((self.ka_host, st.k_pic[l]), (self.va_host, st.v_pic[l])):
                h = torch.empty((anchor_slots.size, hkv, d), dtype=dt, pin_memory=True)
                h.copy_(x.index_select(0, a_rows))
                lst.append(h)
        torch.cuda.synchronize()
        # probe slots index the compact anchor block (query slots stay -1)
        compact = np.full(p.probe_src.size, -1, np.int32)
        compact[anchor_slots] = np.arange(anchor_slots.size, dtype=np.int32)
        self.probe_src_compact = torch.from_numpy(compact).to(dev)
        self.stage_k = [torch.empty((T, hkv, d), dtype=dt, device=dev) for _ in range(self.n_slots)]
        self.stage_v = [torch.empty((T, hkv, d), dtype=dt, device=dev) for _ in range(self.n_slots)]
        self.copy_stream = torch.cuda.Stream(device=dev)
        # the order in which the compute asks for caches: (layer, full?)
        lmax = max(sw.critical_layers)
        self.order = [(l, l in sw.critical_layers) for l in range(lmax + 1)]
        self.order += [(l, True) for l in range(sw.n_layers) if l not in sw.critical_layers]
        self.bytes = sum((T if full else anchor_slots.size) * hkv * d * 2 * st.k_pic[0].element_size()
                         for _, full in self.order)

    def free_device_pic(self):
        """Drop the device-resident caches (the pipeline then holds the only device copies)."""
        st = self.st
        st.k_pic = [None] * len(st.k_pic)
        st.v_pic = [None] * len(st.v_pic)
        torch.cuda.empty_cache()

    def _issue(self, i):
        if i >= len(self.order):
            return
        l, full = self.order[i]
        slot = i % self.n_slots
        with torch.cuda.stream(self.copy_stream):
            if self.slot_free[slot] is not None:
                self.copy_stream.wait_event(self.slot_free[slot])
            src_k = self.k_host[l] if full else self.ka_host[l]
            src_v = self.v_host[l] if full else self.va_host[l]
            n = src_k.shape[0]
            self.stage_k[slot][:n].copy_(src_k, non_blocking=True)
            self.stage_v[slot][:n].copy_(src_v, non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(self.copy_stream)
            self.copied[i] = ev

    def begin(self):
        """Enqueue the first copies, one per slot (call before select())."""
        self.next = 0
        self.copied = {}
        self.slot_free = [None] * self.n_slots
        for i in range(self.n_slots):
            self._issue(i)
        return self

    def get(self, l, full):
        i = self.next
        assert self.order[i] == (l, full), (self.order[i], l, full)
        torch.cuda.current_stream().wait_event(self.copied[i])
        slot = i % self.n_slots
        return self.stage_k[slot], self.stage_v[slot], (self.st.probe_src if full else self.probe_src_compact)

    def release(self, l):
        i = self.next
        slot = i % self.n_slots
        ev = torch.cuda.Event()
        ev.record(torch.cuda.current_stream())
        self.slot_free[slot] = ev
        self.next = i + 1
        self._issue(i + self.n_slots)

    def copy_only(self):
        """The copy sequence alone, back to back on the copy stream (no compute), for
        timing the loads; the current stream waits for the last one."""
        with torch.cuda.stream(self.copy_stream):
            for i, (l, full) in enumerate(self.order):
                src_k = self.k_host[l] if full else self.ka_host[l]
                src_v = self.v_host[l] if full else self.va_host[l]
                n = src_k.shape[0]
                self.stage_k[i % self.n_slots][:n].copy_(src_k, non_blocking=True)
                self.stage_v[i % self.n_slots][:n].copy_(src_v, non_blocking=True)
        torch.cuda.current_stream().wait_stream(self.copy_stream)
