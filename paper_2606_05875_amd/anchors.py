"""Offline per-chunk anchor sets A_i = TopK(G_i, ceil(r_a |c_i|)) (Section 3.3.1, eq. anchor_set).

Two of the paper's ranking rules that need no language model:
  * Sink  -- the first positions of every chunk;
  * Knorm -- the positions whose stored keys have the smallest L2 norm (mean over
             the layers and KV heads of the per-head norm).
The Knorm scores are a plain reduction over the stored caches (torch, offline);
the per-chunk selection is the library's segmented top-k (qcf_select_topk),
with equal scores to the lower position and each chunk's anchors ascending.
"""
from __future__ import annotations

import numpy as np
import torch

from . import qcf

__all__ = ["anchor_count", "anchors_sink", "anchors_knorm"]


def anchor_count(n, ra_bp):
    """ceil(r_a * n) with r_a in basis points."""
    return (int(ra_bp) * int(n) + 9999) // 10000


def anchors_sink(seg_len, ra_bp):
    return [np.arange(anchor_count(n, ra_bp), dtype=np.int32) for n in seg_len]


def anchors_knorm(k_pic, seg_start, seg_len, ra_bp, device="cuda"):
    """k_pic: per-layer device caches [T, H_kv, d] (rows may be padded)."""
    acc = None
    for k in k_pic:
        nrm = torch.linalg.vector_norm(k.float(), dim=-1).mean(dim=-1)   # [T]
        acc = nrm if acc is None else acc + nrm
    score = (-(acc / len(k_pic))).contiguous()
    seg_start = np.asarray(seg_start, np.int64)
    seg_len = np.asarray(seg_len, np.int64)
    seg_k = np.array([anchor_count(n, ra_bp) for n in seg_len], np.int32)
    out_start = np.concatenate([[0], np.cumsum(seg_k)[:-1]]).astype(np.int32)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)
    rows = torch.empty(int(seg_k.sum()), dtype=torch.int32, device=device)
    qcf.qcf_select_topk(rows, score, t(seg_start), t(seg_len), t(seg_k), t(out_start),
                        int(seg_len.max()) if seg_len.size else 0)
    r = rows.cpu().numpy()
    return [r[o:o + k] - a for o, k, a in zip(out_start, seg_k, seg_start)]
