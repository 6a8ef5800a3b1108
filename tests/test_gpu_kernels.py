"""Per-kernel parity of libqcf against the CPU oracle on seeded synthetic inputs.

Every input is drawn here (seeded) and handed to both sides; the oracle never
sees a GPU output.  Sizes span several tiles and end in ragged tails.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import qcfuse as Q
from paper_2606_05875_amd import qcf
from paper_2606_05875_amd.workloads import round_to_bf16
from parity import assert_close, assert_scores, assert_ulp

pytestmark = pytest.mark.gpu
DT = {"bf16": torch.bfloat16, "f32": torch.float32}


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t.to(dtype) if dtype is not None else t


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def padded(a, pad, dtype):
    """[rows, heads, d] device copy of a whose rows are `pad` elements longer than dense."""
    rows = a.shape[0]
    width = int(np.prod(a.shape[1:]))
    base = torch.zeros((rows, width + pad), dtype=dtype, device="cuda")
    view = base[:, :width].view(a.shape)
    view.copy_(dev(a, dtype))
    return view


def draw(rng, shape, dtype, scale=1.0):
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    return round_to_bf16(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype,hkv,d", [("bf16", 8, 128), ("bf16", 2, 64), ("f32", 2, 64), ("f32", 4, 128)])
def test_rerope(dtype, hkv, d):
    say("rerope", dtype, hkv, d)
    rng = np.random.default_rng(1)
    lens = np.array([513, 1, 37, 1024, 300])
    starts = np.concatenate([[0], np.cumsum(lens + 3)[:-1]])       # gaps between segments
    T = int(starts[-1] + lens[-1] + 5)
    delta = np.array([0, 513, 514, 551, 31000])
    k = draw(rng, (T, hkv, d), dtype)
    v = draw(rng, (T, hkv, d), dtype)
    kt, vt = dev(k, DT[dtype]), dev(v, DT[dtype])
    out = torch.full_like(kt, 7.0)
    vout = torch.full_like(vt, 7.0)
    i32 = lambda a: dev(np.asarray(a, np.int32))
    qcf.qcf_rerope(out, kt, i32(starts), i32(lens), i32(delta), int(lens.max()), 5e5, v_out=vout, v_in=vt)
    want = Q.rerope(k, starts, lens, delta, 5e5, dtype)
    inside = np.zeros(T, bool)
    for a, n in zip(starts, lens):
        inside[a:a + n] = True
    got = host(out)
    assert_close(got[inside], want[inside], dtype, "rerope")
    assert_ulp(got[inside], want[inside], dtype, "rerope")
    assert np.all(got[~inside] == 7.0)                                # untouched rows
    np.testing.assert_array_equal(host(vout)[inside], v[inside])     # values stitched unchanged
    assert np.all(host(vout)[~inside] == 7.0)
    # in place gives the same bits
    qcf.qcf_rerope(kt, kt, i32(starts), i32(lens), i32(delta), int(lens.max()), 5e5)
    m = torch.from_numpy(inside).cuda()
    assert torch.equal(kt[m], out[m])


def test_rerope_from_chunk_store():
    # chunks stored in a separate pool, in another order; stitched into the request cache
    say("rerope chunk store")
    rng = np.random.default_rng(11)
    hkv, d = 8, 128
    store_lens = np.array([300, 512, 77, 512])
    store_start = np.concatenate([[0], np.cumsum(store_lens)[:-1]])
    pool_k = draw(rng, (int(store_lens.sum()), hkv, d), "bf16")
    pool_v = draw(rng, (int(store_lens.sum()), hkv, d), "bf16")
    order = np.array([3, 0, 2])                                       # request = chunks 3, 0, 2
    lens = store_lens[order]
    seg_start = np.concatenate([[0], np.cumsum(lens)[:-1]])
    T = int(lens.sum()) + 16                                          # + query slots
    i32 = lambda a: dev(np.asarray(a, np.int32))
    # request cache with padded rows (stride (H_kv + 1) * d), store dense
    ko = padded(np.zeros((T, hkv, d), np.float32), d, torch.bfloat16)
    vo = padded(np.zeros((T, hkv, d), np.float32), d, torch.bfloat16)
    qcf.qcf_rerope(ko, dev(pool_k, torch.bfloat16), i32(seg_start), i32(lens), i32(seg_start), 512, 5e5,
                   v_out=vo, v_in=dev(pool_v, torch.bfloat16), src_start=i32(store_start[order]))
    gk, gv = host(ko), host(vo)
    for s_, c in enumerate(order):
        a, n, src = int(seg_start[s_]), int(lens[s_]), int(store_start[c])
        want = Q.rerope(pool_k[src:src + n], [0], [n], [a], 5e5, "bf16")
        assert_ulp(gk[a:a + n], want, "bf16", f"chunk {c}")
        np.testing.assert_array_equal(gv[a:a + n], pool_v[src:src + n])
    assert np.all(gk[-16:] == 0)
    assert not ko._base[:, hkv * d:].any() and not vo._base[:, hkv * d:].any()   # padding untouched


@pytest.mark.parametrize("dtype,hq,hkv,d,pads", [("bf16", 32, 8, 128, (0, 0, 0)), ("bf16", 16, 2, 64, (0, 0, 0)),
                                                 ("f32", 8, 4, 128, (0, 0, 0)),
                                                 ("bf16", 32, 8, 128, (128, 8, 136)),
                                                 ("f32", 8, 2, 64, (4, 64, 0))])
def test_assemble(dtype, hq, hkv, d, pads):
    """One launch: chunk remap + value stitch, query rows, probe buffer (anchors from the store);
    the cache, the chunk store and the probe buffer may each have their own padded row stride."""
    say("assemble", dtype, hq, hkv, d, pads)
    rng = np.random.default_rng(21)
    theta = 5e5
    store_lens = np.array([513, 1, 300, 77, 1024])
    store_start = np.concatenate([[0], np.cumsum(store_lens + 2)[:-1]])   # gaps in the store
    S_rows = int(store_start[-1] + store_lens[-1] + 3)
    pool_k, pool_v = draw(rng, (S_rows, hkv, d), dtype), draw(rng, (S_rows, hkv, d), dtype)
    order = np.array([4, 1, 0, 3])
    lens = store_lens[order]
    seg_start = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    N = int(lens.sum())
    nq = 37
    T = N + nq + 5
    src_start = store_start[order]
    delta = seg_start.copy()                 # chunk stored at local positions 0..n-1
    # fresh projections for every cache row (only the query rows are read)
    kn, vn = draw(rng, (T, hkv, d), dtype), draw(rng, (T, hkv, d), dtype)
    qn = draw(rng, (T, hq, d), dtype, 3.0)
    qrow = np.arange(N, N + nq)
    qpos = qrow.copy()
    # probe buffer: 3 anchors of each chunk (1 for the 1-row chunk), then the query rows
    anc_src, anc_delta, anc_req = [], [], []
    for s_ in range(len(order)):
        loc = np.sort(rng.choice(lens[s_], min(3, lens[s_]), replace=False))
        anc_src.append(src_start[s_] + loc)
        anc_delta.append(np.full(loc.size, delta[s_]))
        anc_req.append(seg_start[s_] + loc)
    anc_src, anc_delta, anc_req = map(np.concatenate, (anc_src, anc_delta, anc_req))
    na = anc_src.size
    probe_src = np.concatenate([anc_src, np.full(nq, -1)])
    probe_delta = np.concatenate([anc_delta, np.zeros(nq)])
    slot = na + np.arange(nq)
    t = DT[dtype]
    i32 = lambda a: dev(np.asarray(a, np.int32))
    pc, pp, pq = pads
    kc = padded(np.full((T, hkv, d), 7.0, np.float32), pc, t)
    vc = padded(np.full((T, hkv, d), 7.0, np.float32), pc, t)
    qu = torch.empty((nq, hq, d), dtype=t, device="cuda")
    pk = padded(np.zeros((na + nq, hkv, d), np.float32), pq, t)
    pv = padded(np.zeros((na + nq, hkv, d), np.float32), pq, t)
    qcf.qcf_assemble(kc, vc, padded(pool_k, pp, t), padded(pool_v, pp, t), i32(seg_start), i32(lens), i32(delta),
                     int(lens.max()), dev(qn, t), dev(kn, t), dev(vn, t), i32(qrow), i32(qpos), qu, pk, pv,
                     i32(probe_src), i32(probe_delta), theta, src_start=i32(src_start),
                     query_src=i32(qrow), query_slot=i32(slot))
    gk, gv = host(kc), host(vc)
    for s_ in range(len(order)):
        a, n, src = int(seg_start[s_]), int(lens[s_]), int(src_start[s_])
        want = Q.rerope(pool_k[src:src + n], [0], [n], [a], theta, dtype)
        assert_ulp(gk[a:a + n], want, dtype, f"chunk {s_}")
        np.testing.assert_array_equal(gv[a:a + n], pool_v[src:src + n])
    wk = Q.round_storage(Q.rope(kn[qrow], qpos, theta), dtype)
    wq = Q.round_storage(Q.rope(qn[qrow], qpos, theta), dtype)
    assert_ulp(gk[qrow], wk, dtype, "query K")
    np.testing.assert_array_equal(gv[qrow], vn[qrow])
    assert_ulp(host(qu), wq, dtype, "q_u")
    assert np.all(gk[N + nq:] == 7.0) and np.all(gv[N + nq:] == 7.0)     # untouched rows
    # probe buffer: anchors = re-positioned stored rows, equal to their cache rows; then the query
    gpk, gpv = host(pk), host(pv)
    for j in range(na):
        wj = Q.rerope(pool_k[anc_src[j]:anc_src[j] + 1], [0], [1], [anc_delta[j]], theta, dtype)
        assert_ulp(gpk[j:j + 1], wj, dtype, f"anchor {j}")
    np.testing.assert_array_equal(gpk[:na], gk[anc_req])                    # same bits as the cache rows
    np.testing.assert_array_equal(gpv[:na], pool_v[anc_src])
    np.testing.assert_array_equal(gpk[na:], gk[qrow])
    np.testing.assert_array_equal(gpv[na:], gv[qrow])


def test_gather_rows_exact():
    say("gather")
    rng = np.random.default_rng(2)
    src = rng.standard_normal((1000, 8, 128)).astype(np.float32)
    idx = rng.integers(0, 1000, 777).astype(np.int32)
    s = dev(src, torch.bfloat16)
    d = torch.empty((777, 8, 128), dtype=torch.bfloat16, device="cuda")
    qcf.qcf_gather_rows(d, s, dev(idx))
    assert torch.equal(d, s[torch.from_numpy(idx).long().cuda()])
    e = torch.empty((0, 8, 128), dtype=torch.bfloat16, device="cuda")
    qcf.qcf_gather_rows(e, s, dev(np.zeros(0, np.int32)))


@pytest.mark.parametrize("dtype,hq,hkv,d", [("bf16", 32, 8, 128), ("bf16", 8, 8, 64), ("f32", 8, 2, 64)])
def test_scatter_kv(dtype, hq, hkv, d):
    say("scatter", dtype, hq, hkv, d)
    rng = np.random.default_rng(3)
    T, S = 2000, 1500
    kc = draw(rng, (T, hkv, d), dtype)
    vc = draw(rng, (T, hkv, d), dtype)
    kn, vn, qn = draw(rng, (S, hkv, d), dtype), draw(rng, (S, hkv, d), dtype), draw(rng, (S, hq, d), dtype, 3.0)
    rows = np.sort(rng.choice(T, 611, replace=False)).astype(np.int32)
    src = rng.choice(S, 611, replace=False).astype(np.int32)
    pos = rng.integers(0, 33000, 611).astype(np.int32)
    K, V = dev(kc, DT[dtype]), dev(vc, DT[dtype])
    qo = torch.empty((611, hq, d), dtype=DT[dtype], device="cuda")
    qcf.qcf_scatter_kv(K, V, dev(kn, DT[dtype]), dev(vn, DT[dtype]), dev(rows), dev(pos), 1e6,
                       q_new=dev(qn, DT[dtype]), q_out=qo, src_idx=dev(src))
    gk, gv = host(K), host(V)
    wk = Q.round_storage(Q.rope(kn[src], pos, 1e6), dtype)
    wq = Q.round_storage(Q.rope(qn[src], pos, 1e6), dtype)
    assert_close(gk[rows], wk, dtype, "scattered K")
    assert_ulp(gk[rows], wk, dtype, "scattered K")
    assert_ulp(host(qo), wq, dtype, "rotated Q")        # |q| ~ 10: an absolute bound does not apply
    np.testing.assert_array_equal(gv[rows], vn[src])
    keep = np.setdiff1d(np.arange(T), rows)
    np.testing.assert_array_equal(gk[keep], kc[keep])
    np.testing.assert_array_equal(gv[keep], vc[keep])


@pytest.mark.parametrize("lens,ks", [
    ([512, 511, 1, 1024, 700], [153, 0, 1, 1024, 699]),      # per chunk, 256 x 4 slots
    ([4096, 3000, 17], [1228, 3000, 16]),                     # 256 x 16
    ([8192, 8191], [2457, 1]),                                # 512 x 16
    ([16384, 9000], [4915, 8999]),                            # 1024 x 16
    ([20000], [6000]),                                        # global top-k of one request, 1024 x 32
    ([32768, 31000], [9830, 31000]),                          # 1024 x 32, k = n
    ([65536, 40000], [19660, 1]),                             # 1024 x 64
    ([70000, 300], [21000, 90]),                              # longer than the register path
])
def test_select_topk_exact(lens, ks):
    say("topk", lens, ks)
    rng = np.random.default_rng(4)
    n = sum(lens) + 10
    s = rng.random(n).astype(np.float32)
    s[rng.integers(0, n, n // 3)] = 0.25          # many ties
    s[rng.integers(0, n, n // 10)] = 0.0
    s[rng.integers(0, n, n // 10)] = -0.0
    s[rng.integers(0, n, 50)] = 1e-38
    starts = np.concatenate([[5], 5 + np.cumsum(lens)[:-1]]).astype(np.int32)
    out_start = np.concatenate([[0], np.cumsum(ks)[:-1]]).astype(np.int32)
    total = int(sum(ks))
    out = torch.full((total,), -7, dtype=torch.int32, device="cuda")
    pos = torch.full((total,), -7, dtype=torch.int32, device="cuda")
    base = np.full(len(lens), 3, np.int32)
    qcf.qcf_select_topk(out, dev(s), dev(starts), dev(np.array(lens, np.int32)), dev(np.array(ks, np.int32)),
                        dev(out_start), max(lens), out_pos=pos, pos_base=dev(base))
    got = out.cpu().numpy()
    want = np.concatenate([a + Q.select_topk(s[a:a + n_], k) for a, n_, k in zip(starts, lens, ks)])
    np.testing.assert_array_equal(got, want)
    np.testing.assert_array_equal(pos.cpu().numpy(), want - 3)


@pytest.mark.parametrize("n,k", [(32768, 9830), (65536, 1), (5000, 4999)])
def test_select_topk_all_equal(n, k):
    """Every score equal: the k lowest rows, in order (the tie rule alone decides)."""
    say("topk all equal", n, k)
    s = torch.full((n,), 0.5, device="cuda")
    out = torch.full((k,), -7, dtype=torch.int32, device="cuda")
    one = lambda v: dev(np.array([v], np.int32))
    qcf.qcf_select_topk(out, s, one(0), one(n), one(k), one(0), n)
    np.testing.assert_array_equal(out.cpu().numpy(), np.arange(k))


@pytest.mark.parametrize("dtype,nqs,ctxs,hq,hkv,d", [
    ("bf16", [64], [5120], 32, 8, 128),
    ("bf16", [17, 1, 128], [700, 3000, 129], 32, 8, 128),
    ("bf16", [9], [1000], 8, 8, 64),
    ("bf16", [40], [2500], 64, 8, 128),
    ("bf16", [8, 3], [20000, 9000], 32, 8, 128),      # several 128-key sub-tiles per split
    ("f32", [32], [512], 8, 2, 64),
])
def test_probe_scores(dtype, nqs, ctxs, hq, hkv, d):
    say("probe_scores", dtype, nqs, ctxs, hq, hkv, d)
    rng = np.random.default_rng(5)
    B = len(nqs)
    rows = [c + q for c, q in zip(ctxs, nqs)]
    cu_kv = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    k = draw(rng, (int(cu_kv[-1]), hkv, d), dtype, 1 / math.sqrt(d))
    q = draw(rng, (int(cu_q[-1]), hq, d), dtype, 1.5 * math.sqrt(d))
    sc = torch.full((int(cu_kv[-1]),), -5.0, device="cuda")
    scale = 1 / math.sqrt(d)
    args = (dev(q, DT[dtype]), dev(k, DT[dtype]), dev(cu_q), dev(cu_kv), dev(np.array(ctxs, np.int32)),
            max(nqs), max(ctxs), scale)
    qcf.qcf_probe_scores(sc, *args)
    got = sc.double().cpu().numpy()
    for b in range(B):
        a = int(cu_kv[b])
        want = Q.critical_scores(q[cu_q[b]:cu_q[b + 1]], k[a:a + ctxs[b]], scale, hkv)
        assert_scores(got[a:a + ctxs[b]], want, f"scores request {b}")
        assert np.all(got[a + ctxs[b]:cu_kv[b + 1]] == -5.0)          # query slots untouched
    # accumulate mode adds a second layer's scores; runs are bit-identical
    qcf.qcf_probe_scores(sc, *args, accumulate=True)
    np.testing.assert_array_equal(sc.double().cpu().numpy()[:ctxs[0]], 2 * got[:ctxs[0]])


def test_probe_scores_workspace_reuse_across_shapes():
    """One workspace serves calls of different shapes with results identical to fresh
    workspaces (nothing in it carries over from call to call)."""
    say("probe_scores workspace reuse")
    rng = np.random.default_rng(7)
    hq, hkv, d = 32, 8, 128
    shapes = [([64], [5120]), ([5, 33], [300, 2000]), ([128], [777]), ([64], [5120])]
    big = max(qcf.qcf_probe_scores_workspace_size(len(n), max(n), max(c), hq, hkv, d) for n, c in shapes)
    ws = torch.full((big,), 0x5A, dtype=torch.uint8, device="cuda")      # garbage to start
    for nqs, ctxs in shapes:
        rows = [c + q for c, q in zip(ctxs, nqs)]
        cu_kv = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
        cu_q = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
        k = draw(rng, (int(cu_kv[-1]), hkv, d), "bf16", 1 / math.sqrt(d))
        q = draw(rng, (int(cu_q[-1]), hq, d), "bf16", 1.5 * math.sqrt(d))
        args = (dev(q, torch.bfloat16), dev(k, torch.bfloat16), dev(cu_q), dev(cu_kv),
                dev(np.array(ctxs, np.int32)), max(nqs), max(ctxs), 1 / math.sqrt(d))
        a = torch.zeros(int(cu_kv[-1]), device="cuda")
        b = torch.zeros_like(a)
        qcf.qcf_probe_scores(a, *args, workspace=ws)
        qcf.qcf_probe_scores(b, *args)                       # a fresh workspace
        assert torch.equal(a, b)


def test_rope_table():
    """The table holds float32 roundings of the float64 (cos, sin) of pos * theta^(-2j/d)."""
    say("rope_table")
    pos = np.array([0, 1, 7, 513, 4096, 31000, 123456], np.int32)
    for d, theta in ((128, 1e6), (64, 1e4)):
        tab = torch.empty((pos.size, d // 2, 2), dtype=torch.float32, device="cuda")
        qcf.qcf_rope_table(tab, dev(pos), theta)
        a = Q.rope_angles(pos, d, theta)
        want = np.stack([np.cos(a), np.sin(a)], axis=-1)
        got = tab.cpu().numpy()
        # correctly rounded is within half a float32 step; the last float64 digits of two
        # libm implementations may differ, so one step is allowed
        step = np.abs(np.spacing(want.astype(np.float32))).astype(np.float64)
        assert np.all(np.abs(got - want) <= step), "rope table off by more than one float32 step"
        np.testing.assert_array_equal(got[0], np.stack([np.ones(d // 2), np.zeros(d // 2)], -1))


@pytest.mark.parametrize("dtype,nqs,ctxs,hq,hkv,d,pad", [
    ("bf16", [64], [5120], 32, 8, 128, 128),            # 10 x 512-token chunks, padded rows
    ("bf16", [17, 1, 128], [700, 3000, 129], 32, 8, 128, 0),
    ("bf16", [9], [1000], 8, 8, 64, 8),
    ("bf16", [8, 3], [20000, 9000], 32, 8, 128, 0),     # several key chunks per split
    ("f32", [32], [512], 8, 2, 64, 0),
    ("f32", [5, 7], [300, 170], 8, 4, 128, 4),
])
def test_probe_scores_pic(dtype, nqs, ctxs, hq, hkv, d, pad):
    """Scores over keys re-positioned in registers equal, bit for bit, qcf_rerope followed by
    qcf_probe_scores, and match the oracle's scores of the re-positioned keys."""
    say("probe_scores_pic", dtype, nqs, ctxs, hq, hkv, d, pad)
    rng = np.random.default_rng(11)
    B, theta = len(nqs), 1e6
    rows = [c + q for c, q in zip(ctxs, nqs)]
    cu_kv = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    T = int(cu_kv[-1])
    # ragged chunks tile each request's context; a chunk's offset is its first position
    seg_start, seg_len, seg_delta = [], [], []
    for b in range(B):
        a = 0
        while a < ctxs[b]:
            n = min(ctxs[b] - a, int(rng.integers(1, 700)))
            seg_start.append(int(cu_kv[b]) + a)
            seg_len.append(n)
            seg_delta.append(a)
            a += n
    seg_start, seg_len, seg_delta = (np.array(x, np.int32) for x in (seg_start, seg_len, seg_delta))
    n_seg = seg_start.size
    # table rows in shuffled order, so the per-row indirection is exercised
    perm = rng.permutation(n_seg)
    tab_pos = np.zeros(n_seg, np.int32)
    tab_pos[perm] = seg_delta
    key_rot = np.full(T, 10 ** 6, np.int32)          # query rows: never read as keys
    for s in range(n_seg):
        key_rot[seg_start[s]:seg_start[s] + seg_len[s]] = perm[s]
    k_pic = draw(rng, (T, hkv, d), dtype, 1 / math.sqrt(d))
    q = draw(rng, (int(cu_q[-1]), hq, d), dtype, 1.5 * math.sqrt(d))
    table = torch.empty((n_seg, d // 2, 2), dtype=torch.float32, device="cuda")
    qcf.qcf_rope_table(table, dev(tab_pos), theta)
    kp = padded(k_pic, pad, DT[dtype])
    scale = 1 / math.sqrt(d)
    geo = (dev(cu_q), dev(cu_kv), dev(np.array(ctxs, np.int32)), max(nqs), max(ctxs), scale)
    qd = dev(q, DT[dtype])
    fused = torch.full((T,), -5.0, device="cuda")
    qcf.qcf_probe_scores_pic(fused, qd, kp, dev(key_rot), table, *geo)
    # the unfused path: re-position into a request cache, then score it
    k_req = padded(np.zeros_like(k_pic), pad, DT[dtype])
    qcf.qcf_rerope(k_req, kp, dev(seg_start), dev(seg_len), dev(seg_delta), int(seg_len.max()), theta)
    ref = torch.full((T,), -5.0, device="cuda")
    qcf.qcf_probe_scores(ref, qd, k_req, *geo)
    assert torch.equal(fused, ref), "fused scores differ from re-position + scores"
    got = fused.double().cpu().numpy()
    krep = Q.rerope(k_pic, seg_start, seg_len, seg_delta, theta, dtype)
    for b in range(B):
        a = int(cu_kv[b])
        want = Q.critical_scores(q[cu_q[b]:cu_q[b + 1]], krep[a:a + ctxs[b]], scale, hkv)
        assert_scores(got[a:a + ctxs[b]], want, f"fused scores request {b}")
        assert np.all(got[a + ctxs[b]:cu_kv[b + 1]] == -5.0)          # query slots untouched
    # accumulate mode, as over several critical layers
    qcf.qcf_probe_scores_pic(fused, qd, kp, dev(key_rot), table, *geo, accumulate=True)
    qcf.qcf_probe_scores(ref, qd, k_req, *geo, accumulate=True)
    assert torch.equal(fused, ref)


@pytest.mark.parametrize("dtype,hq,hkv,d,n_kv,n_rows", [
    ("bf16", 32, 8, 128, 5184, 700),
    ("bf16", 64, 8, 128, 3000, 333),
    ("bf16", 8, 8, 64, 1000, 129),
    ("bf16", 32, 2, 128, 777, 50),        # group 16
    ("f32", 8, 2, 64, 544, 184),
])
def test_sparse_attention(dtype, hq, hkv, d, n_kv, n_rows):
    say("attention", dtype, hq, hkv, d, n_kv, n_rows)
    rng = np.random.default_rng(6)
    k = draw(rng, (n_kv, hkv, d), dtype, 1 / math.sqrt(d))
    v = draw(rng, (n_kv, hkv, d), dtype, 1 / math.sqrt(d))
    q = draw(rng, (n_rows, hq, d), dtype, math.sqrt(d))
    pos = np.sort(rng.choice(n_kv, n_rows, replace=False)).astype(np.int32)
    pos[0] = 0                                       # a row that sees exactly one key
    scale = 1 / math.sqrt(d)
    out = torch.empty((n_rows, hq, d), dtype=DT[dtype], device="cuda")
    lse = torch.empty((n_rows, hq), dtype=torch.float32, device="cuda")
    qcf.qcf_sparse_prefill_attn(out, dev(q, DT[dtype]), dev(pos), dev(np.array([0, n_rows], np.int32)),
                                dev(k, DT[dtype]), dev(v, DT[dtype]), dev(np.array([0, n_kv], np.int32)),
                                n_rows, n_kv, scale, lse=lse)
    want = Q.round_storage(Q.attention(q, pos, k, v, np.arange(n_kv), scale, hkv), dtype)
    assert_close(host(out), want, dtype, "attention")
    g = hq // hkv
    np.testing.assert_allclose(host(out)[0], np.repeat(v[0], g, axis=0), atol=1e-6)
    # log-sum-exp of the scaled logits, checked on a few rows
    for r in (0, n_rows // 2, n_rows - 1):
        m = pos[r] + 1
        for h in (0, hq - 1):
            lg = (q[r, h].astype(np.float64) @ k[:m, h // g].astype(np.float64).T) * scale
            want_lse = np.log(np.sum(np.exp(lg - lg.max()))) + lg.max()
            assert abs(float(lse[r, h]) - want_lse) < 2e-3 * max(1.0, abs(want_lse))


def test_attention_explicit_positions_and_batch():
    say("attention explicit positions, batch of 3")
    rng = np.random.default_rng(7)
    hq, hkv, d = 32, 8, 128
    n_kv = [200, 37, 1100]
    n_rows = [64, 1, 40]
    cu_kv = np.concatenate([[0], np.cumsum(n_kv)]).astype(np.int32)
    cu_r = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    k = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    v = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    q = draw(rng, (cu_r[-1], hq, d), "bf16", math.sqrt(d))
    kpos = np.concatenate([np.sort(rng.choice(5000, n, replace=False)) for n in n_kv]).astype(np.int32)
    rpos = np.concatenate([rng.integers(0, 5200, n) for n in n_rows]).astype(np.int32)
    out = torch.empty((cu_r[-1], hq, d), dtype=torch.bfloat16, device="cuda")
    qcf.qcf_sparse_prefill_attn(out, dev(q, torch.bfloat16), dev(rpos), dev(cu_r), dev(k, torch.bfloat16),
                                dev(v, torch.bfloat16), dev(cu_kv), max(n_rows), max(n_kv), 1 / math.sqrt(d),
                                kv_pos=dev(kpos))
    got = host(out)
    for b in range(3):
        a, e, ka, ke = cu_r[b], cu_r[b + 1], cu_kv[b], cu_kv[b + 1]
        want = Q.round_storage(Q.attention(q[a:e], rpos[a:e], k[ka:ke], v[ka:ke], kpos[ka:ke],
                                           1 / math.sqrt(d), hkv), "bf16")
        assert_close(got[a:e], want, "bf16", f"request {b}")


def test_empty_calls():
    say("empty calls")
    z = torch.zeros((0, 8, 128), dtype=torch.bfloat16, device="cuda")
    zi = torch.zeros(0, dtype=torch.int32, device="cuda")
    k = torch.zeros((10, 8, 128), dtype=torch.bfloat16, device="cuda")
    qcf.qcf_scatter_kv(k, k.clone(), z, z, zi, zi, 1e4)
    qcf.qcf_select_topk(zi, torch.zeros(10, device="cuda"), zi, zi, zi, zi, 0)
    qz = torch.zeros((0, 32, 128), dtype=torch.bfloat16, device="cuda")
    qcf.qcf_sparse_prefill_attn(qz, qz, zi, torch.zeros(2, dtype=torch.int32, device="cuda"), k, k,
                                torch.tensor([0, 10], dtype=torch.int32, device="cuda"), 0, 10, 0.1)
    torch.cuda.synchronize()


@pytest.mark.parametrize("hq,hkv,d", [(16, 2, 64), (8, 8, 64), (32, 8, 128)])
def test_attention_plain_grid_every_tile(hq, hkv, d):
    """The plain grid (one block per row tile, each block's two wave groups on their own
    schedules: waves 0-3 multiply a tile's P.V in its own step, waves 4-7 in the next one) at
    head sizes 64 and 128 and group sizes 8, 1 and 4: the first and last row of every row tile
    of a ragged batch against the oracle."""
    say("attention plain grid", hq, hkv, d)
    rng = np.random.default_rng(9)
    g = hq // hkv
    rpb = 256 // g                                   # rows per row tile
    first_tiles = -(-512 // (4 * hkv))             # enough row tiles for the plain grid
    n_rows = [first_tiles * rpb + 5, 9 * rpb, 3 * rpb + 1, rpb - 7]
    n_kv = [r * 3 // 2 + 40 for r in n_rows]
    tiles = (max(n_rows) + rpb - 1) // rpb
    assert tiles * len(n_kv) * hkv >= 384, "the case must take the plain grid"
    cu_kv = np.concatenate([[0], np.cumsum(n_kv)]).astype(np.int32)
    cu_r = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    k = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    v = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    q = draw(rng, (cu_r[-1], hq, d), "bf16", math.sqrt(d))
    rpos = np.concatenate([np.sort(rng.choice(nk, nr, replace=False)) for nk, nr in zip(n_kv, n_rows)])
    rpos = rpos.astype(np.int32)
    out = torch.empty((cu_r[-1], hq, d), dtype=torch.bfloat16, device="cuda")
    scale = 1 / math.sqrt(d)
    qcf.qcf_sparse_prefill_attn(out, dev(q, torch.bfloat16), dev(rpos), dev(cu_r), dev(k, torch.bfloat16),
                                dev(v, torch.bfloat16), dev(cu_kv), max(n_rows), max(n_kv), scale)
    got = host(out)
    for b in range(len(n_kv)):
        a, e, ka, ke = cu_r[b], cu_r[b + 1], cu_kv[b], cu_kv[b + 1]
        firsts = np.arange(a, e, rpb)
        pick = np.unique(np.concatenate([firsts, np.minimum(firsts + rpb - 1, e - 1)]))
        want = Q.round_storage(Q.attention(q[pick], rpos[pick], k[ka:ke], v[ka:ke], np.arange(ke - ka),
                                           scale, hkv), "bf16")
        assert_close(got[pick], want, "bf16", f"request {b}")


@pytest.mark.parametrize("hq,hkv,d", [(64, 8, 128), (16, 2, 128), (128, 16, 128), (64, 8, 64)])
def test_attention_one_request_work_queues(hq, hkv, d):
    """One request with four row tiles per CU (1024 blocks of 32 rows x 8 query heads) takes its
    tiles from the per-XCD work queues (8 KV heads: one per queue; 2: four XCDs per queue; 16:
    two heads per queue).  The same call laid out as a batch of two (the second request empty)
    runs the fixed one-block-per-tile order: every row must match it bit for bit, on two calls
    in a row (the counters are reset by the call itself) and with a dirty workspace; sampled
    rows (the last tile, the first, every 16th) also match the oracle.  Head sizes 128 and 64."""
    rpb = 256 // (hq // hkv)
    n_rows = 4 * 256 * rpb // hkv                    # 1024 blocks: the queue threshold on 256 CUs
    n_kv = n_rows + n_rows // 2
    say("attention work queues", hq, hkv, d, n_rows, n_kv)
    rng = np.random.default_rng(21)
    k = draw(rng, (n_kv, hkv, d), "bf16", 1 / math.sqrt(d))
    v = draw(rng, (n_kv, hkv, d), "bf16", 1 / math.sqrt(d))
    q = draw(rng, (n_rows, hq, d), "bf16", math.sqrt(d))
    rpos = np.sort(rng.choice(n_kv, n_rows, replace=False)).astype(np.int32)
    scale = 1 / math.sqrt(d)
    args = (dev(q, torch.bfloat16), dev(rpos))
    kk, vv = dev(k, torch.bfloat16), dev(v, torch.bfloat16)
    need = qcf.qcf_sparse_prefill_attn_workspace_size(1, n_rows, n_kv, hq, hkv, d, torch.bfloat16)
    ws = torch.full((need,), 0xAB, dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(2):
        out = torch.empty((n_rows, hq, d), dtype=torch.bfloat16, device="cuda")
        qcf.qcf_sparse_prefill_attn(out, *args, dev(np.array([0, n_rows], np.int32)), kk, vv,
                                    dev(np.array([0, n_kv], np.int32)), n_rows, n_kv, scale, workspace=ws)
        outs.append(out)
    ref = torch.empty_like(outs[0])
    qcf.qcf_sparse_prefill_attn(ref, *args, dev(np.array([0, n_rows, n_rows], np.int32)), kk, vv,
                                dev(np.array([0, n_kv, n_kv], np.int32)), n_rows, n_kv, scale)
    torch.cuda.synchronize()
    for out in outs:
        assert torch.equal(out, ref), "work-queue grid differs from the fixed-order grid"
    pick = np.unique(np.concatenate([np.arange(n_rows - rpb, n_rows), np.arange(0, rpb, 7),
                                     np.arange(rpb - 1, n_rows, 16 * rpb)]))
    want = Q.round_storage(Q.attention(q[pick], rpos[pick], k, v, np.arange(n_kv), scale, hkv), "bf16")
    assert_close(host(outs[0])[pick], want, "bf16", "work-queue grid")

    # captured in a graph (the counters are reset by a kernel, not a memset): every replay,
    # with eager work and synchronisations between them, equals the eager result
    cu_r1, cu_k1 = dev(np.array([0, n_rows], np.int32)), dev(np.array([0, n_kv], np.int32))
    gout = torch.empty_like(ref)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        qcf.qcf_sparse_prefill_attn(gout, *args, cu_r1, kk, vv, cu_k1, n_rows, n_kv, scale, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        qcf.qcf_sparse_prefill_attn(gout, *args, cu_r1, kk, vv, cu_k1, n_rows, n_kv, scale, workspace=ws)
    for rep in range(3):
        gout.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(gout, ref), f"graph replay {rep} differs"
        eager = torch.empty_like(ref)
        qcf.qcf_sparse_prefill_attn(eager, *args, cu_r1, kk, vv, cu_k1, n_rows, n_kv, scale, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(eager, ref)


@pytest.mark.parametrize("n_kv,n_rows,plain", [
    ([2500, 2500, 400, 3100, 1200, 64], [700, 700, 90, 650, 0, 64], True),
    ([300, 1200, 50, 1200], [100, 400, 10, 0], False)])
def test_attention_ragged_batch(n_kv, n_rows, plain):
    """A ragged batch on both grids: one block per row tile (many tiles; requests taken longest
    first) and the persistent grid (few tiles; cut tiles merged); equal-length requests, a
    request with no rows and a short one; sampled rows against the oracle."""
    say("attention ragged batch", n_kv, n_rows, "plain" if plain else "persistent")
    rng = np.random.default_rng(8)
    hq, hkv, d = 32, 8, 128
    cu_kv = np.concatenate([[0], np.cumsum(n_kv)]).astype(np.int32)
    cu_r = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    k = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    v = draw(rng, (cu_kv[-1], hkv, d), "bf16", 1 / math.sqrt(d))
    q = draw(rng, (cu_r[-1], hq, d), "bf16", math.sqrt(d))
    rpos = np.concatenate([np.sort(rng.choice(nk, nr, replace=False)) for nk, nr in zip(n_kv, n_rows)])
    rpos = rpos.astype(np.int32)
    # the grid choice: one block per (row tile, request, KV head) from 384 such blocks on
    assert ((max(n_rows) + 63) // 64 * len(n_kv) * hkv >= 384) == plain
    out = torch.empty((cu_r[-1], hq, d), dtype=torch.bfloat16, device="cuda")
    scale = 1 / math.sqrt(d)
    qcf.qcf_sparse_prefill_attn(out, dev(q, torch.bfloat16), dev(rpos), dev(cu_r), dev(k, torch.bfloat16),
                                dev(v, torch.bfloat16), dev(cu_kv), max(n_rows), max(n_kv), scale)
    got = host(out)
    for b in range(len(n_kv)):
        a, e, ka, ke = cu_r[b], cu_r[b + 1], cu_kv[b], cu_kv[b + 1]
        if e == a:
            continue
        pick = np.unique(np.concatenate([[a, e - 1], rng.integers(a, e, 4)]))
        want = Q.round_storage(Q.attention(q[pick], rpos[pick], k[ka:ke], v[ka:ke], np.arange(ke - ka),
                                           scale, hkv), "bf16")
        assert_close(got[pick], want, "bf16", f"request {b}")


def test_mfma_loop_yardstick():
    """The matrix-core loop (a yardstick for the attention, not a step of the method) runs, leaves
    finite sums (random operands) and clock counters that give a clock between 0.5 and 3 GHz on
    each of the eight recording blocks."""
    say("mfma loop")
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 2 * n_cu
    ops = torch.randn(1 << 16, generator=torch.Generator().manual_seed(5)).to(torch.bfloat16).cuda()
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda")
    clocks = torch.zeros(32, dtype=torch.int64, device="cuda")
    qcf.qcf_mfma_loop(ops, sink, clocks, blocks, 200)
    torch.cuda.synchronize()
    assert torch.isfinite(sink).all()
    c = clocks.view(8, 4).cpu().numpy().astype(np.float64)
    assert (c[:, 2] > c[:, 0]).all() and (c[:, 3] > c[:, 1]).all()
    ghz = (c[:, 3] - c[:, 1]) / ((c[:, 2] - c[:, 0]) / 100e6) / 1e9
    assert ((ghz > 0.5) & (ghz < 3.0)).all(), ghz
