"""libqcf loads, exports every entry point that include/qcf.h declares, and
rejects bad host arguments before launching anything (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2606_05875_amd import qcf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qcf.h")
OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
A = 0x10000          # a fake, 256-byte aligned address (never dereferenced: calls fail validation)
MIS = 0x10004        # misaligned
F32, BF16 = 0, 1


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    out = {}
    for m in re.finditer(r"\b(?:qcf_status|size_t|int64_t|int|const char\*)\s+(qcf_\w+)\s*\(([^;]*?)\)\s*;", text, re.S):
        args = m.group(2).strip()
        out[m.group(1)] = 0 if args in ("", "void") else args.count(",") + 1
    return out


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(qcf.lib_path()):
        from paper_2606_05875_amd.build import build
        build(verbose=False)
    return qcf.lib()


def test_every_declared_symbol_is_exported(L):
    decl = _declared()
    assert set(decl) == {"qcf_version", "qcf_status_string", "qcf_recommended_row_stride",
                         "qcf_rerope", "qcf_assemble",
                         "qcf_gather_rows",
                         "qcf_scatter_kv", "qcf_probe_scores_workspace_size", "qcf_probe_scores",
                         "qcf_rope_table", "qcf_probe_scores_pic", "qcf_select_topk",
                         "qcf_probe_scores_select", "qcf_probe_scores_select_noalloc",
                         "qcf_sparse_prefill_attn_workspace_size", "qcf_sparse_prefill_attn_rope",
                         "qcf_sparse_prefill_attn", "qcf_mfma_loop"}
    for name, nargs in decl.items():
        assert hasattr(L, name), name
        assert name in qcf.EXPORTS
        assert len(qcf.EXPORTS[name][1]) == nargs, name


def test_version_and_status_strings(L):
    assert L.qcf_version() == 102
    for code in range(5):
        assert L.qcf_status_string(code)
    assert L.qcf_status_string(0) == b"ok"


def test_rerope_validation(L):
    s = None
    r = lambda ko=A, ki=A, vo=None, vi=None, dt=BF16, n=10, d=128, stride=1024, theta=1e4, nseg=1, \
        istride=1024: L.qcf_rerope(ko, ki, vo, vi, dt, n, n, 8, d, stride, istride, nseg, A, A, A, None,
                                   10, theta, s)
    assert r(ko=None, ki=None) == INVALID                 # null tensors with work to do
    assert r(d=96) == UNSUPPORTED
    assert r(dt=7) == UNSUPPORTED
    assert r(stride=512) == INVALID                       # row stride below H_kv * d
    assert r(stride=1028) == INVALID                      # not a 16-byte multiple
    assert r(istride=1000) == INVALID                     # input stride below H_kv * d
    assert r(stride=1152) == INVALID                      # in place with different strides
    assert r(ko=MIS) == INVALID                           # misaligned base
    assert r(theta=0.0) == INVALID
    assert r(n=-1) == INVALID
    assert r(vo=A) == INVALID                             # v_out without v_in
    assert r(vo=A, vi=MIS) == INVALID
    assert r(nseg=70000) == UNSUPPORTED
    # nothing to do: OK without touching the device
    assert L.qcf_rerope(None, None, None, None, BF16, 0, 0, 8, 128, 1024, 1024, 0, None, None, None,
                        None, 0, 1e4, s) == OK


def test_assemble_validation(L):
    def a(**kw):
        g = kw.get
        return [g("kc", A), A, 100, g("stride", 1024), g("kp", A), A, 100, g("pstride", 1024),
                g("nseg", 2), A, A, A, None, 50, g("qn", A), A, A, 100, g("nq", 4), A, A, None,
                g("slot", None), g("qu", A), g("pk", A), A, g("np_", 8), g("qstride", 1024), A, A,
                g("dt", BF16), g("hq", 32), 8, g("d", 128), g("theta", 1e4), None]
    assert L.qcf_assemble(*a(dt=7)) == UNSUPPORTED
    assert L.qcf_assemble(*a(d=96)) == UNSUPPORTED
    assert L.qcf_assemble(*a(hq=36)) == INVALID
    assert L.qcf_assemble(*a(stride=1000)) == INVALID
    assert L.qcf_assemble(*a(pstride=1000)) == INVALID
    assert L.qcf_assemble(*a(qstride=1028)) == INVALID
    assert L.qcf_assemble(*a(theta=0.0)) == INVALID
    assert L.qcf_assemble(*a(kc=None)) == INVALID                 # cache written by segments
    assert L.qcf_assemble(*a(kp=MIS)) == INVALID
    assert L.qcf_assemble(*a(qu=None)) == INVALID                 # query rows need q_u
    assert L.qcf_assemble(*a(pk=None)) == INVALID                 # probe slots to fill
    assert L.qcf_assemble(*a(nq=-1)) == INVALID
    # nothing to do: every pointer may be null
    assert L.qcf_assemble(None, None, 0, 1024, None, None, 0, 1024, 0, None, None, None, None, 0,
                          None, None, None, 0, 0, None, None, None, None, None, None, None, 0, 1024,
                          None, None, BF16, 32, 8, 128, 1e4, None) == OK


def test_recommended_row_stride(L):
    assert L.qcf_recommended_row_stride(8, 128) == 9 * 128      # even: one slice of padding
    assert L.qcf_recommended_row_stride(2, 64) == 3 * 64
    assert L.qcf_recommended_row_stride(1, 128) == 128          # odd: dense rows
    assert L.qcf_recommended_row_stride(5, 64) == 5 * 64
    assert L.qcf_recommended_row_stride(0, 128) == 0
    assert L.qcf_recommended_row_stride(8, 96) == 0
    assert qcf.qcf_recommended_row_stride(8, 128) == 1152


def test_gather_validation(L):
    assert L.qcf_gather_rows(A, A, A, 4, 4, 24, 32, 32, None) == INVALID     # row bytes % 16
    assert L.qcf_gather_rows(A, A, A, 4, 4, 64, 32, 64, None) == INVALID     # row > stride
    assert L.qcf_gather_rows(None, A, A, 4, 4, 32, 32, 32, None) == INVALID
    assert L.qcf_gather_rows(None, None, None, 0, 0, 32, 32, 32, None) == OK


def test_scatter_validation(L):
    args = lambda hq, hkv, d, **kw: [kw.get("kc", A), A, 100, kw.get("stride", hkv * d), A, A,
                                    kw.get("qn", A), kw.get("qo", A), 100, kw.get("src", None), BF16,
                                    kw.get("n", 5), A, A, hq, hkv, d, 1e4, None]
    assert L.qcf_scatter_kv(*args(32, 8, 96)) == UNSUPPORTED
    assert L.qcf_scatter_kv(*args(30, 8, 128)) == INVALID                     # H_q % H_kv
    assert L.qcf_scatter_kv(*args(24, 8, 128)) == UNSUPPORTED                 # group 3
    assert L.qcf_scatter_kv(*args(64, 1, 128)) == UNSUPPORTED                 # group 64 > 32
    assert L.qcf_scatter_kv(*args(32, 8, 128, kc=None)) == INVALID
    assert L.qcf_scatter_kv(*args(32, 8, 128, qn=None)) == INVALID            # q_out without q_new
    assert L.qcf_scatter_kv(*args(32, 8, 128, src=A)) == INVALID              # in-place q with src_idx
    assert L.qcf_scatter_kv(*args(32, 8, 128, stride=8 * 128 + 4)) == INVALID
    assert L.qcf_scatter_kv(*args(32, 8, 128, n=0, kc=None)) == OK


def test_probe_scores_validation_and_workspace(L):
    need = L.qcf_probe_scores_workspace_size(2, 64, 5120, 32, 8, 128)
    assert need > 0 and need % 256 == 0
    assert L.qcf_probe_scores_workspace_size(2, 64, 5120, 32, 8, 96) == 0
    base = lambda **kw: [A, 0, A, 128, A, 10368, kw.get("stride", 1024), BF16, 2, A, A, A, 64, 5120,
                         32, 8, kw.get("d", 128), kw.get("scale", 0.088), kw.get("ws", A),
                         kw.get("wsb", need), None]
    assert L.qcf_probe_scores(*base(wsb=need - 1)) == WORKSPACE
    assert L.qcf_probe_scores(*base(ws=None)) == WORKSPACE
    assert L.qcf_probe_scores(*base(ws=A + 16)) == WORKSPACE                   # not 256-aligned
    assert L.qcf_probe_scores(*base(d=96)) == UNSUPPORTED
    assert L.qcf_probe_scores(*base(scale=0.0)) == INVALID
    assert L.qcf_probe_scores(*base(stride=1000)) == INVALID


def test_rope_table_and_fused_scores_validation(L):
    assert L.qcf_rope_table(A, A, -1, 128, 1e4, None) == INVALID
    assert L.qcf_rope_table(A, A, 10, 96, 1e4, None) == UNSUPPORTED
    assert L.qcf_rope_table(A, A, 10, 128, 0.0, None) == INVALID
    assert L.qcf_rope_table(None, A, 10, 128, 1e4, None) == INVALID
    assert L.qcf_rope_table(MIS, A, 10, 128, 1e4, None) == INVALID               # table not 16-aligned
    assert L.qcf_rope_table(None, None, 0, 128, 1e4, None) == OK                 # empty: nothing launched
    need = L.qcf_probe_scores_workspace_size(2, 64, 5120, 32, 8, 128)
    base = lambda **kw: [A, 0, A, 128, A, 10368, kw.get("stride", 1024), kw.get("rot", A),
                         kw.get("tab", A), kw.get("n_rot", 20), BF16, 2, A, A, A, 64, 5120, 32, 8,
                         kw.get("d", 128), 0.088, A, kw.get("wsb", need), None]
    assert L.qcf_probe_scores_pic(*base(rot=None)) == INVALID
    assert L.qcf_probe_scores_pic(*base(tab=None)) == INVALID
    assert L.qcf_probe_scores_pic(*base(tab=MIS)) == INVALID
    assert L.qcf_probe_scores_pic(*base(n_rot=0)) == INVALID
    assert L.qcf_probe_scores_pic(*base(n_rot=-1)) == INVALID
    assert L.qcf_probe_scores_pic(*base(d=96)) == UNSUPPORTED
    assert L.qcf_probe_scores_pic(*base(stride=1000)) == INVALID
    assert L.qcf_probe_scores_pic(*base(wsb=need - 1)) == WORKSPACE


def test_scores_select_validation(L):
    need = L.qcf_probe_scores_workspace_size(2, 64, 5120, 32, 8, 128)
    base = lambda **kw: [A, 0, A, 128, A, 10368, 1024, BF16, 2, A, A, A, 64, 5120, 32, 8,
                         kw.get("d", 128), 0.088, kw.get("out", A), None, kw.get("n_out", 300),
                         kw.get("n_seg", 20), A, A, A, A, kw.get("req", A), kw.get("msl", 512),
                         A, kw.get("wsb", need), None]
    assert L.qcf_probe_scores_select(*base(out=None)) == INVALID
    assert L.qcf_probe_scores_select(*base(out=MIS + 1)) == INVALID
    assert L.qcf_probe_scores_select(*base(req=None)) == INVALID
    assert L.qcf_probe_scores_select(*base(n_out=-1)) == INVALID
    assert L.qcf_probe_scores_select(*base(msl=-1)) == INVALID
    assert L.qcf_probe_scores_select(*base(d=96)) == UNSUPPORTED
    assert L.qcf_probe_scores_select(*base(wsb=need - 1)) == WORKSPACE
    # no segments: the scores' own checks alone apply
    assert L.qcf_probe_scores_select(*base(n_seg=0, out=None, req=None, wsb=need - 1)) == WORKSPACE


def test_scores_select_noalloc_rejects_oversize_shapes(L):
    # a shape whose scratch need exceeds the fixed array is refused before anything runs
    big = L.qcf_probe_scores_workspace_size(64, 128, 65536, 64, 8, 128)
    assert big > 48 << 20
    args = [A, 0, A, 64 * 128, A, 64 * 65664, 1024, BF16, 64, A, A, A, 128, 65536, 64, 8, 128, 0.088,
            A, None, 300, 20, A, A, A, A, A, 512, None]
    assert L.qcf_probe_scores_select_noalloc(*args) == WORKSPACE


def test_topk_and_attn_validation(L):
    assert L.qcf_select_topk(None, None, 10, A, 100, 2, A, A, A, A, None, 64, None) == INVALID
    assert L.qcf_select_topk(A, None, 10, A, -1, 2, A, A, A, A, None, 64, None) == INVALID
    assert L.qcf_select_topk(None, None, 0, None, 0, 0, None, None, None, None, None, 0, None) == OK
    a = lambda **kw: [A, None, A, A, kw.get("n", 10), A, A, A, 100, kw.get("stride", 1024), A, None,
                      kw.get("dt", BF16), 1, 10, 100, kw.get("hq", 32), 8, 128, 0.088, None, 0, None]
    assert L.qcf_sparse_prefill_attn(*a(dt=3)) == UNSUPPORTED
    r = lambda **kw: [A, None, A, kw.get("src", A), kw.get("nraw", 10), A, 10, A, A, A, 100, 1024, A,
                      kw.get("tab", A), kw.get("ntab", 100), kw.get("dt", BF16), 1, 10, 100, 32, 8, 128,
                      0.088, None, 0, None]
    assert L.qcf_sparse_prefill_attn_rope(*r(tab=None)) == INVALID
    assert L.qcf_sparse_prefill_attn_rope(*r(ntab=0)) == INVALID
    assert L.qcf_sparse_prefill_attn_rope(*r(src=MIS + 1)) == INVALID
    assert L.qcf_sparse_prefill_attn_rope(*r(src=None, nraw=9)) == INVALID
    assert L.qcf_sparse_prefill_attn_rope(*r(dt=F32)) == UNSUPPORTED
    assert L.qcf_sparse_prefill_attn_rope(*r(tab=MIS)) == INVALID
    assert L.qcf_sparse_prefill_attn(*a(hq=36)) == INVALID
    assert L.qcf_sparse_prefill_attn(*a(stride=1000)) == INVALID
    assert L.qcf_sparse_prefill_attn(*a(n=-2)) == INVALID
    assert L.qcf_sparse_prefill_attn_workspace_size(1, 10, 100, 32, 8, 128, BF16) >= 0


def test_mfma_loop_validation(L):
    """The matrix-core yardstick rejects missing buffers and too few blocks before launching."""
    P = ctypes.c_void_p
    buf = P(16)
    assert L.qcf_mfma_loop(None, 1 << 20, buf, 512 * 256, buf, 512, 10, None) == 1
    assert L.qcf_mfma_loop(buf, 8, buf, 512 * 256, buf, 512, 10, None) == 1      # too few operands
    assert L.qcf_mfma_loop(buf, 1 << 20, buf, 100, buf, 512, 10, None) == 1      # sink too small
    assert L.qcf_mfma_loop(buf, 1 << 20, buf, 4 * 256, buf, 4, 10, None) == 1     # fewer than 8 blocks
    assert L.qcf_mfma_loop(buf, 1 << 20, buf, 512 * 256, buf, 512, 0, None) == 1  # no rounds
