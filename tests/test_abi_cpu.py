"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects every invalid call before launching anything
(validation runs on the host, so these calls never reach the device)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2405_13226_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dd_attn.h")

OK, NULL, SHAPE, HEADDIM, DOCLENS, WORKSPACE, ALIGN, ALIAS = range(8)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dd_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libdd_attn.so is not built (python -m paper_2405_13226_amd.build)")
    return _lib.lib()


def test_every_declared_symbol_is_exported(lib):
    names = header_functions()
    assert set(names) == set(_lib.SIGNATURES), names
    raw = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_status_strings(lib):
    for code in range(10):
        s = lib.dd_status_str(code)
        assert s and s != b"unknown status"
    assert lib.dd_status_str(99) == b"unknown status"
    assert lib.dd_status_str(OK) == b"ok"


def test_workspace_bytes(lib):
    n = lib.dd_attn_bwd_workspace_bytes(8, 8192, 16, 128)
    rows = 8 * 8192 * 16 * 4
    assert n >= 2 * rows and n % 256 == 0
    assert lib.dd_attn_bwd_workspace_bytes(1, 1, 1, 64) == 512
    assert lib.dd_attn_bwd_workspace_bytes(1, 1, 1, 80) == 0
    assert lib.dd_attn_bwd_workspace_bytes(0, 1, 1, 64) == 0


def doc_check(lib, cu, total):
    a = np.ascontiguousarray(np.asarray(cu, dtype=np.int32))
    return lib.dd_doclens_check(a.ctypes.data_as(ctypes.c_void_p), a.size - 1, total)


def test_doclens_check(lib):
    assert doc_check(lib, [0, 5, 9, 16], 16) == OK
    assert doc_check(lib, [0, 16], 16) == OK
    assert doc_check(lib, [1, 5, 16], 16) == DOCLENS
    assert doc_check(lib, [0, 5, 5, 16], 16) == DOCLENS
    assert doc_check(lib, [0, 7, 3, 16], 16) == DOCLENS
    assert doc_check(lib, [0, 5, 15], 16) == DOCLENS
    assert doc_check(lib, [0], 16) == DOCLENS
    assert lib.dd_doclens_check(None, 3, 16) == NULL


# Fake, 16-byte aligned, non-overlapping device addresses: validation fails
# before any of them could be dereferenced or a kernel launched.
BASE = 1 << 40
GAP = 1 << 34


def fake(i, off=0):
    return ctypes.c_void_p(BASE + i * GAP + off)


def fwd(lib, q=None, k=None, v=None, o=None, lse=None, B=2, L=64, H=2, D=64, causal=1,
        cu=None, n_docs=0):
    args = [q or fake(0), k or fake(1), v or fake(2), o or fake(3), lse or fake(4)]
    return lib.dd_attn_fwd(*args, B, L, H, D, causal, cu, n_docs, None)


def test_fwd_validation(lib):
    assert lib.dd_attn_fwd(None, fake(1), fake(2), fake(3), fake(4), 2, 64, 2, 64, 1,
                           None, 0, None) == NULL
    assert lib.dd_attn_fwd(fake(0), fake(1), fake(2), fake(3), None, 2, 64, 2, 64, 1,
                           None, 0, None) == NULL
    assert fwd(lib, B=0) == SHAPE
    assert fwd(lib, L=0) == SHAPE
    assert fwd(lib, H=-1) == SHAPE
    assert fwd(lib, B=1 << 16, L=1 << 15, H=1) == SHAPE
    # H * D >= 2^23 (the DMA plans' 32-bit row offsets), with B*L*H < 2^31
    assert fwd(lib, B=1, L=1, H=1 << 16, D=128) == SHAPE
    assert fwd(lib, B=1, L=1, H=1 << 17, D=64) == SHAPE
    # B*H*ceil(L/128) > 2^23 - 8 (a one-block-per-workgroup grid of 512-item
    # workgroups would reach 2^32 work-items), with B*L*H < 2^31
    assert fwd(lib, B=(1 << 23) - 7, L=1, H=1) == SHAPE
    assert fwd(lib, B=(1 << 22) - 3, L=200, H=1) == SHAPE
    assert fwd(lib, B=1 << 20, L=1, H=16) == SHAPE
    assert bwd(lib, B=(1 << 23) - 7, L=1, H=1) == SHAPE
    assert rope_call(lib, B=(1 << 23) - 7, L=1, H=1) == SHAPE
    msg = lib.dd_status_str(SHAPE).decode()
    assert "2^31" in msg and "H*D < 2^23" in msg and "ceil(L/128)" in msg and "RoPE" in msg
    assert fwd(lib, D=80) == HEADDIM
    assert fwd(lib, D=32) == HEADDIM
    assert fwd(lib, cu=fake(5), n_docs=0) == DOCLENS
    assert fwd(lib, cu=None, n_docs=3) == DOCLENS
    assert fwd(lib, cu=fake(5), n_docs=129) == DOCLENS
    assert fwd(lib, cu=fake(5, 2), n_docs=3) == ALIGN
    assert fwd(lib, q=fake(0, 8)) == ALIGN
    assert fwd(lib, o=fake(3, 4)) == ALIGN
    assert fwd(lib, lse=fake(4, 2)) == ALIGN
    assert fwd(lib, o=fake(0, 64)) == ALIAS          # O overlaps Q
    assert fwd(lib, lse=fake(3, 1024)) == ALIAS      # LSE inside O
    assert fwd(lib, o=fake(5), lse=fake(5, 16)) == ALIAS
    assert fwd(lib, cu=fake(3, 32), n_docs=2) == ALIAS


def bwd(lib, ptrs=None, B=2, L=64, H=2, D=64, cu=None, n_docs=0, ws=None, ws_bytes=None):
    p = [fake(i) for i in range(9)]
    if ptrs:
        for i, v in ptrs.items():
            p[i] = v
    need = lib.dd_attn_bwd_workspace_bytes(B, L, H, D)
    ws = ws if ws is not None else fake(9)
    return lib.dd_attn_bwd(*p, B, L, H, D, 1, cu, n_docs, ws,
                           need if ws_bytes is None else ws_bytes, None)


def test_bwd_validation(lib):
    for i in range(9):
        assert bwd(lib, {i: None}) == NULL, i
    assert bwd(lib, B=0) == SHAPE
    assert bwd(lib, D=96) == HEADDIM
    assert bwd(lib, cu=fake(10), n_docs=0) == DOCLENS
    assert bwd(lib, ws=ctypes.c_void_p(0)) == WORKSPACE
    assert bwd(lib, ws_bytes=100) == WORKSPACE
    assert bwd(lib, {0: fake(0, 8)}) == ALIGN
    assert bwd(lib, {5: fake(5, 2)}) == ALIGN
    assert bwd(lib, ws=fake(9, 8)) == ALIGN
    assert bwd(lib, {7: fake(6)}) == ALIAS            # dK == dQ
    assert bwd(lib, {6: fake(4, 16)}) == ALIAS        # dQ overlaps dO
    assert bwd(lib, ws=fake(8, 1024)) == ALIAS        # workspace inside dV
    assert bwd(lib, {8: fake(5)}) == ALIAS            # dV over LSE
    assert bwd(lib, cu=fake(7, 64), n_docs=2) == ALIAS


def rope_call(lib, x=None, y=None, B=2, L=64, H=2, D=64, base=10000.0, inverse=0, cu=None,
              n_docs=0, doc=0):
    return lib.dd_rope(x or fake(0), y or fake(1), B, L, H, D, base, inverse, cu, n_docs, doc, None)


def test_rope_validation(lib):
    assert lib.dd_rope(None, fake(1), 2, 64, 2, 64, 1e4, 0, None, 0, 0, None) == NULL
    assert lib.dd_rope(fake(0), None, 2, 64, 2, 64, 1e4, 0, None, 0, 0, None) == NULL
    assert rope_call(lib, B=0) == SHAPE
    assert rope_call(lib, D=96) == HEADDIM
    for base in (0.0, -1.0, float("inf"), float("nan")):
        assert rope_call(lib, base=base) == SHAPE, base
    assert rope_call(lib, cu=fake(5), n_docs=0) == DOCLENS
    assert rope_call(lib, x=fake(0, 8)) == ALIGN
    assert rope_call(lib, y=fake(0, 64)) == ALIAS      # partial overlap of Y with X
    assert rope_call(lib, y=fake(5), cu=fake(5, 16), n_docs=3) == ALIAS


def test_bwd_rope_validation(lib):
    def call(base=10000.0, **kw):
        p = [fake(i) for i in range(9)]
        for i, v in kw.get("ptrs", {}).items():
            p[i] = v
        B, L, H, D = 2, 64, 2, 64
        need = lib.dd_attn_bwd_workspace_bytes(B, L, H, D)
        return lib.dd_attn_bwd_rope(*p, B, L, H, D, 1, None, 0, base, 0,
                                    kw.get("ws", fake(9)), kw.get("ws_bytes", need), None)
    for base in (0.0, -5.0, float("nan"), float("inf")):
        assert call(base) == SHAPE, base
    for i in range(9):
        assert call(ptrs={i: None}) == NULL, i
    assert call(ws_bytes=10) == WORKSPACE
    assert call(ptrs={7: fake(6)}) == ALIAS


def test_fused_rope_forward_validation(lib):
    def call(ptrs=None, B=2, L=64, H=2, D=64, base=1e4, cu=None, n_docs=0):
        p = [fake(i) for i in range(6)]
        for i, v in (ptrs or {}).items():
            p[i] = v
        return lib.dd_attn_fwd_rope(*p[:5], p[5], B, L, H, D, 1, cu, n_docs, base, 0, None)
    for i in range(5):
        assert call({i: None}) == NULL, i
    for base in (0.0, -1.0, float("nan"), float("inf")):
        assert call(base=base) == SHAPE
    assert call(B=0) == SHAPE
    assert call(D=96) == HEADDIM
    assert call({5: fake(5, 8)}) == ALIGN
    assert call({5: fake(0, 64)}) == ALIAS      # Q_rot overlaps Q
    assert call({5: fake(3, 64)}) == ALIAS      # Q_rot overlaps O
    assert call({5: fake(4)}) == ALIAS          # Q_rot overlaps LSE


def test_block_kernel_validation(lib):
    # GEMM: shapes, strides, alignment, aliasing; rejected on the host.
    def gemm(A=None, B=None, C=None, R=None, M=256, N=256, K=64, lda=None, ldb=None, ldc=None,
             ta=0, tb=0, ws=None, wsb=0):
        lda = lda if lda is not None else (M if ta else K)
        ldb = ldb if ldb is not None else (K if tb else N)
        ldc = ldc if ldc is not None else N
        return lib.dd_gemm(A or fake(0), lda, ta, B or fake(1), ldb, tb, R, C or fake(2), ldc,
                           M, N, K, ws, wsb, None)
    assert lib.dd_gemm(None, 64, 0, fake(1), 256, 0, None, fake(2), 256, 256, 256, 64, None, 0,
                       None) == NULL
    for kw in (dict(M=255), dict(N=300), dict(K=96), dict(M=0), dict(ta=1, tb=1),
               dict(lda=32), dict(ldc=128)):
        assert gemm(**kw) == SHAPE, kw
    assert gemm(lda=68) == ALIGN
    assert gemm(A=fake(0, 8)) == ALIGN
    assert gemm(C=fake(0, 1024)) == ALIAS           # C overlaps A
    assert gemm(R=fake(2, 64)) == ALIAS             # R partly overlaps C
    assert lib.dd_gemm_workspace_bytes(255, 256, 64) == 0
    # LayerNorm
    ln = lambda **kw: lib.dd_layernorm_fwd(kw.get("X", fake(0)), fake(1), fake(2),
                                           kw.get("Y", fake(3)), fake(4), fake(5),
                                           kw.get("rows", 8), kw.get("d", 512),
                                           kw.get("eps", 1e-5), None)
    assert ln(X=None) == NULL
    assert ln(d=256) == SHAPE and ln(d=4096) == SHAPE and ln(rows=0) == SHAPE
    assert ln(eps=0.0) == SHAPE and ln(eps=float("nan")) == SHAPE
    assert ln(Y=fake(0, 64)) == ALIAS
    assert lib.dd_layernorm_bwd_workspace_bytes(8, 300) == 0
    assert lib.dd_layernorm_bwd(fake(0), fake(1), fake(2), fake(3), fake(4), None, fake(5),
                                fake(6), fake(7), 8, 512, fake(8), 0, None) == WORKSPACE
    # SwiGLU
    assert lib.dd_swiglu_fwd(fake(0), fake(1), fake(2), 12, None) == SHAPE
    assert lib.dd_swiglu_fwd(fake(0), fake(1), fake(0, 16), 64, None) == ALIAS
    assert lib.dd_swiglu_bwd(fake(0), fake(1), fake(2), fake(3), fake(3, 16), 64, None) == ALIAS
    # transpose
    tr = lambda **kw: lib.dd_transpose(kw.get("X", fake(0)), kw.get("ldx", 192),
                                       kw.get("Y", fake(1)), kw.get("ldy", 128),
                                       kw.get("rows", 128), kw.get("cols", 192), None)
    assert tr(X=None) == NULL and tr(Y=None) == NULL
    for kw in (dict(rows=0), dict(rows=96), dict(cols=100), dict(ldx=128), dict(ldy=64),
               dict(rows=1 << 19, cols=1 << 18, ldx=1 << 18, ldy=1 << 19)):
        assert tr(**kw) == SHAPE, kw
    assert tr(ldx=196) == ALIGN and tr(X=fake(0, 8)) == ALIGN
    assert tr(Y=fake(0, 1024)) == ALIAS


def test_noalloc_backward_validation(lib):
    # Rejected on the host before the device scratch is touched.
    SCRATCH = 9
    def call(ptrs=None, B=2, L=64, H=2, D=64, cu=None, n_docs=0):
        p = [fake(i) for i in range(9)]
        for i, v in (ptrs or {}).items():
            p[i] = v
        return lib.dd_attn_bwd_noalloc(*p, B, L, H, D, 1, cu, n_docs, None)
    for i in range(9):
        assert call({i: None}) == NULL, i
    assert call(B=0) == SHAPE
    assert call(D=96) == HEADDIM
    assert call(cu=fake(9), n_docs=0) == DOCLENS
    # the scratch covers B*H*L <= 2^21
    assert call(B=8, L=8192, H=33) == SCRATCH
    assert call(B=1, L=(1 << 21) + 1, H=1) == SCRATCH
    assert b"16 MiB" in lib.dd_status_str(SCRATCH)


def test_python_wrapper_checks_metadata_on_cpu():
    torch = pytest.importorskip("torch")
    import paper_2405_13226_amd as dd
    q = torch.zeros(1, 4, 1, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        dd.forward(q, q, q)  # CPU tensors are rejected before any call
    with pytest.raises(ValueError):
        dd.rope(q, 10000.0)
    with pytest.raises(_lib.DDError):
        dd.DocLens([0, 3, 2, 4], 4, torch.device("cpu"))


def test_prof_launches_without_records(lib):
    # Nothing recorded: a count of 0, no device call.  A NULL count, or
    # NULL arrays with a capacity, is rejected.
    n = ctypes.c_longlong(-1)
    assert lib.dd_prof_launches(None, None, 0, ctypes.byref(n)) == OK and n.value == 0
    assert lib.dd_prof_launches(None, None, 0, None) == NULL
    assert lib.dd_prof_launches(None, None, 4, ctypes.byref(n)) == NULL


def test_kernel_ids_match_the_library(lib):
    # The Python table of profiling ids names what the library reports for
    # each id (a host-side lookup, no device call).
    for name, kid in _lib.KERNELS.items():
        assert lib.dd_prof_kernel_name(kid).decode() == name
    assert lib.dd_prof_kernel_name(len(_lib.KERNELS)) is None
    assert lib.dd_prof_kernel_name(-1) is None


def test_bench_counts_the_one_kernel_backward_where_the_library_runs_it():
    # bench.py's FLOP accounting assumes the one-kernel backward runs for
    # D = 64 rows up to the library's limit (kShortMaxRow).
    import bench
    text = open(os.path.join(ROOT, "paper_2405_13226_amd", "csrc", "dd_bwd.hpp")).read()
    m = re.search(r"constexpr int kShortMaxRow = (\d+);", text)
    assert m and int(m.group(1)) == bench.SHORT_MAX_ROW
