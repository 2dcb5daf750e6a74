"""The C ABI on the CPU: liblpv.so loads without a GPU, exports every entry
point that include/lpv.h declares, and rejects bad arguments before any HIP
call (so these run here, with made-up device addresses that are never read)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lpv.h")
LIB = os.path.join(ROOT, "paper_2407_02068_amd", "liblpv.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="liblpv.so not built")

OK, INVALID, SHAPE, DTYPE, BLOCK, ALIAS, ALLOC, HIP = 0, -1, -2, -3, -4, -5, -6, -7
FAKE = 0x7f0000000000  # 16-byte aligned, never dereferenced: every call below fails its checks first


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lpv_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    from paper_2407_02068_amd import lpv
    return lpv.lib()


def test_header_declares_the_boundary():
    names = declared()
    for n in ("lpv_bsr_pack", "lpv_bsr_linear", "lpv_dense_linear", "lpv_bsr_export",
              "lpv_bsr_unpack", "lpv_bsr_destroy", "lpv_bsr_schedule_export"):
        assert n in names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(LIB)
    for name in declared():
        assert hasattr(lib, name), "liblpv.so does not export %s" % name


def test_python_binding_names_match_header():
    from paper_2407_02068_amd import lpv
    assert sorted(lpv.EXPORTED) == declared()


def test_status_strings(L):
    for code, name in ((OK, "LPV_OK"), (INVALID, "LPV_ERR_INVALID_ARG"), (SHAPE, "LPV_ERR_SHAPE"),
                       (DTYPE, "LPV_ERR_DTYPE"), (BLOCK, "LPV_ERR_BLOCK"), (ALIAS, "LPV_ERR_ALIAS"),
                       (ALLOC, "LPV_ERR_ALLOC"), (HIP, "LPV_ERR_HIP")):
        assert L.lpv_status_str(code).decode() == name


def pack(L, W=FAKE, ldw=768, N=3072, K=768, dt=2, b_r=32, b_c=32, mask=FAKE):
    out = ctypes.c_void_p(123)
    st = L.lpv_bsr_pack(W, ldw, N, K, dt, b_r, b_c, mask, None, ctypes.byref(out))
    if st != OK:
        assert out.value is None  # *out is cleared on failure
    return st


@pytest.mark.parametrize("kw,want", [
    (dict(dt=3), DTYPE), (dict(dt=-1), DTYPE),
    (dict(b_r=8), BLOCK), (dict(b_c=128), BLOCK), (dict(b_r=48), BLOCK),
    (dict(N=3072 + 16, b_r=32), SHAPE), (dict(K=768 + 16), SHAPE), (dict(N=0), SHAPE),
    (dict(N=1 << 17), SHAPE), (dict(K=-32), SHAPE),
    (dict(W=0), INVALID), (dict(mask=0), INVALID), (dict(W=FAKE + 8), INVALID),
    (dict(ldw=700), INVALID), (dict(ldw=772), INVALID),
    # 16-bit types: K <= 63424 (a group's walk must fit the kernel's LDS table)
    (dict(K=63456, ldw=63456), SHAPE), (dict(K=65536, ldw=65536, dt=1), SHAPE),
    (dict(K=65536, ldw=65536, dt=0, W=0), INVALID),  # fp32 has no such limit
    (dict(K=63424, ldw=63424, W=0), INVALID),        # the largest 16-bit K passes the shape checks
])
def test_pack_rejects_bad_arguments(L, kw, want):
    assert pack(L, **kw) == want
    assert L.lpv_last_error().decode() != ""


def test_pack_null_out(L):
    assert L.lpv_bsr_pack(FAKE, 768, 3072, 768, 2, 32, 32, FAKE, None, None) == INVALID


def test_pack_alloc_failure_is_reported(L, monkeypatch):
    monkeypatch.setenv("LPV_FAULT_INJECT", "alloc")
    assert pack(L) == ALLOC
    assert "allocation" in L.lpv_last_error().decode()


def dense(L, W=FAKE, ldw=768, N=3072, K=768, dt=2, X=FAKE + (1 << 32), ldx=768, M=197, bias=0,
          Y=FAKE + (2 << 32), ldy=3072, epi=0):
    return L.lpv_dense_linear(W, ldw, N, K, dt, X, ldx, M, bias, Y, ldy, epi, None)


@pytest.mark.parametrize("kw,want", [
    (dict(dt=7), DTYPE), (dict(N=3000), SHAPE), (dict(K=8), SHAPE), (dict(M=-1), SHAPE),
    (dict(ldx=767), INVALID), (dict(ldy=3000), INVALID), (dict(ldx=772), INVALID),
    (dict(X=0), INVALID), (dict(Y=0), INVALID), (dict(X=FAKE + (1 << 32) + 4), INVALID),
    (dict(bias=FAKE + 2), INVALID), (dict(epi=2), INVALID), (dict(W=0), INVALID),
    (dict(Y=FAKE + (1 << 32) + 64), ALIAS), (dict(X=FAKE + (2 << 32) + 1024), ALIAS),
    # leading dimensions above 2^22 elements (32-bit byte offsets in the kernels)
    (dict(ldx=(1 << 22) + 8), INVALID), (dict(ldw=(1 << 22) + 8), INVALID),
    # 16-bit types: K <= 63424
    (dict(K=63440, ldw=63440, ldx=63440), SHAPE), (dict(K=65536, ldw=65536, ldx=65536, dt=1), SHAPE),
])
def test_dense_rejects_bad_arguments(L, kw, want):
    assert dense(L, **kw) == want


def test_dense_m0_is_a_noop(L):
    # M = 0: nothing to do, no HIP call, even with NULL X / Y
    assert dense(L, M=0, X=0, Y=0) == OK


def test_linear_rejects_null_handle(L):
    assert L.lpv_bsr_linear(None, FAKE, 768, 197, None, FAKE + (1 << 32), 3072, 0, None) == INVALID
    from paper_2407_02068_amd.lpv import BsrInfo
    info = BsrInfo()
    assert L.lpv_bsr_info_get(None, ctypes.byref(info)) == INVALID
    assert L.lpv_bsr_export(None, None, None, None, None) == INVALID
    assert L.lpv_bsr_schedule_export(None, None, None, None, None, None, None) == INVALID
    assert L.lpv_bsr_unpack(None, FAKE, 768, None) == INVALID
    L.lpv_bsr_destroy(None)  # NULL-safe


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2407_02068_amd import lpv
    monkeypatch.setattr(lpv, "_lib", None)
    monkeypatch.setattr(lpv, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        lpv.lib()


def mask_topk(L, W=FAKE, ldw=768, N=3072, K=768, dt=2, b_r=32, b_c=32, G=0, ldg=768, p=50,
              mask=FAKE + (1 << 32), scores=FAKE + (2 << 32)):
    return L.lpv_mask_topk(W, ldw, N, K, dt, b_r, b_c, G, ldg, p, mask, scores, None)


@pytest.mark.parametrize("kw,want", [
    (dict(dt=5), DTYPE), (dict(b_r=8), BLOCK), (dict(b_c=24), BLOCK),
    (dict(N=3072 + 16), SHAPE), (dict(K=0), SHAPE), (dict(N=1 << 17), SHAPE),
    (dict(p=-1), INVALID), (dict(p=101), INVALID),
    (dict(W=0), INVALID), (dict(mask=0), INVALID), (dict(scores=0), INVALID),
    (dict(ldw=700), INVALID), (dict(G=FAKE + (3 << 32), ldg=100), INVALID),
    (dict(W=FAKE + 1), INVALID), (dict(scores=FAKE + (2 << 32) + 4), INVALID),
])
def test_mask_topk_rejects_bad_arguments(L, kw, want):
    assert mask_topk(L, **kw) == want
    assert L.lpv_last_error().decode() != ""


def test_backward_rejects_bad_arguments(L):
    out = ctypes.c_void_p(123)
    assert L.lpv_bsr_transpose(None, None, ctypes.byref(out)) == INVALID and out.value is None
    assert L.lpv_bsr_transpose(None, None, None) == INVALID
    assert L.lpv_bsr_grad_w(None, FAKE, 3072, FAKE, 768, 10, FAKE, None) == INVALID
    # bias gradient: every check runs before any HIP call
    bg = lambda G=FAKE, ldg=3072, M=10, N=3072, dt=2, db=FAKE + (1 << 32): \
        L.lpv_bias_grad(G, ldg, M, N, dt, db, None)
    assert bg(dt=7) == DTYPE
    assert bg(N=0) == SHAPE and bg(N=1 << 17) == SHAPE
    assert bg(M=-1) == SHAPE and bg(M=1 << 31) == SHAPE
    assert bg(ldg=3000) == INVALID and bg(ldg=3076) == INVALID and bg(ldg=(1 << 22) + 8) == INVALID
    assert bg(db=0) == INVALID and bg(db=FAKE + 1) == INVALID
    assert bg(G=0) == INVALID and bg(G=FAKE + 8) == INVALID
    assert L.lpv_last_error().decode() != ""
    # the no-allocation variant runs the same checks before any HIP call
    bn = lambda G=FAKE, ldg=3072, M=10, N=3072, dt=2, db=FAKE + (1 << 32): \
        L.lpv_bias_grad_noalloc(G, ldg, M, N, dt, db, None)
    assert bn(dt=7) == DTYPE
    assert bn(N=0) == SHAPE and bn(N=1 << 17) == SHAPE
    assert bn(M=-1) == SHAPE and bn(M=1 << 31) == SHAPE
    assert bn(ldg=3000) == INVALID and bn(ldg=3076) == INVALID
    assert bn(db=0) == INVALID and bn(db=FAKE + 1) == INVALID
    assert bn(G=0) == INVALID and bn(G=FAKE + 8) == INVALID
    assert L.lpv_last_error().decode() != ""


def test_delta_curve_rejects_bad_arguments(L):
    pc = (ctypes.c_int32 * 3)(0, 50, 100)
    bad = (ctypes.c_int32 * 3)(0, 60, 50)

    def dc(W=FAKE, ldw=768, N=3072, K=768, dt=2, b_r=32, b_c=32, grad=FAKE + (1 << 32), ldg=768,
           S=FAKE + (2 << 32), lds=768, stride=3072 * 768, n=4, kappa=0.1, pcts=pc, npt=3,
           out=FAKE + (3 << 32)):
        return L.lpv_delta_curve(W, ldw, N, K, dt, b_r, b_c, grad, ldg, S, lds, stride, n,
                                 ctypes.c_double(kappa), pcts, npt, out, None)
    assert dc(dt=9) == DTYPE and dc(b_r=8) == BLOCK
    assert dc(N=3072 + 16) == SHAPE and dc(N=1 << 17) == SHAPE and dc(n=-1) == SHAPE
    assert dc(n=70000) == SHAPE
    assert dc(N=16384, K=16384, b_r=16, b_c=16, ldw=16384, ldg=16384, lds=16384,
              stride=16384 * 16384) == SHAPE  # more than 2^17 blocks
    assert dc(pcts=bad) == INVALID and dc(npt=0) == INVALID and dc(npt=200) == INVALID
    assert dc(pcts=None) == INVALID and dc(kappa=float("nan")) == INVALID
    assert dc(W=0) == INVALID and dc(grad=0) == INVALID and dc(out=0) == INVALID
    assert dc(S=0) == INVALID and dc(W=FAKE + 8) == INVALID and dc(out=FAKE + (3 << 32) + 4) == INVALID
    assert dc(ldw=700) == INVALID and dc(lds=770) == INVALID and dc(stride=100) == INVALID
    assert L.lpv_last_error().decode() != ""


def test_delta_curve_workspace_size_and_checks(L):
    sz = ctypes.c_size_t(0)

    def ws(N=3072, K=768, b_r=32, b_c=32, n=4, npt=21, out=True):
        return L.lpv_delta_curve_workspace_size(N, K, b_r, b_c, n, npt,
                                                ctypes.byref(sz) if out else None)
    assert ws() == OK
    # scores, dots of n + 2 vectors, per-point step sums and terms (float64),
    # the permutation (int32)
    nb = 96 * 24
    assert sz.value == (nb + 6 * nb + 21 * 6 + 21) * 8 + nb * 4
    big = ws(N=768, K=3072, n=64, npt=128) == OK and sz.value
    assert big > (66 * 2304) * 8
    assert ws(b_r=8) == BLOCK and ws(N=3072 + 16) == SHAPE and ws(N=1 << 17) == SHAPE
    assert ws(N=16384, K=16384, b_r=16, b_c=16) == SHAPE
    assert ws(n=-1) == INVALID and ws(npt=0) == INVALID and ws(npt=129) == INVALID
    assert ws(out=False) == INVALID
    pc = (ctypes.c_int32 * 3)(0, 50, 100)

    def dw(buf=FAKE + (4 << 32), nbytes=1 << 30, N=3072):
        return L.lpv_delta_curve_ws(FAKE, 768, N, 768, 2, 32, 32, FAKE + (1 << 32), 768,
                                    FAKE + (2 << 32), 768, 3072 * 768, 4, ctypes.c_double(0.1),
                                    pc, 3, FAKE + (3 << 32), buf, nbytes, None)
    assert dw(buf=0) == INVALID and dw(nbytes=64) == INVALID and dw(buf=FAKE + 8) == INVALID
    assert dw(N=3072 + 16) == SHAPE


def test_encoder_calls_reject_bad_arguments(L):
    # every check runs before any HIP call; empty batches return OK untouched
    ln = lambda x=FAKE, y=0, M=10, D=768, dt=2, g=FAKE + (1 << 32), b=FAKE + (2 << 32), eps=1e-6, \
        S=0, out=FAKE + (3 << 32): L.lpv_add_layernorm(x, y, M, D, dt, g, b, ctypes.c_double(eps),
                                                       S, out, None)
    assert ln(dt=0) == DTYPE and ln(dt=9) == DTYPE
    assert ln(D=2) == SHAPE and ln(D=770) == SHAPE and ln(D=4096) == SHAPE
    assert ln(M=-1) == SHAPE and ln(M=1 << 31) == SHAPE
    assert ln(eps=-1.0) == INVALID and ln(eps=float("inf")) == INVALID
    assert ln(g=0) == INVALID and ln(b=FAKE + 4) == INVALID and ln(x=0) == INVALID
    assert ln(out=FAKE + 2) == INVALID and ln(y=FAKE + 6) == INVALID and ln(S=FAKE + 4) == INVALID
    assert ln(M=0, x=0, out=0) == OK
    at = lambda q=FAKE, n=4, T=197, H=12, hd=64, dt=2, out=FAKE + (1 << 32): \
        L.lpv_attention(q, n, T, H, hd, dt, out, None)
    assert at(dt=0) == DTYPE and at(hd=32) == SHAPE and at(hd=128) == SHAPE
    assert at(T=0) == SHAPE and at(T=513) == SHAPE and at(H=0) == SHAPE and at(H=65) == SHAPE
    assert at(n=-1) == SHAPE and at(n=1 << 24) == SHAPE
    assert at(q=0) == INVALID and at(out=FAKE + 8) == INVALID
    assert at(out=FAKE + 64) == ALIAS
    assert at(n=0, q=0, out=0) == OK
    assert L.lpv_last_error().decode() != ""
