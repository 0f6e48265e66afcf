"""Host-side checks of the C ABI: the built library exports every function the
header declares, the status strings and workspace sizes, and argument
validation (calls that must return L1CSR_EINVAL before launching anything).

No call here launches a kernel.  The validation calls run only on a machine
without a GPU device node, so that a validation mistake can never reach a
kernel with the placeholder pointers used here.
"""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "l1csr.h")
LIB = os.path.join(ROOT, "paper_1905_07931_amd", "libl1csr.so")

OK, EINVAL, ECAPACITY, EBADCSR, EHIP, EUNSUPPORTED, ESCRATCH = 0, -1, -2, -3, -4, -5, -6
NO_GPU = not os.path.exists("/dev/kfd")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?(?:int|size_t|char)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_1905_07931_amd import build
        build.build(verbose=False)
    lib = C.CDLL(LIB)
    lib.l1csr_status_str.restype = C.c_char_p
    lib.l1csr_status_str.argtypes = [C.c_int]
    lib.l1csr_workspace_bytes.restype = C.c_size_t
    lib.l1csr_workspace_bytes.argtypes = [C.c_int, C.c_int32, C.c_int32, C.c_int64, C.c_int32]
    return lib


def test_header_declares_the_hot_path_calls():
    names = declared_functions()
    for n in ["csr_spmm_fwd", "csr_spmm_bwd_t", "dense_wgrad", "sddmm_masked_wgrad", "prox_l1_step",
              "csr_recompress", "prox_l1_recompress", "csc_build", "csc_update_vals", "csr_compact",
              "csr_validate", "l1csr_workspace_bytes", "l1csr_status_str", "prox_adaptive_step",
              "prox_adaptive_recompress", "prox_l1_recompress_noalloc"]:
        assert n in names, n


def test_library_exports_every_declared_function(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(lib):
    seen = set()
    for code in (OK, EINVAL, ECAPACITY, EBADCSR, EHIP, EUNSUPPORTED, ESCRATCH):
        s = lib.l1csr_status_str(code).decode()
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 7
    assert lib.l1csr_status_str(12345).decode() == "unknown status"


def test_workspace_sizes(lib):
    ws = lib.l1csr_workspace_bytes
    assert ws(99, 10, 10, 10, 10) == 0                 # unknown op
    assert ws(1, -1, 10, 10, 10) == 0                  # negative size
    for op in range(1, 9):
        for dims in [(1, 1, 1, 1), (300, 784, 23520, 64), (4096, 9216, 3397386, 1024)]:
            b = ws(op, *dims)
            assert b % 256 == 0, (op, dims, b)
    # the sizes grow with the problem
    assert ws(1, 4096, 9216, 3397386, 0) >= ws(1, 300, 784, 23520, 0) > 0
    assert ws(4, 4096, 9216, 3397386, 1024) > ws(4, 4096, 300, 200000, 1024) > 0
    assert ws(3, 4096, 9216, 3397386, 1024) > 0
    assert ws(2, 4096, 9216, 0, 0) >= 4 * 4097
    assert ws(7, 4096, 9216, 0, 0) >= 4 * 4097


P = C.c_void_p(4096)  # placeholder non-null pointer; never dereferenced by a rejected call
NUL = None
S = None              # default stream


def _f(x):
    return C.c_float(x)


def _setup(lib):
    lib.csr_spmm_fwd.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_int64, C.c_void_p,
                                 C.c_size_t, C.c_void_p]
    lib.dense_wgrad.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int64, C.c_void_p,
                                C.c_int64, C.c_void_p, C.c_int64, C.c_int, C.c_void_p, C.c_size_t,
                                C.c_void_p]
    lib.csr_validate.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p]
    lib.prox_l1_step.argtypes = [C.c_int, C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_int64, C.c_float, C.c_float, C.c_void_p,
                                 C.c_int64, C.c_void_p, C.c_void_p]
    lib.csr_recompress.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_int64, C.c_float, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.prox_l1_recompress.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_int64, C.c_float, C.c_float,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.sddmm_masked_wgrad.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_int64, C.c_void_p, C.c_int64, C.c_int32,
                                       C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.csc_build.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p,
                              C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                              C.c_void_p, C.c_size_t, C.c_void_p]
    lib.csr_spmm_bwd_t.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_int64, C.c_int32, C.c_void_p, C.c_int64, C.c_void_p,
                                   C.c_size_t, C.c_void_p]


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_sizes_beyond_the_int32_layout_are_unsupported(lib):
    # row pointers are int32: an N x K output above 2^31 - 1 entries cannot be
    # addressed; grid limits bound the batch and the row tiles
    _setup(lib)
    big = 65536  # 65536 * 65536 = 2^32 entries
    assert lib.csr_recompress(big, big, P, big, 0.0, NUL, P, P, P, 16, NUL, NUL, P, 1 << 30, S) == EUNSUPPORTED
    Q = C.c_void_p(8192)  # an output CSR distinct from the input
    assert lib.prox_l1_recompress(big, big, 0, P, P, P, P, big, 0.1, 0.1, Q, Q, Q, 16, NUL, NUL, P, 1 << 30,
                                  S) == EUNSUPPORTED
    assert lib.dense_wgrad(128 * 65536 + 1, 4, 8, P, 8, P, 8, P, 4, 0, NUL, 0, S) == EUNSUPPORTED
    assert lib.csr_spmm_fwd(4, 4, 3, P, P, P, P, 64 * 65536 + 64, 64 * 65536 + 64, P, 64 * 65536 + 64,
                            NUL, 0, S) == EUNSUPPORTED
    # the largest supported N x K passes the size check (it fails later only on the missing workspace)
    n = 46340  # 46340^2 = 2,147,395,600 < 2^31
    assert lib.csr_recompress(n, n, P, n, 0.0, NUL, P, P, P, 16, NUL, NUL, NUL, 0, S) == EINVAL


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_invalid_arguments_are_rejected_before_launch(lib):
    _setup(lib)
    # SpMM: negative size, missing pointer, short leading dimension, nnz > N*K, short workspace
    assert lib.csr_spmm_fwd(-1, 4, 0, P, P, P, P, 8, 8, P, 8, NUL, 0, S) == EINVAL
    assert lib.csr_spmm_fwd(4, 4, 3, NUL, P, P, P, 8, 8, P, 8, NUL, 0, S) == EINVAL
    assert lib.csr_spmm_fwd(4, 4, 3, P, P, P, P, 7, 8, P, 8, NUL, 0, S) == EINVAL
    assert lib.csr_spmm_fwd(4, 4, 3, P, P, P, P, 8, 8, P, 7, NUL, 0, S) == EINVAL
    assert lib.csr_spmm_fwd(4, 4, 17, P, P, P, P, 8, 8, P, 8, NUL, 0, S) == EINVAL
    assert lib.l1csr_workspace_bytes(4, 4096, 300, 200000, 1024) > 1
    assert lib.csr_spmm_fwd(4096, 300, 200000, P, P, P, P, 1024, 1024, P, 1024, P, 1, S) == EINVAL
    # dense dW: short ld, missing output, unknown precision
    assert lib.dense_wgrad(4, 4, 8, P, 7, P, 8, P, 4, 0, NUL, 0, S) == EINVAL
    assert lib.dense_wgrad(4, 4, 8, P, 8, P, 8, P, 3, 0, NUL, 0, S) == EINVAL
    assert lib.dense_wgrad(4, 4, 8, P, 8, P, 8, NUL, 4, 1, NUL, 0, S) == EINVAL
    assert lib.dense_wgrad(4, 4, 8, P, 8, P, 8, P, 4, 3, NUL, 0, S) == EINVAL
    assert lib.dense_wgrad(4, 4, 8, P, 8, P, 8, P, 4, -1, NUL, 0, S) == EINVAL
    # a workspace shorter than the split reduction of a skinny product needs
    need = lib.l1csr_workspace_bytes(8, 50, 500, 0, 16384)
    assert need >= 4 * 50 * 500 * 2
    assert lib.dense_wgrad(50, 500, 16384, P, 16384, P, 16384, P, 500, 0, P, need - 4096, S) == EINVAL
    # CSR check: negative sizes, missing status or columns
    assert lib.csr_validate(-1, 4, 0, P, P, P, S) == EINVAL
    assert lib.csr_validate(4, 4, 3, P, P, NUL, S) == EINVAL
    assert lib.csr_validate(4, 4, 3, P, NUL, P, S) == EINVAL
    assert lib.csr_validate(4, 4, -2, P, P, P, S) == EINVAL
    # prox: non-finite or negative eta / lambda, bad mode
    nan, inf = float("nan"), float("inf")
    for eta, lam in [(nan, 0.1), (0.1, nan), (inf, 0.1), (0.1, -1.0), (-0.1, 0.1)]:
        assert lib.prox_l1_step(0, 4, 4, 3, P, P, P, P, 4, eta, lam, P, 4, NUL, S) == EINVAL
    assert lib.prox_l1_step(7, 4, 4, 3, P, P, P, P, 4, 0.1, 0.1, P, 4, NUL, S) == EINVAL
    assert lib.prox_l1_step(0, 4, 4, 3, P, P, P, P, 3, 0.1, 0.1, P, 4, NUL, S) == EINVAL
    # recompress: non-finite threshold, missing outputs, short workspace
    assert lib.csr_recompress(4, 4, P, 4, nan, NUL, P, P, P, 16, NUL, NUL, P, 4096, S) == EINVAL
    assert lib.csr_recompress(4, 4, P, 4, 0.0, NUL, NUL, P, P, 16, NUL, NUL, P, 4096, S) == EINVAL
    assert lib.csr_recompress(4, 4, P, 4, 0.0, NUL, P, P, P, 16, NUL, NUL, P, 1, S) == EINVAL
    # fused prox + recompress: output aliasing the input CSR, short workspace
    assert lib.prox_l1_recompress(4, 4, 3, P, P, P, P, 4, 0.1, 0.1, P, P, P, 16, NUL, NUL, P, 4096,
                                  S) == EINVAL
    Q = C.c_void_p(8192)
    assert lib.prox_l1_recompress(4, 4, 3, P, P, P, P, 4, 0.1, 0.1, Q, Q, Q, 16, NUL, NUL, P, 1,
                                  S) == EINVAL
    # SDDMM: missing output
    assert lib.sddmm_masked_wgrad(4, 4, 3, P, P, P, 8, P, 8, 8, NUL, P, 1 << 20, S) == EINVAL
    # CSC build: missing workspace
    assert lib.csc_build(4, 4, 3, P, P, P, NUL, NUL, P, P, P, P, NUL, 0, S) == EINVAL
    # CSC build: half a bitmap index
    assert lib.csc_build(4, 4, 3, P, P, P, P, NUL, P, P, P, P, P, 1 << 20, S) == EINVAL
    # backward: half a CSC (row_idx without col_ptr)
    assert lib.csr_spmm_bwd_t(4, 4, 3, P, P, P, NUL, P, NUL, P, 8, 8, P, 8, NUL, 0, S) == EINVAL


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_adaptive_prox_arguments_are_rejected_before_launch(lib):
    vp, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
    lib.prox_adaptive_step.argtypes = [C.c_int, C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, vp, vp, i64,
                                       f32, f32, f32, f32, f32, i64, vp, i64, vp, vp, C.c_size_t, vp]
    lib.prox_adaptive_recompress.argtypes = [C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, vp, vp, i64,
                                             f32, f32, f32, f32, f32, i64, vp, vp, vp, i64, vp, vp, vp,
                                             C.c_size_t, vp]
    # distinct, far-apart placeholder buffers: W arrays, G, m, v, Z, outputs, workspace
    Wp, G, M, V, Z, O, WS = (C.c_void_p(a << 24) for a in range(1, 8))
    ws = lib.l1csr_workspace_bytes(7, 4, 4, 3, 0)
    step, rec = lib.prox_adaptive_step, lib.prox_adaptive_recompress
    nan, inf = float("nan"), float("inf")

    def dense(solver=2, eta=0.01, lam=0.1, eps=1e-8, b1=0.9, b2=0.999, t=1, m=M, v=V, z=Z, g=G,
              ldg=4, lds=4, ldz=4, w=WS, wb=None):
        return step(0, solver, 4, 4, 3, Wp, Wp, Wp, g, ldg, m, v, lds, eta, lam, eps, b1, b2, t, z, ldz,
                    NUL, w, ws if wb is None else wb, S)

    def fused(solver=2, eta=0.01, lam=0.1, eps=1e-8, b1=0.9, b2=0.999, t=1, m=M, v=V, g=G, out=O,
              w=WS, wb=None):
        return rec(solver, 4, 4, 3, Wp, Wp, Wp, g, 4, m, v, 4, eta, lam, eps, b1, b2, t, out, out, out,
                   16, NUL, NUL, w, ws if wb is None else wb, S)

    for f in (dense, fused):
        # solver codes, step, threshold and safeguard parameters (Algorithms 1-2)
        for bad in [dict(solver=0), dict(solver=3), dict(eta=0.0), dict(eta=nan), dict(lam=-1.0),
                    dict(lam=inf), dict(eps=0.0), dict(eps=-1e-8), dict(eps=nan), dict(b2=1.0),
                    dict(b2=-0.1), dict(b1=1.0), dict(b1=-0.5), dict(t=0), dict(t=-3)]:
            assert f(**bad) == EINVAL, (f.__name__, bad)
        # ADAM needs m; G, m, v must be distinct buffers; a short workspace
        assert f(m=NUL) == EINVAL
        assert f(m=V) == EINVAL and f(v=G) == EINVAL and f(m=G) == EINVAL
        assert f(w=NUL) == EINVAL and f(wb=1) == EINVAL
    # dense form: Z over the state, short leading dimensions
    assert dense(z=V) == EINVAL and dense(solver=1, m=NUL, z=V) == EINVAL
    assert dense(ldg=3) == EINVAL and dense(lds=3) == EINVAL and dense(ldz=3) == EINVAL
    # fused: the output CSR must not be W's
    assert fused(out=Wp) == EINVAL
    # stored-entry form: missing state, state over the gradient or the values
    assert step(1, 2, 4, 4, 3, Wp, Wp, Wp, G, 0, NUL, V, 0, 0.01, 0.0, 1e-8, 0.9, 0.999, 1, NUL, 0,
                NUL, NUL, 0, S) == EINVAL
    assert step(1, 1, 4, 4, 3, Wp, Wp, Wp, G, 0, NUL, G, 0, 0.01, 0.0, 1e-8, 0.9, 0.999, 1, NUL, 0,
                NUL, NUL, 0, S) == EINVAL
    assert step(1, 1, 4, 4, 3, Wp, Wp, V, G, 0, NUL, V, 0, 0.01, 0.0, 1e-8, 0.9, 0.999, 1, NUL, 0,
                NUL, NUL, 0, S) == EINVAL
    assert step(5, 1, 4, 4, 3, Wp, Wp, Wp, G, 4, NUL, V, 4, 0.01, 0.0, 1e-8, 0.9, 0.999, 1, Z, 4,
                NUL, WS, ws, S) == EINVAL


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_fused_updates_reject_outputs_overlapping_inputs(lib):
    """prox_l1_recompress / prox_adaptive_recompress write W' while other
    workgroups still read W, G and the states: any byte overlap between an
    output array (row_ptr_out [N+1], col_idx_out / vals_out [capacity]) and
    an input, or between two outputs, is rejected before launch.  With every
    buffer distinct the same calls get past validation (and, with no GPU,
    fail only at the launch)."""
    _setup(lib)
    vp, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
    lib.prox_adaptive_recompress.argtypes = [C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, vp, vp, i64,
                                             f32, f32, f32, f32, f32, i64, vp, vp, vp, i64, vp, vp, vp,
                                             C.c_size_t, vp]
    N = K = 64
    nnz, cap = 100, N * K
    base = {n: (i + 1) << 24 for i, n in enumerate(["rp", "ci", "v", "G", "m", "vv", "rpo", "cio", "vo", "ws"])}
    ws = lib.l1csr_workspace_bytes(7, N, K, nnz, 0)

    def plain(**o):
        a = dict(base, **o)
        p = {k: C.c_void_p(x) for k, x in a.items()}
        return lib.prox_l1_recompress(N, K, nnz, p["rp"], p["ci"], p["v"], p["G"], K, 0.1, 0.1, p["rpo"],
                                      p["cio"], p["vo"], cap, NUL, NUL, p["ws"], ws, S)

    def adam(**o):
        a = dict(base, **o)
        p = {k: C.c_void_p(x) for k, x in a.items()}
        return lib.prox_adaptive_recompress(2, N, K, nnz, p["rp"], p["ci"], p["v"], p["G"], K, p["m"],
                                            p["vv"], K, 0.01, 0.1, 1e-8, 0.9, 0.999, 1, p["rpo"], p["cio"],
                                            p["vo"], cap, NUL, NUL, p["ws"], ws, S)

    for f in (plain, adam):
        assert f() == EHIP  # valid arguments: only the launch fails here
        inside = lambda name, off=64: base[name] + off
        for bad in [dict(cio=inside("v")), dict(vo=inside("ci")), dict(vo=inside("G", 4 * (N * K - 1))),
                    dict(rpo=inside("ci", 4 * (nnz - 1))), dict(cio=inside("rp", -4 * cap + 8)),
                    dict(vo=inside("cio", 4 * (cap - 1))), dict(rpo=inside("vo"))]:
            assert f(**bad) == EINVAL, (f.__name__, bad)
        # just past the end of an input is fine
        assert f(cio=base["v"] + 4 * nnz) == EHIP
    for bad in [dict(vo=inside("m")), dict(cio=inside("vv", 4 * (N * K - 1)))]:
        assert adam(**bad) == EINVAL, bad
    assert plain(vo=inside("m")) == EHIP  # the plain update has no state


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_noalloc_prox_checks_its_arguments_and_scratch_before_launch(lib):
    """prox_l1_recompress_noalloc validates like prox_l1_recompress and
    rejects a layer whose slab scratch exceeds the 16 MiB static array with
    L1CSR_ESCRATCH, before any runtime call."""
    vp, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
    f = lib.prox_l1_recompress_noalloc
    f.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, f32, f32, vp, vp, vp, i64, vp, vp, vp]
    a = {n: C.c_void_p((i + 1) << 28) for i, n in enumerate(["rp", "ci", "v", "G", "rpo", "cio", "vo"])}

    def call(N, K, nnz=0, eta=0.01, lam=1e-4, ldg=None, rpo=None, cap=None):
        return f(N, K, nnz, a["rp"], a["ci"], a["v"], a["G"], K if ldg is None else ldg, eta, lam,
                 a["rpo"] if rpo is None else rpo, a["cio"], a["vo"], N * K if cap is None else cap, NUL,
                 NUL, S)

    assert lib.l1csr_workspace_bytes(7, 2_000_000, 1, 0, 0) > 16 << 20
    assert call(2_000_000, 1) == ESCRATCH
    assert call(64, 64, eta=float("nan")) == EINVAL
    assert call(64, 64, ldg=63) == EINVAL
    assert call(64, 64, rpo=C.c_void_p(0)) == EINVAL  # no row pointers
    assert call(64, 64, nnz=10, rpo=a["ci"]) == EINVAL   # output over W's columns
    assert call(65536, 65536) == EUNSUPPORTED            # beyond the int32 layout


@pytest.mark.skipif(not NO_GPU, reason="validation calls use placeholder pointers; run without a GPU")
def test_fused_weight_update_arguments_are_rejected_before_launch(lib):
    """dense_wgrad_prox, csr_recompress_counted and csr_bitmap_build check
    their arguments on the host: sizes, precision, eta / lambda, a missing
    bitmap or counts array, leading dimensions, a short workspace, and every
    output apart from every input."""
    vp, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
    f = lib.dense_wgrad_prox
    f.argtypes = [i32, i32, i32, vp, i64, vp, i64, C.c_int, i64, vp, vp, vp, vp, vp, f32, f32, vp, i64, vp, vp,
                  C.c_size_t, vp]
    g = lib.csr_recompress_counted
    g.argtypes = [i32, i32, vp, i64, vp, vp, vp, vp, i64, vp, vp, vp, C.c_size_t, vp]
    bb = lib.csr_bitmap_build
    bb.argtypes = [i32, i32, i64, vp, vp, vp, vp, vp]
    N, K, B, nnz = 64, 100, 16, 300
    names = ["dY", "X", "rp", "ci", "v", "Z", "wc", "mk", "ps", "rpo", "cio", "vo", "ws"]
    base = {n: (i + 1) << 26 for i, n in enumerate(names)}

    def prox(**o):
        a = dict(base)
        a.update({k: v for k, v in o.items() if k in a})
        p = {k: (None if x is None else C.c_void_p(x)) for k, x in a.items()}
        return f(o.get("N", N), o.get("K", K), B, p["dY"], o.get("ldy", B), p["X"], B, o.get("prec", 0), nnz,
                 p["rp"], p["ci"], p["v"], p["mk"], p["ps"], o.get("eta", 0.01), o.get("lam", 1e-4), p["Z"],
                 o.get("ldz", K), p["wc"], p["ws"], 0, S)

    def rec(**o):
        a = dict(base)
        a.update({k: v for k, v in o.items() if k in a})
        p = {k: (None if x is None else C.c_void_p(x)) for k, x in a.items()}
        return g(o.get("N", N), o.get("K", K), p["Z"], o.get("ldz", K), p["wc"], p["rpo"], p["cio"], p["vo"],
                 N * K, None, None, p["ws"], o.get("wsb", lib.l1csr_workspace_bytes(2, N, K, 0, 0)), S)

    assert lib.l1csr_workspace_bytes(9, N, K, nnz, B) == 0  # no split at this shape
    assert prox() == EHIP and rec() == EHIP  # valid: only the launch fails without a GPU
    for bad in [dict(prec=3), dict(N=-1), dict(eta=0.0), dict(lam=float("nan")), dict(ldy=B - 1), dict(ldz=K - 1),
                dict(mk=None), dict(ps=None), dict(wc=None), dict(Z=base["dY"] + 8), dict(wc=base["Z"] + 4),
                dict(Z=base["mk"] + 4), dict(wc=base["ci"])]:
        assert prox(**bad) == EINVAL, bad
    assert prox(N=65536, K=65536, ldz=65536) == EUNSUPPORTED
    # the workspace: row totals (N + 1) and one total per block of 16 or more rows
    assert lib.l1csr_workspace_bytes(2, N, K, 0, 0) >= 4 * (N + 1 + (N + 15) // 16)
    for bad in [dict(N=-1), dict(ldz=K - 1), dict(wc=None), dict(rpo=None), dict(wsb=4 * (N + 1)), dict(ws=None),
                dict(cio=base["Z"] + 4), dict(vo=base["wc"]), dict(rpo=base["cio"] + 4 * (N * K - 1)),
                dict(vo=base["ws"])]:
        assert rec(**bad) == EINVAL, bad
    assert rec(N=65536, K=65536, ldz=65536) == EUNSUPPORTED
    P, Q = C.c_void_p(1 << 26), C.c_void_p(2 << 26)
    assert bb(-1, 4, 0, P, P, P, Q, S) == EINVAL
    assert bb(4, 4, 3, P, P, None, Q, S) == EINVAL
    assert bb(4, 64, 3, P, P, P, C.c_void_p((1 << 26) + 8), S) == EINVAL  # mask and pos overlap


def test_planned_product_arguments_are_rejected_before_launch(lib):
    """csr_spmm_plan / csr_spmm_planned check the CSR, B, the dense operands
    and the plan buffer on the host; a shape without a tiled plan needs no
    buffer and enqueues nothing."""
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    pl = lib.csr_spmm_plan
    pl.argtypes = [i32, i32, i64, vp, vp, vp, i32, vp, sz, vp]
    pd = lib.csr_spmm_planned
    pd.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, i32, vp, i64, vp, sz, vp]
    names = ["rp", "ci", "v", "X", "Y", "plan"]
    base = {n: (i + 1) << 30 for i, n in enumerate(names)}
    N, K, B, nnz = 4096, 512, 512, 400000
    need = lib.l1csr_workspace_bytes(4, N, K, nnz, B)  # L1CSR_OP_SPMM
    assert need > 0  # the tiled path at this shape

    def args(o):
        a = dict(base)
        a.update({k: v for k, v in o.items() if k in a})
        return {k: (None if x is None else C.c_void_p(x)) for k, x in a.items()}

    def plan(**o):
        p = args(o)
        return pl(o.get("N", N), K, nnz, p["rp"], p["ci"], p["v"], o.get("B", B), p["plan"], o.get("pb", need), S)

    def planned(**o):
        p = args(o)
        return pd(o.get("N", N), K, nnz, p["rp"], p["ci"], p["v"], p["X"], o.get("ldx", B), o.get("B", B), p["Y"],
                  o.get("ldy", B), p["plan"], o.get("pb", need), S)

    assert plan() == EHIP and planned() == EHIP  # valid: only the launch fails without a GPU
    for bad in [dict(B=-1), dict(N=-1), dict(rp=None), dict(plan=None), dict(pb=need - 1)]:
        assert plan(**bad) == EINVAL, bad
    for bad in [dict(B=-1), dict(rp=None), dict(X=None), dict(ldx=B - 1), dict(ldy=B - 1), dict(plan=None),
                dict(pb=need - 1), dict(Y=base["plan"] + 4096)]:
        assert planned(**bad) == EINVAL, bad
    # no tiled plan at a small shape: nothing to plan, no buffer needed
    assert lib.l1csr_workspace_bytes(4, 64, 100, 300, 16) == 0
    assert pl(64, 100, 300, C.c_void_p(1 << 30), C.c_void_p(2 << 30), C.c_void_p(3 << 30), 16, None, 0, S) == OK


def test_mapped_host_memory_arguments_are_checked(lib):
    """l1csr_host_alloc_mapped rejects a zero size and missing out-pointers
    before it asks the runtime for anything; freeing NULL is an error too."""
    a = lib.l1csr_host_alloc_mapped
    a.argtypes = [C.c_size_t, C.POINTER(C.c_void_p), C.POINTER(C.c_void_p)]
    f = lib.l1csr_host_free_mapped
    f.argtypes = [C.c_void_p]
    h, d = C.c_void_p(), C.c_void_p()
    assert a(0, C.byref(h), C.byref(d)) == EINVAL
    assert a(64, None, C.byref(d)) == EINVAL
    assert a(64, C.byref(h), None) == EINVAL
    assert f(None) == EINVAL


def test_binding_and_torch_share_one_hip_runtime():
    """The binding loads the library after torch, so that the library binds
    torch's own HIP runtime: a second runtime in the process would not know
    torch's streams or memory.  Checked in a fresh interpreter that asks for
    the library before anything else imports torch."""
    import ast
    import subprocess
    import sys
    if not os.path.exists(LIB):
        from paper_1905_07931_amd import build
        build.build(verbose=False)
    code = ("import paper_1905_07931_amd as L1\n"
            "L1.lib()\n"
            "import torch\n"
            "print(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    runtimes = ast.literal_eval(r.stdout.strip().splitlines()[-1])
    assert len(runtimes) == 1, runtimes
