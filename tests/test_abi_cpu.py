"""The C ABI without a GPU: the library loads, exports every declared symbol
and rejects invalid arguments before touching the HIP runtime."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2512_04632_amd import _lib as tm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "turbomuon.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w ]*\*?\s*(tm_\w+)\s*\(", text, re.M)))


def header_defines():
    text = open(HEADER).read()
    return {k: int(v) for k, v in re.findall(r"#define\s+(TM_\w+)\s+\(?(-?\d+)\)?", text)}


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 9
    L = tm.lib()
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(tm._SIGNATURES)


def test_constants_match_header():
    d = header_defines()
    assert d["TM_OK"] == tm.TM_OK and d["TM_ERR_INVALID_ARG"] == tm.TM_ERR_INVALID_ARG
    assert d["TM_ERR_UNSUPPORTED"] == tm.TM_ERR_UNSUPPORTED
    assert d["TM_ERR_NO_MEMORY"] == tm.TM_ERR_NO_MEMORY and d["TM_ERR_HIP"] == tm.TM_ERR_HIP
    assert d["TM_PRECOND_NONE"] == tm.PRECOND["none"]
    assert d["TM_PRECOND_FROBENIUS"] == tm.PRECOND["frobenius"]
    assert d["TM_PRECOND_AOL"] == tm.PRECOND["aol"]
    assert d["TM_PRECOND_SCHATTEN4"] == tm.PRECOND["schatten4"]
    phases = {k[len("TM_PHASE_"):].lower(): v for k, v in d.items() if k.startswith("TM_PHASE_")}
    assert phases == tm.PHASES and d["TM_NUM_PHASES"] == len(tm.PHASES)
    assert d["TM_MAX_DIM"] == tm.TM_MAX_DIM and d["TM_MAX_ITERS"] == tm.TM_MAX_ITERS


def test_status_strings_and_version():
    for code, name in [(0, "TM_OK"), (-1, "TM_ERR_INVALID_ARG"), (-2, "TM_ERR_UNSUPPORTED"),
                       (-3, "TM_ERR_NO_MEMORY"), (-4, "TM_ERR_HIP")]:
        assert tm.status_string(code) == name
    assert tm.status_string(7) == "TM_ERR_UNKNOWN"
    assert re.fullmatch(r"\d+\.\d+\.\d+", tm.version())


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails or batch = 0


@pytest.mark.parametrize("fn", ["tm_orthogonalize", "tm_orthogonalize_f32"])
@pytest.mark.parametrize("m,n,batch,iters,precond,code", [
    (0, 4, 1, 4, 2, tm.TM_ERR_INVALID_ARG),
    (4, 0, 1, 4, 2, tm.TM_ERR_INVALID_ARG),
    (-3, 4, 1, 4, 2, tm.TM_ERR_INVALID_ARG),
    (65537, 4, 1, 4, 2, tm.TM_ERR_INVALID_ARG),
    (4, 4, -1, 4, 2, tm.TM_ERR_INVALID_ARG),
    (4, 4, 1, -1, 2, tm.TM_ERR_INVALID_ARG),
    (4, 4, 1, 65, 2, tm.TM_ERR_INVALID_ARG),
    (4, 4, 1, 4, 4, tm.TM_ERR_INVALID_ARG),
    (4, 4, 1, 4, -1, tm.TM_ERR_INVALID_ARG),
    (4, 4, 0, 4, 2, tm.TM_OK),                 # empty batch: no-op
])
def test_batched_validation(fn, m, n, batch, iters, precond, code):
    f = getattr(tm.lib(), fn)
    assert f(FAKE, m, n, batch, iters, None, precond, None) == code
    if code != tm.TM_OK:
        assert tm.last_error() != ""


def test_null_and_misaligned_pointers():
    L = tm.lib()
    assert L.tm_orthogonalize(None, 4, 4, 1, 4, None, 2, None) == tm.TM_ERR_INVALID_ARG
    assert L.tm_orthogonalize(ctypes.c_void_p(0x1001), 4, 4, 1, 4, None, 2, None) == tm.TM_ERR_UNSUPPORTED
    assert L.tm_orthogonalize_f32(ctypes.c_void_p(0x1002), 4, 4, 1, 4, None, 2, None) == tm.TM_ERR_UNSUPPORTED
    # a null pointer with an empty batch is still a no-op
    assert L.tm_orthogonalize(None, 4, 4, 0, 4, None, 2, None) == tm.TM_OK


@pytest.mark.parametrize("fn", ["tm_orthogonalize_grouped", "tm_orthogonalize_grouped_f32"])
def test_grouped_validation(fn):
    f = getattr(tm.lib(), fn)
    ptrs = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    ms = (ctypes.c_int64 * 2)(8, 16)
    ns = (ctypes.c_int64 * 2)(8, 0)
    assert f(ptrs, ms, ns, 2, 4, None, 2, None) == tm.TM_ERR_INVALID_ARG
    assert "matrix 1" in tm.last_error()
    ns[1] = 4
    assert f(ptrs, ms, ns, 2, 4, None, 9, None) == tm.TM_ERR_INVALID_ARG
    assert f(ptrs, ms, ns, -1, 4, None, 2, None) == tm.TM_ERR_INVALID_ARG
    assert f(None, ms, ns, 2, 4, None, 2, None) == tm.TM_ERR_INVALID_ARG
    nulls = (ctypes.c_void_p * 2)(0x1000, None)
    assert f(nulls, ms, ns, 2, 4, None, 2, None) == tm.TM_ERR_INVALID_ARG
    assert f(ptrs, ms, ns, 0, 4, None, 2, None) == tm.TM_OK


def test_workspace_bytes():
    # per matrix: two Y buffers (kp x Np), A and B (kp x kp), the fp32 first Gram,
    # s, the row-sum partials [ceil(kp/64)][kp] and 32 Frobenius partials
    def a256(v):
        return (v + 255) // 256 * 256

    def layout(kp, Np, e):
        return (2 * a256(kp * Np * e) + 2 * a256(kp * kp * e) + a256(4 * kp * kp) + a256(4 * kp)
                + a256(4 * kp * ((kp + 63) // 64)) + a256(4 * 32))

    shapes = [(768, 3072), (3072, 768), (17, 33), (1, 1)]
    # fp32: A and B rows padded to 8, Y unpadded
    f32 = sum(layout((min(m, n) + 7) // 8 * 8, max(m, n), 4) for m, n in shapes)
    assert tm.workspace_bytes(shapes, 4) == f32
    # bf16: every dim padded to the call's square tile T (one of 256, 128, 64)
    bf = tm.workspace_bytes(shapes, 2)
    cands = [sum(layout(-(-min(m, n) // T) * T, -(-max(m, n) // T) * T, 2) for m, n in shapes)
             for T in (256, 128, 64)]
    assert bf in cands
    assert tm.workspace_bytes([(4096, 14336)], 2) == layout(4096, 14336, 2)
    assert tm.workspace_bytes([(0, 4)], 2) == 0
    assert tm.workspace_bytes([(4, 4)], 3) == 0


def test_muon_step_validation():
    f = tm.lib().tm_muon_step_grouped
    P3 = ctypes.c_void_p * 2
    W, G, M = P3(0x1000, 0x2000), P3(0x3000, 0x4000), P3(0x5000, 0x6000)
    ms = (ctypes.c_int64 * 2)(8, 16)
    ns = (ctypes.c_int64 * 2)(8, 4)
    args = (0.02, 0.95, 1, 0.0, 1, 4, None, 2, None)
    assert f(W, G, M, ms, ns, 0, *args) == tm.TM_OK                    # empty group: no-op
    assert f(W, G, M, ms, ns, -1, *args) == tm.TM_ERR_INVALID_ARG
    assert f(None, G, M, ms, ns, 2, *args) == tm.TM_ERR_INVALID_ARG
    ns[1] = 0
    assert f(W, G, M, ms, ns, 2, *args) == tm.TM_ERR_INVALID_ARG
    assert "matrix 1" in tm.last_error()
    ns[1] = 4
    M[1] = None
    assert f(W, G, M, ms, ns, 2, *args) == tm.TM_ERR_INVALID_ARG
    M[1] = 0x6002
    assert f(W, G, M, ms, ns, 2, *args) == tm.TM_ERR_UNSUPPORTED
    M[1] = 0x6000
    assert f(W, G, M, ms, ns, 2, 0.02, 0.95, 1, 0.0, 1, 65, None, 2, None) == tm.TM_ERR_INVALID_ARG
    assert f(W, G, M, ms, ns, 2, 0.02, 0.95, 1, 0.0, 1, 4, None, 7, None) == tm.TM_ERR_INVALID_ARG


def test_optimizer_rejects_non_matrix_parameters():
    torch = pytest.importorskip("torch")
    from paper_2512_04632_amd.optim import TurboMuon
    with pytest.raises(ValueError):
        TurboMuon([torch.nn.Parameter(torch.zeros(5))])
    with pytest.raises(ValueError):
        TurboMuon([torch.nn.Parameter(torch.zeros(4, 4, dtype=torch.float64))])
    TurboMuon([torch.nn.Parameter(torch.zeros(4, 6))], lr=0.1)


def test_schedule_tail_points_at_the_last_rows():
    """tm_schedule_tail returns the last `iters` rows of a schedule (values rounded
    to float32 only) and rejects out-of-range requests."""
    sched = [(3.0, -3.5, 1.5), (2.6, -2.7, 1.1), (2.2, -1.9, 0.7), (1.875, -1.25, 0.375),
             (1.6, -0.7, 0.1)]
    f32 = lambda rows: [tuple(float(np.float32(v)) for v in r) for r in rows]  # noqa: E731
    assert tm.schedule_tail(sched, 4) == f32(sched[1:])
    assert tm.schedule_tail(sched, 5) == f32(sched)
    assert tm.schedule_tail(sched, 1) == f32(sched[4:])
    assert tm.schedule_tail(sched, 0) == []
    for bad in (6, -1):
        with pytest.raises(tm.TurboMuonError):
            tm.schedule_tail(sched, bad)
    L = tm.lib()
    assert not L.tm_schedule_tail(None, 3, 1)
    arr = (ctypes.c_float * 3)(1.0, 2.0, 3.0)
    assert not L.tm_schedule_tail(arr, 0, 0)
    assert not L.tm_schedule_tail(arr, tm.TM_MAX_ITERS + 1, 1)
    base = ctypes.cast(arr, ctypes.c_void_p).value
    p = L.tm_schedule_tail(arr, 1, 0)
    assert ctypes.cast(p, ctypes.c_void_p).value == base + 12
