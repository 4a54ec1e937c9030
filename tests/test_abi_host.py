"""Host-side checks of the C ABI (CPU only): the library loads, exports every function that
include/tacg.h declares, sizes its workspaces, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_01007_amd as tacg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tacg.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tacg_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(tacg.LIB_PATH):
        pytest.skip("libtacg.so not built")
    return tacg.lib()


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert {"tacg_coact_build", "tacg_reweight", "tacg_eval_placements", "tacg_jain"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_coact_kernel_choice(L):
    """The co-activation build's kernel choice (a host-only query): matrix cores at E <= 64 from top-4,
    at E <= 128 for top-8 to top-12, the LDS histogram otherwise; 0 for shapes the build rejects."""
    use = L.tacg_coact_uses_matrix_cores
    assert [use(64, k) for k in (1, 2, 3, 4, 6, 16)] == [0, 0, 0, 1, 1, 1]
    assert [use(32, k) for k in (3, 4, 12)] == [0, 1, 1]
    assert [use(128, k) for k in (4, 6, 7, 8, 10, 12, 13, 16)] == [0, 0, 0, 1, 1, 1, 0, 0]
    assert [use(65, 8), use(129, 8), use(256, 8), use(256, 4)] == [1, 0, 0, 0]
    assert [use(0, 4), use(64, 0), use(64, 17), use(4, 6), use(257, 8), use(-1, 8)] == [0] * 6
    assert tacg.coact_uses_matrix_cores(60, 4) and not tacg.coact_uses_matrix_cores(256, 8)


def test_strerror(L):
    for code in (0, -1, -2, -3, 7):
        assert isinstance(L.tacg_strerror(code), bytes)


def test_workspace_sizes(L):
    # coact: (W + L*F) slots of the triangle; at E = 256 one workgroup per CU (256)
    tri = 256 * 255 // 2
    n = L.tacg_coact_workspace_bytes(1 << 23, 58, 8, 256, 16)
    assert n >= (256 + 58 * 16) * tri * 4 and n % 256 == 0
    assert L.tacg_coact_workspace_bytes(6144, 2, 2, 8, 3) >= 3 * 2 * 28 * 4
    assert L.tacg_coact_workspace_bytes(-1, 2, 2, 8, 3) == 0
    assert L.tacg_reweight_workspace_bytes(16, 58, 256) >= 58 * 256 * 256 * 8
    assert L.tacg_eval_workspace_bytes(1 << 23, 58, 256, 32, 1024, 16) > 0
    assert L.tacg_eval_workspace_bytes(10, 0, 8, 4, 1, 1) == 0


FAKE = ctypes.c_void_p(1 << 20)   # never dereferenced: every call below fails validation first


def _coact(L, **kw):
    a = dict(trace=FAKE, N=100, Ly=2, k=2, E=8, off=np.array([0, 50, 100], dtype=np.int64), F=2, D=FAKE, C=FAKE,
             flags=0, err=FAKE, ws=FAKE, wsb=1 << 30)
    a.update(kw)
    return L.tacg_coact_build(a["trace"], a["N"], a["Ly"], a["k"], a["E"],
                              a["off"].ctypes.data_as(ctypes.c_void_p) if a["off"] is not None else None,
                              a["F"], a["D"], a["C"], a["flags"], a["err"], a["ws"], a["wsb"], None)


def test_coact_argument_errors(L):
    assert _coact(L, Ly=0) == tacg.E_INVAL
    assert _coact(L, k=9) == tacg.E_INVAL                       # k > E
    assert _coact(L, E=300, k=2) == tacg.E_UNSUPPORTED
    assert _coact(L, k=17, E=32) == tacg.E_UNSUPPORTED
    assert _coact(L, off=np.array([0, 60, 50], dtype=np.int64)) == tacg.E_INVAL   # not monotone / end != N
    assert _coact(L, off=np.array([0, 60, 99], dtype=np.int64)) == tacg.E_INVAL
    assert _coact(L, off=np.array([1, 60, 100], dtype=np.int64)) == tacg.E_INVAL
    assert _coact(L, off=None) == tacg.E_INVAL
    assert _coact(L, trace=None) == tacg.E_INVAL
    assert _coact(L, trace=ctypes.c_void_p((1 << 20) + 2)) == tacg.E_INVAL   # misaligned trace
    assert _coact(L, D=None) == tacg.E_INVAL
    assert _coact(L, err=None) == tacg.E_INVAL
    assert _coact(L, flags=4) == tacg.E_INVAL
    assert _coact(L, wsb=16) == tacg.E_INVAL
    assert _coact(L, ws=ctypes.c_void_p((1 << 20) + 64)) == tacg.E_INVAL   # workspace not 256-aligned
    assert _coact(L, N=1 << 31, k=2, off=np.array([0, 1 << 30, 1 << 31], dtype=np.int64)) == tacg.E_UNSUPPORTED
    assert _coact(L, F=65, off=np.zeros(66, dtype=np.int64)) in (tacg.E_UNSUPPORTED, tacg.E_INVAL)


def test_reweight_argument_errors(L):
    f = L.tacg_reweight
    ok = dict(D=FAKE, C=FAKE, F=3, Ly=2, E=8, k=2, alpha=0.25, tau=1.0, eps=1e-8, pref=FAKE, at=FAKE, ah=None,
              ws=FAKE, wsb=1 << 30)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["D"], a["C"], a["F"], a["Ly"], a["E"], a["k"], a["alpha"], a["tau"], a["eps"], a["pref"],
                 a["at"], a["ah"], a["ws"], a["wsb"], None)

    assert call(F=1) == tacg.E_INVAL
    assert call(alpha=1.5) == tacg.E_INVAL
    assert call(tau=0.0) == tacg.E_INVAL
    assert call(eps=-1.0) == tacg.E_INVAL
    assert call(D=None) == tacg.E_INVAL
    assert call(wsb=8) == tacg.E_INVAL
    assert call(E=512) == tacg.E_UNSUPPORTED


def test_eval_argument_errors(L):
    off = np.array([0, 60, 100], dtype=np.int64)
    hs = np.array([0, 2], dtype=np.int32)
    hz = np.array([2, 2], dtype=np.int32)

    def call(G=4, P=3, R=0, sec=None, ref=None, hs_=hs, hz_=hz, flags=0, tn=3, td=20, wsb=1 << 30, off_=off):
        return L.tacg_eval_placements(FAKE, 100, 2, 2, 8, off_.ctypes.data_as(ctypes.c_void_p), 2,
                                      hs_.ctypes.data_as(ctypes.c_void_p), hz_.ctypes.data_as(ctypes.c_void_p),
                                      G, P, FAKE, sec, R, ref, tn, td, FAKE, FAKE, FAKE, None, flags, FAKE, FAKE,
                                      wsb, None)

    assert call(G=33) == tacg.E_UNSUPPORTED
    assert call(G=0) == tacg.E_INVAL
    assert call(P=0) == tacg.E_INVAL
    assert call(R=5, sec=FAKE, ref=FAKE) == tacg.E_UNSUPPORTED
    assert call(R=2, sec=None, ref=FAKE) == tacg.E_INVAL
    assert call(R=2, sec=FAKE, ref=None) == tacg.E_INVAL
    assert call(hz_=np.array([2, 0], dtype=np.int32)) == tacg.E_INVAL
    assert call(hs_=np.array([0, 3], dtype=np.int32)) == tacg.E_INVAL     # band past G
    assert call(flags=1) == tacg.E_INVAL
    assert call(tn=-1) == tacg.E_INVAL
    assert call(tn=(1 << 20) + 1) == tacg.E_INVAL
    assert call(td=(1 << 20) + 1) == tacg.E_INVAL
    assert call(wsb=1) == tacg.E_INVAL
    assert call(off_=np.array([0, 60, 90], dtype=np.int64)) == tacg.E_INVAL


def test_eval_trace_stats_argument_errors(L):
    off = np.array([0, 60, 100], dtype=np.int64)
    hs = np.array([0, 2], dtype=np.int32)
    hz = np.array([2, 2], dtype=np.int32)

    def call(G=4, P=3, hs_=hs, hz_=hz, flags=0, wsb=1 << 30, sf=FAKE, cf=FAKE, mf=FAKE):
        return L.tacg_eval_trace_stats(FAKE, 100, 2, 2, 8, off.ctypes.data_as(ctypes.c_void_p), 2,
                                       hs_.ctypes.data_as(ctypes.c_void_p), hz_.ctypes.data_as(ctypes.c_void_p),
                                       G, P, FAKE, None, 0, None, 3, 20, FAKE, FAKE, FAKE, sf, cf, mf, flags, FAKE,
                                       FAKE, wsb, None)

    assert call(G=33) == tacg.E_UNSUPPORTED
    assert call(P=0) == tacg.E_INVAL
    assert call(flags=1) == tacg.E_INVAL
    assert call(wsb=1) == tacg.E_INVAL
    assert call(sf=None) == tacg.E_INVAL
    assert call(cf=None) == tacg.E_INVAL
    assert call(mf=None) == tacg.E_INVAL
    # the distinct family bands must tile the GPUs: overlapping bands, or a GPU outside every band
    assert call(hs_=np.array([0, 1], dtype=np.int32), hz_=np.array([2, 3], dtype=np.int32)) == tacg.E_UNSUPPORTED
    assert call(hs_=np.array([0, 0], dtype=np.int32), hz_=np.array([2, 2], dtype=np.int32)) == tacg.E_UNSUPPORTED
    assert call(hs_=np.array([0, 0], dtype=np.int32), hz_=np.array([2, 4], dtype=np.int32)) == tacg.E_UNSUPPORTED


def test_eval_online_argument_errors(L):
    off = np.array([0, 60, 100], dtype=np.int64)
    hs = np.array([0, 2], dtype=np.int32)
    hz = np.array([2, 2], dtype=np.int32)

    def call(G=4, P=3, R=0, sec=None, rho=0.995, hs_=hs, hz_=hz, flags=0, tn=3, td=20, off_=off, ch=FAKE):
        return L.tacg_eval_online(FAKE, 100, 2, 2, 8, off_.ctypes.data_as(ctypes.c_void_p), 2,
                                  hs_.ctypes.data_as(ctypes.c_void_p), hz_.ctypes.data_as(ctypes.c_void_p),
                                  G, P, FAKE, sec, R, rho, tn, td, None, None, ch, FAKE, FAKE, None, flags, FAKE,
                                  None)

    assert call(G=33) == tacg.E_UNSUPPORTED
    assert call(G=0) == tacg.E_INVAL
    assert call(P=0) == tacg.E_INVAL
    assert call(R=5, sec=FAKE) == tacg.E_UNSUPPORTED
    assert call(R=2, sec=None) == tacg.E_INVAL
    assert call(rho=1.0) == tacg.E_INVAL
    assert call(rho=-0.1) == tacg.E_INVAL
    assert call(rho=float("nan")) == tacg.E_INVAL
    assert call(hz_=np.array([2, 0], dtype=np.int32)) == tacg.E_INVAL
    assert call(hs_=np.array([0, 3], dtype=np.int32)) == tacg.E_INVAL
    assert call(flags=1) == tacg.E_INVAL
    assert call(td=-1) == tacg.E_INVAL
    assert call(tn=(1 << 20) + 1) == tacg.E_INVAL
    assert call(td=(1 << 20) + 1) == tacg.E_INVAL
    assert call(ch=None) == tacg.E_INVAL
    assert call(off_=np.array([0, 60, 90], dtype=np.int64)) == tacg.E_INVAL


def test_diagnostics_argument_errors(L):
    assert L.tacg_activation_distance(None, 2, 2, 8, 2, FAKE, None) == tacg.E_INVAL
    assert L.tacg_activation_distance(FAKE, 2, 2, 300, 2, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_pair_jaccard(FAKE, 2, 2, 1, 64, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_pair_jaccard(FAKE, 2, 2, 8, 0, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_pair_jaccard(FAKE, 2, 2, 8, 5000, FAKE, FAKE, None) == tacg.E_UNSUPPORTED


def test_gesr_scores_argument_errors(L):
    assert L.tacg_gesr_scores(FAKE, FAKE, 2, 2, 300, 2, FAKE, FAKE, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_gesr_scores(FAKE, FAKE, 0, 2, 8, 2, FAKE, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_gesr_scores(FAKE, FAKE, 2, 2, 8, 9, FAKE, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_gesr_scores(None, FAKE, 2, 2, 8, 2, FAKE, FAKE, FAKE, None) == tacg.E_INVAL


def test_group_objective_argument_errors(L):
    assert L.tacg_group_objective(FAKE, 2, 300, FAKE, 3, 4, FAKE, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_group_objective(FAKE, 2, 8, FAKE, 3, 40, FAKE, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_group_objective(None, 2, 8, FAKE, 3, 4, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_group_objective(FAKE, 0, 8, FAKE, 3, 4, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_group_objective(FAKE, 2, 8, FAKE, 0, 4, FAKE, FAKE, None) == tacg.OK      # nothing to do


def test_jain_and_load_argument_errors(L):
    assert L.tacg_jain(FAKE, 2, 1, 33, 0, FAKE, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_jain(FAKE, 2, 1, 4, 2, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_jain(None, 2, 1, 4, 0, FAKE, FAKE, None) == tacg.E_INVAL
    assert L.tacg_jain(FAKE, 0, 1, 4, 0, FAKE, FAKE, None) == tacg.OK        # nothing to do
    assert L.tacg_placement_load(FAKE, 2, 2, 8, FAKE, 3, 40, FAKE, FAKE, None) == tacg.E_UNSUPPORTED
    assert L.tacg_placement_load(None, 2, 2, 8, FAKE, 3, 4, FAKE, FAKE, None) == tacg.E_INVAL


def test_binding_refuses_host_tensors():
    import torch
    if not os.path.exists(tacg.LIB_PATH):
        pytest.skip("libtacg.so not built")
    tr = torch.zeros((1, 4, 2), dtype=torch.int16)
    with pytest.raises(ValueError):
        tacg.coact_build(tr, [0, 4], 8, D=torch.zeros((1, 1, 8), dtype=torch.int32),
                         C=torch.zeros((1, 1, 8, 8), dtype=torch.int32), ws=torch.zeros(1 << 12, dtype=torch.uint8),
                         err=torch.zeros(1, dtype=torch.int32))


def test_binding_checks_element_types_and_shapes():
    """A tensor of another element type or shape than the C ABI assumes is refused before any call
    (a kernel would otherwise read or write past a smaller buffer).  Without a GPU the public calls
    stop at the first tensor argument (host tensors are refused too), so the later arguments' check is
    exercised through the helper that every call uses."""
    import torch
    if not os.path.exists(tacg.LIB_PATH):
        pytest.skip("libtacg.so not built")
    ws = torch.zeros(1 << 12, dtype=torch.uint8)
    err = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(ValueError, match="trace"):
        tacg.coact_build(torch.zeros((1, 4, 2), dtype=torch.int32), [0, 4], 8, ws=ws, err=err)
    with pytest.raises(ValueError, match="trace"):
        tacg.coact_build(torch.zeros((4, 2), dtype=torch.int16), [0, 4], 8, ws=ws, err=err)
    with pytest.raises(ValueError, match="trace"):
        tacg.eval_placements(torch.zeros((1, 4, 2), dtype=torch.int64), [0, 4], 8, [0], [1], 1,
                             torch.zeros((1, 1, 8), dtype=torch.uint8))
    with pytest.raises(ValueError, match="load: expected torch.int32"):
        tacg.jain_index(torch.zeros((2, 1, 4), dtype=torch.int64))
    with pytest.raises(ValueError, match="a_tilde: expected torch.float32"):
        tacg.group_objective(torch.zeros((1, 8, 8), dtype=torch.float64), torch.zeros((2, 1, 8), dtype=torch.uint8), 4,
                             err=err)
    with pytest.raises(ValueError, match="D: expected"):
        tacg.placement_load(torch.zeros((1, 1, 8), dtype=torch.int16), torch.zeros((2, 1, 8), dtype=torch.uint8), 4,
                            err=err)
    # the helper: element type, then shape, then device
    with pytest.raises(ValueError, match=r"D: expected torch.int32 \(1, 1, 8\), got torch.int16"):
        tacg._arg(torch.zeros((1, 1, 8), dtype=torch.int16), "D", torch.int32, (1, 1, 8))
    with pytest.raises(ValueError, match=r"primary: expected torch.uint8 \(2, 1, 8\), got torch.uint8 \(2, 1, 9\)"):
        tacg._arg(torch.zeros((2, 1, 9), dtype=torch.uint8), "primary", torch.uint8, (2, 1, 8))
    with pytest.raises(ValueError, match="device tensor"):
        tacg._arg(torch.zeros((2, 1, 8), dtype=torch.uint8), "primary", torch.uint8, (2, 1, 8))
    assert tacg._arg(None, "secondary", torch.uint8, (1,)) is None


def test_binding_checks_family_offsets_and_bands():
    """The C ABI reads F + 1 family offsets and F entries of each home-band array; a shorter or
    multi-dimensional list is refused with ValueError before any call (it would otherwise be an
    out-of-bounds host read)."""
    import torch
    if not os.path.exists(tacg.LIB_PATH):
        pytest.skip("libtacg.so not built")
    tr = torch.zeros((1, 4, 2), dtype=torch.int16)
    prim = torch.zeros((1, 1, 8), dtype=torch.uint8)
    for call in (tacg.eval_placements, tacg.eval_trace_stats, tacg.eval_online):
        with pytest.raises(ValueError, match="home_start / home_size"):
            call(tr, [0, 2, 4], 8, [0], [1, 1], 2, prim)            # F = 2, one start
        with pytest.raises(ValueError, match="home_start / home_size"):
            call(tr, [0, 2, 4], 8, [0, 1], [1], 2, prim)            # F = 2, one size
        with pytest.raises(ValueError, match="home_start / home_size"):
            call(tr, [0, 4], 8, [[0]], [[1]], 2, prim)              # not 1-D
        with pytest.raises(ValueError, match="fam_off"):
            call(tr, [4], 8, [], [], 2, prim)                       # no family
        with pytest.raises(ValueError, match="fam_off"):
            call(tr, [[0, 4]], 8, [0], [1], 2, prim)                # not 1-D
    with pytest.raises(ValueError, match="fam_off"):
        tacg.coact_build(tr, [4], 8)


def _noalloc(L, **kw):
    a = dict(trace=FAKE, N=100, Ly=2, k=2, E=8, off=np.array([0, 50, 100], dtype=np.int64), F=2,
             hs=np.array([0, 1], dtype=np.int32), hz=np.array([1, 1], dtype=np.int32), G=2, P=4, prim=FAKE,
             sec=None, R=0, ref=None, tn=3, td=20, ch=FAKE, cs=FAKE, load=FAKE, fam=None, flags=0, err=FAKE)
    a.update(kw)
    return L.tacg_eval_placements_noalloc(
        a["trace"], a["N"], a["Ly"], a["k"], a["E"], a["off"].ctypes.data_as(ctypes.c_void_p), a["F"],
        a["hs"].ctypes.data_as(ctypes.c_void_p), a["hz"].ctypes.data_as(ctypes.c_void_p), a["G"], a["P"],
        a["prim"], a["sec"], a["R"], a["ref"], a["tn"], a["td"], a["ch"], a["cs"], a["load"], a["fam"], a["flags"],
        a["err"], None)


def test_noalloc_argument_errors_and_scratch_limit(L):
    """The no-allocation entry point checks its arguments like tacg_eval_placements and refuses, before
    anything is enqueued, an input whose scratch need exceeds the fixed device array."""
    assert tacg.NOALLOC_SCRATCH_BYTES == 32 << 20
    assert _noalloc(L, G=0) == tacg.E_INVAL
    assert _noalloc(L, G=33) == tacg.E_UNSUPPORTED
    assert _noalloc(L, prim=None) == tacg.E_INVAL
    assert _noalloc(L, R=1) == tacg.E_INVAL                    # secondaries without tables
    assert _noalloc(L, flags=1) == tacg.E_INVAL
    assert _noalloc(L, hz=np.array([1, 2], dtype=np.int32)) == tacg.E_INVAL   # band past G
    # 58 layers, E = 256, G = 32, 16 families: about 2100 placements fit in 32 MiB
    big = dict(N=1 << 10, Ly=58, k=8, E=256, off=np.linspace(0, 1 << 10, 17).astype(np.int64), F=16,
               hs=np.arange(16, dtype=np.int32) * 2, hz=np.full(16, 2, dtype=np.int32), G=32)
    fits = [P for P in range(1900, 2300) if L.tacg_eval_workspace_bytes(1 << 10, 58, 256, 32, P, 16)
            <= tacg.NOALLOC_SCRATCH_BYTES]
    assert fits and fits[0] == 1900 and 2000 < fits[-1] < 2299
    assert _noalloc(L, P=fits[-1] + 1, **big) == tacg.E_SCRATCH
    assert b"no-allocation" in L.tacg_strerror(tacg.E_SCRATCH)
