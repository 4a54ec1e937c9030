"""MI355X-native trace passes of TACG/GESR (task-aware co-activation grouping with generic-expert
shared replication).

Thin ctypes binding of libtacg.so (HIP kernels for gfx950 behind the C ABI of include/tacg.h).
PyTorch supplies device memory and the current HIP stream; every step runs in the library's
kernels.  There is no fallback: if the library or the GPU is missing, the calls raise.

    D, C, err = coact_build(trace, fam_off, n_experts)
    pref, a_tilde, a_hat = reweight(D, C, top_k, alpha=0.25, tau=1.0, eps=1e-8)
    load_ref = placement_load(D, primary, n_gpus)
    out = eval_placements(trace, fam_off, n_experts, home_start, home_size, n_gpus, primary,
                          secondary, load_ref, theta=(3, 20))
    jain, maxvio = jain_index(out["load"])

Unsigned 32-bit device outputs are held in torch.int32 tensors (same bits) and unsigned 64-bit ones in
torch.int64 tensors; `as_u32` converts the former to int64 values.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# TACG_LIBRARY names another build of the library to load (a host-sanitized build, for instance)
LIB_PATH = os.environ.get("TACG_LIBRARY") or os.path.join(_PKG, "libtacg.so")

OK, E_INVAL, E_UNSUPPORTED, E_DEVICE, E_SCRATCH = 0, -1, -2, -3, -4
NOALLOC_SCRATCH_BYTES = 32 << 20
ERR_ID_RANGE, ERR_ID_DUP, ERR_TABLE, ERR_LIMIT = 0x1, 0x2, 0x4, 0x8
ACCUMULATE = 0x1
NONE = 0xFF

_lock = threading.Lock()
_lib = None


class TacgError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({lib().tacg_strerror(status).decode()})")
        self.status = status


def lib():
    """The loaded libtacg.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_01007_amd.build`")
            L = ctypes.CDLL(LIB_PATH)
            P, i32, i64, u32, sz, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                         ctypes.c_size_t, ctypes.c_double)
            L.tacg_coact_build.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, u32, P, P, sz, P]
            L.tacg_coact_workspace_bytes.argtypes = [i64, i32, i32, i32, i32]
            L.tacg_coact_workspace_bytes.restype = sz
            L.tacg_coact_uses_matrix_cores.argtypes = [i32, i32]
            L.tacg_coact_uses_matrix_cores.restype = ctypes.c_int
            L.tacg_reweight.argtypes = [P, P, i32, i32, i32, i32, f64, f64, f64, P, P, P, P, sz, P]
            L.tacg_reweight_workspace_bytes.argtypes = [i32, i32, i32]
            L.tacg_reweight_workspace_bytes.restype = sz
            L.tacg_placement_load.argtypes = [P, i32, i32, i32, P, i32, i32, P, P, P]
            L.tacg_eval_placements.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, P, P, i32, P, i32, i32,
                                               P, P, P, P, u32, P, P, sz, P]
            L.tacg_eval_placements_noalloc.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, P, P, i32, P,
                                                       i32, i32, P, P, P, P, u32, P, P]
            L.tacg_eval_trace_stats.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, P, P, i32, P, i32,
                                                i32, P, P, P, P, P, P, u32, P, P, sz, P]
            L.tacg_eval_workspace_bytes.argtypes = [i64, i32, i32, i32, i32, i32]
            L.tacg_eval_workspace_bytes.restype = sz
            L.tacg_eval_online.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, P, P, i32, f64, i32, i32,
                                           P, P, P, P, P, P, u32, P, P]
            L.tacg_activation_distance.argtypes = [P, i32, i32, i32, i32, P, P]
            L.tacg_pair_jaccard.argtypes = [P, i32, i32, i32, i32, P, P, P]
            L.tacg_gesr_scores.argtypes = [P, P, i32, i32, i32, i32, P, P, P, P]
            L.tacg_group_objective.argtypes = [P, i32, i32, P, i32, i32, P, P, P]
            L.tacg_jain.argtypes = [P, i32, i32, i32, i32, P, P, P]
            L.tacg_strerror.argtypes = [ctypes.c_int]
            L.tacg_strerror.restype = ctypes.c_char_p
            for name in ("tacg_coact_build", "tacg_reweight", "tacg_placement_load", "tacg_eval_placements",
                         "tacg_eval_placements_noalloc", "tacg_eval_trace_stats", "tacg_jain"):
                getattr(L, name).restype = ctypes.c_int
            _lib = L
    return _lib


def _check(fn: str, status: int):
    if status != OK:
        raise TacgError(fn, status)


def _dptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _arg(t: Optional[torch.Tensor], name: str, dtype: torch.dtype, shape) -> Optional[ctypes.c_void_p]:
    """Device pointer of `t` after checking the element type and shape the C ABI assumes (a kernel
    would otherwise read or write past a smaller buffer)."""
    if t is None:
        return None
    if t.dtype != dtype or tuple(t.shape) != tuple(int(x) for x in shape):
        raise ValueError(f"{name}: expected {dtype} {tuple(int(x) for x in shape)}, got {t.dtype} {tuple(t.shape)}")
    return _dptr(t)


def _trace_dims(trace: torch.Tensor):
    if trace.dtype != torch.int16 or trace.dim() != 3:
        raise ValueError(f"trace: expected int16 [L][N][k], got {trace.dtype} {tuple(trace.shape)}")
    return trace.shape


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _host_i64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int64))


def _host_i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _hptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _fam_off(fam_off) -> np.ndarray:
    """fam_off as int64 [F+1] with F >= 1 (the C ABI reads F + 1 entries)."""
    off = _host_i64(fam_off)
    if off.ndim != 1 or off.size < 2:
        raise ValueError(f"fam_off: expected a 1-D sequence of F + 1 >= 2 offsets, got shape {off.shape}")
    return off


def _bands(home_start, home_size, F: int):
    """home_start, home_size as int32 [F] each (the C ABI reads F entries of both)."""
    hs, hz = _host_i32(home_start), _host_i32(home_size)
    if hs.ndim != 1 or hz.ndim != 1 or hs.size != F or hz.size != F:
        raise ValueError(f"home_start / home_size: expected {F} entries each (one per family), "
                         f"got shapes {hs.shape} and {hz.shape}")
    return hs, hz


def as_u32(t: torch.Tensor) -> torch.Tensor:
    """int64 values of a uint32 buffer held in an int32 tensor."""
    return t.to(torch.int64) & 0xFFFFFFFF


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _err_tensor(device) -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device=device)


# ------------------------------------------------------------------------------------------------
def coact_uses_matrix_cores(n_experts: int, top_k: int) -> bool:
    """Whether tacg_coact_build counts this shape on the matrix cores (else the LDS pair histogram)."""
    return bool(lib().tacg_coact_uses_matrix_cores(int(n_experts), int(top_k)))


def coact_build(trace: torch.Tensor, fam_off, n_experts: int, D: Optional[torch.Tensor] = None,
                C: Optional[torch.Tensor] = None, accumulate: bool = False, ws: Optional[torch.Tensor] = None,
                err: Optional[torch.Tensor] = None, stream=None):
    """Counts D [F][L][E] and C [F][L][E][E] (uint32 bits in int32 tensors) and the d_err tensor."""
    L_, N, k = _trace_dims(trace)
    off = _fam_off(fam_off)
    F = off.size - 1
    dev = trace.device
    if D is None:
        D = torch.empty((F, L_, n_experts), dtype=torch.int32, device=dev)
    if C is None:
        C = torch.empty((F, L_, n_experts, n_experts), dtype=torch.int32, device=dev)
    need = lib().tacg_coact_workspace_bytes(N, L_, k, n_experts, F)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    if err is None:
        err = _err_tensor(dev)
    st = lib().tacg_coact_build(_dptr(trace), N, L_, k, n_experts, _hptr(off), F,
                                _arg(D, "D", torch.int32, (F, L_, n_experts)),
                                _arg(C, "C", torch.int32, (F, L_, n_experts, n_experts)),
                                ACCUMULATE if accumulate else 0, _arg(err, "err", torch.int32, (1,)),
                                _dptr(ws), ws.numel(), _stream(stream))
    _check("tacg_coact_build", st)
    return D, C, err


def reweight(D: torch.Tensor, C: torch.Tensor, top_k: int, alpha: float = 0.25, tau: float = 1.0,
             eps: float = 1e-8, want_hat: bool = False, ws: Optional[torch.Tensor] = None, stream=None):
    """pref [L][E][F], a_tilde [L][E][E] (float32), a_hat or None."""
    F, L_, E = D.shape
    dev = D.device
    pref = torch.empty((L_, E, F), dtype=torch.float32, device=dev)
    at = torch.empty((L_, E, E), dtype=torch.float32, device=dev)
    ah = torch.empty((L_, E, E), dtype=torch.float32, device=dev) if want_hat else None
    need = lib().tacg_reweight_workspace_bytes(F, L_, E)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    st = lib().tacg_reweight(_arg(D, "D", torch.int32, (F, L_, E)), _arg(C, "C", torch.int32, (F, L_, E, E)), F, L_,
                             E, top_k, float(alpha), float(tau), float(eps),
                             _dptr(pref), _dptr(at), _dptr(ah), _dptr(ws), ws.numel(), _stream(stream))
    _check("tacg_reweight", st)
    return pref, at, ah


def placement_load(D: torch.Tensor, primary: torch.Tensor, n_gpus: int, err: Optional[torch.Tensor] = None,
                   stream=None):
    """int64 load_ref [P][L][G]."""
    F, L_, E = D.shape
    P = primary.shape[0]
    out = torch.empty((P, L_, n_gpus), dtype=torch.int64, device=D.device)
    if err is None:
        err = _err_tensor(D.device)
    st = lib().tacg_placement_load(_arg(D, "D", torch.int32, (F, L_, E)), F, L_, E,
                                   _arg(primary, "primary", torch.uint8, (P, L_, E)), P, n_gpus, _dptr(out),
                                   _arg(err, "err", torch.int32, (1,)), _stream(stream))
    _check("tacg_placement_load", st)
    return out


def eval_placements(trace: torch.Tensor, fam_off, n_experts: int, home_start, home_size, n_gpus: int,
                    primary: torch.Tensor, secondary: Optional[torch.Tensor] = None,
                    load_ref: Optional[torch.Tensor] = None, theta=(3, 20), want_fam: bool = True,
                    ws: Optional[torch.Tensor] = None, err: Optional[torch.Tensor] = None, out: Optional[dict] = None,
                    stream=None) -> dict:
    """dict(cost_home [P] int64, cost_span [P] int64, load [P][L][G] (uint32 bits), cost_home_fam, err)."""
    L_, N, k = _trace_dims(trace)
    off = _fam_off(fam_off)
    F = off.size - 1
    hs, hz = _bands(home_start, home_size, F)
    P = primary.shape[0]
    dev = trace.device
    R = 0 if secondary is None else int(secondary.shape[-1])
    if out is None:
        out = dict(cost_home=torch.empty(P, dtype=torch.int64, device=dev),
                   cost_span=torch.empty(P, dtype=torch.int64, device=dev),
                   load=torch.empty((P, L_, n_gpus), dtype=torch.int32, device=dev),
                   cost_home_fam=torch.empty((P, F), dtype=torch.int64, device=dev) if want_fam else None)
    need = lib().tacg_eval_workspace_bytes(N, L_, n_experts, n_gpus, P, F)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    if err is None:
        err = _err_tensor(dev)
    tn, td = theta if theta is not None else (0, 0)
    st = lib().tacg_eval_placements(
        _dptr(trace), N, L_, k, n_experts, _hptr(off), F, _hptr(hs), _hptr(hz), n_gpus, P,
        _arg(primary, "primary", torch.uint8, (P, L_, n_experts)),
        _arg(secondary, "secondary", torch.uint8, (P, L_, n_experts, R)) if R > 0 else None, R,
        _arg(load_ref, "load_ref", torch.int64, (P, L_, n_gpus)) if R > 0 else None, int(tn), int(td),
        _arg(out["cost_home"], "cost_home", torch.int64, (P,)), _arg(out["cost_span"], "cost_span", torch.int64, (P,)),
        _arg(out["load"], "load", torch.int32, (P, L_, n_gpus)),
        _arg(out["cost_home_fam"], "cost_home_fam", torch.int64, (P, F)), 0,
        _arg(err, "err", torch.int32, (1,)), _dptr(ws), ws.numel(), _stream(stream))
    _check("tacg_eval_placements", st)
    out["err"] = err
    return out


def eval_placements_noalloc(trace: torch.Tensor, fam_off, n_experts: int, home_start, home_size, n_gpus: int,
                            primary: torch.Tensor, secondary: Optional[torch.Tensor] = None,
                            load_ref: Optional[torch.Tensor] = None, theta=(3, 20), err: Optional[torch.Tensor] = None,
                            out: Optional[dict] = None, stream=None) -> dict:
    """eval_placements through tacg_eval_placements_noalloc: no workspace; the library's own device
    scratch (NOALLOC_SCRATCH_BYTES per GPU) serves instead.  Pass `out` (and `err`) to make the call
    itself allocate nothing.  Same dict as eval_placements."""
    L_, N, k = _trace_dims(trace)
    off = _fam_off(fam_off)
    F = off.size - 1
    hs, hz = _bands(home_start, home_size, F)
    P = primary.shape[0]
    dev = trace.device
    R = 0 if secondary is None else int(secondary.shape[-1])
    if out is None:
        out = dict(cost_home=torch.empty(P, dtype=torch.int64, device=dev),
                   cost_span=torch.empty(P, dtype=torch.int64, device=dev),
                   load=torch.empty((P, L_, n_gpus), dtype=torch.int32, device=dev),
                   cost_home_fam=torch.empty((P, F), dtype=torch.int64, device=dev))
    if err is None:
        err = _err_tensor(dev)
    tn, td = theta if theta is not None else (0, 0)
    st = lib().tacg_eval_placements_noalloc(
        _dptr(trace), N, L_, k, n_experts, _hptr(off), F, _hptr(hs), _hptr(hz), n_gpus, P,
        _arg(primary, "primary", torch.uint8, (P, L_, n_experts)),
        _arg(secondary, "secondary", torch.uint8, (P, L_, n_experts, R)) if R > 0 else None, R,
        _arg(load_ref, "load_ref", torch.int64, (P, L_, n_gpus)) if R > 0 else None, int(tn), int(td),
        _arg(out["cost_home"], "cost_home", torch.int64, (P,)), _arg(out["cost_span"], "cost_span", torch.int64, (P,)),
        _arg(out["load"], "load", torch.int32, (P, L_, n_gpus)),
        _arg(out.get("cost_home_fam"), "cost_home_fam", torch.int64, (P, F)), 0,
        _arg(err, "err", torch.int32, (1,)), _stream(stream))
    _check("tacg_eval_placements_noalloc", st)
    out["err"] = err
    return out


def eval_trace_stats(trace: torch.Tensor, fam_off, n_experts: int, home_start, home_size, n_gpus: int,
                     primary: torch.Tensor, secondary: Optional[torch.Tensor] = None,
                     load_ref: Optional[torch.Tensor] = None, theta=(3, 20), ws: Optional[torch.Tensor] = None,
                     err: Optional[torch.Tensor] = None, stream=None) -> dict:
    """Snapshot scoring plus the per-token statistics of App. C (tacg_eval_trace_stats).
    dict(cost_home, cost_span, load, span_fam, cross_fam, home_mass_fam ([P][F] int64), err)."""
    L_, N, k = _trace_dims(trace)
    off = _fam_off(fam_off)
    F = off.size - 1
    hs, hz = _bands(home_start, home_size, F)
    P = primary.shape[0]
    dev = trace.device
    R = 0 if secondary is None else int(secondary.shape[-1])
    out = dict(cost_home=torch.empty(P, dtype=torch.int64, device=dev),
               cost_span=torch.empty(P, dtype=torch.int64, device=dev),
               load=torch.empty((P, L_, n_gpus), dtype=torch.int32, device=dev),
               span_fam=torch.empty((P, F), dtype=torch.int64, device=dev),
               cross_fam=torch.empty((P, F), dtype=torch.int64, device=dev),
               home_mass_fam=torch.empty((P, F), dtype=torch.int64, device=dev))
    need = lib().tacg_eval_workspace_bytes(N, L_, n_experts, n_gpus, P, F)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    if err is None:
        err = _err_tensor(dev)
    tn, td = theta if theta is not None else (0, 0)
    st = lib().tacg_eval_trace_stats(
        _dptr(trace), N, L_, k, n_experts, _hptr(off), F, _hptr(hs), _hptr(hz), n_gpus, P,
        _arg(primary, "primary", torch.uint8, (P, L_, n_experts)),
        _arg(secondary, "secondary", torch.uint8, (P, L_, n_experts, R)) if R > 0 else None, R,
        _arg(load_ref, "load_ref", torch.int64, (P, L_, n_gpus)) if R > 0 else None, int(tn), int(td),
        _dptr(out["cost_home"]), _dptr(out["cost_span"]), _dptr(out["load"]), _dptr(out["span_fam"]),
        _dptr(out["cross_fam"]), _dptr(out["home_mass_fam"]), 0, _arg(err, "err", torch.int32, (1,)), _dptr(ws),
        ws.numel(), _stream(stream))
    _check("tacg_eval_trace_stats", st)
    out["err"] = err
    return out


def eval_online(trace: torch.Tensor, fam_off, n_experts: int, home_start, home_size, n_gpus: int,
                primary: torch.Tensor, secondary: Optional[torch.Tensor] = None, rho: float = 0.995, theta=(3, 20),
                state: Optional[torch.Tensor] = None, want_state: bool = True, want_fam: bool = True,
                err: Optional[torch.Tensor] = None, out: Optional[dict] = None, stream=None) -> dict:
    """Scoring with decayed per-GPU loads (tacg_eval_online).  state: float64 [P][L][G] initial loads
    or None (zero).  dict(cost_home, cost_span, load, cost_home_fam, state (final loads), err)."""
    L_, N, k = _trace_dims(trace)
    off = _fam_off(fam_off)
    F = off.size - 1
    hs, hz = _bands(home_start, home_size, F)
    P = primary.shape[0]
    dev = trace.device
    R = 0 if secondary is None else int(secondary.shape[-1])
    if out is None:
        out = dict(cost_home=torch.empty(P, dtype=torch.int64, device=dev),
                   cost_span=torch.empty(P, dtype=torch.int64, device=dev),
                   load=torch.empty((P, L_, n_gpus), dtype=torch.int32, device=dev),
                   cost_home_fam=torch.empty((P, F), dtype=torch.int64, device=dev) if want_fam else None,
                   state=torch.empty((P, L_, n_gpus), dtype=torch.float64, device=dev) if want_state else None)
    if state is not None and (state.dtype != torch.float64 or tuple(state.shape) != (P, L_, n_gpus)):
        raise ValueError("state must be float64 [P][L][G]")
    if err is None:
        err = _err_tensor(dev)
    tn, td = theta if theta is not None else (0, 0)
    st = lib().tacg_eval_online(
        _dptr(trace), N, L_, k, n_experts, _hptr(off), F, _hptr(hs), _hptr(hz), n_gpus, P,
        _arg(primary, "primary", torch.uint8, (P, L_, n_experts)),
        _arg(secondary, "secondary", torch.uint8, (P, L_, n_experts, R)) if R > 0 else None, R, float(rho),
        int(tn), int(td), _dptr(state),
        _arg(out.get("state"), "state", torch.float64, (P, L_, n_gpus)),
        _arg(out["cost_home"], "cost_home", torch.int64, (P,)), _arg(out["cost_span"], "cost_span", torch.int64, (P,)),
        _arg(out["load"], "load", torch.int32, (P, L_, n_gpus)),
        _arg(out["cost_home_fam"], "cost_home_fam", torch.int64, (P, F)), 0,
        _arg(err, "err", torch.int32, (1,)), _stream(stream))
    _check("tacg_eval_online", st)
    out["err"] = err
    return out


def activation_distance(D: torch.Tensor, top_k: int, stream=None) -> torch.Tensor:
    """float64 [F][F] Frobenius distances of the families' expert-activation distributions."""
    F, L_, E = D.shape
    out = torch.empty((F, F), dtype=torch.float64, device=D.device)
    st = lib().tacg_activation_distance(_arg(D, "D", torch.int32, (F, L_, E)), F, L_, E, top_k, _dptr(out),
                                        _stream(stream))
    _check("tacg_activation_distance", st)
    return out


def pair_jaccard(C: torch.Tensor, top_n: int = 64, stream=None):
    """(top_pairs int32 [F][L][top_n], jaccard float64 [L][F][F]) of the co-activation counts."""
    F, L_, E, _ = C.shape
    pairs = torch.empty((F, L_, top_n), dtype=torch.int32, device=C.device)
    jac = torch.empty((L_, F, F), dtype=torch.float64, device=C.device)
    st = lib().tacg_pair_jaccard(_arg(C, "C", torch.int32, (F, L_, E, E)), F, L_, E, top_n, _dptr(pairs), _dptr(jac),
                                 _stream(stream))
    _check("tacg_pair_jaccard", st)
    return pairs, jac


def gesr_scores(D: torch.Tensor, C: torch.Tensor, top_k: int, stream=None):
    """float64 cent, cons, spec [L][E] (tacg_gesr_scores)."""
    F, L_, E = D.shape
    cent = torch.empty((L_, E), dtype=torch.float64, device=D.device)
    cons = torch.empty_like(cent)
    spec = torch.empty_like(cent)
    st = lib().tacg_gesr_scores(_arg(D, "D", torch.int32, (F, L_, E)), _arg(C, "C", torch.int32, (F, L_, E, E)),
                                F, L_, E, top_k, _dptr(cent), _dptr(cons), _dptr(spec),
                                _stream(stream))
    _check("tacg_gesr_scores", st)
    return cent, cons, spec


def group_objective(a_tilde: torch.Tensor, primary: torch.Tensor, n_gpus: int, err: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """float64 [P][L] within-group affinity of every placement (tacg_group_objective)."""
    L_, E, _ = a_tilde.shape
    P = primary.shape[0]
    out = torch.empty((P, L_), dtype=torch.float64, device=a_tilde.device)
    if err is None:
        err = _err_tensor(a_tilde.device)
    st = lib().tacg_group_objective(_arg(a_tilde, "a_tilde", torch.float32, (L_, E, E)), L_, E,
                                    _arg(primary, "primary", torch.uint8, (P, L_, E)), P, n_gpus, _dptr(out),
                                    _arg(err, "err", torch.int32, (1,)),
                                    _stream(stream))
    _check("tacg_group_objective", st)
    return out


def jain_index(load: torch.Tensor, per_layer: bool = False, stream=None):
    """float32 Jain and MaxVio, [P] (sum over layers) or [P][L]."""
    P, L_, G = load.shape
    shape = (P, L_) if per_layer else (P,)
    j = torch.empty(shape, dtype=torch.float32, device=load.device)
    v = torch.empty(shape, dtype=torch.float32, device=load.device)
    st = lib().tacg_jain(_arg(load, "load", torch.int32, (P, L_, G)), P, L_, G, 1 if per_layer else 0, _dptr(j),
                         _dptr(v), _stream(stream))
    _check("tacg_jain", st)
    return j, v
