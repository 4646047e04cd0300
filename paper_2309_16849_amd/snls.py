"""Python binding of libsnls.so (the C ABI declared in include/snls.h).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
There is no CPU fallback -- if libsnls.so is missing or fails to load, every
call raises.

Functions carry the C names: snls_search, snls_topk, snls_aggregate,
snls_backward, snls_aggregate_stacked, snls_chain_flows, snls_aggregate_static,
snls_gather_stacked, snls_stacked_reduce, snls_gather_reduce, snls_workspace_size,
snls_status_string, snls_abi_version.
Parameters are plain dicts with keys B, T, C, H, W, HD, ws, wt, ps, stride0,
stride1, k, dist_type (see ``params_from_dict``).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsnls.so")

SNLS_OK, SNLS_ERR_INVALID_ARG, SNLS_ERR_UNSUPPORTED, SNLS_ERR_HIP, SNLS_ERR_WORKSPACE, SNLS_ERR_SCRATCH = range(6)
SNLS_DIST_PROD, SNLS_DIST_L2 = 0, 1
SNLS_OP_SEARCH, SNLS_OP_AGGREGATE, SNLS_OP_BACKWARD, SNLS_OP_AGGREGATE_STACKED = 0, 1, 2, 3
SNLS_OP_GATHER_STACKED, SNLS_OP_GATHER_REDUCE = 4, 5
SNLS_MAX_K = 128
SNLS_STATIC_SCRATCH_BYTES = 64 << 20
SYMBOLS = ("snls_search", "snls_topk", "snls_aggregate", "snls_backward", "snls_workspace_size",
           "snls_status_string", "snls_abi_version", "snls_aggregate_stacked", "snls_chain_flows",
           "snls_aggregate_static", "snls_gather_stacked", "snls_stacked_reduce", "snls_gather_reduce")


class SnlsParams(ctypes.Structure):
    """Mirror of the C struct snls_params."""
    _fields_ = [("struct_size", ctypes.c_uint32)] + [
        (n, ctypes.c_int32) for n in ("B", "T", "C", "H", "W", "HD", "ws", "wt", "ps", "stride0")
    ] + [("stride1", ctypes.c_float), ("k", ctypes.c_int32), ("dist_type", ctypes.c_int32)]


class SnlsError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s failed: %s (status %d)" % (where, snls_status_string(status), status))
        self.status = status


_lib = None


def load_library():
    """Load libsnls.so once (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsnls.so is not built (%s); run python -m paper_2309_16849_amd.build" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        P, F32, I32, I64, SZ = ctypes.c_void_p, ctypes.c_float, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        PP = ctypes.POINTER(SnlsParams)
        lib.snls_search.argtypes = [P, P, P, PP, P, P, P, SZ, P]
        lib.snls_topk.argtypes = [P, P, I64, I32, I32, I32, P, P, P]
        lib.snls_aggregate.argtypes = [P, P, P, PP, F32, P, P, SZ, P]
        lib.snls_backward.argtypes = [P] * 8 + [PP, F32, P, P, P, P, P, SZ, P]
        lib.snls_aggregate_stacked.argtypes = [P, P, P, PP, F32, P, P, SZ, P]
        lib.snls_chain_flows.argtypes = [P, P, I32, I32, I32, I32, I32, P, P]
        lib.snls_aggregate_static.argtypes = [P, P, P, PP, F32, P, P]
        lib.snls_gather_stacked.argtypes = [P, P, P, PP, P, P, SZ, P]
        lib.snls_stacked_reduce.argtypes = [P, P, PP, I32, P, P]
        lib.snls_gather_reduce.argtypes = [P, P, P, P, PP, I32, P, P, SZ, P]
        lib.snls_workspace_size.argtypes = [ctypes.c_int, PP]
        lib.snls_workspace_size.restype = SZ
        lib.snls_status_string.argtypes = [ctypes.c_int]
        lib.snls_status_string.restype = ctypes.c_char_p
        lib.snls_abi_version.argtypes = []
        for f in ("snls_search", "snls_topk", "snls_aggregate", "snls_backward", "snls_abi_version",
                  "snls_aggregate_stacked", "snls_chain_flows", "snls_aggregate_static", "snls_gather_stacked",
                  "snls_stacked_reduce", "snls_gather_reduce"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def params_from_dict(p: dict) -> SnlsParams:
    s = SnlsParams()
    s.struct_size = ctypes.sizeof(SnlsParams)
    for n in ("B", "T", "C", "H", "W", "HD", "ws", "wt", "ps", "stride0", "k", "dist_type"):
        setattr(s, n, int(p[n]))
    s.stride1 = float(p["stride1"])
    return s


def grid(p: dict):
    return (p["H"] - 1) // p["stride0"] + 1, (p["W"] - 1) // p["stride0"] + 1


def n_cand(p: dict) -> int:
    return (2 * p["wt"] + 1) * p["ws"] ** 2


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _dev(t, name, shape=None):
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
        raise ValueError("%s must be a contiguous float32 tensor on the GPU" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return t


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, where):
    if status != SNLS_OK:
        raise SnlsError(status, where)


def snls_status_string(status: int) -> str:
    return load_library().snls_status_string(int(status)).decode()


def snls_abi_version() -> int:
    return load_library().snls_abi_version()


def snls_workspace_size(op: int, p: dict) -> int:
    prm = params_from_dict(p)
    return load_library().snls_workspace_size(op, ctypes.byref(prm))


def video_shape(p: dict):
    return (p["B"], p["T"], p["C"], p["H"], p["W"])


def flow_shape(p: dict):
    return (p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"])


def out_shape(p: dict):
    nH, nW = grid(p)
    kk = p["k"] if p["k"] > 0 else n_cand(p)
    return (p["B"], p["HD"], p["T"], nH, nW, kk)


def snls_search(q, k, flows, p: dict, dists=None, inds=None, workspace=None, stream=None):
    """Shifted non-local search; returns (dists, inds) (see include/snls.h).
    The workspace is allocated here when not given (its size may be 0)."""
    lib = load_library()
    _dev(q, "q", video_shape(p))
    _dev(k, "k", video_shape(p))
    if p["wt"] > 0 or flows is not None:
        _dev(flows, "flows", flow_shape(p))
    shp = out_shape(p)
    if dists is None:
        dists = torch.empty(shp, device=q.device, dtype=torch.float32)
    if inds is None:
        inds = torch.empty(shp + (3,), device=q.device, dtype=torch.float32)
    _dev(dists, "dists", shp)
    _dev(inds, "inds", shp + (3,))
    if workspace is None:
        workspace = workspace_for(SNLS_OP_SEARCH, p, q.device)
    prm = params_from_dict(p)
    _check(lib.snls_search(_ptr(q), _ptr(k), _ptr(flows), ctypes.byref(prm), _ptr(dists), _ptr(inds),
                           _ptr(workspace), workspace.numel() * 4, _stream(stream)), "snls_search")
    return dists, inds


def snls_topk(dists_all, inds_all, k: int, dist_type: int, dists=None, inds=None, stream=None):
    """top-k of rows of candidate scores; dists_all (..., n_cand), inds_all (..., n_cand, 3)."""
    lib = load_library()
    _dev(dists_all, "dists_all")
    n_c = dists_all.shape[-1]
    lead = tuple(dists_all.shape[:-1])
    _dev(inds_all, "inds_all", lead + (n_c, 3))
    rows = dists_all.numel() // max(n_c, 1)
    if dists is None:
        dists = torch.empty(lead + (k,), device=dists_all.device, dtype=torch.float32)
    if inds is None:
        inds = torch.empty(lead + (k, 3), device=dists_all.device, dtype=torch.float32)
    _dev(dists, "dists", lead + (k,))
    _dev(inds, "inds", lead + (k, 3))
    _check(lib.snls_topk(_ptr(dists_all), _ptr(inds_all), rows, n_c, k, dist_type, _ptr(dists), _ptr(inds),
                         _stream(stream)), "snls_topk")
    return dists, inds


def workspace_for(op: int, p: dict, device):
    """A device buffer of snls_workspace_size(op, p) bytes (torch allocations are 256-byte aligned)."""
    need = snls_workspace_size(op, p)
    if need == ctypes.c_size_t(-1).value:
        raise SnlsError(SNLS_ERR_INVALID_ARG, "snls_workspace_size")
    return torch.empty(max((need + 3) // 4, 1), device=device, dtype=torch.float32)


def snls_aggregate(v, dists, inds, p: dict, scale: float = 1.0, out=None, workspace=None, stream=None):
    """Softmax-weighted patch aggregation; returns out (B,T,C,H,W)."""
    lib = load_library()
    _dev(v, "v", video_shape(p))
    shp = out_shape(p)
    _dev(dists, "dists", shp)
    _dev(inds, "inds", shp + (3,))
    if out is None:
        out = torch.empty(video_shape(p), device=v.device, dtype=torch.float32)
    _dev(out, "out", video_shape(p))
    if workspace is None:
        workspace = workspace_for(SNLS_OP_AGGREGATE, p, v.device)
    prm = params_from_dict(p)
    _check(lib.snls_aggregate(_ptr(v), _ptr(dists), _ptr(inds), ctypes.byref(prm), float(scale), _ptr(out),
                              _ptr(workspace), workspace.numel() * 4, _stream(stream)), "snls_aggregate")
    return out


def snls_aggregate_static(v, dists, inds, p: dict, scale: float = 1.0, out=None, stream=None):
    """snls_aggregate with the library's static scratch array as workspace
    (nothing allocated on the device beyond ``out`` when it is not given)."""
    lib = load_library()
    _dev(v, "v", video_shape(p))
    shp = out_shape(p)
    _dev(dists, "dists", shp)
    _dev(inds, "inds", shp + (3,))
    if out is None:
        out = torch.empty(video_shape(p), device=v.device, dtype=torch.float32)
    _dev(out, "out", video_shape(p))
    prm = params_from_dict(p)
    _check(lib.snls_aggregate_static(_ptr(v), _ptr(dists), _ptr(inds), ctypes.byref(prm), float(scale), _ptr(out),
                                     _stream(stream)), "snls_aggregate_static")
    return out


def snls_backward(q, k, v, flows, dists, inds, grad_out, p: dict, scale: float = 1.0, grad_dists=None,
                  workspace=None, stream=None):
    """Gradients (grad_q, grad_k, grad_v, grad_flows) of search + aggregation."""
    lib = load_library()
    vs, shp = video_shape(p), out_shape(p)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (grad_out, "grad_out")):
        _dev(t, n, vs)
    _dev(dists, "dists", shp)
    _dev(inds, "inds", shp + (3,))
    if grad_dists is not None:
        _dev(grad_dists, "grad_dists", shp)
    if p["wt"] > 0 or flows is not None:
        _dev(flows, "flows", flow_shape(p))
    gq, gk, gv = (torch.empty(vs, device=q.device, dtype=torch.float32) for _ in range(3))
    gf = torch.empty(flow_shape(p), device=q.device, dtype=torch.float32)
    if workspace is None:
        workspace = workspace_for(SNLS_OP_BACKWARD, p, q.device)
    prm = params_from_dict(p)
    _check(lib.snls_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(flows), _ptr(dists), _ptr(inds), _ptr(grad_out),
                             _ptr(grad_dists), ctypes.byref(prm), float(scale), _ptr(gq), _ptr(gk), _ptr(gv),
                             _ptr(gf), _ptr(workspace), workspace.numel() * 4, _stream(stream)), "snls_backward")
    return gq, gk, gv, gf


def snls_aggregate_stacked(v, dists, inds, p: dict, scale: float = 1.0, stacked=None, workspace=None, stream=None):
    """Aggregation with the k neighbours kept apart; returns (B, HD, k, T, C/HD, H, W)."""
    lib = load_library()
    _dev(v, "v", video_shape(p))
    shp = out_shape(p)
    _dev(dists, "dists", shp)
    _dev(inds, "inds", shp + (3,))
    st_shape = (p["B"], p["HD"], p["k"], p["T"], p["C"] // p["HD"], p["H"], p["W"])
    if stacked is None:
        stacked = torch.empty(st_shape, device=v.device, dtype=torch.float32)
    _dev(stacked, "stacked", st_shape)
    if workspace is None:
        workspace = workspace_for(SNLS_OP_AGGREGATE_STACKED, p, v.device)
    prm = params_from_dict(p)
    _check(lib.snls_aggregate_stacked(_ptr(v), _ptr(dists), _ptr(inds), ctypes.byref(prm), float(scale),
                                      _ptr(stacked), _ptr(workspace), workspace.numel() * 4, _stream(stream)),
           "snls_aggregate_stacked")
    return stacked


def snls_chain_flows(fflow, bflow, wt: int, flows=None, stream=None):
    """Window offsets (B, T, 2wt, 2, H, W) composed from one-step flows (B, T, 2, H, W)."""
    lib = load_library()
    _dev(fflow, "fflow")
    B, T, two, H, W = fflow.shape
    if two != 2:
        raise ValueError("fflow must be (B, T, 2, H, W)")
    _dev(bflow, "bflow", tuple(fflow.shape))
    if flows is None:
        flows = torch.empty((B, T, 2 * wt, 2, H, W), device=fflow.device, dtype=torch.float32)
    _dev(flows, "flows", (B, T, 2 * wt, 2, H, W))
    _check(lib.snls_chain_flows(_ptr(fflow), _ptr(bflow), B, T, H, W, int(wt), _ptr(flows), _stream(stream)),
           "snls_chain_flows")
    return flows


def stacked_shape(p: dict):
    return (p["B"], p["HD"], p["k"], p["T"], p["C"] // p["HD"], p["H"], p["W"])


def snls_gather_stacked(v, weights, inds, p: dict, stacked=None, workspace=None, stream=None):
    """The example's gather with caller weights; returns (B, HD, k, T, C/HD, H, W)."""
    lib = load_library()
    _dev(v, "v", video_shape(p))
    shp = out_shape(p)
    _dev(weights, "weights", shp)
    _dev(inds, "inds", shp + (3,))
    if stacked is None:
        stacked = torch.empty(stacked_shape(p), device=v.device, dtype=torch.float32)
    _dev(stacked, "stacked", stacked_shape(p))
    if workspace is None:
        workspace = workspace_for(SNLS_OP_GATHER_STACKED, p, v.device)
    prm = params_from_dict(p)
    _check(lib.snls_gather_stacked(_ptr(v), _ptr(weights), _ptr(inds), ctypes.byref(prm), _ptr(stacked),
                                   _ptr(workspace), workspace.numel() * 4, _stream(stream)), "snls_gather_stacked")
    return stacked


def snls_stacked_reduce(stacked, proj, p: dict, out=None, stream=None):
    """Reduction over the k neighbours with kernel proj (Cout, C, k); returns (B, T, Cout, H, W)."""
    lib = load_library()
    _dev(stacked, "stacked", stacked_shape(p))
    _dev(proj, "proj")
    cout = proj.shape[0]
    if tuple(proj.shape) != (cout, p["C"], p["k"]):
        raise ValueError("proj must be (Cout, C, k)")
    if out is None:
        out = torch.empty((p["B"], p["T"], cout, p["H"], p["W"]), device=stacked.device, dtype=torch.float32)
    _dev(out, "out", (p["B"], p["T"], cout, p["H"], p["W"]))
    prm = params_from_dict(p)
    _check(lib.snls_stacked_reduce(_ptr(stacked), _ptr(proj), ctypes.byref(prm), cout, _ptr(out), _stream(stream)),
           "snls_stacked_reduce")
    return out


def snls_gather_reduce(v, weights, inds, proj, p: dict, out=None, workspace=None, stream=None):
    """Gather with caller weights and reduction over the k neighbours in one pass; returns (B, T, Cout, H, W)."""
    lib = load_library()
    _dev(v, "v", video_shape(p))
    shp = out_shape(p)
    _dev(weights, "weights", shp)
    _dev(inds, "inds", shp + (3,))
    _dev(proj, "proj")
    cout = proj.shape[0]
    if tuple(proj.shape) != (cout, p["C"], p["k"]):
        raise ValueError("proj must be (Cout, C, k)")
    if out is None:
        out = torch.empty((p["B"], p["T"], cout, p["H"], p["W"]), device=v.device, dtype=torch.float32)
    _dev(out, "out", (p["B"], p["T"], cout, p["H"], p["W"]))
    if workspace is None:
        workspace = workspace_for(SNLS_OP_GATHER_REDUCE, p, v.device)
    prm = params_from_dict(p)
    _check(lib.snls_gather_reduce(_ptr(v), _ptr(weights), _ptr(inds), _ptr(proj), ctypes.byref(prm), cout, _ptr(out),
                                  _ptr(workspace), workspace.numel() * 4, _stream(stream)), "snls_gather_reduce")
    return out
