"""ctypes binding of libmoe_gemm2.so: argument marshalling only.

Every step of the stage runs in the library's HIP kernel; PyTorch is used
here for device memory and the current stream.  If the library is missing
this module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe_gemm2.so")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_ALIGNMENT = -2
MOE_ERR_WORKSPACE = -3
MOE_ERR_NO_LEGAL_PARTITION = -4
MOE_ERR_HIP = -5
MOE_ERR_TIMEOUT = -6
MOE_ERR_UNSUPPORTED = -7
MOE_ERR_BAD_ROUTING = -8

EXPORTED = (
    "moe_select_partition", "moe_select_evaluate", "moe_gemm2_default_params",
    "moe_gemm2_workspace_size", "moe_gemm2_workspace_init", "moe_gemm2_combine",
    "moe_gemm2_combine_traced", "moe_gemm2_trace_size", "moe_gemm2_status",
    "moe_strerror", "moe_gemm2_abi_version", "moe_gemm2_default_params_ex",
    "moe_gemm2_combine_ex", "moe_gemm2_launch_params", "moe_gemm1_pack_weights",
    "moe_gemm1_swiglu", "moe_layer_workspace_size", "moe_layer_forward",
    "moe_gemm2_combine_noalloc", "moe_select_partition_splits", "moe_select_candidate",
)

# size of the library's own scratch behind moe_gemm2_combine_noalloc
NOALLOC_SCRATCH_BYTES = 96 << 20

MODE_OWNER_WRITE = 0
MODE_ATOMIC_SCATTER = 1
MODE_TOKEN_BANDS = 2


class Workload(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("I", ctypes.c_int32),
                ("E", ctypes.c_int32), ("topk", ctypes.c_int32), ("splits", ctypes.c_int32),
                ("ranks", ctypes.c_int32), ("rows", ctypes.c_int64),
                ("host_expert_counts", ctypes.POINTER(ctypes.c_int32))]


class SelectParams(ctypes.Structure):
    _fields_ = [("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("comm_tile_m", ctypes.c_int32), ("comm_tile_n", ctypes.c_int32),
                ("occ_comp", ctypes.c_int32), ("occ_comm", ctypes.c_int32),
                ("num_cus", ctypes.c_int32), ("c_min", ctypes.c_int32),
                ("c_max", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("rho_ref_num", ctypes.c_int64), ("rho_ref_den", ctypes.c_int64),
                ("k_ref", ctypes.c_int32), ("tile_m_ref", ctypes.c_int32),
                ("tile_n_ref", ctypes.c_int32), ("d_ref", ctypes.c_int32),
                ("split_axis", ctypes.c_int32), ("drain", ctypes.c_int32),
                ("rho_kh", ctypes.c_int32), ("topk_ref", ctypes.c_int32),
                ("comm_tile_n_ref", ctypes.c_int32), ("readiness", ctypes.c_int32),
                ("comm_tile_m_last", ctypes.c_int32),
                ("split_cost_num", ctypes.c_int64), ("split_cost_den", ctypes.c_int64)]


class Partition(ctypes.Structure):
    _fields_ = [("C", ctypes.c_int32), ("R", ctypes.c_int32), ("P", ctypes.c_int32),
                ("delta_comp", ctypes.c_int32), ("T_num", ctypes.c_int64),
                ("T_den", ctypes.c_int64), ("W_comp", ctypes.c_int64),
                ("W_comm", ctypes.c_int64)]


class MoeError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        self.code = code
        super().__init__(f"{what}: {strerror(code)} ({code})" if what else strerror(code))


_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(
                    f"{LIB_PATH} is missing: build it with "
                    "`python -m paper_2609_07536_amd.build`")
            # torch first: it brings its own HIP runtime, which then also
            # serves this library (same soname).  Loaded the other way
            # round, the process would hold two HIP runtimes, and torch's
            # device memory and streams would be invalid in ours.
            import torch  # noqa: F401
            L = ctypes.CDLL(LIB_PATH)
            vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
            L.moe_select_partition.argtypes = [ctypes.POINTER(Workload),
                                               ctypes.POINTER(SelectParams),
                                               ctypes.POINTER(Partition)]
            L.moe_select_partition.restype = ctypes.c_int
            L.moe_select_partition_splits.argtypes = [ctypes.POINTER(Workload),
                                                      ctypes.POINTER(SelectParams), i32, i32,
                                                      ctypes.POINTER(Partition),
                                                      ctypes.POINTER(ctypes.c_int32)]
            L.moe_select_partition_splits.restype = ctypes.c_int
            L.moe_select_evaluate.argtypes = [ctypes.POINTER(Workload),
                                              ctypes.POINTER(SelectParams),
                                              ctypes.POINTER(ctypes.c_int64), i32,
                                              ctypes.POINTER(ctypes.c_int64)]
            L.moe_select_evaluate.restype = ctypes.c_int
            L.moe_gemm2_default_params.argtypes = [ctypes.c_int, ctypes.POINTER(SelectParams)]
            L.moe_gemm2_default_params.restype = ctypes.c_int
            L.moe_gemm2_default_params_ex.argtypes = [ctypes.c_int, i32, i32,
                                                      ctypes.POINTER(SelectParams)]
            L.moe_gemm2_default_params_ex.restype = ctypes.c_int
            L.moe_gemm2_launch_params.argtypes = [ctypes.c_int, i32, ctypes.POINTER(Workload),
                                                  ctypes.POINTER(SelectParams)]
            L.moe_gemm2_launch_params.restype = ctypes.c_int
            L.moe_gemm2_workspace_size.argtypes = [ctypes.POINTER(Workload)]
            L.moe_gemm2_workspace_size.restype = sz
            L.moe_gemm2_trace_size.argtypes = [ctypes.POINTER(Workload)]
            L.moe_gemm2_trace_size.restype = sz
            L.moe_gemm2_workspace_init.argtypes = [vp, sz, vp]
            L.moe_gemm2_workspace_init.restype = ctypes.c_int
            L.moe_gemm2_combine.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.POINTER(Workload),
                                            i32, vp, sz, vp]
            L.moe_gemm2_combine.restype = ctypes.c_int
            L.moe_gemm2_combine_traced.argtypes = [vp, vp, vp, vp, vp, vp,
                                                   ctypes.POINTER(Workload), i32, vp, sz, vp,
                                                   vp, sz]
            L.moe_gemm2_combine_traced.restype = ctypes.c_int
            L.moe_gemm2_combine_ex.argtypes = [vp, vp, vp, vp, vp, vp,
                                               ctypes.POINTER(Workload), i32, i32, vp, sz,
                                               vp, vp, sz]
            L.moe_gemm2_combine_ex.restype = ctypes.c_int
            L.moe_gemm2_combine_noalloc.argtypes = [vp, vp, vp, vp, vp, vp,
                                                    ctypes.POINTER(Workload), i32, i32, vp]
            L.moe_gemm2_combine_noalloc.restype = ctypes.c_int
            L.moe_gemm1_pack_weights.argtypes = [vp, vp, i32, i32, i32, vp]
            L.moe_gemm1_pack_weights.restype = ctypes.c_int
            L.moe_gemm1_swiglu.argtypes = [vp, vp, vp, vp, vp, ctypes.POINTER(Workload), vp, sz, vp]
            L.moe_gemm1_swiglu.restype = ctypes.c_int
            L.moe_layer_workspace_size.argtypes = [ctypes.POINTER(Workload)]
            L.moe_layer_workspace_size.restype = sz
            L.moe_layer_forward.argtypes = [vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(Workload),
                                            i32, vp, sz, vp]
            L.moe_layer_forward.restype = ctypes.c_int
            L.moe_gemm2_status.argtypes = [vp, vp, ctypes.c_int]
            L.moe_gemm2_status.restype = ctypes.c_int
            L.moe_strerror.argtypes = [ctypes.c_int]
            L.moe_strerror.restype = ctypes.c_char_p
            L.moe_select_candidate.argtypes = [ctypes.POINTER(Workload),
                                               ctypes.POINTER(SelectParams), i32,
                                               ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(ctypes.c_int64), i32]
            L.moe_select_candidate.restype = ctypes.c_int
            L.moe_gemm2_abi_version.argtypes = []
            L.moe_gemm2_abi_version.restype = ctypes.c_int
            _lib = L
        return _lib


def strerror(code: int) -> str:
    return lib().moe_strerror(int(code)).decode()


def make_workload(T: int, H: int, I: int, E: int, topk: int, splits: int = 1,
                  counts: Optional[Sequence[int]] = None, rows: int = 0,
                  ranks: int = 1):
    """A moe_workload_t; the returned tuple keeps the counts array alive."""
    wl = Workload(T=T, H=H, I=I, E=E, topk=topk, splits=splits, ranks=ranks, rows=rows)
    keep = None
    if counts is not None:
        keep = np.ascontiguousarray(np.asarray(counts, dtype=np.int32))
        wl.host_expert_counts = keep.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    return wl, keep


def select_partition(wl: Workload, params: SelectParams):
    out = Partition()
    r = lib().moe_select_partition(ctypes.byref(wl), ctypes.byref(params), ctypes.byref(out))
    return r, out


def select_partition_splits(wl: Workload, params: SelectParams, l_min: int, l_max: int):
    """moe_select_partition_splits: returns (C or error, L, Partition)."""
    out = Partition()
    L = ctypes.c_int32(0)
    r = lib().moe_select_partition_splits(ctypes.byref(wl), ctypes.byref(params), int(l_min),
                                          int(l_max), ctypes.byref(out), ctypes.byref(L))
    return r, L.value, out


def select_candidate(wl: Workload, params: SelectParams, C: int):
    """moe_select_candidate: (entries or error, rho_num, rho_den, A, F) with
    A and F the split arrival and finish times in units of 1/rho_den compute
    waves."""
    num, den = ctypes.c_int64(0), ctypes.c_int64(0)
    n = lib().moe_select_candidate(ctypes.byref(wl), ctypes.byref(params), int(C), None, None,
                                   None, None, 0)
    if n < 0:
        return n, 0, 0, [], []
    A = (ctypes.c_int64 * n)()
    F = (ctypes.c_int64 * n)()
    r = lib().moe_select_candidate(ctypes.byref(wl), ctypes.byref(params), int(C),
                                   ctypes.byref(num), ctypes.byref(den), A, F, n)
    k = max(r, 0)
    return r, num.value, den.value, [A[i] for i in range(k)], [F[i] for i in range(k)]


def select_evaluate(wl: Workload, params: SelectParams):
    n = params.c_max - params.c_min + 1
    buf = (ctypes.c_int64 * max(n, 1))()
    den = ctypes.c_int64(0)
    r = lib().moe_select_evaluate(ctypes.byref(wl), ctypes.byref(params), buf, n,
                                  ctypes.byref(den))
    return r, [buf[i] for i in range(max(r, 0))], den.value


def default_params(device: int = 0, mode: Optional[int] = None, topk: int = 1) -> SelectParams:
    """moe_gemm2_default_params, or moe_gemm2_default_params_ex for a mode."""
    p = SelectParams()
    if mode is None:
        r = lib().moe_gemm2_default_params(device, ctypes.byref(p))
    else:
        r = lib().moe_gemm2_default_params_ex(device, int(mode), int(topk), ctypes.byref(p))
    if r < 0:
        raise MoeError(r, "moe_gemm2_default_params")
    return p


def launch_params(wl: Workload, mode: int = 0, device: int = 0) -> SelectParams:
    """moe_gemm2_launch_params: the selector parameters a launch of this
    workload uses (its consumer task size and the matching rho_ref)."""
    p = SelectParams()
    r = lib().moe_gemm2_launch_params(device, int(mode), ctypes.byref(wl), ctypes.byref(p))
    if r < 0:
        raise MoeError(r, "moe_gemm2_launch_params")
    return p


def workspace_size(wl: Workload) -> int:
    return int(lib().moe_gemm2_workspace_size(ctypes.byref(wl)))


def trace_size(wl: Workload) -> int:
    return int(lib().moe_gemm2_trace_size(ctypes.byref(wl)))


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Workspace:
    """Device workspace (torch-owned memory), zeroed once on creation."""

    def __init__(self, nbytes: int, device=None, stream=None):
        import torch
        self.nbytes = int(nbytes)
        self.tensor = torch.empty(max(self.nbytes, 256) + 256, dtype=torch.uint8,
                                  device=device or "cuda")
        base = self.tensor.data_ptr()
        self.ptr = (base + 255) // 256 * 256
        r = lib().moe_gemm2_workspace_init(ctypes.c_void_p(self.ptr),
                                           ctypes.c_size_t(self.nbytes), _stream(stream))
        if r < 0:
            raise MoeError(r, "moe_gemm2_workspace_init")

    def status(self, stream=None, clear: bool = False) -> int:
        return lib().moe_gemm2_status(ctypes.c_void_p(self.ptr), _stream(stream), int(clear))


def _call_workspace(nbytes: int, device, stream) -> "Workspace":
    """A workspace for one call that was given none.

    It is allocated (and zeroed) on the launch's own stream: torch's caching
    allocator then reuses its memory only for later work on that stream,
    which runs after the launch, never while the kernel may still write
    its flags, inverse map and Y staging.  This path allocates on every
    call; pass a Workspace to avoid that."""
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    with torch.cuda.stream(s):
        ws = Workspace(nbytes, device=device, stream=s)
    ws.tensor.record_stream(s)
    return ws


def combine(x_perm, w2, expert_offsets, token_ids, gate_w, T: int, splits: int = 1,
            topk: Optional[int] = None, counts: Optional[Sequence[int]] = None,
            num_consumers: int = -1, out=None, workspace: Optional[Workspace] = None,
            stream=None, trace=None, mode: Optional[int] = None):
    """Run the stage on torch device tensors: moe_gemm2_combine (or
    moe_gemm2_combine_traced with a trace buffer) when mode is None,
    moe_gemm2_combine_ex with that mode otherwise.

    x_perm bf16 [rows, I], w2 bf16 [E, I, H], expert_offsets int32 [E+1],
    token_ids int32 [rows], gate_w fp32 [rows]; returns (out [T, H] fp32, C).
    Without a (large enough) workspace, one is allocated for this call on
    the launch's stream.
    """
    import torch
    rows, I = int(x_perm.shape[0]), int(x_perm.shape[1])
    E, H = int(w2.shape[0]), int(w2.shape[2])
    if topk is None:
        topk = max(1, -(-rows // max(T, 1)))
    for t, dt in ((x_perm, torch.bfloat16), (w2, torch.bfloat16),
                  (expert_offsets, torch.int32), (token_ids, torch.int32),
                  (gate_w, torch.float32)):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise TypeError(f"expected a contiguous CUDA {dt} tensor, got {t.dtype}")
    wl, keep = make_workload(T, H, I, E, topk, splits, counts, rows=rows)
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=x_perm.device)
    need = workspace_size(wl)
    if need == 0:
        raise MoeError(MOE_ERR_UNSUPPORTED, "moe_gemm2_workspace_size")
    if workspace is None or workspace.nbytes < need:
        workspace = _call_workspace(need, x_perm.device, stream)
    vp = ctypes.c_void_p
    args = [vp(x_perm.data_ptr()), vp(w2.data_ptr()), vp(expert_offsets.data_ptr()),
            vp(token_ids.data_ptr()), vp(gate_w.data_ptr()), vp(out.data_ptr()),
            ctypes.byref(wl), int(num_consumers), vp(workspace.ptr),
            ctypes.c_size_t(workspace.nbytes), _stream(stream)]
    if mode is not None:
        tp = vp(trace.data_ptr()) if trace is not None else vp(0)
        tb = trace.numel() * trace.element_size() if trace is not None else 0
        r = lib().moe_gemm2_combine_ex(*args[:8], int(mode), *args[8:], tp, ctypes.c_size_t(tb))
    elif trace is None:
        r = lib().moe_gemm2_combine(*args)
    else:
        r = lib().moe_gemm2_combine_traced(*args, vp(trace.data_ptr()),
                                           ctypes.c_size_t(trace.numel() * trace.element_size()))
    del keep
    if r < 0:
        raise MoeError(r, "moe_gemm2_combine")
    return out, r


def combine_noalloc(x_perm, w2, expert_offsets, token_ids, gate_w, out, T: int,
                    splits: int = 1, topk: Optional[int] = None,
                    counts: Optional[Sequence[int]] = None, num_consumers: int = -1,
                    mode: int = 0, stream=None) -> int:
    """moe_gemm2_combine_noalloc: the stage into the caller's `out` (fp32
    [T, H]) with the library's own scratch as workspace; nothing is
    allocated.  Returns C."""
    import torch
    rows, I = int(x_perm.shape[0]), int(x_perm.shape[1])
    E, H = int(w2.shape[0]), int(w2.shape[2])
    if topk is None:
        topk = max(1, -(-rows // max(T, 1)))
    for t, dt in ((x_perm, torch.bfloat16), (w2, torch.bfloat16),
                  (expert_offsets, torch.int32), (token_ids, torch.int32),
                  (gate_w, torch.float32), (out, torch.float32)):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise TypeError(f"expected a contiguous CUDA {dt} tensor, got {t.dtype}")
    wl, keep = make_workload(T, H, I, E, topk, splits, counts, rows=rows)
    vp = ctypes.c_void_p
    r = lib().moe_gemm2_combine_noalloc(
        vp(x_perm.data_ptr()), vp(w2.data_ptr()), vp(expert_offsets.data_ptr()),
        vp(token_ids.data_ptr()), vp(gate_w.data_ptr()), vp(out.data_ptr()),
        ctypes.byref(wl), int(num_consumers), int(mode), _stream(stream))
    del keep
    if r < 0:
        raise MoeError(r, "moe_gemm2_combine_noalloc")
    return r


# ---- the up-projection and the whole post-router layer -----------------------------

def _check_tensor(t, dt, what):
    if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
        raise TypeError(f"{what}: expected a contiguous CUDA {dt} tensor, got {t.dtype}")


def pack_w1(w_gate_up, stream=None):
    """moe_gemm1_pack_weights: [E, H, 2I] (gate columns, then up columns) to
    the packed layout the up-projection reads; returns a new tensor."""
    import torch
    _check_tensor(w_gate_up, torch.bfloat16, "w_gate_up")
    E, H, N = (int(d) for d in w_gate_up.shape)
    out = torch.empty_like(w_gate_up)
    r = lib().moe_gemm1_pack_weights(ctypes.c_void_p(w_gate_up.data_ptr()),
                                     ctypes.c_void_p(out.data_ptr()), E, H, N // 2, _stream(stream))
    if r < 0:
        raise MoeError(r, "moe_gemm1_pack_weights")
    return out


def layer_workspace_size(wl: Workload) -> int:
    return int(lib().moe_layer_workspace_size(ctypes.byref(wl)))


def gemm1_swiglu(hidden, w1_packed, expert_offsets, token_ids, topk: int, rows: int,
                 counts=None, out=None, workspace: Optional[Workspace] = None, stream=None):
    """moe_gemm1_swiglu on torch device tensors: hidden bf16 [T, H], w1_packed
    bf16 [E, H, 2I]; returns x_perm bf16 [rows, I]."""
    import torch
    _check_tensor(hidden, torch.bfloat16, "hidden")
    _check_tensor(w1_packed, torch.bfloat16, "w1")
    _check_tensor(expert_offsets, torch.int32, "expert_offsets")
    _check_tensor(token_ids, torch.int32, "token_ids")
    T, H = int(hidden.shape[0]), int(hidden.shape[1])
    E, I = int(w1_packed.shape[0]), int(w1_packed.shape[2]) // 2
    wl, keep = make_workload(T, H, I, E, topk, 1, counts, rows=rows)
    if out is None:
        out = torch.empty((max(rows, 1), I), dtype=torch.bfloat16, device=hidden.device)
    if workspace is None:
        workspace = _call_workspace(512, hidden.device, stream)
    vp = ctypes.c_void_p
    r = lib().moe_gemm1_swiglu(vp(hidden.data_ptr()), vp(w1_packed.data_ptr()),
                               vp(expert_offsets.data_ptr()), vp(token_ids.data_ptr()),
                               vp(out.data_ptr()), ctypes.byref(wl), vp(workspace.ptr),
                               ctypes.c_size_t(workspace.nbytes), _stream(stream))
    del keep
    if r < 0:
        raise MoeError(r, "moe_gemm1_swiglu")
    return out


def layer_forward(hidden, w1_packed, w2, expert_offsets, token_ids, gate_w, topk: int,
                  splits: int = 1, counts=None, num_consumers: int = -1, out=None,
                  workspace: Optional[Workspace] = None, stream=None):
    """moe_layer_forward: the up-projection then the down-projection with the
    combine; returns (out fp32 [T, H], C of the second launch)."""
    import torch
    for t, dt, what in ((hidden, torch.bfloat16, "hidden"), (w1_packed, torch.bfloat16, "w1"),
                        (w2, torch.bfloat16, "w2"), (expert_offsets, torch.int32, "offsets"),
                        (token_ids, torch.int32, "token_ids"), (gate_w, torch.float32, "gate_w")):
        _check_tensor(t, dt, what)
    T, H = int(hidden.shape[0]), int(hidden.shape[1])
    E, I = int(w2.shape[0]), int(w2.shape[1])
    rows = int(token_ids.shape[0])
    wl, keep = make_workload(T, H, I, E, topk, splits, counts, rows=rows)
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    need = layer_workspace_size(wl)
    if need == 0:
        raise MoeError(MOE_ERR_UNSUPPORTED, "moe_layer_workspace_size")
    if workspace is None or workspace.nbytes < need:
        workspace = _call_workspace(need, hidden.device, stream)
    vp = ctypes.c_void_p
    r = lib().moe_layer_forward(vp(hidden.data_ptr()), vp(w1_packed.data_ptr()), vp(w2.data_ptr()),
                                vp(expert_offsets.data_ptr()), vp(token_ids.data_ptr()),
                                vp(gate_w.data_ptr()), vp(out.data_ptr()), ctypes.byref(wl),
                                int(num_consumers), vp(workspace.ptr),
                                ctypes.c_size_t(workspace.nbytes), _stream(stream))
    del keep
    if r < 0:
        raise MoeError(r, "moe_layer_forward")
    return out, r
