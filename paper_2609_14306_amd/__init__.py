"""Python binding of libvpce.so: fused vocabulary-projection softmax cross-entropy on MI355X.

Argument marshalling only.  Every step of the computation runs in the HIP
kernels behind the C ABI of ``include/vpce.h``; PyTorch supplies device memory
and the current stream.  There is no fallback: if the library is missing or a
call fails, an exception is raised.

The low-level functions carry the C names (``vp_ce_workspace_size``,
``vp_ce_forward``, ``vp_ce_backward``, ``vp_ce_check``, ``vp_status_str``,
``vp_abi_version``) and take torch tensors; ``forward`` and ``backward``
allocate outputs and workspace and call them.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvpce.so")

VP_OK, VP_ERR_NULL, VP_ERR_SHAPE, VP_ERR_DTYPE, VP_ERR_ORDER = 0, 1, 2, 3, 4
VP_ERR_ALIGN, VP_ERR_WORKSPACE, VP_ERR_TARGET, VP_ERR_HIP, VP_ERR_UNSUPPORTED = 5, 6, 7, 8, 9
VP_F32, VP_BF16 = 0, 1
VP_ACCUMULATE_DW = 1
VP_MAX_SHARDS = 64

EXPORTED = ("vp_ce_workspace_size", "vp_ce_forward", "vp_ce_forward_noalloc", "vp_ce_backward",
            "vp_ce_state_init",
            "vp_ce_fold_shard", "vp_ce_fold_finalize", "vp_ce_plan_info", "vp_ce_check",
            "vp_status_str", "vp_abi_version")


class VpError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {vp_status_str(status)} (status {status})")
        self.status = status


class vp_plan_info(ctypes.Structure):
    _fields_ = [("Tc", ctypes.c_int64), ("Vc", ctypes.c_int64), ("strips", ctypes.c_int64),
                ("stage_launches", ctypes.c_int64)]


class vp_problem(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int64),
        ("d", ctypes.c_int64),
        ("P", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("shard_rows", ctypes.POINTER(ctypes.c_int64)),
        ("order", ctypes.POINTER(ctypes.c_int32)),
        ("ignore_index", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
        ("strip_elems", ctypes.c_int64),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libvpce.so (built by ``paper_2609_14306_amd.build``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_14306_amd.build` "
                           "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp = P(vp_problem)
    vptr = ctypes.c_void_p
    lib.vp_abi_version.restype = ctypes.c_int
    lib.vp_abi_version.argtypes = []
    lib.vp_status_str.restype = ctypes.c_char_p
    lib.vp_status_str.argtypes = [ctypes.c_int]
    lib.vp_ce_workspace_size.restype = ctypes.c_int
    lib.vp_ce_workspace_size.argtypes = [vp, P(ctypes.c_size_t), P(ctypes.c_size_t)]
    lib.vp_ce_forward.restype = ctypes.c_int
    lib.vp_ce_forward.argtypes = [vp, vptr, P(vptr), vptr, vptr, vptr, vptr, ctypes.c_size_t, vptr]
    lib.vp_ce_forward_noalloc.restype = ctypes.c_int
    lib.vp_ce_forward_noalloc.argtypes = [vp, vptr, P(vptr), vptr, vptr, vptr, vptr]
    lib.vp_ce_backward.restype = ctypes.c_int
    lib.vp_ce_backward.argtypes = [vp, vptr, P(vptr), vptr, vptr, vptr, vptr, P(vptr), vptr,
                                   ctypes.c_size_t, vptr]
    lib.vp_ce_state_init.restype = ctypes.c_int
    lib.vp_ce_state_init.argtypes = [vptr, ctypes.c_int64, vptr]
    lib.vp_ce_fold_shard.restype = ctypes.c_int
    lib.vp_ce_fold_shard.argtypes = [vp, ctypes.c_int64, vptr, vptr, vptr, vptr, vptr, ctypes.c_size_t,
                                     vptr]
    lib.vp_ce_fold_finalize.restype = ctypes.c_int
    lib.vp_ce_fold_finalize.argtypes = [vp, vptr, vptr, vptr, vptr, vptr, ctypes.c_size_t, vptr]
    lib.vp_ce_plan_info.restype = ctypes.c_int
    lib.vp_ce_plan_info.argtypes = [vp, P(vp_plan_info)]
    lib.vp_ce_check.restype = ctypes.c_int
    lib.vp_ce_check.argtypes = [vptr, vptr, P(ctypes.c_int64)]
    _lib = lib
    return lib


def vp_abi_version() -> int:
    return int(load_library().vp_abi_version())


def vp_status_str(status: int) -> str:
    return load_library().vp_status_str(int(status)).decode()


class Problem:
    """Owns a ``vp_problem`` and the host arrays it points to."""

    def __init__(self, T: int, d: int, shard_rows: Sequence[int], dtype: int,
                 order: Optional[Sequence[int]] = None, ignore_index: int = -100, flags: int = 0,
                 strip_elems: int = 0):
        P = len(shard_rows)
        self._rows = (ctypes.c_int64 * max(P, 1))(*[int(r) for r in shard_rows])
        self._order = None if order is None else (ctypes.c_int32 * max(P, 1))(*[int(o) for o in order])
        self.c = vp_problem(
            T=int(T), d=int(d), P=P, dtype=int(dtype),
            shard_rows=ctypes.cast(self._rows, ctypes.POINTER(ctypes.c_int64)),
            order=(ctypes.cast(self._order, ctypes.POINTER(ctypes.c_int32)) if self._order is not None
                   else ctypes.POINTER(ctypes.c_int32)()),
            ignore_index=int(ignore_index), flags=int(flags), strip_elems=int(strip_elems))
        self.T, self.d, self.P = int(T), int(d), P
        self.shard_rows = [int(r) for r in shard_rows]


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _ptr_array(ts) -> ctypes.Array:
    return (ctypes.c_void_p * max(len(ts), 1))(*[(_ptr(t) if t is not None and t.numel() else None)
                                                  for t in ts])


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return int(stream)
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def _check(status: int, what: str) -> None:
    if status != VP_OK:
        raise VpError(status, what)


# ---------------------------------------------------------------------------
# Tensor checks.  The C ABI receives bare pointers: element types, widths and
# strides are whatever the caller's tensors hold, so each tensor is checked here
# against the problem before its pointer is taken (a wrong dtype or width would
# make the kernels read or write outside the tensor).  Shape, dtype and layout are
# checked first and the device last, so that every refusal is raised on the host.
def _torch_dtype(code: int):
    import torch
    return torch.bfloat16 if code == VP_BF16 else torch.float32


def _need(t, name: str, dtype, shape) -> None:
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous (row-major)")


def _same_device(named) -> None:
    devs = {(t.device.type, t.device.index) for _, t in named if t is not None}
    if len(devs) > 1:
        raise ValueError("tensors are on different devices: " +
                         ", ".join(f"{n} on {t.device}" for n, t in named if t is not None))
    for n, t in named:
        if t is not None and t.device.type != "cuda":
            raise ValueError(f"{n}: must be on a GPU device, found {t.device}")


def _need_ws(ws, nbytes: int):
    import torch
    if not isinstance(ws, torch.Tensor) or not ws.is_contiguous():
        raise ValueError("ws: expected a contiguous torch.Tensor")
    if ws.numel() * ws.element_size() < nbytes:
        raise ValueError(f"ws: {ws.numel() * ws.element_size()} bytes, the call needs {nbytes}")


def _check_inputs(prob: Problem, H, W_shards, targets):
    import torch
    if len(W_shards) != prob.P:
        raise ValueError(f"W_shards: {len(W_shards)} shards, the problem has {prob.P}")
    dt = _torch_dtype(prob.c.dtype)
    _need(H, "H", dt, (prob.T, prob.d))
    for p, (w, r) in enumerate(zip(W_shards, prob.shard_rows)):
        _need(w, f"W_shards[{p}]", dt, (r, prob.d))
    _need(targets, "targets", torch.int64, (prob.T,))
    return [("H", H), ("targets", targets)] + [(f"W_shards[{p}]", w) for p, w in enumerate(W_shards)]


def vp_ce_workspace_size(prob: Problem) -> Tuple[int, int]:
    f = ctypes.c_size_t(0)
    b = ctypes.c_size_t(0)
    _check(load_library().vp_ce_workspace_size(ctypes.byref(prob.c), ctypes.byref(f), ctypes.byref(b)),
           "vp_ce_workspace_size")
    return int(f.value), int(b.value)


def vp_ce_state_init(state, T: int, stream=None) -> None:
    import torch
    _need(state, "state", torch.float32, (3 * int(T),))
    _same_device([("state", state)])
    _check(load_library().vp_ce_state_init(_ptr(state), int(T), _stream(stream)), "vp_ce_state_init")


def vp_ce_fold_shard(shard: Problem, id_offset: int, H, W_shard, targets, state, ws,
                     stream=None) -> None:
    import torch
    if shard.P != 1:
        raise ValueError("vp_ce_fold_shard: the shard problem must have P == 1")
    named = _check_inputs(shard, H, [W_shard], targets)
    _need(state, "state", torch.float32, (3 * shard.T,))
    _need_ws(ws, vp_ce_workspace_size(shard)[0] if shard.shard_rows[0] > 0 else 0)
    _same_device(named + [("state", state), ("ws", ws)])
    st = load_library().vp_ce_fold_shard(ctypes.byref(shard.c), int(id_offset), _ptr(H),
                                         _ptr(W_shard) if W_shard is not None and W_shard.numel() else None,
                                         _ptr(targets), _ptr(state), _ptr(ws),
                                         ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "vp_ce_fold_shard")


def vp_ce_fold_finalize(prob: Problem, targets, state, loss, lse, ws, stream=None) -> None:
    import torch
    _need(targets, "targets", torch.int64, (prob.T,))
    _need(state, "state", torch.float32, (3 * prob.T,))
    _need(loss, "loss", torch.float32, (prob.T,))
    _need(lse, "lse", torch.float32, (prob.T,))
    _need_ws(ws, 256)
    _same_device([("targets", targets), ("state", state), ("loss", loss), ("lse", lse), ("ws", ws)])
    st = load_library().vp_ce_fold_finalize(ctypes.byref(prob.c), _ptr(targets), _ptr(state), _ptr(loss),
                                            _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(),
                                            _stream(stream))
    _check(st, "vp_ce_fold_finalize")


def vp_ce_plan_info(prob: Problem) -> dict:
    """The backward's strip plan: Tc, Vc, strips and stage_launches (host only)."""
    info = vp_plan_info()
    _check(load_library().vp_ce_plan_info(ctypes.byref(prob.c), ctypes.byref(info)), "vp_ce_plan_info")
    return {"Tc": int(info.Tc), "Vc": int(info.Vc), "strips": int(info.strips),
            "stage_launches": int(info.stage_launches)}


def vp_ce_forward(prob: Problem, H, W_shards, targets, loss, lse, ws, stream=None) -> None:
    import torch
    named = _check_inputs(prob, H, W_shards, targets)
    _need(loss, "loss", torch.float32, (prob.T,))
    _need(lse, "lse", torch.float32, (prob.T,))
    _need_ws(ws, vp_ce_workspace_size(prob)[0])
    _same_device(named + [("loss", loss), ("lse", lse), ("ws", ws)])
    st = load_library().vp_ce_forward(ctypes.byref(prob.c), _ptr(H), _ptr_array(W_shards), _ptr(targets),
                                      _ptr(loss), _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(),
                                      _stream(stream))
    _check(st, "vp_ce_forward")


def vp_ce_forward_noalloc(prob: Problem, H, W_shards, targets, loss, lse, stream=None) -> None:
    """vp_ce_forward with the library's own 16 MiB device workspace (no allocation)."""
    import torch
    named = _check_inputs(prob, H, W_shards, targets)
    _need(loss, "loss", torch.float32, (prob.T,))
    _need(lse, "lse", torch.float32, (prob.T,))
    _same_device(named + [("loss", loss), ("lse", lse)])
    st = load_library().vp_ce_forward_noalloc(ctypes.byref(prob.c), _ptr(H), _ptr_array(W_shards),
                                              _ptr(targets), _ptr(loss), _ptr(lse), _stream(stream))
    _check(st, "vp_ce_forward_noalloc")


def vp_ce_backward(prob: Problem, H, W_shards, targets, lse, grad_loss, dH, dW_shards, ws,
                   stream=None) -> None:
    import torch
    named = _check_inputs(prob, H, W_shards, targets)
    _need(lse, "lse", torch.float32, (prob.T,))
    _need(grad_loss, "grad_loss", torch.float32, (prob.T,))
    _need(dH, "dH", torch.float32, (prob.T, prob.d))
    if len(dW_shards) != prob.P:
        raise ValueError(f"dW_shards: {len(dW_shards)} shards, the problem has {prob.P}")
    for p, (w, r) in enumerate(zip(dW_shards, prob.shard_rows)):
        _need(w, f"dW_shards[{p}]", torch.float32, (r, prob.d))
    _need_ws(ws, vp_ce_workspace_size(prob)[1])
    _same_device(named + [("lse", lse), ("grad_loss", grad_loss), ("dH", dH), ("ws", ws)] +
                 [(f"dW_shards[{p}]", w) for p, w in enumerate(dW_shards)])
    st = load_library().vp_ce_backward(ctypes.byref(prob.c), _ptr(H), _ptr_array(W_shards),
                                       _ptr(targets), _ptr(lse), _ptr(grad_loss), _ptr(dH),
                                       _ptr_array(dW_shards), _ptr(ws),
                                       ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "vp_ce_backward")


def vp_ce_check(ws, stream=None) -> int:
    """Synchronises the stream and returns the number of out-of-range targets found."""
    n = ctypes.c_int64(0)
    st = load_library().vp_ce_check(_ptr(ws), _stream(stream), ctypes.byref(n))
    if st not in (VP_OK, VP_ERR_TARGET):
        _check(st, "vp_ce_check")
    return int(n.value)


# ---------------------------------------------------------------------------
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return VP_BF16
    if t.dtype == torch.float32:
        return VP_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def problem_for(H, W_shards, ignore_index: int = -100, order=None, flags: int = 0,
                strip_elems: int = 0) -> Problem:
    return Problem(H.shape[0], H.shape[1], [w.shape[0] for w in W_shards], _dtype_code(H), order,
                   ignore_index, flags, strip_elems)


def forward(H, W_shards: List, targets, ignore_index: int = -100, order=None, ws=None,
            strip_elems: int = 0):
    """(loss, lse) float32 [T] for hidden states H [T, d] and vocabulary shards W_p [V_p, d]."""
    import torch
    prob = problem_for(H, W_shards, ignore_index, order, 0, strip_elems)
    fwd_b, _ = vp_ce_workspace_size(prob)
    if ws is None:
        ws = torch.empty(fwd_b, dtype=torch.uint8, device=H.device)
    loss = torch.empty(prob.T, dtype=torch.float32, device=H.device)
    lse = torch.empty(prob.T, dtype=torch.float32, device=H.device)
    vp_ce_forward(prob, H, W_shards, targets, loss, lse, ws)
    return loss, lse


def new_state(T: int, device):
    """A fold state float32 [3 * T] set to (-inf, 0, 0) on `device`."""
    import torch
    state = torch.empty(3 * int(T), dtype=torch.float32, device=device)
    vp_ce_state_init(state, T)
    return state


def fold_shard(H, W_shard, id_offset: int, targets, state, ws=None) -> None:
    """Folds the shard W_shard [V_q, d] owning global ids [id_offset, id_offset + V_q) into
    `state` (one meeting of Algorithm 2, in place)."""
    import torch
    if W_shard.shape[0] == 0:
        return  # an empty strip leaves the state unchanged
    shard = problem_for(H, [W_shard])
    fwd_b, _ = vp_ce_workspace_size(shard)
    if ws is None or ws.numel() * ws.element_size() < fwd_b:
        ws = torch.empty(fwd_b, dtype=torch.uint8, device=H.device)
    vp_ce_fold_shard(shard, id_offset, H, W_shard, targets, state, ws)


def fold_finalize(targets, state, shard_rows: Sequence[int], ignore_index: int = -100, ws=None):
    """(loss, lse) float32 [T] from a state that has met every shard of the vocabulary
    whose shards have `shard_rows` rows."""
    import torch
    T = int(targets.shape[0])
    prob = Problem(T, 8, list(shard_rows), VP_BF16, None, ignore_index)
    if ws is None:
        ws = torch.empty(256, dtype=torch.uint8, device=targets.device)
    loss = torch.empty(T, dtype=torch.float32, device=targets.device)
    lse = torch.empty(T, dtype=torch.float32, device=targets.device)
    vp_ce_fold_finalize(prob, targets, state, loss, lse, ws)
    return loss, lse


def backward(H, W_shards: List, targets, lse, grad_loss, ignore_index: int = -100, order=None,
             dW_shards=None, accumulate: bool = False, ws=None, strip_elems: int = 0):
    """(dH [T, d], [dW_p [V_p, d]]) float32, recomputing the logits from the saved lse."""
    import torch
    flags = VP_ACCUMULATE_DW if accumulate else 0
    prob = problem_for(H, W_shards, ignore_index, order, flags, strip_elems)
    _, bwd_b = vp_ce_workspace_size(prob)
    if ws is None:
        ws = torch.empty(bwd_b, dtype=torch.uint8, device=H.device)
    dH = torch.empty(prob.T, prob.d, dtype=torch.float32, device=H.device)
    if dW_shards is None:
        dW_shards = [torch.empty(w.shape[0], prob.d, dtype=torch.float32, device=H.device)
                     for w in W_shards]
    vp_ce_backward(prob, H, W_shards, targets, lse, grad_loss, dH, dW_shards, ws)
    return dH, dW_shards
