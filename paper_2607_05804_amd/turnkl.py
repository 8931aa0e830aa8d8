"""Python binding of libturnkl.so: argument marshalling only.

Every step of the fused turn-KL path runs in the library's HIP kernels; this
module turns torch tensors into device pointers and the current HIP stream,
calls the C ABI (include/turnkl.h) and raises on error.  It loads the
in-tree library and fails loudly if it is missing; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libturnkl.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_ALIAS = -2
ERR_WORKSPACE = -3
ERR_UNSORTED = -4
ERR_TURN_RANGE = -5
ERR_PAD_MASK = -6
ERR_HIP = -7
ERR_SYNC_TIMEOUT = -8
ERR_TOPK_ID = -9
ERR_OUTCOME = -10
ERR_SCRATCH = -11

# Size of the scratch array of turnkl_fwd_bwd_noalloc (TURNKL_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 32 << 20

BF16 = 0
F32 = 1

# Names of every entry point include/turnkl.h declares.
EXPORTS = ("turnkl_workspace_bytes", "turnkl_fwd_bwd", "turnkl_fwd_bwd_noalloc",
           "turnkl_get_status", "turnkl_get_segments", "turnkl_alpha_schedule",
           "turnkl_status_string", "turnkl_topk_workspace_bytes", "turnkl_fwd_bwd_topk",
           "turnkl_depth_default_config", "turnkl_depth_init", "turnkl_depth_plan",
           "turnkl_depth_update", "turnkl_loss_share", "turnkl_budget_report",
           "turnkl_outcome_gap")
# ... and every entry point include/turnkl_testing.h declares (measurement and
# test hooks).
TESTING_EXPORTS = ("turnkl_profile_row_kernel", "turnkl_set_row_tiling",
                   "turnkl_testing_workspace_bytes", "turnkl_set_spin_limit")

STAT_DTYPE = np.dtype([("n_tokens", "<i8"), ("n_traj", "<i8"), ("kl_mean", "<f8"),
                       ("kl_m2", "<f8"), ("kl_var", "<f8"), ("loss_mass", "<f8")])
STAT_FIELDS = 6  # int64, int64, 4 x float64 -> 48 bytes

_lib = None
# The tiling override of turnkl_set_row_tiling is per host thread in the
# library; this mirror lets the binding size workspaces for it.
_thread = threading.local()


class Options(ctypes.Structure):
    """turnkl_options (include/turnkl.h)."""
    _fields_ = [("support_floor", ctypes.c_int32), ("support_frac", ctypes.c_double),
                ("success", ctypes.c_void_p), ("outcome_stats_out", ctypes.c_void_p),
                ("token_weight_out", ctypes.c_void_p), ("token_lse_out", ctypes.c_void_p)]


class DepthConfig(ctypes.Structure):
    """turnkl_depth_config (include/turnkl.h)."""
    _fields_ = [("h_min", ctypes.c_int32), ("h_max", ctypes.c_int32),
                ("warmup_steps", ctypes.c_int32), ("probe_interval", ctypes.c_int32),
                ("min_cov_traj", ctypes.c_int32), ("coverage_quantile", ctypes.c_double),
                ("ema_alpha", ctypes.c_double), ("eps", ctypes.c_double)]


class DepthState(ctypes.Structure):
    """turnkl_depth_state (include/turnkl.h)."""
    _fields_ = [("h_bar", ctypes.c_double), ("h_eff_bar", ctypes.c_double),
                ("h_eff", ctypes.c_int32), ("h_cov", ctypes.c_int32),
                ("h_ctrl", ctypes.c_int32), ("n_probes", ctypes.c_int32)]


class Budget(ctypes.Structure):
    """turnkl_budget (include/turnkl.h)."""
    _fields_ = [("n_min", ctypes.c_int64), ("prefix", ctypes.c_int32), ("third", ctypes.c_int32),
                ("shallow_budget", ctypes.c_double), ("deep_budget", ctypes.c_double),
                ("deep_support", ctypes.c_double), ("deep_shallow_kl", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


class TurnKLError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {status_string(code)} ({code})")
        self.code = code


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; "
                               "g.build()'` (no CPU fallback exists)")
        l = ctypes.CDLL(LIB_PATH)
        c = ctypes
        l.turnkl_workspace_bytes.restype = c.c_size_t
        l.turnkl_workspace_bytes.argtypes = [c.c_int64, c.c_int64, c.c_int, c.c_int32, c.c_int]
        l.turnkl_testing_workspace_bytes.restype = c.c_size_t
        l.turnkl_testing_workspace_bytes.argtypes = [c.c_int64, c.c_int64, c.c_int, c.c_int32,
                                                     c.c_int, c.c_int]
        l.turnkl_fwd_bwd.restype = c.c_int
        l.turnkl_fwd_bwd.argtypes = [
            c.c_void_p, c.c_int64, c.c_void_p, c.c_int64, c.c_int, c.c_int64, c.c_int64,
            c.c_void_p, c.c_void_p, c.c_void_p, c.c_double, c.c_float, c.c_void_p, c.c_void_p,
            c.c_int64, c.c_void_p, c.c_int32, c.c_int, c.c_void_p, c.POINTER(Options),
            c.c_void_p, c.c_size_t, c.c_void_p]
        l.turnkl_fwd_bwd_noalloc.restype = c.c_int
        l.turnkl_fwd_bwd_noalloc.argtypes = [
            c.c_void_p, c.c_int64, c.c_void_p, c.c_int64, c.c_int, c.c_int64, c.c_int64,
            c.c_void_p, c.c_void_p, c.c_void_p, c.c_double, c.c_float, c.c_void_p, c.c_void_p,
            c.c_int64, c.c_void_p, c.c_int32, c.c_int, c.c_void_p, c.POINTER(Options),
            c.c_void_p, c.c_void_p]
        l.turnkl_get_status.restype = c.c_int
        l.turnkl_get_status.argtypes = [c.c_void_p, c.c_void_p]
        l.turnkl_get_segments.restype = c.c_int
        l.turnkl_get_segments.argtypes = [c.c_void_p, c.c_int64, c.c_void_p,
                                          c.POINTER(c.c_int32)] + [c.c_void_p] * 5
        l.turnkl_alpha_schedule.restype = c.c_double
        l.turnkl_alpha_schedule.argtypes = [c.c_int64, c.c_int64, c.c_double, c.c_double]
        l.turnkl_status_string.restype = c.c_char_p
        l.turnkl_status_string.argtypes = [c.c_int]
        l.turnkl_profile_row_kernel.restype = c.c_int
        l.turnkl_profile_row_kernel.argtypes = [c.c_void_p, c.c_void_p]
        l.turnkl_set_row_tiling.restype = c.c_int
        l.turnkl_set_row_tiling.argtypes = [c.c_int]
        l.turnkl_set_spin_limit.restype = c.c_int
        l.turnkl_set_spin_limit.argtypes = [c.c_int]
        l.turnkl_topk_workspace_bytes.restype = c.c_size_t
        l.turnkl_topk_workspace_bytes.argtypes = [c.c_int64, c.c_int32, c.c_int32]
        l.turnkl_fwd_bwd_topk.restype = c.c_int
        l.turnkl_fwd_bwd_topk.argtypes = [
            c.c_void_p, c.c_int64, c.c_int, c.c_int64, c.c_int64, c.c_void_p, c.c_void_p,
            c.c_int64, c.c_int32, c.c_void_p, c.c_void_p, c.c_void_p, c.c_double, c.c_float,
            c.c_void_p, c.c_void_p, c.c_int64, c.c_void_p, c.c_int64, c.c_void_p, c.c_int32,
            c.c_int, c.c_void_p, c.POINTER(Options), c.c_void_p, c.c_size_t, c.c_void_p]
        l.turnkl_depth_default_config.restype = None
        l.turnkl_depth_default_config.argtypes = [c.POINTER(DepthConfig)]
        l.turnkl_depth_init.restype = c.c_int
        l.turnkl_depth_init.argtypes = [c.POINTER(DepthConfig), c.POINTER(DepthState)]
        l.turnkl_depth_plan.restype = c.c_int
        l.turnkl_depth_plan.argtypes = [c.POINTER(DepthConfig), c.POINTER(DepthState), c.c_int64,
                                        c.POINTER(c.c_int32), c.POINTER(c.c_int32),
                                        c.POINTER(c.c_int32)]
        l.turnkl_depth_update.restype = c.c_int
        l.turnkl_depth_update.argtypes = [c.POINTER(DepthConfig), c.POINTER(DepthState), c.c_void_p,
                                          c.c_int32, c.c_void_p, c.c_int64]
        l.turnkl_loss_share.restype = c.c_int
        l.turnkl_loss_share.argtypes = [c.c_void_p, c.c_int32, c.c_void_p]
        l.turnkl_budget_report.restype = c.c_int
        l.turnkl_budget_report.argtypes = [c.c_void_p, c.c_int32, c.c_int64, c.c_int32, c.c_double,
                                           c.POINTER(Budget)]
        l.turnkl_outcome_gap.restype = c.c_int
        l.turnkl_outcome_gap.argtypes = [c.c_void_p, c.c_int32, c.c_void_p]
        _lib = l
    return _lib


def status_string(code: int) -> str:
    return lib().turnkl_status_string(code).decode()


def alpha_schedule(k: int, K: int, s: float = 0.0, e: float = 1.0) -> float:
    return float(lib().turnkl_alpha_schedule(k, K, s, e))


def workspace_bytes(n_tokens: int, vocab: int, dtype: int, max_turns: int,
                    aligned_rows: bool = True) -> int:
    """turnkl_workspace_bytes; under a tiling override of this thread
    (set_row_tiling), turnkl_testing_workspace_bytes for that tiling."""
    vpt = getattr(_thread, "vpt", 0)
    if vpt:
        return int(lib().turnkl_testing_workspace_bytes(n_tokens, vocab, dtype, max_turns,
                                                        int(bool(aligned_rows)), vpt))
    return int(lib().turnkl_workspace_bytes(n_tokens, vocab, dtype, max_turns,
                                            int(bool(aligned_rows))))


def set_row_tiling(vectors_per_thread: int) -> None:
    """Tiling override for this thread (turnkl_testing.h); 0 restores the default."""
    rc = lib().turnkl_set_row_tiling(vectors_per_thread)
    if rc != OK:
        raise TurnKLError(rc, "turnkl_set_row_tiling")
    _thread.vpt = int(vectors_per_thread)


def set_spin_limit(polls: int) -> None:
    """Bound on the row kernel's cross-workgroup wait for this thread (0: default)."""
    rc = lib().turnkl_set_spin_limit(polls)
    if rc != OK:
        raise TurnKLError(rc, "turnkl_set_spin_limit")


def profile_row_kernel(before, after) -> None:
    """Record torch.cuda.Event objects around the row kernel of later calls (None, None: stop)."""
    b = ctypes.c_void_p(before.cuda_event) if before is not None else None
    a = ctypes.c_void_p(after.cuda_event) if after is not None else None
    lib().turnkl_profile_row_kernel(b, a)


def _options(n: int, support_floor: int, support_frac: float, success, outcome_stats,
             token_weights=None, token_lse=None, device=None):
    """turnkl_options for the keyword arguments, or None when all are off."""
    for t, name in ((success, "success"), (token_weights, "token_weights"),
                    (token_lse, "token_lse")):
        if t is not None and device is not None and t.device != device:
            raise ValueError(f"{name} must be on {device}, not {t.device}")
    if (not support_floor and not support_frac and success is None and outcome_stats is None
            and token_weights is None and token_lse is None):
        return None
    if success is not None and (success.dtype != torch.uint8 or success.numel() != n):
        raise ValueError("success must be uint8 with one entry per row")
    for t, per, name in ((token_weights, 1, "token_weights"), (token_lse, 2, "token_lse")):
        if t is not None and (t.dtype != torch.float32 or t.numel() != per * n
                              or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 tensor of {per} x n_tokens")
    return ctypes.byref(Options(int(support_floor), float(support_frac), _ptr(success),
                                _ptr(outcome_stats), _ptr(token_weights), _ptr(token_lse)))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _row_stride(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("logits must be 2-D with unit column stride")
    return int(t.stride(0)) if t.shape[0] > 1 else int(max(t.stride(0), t.shape[1]))


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need(t: torch.Tensor | None, nbytes: int, name: str, device, dtype=None) -> None:
    """A caller buffer the kernels write or read by size: on the logits'
    device, contiguous, of the given dtype and at least nbytes long (the C ABI
    takes bare pointers and cannot check this)."""
    if t is None:
        return
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, not {t.device}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, not {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes; the call needs {nbytes}")


def _check_common(student, n, max_turns, turn_id, traj_id, loss_mask, turn_stats, outcome_stats,
                  kl_t, grad_t):
    dev = student.device
    for t, name in ((turn_id, "turn_id"), (traj_id, "traj_id"), (loss_mask, "loss_mask")):
        _need(t, 0, name, dev)
    stat_bytes = int(max_turns) * STAT_DTYPE.itemsize
    _need(turn_stats, stat_bytes, "turn_stats", dev)
    _need(outcome_stats, 2 * stat_bytes, "outcome_stats", dev)
    _need(kl_t, 4 * n, "token_kl", dev, torch.float32)
    if grad_t is not None and grad_t is not student:
        if grad_t.device != dev or grad_t.dtype != student.dtype or grad_t.shape != student.shape:
            raise ValueError("grad must match the student logits' device, dtype and shape")


def _rows_aligned(*tensors) -> bool:
    """Whether every row of these logit or gradient matrices starts on a
    16-byte boundary (base address and row stride in bytes)."""
    for t in tensors:
        if t is None or t.dim() != 2 or t.shape[0] == 0:
            continue
        if t.data_ptr() % 16 or (t.stride(0) * t.element_size()) % 16:
            return False
    return True


class Workspace:
    """Caller-owned device scratch for turnkl_fwd_bwd (a uint8 torch tensor).

    aligned_rows: the calls it serves pass logit and gradient rows that start
    on 16-byte boundaries (turnkl_workspace_bytes); False sizes it for any
    rows."""

    def __init__(self, n_tokens: int, vocab: int, dtype: int, max_turns: int, device="cuda",
                 aligned_rows: bool = True):
        nbytes = workspace_bytes(n_tokens, vocab, dtype, max_turns, aligned_rows)
        if nbytes == 0:
            raise TurnKLError(ERR_INVALID_ARG, "turnkl_workspace_bytes")
        self.tensor = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.nbytes = nbytes
        self.n_tokens = n_tokens

    def status(self) -> int:
        stream = torch.cuda.current_stream().cuda_stream
        return int(lib().turnkl_get_status(_ptr(self.tensor), ctypes.c_void_p(stream)))

    def segments(self, device="cuda") -> dict:
        n = self.n_tokens
        bufs = [torch.empty(max(n, 1), dtype=torch.int32, device=device) for _ in range(5)]
        n_seg = ctypes.c_int32(0)
        stream = torch.cuda.current_stream().cuda_stream
        rc = lib().turnkl_get_segments(_ptr(self.tensor), n, ctypes.c_void_p(stream),
                                       ctypes.byref(n_seg), *[_ptr(b) for b in bufs])
        if rc != OK:
            raise TurnKLError(rc, "turnkl_get_segments")
        k = n_seg.value
        names = ("start", "length", "traj", "turn", "n_sup")
        return {nm: b[:k].cpu().numpy().astype(np.int64) for nm, b in zip(names, bufs)}


def _check_fused_inputs(student, teacher, turn_id, traj_id, loss_mask):
    """dtype code, n_tokens and vocab of a fused call, after checking its inputs."""
    dt = _dtype_code(student)
    if teacher.dtype != student.dtype:
        raise TypeError("student and teacher logits must share a dtype")
    if teacher.shape != student.shape or teacher.device != student.device:
        raise ValueError("student and teacher logits must share a shape and a device")
    n, v = (int(student.shape[0]), int(student.shape[1])) if student.dim() == 2 else (0, 0)
    for t in (turn_id, traj_id):
        if t.dtype != torch.int32 or t.numel() != n:
            raise ValueError("turn_id / traj_id must be int32 with one entry per row")
    if loss_mask.dtype != torch.uint8 or loss_mask.numel() != n:
        raise ValueError("loss_mask must be uint8 with one entry per row")
    return dt, n, v


def _fused_args(student, teacher, dt, n, v, turn_id, traj_id, loss_mask, alpha, grad_scale,
                loss, grad_t, turn_stats, max_turns, accumulate_stats, kl_t, options):
    """The arguments turnkl_fwd_bwd and turnkl_fwd_bwd_noalloc share, in order."""
    return [_ptr(student), _row_stride(student) if n else v, _ptr(teacher),
            _row_stride(teacher) if n else v, dt, n, v, _ptr(turn_id), _ptr(traj_id),
            _ptr(loss_mask), float(alpha), float(grad_scale), _ptr(loss), _ptr(grad_t),
            (_row_stride(grad_t) if n else v) if grad_t is not None else 0, _ptr(turn_stats),
            int(max_turns), int(bool(accumulate_stats)), _ptr(kl_t), options]


def fwd_bwd(student: torch.Tensor, teacher: torch.Tensor, turn_id: torch.Tensor,
            traj_id: torch.Tensor, loss_mask: torch.Tensor, alpha: float, *,
            grad_scale: float = 1.0, grad: str | torch.Tensor | None = "new",
            max_turns: int = 64, turn_stats: torch.Tensor | None = None,
            accumulate_stats: bool = False, token_kl: bool | torch.Tensor = False,
            workspace: Workspace | None = None, check: bool = True, support_floor: int = 0,
            support_frac: float = 0.0, success: torch.Tensor | None = None,
            outcome_stats: torch.Tensor | None = None, token_weights: torch.Tensor | None = None,
            token_lse: torch.Tensor | None = None):
    """One fused forward + backward call on the current stream.

    grad: "new" allocates the gradient, "inplace" writes it over `student`,
    a tensor is used as the output, None computes the forward only.
    turn_stats: optional [max_turns * 6] float64-compatible device buffer in
    the turnkl_turn_stat layout (use new_turn_stats()); accumulate_stats
    merges into it.  support_floor / support_frac: the turn-support floor of
    the turn term; success (uint8 per token) with outcome_stats (a
    new_turn_stats(2 * max_turns) buffer: failed, then successful): the
    per-outcome statistics (turnkl_options).  token_weights (float32 [N]) and
    token_lse (float32 [N, 2]) receive each token's weight w_i and the
    log-partition functions of its student and teacher rows (NaN for
    unsupervised tokens).  Returns (loss[3] tensor, grad or None, turn_stats or
    None, token_kl or None, workspace).
    """
    dt, n, v = _check_fused_inputs(student, teacher, turn_id, traj_id, loss_mask)
    dev = student.device
    if isinstance(grad, str):
        if grad == "new":
            grad_t = torch.empty_like(student)
        elif grad == "inplace":
            grad_t = student
        else:
            raise ValueError(grad)
    else:
        grad_t = grad
    if workspace is None:
        workspace = Workspace(n, v, dt, max_turns, device=dev,
                              aligned_rows=_rows_aligned(student, teacher, grad_t))
    loss = torch.empty(3, dtype=torch.float32, device=dev)
    if isinstance(token_kl, torch.Tensor):
        kl_t = token_kl
    else:
        kl_t = torch.empty(max(n, 1), dtype=torch.float32, device=dev) if token_kl else None
    _check_common(student, n, max_turns, turn_id, traj_id, loss_mask, turn_stats, outcome_stats,
                  kl_t, grad_t)
    stream = torch.cuda.current_stream(dev).cuda_stream
    opts = _options(n, support_floor, support_frac, success, outcome_stats, token_weights,
                    token_lse, dev)
    rc = lib().turnkl_fwd_bwd(
        *_fused_args(student, teacher, dt, n, v, turn_id, traj_id, loss_mask, alpha, grad_scale,
                     loss, grad_t, turn_stats, max_turns, accumulate_stats, kl_t, opts),
        _ptr(workspace.tensor), workspace.nbytes, ctypes.c_void_p(stream))
    if rc != OK:
        raise TurnKLError(rc, "turnkl_fwd_bwd")
    if check:
        st = workspace.status()
        if st != OK:
            raise TurnKLError(st, "turnkl_fwd_bwd (device)")
    return loss, grad_t, turn_stats, kl_t, workspace


def fwd_bwd_noalloc(student: torch.Tensor, teacher: torch.Tensor, turn_id: torch.Tensor,
                    traj_id: torch.Tensor, loss_mask: torch.Tensor, alpha: float,
                    loss: torch.Tensor, *, grad_scale: float = 1.0,
                    grad: str | torch.Tensor | None = None, max_turns: int = 64,
                    turn_stats: torch.Tensor | None = None, accumulate_stats: bool = False,
                    token_kl: torch.Tensor | None = None, status: torch.Tensor | None = None,
                    support_floor: int = 0, support_frac: float = 0.0,
                    success: torch.Tensor | None = None,
                    outcome_stats: torch.Tensor | None = None,
                    token_weights: torch.Tensor | None = None,
                    token_lse: torch.Tensor | None = None) -> None:
    """turnkl_fwd_bwd_noalloc on the current stream: the fused call with the
    library's built-in scratch instead of a workspace.  Neither the library
    nor this function allocates: every output is the caller's tensor.

    loss: float32 [3]; grad: a tensor, "inplace" or None (forward only);
    token_kl: float32 [N] or None; status: int32 [1] or None, receives the
    device-side status (OK or the data error) when the call's last kernel
    runs.  The other arguments are those of fwd_bwd.  Calls that can overlap
    in time on one GPU share the scratch and race.
    """
    dt, n, v = _check_fused_inputs(student, teacher, turn_id, traj_id, loss_mask)
    dev = student.device
    grad_t = student if (isinstance(grad, str) and grad == "inplace") else grad
    if isinstance(grad_t, str):
        raise ValueError(grad)
    _need(loss, 12, "loss", dev, torch.float32)
    _need(status, 4, "status", dev, torch.int32)
    _check_common(student, n, max_turns, turn_id, traj_id, loss_mask, turn_stats, outcome_stats,
                  token_kl, grad_t)
    stream = torch.cuda.current_stream(dev).cuda_stream
    opts = _options(n, support_floor, support_frac, success, outcome_stats, token_weights,
                    token_lse, dev)
    rc = lib().turnkl_fwd_bwd_noalloc(
        *_fused_args(student, teacher, dt, n, v, turn_id, traj_id, loss_mask, alpha, grad_scale,
                     loss, grad_t, turn_stats, max_turns, accumulate_stats, token_kl, opts),
        _ptr(status), ctypes.c_void_p(stream))
    if rc != OK:
        raise TurnKLError(rc, "turnkl_fwd_bwd_noalloc")


class TopkWorkspace(Workspace):
    """Caller-owned device scratch for turnkl_fwd_bwd_topk."""

    def __init__(self, n_tokens: int, k: int, max_turns: int, device="cuda"):
        nbytes = int(lib().turnkl_topk_workspace_bytes(n_tokens, k, max_turns))
        if nbytes == 0:
            raise TurnKLError(ERR_INVALID_ARG, "turnkl_topk_workspace_bytes")
        self.tensor = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.nbytes = nbytes
        self.n_tokens = n_tokens


def fwd_bwd_topk(student: torch.Tensor, teacher_ids: torch.Tensor, teacher_vals: torch.Tensor,
                 turn_id: torch.Tensor, traj_id: torch.Tensor, loss_mask: torch.Tensor,
                 alpha: float, *, grad_scale: float = 1.0,
                 grad: str | torch.Tensor | None = "new", grad_topk: bool | torch.Tensor = False,
                 max_turns: int = 64, turn_stats: torch.Tensor | None = None,
                 accumulate_stats: bool = False, token_kl: bool | torch.Tensor = False,
                 workspace: TopkWorkspace | None = None, check: bool = True,
                 support_floor: int = 0, support_frac: float = 0.0,
                 success: torch.Tensor | None = None, outcome_stats: torch.Tensor | None = None,
                 token_weights: torch.Tensor | None = None, token_lse: torch.Tensor | None = None):
    """The top-K variant (turnkl_fwd_bwd_topk) on the current stream.

    teacher_ids: int32 [N, K]; teacher_vals: float32 [N, K].  grad as in
    fwd_bwd (dense, zero off the support); grad_topk: True allocates, or a
    float32 [N, K] tensor receives, the gradient on the support; the options
    as in fwd_bwd (token_lse: log-partition functions over each token's
    support).  Returns
    (loss[3], grad or None, grad_topk or None, turn_stats or None,
    token_kl or None, workspace).
    """
    dt = _dtype_code(student)
    n, v = (int(student.shape[0]), int(student.shape[1])) if student.dim() == 2 else (0, 0)
    if teacher_ids.dtype != torch.int32 or teacher_vals.dtype != torch.float32:
        raise TypeError("teacher_ids must be int32 and teacher_vals float32")
    if teacher_ids.dim() != 2 or teacher_ids.shape != teacher_vals.shape or teacher_ids.shape[0] != n:
        raise ValueError("teacher_ids / teacher_vals must both be [n_tokens, K]")
    if teacher_ids.stride() != teacher_vals.stride():
        raise ValueError("teacher_ids and teacher_vals must share a row stride")
    k = int(teacher_ids.shape[1])
    for t in (turn_id, traj_id):
        if t.dtype != torch.int32 or t.numel() != n:
            raise ValueError("turn_id / traj_id must be int32 with one entry per row")
    if loss_mask.dtype != torch.uint8 or loss_mask.numel() != n:
        raise ValueError("loss_mask must be uint8 with one entry per row")
    dev = student.device
    if isinstance(grad, str):
        if grad == "new":
            grad_t = torch.empty_like(student)
        elif grad == "inplace":
            grad_t = student
        else:
            raise ValueError(grad)
    else:
        grad_t = grad
    if isinstance(grad_topk, torch.Tensor):
        gk = grad_topk
    else:
        gk = torch.empty((max(n, 1), k), dtype=torch.float32, device=dev) if grad_topk else None
    if workspace is None:
        workspace = TopkWorkspace(n, k, max_turns, device=dev)
    loss = torch.empty(3, dtype=torch.float32, device=dev)
    if isinstance(token_kl, torch.Tensor):
        kl_t = token_kl
    else:
        kl_t = torch.empty(max(n, 1), dtype=torch.float32, device=dev) if token_kl else None
    _check_common(student, n, max_turns, turn_id, traj_id, loss_mask, turn_stats, outcome_stats,
                  kl_t, grad_t)
    for t, name in ((teacher_ids, "teacher_ids"), (teacher_vals, "teacher_vals")):
        if t.device != dev or (n and t.stride(1) != 1):
            raise ValueError(f"{name} must be on the logits' device with unit column stride")
    if gk is not None and (gk.device != dev or gk.dtype != torch.float32 or gk.dim() != 2
                           or gk.shape[0] < n or gk.shape[1] != k or (n and gk.stride(1) != 1)):
        raise ValueError("grad_topk must be float32 [n_tokens, K] with unit column stride")
    stream = torch.cuda.current_stream(dev).cuda_stream
    ld_k = int(teacher_ids.stride(0)) if n else k
    rc = lib().turnkl_fwd_bwd_topk(
        _ptr(student), _row_stride(student) if n else v, dt, n, v, _ptr(teacher_ids),
        _ptr(teacher_vals), ld_k, k, _ptr(turn_id), _ptr(traj_id), _ptr(loss_mask), float(alpha),
        float(grad_scale), _ptr(loss), _ptr(grad_t),
        (_row_stride(grad_t) if n else v) if grad_t is not None else 0, _ptr(gk),
        (int(gk.stride(0)) if n else k) if gk is not None else 0, _ptr(turn_stats),
        int(max_turns), int(bool(accumulate_stats)), _ptr(kl_t),
        _options(n, support_floor, support_frac, success, outcome_stats, token_weights, token_lse,
                 dev),
        _ptr(workspace.tensor),
        workspace.nbytes, ctypes.c_void_p(stream))
    if rc != OK:
        raise TurnKLError(rc, "turnkl_fwd_bwd_topk")
    if check:
        st = workspace.status()
        if st != OK:
            raise TurnKLError(st, "turnkl_fwd_bwd_topk (device)")
    return loss, grad_t, gk, turn_stats, kl_t, workspace


def new_turn_stats(max_turns: int, device="cuda") -> torch.Tensor:
    """Zeroed [max_turns] turnkl_turn_stat buffer (48 bytes each) as a uint8 tensor."""
    return torch.zeros(max_turns * STAT_DTYPE.itemsize, dtype=torch.uint8, device=device)


def read_turn_stats(buf: torch.Tensor) -> np.ndarray:
    return buf.cpu().numpy().view(STAT_DTYPE)


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise TurnKLError(rc, what)


class DepthController:
    """The adaptive rollout-depth controller (turnkl_depth_*; host code).

    plan(k) -> (cap, probe, rollout_depth) for step k = 1, 2, ...;
    update(stats, success_lengths) after a probe step, with the probe batch's
    per-turn statistics (the buffer turnkl_fwd_bwd filled, on any device, or
    a STAT_DTYPE array) and the turn counts of its successful trajectories.
    """

    def __init__(self, **overrides):
        l = lib()
        self.config = DepthConfig()
        l.turnkl_depth_default_config(ctypes.byref(self.config))
        for k, v in overrides.items():
            setattr(self.config, k, v)
        self.state = DepthState()
        _check(l.turnkl_depth_init(ctypes.byref(self.config), ctypes.byref(self.state)),
               "turnkl_depth_init")

    def plan(self, step: int):
        cap, probe, roll = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().turnkl_depth_plan(ctypes.byref(self.config), ctypes.byref(self.state), step,
                                       ctypes.byref(cap), ctypes.byref(probe), ctypes.byref(roll)),
               "turnkl_depth_plan")
        return cap.value, bool(probe.value), roll.value

    def update(self, stats, success_lengths=()) -> None:
        if isinstance(stats, torch.Tensor):
            stats = read_turn_stats(stats)
        st = np.ascontiguousarray(stats, dtype=STAT_DTYPE)
        ln = np.ascontiguousarray(np.asarray(success_lengths, dtype=np.int32))
        _check(lib().turnkl_depth_update(ctypes.byref(self.config), ctypes.byref(self.state),
                                         st.ctypes.data, st.shape[0],
                                         ln.ctypes.data if ln.size else None, ln.size),
               "turnkl_depth_update")


def _host_stats(stats) -> np.ndarray:
    if isinstance(stats, torch.Tensor):
        stats = read_turn_stats(stats)
    return np.ascontiguousarray(stats, dtype=STAT_DTYPE).reshape(-1)


def loss_share(stats) -> np.ndarray:
    """s_t of a batch's per-turn statistics (turnkl_loss_share; host code)."""
    st = _host_stats(stats)
    out = np.zeros(st.shape[0], np.float64)
    _check(lib().turnkl_loss_share(st.ctypes.data, st.shape[0], out.ctypes.data),
           "turnkl_loss_share")
    return out


def budget_report(stats, n_traj: int, support_floor: int = 8, support_frac: float = 0.15) -> dict:
    """Deep/shallow budget, support and raw-KL ratio over the reliable turn
    prefix (turnkl_budget_report; host code)."""
    st = _host_stats(stats)
    b = Budget()
    _check(lib().turnkl_budget_report(st.ctypes.data, st.shape[0], int(n_traj), int(support_floor),
                                      float(support_frac), ctypes.byref(b)),
           "turnkl_budget_report")
    return b.as_dict()


def outcome_gap(outcome_stats) -> np.ndarray:
    """G_t from the [2 * T] per-outcome statistics (turnkl_outcome_gap)."""
    st = _host_stats(outcome_stats)
    if st.shape[0] % 2:
        raise ValueError("outcome statistics hold 2 * max_turns entries")
    out = np.zeros(st.shape[0] // 2, np.float64)
    _check(lib().turnkl_outcome_gap(st.ctypes.data, st.shape[0] // 2, out.ctypes.data),
           "turnkl_outcome_gap")
    return out
