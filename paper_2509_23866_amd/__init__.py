"""Python binding of libdart (the C ABI declared in include/dart.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
``csrc/dart.hip``. torch supplies device memory and the stream. The library must
be built (``__graft_entry__.build()``); if it is missing, importing a function
raises — there is no CPU fallback.

Functions carry the C names: ``dart_tok_stats``, ``dart_step_select``,
``dart_tis_loss_fwd_bwd`` (and its halves ``dart_tis_loss_fwd`` /
``dart_tis_grad``), the ``_ex`` variants (inverse temperature, the KL term,
aggregation and ratio level, zero-row skipping), ``dart_tis_loss_workspace_bytes``,
``dart_kept_steps`` and ``dart_status_string``. ``policy_update`` chains the
device calls.
"""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdart.so")

DART_OK = 0
DART_ERR_INVALID_ARG = 1
DART_ERR_UNSUPPORTED = 2
DART_ERR_HIP = 3
DART_F32 = 0
DART_BF16 = 1

DART_KL = {"none": 0, "k1": 1, "k2": 2, "k3": 3}
DART_AGG = {"token_mean": 0, "token_mean_all": 1, "step_mean": 2}
DART_RATIO = {"token": 0, "step_geomean": 1, "step_product": 2}
DART_GRAD_SKIP_ZERO_ROWS = 1
DART_LMHEAD_SKIP_ZERO_ROWS = 1
DART_LMHEAD_BF16_GRADS = 4

EXPORTED = ("dart_tok_stats", "dart_step_select", "dart_tis_loss_fwd_bwd", "dart_tis_loss_fwd",
            "dart_tis_grad", "dart_tis_loss_fwd_bwd_noalloc", "dart_select_tis_loss_fwd",
            "dart_tok_stats_ex", "dart_tis_loss_fwd_ex", "dart_tis_grad_ex",
            "dart_grpo_advantage", "dart_step_select_groups", "dart_tis_loss_workspace_bytes",
            "dart_lmhead_tok_stats", "dart_lmhead_tok_stats_ex", "dart_lmhead_stats_workspace_bytes",
            "dart_lmhead_dlogits", "dart_lmhead_dlogits_ex",
            "dart_lmhead_backward", "dart_lmhead_backward_workspace_bytes",
            "dart_lmhead_backward_ex", "dart_lmhead_backward_ex_workspace_bytes", "dart_kept_steps",
            "dart_status_string")


class dart_loss_config_t(ctypes.Structure):
    """Mirror of the C struct dart_loss_config_t."""

    _fields_ = [("eps_low", ctypes.c_float), ("eps_high", ctypes.c_float), ("C", ctypes.c_float),
                ("kl", ctypes.c_int32), ("beta", ctypes.c_float), ("aggregation", ctypes.c_int32),
                ("ratio", ctypes.c_int32)]


class DartError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} failed: {dart_status_string(code)} ({code})")
        self.code = code


_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def load_library():
    """Open libdart.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        lib.dart_tok_stats.restype = ctypes.c_int
        lib.dart_tok_stats.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P]
        lib.dart_step_select.restype = ctypes.c_int
        lib.dart_step_select.argtypes = [_P, _I64, _P, _I64, ctypes.c_double, _P, _P, _P, _P]
        lib.dart_tis_loss_fwd_bwd.restype = ctypes.c_int
        lib.dart_tis_loss_fwd_bwd.argtypes = [
            _P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _I64, _P,
            ctypes.c_float, ctypes.c_float, ctypes.c_float, _P, _I64, _P, _P, _P, _P,
            ctypes.c_size_t, _P]
        lib.dart_tis_loss_fwd_bwd_noalloc.restype = ctypes.c_int
        lib.dart_tis_loss_fwd_bwd_noalloc.argtypes = [
            _P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _I64, _P,
            ctypes.c_float, ctypes.c_float, ctypes.c_float, _P, _I64, _P, _P, _P, _P]
        lib.dart_tis_loss_fwd.restype = ctypes.c_int
        lib.dart_tis_loss_fwd.argtypes = [_I64, _P, _P, _P, _P, _P, _I64, _P, ctypes.c_float,
                                          ctypes.c_float, ctypes.c_float, _P, _P, _P, _P,
                                          ctypes.c_size_t, _P]
        lib.dart_select_tis_loss_fwd.restype = ctypes.c_int
        lib.dart_select_tis_loss_fwd.argtypes = [
            _I64, _P, _P, _P, _P, _P, _P, _I64, ctypes.c_double, ctypes.c_float, ctypes.c_float,
            ctypes.c_float, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
        lib.dart_tis_loss_workspace_bytes.restype = ctypes.c_size_t
        lib.dart_tis_loss_workspace_bytes.argtypes = [_I64]
        lib.dart_tis_grad.restype = ctypes.c_int
        lib.dart_tis_grad.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P,
                                      _I64, _P]
        lib.dart_tok_stats_ex.restype = ctypes.c_int
        lib.dart_tok_stats_ex.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, ctypes.c_float,
                                          _P, _P, _P, _P]
        lib.dart_tis_loss_fwd_ex.restype = ctypes.c_int
        lib.dart_tis_loss_fwd_ex.argtypes = [_I64, _P, _P, _P, _P, _P, _P, _I64, _P,
                                             ctypes.POINTER(dart_loss_config_t), _P, _P, _P, _P,
                                             ctypes.c_size_t, _P]
        lib.dart_tis_grad_ex.restype = ctypes.c_int
        lib.dart_tis_grad_ex.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P,
                                         ctypes.c_float, ctypes.c_uint32, _P, _I64, _P]
        lib.dart_grpo_advantage.restype = ctypes.c_int
        lib.dart_grpo_advantage.argtypes = [_P, _I64, _P, _P, _I64, _P, _I64, _I64, _P, _P, _P, _P]
        lib.dart_step_select_groups.restype = ctypes.c_int
        lib.dart_step_select_groups.argtypes = [_P, _I64, _P, _I64, _P, _I64, ctypes.c_double, _P,
                                                _P, _P, _P]
        lib.dart_lmhead_tok_stats.restype = ctypes.c_int
        lib.dart_lmhead_tok_stats.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _P, _P,
                                              _P, ctypes.c_size_t, _P]
        lib.dart_lmhead_tok_stats_ex.restype = ctypes.c_int
        lib.dart_lmhead_tok_stats_ex.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P,
                                                 ctypes.c_float, _P, _P, _P, _P, ctypes.c_size_t,
                                                 _P]
        lib.dart_lmhead_stats_workspace_bytes.restype = ctypes.c_size_t
        lib.dart_lmhead_stats_workspace_bytes.argtypes = [_I64, _I64]
        lib.dart_lmhead_dlogits.restype = ctypes.c_int
        lib.dart_lmhead_dlogits.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _P, _P,
                                            _P, _I64, _P]
        lib.dart_lmhead_dlogits_ex.restype = ctypes.c_int
        lib.dart_lmhead_dlogits_ex.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _P,
                                               _P, ctypes.c_float, _P, _I64, _P]
        lib.dart_lmhead_backward.restype = ctypes.c_int
        lib.dart_lmhead_backward.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _P, _P,
                                             _P, _I64, _P, _I64, _I64, _P, ctypes.c_size_t, _P]
        lib.dart_lmhead_backward_workspace_bytes.restype = ctypes.c_size_t
        lib.dart_lmhead_backward_workspace_bytes.argtypes = [_I64, _I64]
        lib.dart_lmhead_backward_ex.restype = ctypes.c_int
        lib.dart_lmhead_backward_ex.argtypes = [_P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _P,
                                                _P, ctypes.c_float, _P, _I64, _P, _I64, _I64,
                                                _I64, ctypes.c_uint32, _P, ctypes.c_size_t, _P]
        lib.dart_lmhead_backward_ex_workspace_bytes.restype = ctypes.c_size_t
        lib.dart_lmhead_backward_ex_workspace_bytes.argtypes = [_I64, _I64, _I64, _I64, _I64,
                                                                ctypes.c_uint32]
        lib.dart_kept_steps.restype = _I64
        lib.dart_kept_steps.argtypes = [_I64, ctypes.c_double]
        lib.dart_status_string.restype = ctypes.c_char_p
        lib.dart_status_string.argtypes = [ctypes.c_int]
        _lib = lib
    return _lib


def dart_status_string(code: int) -> str:
    return load_library().dart_status_string(int(code)).decode()


def dart_kept_steps(S: int, rho: float) -> int:
    return int(load_library().dart_kept_steps(int(S), float(rho)))


def _torch():
    import torch

    return torch


def _stream_handle(stream, device):
    """The HIP stream a call enqueues on: for None the current stream of the
    inputs' device (not of the current device); a torch stream, which must
    belong to the inputs' device; or a raw hipStream_t handle, taken as given."""
    torch = _torch()
    if stream is None:
        return torch.cuda.current_stream(device).cuda_stream
    if hasattr(stream, "cuda_stream"):
        if torch.device(stream.device) != torch.device(device):
            raise ValueError(f"the stream is on {stream.device}, the inputs on {device}")
        return stream.cuda_stream
    return int(stream)


def _ptr(t):
    return None if t is None else t.data_ptr()


def dart_tis_loss_workspace_bytes(T: int) -> int:
    return int(load_library().dart_tis_loss_workspace_bytes(int(T)))


def _workspace(workspace, T, device, stream):
    """(pointer, bytes, tensor) for the loss workspace: "auto" allocates one
    from torch's caching allocator (kept for the stream the call runs on),
    None passes NULL (one-workgroup loss), a uint8 tensor is used as given."""
    torch = _torch()
    if workspace is None:
        return None, 0, None
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError('workspace must be "auto", None or a uint8 device tensor')
        workspace = torch.empty(dart_tis_loss_workspace_bytes(T), dtype=torch.uint8, device=device)
        if isinstance(stream, torch.cuda.Stream):
            workspace.record_stream(stream)
    if (not isinstance(workspace, torch.Tensor) or workspace.dtype != torch.uint8
            or workspace.device != device or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor on the device of the inputs")
    return workspace.data_ptr(), workspace.numel(), workspace


def _check_vec(name, t, dtype, n, device):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != dtype or t.device != device or t.dim() != 1 or t.numel() != n or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} vector of {n} elements on {device}")


def _logits_meta(logits):
    torch = _torch()
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a 2-D tensor with contiguous rows")
    if logits.dtype == torch.bfloat16:
        dt = DART_BF16
    elif logits.dtype == torch.float32:
        dt = DART_F32
    else:
        raise TypeError("logits must be bfloat16 or float32")
    if not logits.is_cuda:
        raise ValueError("logits must be on a GPU")
    return dt, logits.shape[0], logits.shape[1], logits.stride(0)


def dart_tok_stats(logits, target, logp=None, entropy=None, lse=None, stream=None, inv_temp=1.0):
    """Per-token log-prob of the target, entropy and log-normaliser (float32 [T]
    each) of softmax(inv_temp * logits)."""
    torch = _torch()
    dt, T, V, ld = _logits_meta(logits)
    dev = logits.device
    _check_vec("target", target, torch.int32, T, dev)
    logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
    entropy = torch.empty(T, dtype=torch.float32, device=dev) if entropy is None else entropy
    lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
    for n, v in (("logp", logp), ("entropy", entropy), ("lse", lse)):
        _check_vec(n, v, torch.float32, T, dev)
    if inv_temp == 1.0:
        rc = load_library().dart_tok_stats(logits.data_ptr(), dt, T, V, ld, target.data_ptr(),
                                           logp.data_ptr(), entropy.data_ptr(), lse.data_ptr(),
                                           _stream_handle(stream, dev))
        name = "dart_tok_stats"
    else:
        rc = load_library().dart_tok_stats_ex(logits.data_ptr(), dt, T, V, ld, target.data_ptr(),
                                              float(inv_temp), logp.data_ptr(),
                                              entropy.data_ptr(), lse.data_ptr(),
                                              _stream_handle(stream, dev))
        name = "dart_tok_stats_ex"
    if rc != DART_OK:
        raise DartError(name, rc)
    return logp, entropy, lse


def dart_step_select(entropy, step_offsets, rho, step_entropy=None, step_mask=None,
                     n_kept_steps=None, stream=None):
    """Per-step mean entropy (float32 [S]), kept-step mask (uint8 [S]) and the
    kept count (int32 [1])."""
    torch = _torch()
    dev = entropy.device
    T = entropy.numel()
    S = step_offsets.numel() - 1
    _check_vec("entropy", entropy, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    step_entropy = torch.empty(S, dtype=torch.float32, device=dev) if step_entropy is None else step_entropy
    step_mask = torch.empty(S, dtype=torch.uint8, device=dev) if step_mask is None else step_mask
    n_kept_steps = torch.empty(1, dtype=torch.int32, device=dev) if n_kept_steps is None else n_kept_steps
    _check_vec("step_entropy", step_entropy, torch.float32, S, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    _check_vec("n_kept_steps", n_kept_steps, torch.int32, 1, dev)
    rc = load_library().dart_step_select(entropy.data_ptr(), T, step_offsets.data_ptr(), S,
                                         float(rho), step_entropy.data_ptr(), step_mask.data_ptr(),
                                         n_kept_steps.data_ptr(), _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_step_select", rc)
    return step_entropy, step_mask, n_kept_steps


def dart_tis_loss_fwd_bwd(logits, target, logp, lse, logp_old, logp_rollout, adv, step_offsets,
                          step_mask, eps_low, eps_high, C, dlogits=None, loss=None, tok_coef=None,
                          stats=None, with_stats=True, stream=None, workspace="auto"):
    """Loss (float64 [1]), dlogits (dtype and shape of logits; pass ``dlogits=logits``
    for the in-place gradient), per-token coefficient (float32 [T]) and stats
    (float32 [4]: clip fraction, mean TIS weight, capped fraction, N).
    ``workspace``: "auto" (allocated here), None (one-workgroup loss, no
    workspace) or a uint8 device tensor of dart_tis_loss_workspace_bytes(T)."""
    torch = _torch()
    dt, T, V, ld = _logits_meta(logits)
    dev = logits.device
    S = step_offsets.numel() - 1
    _check_vec("target", target, torch.int32, T, dev)
    for n, v in (("logp", logp), ("lse", lse), ("logp_old", logp_old),
                 ("logp_rollout", logp_rollout), ("adv", adv)):
        _check_vec(n, v, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    if dlogits is None:
        dlogits = torch.empty((T, V), dtype=logits.dtype, device=dev)
    if (dlogits.dtype != logits.dtype or dlogits.dim() != 2 or tuple(dlogits.shape) != (T, V)
            or dlogits.stride(1) != 1 or dlogits.device != dev):
        raise ValueError("dlogits must match logits in dtype and shape, with contiguous rows")
    loss = torch.empty(1, dtype=torch.float64, device=dev) if loss is None else loss
    tok_coef = torch.empty(T, dtype=torch.float32, device=dev) if tok_coef is None else tok_coef
    if stats is None and with_stats:
        stats = torch.empty(4, dtype=torch.float32, device=dev)
    _check_vec("loss", loss, torch.float64, 1, dev)
    _check_vec("tok_coef", tok_coef, torch.float32, T, dev)
    if stats is not None:
        _check_vec("stats", stats, torch.float32, 4, dev)
    ws, ws_bytes, _ws = _workspace(workspace, T, dev, stream)
    rc = load_library().dart_tis_loss_fwd_bwd(
        logits.data_ptr(), dt, T, V, ld, target.data_ptr(), logp.data_ptr(), lse.data_ptr(),
        logp_old.data_ptr(), logp_rollout.data_ptr(), adv.data_ptr(), step_offsets.data_ptr(), S,
        step_mask.data_ptr(), float(eps_low), float(eps_high), float(C), dlogits.data_ptr(),
        dlogits.stride(0), loss.data_ptr(), tok_coef.data_ptr(), _ptr(stats), ws, ws_bytes,
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_tis_loss_fwd_bwd", rc)
    return loss, dlogits, tok_coef, stats


def dart_tis_loss_fwd_bwd_noalloc(logits, target, logp, lse, logp_old, logp_rollout, adv,
                                  step_offsets, step_mask, eps_low, eps_high, C, dlogits=None,
                                  loss=None, tok_coef=None, stats=None, with_stats=True,
                                  stream=None):
    """dart_tis_loss_fwd_bwd with the loss workspace in the library's fixed
    per-GPU scratch array (the C call allocates nothing; outputs not given are
    allocated here by torch). Calls on one GPU that may overlap race."""
    torch = _torch()
    dt, T, V, ld = _logits_meta(logits)
    dev = logits.device
    S = step_offsets.numel() - 1
    _check_vec("target", target, torch.int32, T, dev)
    for n, v in (("logp", logp), ("lse", lse), ("logp_old", logp_old),
                 ("logp_rollout", logp_rollout), ("adv", adv)):
        _check_vec(n, v, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    if dlogits is None:
        dlogits = torch.empty((T, V), dtype=logits.dtype, device=dev)
    if (dlogits.dtype != logits.dtype or dlogits.dim() != 2 or tuple(dlogits.shape) != (T, V)
            or dlogits.stride(1) != 1 or dlogits.device != dev):
        raise ValueError("dlogits must match logits in dtype and shape, with contiguous rows")
    loss = torch.empty(1, dtype=torch.float64, device=dev) if loss is None else loss
    tok_coef = torch.empty(T, dtype=torch.float32, device=dev) if tok_coef is None else tok_coef
    if stats is None and with_stats:
        stats = torch.empty(4, dtype=torch.float32, device=dev)
    _check_vec("loss", loss, torch.float64, 1, dev)
    _check_vec("tok_coef", tok_coef, torch.float32, T, dev)
    if stats is not None:
        _check_vec("stats", stats, torch.float32, 4, dev)
    rc = load_library().dart_tis_loss_fwd_bwd_noalloc(
        logits.data_ptr(), dt, T, V, ld, target.data_ptr(), logp.data_ptr(), lse.data_ptr(),
        logp_old.data_ptr(), logp_rollout.data_ptr(), adv.data_ptr(), step_offsets.data_ptr(), S,
        step_mask.data_ptr(), float(eps_low), float(eps_high), float(C), dlogits.data_ptr(),
        dlogits.stride(0), loss.data_ptr(), tok_coef.data_ptr(), _ptr(stats),
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_tis_loss_fwd_bwd_noalloc", rc)
    return loss, dlogits, tok_coef, stats


def dart_tis_loss_fwd(logp, logp_old, logp_rollout, adv, step_offsets, step_mask, eps_low,
                      eps_high, C, loss=None, tok_coef=None, stats=None, with_stats=True,
                      stream=None, workspace="auto"):
    """Loss (float64 [1]), per-token coefficient (float32 [T]) and stats; the
    logits are not needed. ``workspace`` as for dart_tis_loss_fwd_bwd."""
    torch = _torch()
    dev = logp.device
    T = logp.numel()
    S = step_offsets.numel() - 1
    for n, v in (("logp", logp), ("logp_old", logp_old), ("logp_rollout", logp_rollout),
                 ("adv", adv)):
        _check_vec(n, v, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev) if loss is None else loss
    tok_coef = torch.empty(T, dtype=torch.float32, device=dev) if tok_coef is None else tok_coef
    if stats is None and with_stats:
        stats = torch.empty(4, dtype=torch.float32, device=dev)
    _check_vec("loss", loss, torch.float64, 1, dev)
    _check_vec("tok_coef", tok_coef, torch.float32, T, dev)
    if stats is not None:
        _check_vec("stats", stats, torch.float32, 4, dev)
    ws, ws_bytes, _ws = _workspace(workspace, T, dev, stream)
    rc = load_library().dart_tis_loss_fwd(
        T, logp.data_ptr(), logp_old.data_ptr(), logp_rollout.data_ptr(), adv.data_ptr(),
        step_offsets.data_ptr(), S, step_mask.data_ptr(), float(eps_low), float(eps_high),
        float(C), loss.data_ptr(), tok_coef.data_ptr(), _ptr(stats), ws, ws_bytes,
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_tis_loss_fwd", rc)
    return loss, tok_coef, stats


def dart_select_tis_loss_fwd(entropy, logp, logp_old, logp_rollout, adv, step_offsets, rho,
                             eps_low, eps_high, C, step_entropy=None, step_mask=None,
                             n_kept_steps=None, loss=None, tok_coef=None, stats=None,
                             with_stats=True, stream=None, workspace="auto"):
    """dart_step_select then dart_tis_loss_fwd in one call (one launch up to
    4096 tokens and 8192 steps). Returns (step_entropy, step_mask,
    n_kept_steps, loss, tok_coef, stats). ``workspace`` as for
    dart_tis_loss_fwd_bwd."""
    torch = _torch()
    dev = logp.device
    T = logp.numel()
    S = step_offsets.numel() - 1
    for n, v in (("entropy", entropy), ("logp", logp), ("logp_old", logp_old),
                 ("logp_rollout", logp_rollout), ("adv", adv)):
        _check_vec(n, v, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    step_entropy = torch.empty(S, dtype=torch.float32, device=dev) if step_entropy is None else step_entropy
    step_mask = torch.empty(S, dtype=torch.uint8, device=dev) if step_mask is None else step_mask
    n_kept_steps = torch.empty(1, dtype=torch.int32, device=dev) if n_kept_steps is None else n_kept_steps
    loss = torch.empty(1, dtype=torch.float64, device=dev) if loss is None else loss
    tok_coef = torch.empty(T, dtype=torch.float32, device=dev) if tok_coef is None else tok_coef
    if stats is None and with_stats:
        stats = torch.empty(4, dtype=torch.float32, device=dev)
    _check_vec("step_entropy", step_entropy, torch.float32, S, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    _check_vec("n_kept_steps", n_kept_steps, torch.int32, 1, dev)
    _check_vec("loss", loss, torch.float64, 1, dev)
    _check_vec("tok_coef", tok_coef, torch.float32, T, dev)
    if stats is not None:
        _check_vec("stats", stats, torch.float32, 4, dev)
    ws, ws_bytes, _ws = _workspace(workspace, T, dev, stream)
    rc = load_library().dart_select_tis_loss_fwd(
        T, entropy.data_ptr(), logp.data_ptr(), logp_old.data_ptr(), logp_rollout.data_ptr(),
        adv.data_ptr(), step_offsets.data_ptr(), S, float(rho), float(eps_low), float(eps_high),
        float(C), step_entropy.data_ptr(), step_mask.data_ptr(), n_kept_steps.data_ptr(),
        loss.data_ptr(), tok_coef.data_ptr(), _ptr(stats), ws, ws_bytes,
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_select_tis_loss_fwd", rc)
    return step_entropy, step_mask, n_kept_steps, loss, tok_coef, stats


def dart_tis_loss_fwd_ex(logp, logp_old, logp_rollout, adv, step_offsets, step_mask, eps_low,
                         eps_high, C, logp_ref=None, kl="none", beta=0.0, aggregation="token_mean",
                         ratio="token", loss=None, tok_coef=None, stats=None, with_stats=True,
                         stream=None, workspace="auto"):
    """The loss with the KL term, aggregation and ratio level selectable.
    Returns (loss float64 [1], tok_coef float32 [T], stats float32 [6]).
    ``workspace`` as for dart_tis_loss_fwd_bwd."""
    torch = _torch()
    dev = logp.device
    T = logp.numel()
    S = step_offsets.numel() - 1
    for n, v in (("logp", logp), ("logp_old", logp_old), ("logp_rollout", logp_rollout),
                 ("adv", adv)):
        _check_vec(n, v, torch.float32, T, dev)
    if DART_KL[kl] != 0:
        _check_vec("logp_ref", logp_ref, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    _check_vec("step_mask", step_mask, torch.uint8, S, dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev) if loss is None else loss
    tok_coef = torch.empty(T, dtype=torch.float32, device=dev) if tok_coef is None else tok_coef
    if stats is None and with_stats:
        stats = torch.empty(6, dtype=torch.float32, device=dev)
    _check_vec("loss", loss, torch.float64, 1, dev)
    _check_vec("tok_coef", tok_coef, torch.float32, T, dev)
    if stats is not None:
        _check_vec("stats", stats, torch.float32, 6, dev)
    cfg = dart_loss_config_t(float(eps_low), float(eps_high), float(C), DART_KL[kl], float(beta),
                             DART_AGG[aggregation], DART_RATIO[ratio])
    ws, ws_bytes, _ws = _workspace(workspace, T, dev, stream)
    rc = load_library().dart_tis_loss_fwd_ex(
        T, logp.data_ptr(), logp_old.data_ptr(), logp_rollout.data_ptr(),
        None if DART_KL[kl] == 0 else logp_ref.data_ptr(), adv.data_ptr(),
        step_offsets.data_ptr(), S, step_mask.data_ptr(), ctypes.byref(cfg), loss.data_ptr(),
        tok_coef.data_ptr(), _ptr(stats), ws, ws_bytes, _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_tis_loss_fwd_ex", rc)
    return loss, tok_coef, stats


def dart_tis_grad(logits, target, logp, lse, tok_coef, dlogits=None, stream=None, inv_temp=1.0,
                  skip_zero_rows=False):
    """dlogits = inv_temp * tok_coef * (onehot(target) - softmax(inv_temp * logits)),
    dtype of logits; ``skip_zero_rows`` writes rows with a zero coefficient
    without reading them."""
    torch = _torch()
    dt, T, V, ld = _logits_meta(logits)
    dev = logits.device
    _check_vec("target", target, torch.int32, T, dev)
    for n, v in (("logp", logp), ("lse", lse), ("tok_coef", tok_coef)):
        _check_vec(n, v, torch.float32, T, dev)
    if dlogits is None:
        dlogits = torch.empty((T, V), dtype=logits.dtype, device=dev)
    if (dlogits.dtype != logits.dtype or dlogits.dim() != 2 or tuple(dlogits.shape) != (T, V)
            or dlogits.stride(1) != 1 or dlogits.device != dev):
        raise ValueError("dlogits must match logits in dtype and shape, with contiguous rows")
    if inv_temp == 1.0 and not skip_zero_rows:
        rc = load_library().dart_tis_grad(
            logits.data_ptr(), dt, T, V, ld, target.data_ptr(), logp.data_ptr(), lse.data_ptr(),
            tok_coef.data_ptr(), dlogits.data_ptr(), dlogits.stride(0), _stream_handle(stream, dev))
        name = "dart_tis_grad"
    else:
        rc = load_library().dart_tis_grad_ex(
            logits.data_ptr(), dt, T, V, ld, target.data_ptr(), logp.data_ptr(), lse.data_ptr(),
            tok_coef.data_ptr(), float(inv_temp),
            DART_GRAD_SKIP_ZERO_ROWS if skip_zero_rows else 0, dlogits.data_ptr(),
            dlogits.stride(0), _stream_handle(stream, dev))
        name = "dart_tis_grad_ex"
    if rc != DART_OK:
        raise DartError(name, rc)
    return dlogits


def dart_grpo_advantage(reward, traj_step_offsets, group_traj_offsets, step_offsets, T=None,
                        adv=None, group_mean=None, group_std=None, stream=None):
    """Step-wise GRPO advantage per token (float32 [T]) and per-group mean/std."""
    torch = _torch()
    dev = reward.device
    n_traj = reward.numel()
    G = group_traj_offsets.numel() - 1
    S = step_offsets.numel() - 1
    _check_vec("reward", reward, torch.float32, n_traj, dev)
    _check_vec("traj_step_offsets", traj_step_offsets, torch.int32, n_traj + 1, dev)
    _check_vec("group_traj_offsets", group_traj_offsets, torch.int32, G + 1, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    if T is None:
        T = int(step_offsets[-1].item())
    adv = torch.empty(T, dtype=torch.float32, device=dev) if adv is None else adv
    group_mean = torch.empty(G, dtype=torch.float32, device=dev) if group_mean is None else group_mean
    group_std = torch.empty(G, dtype=torch.float32, device=dev) if group_std is None else group_std
    _check_vec("adv", adv, torch.float32, T, dev)
    rc = load_library().dart_grpo_advantage(
        reward.data_ptr(), n_traj, traj_step_offsets.data_ptr(), group_traj_offsets.data_ptr(), G,
        step_offsets.data_ptr(), S, T, adv.data_ptr(), _ptr(group_mean), _ptr(group_std),
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_grpo_advantage", rc)
    return adv, group_mean, group_std


def dart_step_select_groups(entropy, step_offsets, group_step_offsets, rho, step_entropy=None,
                            step_mask=None, n_kept_steps=None, stream=None):
    """Per-step entropy, mask and kept count per group (top ceil(rho S_g) of each group)."""
    torch = _torch()
    dev = entropy.device
    T = entropy.numel()
    S = step_offsets.numel() - 1
    G = group_step_offsets.numel() - 1
    _check_vec("entropy", entropy, torch.float32, T, dev)
    _check_vec("step_offsets", step_offsets, torch.int32, S + 1, dev)
    _check_vec("group_step_offsets", group_step_offsets, torch.int32, G + 1, dev)
    step_entropy = torch.empty(S, dtype=torch.float32, device=dev) if step_entropy is None else step_entropy
    step_mask = torch.empty(S, dtype=torch.uint8, device=dev) if step_mask is None else step_mask
    n_kept_steps = torch.empty(G, dtype=torch.int32, device=dev) if n_kept_steps is None else n_kept_steps
    rc = load_library().dart_step_select_groups(
        entropy.data_ptr(), T, step_offsets.data_ptr(), S, group_step_offsets.data_ptr(), G,
        float(rho), step_entropy.data_ptr(), step_mask.data_ptr(), n_kept_steps.data_ptr(),
        _stream_handle(stream, dev))
    if rc != DART_OK:
        raise DartError("dart_step_select_groups", rc)
    return step_entropy, step_mask, n_kept_steps


def dart_lmhead_stats_workspace_bytes(T: int, V: int) -> int:
    return int(load_library().dart_lmhead_stats_workspace_bytes(int(T), int(V)))


def _matrix_bf16(name, t, device=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or t.dtype != torch.bfloat16 or t.dim() != 2:
        raise TypeError(f"{name} must be a 2-D bfloat16 tensor")
    if t.stride(1) != 1 or t.stride(0) % 8 or t.data_ptr() % 16 or not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU with contiguous rows, a row stride that is a "
                         "multiple of 8 and a 16-byte aligned base")
    if device is not None and t.device != device:
        raise ValueError(f"{name} must be on {device}")


def dart_lmhead_tok_stats(hidden, weight, target, logp=None, entropy=None, lse=None,
                          workspace="auto", stream=None):
    """(logp, entropy, lse) float32 [T] of softmax(hidden @ weight^T) without
    materialising the logits: hidden [T, d] and weight [V, d] bfloat16 (d a
    multiple of 8). ``workspace``: "auto" (allocated here) or a uint8 device
    tensor of dart_lmhead_stats_workspace_bytes(T, V) bytes."""
    return _lmhead_tok_stats(None, hidden, weight, target, logp, entropy, lse, workspace, stream)


def dart_lmhead_tok_stats_ex(hidden, weight, target, inv_temp, logp=None, entropy=None,
                             lse=None, workspace="auto", stream=None):
    """dart_lmhead_tok_stats of softmax(inv_temp * hidden @ weight^T)."""
    return _lmhead_tok_stats(float(inv_temp), hidden, weight, target, logp, entropy, lse,
                             workspace, stream)


def _lmhead_tok_stats(inv_temp, hidden, weight, target, logp, entropy, lse, workspace, stream):
    torch = _torch()
    _matrix_bf16("hidden", hidden)
    dev = hidden.device
    _matrix_bf16("weight", weight, dev)
    T, d = hidden.shape
    V = weight.shape[0]
    if weight.shape[1] != d:
        raise ValueError("hidden and weight must have the same inner size d")
    _check_vec("target", target, torch.int32, T, dev)
    logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
    entropy = torch.empty(T, dtype=torch.float32, device=dev) if entropy is None else entropy
    lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
    for n, v in (("logp", logp), ("entropy", entropy), ("lse", lse)):
        _check_vec(n, v, torch.float32, T, dev)
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError('workspace must be "auto" or a uint8 device tensor')
        workspace = torch.empty(dart_lmhead_stats_workspace_bytes(T, V), dtype=torch.uint8,
                                device=dev)
        if isinstance(stream, torch.cuda.Stream):
            workspace.record_stream(stream)
    if (not isinstance(workspace, torch.Tensor) or workspace.dtype != torch.uint8
            or workspace.device != dev or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor on the device of the inputs")
    args = [hidden.data_ptr(), T, d, hidden.stride(0), weight.data_ptr(), V, weight.stride(0),
            target.data_ptr()]
    name = "dart_lmhead_tok_stats"
    if inv_temp is not None:
        args.append(inv_temp)
        name += "_ex"
    args += [logp.data_ptr(), entropy.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
             workspace.numel(), _stream_handle(stream, dev)]
    rc = getattr(load_library(), name)(*args)
    if rc != DART_OK:
        raise DartError(name, rc)
    return logp, entropy, lse


def dart_lmhead_backward_workspace_bytes(chunk_rows: int, V: int) -> int:
    return int(load_library().dart_lmhead_backward_workspace_bytes(int(chunk_rows), int(V)))


def dart_lmhead_backward_ex_workspace_bytes(T: int, d: int, V: int, chunk_rows: int,
                                            chunk_cols: int, flags: int) -> int:
    return int(load_library().dart_lmhead_backward_ex_workspace_bytes(
        int(T), int(d), int(V), int(chunk_rows), int(chunk_cols), int(flags)))


def _lmhead_common(hidden, weight, target, lse, logp, tok_coef):
    torch = _torch()
    _matrix_bf16("hidden", hidden)
    dev = hidden.device
    _matrix_bf16("weight", weight, dev)
    T, d = hidden.shape
    if weight.shape[1] != d:
        raise ValueError("hidden and weight must have the same inner size d")
    _check_vec("target", target, torch.int32, T, dev)
    for n, v in (("lse", lse), ("logp", logp), ("tok_coef", tok_coef)):
        _check_vec(n, v, torch.float32, T, dev)
    return dev, T, d, weight.shape[0]


def dart_lmhead_dlogits(hidden, weight, target, lse, logp, tok_coef, dlogits=None, stream=None,
                        inv_temp=None):
    """bfloat16 [T, V] dlogits = tok_coef (onehot - softmax(hidden @ weight^T)), the
    logits recomputed on the matrix cores; lse and logp from dart_lmhead_tok_stats.
    With inv_temp (dart_lmhead_dlogits_ex): inv_temp tok_coef (onehot -
    softmax(inv_temp hidden @ weight^T)), lse and logp from dart_lmhead_tok_stats_ex."""
    torch = _torch()
    dev, T, d, V = _lmhead_common(hidden, weight, target, lse, logp, tok_coef)
    if dlogits is None:
        dlogits = torch.empty((T, V), dtype=torch.bfloat16, device=dev)
    _matrix_bf16("dlogits", dlogits, dev)
    if tuple(dlogits.shape) != (T, V):
        raise ValueError(f"dlogits must have shape ({T}, {V})")
    args = [hidden.data_ptr(), T, d, hidden.stride(0), weight.data_ptr(), V, weight.stride(0),
            target.data_ptr(), lse.data_ptr(), logp.data_ptr(), tok_coef.data_ptr()]
    name = "dart_lmhead_dlogits"
    if inv_temp is not None:
        args.append(float(inv_temp))
        name += "_ex"
    args += [dlogits.data_ptr(), dlogits.stride(0), _stream_handle(stream, dev)]
    rc = getattr(load_library(), name)(*args)
    if rc != DART_OK:
        raise DartError(name, rc)
    return dlogits


def _lmhead_backward(name, flags, hidden, weight, target, lse, logp, tok_coef, chunk_rows,
                     chunk_cols, dhidden, dweight, workspace, stream, inv_temp=1.0):
    torch = _torch()
    dev, T, d, V = _lmhead_common(hidden, weight, target, lse, logp, tok_coef)
    f = 0 if flags is None else int(flags)
    chunk_rows = max(1, min(int(chunk_rows), T))
    chunk_cols = max(1, min(int(chunk_cols), V))
    gdt = torch.bfloat16 if f & DART_LMHEAD_BF16_GRADS else torch.float32
    dhidden = torch.empty((T, d), dtype=gdt, device=dev) if dhidden is None else dhidden
    dweight = torch.empty((V, d), dtype=gdt, device=dev) if dweight is None else dweight
    for n, m, shape in (("dhidden", dhidden, (T, d)), ("dweight", dweight, (V, d))):
        if (not isinstance(m, torch.Tensor) or m.dtype != gdt or m.device != dev
                or tuple(m.shape) != shape or m.stride(1) != 1):
            raise ValueError(f"{n} must be a {gdt} {shape} tensor on {dev} with contiguous rows")
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError('workspace must be "auto" or a uint8 device tensor')
        nbytes = (dart_lmhead_backward_workspace_bytes(chunk_rows, V) if flags is None else
                  dart_lmhead_backward_ex_workspace_bytes(T, d, V, chunk_rows, chunk_cols, f))
        if nbytes == 0:
            raise ValueError(f"{name}: bad sizes or flags")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        if isinstance(stream, torch.cuda.Stream):
            workspace.record_stream(stream)
    if (not isinstance(workspace, torch.Tensor) or workspace.dtype != torch.uint8
            or workspace.device != dev or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor on the device of the inputs")
    args = [hidden.data_ptr(), T, d, hidden.stride(0), weight.data_ptr(), V, weight.stride(0),
            target.data_ptr(), lse.data_ptr(), logp.data_ptr(), tok_coef.data_ptr()]
    if flags is not None:
        args.append(float(inv_temp))
    args += [dhidden.data_ptr(), dhidden.stride(0), dweight.data_ptr(), dweight.stride(0),
             chunk_rows]
    if flags is not None:
        args += [chunk_cols, f]
    args += [workspace.data_ptr(), workspace.numel(), _stream_handle(stream, dev)]
    rc = getattr(load_library(), name)(*args)
    if rc != DART_OK:
        raise DartError(name, rc)
    return dhidden, dweight


def dart_lmhead_backward(hidden, weight, target, lse, logp, tok_coef, chunk_rows=1024,
                         dhidden=None, dweight=None, workspace="auto", stream=None):
    """(dhidden float32 [T, d], dweight float32 [V, d]) of the loss through the LM
    head, dlogits formed chunk_rows rows at a time in ``workspace`` ("auto" or a
    uint8 device tensor of dart_lmhead_backward_workspace_bytes(min(chunk_rows, T), V)
    bytes)."""
    return _lmhead_backward("dart_lmhead_backward", None, hidden, weight, target, lse, logp,
                            tok_coef, chunk_rows, weight.shape[0], dhidden, dweight, workspace,
                            stream)


def dart_lmhead_backward_ex(hidden, weight, target, lse, logp, tok_coef, chunk_rows=None,
                            chunk_cols=None, flags=0, dhidden=None, dweight=None,
                            workspace="auto", stream=None, inv_temp=1.0):
    """dart_lmhead_backward in blocks of chunk_rows rows x chunk_cols vocabulary
    entries (both None: lmhead_backward_plan's block), at inverse temperature
    inv_temp (lse and logp from dart_lmhead_tok_stats_ex at the same value),
    with flags (bitwise or):
    DART_LMHEAD_BF16_GRADS: dhidden and dweight in bfloat16;
    DART_LMHEAD_SKIP_ZERO_ROWS: the GEMMs over the rows with tok_coef != 0 only
    (the call synchronises the stream once).
    ``workspace`` is "auto" or a uint8 device tensor of
    dart_lmhead_backward_ex_workspace_bytes(T, d, V, chunk_rows, chunk_cols, flags)
    bytes."""
    if chunk_rows is None and chunk_cols is None:
        chunk_rows, chunk_cols = lmhead_backward_plan(hidden.shape[0], weight.shape[0])
    elif chunk_rows is None or chunk_cols is None:
        raise ValueError("give both chunk_rows and chunk_cols, or neither")
    return _lmhead_backward("dart_lmhead_backward_ex", int(flags), hidden, weight, target, lse,
                            logp, tok_coef, chunk_rows, chunk_cols, dhidden, dweight, workspace,
                            stream, inv_temp)


def lmhead_backward_plan(T: int, V: int, budget_bytes: int = 512 << 20):
    """(chunk_rows, chunk_cols) for dart_lmhead_backward_ex: the block whose bf16
    dlogits fit budget_bytes and that rewrites the summed outputs least. Each of
    the ceil(T / rows) row blocks rewrites the [V, d] dweight and each of the
    ceil(V / cols) vocabulary blocks the [T, d] dhidden, so the cost is
    ceil(T / rows) V + ceil(V / cols) T; blocks are whole 256-wide tiles (or all
    of T, V). All rows when T << V, square blocks when T ~ V."""
    T, V = int(T), int(V)
    elems = max(budget_bytes // 2, 256 * 256)
    best = None
    for rows in sorted({T} | set(range(256, T, 256))):
        cols = V if rows * V <= elems else (elems // rows) // 256 * 256
        if cols < 256:
            continue
        cost = -(-T // rows) * V + -(-V // cols) * T
        if best is None or cost < best[0]:
            best = (cost, rows, cols)
    if best is None:
        return min(T, 256), min(V, 256)
    return best[1], best[2]


def policy_update(logits, target, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                  eps_high, C, dlogits=None, stream=None):
    """tok_stats -> select_tis_loss_fwd -> tis_grad on one stream. Returns a dict
    of device tensors (nothing is synchronised)."""
    logp, ent, lse = dart_tok_stats(logits, target, stream=stream)
    step_ent, mask, n_kept, loss, coef, stats = dart_select_tis_loss_fwd(
        ent, logp, logp_old, logp_rollout, adv, step_offsets, rho, eps_low, eps_high, C,
        stream=stream)
    dz = dart_tis_grad(logits, target, logp, lse, coef, dlogits, stream=stream)
    return dict(logp=logp, entropy=ent, lse=lse, step_entropy=step_ent, step_mask=mask,
                n_kept_steps=n_kept, loss=loss, dlogits=dz, tok_coef=coef, stats=stats)
