"""ctypes binding of libbgpo (include/bgpo.h).

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity and passed as raw device pointers together with torch's current
HIP stream.  Every step of the computation runs in the library's HIP kernels;
there is no fallback, and importing this module raises if the library has not
been built (``python -m paper_2510_11683_amd.build``).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbgpo.so")

BGPO_OK = 0
BGPO_ERR_INVALID_ARG = -1
BGPO_ERR_WORKSPACE = -2
BGPO_ERR_HIP = -3
BGPO_ERR_UNSUPPORTED = -4
BGPO_ERR_BUDGET = -5
BGPO_BF16, BGPO_F32 = 0, 1
BGPO_T_IID = 0
BGPO_T_STRATIFIED = 1
BGPO_FLAG_NONFINITE = 1
BGPO_BOUND_PAPER, BGPO_BOUND_TAYLOR, BGPO_BOUND_JENSEN, BGPO_BOUND_EXACT = 0, 1, 2, 3
KERNEL_CLASSES = ("transpose_w", "mask", "gather", "fwd", "ell", "softmax_grad", "dx", "dx_reduce", "dw",
                  "recompute")


class _Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("L", ctypes.c_int32), ("d", ctypes.c_int32),
                ("V", ctypes.c_int32), ("n_t", ctypes.c_int32), ("j_begin", ctypes.c_int32),
                ("j_count", ctypes.c_int32), ("t_mode", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("seq_id_base", ctypes.c_uint32),
                ("bound", ctypes.c_int32), ("sample_stride", ctypes.c_int64),
                ("norm_eps", ctypes.c_float), ("retain_samples", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("vocab_chunk", ctypes.c_int32),
                ("ws_budget", ctypes.c_uint64)]


class _PlanInfo(ctypes.Structure):
    _fields_ = [("samples_per_unit", ctypes.c_int32), ("dw_batch", ctypes.c_int32),
                ("dx_splits", ctypes.c_int32), ("vocab_chunk", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_uint64), ("w_copy", ctypes.c_int32)]


class Timing(ctypes.Structure):
    """Per-kernel-class elapsed milliseconds and launch counts (bgpo_timing)."""
    _fields_ = [("ms", ctypes.c_double * len(KERNEL_CLASSES)),
                ("launches", ctypes.c_int64 * len(KERNEL_CLASSES))]

    def as_dict(self):
        return {k: (self.ms[i], int(self.launches[i])) for i, k in enumerate(KERNEL_CLASSES)}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2510_11683_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.bgpo_version.restype = ctypes.c_int
    lib.bgpo_status_string.restype = ctypes.c_char_p
    lib.bgpo_status_string.argtypes = [ctypes.c_int]
    lib.bgpo_workspace_size.argtypes = [P(_Problem), P(sz)]
    lib.bgpo_workspace_plan.argtypes = [P(_Problem), P(_PlanInfo)]
    lib.bgpo_sample_masks.argtypes = [P(_Problem), vp, i32, vp, vp, vp, vp]
    lib.bgpo_elbo_fwd.argtypes = [P(_Problem), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp, P(Timing)]
    lib.bgpo_elbo_bwd_accumulate.argtypes = [P(_Problem), vp, vp, vp, vp, vp, vp, ctypes.c_double,
                                             vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp, P(Timing)]
    lib.bgpo_elbo_fwd_rmsnorm.argtypes = [P(_Problem), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp,
                                          P(Timing)]
    lib.bgpo_elbo_bwd_accumulate_rmsnorm.argtypes = [P(_Problem), vp, vp, vp, vp, vp, vp, vp,
                                                     ctypes.c_double, vp, vp, vp, vp, vp, vp, vp,
                                                     vp, vp, vp, sz, vp, P(Timing)]
    lib.bgpo_elbo_bwd_accumulate_noalloc.argtypes = [P(_Problem), vp, vp, vp, vp, vp, vp,
                                                     ctypes.c_double, vp, vp, vp, vp, vp, vp, vp,
                                                     vp, vp]
    lib.bgpo_noalloc_scratch_bytes.restype = sz
    lib.bgpo_noalloc_scratch_bytes.argtypes = []
    lib.bgpo_moments_update.argtypes = [vp, vp, vp, ctypes.c_int64, i32, vp]
    lib.bgpo_moments_workspace_size.restype = sz
    lib.bgpo_moments_workspace_size.argtypes = []
    lib.bgpo_moments_summary.argtypes = [vp, vp, vp, ctypes.c_int64, i32, vp, vp, sz, vp]
    lib.bgpo_test_gemm_nt.argtypes = [vp, vp, vp, i32, i32, i32, vp]
    lib.bgpo_test_gemm_split.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp]
    lib.bgpo_test_gemm_tn.argtypes = [vp, vp, vp, i32, i32, i32, vp]
    lib.bgpo_test_mask_scratch_bytes.restype = sz
    lib.bgpo_test_mask_scratch_bytes.argtypes = [P(_Problem)]
    lib.bgpo_test_mask_multiblock.argtypes = [P(_Problem), vp, i32, vp, vp, vp, vp, sz, vp]
    for f in ("bgpo_workspace_size", "bgpo_workspace_plan", "bgpo_sample_masks", "bgpo_elbo_fwd",
              "bgpo_elbo_bwd_accumulate", "bgpo_elbo_bwd_accumulate_noalloc", "bgpo_elbo_fwd_rmsnorm",
              "bgpo_elbo_bwd_accumulate_rmsnorm", "bgpo_moments_update", "bgpo_moments_summary",
              "bgpo_test_gemm_nt", "bgpo_test_gemm_split", "bgpo_test_gemm_tn",
              "bgpo_test_mask_multiblock"):
        getattr(lib, f).restype = ctypes.c_int
    return lib


_lib = _load()


class BgpoError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {_lib.bgpo_status_string(status).decode()} ({status})")
        self.status = status


def _check(status: int, where: str):
    if status != BGPO_OK:
        raise BgpoError(status, where)


@dataclasses.dataclass
class Problem:
    """Mirror of bgpo_problem; j_count None means the rest of [j_begin, n_t)."""
    B: int
    L: int
    d: int
    V: int
    n_t: int
    j_begin: int = 0
    j_count: Optional[int] = None
    seed: int = 0
    seq_id_base: int = 0
    t_mode: int = BGPO_T_IID
    bound: int = BGPO_BOUND_PAPER
    sample_stride: int = 0        # elements between per-sample head inputs / dX; 0 = shared
    norm_eps: float = 1e-6        # final RMSNorm epsilon (the _rmsnorm calls)
    retain_samples: int = 0       # 1: exact objective keeping every sample's state (memory ~ n_t)
    in_dtype: int = BGPO_BF16     # element type of hidden / x and W_head (BGPO_F32: rounded on device)
    vocab_chunk: int = 0          # > 0: recompute backward with vocabulary chunks of this width
    ws_budget: int = 0            # workspace byte budget (0: none); picks the backward's layout

    @property
    def jc(self) -> int:
        return self.n_t - self.j_begin if self.j_count is None else self.j_count

    def c(self) -> _Problem:
        return _Problem(self.B, self.L, self.d, self.V, self.n_t, self.j_begin, self.jc, self.t_mode,
                        self.seed & 0xFFFFFFFFFFFFFFFF, self.seq_id_base & 0xFFFFFFFF, self.bound,
                        self.sample_stride, self.norm_eps, self.retain_samples, self.in_dtype,
                        self.vocab_chunk, self.ws_budget & 0xFFFFFFFFFFFFFFFF)


def _ptr(t: Optional[torch.Tensor], name: str, dtypes=None, shape=None, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)


def _in_types(prob: "Problem"):
    """Accepted dtypes of hidden / x and W_head for the problem's in_dtype."""
    return (torch.float32,) if prob.in_dtype == BGPO_F32 else _BF16


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def bgpo_version() -> int:
    return _lib.bgpo_version()


def bgpo_workspace_size(prob: Problem) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.bgpo_workspace_size(ctypes.byref(prob.c()), ctypes.byref(n)), "bgpo_workspace_size")
    return int(n.value)


def bgpo_workspace_plan(prob: Problem) -> dict:
    """The layout the problem's workspace takes (mode, unit size, chunk, bytes)."""
    info = _PlanInfo()
    _check(_lib.bgpo_workspace_plan(ctypes.byref(prob.c()), ctypes.byref(info)), "bgpo_workspace_plan")
    d = {k: int(getattr(info, k)) for k, _ in _PlanInfo._fields_}
    d["mode"] = "recompute" if d["vocab_chunk"] else "stored"
    return d


def alloc_workspace(prob: Problem, device="cuda") -> torch.Tensor:
    """A caller-owned workspace of bgpo_workspace_size() bytes (256-byte aligned)."""
    return torch.empty(bgpo_workspace_size(prob), dtype=torch.uint8, device=device)


def bgpo_sample_masks(prob: Problem, resp_mask, j: int, idx, n_masked, t_out=None, stream=None):
    B, L = prob.B, prob.L
    _check(_lib.bgpo_sample_masks(ctypes.byref(prob.c()),
                                  _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)), int(j),
                                  _ptr(idx, "idx", (torch.int32,), (B * L,)),
                                  _ptr(n_masked, "n_masked", (torch.int32,), (B,)),
                                  _ptr(t_out, "t_out", (torch.float32,), (B,), allow_none=True),
                                  _stream(stream)), "bgpo_sample_masks")


def bgpo_test_mask_multiblock(prob: Problem, resp_mask, j: int, idx, n_masked, t_out=None,
                              stream=None):
    """Test hook: the multi-block mask passes (any size); allocates their scratch."""
    B, L = prob.B, prob.L
    pc = prob.c()
    scratch = torch.empty(int(_lib.bgpo_test_mask_scratch_bytes(ctypes.byref(pc))) + 256,
                          dtype=torch.uint8, device=resp_mask.device)
    _check(_lib.bgpo_test_mask_multiblock(
        ctypes.byref(pc), _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)), int(j),
        _ptr(idx, "idx", (torch.int32,), (B * L,)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B,)),
        _ptr(t_out, "t_out", (torch.float32,), (B,), allow_none=True),
        _ptr(scratch, "scratch", (torch.uint8,)), scratch.numel(), _stream(stream)),
        "bgpo_test_mask_multiblock")
    return scratch


def _act_shape(prob: Problem):
    """Shape of the head input (and dX): [B, L, d], or [j_count, B, L, d] with a
    sample stride of exactly B*L*d elements (other strides: pass a flat tensor
    through the C ABI directly)."""
    B, L, d = prob.B, prob.L, prob.d
    if prob.sample_stride == 0:
        return (B, L, d)
    if prob.sample_stride != B * L * d:
        raise ValueError("the binding supports sample_stride 0 or B*L*d")
    return (prob.jc, B, L, d)


def bgpo_elbo_fwd(prob: Problem, hidden, W_head, targets, resp_mask, ell, n_masked, t_out,
                  workspace, stream=None, timing: Optional[Timing] = None):
    B, L, d, V, nt = prob.B, prob.L, prob.d, prob.V, prob.n_t
    _check(_lib.bgpo_elbo_fwd(
        ctypes.byref(prob.c()), _ptr(hidden, "hidden", _in_types(prob), _act_shape(prob)),
        _ptr(W_head, "W_head", _in_types(prob), (d, V)), _ptr(targets, "targets", (torch.int32,), (B, L)),
        _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)),
        _ptr(ell, "ell", (torch.float64,), (B, nt)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B, nt)),
        _ptr(t_out, "t_out", (torch.float32,), (B, nt), allow_none=True),
        _ptr(workspace, "workspace", (torch.uint8,)), workspace.numel(), _stream(stream),
        ctypes.byref(timing) if timing is not None else None), "bgpo_elbo_fwd")


def bgpo_elbo_bwd_accumulate(prob: Problem, hidden, W_head, targets, resp_mask, adv, ell_old,
                             loss_scale: float, dX, dW, ell, g, loss, n_masked, t_out,
                             status_flags, workspace, stream=None,
                             timing: Optional[Timing] = None):
    B, L, d, V, nt = prob.B, prob.L, prob.d, prob.V, prob.n_t
    _check(_lib.bgpo_elbo_bwd_accumulate(
        ctypes.byref(prob.c()), _ptr(hidden, "hidden", _in_types(prob), _act_shape(prob)),
        _ptr(W_head, "W_head", _in_types(prob), (d, V)), _ptr(targets, "targets", (torch.int32,), (B, L)),
        _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)),
        _ptr(adv, "adv", (torch.float32,), (B,)),
        _ptr(ell_old, "ell_old", (torch.float64,), (B, nt), allow_none=True),
        float(loss_scale),
        _ptr(dX, "dX", (torch.float32,), _act_shape(prob)), _ptr(dW, "dW", (torch.float32,), (d, V)),
        _ptr(ell, "ell", (torch.float64,), (B, nt)), _ptr(g, "g", (torch.float64,), (B, nt)),
        _ptr(loss, "loss", (torch.float64,), (1,)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B, nt)),
        _ptr(t_out, "t_out", (torch.float32,), (B, nt), allow_none=True),
        _ptr(status_flags, "status_flags", (torch.int32,), (1,), allow_none=True),
        _ptr(workspace, "workspace", (torch.uint8,)), workspace.numel(), _stream(stream),
        ctypes.byref(timing) if timing is not None else None), "bgpo_elbo_bwd_accumulate")


def bgpo_elbo_bwd_accumulate_noalloc(prob: Problem, hidden, W_head, targets, resp_mask, adv,
                                     ell_old, loss_scale: float, dX, dW, ell, g, loss, n_masked,
                                     t_out, status_flags, stream=None):
    """bgpo_elbo_bwd_accumulate on the library's static scratch (no workspace)."""
    B, L, d, V, nt = prob.B, prob.L, prob.d, prob.V, prob.n_t
    _check(_lib.bgpo_elbo_bwd_accumulate_noalloc(
        ctypes.byref(prob.c()), _ptr(hidden, "hidden", _in_types(prob), _act_shape(prob)),
        _ptr(W_head, "W_head", _in_types(prob), (d, V)),
        _ptr(targets, "targets", (torch.int32,), (B, L)),
        _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)),
        _ptr(adv, "adv", (torch.float32,), (B,)),
        _ptr(ell_old, "ell_old", (torch.float64,), (B, nt), allow_none=True),
        float(loss_scale),
        _ptr(dX, "dX", (torch.float32,), _act_shape(prob)), _ptr(dW, "dW", (torch.float32,), (d, V)),
        _ptr(ell, "ell", (torch.float64,), (B, nt)), _ptr(g, "g", (torch.float64,), (B, nt)),
        _ptr(loss, "loss", (torch.float64,), (1,)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B, nt)),
        _ptr(t_out, "t_out", (torch.float32,), (B, nt), allow_none=True),
        _ptr(status_flags, "status_flags", (torch.int32,), (1,), allow_none=True),
        _stream(stream)), "bgpo_elbo_bwd_accumulate_noalloc")


def bgpo_noalloc_scratch_bytes() -> int:
    return int(_lib.bgpo_noalloc_scratch_bytes())


def bgpo_elbo_fwd_rmsnorm(prob: Problem, x, norm_weight, W_head, targets, resp_mask, ell,
                          n_masked, t_out, workspace, stream=None,
                          timing: Optional[Timing] = None):
    B, L, d, V, nt = prob.B, prob.L, prob.d, prob.V, prob.n_t
    _check(_lib.bgpo_elbo_fwd_rmsnorm(
        ctypes.byref(prob.c()), _ptr(x, "x", _in_types(prob), _act_shape(prob)),
        _ptr(norm_weight, "norm_weight", (torch.float32,), (d,)),
        _ptr(W_head, "W_head", _in_types(prob), (d, V)), _ptr(targets, "targets", (torch.int32,), (B, L)),
        _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)),
        _ptr(ell, "ell", (torch.float64,), (B, nt)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B, nt)),
        _ptr(t_out, "t_out", (torch.float32,), (B, nt), allow_none=True),
        _ptr(workspace, "workspace", (torch.uint8,)), workspace.numel(), _stream(stream),
        ctypes.byref(timing) if timing is not None else None), "bgpo_elbo_fwd_rmsnorm")


def bgpo_elbo_bwd_accumulate_rmsnorm(prob: Problem, x, norm_weight, W_head, targets, resp_mask,
                                     adv, ell_old, loss_scale: float, dx, d_norm_weight, dW, ell,
                                     g, loss, n_masked, t_out, status_flags, workspace,
                                     stream=None, timing: Optional[Timing] = None):
    B, L, d, V, nt = prob.B, prob.L, prob.d, prob.V, prob.n_t
    _check(_lib.bgpo_elbo_bwd_accumulate_rmsnorm(
        ctypes.byref(prob.c()), _ptr(x, "x", _in_types(prob), _act_shape(prob)),
        _ptr(norm_weight, "norm_weight", (torch.float32,), (d,)),
        _ptr(W_head, "W_head", _in_types(prob), (d, V)), _ptr(targets, "targets", (torch.int32,), (B, L)),
        _ptr(resp_mask, "resp_mask", (torch.uint8,), (B, L)),
        _ptr(adv, "adv", (torch.float32,), (B,)),
        _ptr(ell_old, "ell_old", (torch.float64,), (B, nt), allow_none=True),
        float(loss_scale),
        _ptr(dx, "dx", (torch.float32,), _act_shape(prob)),
        _ptr(d_norm_weight, "d_norm_weight", (torch.float32,), (d,)),
        _ptr(dW, "dW", (torch.float32,), (d, V)),
        _ptr(ell, "ell", (torch.float64,), (B, nt)), _ptr(g, "g", (torch.float64,), (B, nt)),
        _ptr(loss, "loss", (torch.float64,), (1,)),
        _ptr(n_masked, "n_masked", (torch.int32,), (B, nt)),
        _ptr(t_out, "t_out", (torch.float32,), (B, nt), allow_none=True),
        _ptr(status_flags, "status_flags", (torch.int32,), (1,), allow_none=True),
        _ptr(workspace, "workspace", (torch.uint8,)), workspace.numel(), _stream(stream),
        ctypes.byref(timing) if timing is not None else None), "bgpo_elbo_bwd_accumulate_rmsnorm")


def bgpo_moments_update(g, mean, m2, count: int, stream=None):
    """Fold estimate number `count` (0-based) of a gradient into running moments."""
    n = g.numel()
    _check(_lib.bgpo_moments_update(_ptr(g, "g", (torch.float32,)),
                                    _ptr(mean, "mean", (torch.float32,), tuple(g.shape)),
                                    _ptr(m2, "m2", (torch.float32,), tuple(g.shape)), n, int(count),
                                    _stream(stream)), "bgpo_moments_update")


def moments_workspace(device="cuda") -> torch.Tensor:
    return torch.empty(_lib.bgpo_moments_workspace_size(), dtype=torch.uint8, device=device)


def bgpo_moments_summary(mean, m2, ref, count: int, out, workspace, stream=None):
    """out[0] mean per-element sample std, out[1] mean |mean - ref|, out[2] mean |ref|."""
    _check(_lib.bgpo_moments_summary(_ptr(mean, "mean", (torch.float32,)),
                                     _ptr(m2, "m2", (torch.float32,), tuple(mean.shape)),
                                     _ptr(ref, "ref", (torch.float32,), tuple(mean.shape), allow_none=True),
                                     mean.numel(), int(count),
                                     _ptr(out, "out", (torch.float64,), (3,)),
                                     _ptr(workspace, "workspace", (torch.uint8,)), workspace.numel(),
                                     _stream(stream)), "bgpo_moments_summary")


def bgpo_test_gemm_nt(A, B, C, stream=None):
    """Test hook: C[m, n] = sum_k A[m, k] B[n, k] through the MFMA GEMM core of
    the dX GEMM, in its operand layouts: A K-slab-major [K/64, M, 64]
    (element (m, k) at [k // 64, m, k % 64]), B row-major [N, K]."""
    S, M, _ = A.shape
    N, K = B.shape
    _check(_lib.bgpo_test_gemm_nt(_ptr(A, "A", _BF16, (K // 64, M, 64)), _ptr(B, "B", _BF16, (N, K)),
                                  _ptr(C, "C", (torch.float32,), (M, N)), M, N, K, _stream(stream)),
           "bgpo_test_gemm_nt")


def bgpo_test_gemm_split(A, B, C, n_split: int, stream=None):
    """Test hook: the GEMM core with K in n_split slices, slice s's product in
    C[s] (C float32 [n_split, M, N]); A, B as in bgpo_test_gemm_nt."""
    S, M, _ = A.shape
    N, K = B.shape
    _check(_lib.bgpo_test_gemm_split(_ptr(A, "A", _BF16, (K // 64, M, 64)), _ptr(B, "B", _BF16, (N, K)),
                                     _ptr(C, "C", (torch.float32,), (n_split, M, N)), M, N, K,
                                     int(n_split), _stream(stream)),
           "bgpo_test_gemm_split")


def bgpo_test_gemm_tn(A, B, C, stream=None):
    """Test hook: C[n, m] += sum_k A[m, k] B[n, k] through the dW GEMM's kernel,
    in its operand layouts: A [M/64, K, 64] (element (m, k) at
    [m // 64, k, m % 64]), B K-slab-major [K/64, N, 64] (element (n, k) at
    [k // 64, n, k % 64]), C float32 [N, M]."""
    MS, K, _ = A.shape
    KS, N, _ = B.shape
    M = MS * 64
    _check(_lib.bgpo_test_gemm_tn(_ptr(A, "A", _BF16, (MS, K, 64)), _ptr(B, "B", _BF16, (K // 64, N, 64)),
                                  _ptr(C, "C", (torch.float32,), (N, M)), M, N, K, _stream(stream)),
           "bgpo_test_gemm_tn")


def device_inputs(x: dict, device="cuda") -> dict:
    """numpy inputs from the workload generator -> device tensors of the ABI dtypes."""
    import numpy as np
    out = {
        "hidden": torch.from_numpy(x["hidden"].view(np.int16)).to(device).view(torch.bfloat16),
        "targets": torch.from_numpy(x["targets"].astype(np.int32)).to(device),
        "resp_mask": torch.from_numpy(x["resp_mask"].astype(np.uint8)).to(device),
        "adv": torch.from_numpy(x["adv"].astype(np.float32)).to(device),
    }
    if x.get("W") is not None:
        out["W"] = torch.from_numpy(x["W"].view(np.int16)).to(device).view(torch.bfloat16)
    return out
