"""Thin ctypes binding of liblocal.so (argument marshalling only).

Every function here checks and marshals torch tensors to the C ABI declared in
include/local.h and enqueues the library's HIP kernels on the current torch
stream; `KVManager` marshals numpy arrays to the host-side KV manager of
include/local_kv.h. No computation happens in Python and there is no
fallback: if the built library is missing or fails to load, every call
raises.

torch is imported before the library is loaded so that the library binds to
the HIP runtime torch already loaded (both use the soname libamdhip64.so.7),
which lets it run on torch's streams and memory.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblocal.so")
BLOCK_SIZE = 16

EXPORTS = ("local_last_error", "local_version", "local_lora_linear",
           "local_lora_linear_grouped", "local_paged_attn_decode", "local_paged_attn_prefill",
           "local_block_version_check", "local_lora_grad", "local_lora_grad_input",
           "local_lora_grad_grouped", "local_paged_attn_decode_noalloc",
           "local_paged_attn_decode_checked", "local_kv_pool_import", "local_kv_pool_export",
           # host-side KV manager (local_kv.h)
           "local_kvm_default_params", "local_kvm_create", "local_kvm_destroy",
           "local_kvm_tags", "local_kvm_set_committed", "local_kvm_stage", "local_kvm_publish",
           "local_kvm_discard_staged", "local_kvm_versions", "local_kvm_alloc",
           "local_kvm_release", "local_kvm_pin", "local_kvm_unpin", "local_kvm_lookup",
           "local_kvm_insert",
           "local_kvm_plan_stale_prefill", "local_kvm_path", "local_kvm_evict",
           "local_kvm_scores", "local_kvm_stats",
           # host-side cooperative scheduler (local_sched.h)
           "local_sched_default_params", "local_sched_create", "local_sched_destroy",
           "local_sched_submit", "local_sched_cancel", "local_sched_next",
           "local_sched_should_yield", "local_sched_complete", "local_sched_yield",
           "local_sched_estimates", "local_sched_prefill_estimate", "local_sched_stats")

_STATUS = {0: "LOCAL_OK", 1: "LOCAL_ERR_NULL", 2: "LOCAL_ERR_SHAPE",
           3: "LOCAL_ERR_UNSUPPORTED", 4: "LOCAL_ERR_WORKSPACE", 5: "LOCAL_ERR_HIP"}


class LocalError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (_STATUS.get(status, str(status)), message))
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load liblocal.so and declare its signatures. Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(
            "liblocal.so is not built (%s); run `python -m paper_2608_15241_amd.build`" % path)
    lib = ctypes.CDLL(path)
    P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    SZ = ctypes.POINTER(ctypes.c_size_t)
    lib.local_last_error.restype = ctypes.c_char_p
    lib.local_last_error.argtypes = []
    lib.local_version.restype = i32
    lib.local_version.argtypes = []
    lib.local_lora_linear.restype = ctypes.c_int
    lib.local_lora_linear.argtypes = [P, i64, i64, P, i64, P, P, i32, i32, P, P, P, P, P,
                                      P, SZ, P]
    lib.local_lora_linear_grouped.restype = ctypes.c_int
    lib.local_lora_linear_grouped.argtypes = [P, i64, i64, i32, P, P, P, P, i32, i32, P, P, P,
                                              P, P, SZ, P]
    lib.local_paged_attn_decode.restype = ctypes.c_int
    lib.local_paged_attn_decode.argtypes = [P, i32, i32, i32, i32, P, P, P, P, i64, i32, P,
                                            i32, P, P, P, f32, P, P, P, SZ, P]
    lib.local_paged_attn_decode_checked.restype = ctypes.c_int
    lib.local_paged_attn_decode_checked.argtypes = [P, i32, i32, i32, i32, P, P, P, P, i64,
                                                    i32, P, i32, P, P, P, f32, P, P, P, i64,
                                                    P, P, P, SZ, P]
    lib.local_paged_attn_decode_noalloc.restype = ctypes.c_int
    lib.local_paged_attn_decode_noalloc.argtypes = [P, i32, i32, i32, i32, P, P, P, P, i64,
                                                    i32, P, i32, P, P, P, f32, P, P, P]
    lib.local_paged_attn_prefill.restype = ctypes.c_int
    lib.local_paged_attn_prefill.argtypes = [P, P, i32, i64, i32, i32, i32, P, P, P, P, i64,
                                             i32, P, i32, P, P, P, f32, P, P, P, SZ, P]
    lib.local_block_version_check.restype = ctypes.c_int
    lib.local_block_version_check.argtypes = [P, i32, i32, P, i32, P, i64, P, P, i64, P, P,
                                              P, SZ, P]
    lib.local_lora_grad.restype = ctypes.c_int
    lib.local_lora_grad.argtypes = [P, i64, i64, P, i64, P, P, i32, i32, P, P, P, P, P, P, SZ,
                                    P]
    lib.local_lora_grad_grouped.restype = ctypes.c_int
    lib.local_lora_grad_grouped.argtypes = [P, i64, i64, i32, P, P, P, P, i32, i32, P, P, P,
                                            P, P, P, SZ, P]
    lib.local_lora_grad_input.restype = ctypes.c_int
    lib.local_lora_grad_input.argtypes = [P, i64, i64, P, i64, P, P, i32, i32, P, P, P, P, P,
                                          SZ, P]
    for name in ("local_kv_pool_import", "local_kv_pool_export"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [P, P, i64, i32, i32, i32, P, P, P]
    _declare_kvm(lib)
    _declare_sched(lib)
    _lib = lib
    return lib


class KvmParams(ctypes.Structure):
    """local_kvm_params_t (local_kv.h)."""
    _fields_ = [(n, ctypes.c_double) for n in (
        "lambda_p", "lambda_a", "beta", "chi", "eta", "zeta", "eps", "alpha_l", "l_max",
        "c_tok", "c_ctx", "block_bytes")]


def _declare_kvm(lib):
    P, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    I32P, I64P, F64P = (ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
                        ctypes.POINTER(ctypes.c_double))
    sig = {
        "local_kvm_default_params": (None, [ctypes.POINTER(KvmParams)]),
        "local_kvm_create": (P, [i32, ctypes.POINTER(KvmParams)]),
        "local_kvm_destroy": (None, [P]),
        "local_kvm_tags": (I32P, [P]),
        "local_kvm_set_committed": (ctypes.c_int, [P, i32, i32]),
        "local_kvm_stage": (ctypes.c_int, [P, i32, i32]),
        "local_kvm_publish": (ctypes.c_int, [P, i32, I32P]),
        "local_kvm_discard_staged": (ctypes.c_int, [P, i32, I32P]),
        "local_kvm_versions": (ctypes.c_int, [P, i32, I32P, I32P]),
        "local_kvm_alloc": (ctypes.c_int, [P, i32, i32, I32P]),
        "local_kvm_release": (ctypes.c_int, [P, I32P, i32]),
        "local_kvm_pin": (ctypes.c_int, [P, I32P, i32]),
        "local_kvm_unpin": (ctypes.c_int, [P, I32P, i32]),
        "local_kvm_lookup": (ctypes.c_int, [P, i32, i32, i32, I32P, i64, f64, f64, f64, I32P,
                                            i32, I32P]),
        "local_kvm_insert": (ctypes.c_int, [P, i32, i32, i32, I32P, i64, i32, I32P, i32,
                                            I32P]),
        "local_kvm_plan_stale_prefill": (ctypes.c_int, [P, i32, i32, I32P, I32P, I32P, I32P]),
        "local_kvm_path": (ctypes.c_int, [P, i32, I32P, I32P, i64, I64P]),
        "local_kvm_evict": (ctypes.c_int, [P, i32, I32P, i32, I32P]),
        "local_kvm_scores": (ctypes.c_int, [P, i32, i32, i32, F64P, F64P, F64P, F64P]),
        "local_kvm_stats": (ctypes.c_int, [P, I32P, I32P, I32P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args


class SchedParams(ctypes.Structure):
    """local_sched_params_t (local_sched.h)."""
    _fields_ = [(n, ctypes.c_double) for n in (
        "alpha_judge", "alpha_train", "alpha_prefill", "reserve", "window", "delta")]


class SchedTask(ctypes.Structure):
    """local_sched_task_t (local_sched.h)."""
    _fields_ = [("cls", ctypes.c_int32), ("priority", ctypes.c_int32),
                ("adapter", ctypes.c_int32), ("version", ctypes.c_int32),
                ("duration", ctypes.c_double), ("mem", ctypes.c_double),
                ("max_nonyield", ctypes.c_double), ("utility", ctypes.c_double),
                ("deadline", ctypes.c_double), ("tokens", ctypes.c_int32),
                ("prefix_len", ctypes.c_int32)]


def _declare_sched(lib):
    P, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    I32P, I64P, F64P = (ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
                        ctypes.POINTER(ctypes.c_double))
    sig = {
        "local_sched_default_params": (None, [ctypes.POINTER(SchedParams)]),
        "local_sched_create": (ctypes.c_int, [ctypes.POINTER(SchedParams),
                                              ctypes.POINTER(ctypes.c_void_p)]),
        "local_sched_destroy": (None, [P]),
        "local_sched_submit": (ctypes.c_int, [P, ctypes.POINTER(SchedTask), I64P]),
        "local_sched_cancel": (ctypes.c_int, [P, i64]),
        "local_sched_next": (ctypes.c_int, [P, f64, f64, i32, I32P, I64P, F64P, F64P]),
        "local_sched_should_yield": (i32, [P]),
        "local_sched_complete": (ctypes.c_int, [P, i64, f64]),
        "local_sched_yield": (ctypes.c_int, [P, i64, i32]),
        "local_sched_estimates": (ctypes.c_int, [P, i32, F64P, F64P, F64P]),
        "local_sched_prefill_estimate": (ctypes.c_int, [P, i32, i32, F64P]),
        "local_sched_stats": (ctypes.c_int, [P, I32P, I32P, I64P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args


def _check(status: int):
    if status != 0:
        raise LocalError(status, _lib.local_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _req(t: torch.Tensor, name: str, dtype, ndim: Optional[int] = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must have %d dims, got %d" % (name, ndim, t.dim()))
    return t


class Workspace:
    """A grow-only device byte buffer reused across calls on one stream."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                   device=self.device or "cuda")
        return self.buf


_default_ws = {}


def _ws_for(device) -> Workspace:
    key = torch.device(device).index
    if key not in _default_ws:
        _default_ws[key] = Workspace(device)
    return _default_ws[key]


class Call:
    """One prepared C-ABI call: arguments marshalled once, replayed cheaply.

    The workspace size is queried once at preparation. Each call enqueues on
    the torch stream current at call time, so a sequence of prepared calls
    can be captured into a HIP graph (torch.cuda.graph) and replayed.
    """

    def __init__(self, fn, args_before_ws, workspace: Optional[Workspace], device,
                 keep=()):
        # The call holds raw device pointers: keep every tensor it points to
        # alive for as long as the call can run (including graph replays).
        self.keep = tuple(t for t in keep if t is not None)
        n = ctypes.c_size_t(0)
        _check(fn(*args_before_ws, None, ctypes.byref(n), _stream()))
        self.ws = (workspace or _ws_for(device)).get(n.value)
        self.ws_bytes = ctypes.c_size_t(self.ws.numel())
        self.fn = fn
        self.args = tuple(args_before_ws) + (_ptr(self.ws), ctypes.byref(self.ws_bytes))
        self.outputs = None

    def __call__(self):
        _check(self.fn(*self.args, _stream()))
        return self.outputs


def prepare_lora_linear(x, W, A=None, B=None, ranks=None, adapter_idx=None, scale=None,
                        residual=None, out=None, workspace: Optional[Workspace] = None) -> Call:
    """Prepared y = residual + x W^T + scale_t (x A_a^T) B_a^T (bf16 in and out)."""
    lib = load_library()
    _req(x, "x", torch.bfloat16, 2)
    _req(W, "W", torch.bfloat16, 2)
    T, K = x.shape
    N = W.shape[0]
    if W.shape[1] != K:
        raise ValueError("W must be [N, K=%d], got %s" % (K, tuple(W.shape)))
    n_ad, r_max = 0, 0
    if A is not None:
        _req(A, "A", torch.bfloat16, 3)
        _req(B, "B", torch.bfloat16, 3)
        n_ad, r_max = A.shape[0], A.shape[1]
        if A.shape[2] != K or tuple(B.shape) != (n_ad, N, r_max):
            raise ValueError("A must be [n_ad, r_max, K] and B [n_ad, N, r_max]")
        _req(adapter_idx, "adapter_idx", torch.int32, 1)
        _req(scale, "scale", torch.float32, 1)
        if adapter_idx.shape[0] != T or scale.shape[0] != T:
            raise ValueError("adapter_idx and scale must have T=%d entries" % T)
        if ranks is not None:
            _req(ranks, "ranks", torch.int32, 1)
            if ranks.shape[0] != n_ad:
                raise ValueError("ranks must have n_adapters entries")
    if residual is not None:
        _req(residual, "residual", torch.bfloat16, 2)
        if tuple(residual.shape) != (T, N):
            raise ValueError("residual must be [T, N]")
    if out is None:
        out = torch.empty((T, N), dtype=torch.bfloat16, device=x.device)
    _req(out, "out", torch.bfloat16, 2)
    if tuple(out.shape) != (T, N):
        raise ValueError("out must be [T, N]")
    args = [_ptr(x), T, K, _ptr(W), N, _ptr(A), _ptr(B), n_ad, r_max, _ptr(ranks),
            _ptr(adapter_idx), _ptr(scale), _ptr(residual), _ptr(out)]
    c = Call(lib.local_lora_linear, args, workspace, x.device,
             keep=(x, W, A, B, ranks, adapter_idx, scale, residual, out))
    c.outputs = out
    return c


def local_lora_linear(*args, **kwargs):
    """y = residual + x W^T + scale_t (x A_a^T) B_a^T per token (bf16 in and out)."""
    return prepare_lora_linear(*args, **kwargs)()


def _adapter_checks(A, B, ranks, adapter_idx, scale, T, K, N):
    _req(A, "A", torch.bfloat16, 3)
    _req(B, "B", torch.bfloat16, 3)
    n_ad, r_max = A.shape[0], A.shape[1]
    if A.shape[2] != K or tuple(B.shape) != (n_ad, N, r_max):
        raise ValueError("A must be [n_ad, r_max, K=%d] and B [n_ad, N=%d, r_max]" % (K, N))
    _req(adapter_idx, "adapter_idx", torch.int32, 1)
    _req(scale, "scale", torch.float32, 1)
    if adapter_idx.shape[0] != T or scale.shape[0] != T:
        raise ValueError("adapter_idx and scale must have T=%d entries" % T)
    if ranks is not None:
        _req(ranks, "ranks", torch.int32, 1)
        if ranks.shape[0] != n_ad:
            raise ValueError("ranks must have n_adapters entries")
    return n_ad, r_max


def prepare_lora_grad(x, dy, A, B, ranks, adapter_idx, scale, dA=None, dB=None,
                      workspace: Optional[Workspace] = None) -> Call:
    """Prepared adapter gradients of the mixed-adapter projection: returns
    (dA [n_ad, r_max, K], dB [n_ad, N, r_max]) in float32."""
    lib = load_library()
    _req(x, "x", torch.bfloat16, 2)
    _req(dy, "dy", torch.bfloat16, 2)
    T, K = x.shape
    N = dy.shape[1]
    if dy.shape[0] != T:
        raise ValueError("dy must be [T=%d, N]" % T)
    n_ad, r_max = _adapter_checks(A, B, ranks, adapter_idx, scale, T, K, N)
    if dA is None:
        dA = torch.empty((n_ad, r_max, K), dtype=torch.float32, device=x.device)
    if dB is None:
        dB = torch.empty((n_ad, N, r_max), dtype=torch.float32, device=x.device)
    _req(dA, "dA", torch.float32, 3)
    _req(dB, "dB", torch.float32, 3)
    if tuple(dA.shape) != (n_ad, r_max, K) or tuple(dB.shape) != (n_ad, N, r_max):
        raise ValueError("dA must be [n_ad, r_max, K] and dB [n_ad, N, r_max]")
    args = [_ptr(x), T, K, _ptr(dy), N, _ptr(A), _ptr(B), n_ad, r_max, _ptr(ranks),
            _ptr(adapter_idx), _ptr(scale), _ptr(dA), _ptr(dB)]
    c = Call(lib.local_lora_grad, args, workspace, x.device,
             keep=(x, dy, A, B, ranks, adapter_idx, scale, dA, dB))
    c.outputs = (dA, dB)
    return c


def local_lora_grad(*args, **kwargs):
    """(dA, dB) of the mixed-adapter projection (see prepare_lora_grad)."""
    return prepare_lora_grad(*args, **kwargs)()


def prepare_lora_grad_grouped(x, dys, As, Bs, ranks, adapter_idx, scale, dAs=None, dBs=None,
                              workspace: Optional[Workspace] = None) -> Call:
    """Prepared adapter gradients of up to 4 projections of one x: returns
    ([dA_g [n_ad, r_max, K]], [dB_g [n_ad, N_g, r_max]]) in float32."""
    lib = load_library()
    _req(x, "x", torch.bfloat16, 2)
    T, K = x.shape
    G = len(dys)
    if not 1 <= G <= 4 or len(As) != G or len(Bs) != G:
        raise ValueError("dys, As and Bs must have the same length, 1..4")
    ranks = list(ranks) if ranks is not None else [None] * G
    Ns = []
    for g in range(G):
        _req(dys[g], "dy", torch.bfloat16, 2)
        if dys[g].shape[0] != T:
            raise ValueError("dy must be [T=%d, N]" % T)
        Ns.append(dys[g].shape[1])
        n_ad, r_max = _adapter_checks(As[g], Bs[g], ranks[g], adapter_idx, scale, T, K, Ns[g])
        if g and (n_ad, r_max) != (As[0].shape[0], As[0].shape[1]):
            raise ValueError("every projection needs the same n_adapters and r_max")
    n_ad, r_max = As[0].shape[0], As[0].shape[1]
    dAs = dAs or [torch.empty((n_ad, r_max, K), dtype=torch.float32, device=x.device)
                  for _ in range(G)]
    dBs = dBs or [torch.empty((n_ad, Ns[g], r_max), dtype=torch.float32, device=x.device)
                  for g in range(G)]
    for g in range(G):
        _req(dAs[g], "dA", torch.float32, 3)
        _req(dBs[g], "dB", torch.float32, 3)
        if tuple(dAs[g].shape) != (n_ad, r_max, K) or tuple(dBs[g].shape) != (n_ad, Ns[g], r_max):
            raise ValueError("dA must be [n_ad, r_max, K] and dB [n_ad, N, r_max]")
    n_arr = (ctypes.c_int64 * G)(*Ns)
    dy_arr, dy_p = _ptr_array(dys)
    a_arr, a_p = _ptr_array(As)
    b_arr, b_p = _ptr_array(Bs)
    r_arr, r_p = _ptr_array(ranks)
    da_arr, da_p = _ptr_array(dAs)
    db_arr, db_p = _ptr_array(dBs)
    args = [_ptr(x), T, K, G, dy_p, ctypes.cast(n_arr, ctypes.c_void_p), a_p, b_p, n_ad, r_max,
            r_p, _ptr(adapter_idx), _ptr(scale), da_p, db_p]
    keep = (x, adapter_idx, scale, n_arr, dy_arr, a_arr, b_arr, r_arr, da_arr, db_arr) + \
        tuple(dys) + tuple(As) + tuple(Bs) + tuple(ranks) + tuple(dAs) + tuple(dBs)
    c = Call(lib.local_lora_grad_grouped, args, workspace, x.device, keep=keep)
    c.outputs = (dAs, dBs)
    return c


def local_lora_grad_grouped(*args, **kwargs):
    """Adapter gradients of up to 4 projections of one x (see prepare_lora_grad_grouped)."""
    return prepare_lora_grad_grouped(*args, **kwargs)()


def prepare_lora_grad_input(dy, Wt, A, B, ranks, adapter_idx, scale, out=None,
                            workspace: Optional[Workspace] = None) -> Call:
    """Prepared dx = dy W + scale_t (dy B_a) A_a (bf16), with the frozen base
    weight given transposed, Wt = W^T [K, N]."""
    lib = load_library()
    _req(dy, "dy", torch.bfloat16, 2)
    _req(Wt, "Wt", torch.bfloat16, 2)
    T, N = dy.shape
    K = Wt.shape[0]
    if Wt.shape[1] != N:
        raise ValueError("Wt must be [K, N=%d], got %s" % (N, tuple(Wt.shape)))
    n_ad, r_max = _adapter_checks(A, B, ranks, adapter_idx, scale, T, K, N)
    if out is None:
        out = torch.empty((T, K), dtype=torch.bfloat16, device=dy.device)
    _req(out, "out", torch.bfloat16, 2)
    if tuple(out.shape) != (T, K):
        raise ValueError("out must be [T, K]")
    args = [_ptr(dy), T, N, _ptr(Wt), K, _ptr(A), _ptr(B), n_ad, r_max, _ptr(ranks),
            _ptr(adapter_idx), _ptr(scale), _ptr(out)]
    c = Call(lib.local_lora_grad_input, args, workspace, dy.device,
             keep=(dy, Wt, A, B, ranks, adapter_idx, scale, out))
    c.outputs = out
    return c


def local_lora_grad_input(*args, **kwargs):
    """dx of the mixed-adapter projection (see prepare_lora_grad_input)."""
    return prepare_lora_grad_input(*args, **kwargs)()


def _ptr_array(ts):
    """A host array of device pointers (NULL for None)."""
    arr = (ctypes.c_void_p * len(ts))(*[t.data_ptr() if t is not None else None for t in ts])
    return arr, ctypes.cast(arr, ctypes.c_void_p)


def prepare_lora_linear_grouped(x, Ws, As=None, Bs=None, ranks=None, adapter_idx=None,
                                scale=None, outs=None,
                                workspace: Optional[Workspace] = None) -> Call:
    """Prepared y_g = x W_g^T + scale_t (x A_g,a^T) B_g,a^T for up to 4 projections g that
    share x and the adapter routing (one adapter set shape for all of them)."""
    lib = load_library()
    _req(x, "x", torch.bfloat16, 2)
    T, K = x.shape
    G = len(Ws)
    if not 1 <= G <= 4:
        raise ValueError("1 to 4 projections, got %d" % G)
    for W in Ws:
        _req(W, "W", torch.bfloat16, 2)
        if W.shape[1] != K:
            raise ValueError("every W must be [N, K=%d], got %s" % (K, tuple(W.shape)))
    Ns = [W.shape[0] for W in Ws]
    n_ad, r_max = 0, 0
    if As is not None:
        if len(As) != G or len(Bs) != G:
            raise ValueError("one A and one B per projection")
        n_ad, r_max = As[0].shape[0], As[0].shape[1]
        for A, B, N in zip(As, Bs, Ns):
            _req(A, "A", torch.bfloat16, 3)
            _req(B, "B", torch.bfloat16, 3)
            if tuple(A.shape) != (n_ad, r_max, K) or tuple(B.shape) != (n_ad, N, r_max):
                raise ValueError("A must be [n_ad, r_max, K] and B [n_ad, N, r_max], with one "
                                 "n_ad and r_max for every projection")
        _req(adapter_idx, "adapter_idx", torch.int32, 1)
        _req(scale, "scale", torch.float32, 1)
        if adapter_idx.shape[0] != T or scale.shape[0] != T:
            raise ValueError("adapter_idx and scale must have T=%d entries" % T)
        if ranks is not None:
            if len(ranks) != G:
                raise ValueError("one ranks tensor (or None) per projection")
            for r in ranks:
                if r is not None:
                    _req(r, "ranks", torch.int32, 1)
                    if r.shape[0] != n_ad:
                        raise ValueError("ranks must have n_adapters entries")
    if outs is None:
        outs = [torch.empty((T, N), dtype=torch.bfloat16, device=x.device) for N in Ns]
    for o, N in zip(outs, Ns):
        _req(o, "out", torch.bfloat16, 2)
        if tuple(o.shape) != (T, N):
            raise ValueError("each out must be [T, N_g]")
    w_arr, w_p = _ptr_array(Ws)
    n_arr = (ctypes.c_int64 * G)(*Ns)
    a_arr, a_p = _ptr_array(As) if As is not None else (None, None)
    b_arr, b_p = _ptr_array(Bs) if Bs is not None else (None, None)
    r_arr, r_p = _ptr_array(ranks) if ranks is not None else (None, None)
    y_arr, y_p = _ptr_array(outs)
    args = [_ptr(x), T, K, G, w_p, ctypes.cast(n_arr, ctypes.c_void_p), a_p, b_p, n_ad, r_max,
            r_p, _ptr(adapter_idx), _ptr(scale), y_p]
    keep = (x, adapter_idx, scale, w_arr, n_arr, a_arr, b_arr, r_arr, y_arr) + tuple(Ws) + \
        tuple(As or ()) + tuple(Bs or ()) + tuple(ranks or ()) + tuple(outs)
    c = Call(lib.local_lora_linear_grouped, args, workspace, x.device, keep=keep)
    c.outputs = tuple(outs)
    return c


def local_lora_linear_grouped(*args, **kwargs):
    """Outputs of up to 4 LoRA projections of one x (see prepare_lora_linear_grouped)."""
    return prepare_lora_linear_grouped(*args, **kwargs)()


def _pool_checks(k_cache, v_cache, Hkv, D):
    _req(k_cache, "k_cache", torch.bfloat16)
    _req(v_cache, "v_cache", torch.bfloat16)
    per_block = Hkv * BLOCK_SIZE * D
    if k_cache.numel() % per_block or k_cache.numel() != v_cache.numel():
        raise ValueError("k_cache/v_cache must hold num_blocks * Hkv * 16 * D elements")
    return k_cache.numel() // per_block


def _meta_checks(block_table, ctx_lens, block_version, req_version, B,
                 num_blocks: Optional[int] = None):
    _req(block_table, "block_table", torch.int32, 2)
    _req(ctx_lens, "ctx_lens", torch.int32, 1)
    _req(block_version, "block_version", torch.int32, 1)
    _req(req_version, "req_version", torch.int32, 1)
    if block_table.shape[0] != B or ctx_lens.shape[0] != B or req_version.shape[0] != B:
        raise ValueError("block_table, ctx_lens and req_version must have B=%d rows" % B)
    if num_blocks is not None and block_version.numel() < num_blocks:
        raise ValueError("block_version must have a tag for each of the pool's %d blocks, "
                         "got %d" % (num_blocks, block_version.numel()))


def _attn_out_checks(out, lse, rows, Hq, D, device):
    """out [rows, Hq, D] bf16 and lse [rows, Hq] float32 (allocated when None)."""
    if out is None:
        out = torch.empty((rows, Hq, D), dtype=torch.bfloat16, device=device)
    if lse is None:
        lse = torch.empty((rows, Hq), dtype=torch.float32, device=device)
    _req(out, "out", torch.bfloat16, 3)
    _req(lse, "lse", torch.float32, 2)
    if tuple(out.shape) != (rows, Hq, D):
        raise ValueError("out must be [%d, %d, %d], got %s" % (rows, Hq, D, tuple(out.shape)))
    if tuple(lse.shape) != (rows, Hq):
        raise ValueError("lse must be [%d, %d], got %s" % (rows, Hq, tuple(lse.shape)))
    return out, lse


def prepare_paged_attn_decode(q, k_cache, v_cache, block_table, ctx_lens, block_version,
                              req_version, sm_scale: float, k_new=None, v_new=None,
                              Hkv: Optional[int] = None, out=None, lse=None,
                              workspace: Optional[Workspace] = None) -> Call:
    """Prepared decode attention; the call returns (out, lse)."""
    lib = load_library()
    _req(q, "q", torch.bfloat16, 3)
    B, Hq, D = q.shape
    if Hkv is None:
        if k_new is None:
            raise ValueError("Hkv is required when k_new is not given")
        Hkv = k_new.shape[1]
    num_blocks = _pool_checks(k_cache, v_cache, Hkv, D)
    _meta_checks(block_table, ctx_lens, block_version, req_version, B, num_blocks)
    if k_new is not None:
        _req(k_new, "k_new", torch.bfloat16, 3)
        _req(v_new, "v_new", torch.bfloat16, 3)
        if tuple(k_new.shape) != (B, Hkv, D) or tuple(v_new.shape) != (B, Hkv, D):
            raise ValueError("k_new/v_new must be [B, Hkv, D]")
    out, lse = _attn_out_checks(out, lse, B, Hq, D, q.device)
    args = [_ptr(q), B, Hq, Hkv, D, _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
            num_blocks, BLOCK_SIZE, _ptr(block_table), block_table.shape[1], _ptr(ctx_lens),
            _ptr(block_version), _ptr(req_version), float(sm_scale), _ptr(out), _ptr(lse)]
    c = Call(lib.local_paged_attn_decode, args, workspace, q.device,
             keep=(q, k_new, v_new, k_cache, v_cache, block_table, ctx_lens, block_version,
                   req_version, out, lse))
    c.outputs = (out, lse)
    return c


def local_paged_attn_decode(*args, **kwargs):
    """One query token per request over its paged, version-masked KV cache.

    q [B, Hq, D]; pools as documented in include/local.h; returns (out, lse).
    """
    return prepare_paged_attn_decode(*args, **kwargs)()


def prepare_paged_attn_decode_checked(q, k_cache, v_cache, block_table, ctx_lens,
                                      block_version, req_version, sm_scale: float, k_new=None,
                                      v_new=None, Hkv: Optional[int] = None, out=None, lse=None,
                                      cap: Optional[int] = None, stale_pairs=None, n_stale=None,
                                      valid_tokens=None,
                                      workspace: Optional[Workspace] = None) -> Call:
    """Prepared decode attention with the version check of the same requests;
    the call returns (out, lse, stale_pairs, n_stale, valid_tokens)."""
    lib = load_library()
    _req(q, "q", torch.bfloat16, 3)
    B, Hq, D = q.shape
    if Hkv is None:
        if k_new is None:
            raise ValueError("Hkv is required when k_new is not given")
        Hkv = k_new.shape[1]
    num_blocks = _pool_checks(k_cache, v_cache, Hkv, D)
    _meta_checks(block_table, ctx_lens, block_version, req_version, B, num_blocks)
    if k_new is not None:
        _req(k_new, "k_new", torch.bfloat16, 3)
        _req(v_new, "v_new", torch.bfloat16, 3)
        if tuple(k_new.shape) != (B, Hkv, D) or tuple(v_new.shape) != (B, Hkv, D):
            raise ValueError("k_new/v_new must be [B, Hkv, D]")
    out, lse = _attn_out_checks(out, lse, B, Hq, D, q.device)
    dev = q.device
    if cap is None:
        cap = block_table.numel()
    if stale_pairs is None:
        stale_pairs = torch.empty((max(cap, 1), 2), dtype=torch.int32, device=dev)
    if n_stale is None:
        n_stale = torch.empty((1,), dtype=torch.int32, device=dev)
    if valid_tokens is None:
        valid_tokens = torch.empty((B,), dtype=torch.int32, device=dev)
    _req(stale_pairs, "stale_pairs", torch.int32, 2)
    _req(n_stale, "n_stale", torch.int32, 1)
    _req(valid_tokens, "valid_tokens", torch.int32, 1)
    if stale_pairs.shape[0] < cap or stale_pairs.shape[1] != 2 or valid_tokens.shape[0] != B:
        raise ValueError("stale_pairs must be [>= cap, 2] and valid_tokens [B]")
    args = [_ptr(q), B, Hq, Hkv, D, _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
            num_blocks, BLOCK_SIZE, _ptr(block_table), block_table.shape[1], _ptr(ctx_lens),
            _ptr(block_version), _ptr(req_version), float(sm_scale), _ptr(out), _ptr(lse),
            _ptr(stale_pairs), cap, _ptr(n_stale), _ptr(valid_tokens)]
    c = Call(lib.local_paged_attn_decode_checked, args, workspace, q.device,
             keep=(q, k_new, v_new, k_cache, v_cache, block_table, ctx_lens, block_version,
                   req_version, out, lse, stale_pairs, n_stale, valid_tokens))
    c.outputs = (out, lse, stale_pairs, n_stale, valid_tokens)
    return c


def local_paged_attn_decode_checked(*args, **kwargs):
    """Decode attention plus the version check of the same requests (see
    include/local.h); returns (out, lse, stale_pairs, n_stale, valid_tokens)."""
    return prepare_paged_attn_decode_checked(*args, **kwargs)()


class NoWorkspaceCall:
    """A prepared C-ABI call of an entry point that takes no workspace."""

    def __init__(self, fn, args, keep=()):
        self.keep = tuple(t for t in keep if t is not None)
        self.fn = fn
        self.args = tuple(args)
        self.outputs = None

    def __call__(self):
        _check(self.fn(*self.args, _stream()))
        return self.outputs


def prepare_paged_attn_decode_noalloc(q, k_cache, v_cache, block_table, ctx_lens,
                                      block_version, req_version, sm_scale: float, k_new=None,
                                      v_new=None, Hkv: Optional[int] = None, out=None,
                                      lse=None) -> NoWorkspaceCall:
    """Prepared decode attention through local_paged_attn_decode_noalloc (no
    workspace: the library's own scratch); the call returns (out, lse)."""
    lib = load_library()
    _req(q, "q", torch.bfloat16, 3)
    B, Hq, D = q.shape
    if Hkv is None:
        if k_new is None:
            raise ValueError("Hkv is required when k_new is not given")
        Hkv = k_new.shape[1]
    num_blocks = _pool_checks(k_cache, v_cache, Hkv, D)
    _meta_checks(block_table, ctx_lens, block_version, req_version, B, num_blocks)
    if k_new is not None:
        _req(k_new, "k_new", torch.bfloat16, 3)
        _req(v_new, "v_new", torch.bfloat16, 3)
        if tuple(k_new.shape) != (B, Hkv, D) or tuple(v_new.shape) != (B, Hkv, D):
            raise ValueError("k_new/v_new must be [B, Hkv, D]")
    out, lse = _attn_out_checks(out, lse, B, Hq, D, q.device)
    args = [_ptr(q), B, Hq, Hkv, D, _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
            num_blocks, BLOCK_SIZE, _ptr(block_table), block_table.shape[1], _ptr(ctx_lens),
            _ptr(block_version), _ptr(req_version), float(sm_scale), _ptr(out), _ptr(lse)]
    c = NoWorkspaceCall(lib.local_paged_attn_decode_noalloc, args,
                        keep=(q, k_new, v_new, k_cache, v_cache, block_table, ctx_lens,
                              block_version, req_version, out, lse))
    c.outputs = (out, lse)
    return c


def local_paged_attn_decode_noalloc(*args, **kwargs):
    """local_paged_attn_decode without a workspace (see include/local.h)."""
    return prepare_paged_attn_decode_noalloc(*args, **kwargs)()


def prepare_paged_attn_prefill(q, q_indptr, k_cache, v_cache, block_table, ctx_lens,
                               block_version, req_version, sm_scale: float, k_new=None,
                               v_new=None, Hkv: Optional[int] = None, out=None, lse=None,
                               workspace: Optional[Workspace] = None) -> Call:
    """Prepared chunked-prefill attention; the call returns (out, lse)."""
    lib = load_library()
    _req(q, "q", torch.bfloat16, 3)
    T, Hq, D = q.shape
    _req(q_indptr, "q_indptr", torch.int32, 1)
    B = q_indptr.shape[0] - 1
    if Hkv is None:
        if k_new is None:
            raise ValueError("Hkv is required when k_new is not given")
        Hkv = k_new.shape[1]
    num_blocks = _pool_checks(k_cache, v_cache, Hkv, D)
    _meta_checks(block_table, ctx_lens, block_version, req_version, B, num_blocks)
    if k_new is not None:
        _req(k_new, "k_new", torch.bfloat16, 3)
        _req(v_new, "v_new", torch.bfloat16, 3)
        if tuple(k_new.shape) != (T, Hkv, D) or tuple(v_new.shape) != (T, Hkv, D):
            raise ValueError("k_new/v_new must be [T, Hkv, D]")
    out, lse = _attn_out_checks(out, lse, T, Hq, D, q.device)
    args = [_ptr(q), _ptr(q_indptr), B, T, Hq, Hkv, D, _ptr(k_new), _ptr(v_new),
            _ptr(k_cache), _ptr(v_cache), num_blocks, BLOCK_SIZE, _ptr(block_table),
            block_table.shape[1], _ptr(ctx_lens), _ptr(block_version), _ptr(req_version),
            float(sm_scale), _ptr(out), _ptr(lse)]
    c = Call(lib.local_paged_attn_prefill, args, workspace, q.device,
             keep=(q, q_indptr, k_new, v_new, k_cache, v_cache, block_table, ctx_lens,
                   block_version, req_version, out, lse))
    c.outputs = (out, lse)
    return c


def local_paged_attn_prefill(*args, **kwargs):
    """Chunked prefill: append each request's chunk, then causal attention.

    q [T, Hq, D], q_indptr [B+1]; returns (out [T, Hq, D], lse [T, Hq]).
    """
    return prepare_paged_attn_prefill(*args, **kwargs)()


def prepare_block_version_check(block_table, ctx_lens, block_version, req_version,
                                cap: Optional[int] = None, stale_pairs=None, n_stale=None,
                                valid_tokens=None, workspace: Optional[Workspace] = None
                                ) -> Call:
    """Prepared version check; the call returns (stale_pairs, n_stale, valid_tokens)."""
    lib = load_library()
    _req(block_table, "block_table", torch.int32, 2)
    B, max_blocks = block_table.shape
    _meta_checks(block_table, ctx_lens, block_version, req_version, B)
    dev = block_table.device
    if cap is None:
        cap = B * max_blocks
    if stale_pairs is None:
        stale_pairs = torch.empty((max(cap, 1), 2), dtype=torch.int32, device=dev)
    if n_stale is None:
        n_stale = torch.empty((1,), dtype=torch.int32, device=dev)
    if valid_tokens is None:
        valid_tokens = torch.empty((B,), dtype=torch.int32, device=dev)
    _req(stale_pairs, "stale_pairs", torch.int32, 2)
    _req(n_stale, "n_stale", torch.int32, 1)
    _req(valid_tokens, "valid_tokens", torch.int32, 1)
    if stale_pairs.shape[0] < cap:
        raise ValueError("stale_pairs must have at least cap rows")
    args = [_ptr(block_table), B, max_blocks, _ptr(ctx_lens), BLOCK_SIZE,
            _ptr(block_version), block_version.numel(), _ptr(req_version), _ptr(stale_pairs),
            cap, _ptr(n_stale), _ptr(valid_tokens)]
    c = Call(lib.local_block_version_check, args, workspace, dev,
             keep=(block_table, ctx_lens, block_version, req_version, stale_pairs, n_stale,
                   valid_tokens))
    c.outputs = (stale_pairs, n_stale, valid_tokens)
    return c


def local_block_version_check(*args, **kwargs
                              ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Returns (stale_pairs [cap, 2], n_stale [1], valid_tokens [B]) on the device.

    Only the first min(n_stale, cap) rows of stale_pairs are written.
    """
    return prepare_block_version_check(*args, **kwargs)()


def _pool_pair(a, b, what):
    _req(a, what[0], torch.bfloat16, 4)
    _req(b, what[1], torch.bfloat16, 4)
    if a.shape != b.shape:
        raise ValueError("%s and %s must have one shape" % what)


def local_kv_pool_import(k_tok, v_tok, k_cache=None, v_cache=None):
    """Token-major pools [num_blocks, Hkv, 16, D] (bf16) -> the library's pool
    layout; returns (k_cache [num_blocks, Hkv, 16*D], v_cache alike)."""
    lib = load_library()
    _pool_pair(k_tok, v_tok, ("k_tok", "v_tok"))
    nb, hkv, bs, D = k_tok.shape
    if k_cache is None:
        k_cache = torch.empty((nb, hkv, bs * D), dtype=torch.bfloat16, device=k_tok.device)
    if v_cache is None:
        v_cache = torch.empty((nb, hkv, bs * D), dtype=torch.bfloat16, device=k_tok.device)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _req(t, n, torch.bfloat16, 3)
        if tuple(t.shape) != (nb, hkv, bs * D):
            raise ValueError("%s must be [num_blocks, Hkv, 16*D]" % n)
    _check(lib.local_kv_pool_import(_ptr(k_tok), _ptr(v_tok), nb, hkv, D, bs, _ptr(k_cache),
                                    _ptr(v_cache), _stream()))
    return k_cache, v_cache


def local_kv_pool_export(k_cache, v_cache, D, k_tok=None, v_tok=None):
    """The library's pools [num_blocks, Hkv, 16*D] (bf16) -> token-major
    [num_blocks, Hkv, 16, D]; returns (k_tok, v_tok)."""
    lib = load_library()
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _req(t, n, torch.bfloat16, 3)
    if k_cache.shape != v_cache.shape or k_cache.shape[2] != BLOCK_SIZE * D:
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16*D]")
    nb, hkv = k_cache.shape[0], k_cache.shape[1]
    if k_tok is None:
        k_tok = torch.empty((nb, hkv, BLOCK_SIZE, D), dtype=torch.bfloat16, device=k_cache.device)
    if v_tok is None:
        v_tok = torch.empty((nb, hkv, BLOCK_SIZE, D), dtype=torch.bfloat16, device=k_cache.device)
    _pool_pair(k_tok, v_tok, ("k_tok", "v_tok"))
    if tuple(k_tok.shape) != (nb, hkv, BLOCK_SIZE, D):
        raise ValueError("k_tok and v_tok must be [num_blocks, Hkv, 16, D]")
    _check(lib.local_kv_pool_export(_ptr(k_cache), _ptr(v_cache), nb, hkv, D, BLOCK_SIZE,
                                    _ptr(k_tok), _ptr(v_tok), _stream()))
    return k_tok, v_tok


# ------------------------------------------------------------ KV manager

def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p32(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


class KVManager:
    """The host-side KV cache manager of local_kv.h (argument marshalling
    only). Methods take the names of the C calls without the prefix."""

    def __init__(self, num_blocks: int, params: Optional[dict] = None):
        lib = load_library()
        p = KvmParams()
        lib.local_kvm_default_params(ctypes.byref(p))
        for k, v in (params or {}).items():
            setattr(p, k, float(v))
        h = lib.local_kvm_create(int(num_blocks), ctypes.byref(p))
        if not h:
            raise LocalError(2, lib.local_last_error().decode())
        self._lib, self._h, self.num_blocks = lib, ctypes.c_void_p(h), int(num_blocks)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.local_kvm_destroy(h)
            self._h = None

    def tags(self) -> np.ndarray:
        """Copy of the version tag of every block (the `block_version` array)."""
        ptr = self._lib.local_kvm_tags(self._h)
        return np.ctypeslib.as_array(ptr, shape=(self.num_blocks,)).copy()

    def set_committed(self, adapter: int, version: int):
        _check(self._lib.local_kvm_set_committed(self._h, adapter, version))

    def stage(self, adapter: int, version: int):
        _check(self._lib.local_kvm_stage(self._h, adapter, version))

    def publish(self, adapter: int) -> int:
        old = ctypes.c_int32()
        _check(self._lib.local_kvm_publish(self._h, adapter, ctypes.byref(old)))
        return old.value

    def discard_staged(self, adapter: int) -> int:
        n = ctypes.c_int32()
        _check(self._lib.local_kvm_discard_staged(self._h, adapter, ctypes.byref(n)))
        return n.value

    def versions(self, adapter: int) -> Tuple[int, int]:
        c, st = ctypes.c_int32(), ctypes.c_int32()
        _check(self._lib.local_kvm_versions(self._h, adapter, ctypes.byref(c), ctypes.byref(st)))
        return c.value, st.value

    def alloc(self, n: int, version: int) -> np.ndarray:
        out = np.zeros(max(n, 0), dtype=np.int32)
        _check(self._lib.local_kvm_alloc(self._h, n, version, _p32(out)))
        return out

    def release(self, blocks):
        b = _i32(blocks)
        _check(self._lib.local_kvm_release(self._h, _p32(b), b.size))

    def pin(self, blocks):
        b = _i32(blocks)
        _check(self._lib.local_kvm_pin(self._h, _p32(b), b.size))

    def unpin(self, blocks):
        b = _i32(blocks)
        _check(self._lib.local_kvm_unpin(self._h, _p32(b), b.size))

    def lookup(self, ns: int, adapter: int, version: int, tokens, d_prefix: float = 0.0,
               s_prefix: float = 0.0, d_adapter: float = 0.0,
               max_blocks: Optional[int] = None) -> np.ndarray:
        t = _i32(tokens)
        mb = t.size // BLOCK_SIZE if max_blocks is None else int(max_blocks)
        out = np.zeros(max(mb, 1), dtype=np.int32)
        n = ctypes.c_int32()
        _check(self._lib.local_kvm_lookup(self._h, ns, adapter, version, _p32(t), t.size,
                                          d_prefix, s_prefix, d_adapter, _p32(out), mb,
                                          ctypes.byref(n)))
        return out[:n.value].copy()

    def insert(self, ns: int, adapter: int, version: int, tokens, blocks,
               first: int = 0) -> np.ndarray:
        t, b = _i32(tokens), _i32(blocks)
        rec = np.zeros(max(b.size, 1), dtype=np.int32)
        _check(self._lib.local_kvm_insert(self._h, ns, adapter, version, _p32(t), t.size,
                                          int(first), _p32(b), b.size, _p32(rec)))
        return rec[:b.size].copy()

    def plan_stale_prefill(self, adapter: int, max_prefixes: int = 8):
        """[(node, covered_blocks, total_blocks)] ranked hottest first."""
        m = max(int(max_prefixes), 1)
        nodes, cov, tot = (np.zeros(m, dtype=np.int32) for _ in range(3))
        n = ctypes.c_int32()
        _check(self._lib.local_kvm_plan_stale_prefill(self._h, adapter, int(max_prefixes),
                                                      _p32(nodes), _p32(cov), _p32(tot),
                                                      ctypes.byref(n)))
        return [(int(nodes[i]), int(cov[i]), int(tot[i])) for i in range(n.value)]

    def path(self, node: int) -> Tuple[int, np.ndarray]:
        """(namespace, tokens of the path from the root to `node`)."""
        ns, n = ctypes.c_int32(), ctypes.c_int64()
        _check(self._lib.local_kvm_path(self._h, node, ctypes.byref(ns), None, 0,
                                        ctypes.byref(n)))
        out = np.zeros(max(n.value, 1), dtype=np.int32)
        _check(self._lib.local_kvm_path(self._h, node, ctypes.byref(ns), _p32(out), n.value,
                                        ctypes.byref(n)))
        return ns.value, out[:n.value].copy()

    def evict(self, n_free: int) -> np.ndarray:
        out = np.zeros(max(self.num_blocks, 1), dtype=np.int32)
        n = ctypes.c_int32()
        _check(self._lib.local_kvm_evict(self._h, n_free, _p32(out), self.num_blocks,
                                         ctypes.byref(n)))
        return out[:n.value].copy()

    def scores(self, node: int, adapter: int, version: int) -> Tuple[float, float, float, float]:
        """(H_P, H_A, H_KV, Pi_keep) at the current clock."""
        v = [ctypes.c_double() for _ in range(4)]
        _check(self._lib.local_kvm_scores(self._h, node, adapter, version,
                                          *[ctypes.byref(x) for x in v]))
        return tuple(x.value for x in v)

    def stats(self) -> Tuple[int, int, int]:
        """(free blocks, recorded blocks, trie nodes)."""
        v = [ctypes.c_int32() for _ in range(3)]
        _check(self._lib.local_kvm_stats(self._h, *[ctypes.byref(x) for x in v]))
        return tuple(x.value for x in v)


class Scheduler:
    """The host-side cooperative scheduler of local_sched.h (argument
    marshalling only). Methods take the names of the C calls without the
    prefix; a task is given as keyword arguments of local_sched_task_t."""

    FOREGROUND, JUDGE, TRAIN, PREFILL = 0, 1, 2, 3
    RUN, BUSY, IDLE, OFFLOAD = 0, 1, 2, 3

    def __init__(self, params: Optional[dict] = None):
        lib = load_library()
        p = SchedParams()
        lib.local_sched_default_params(ctypes.byref(p))
        for k, v in (params or {}).items():
            setattr(p, k, float(v))
        h = ctypes.c_void_p()
        _check(lib.local_sched_create(ctypes.byref(p), ctypes.byref(h)))
        self._lib, self._h = lib, h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.local_sched_destroy(h)
            self._h = None

    def submit(self, cls, priority=0, adapter=0, version=0, duration=-1.0, mem=0.0,
               max_nonyield=0.0, utility=0.0, deadline=-1.0, tokens=0, prefix_len=0) -> int:
        t = SchedTask(int(cls), int(priority), int(adapter), int(version), float(duration),
                      float(mem), float(max_nonyield), float(utility), float(deadline),
                      int(tokens), int(prefix_len))
        i = ctypes.c_int64(-1)
        _check(self._lib.local_sched_submit(self._h, ctypes.byref(t), ctypes.byref(i)))
        return i.value

    def cancel(self, task_id: int):
        _check(self._lib.local_sched_cancel(self._h, int(task_id)))

    def next(self, now: float, mem_free: float, turn_window: bool = False):
        """(decision, task id or -1, duration estimate or -1, deficit bytes)."""
        d, t = ctypes.c_int32(), ctypes.c_int64()
        e, df = ctypes.c_double(), ctypes.c_double()
        _check(self._lib.local_sched_next(self._h, float(now), float(mem_free),
                                          1 if turn_window else 0, ctypes.byref(d),
                                          ctypes.byref(t), ctypes.byref(e), ctypes.byref(df)))
        return d.value, t.value, e.value, df.value

    def should_yield(self) -> bool:
        return bool(self._lib.local_sched_should_yield(self._h))

    def complete(self, task_id: int, seconds: float):
        _check(self._lib.local_sched_complete(self._h, int(task_id), float(seconds)))

    def yield_(self, task_id: int, requeue: bool = True):
        _check(self._lib.local_sched_yield(self._h, int(task_id), 1 if requeue else 0))

    def estimates(self, prefix_len: int = 0):
        """(judge EMA, training EMA, prefill rate of bucket b(prefix_len)); -1 if unset."""
        j, t, r = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        _check(self._lib.local_sched_estimates(self._h, int(prefix_len), ctypes.byref(j),
                                               ctypes.byref(t), ctypes.byref(r)))
        return j.value, t.value, r.value

    def prefill_estimate(self, tokens: int, prefix_len: int) -> float:
        v = ctypes.c_double()
        _check(self._lib.local_sched_prefill_estimate(self._h, int(tokens), int(prefix_len),
                                                      ctypes.byref(v)))
        return v.value

    def stats(self):
        """(queued foreground, queued background, running task id or -1)."""
        f, b, r = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
        _check(self._lib.local_sched_stats(self._h, ctypes.byref(f), ctypes.byref(b),
                                           ctypes.byref(r)))
        return f.value, b.value, r.value
