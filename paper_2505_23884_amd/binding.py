"""ctypes binding of liblact.so with the names of the C ABI (include/lact.h)."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblact.so")

APPLY_THEN_UPDATE, UPDATE_THEN_APPLY = 0, 1
IO_BF16, IO_FP32 = 0, 1
KCLASS_NAMES = ("fwd", "bwd", "update", "ns", "prep", "io")

_ERRORS = {0: "LACT_OK", -1: "LACT_EINVAL", -2: "LACT_EALIGN", -3: "LACT_EWORKSPACE",
           -4: "LACT_EUNSUPPORTED", -5: "LACT_EHIP", -6: "LACT_ESCRATCH"}
NOALLOC_SCRATCH_BYTES = 128 << 20   # LACT_NOALLOC_SCRATCH_BYTES


class LactError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERRORS.get(code, code)}: {msg}")
        self.code = code


class LactDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("h", ctypes.c_int32), ("n_kv", ctypes.c_int64), ("n_q", ctypes.c_int64),
                ("chunk", ctypes.c_int64), ("order", ctypes.c_int32), ("use_muon", ctypes.c_int32),
                ("ns_steps", ctypes.c_int32), ("io_dtype", ctypes.c_int32), ("eta_per_matrix", ctypes.c_int32),
                ("fast_weight", ctypes.c_int32)]


FW_SWIGLU, FW_LINEAR = 0, 1


SEG_APPLY_THEN_UPDATE, SEG_UPDATE_THEN_APPLY, SEG_UPDATE_ONLY, SEG_APPLY_ONLY = 0, 1, 2, 3
SEG_MODES = {"apply_then_update": 0, "update_then_apply": 1, "update_only": 2, "apply_only": 3}


class LactSegment(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("reserved", ctypes.c_int32), ("begin", ctypes.c_int64),
                ("end", ctypes.c_int64)]


_lib = None


def load_library(path: str | None = None):
    """Load liblact.so (raises if it has not been built: there is no fallback)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise LactError(-5, f"{p} is missing; build it with paper_2505_23884_amd.build.build()")
    L = ctypes.CDLL(p)
    vp, sz, i32, i64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int64
    dp = ctypes.POINTER(LactDesc)
    L.lact_workspace_bytes.argtypes = [dp, ctypes.POINTER(i32)]
    L.lact_workspace_bytes.restype = sz
    L.lact_check_desc.argtypes = [dp]
    L.lact_check_desc.restype = i32
    L.lact_forward.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.lact_forward.restype = i32
    L.lact_forward_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.lact_forward_noalloc.restype = i32
    L.lact_forward_momentum.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.lact_forward_momentum.restype = i32
    L.lact_forward_schedule.argtypes = [dp, ctypes.POINTER(LactSegment), i64] + [vp] * 13 + [sz, vp]
    L.lact_forward_schedule.restype = i32
    L.lact_backward_workspace_bytes.argtypes = [dp, ctypes.POINTER(i32)]
    L.lact_backward_workspace_bytes.restype = sz
    L.lact_backward_linear.argtypes = [dp] + [vp] * 12 + [vp, sz, vp]
    L.lact_backward_linear.restype = i32
    L.lact_backward.argtypes = [dp] + [vp] * 19 + [sz, vp]
    L.lact_backward.restype = i32
    L.lact_backward_momentum_workspace_bytes.argtypes = [dp, ctypes.POINTER(i32)]
    L.lact_backward_momentum_workspace_bytes.restype = sz
    L.lact_backward_momentum.argtypes = [dp] + [vp] * 30 + [sz, vp]
    L.lact_backward_momentum.restype = i32
    L.lact_backward_schedule_workspace_bytes.argtypes = [dp, ctypes.POINTER(LactSegment), i64, i32,
                                                         ctypes.POINTER(i32)]
    L.lact_backward_schedule_workspace_bytes.restype = sz
    L.lact_backward_schedule.argtypes = [dp, ctypes.POINTER(LactSegment), i64] + [vp] * 30 + [sz, vp]
    L.lact_backward_schedule.restype = i32
    f32 = ctypes.c_float
    L.lact_prologue.argtypes = [dp, vp, vp, f32, vp, vp, vp, vp, vp, vp, vp]
    L.lact_prologue.restype = i32
    L.lact_rmsnorm_out.argtypes = [dp, vp, vp, f32, vp, vp]
    L.lact_prologue_backward.argtypes = [dp, vp, vp, f32] + [vp] * 10
    L.lact_prologue_backward.restype = i32
    L.lact_rmsnorm_out_backward_workspace_bytes.argtypes = [dp, i32, ctypes.POINTER(i32)]
    L.lact_rmsnorm_out_backward_workspace_bytes.restype = sz
    L.lact_rmsnorm_out_backward.argtypes = [dp, vp, vp, f32, vp, vp, vp, vp, sz, vp]
    L.lact_rmsnorm_out_backward.restype = i32
    L.lact_rmsnorm_out.restype = i32
    L.lact_timing_enable.argtypes = [i32]
    L.lact_timing_enable.restype = i32
    L.lact_timing_reset.argtypes = []
    L.lact_timing_reset.restype = i32
    L.lact_timing_read.argtypes = [i32, ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_double)]
    L.lact_timing_read.restype = i32
    for f in ("lact_strerror",):
        getattr(L, f).argtypes = [i32]
        getattr(L, f).restype = ctypes.c_char_p
    for f in ("lact_last_hip_error", "lact_version"):
        getattr(L, f).argtypes = []
        getattr(L, f).restype = ctypes.c_char_p
    if path is None:
        _lib = L
    return L


def lib():
    return load_library()


def _raise(code: int):
    L = lib()
    msg = L.lact_strerror(code).decode()
    if code == -5:
        msg += ": " + L.lact_last_hip_error().decode()
    raise LactError(code, msg)


def make_desc(B, H, d, h, n_kv, n_q, chunk, order=0, use_muon=False, ns_steps=5, io_dtype=IO_BF16,
              eta_per_matrix=False, fast_weight=FW_SWIGLU):
    return LactDesc(int(B), int(H), int(d), int(h), int(n_kv), int(n_q), int(chunk), int(order),
                    int(bool(use_muon)), int(ns_steps), int(io_dtype), int(bool(eta_per_matrix)), int(fast_weight))


def check_desc(desc: LactDesc) -> int:
    return lib().lact_check_desc(ctypes.byref(desc))


def workspace_bytes(desc: LactDesc) -> int:
    err = ctypes.c_int(0)
    n = lib().lact_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    if err.value:
        _raise(err.value)
    return int(n)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _marshal(q, k, v, eta, W1, W2, W3, extra, chunk, order, use_muon, ns_steps, out, workspace, stream,
             fast_weight=FW_SWIGLU, need_workspace=True):
    """Checks shapes and dtypes; returns (desc, out, workspace, stream handle)
    (workspace None when need_workspace is False)."""
    import torch
    if q.dim() == 4:
        B, H = q.shape[0], q.shape[1]
    elif q.dim() == 3:
        B, H = q.shape[0], 1
    else:
        raise LactError(-1, "q must be [B, H, n_q, d] or [BH, n_q, d]")
    n_q, d = q.shape[-2], q.shape[-1]
    n_kv = k.shape[-2]
    h = W1.shape[-2]
    if q.dtype == torch.bfloat16:
        io = IO_BF16
    elif q.dtype == torch.float32:
        io = IO_FP32
    else:
        raise LactError(-1, f"unsupported q dtype {q.dtype}")
    named = [(q, "q"), (k, "k"), (v, "v"), (eta, "eta"), (W1, "W1"), (W2, "W2"), (W3, "W3"), *extra]
    for t, name in named:
        if not t.is_cuda or not t.is_contiguous():
            raise LactError(-1, f"{name} must be a contiguous device tensor")
    if k.dtype != q.dtype or v.dtype != q.dtype:
        raise LactError(-1, "q, k, v must share one dtype")
    if eta.dtype != torch.float32 or any(t.dtype != torch.float32 for t, _ in named[4:]):
        raise LactError(-1, "eta, beta, the fast weights and the momentum are fp32")
    BH = B * H
    # per-matrix rates: eta [.., n_kv, 3] (one more trailing dim than k's token axis)
    lr3 = eta.dim() == k.dim() and eta.shape[-1] == 3
    if (k.numel() != BH * n_kv * d or v.numel() != BH * n_kv * d or eta.numel() != BH * n_kv * (3 if lr3 else 1)
            or W1.numel() != BH * h * d or W3.numel() != BH * h * d or W2.numel() != BH * d * h
            or W2.shape[-2] != d or W2.shape[-1] != h or W1.shape[-1] != d):
        raise LactError(-1, "inconsistent tensor shapes")
    desc = make_desc(B, H, d, h, n_kv, n_q, chunk, order, use_muon, ns_steps, io, lr3, fast_weight)
    if need_workspace and workspace is None:
        workspace = torch.empty(max(workspace_bytes(desc), 1), dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    if stream is None:
        stream = torch.cuda.current_stream(q.device).cuda_stream
    return desc, out, workspace, stream


def forward(q, k, v, eta, W1, W2, W3, chunk, order=APPLY_THEN_UPDATE, use_muon=False,
            ns_steps=5, out=None, workspace=None, stream=None):
    """LaCT fast-weight path on the GPU (see include/lact.h for the semantics).

    q [B, H, n_q, d] (or [BH, n_q, d]); k, v [.., n_kv, d]; bf16 or fp32 (same dtype);
    eta [.., n_kv] fp32; W1, W3 [.., h, d], W2 [.., d, h] fp32, updated IN PLACE.
    Returns o with q's shape and dtype. Runs on torch's current stream unless a
    stream is given; allocates the workspace unless one is passed.
    """
    desc, out, workspace, stream = _marshal(q, k, v, eta, W1, W2, W3, [], chunk, order, use_muon,
                                            ns_steps, out, workspace, stream)
    rc = lib().lact_forward(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(W1),
                            _ptr(W2), _ptr(W3), _ptr(out), _ptr(workspace),
                            ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                            ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return out


def forward_noalloc(q, k, v, eta, W1, W2, W3, chunk, order=APPLY_THEN_UPDATE, use_muon=False, ns_steps=5,
                    out=None, stream=None):
    """forward() through lact_forward_noalloc: no workspace argument; the
    library's fixed per-device scratch array serves as the workspace (calls
    that may overlap on one device race on it). ``out`` is allocated here
    when not given (pass it to allocate nothing)."""
    desc, out, _, stream = _marshal(q, k, v, eta, W1, W2, W3, [], chunk, order, use_muon, ns_steps, out, None,
                                    stream, need_workspace=False)
    rc = lib().lact_forward_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(W1),
                                    _ptr(W2), _ptr(W3), _ptr(out), ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return out


def forward_momentum(q, k, v, eta, beta, W1, W2, W3, M1=None, M2=None, M3=None, *, chunk,
                     order=APPLY_THEN_UPDATE, use_muon=False, ns_steps=5, out=None, workspace=None,
                     stream=None):
    """The path with the momentum test-time optimizer (lact_forward_momentum).

    beta [.., n_kv] fp32 per-token momentum factor; M1, M3 [.., h, d], M2 [.., d, h]
    fp32 momentum, updated IN PLACE (zeros are allocated when omitted). W as in
    forward(). Returns (o, (M1, M2, M3)).
    """
    import torch
    if M1 is None and M2 is None and M3 is None:
        M1, M2, M3 = (torch.zeros_like(w) for w in (W1, W2, W3))
    if M1 is None or M2 is None or M3 is None:
        raise LactError(-1, "pass all three momentum tensors or none")
    for m, w, name in ((M1, W1, "M1"), (M2, W2, "M2"), (M3, W3, "M3")):
        if m.shape != w.shape:
            raise LactError(-1, f"{name} must have the shape of its fast weight")
    if beta.numel() != k.numel() // k.shape[-1]:
        raise LactError(-1, "beta must be [.., n_kv]")
    extra = [(beta, "beta"), (M1, "M1"), (M2, "M2"), (M3, "M3")]
    desc, out, workspace, stream = _marshal(q, k, v, eta, W1, W2, W3, extra, chunk, order, use_muon,
                                            ns_steps, out, workspace, stream)
    rc = lib().lact_forward_momentum(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta),
                                     _ptr(beta), _ptr(W1), _ptr(W2), _ptr(W3), _ptr(M1), _ptr(M2),
                                     _ptr(M3), _ptr(out), _ptr(workspace),
                                     ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                     ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return out, (M1, M2, M3)


def forward_linear(q, k, v, eta, W, chunk, order=APPLY_THEN_UPDATE, use_muon=False, ns_steps=5, beta=None, M=None,
                   out=None, workspace=None, stream=None):
    """The path with the linear fast weight f_W(x) = W x (lact_desc.fast_weight =
    LACT_FW_LINEAR): W [.., d, d] fp32, updated IN PLACE; q, k, v, eta as in
    forward(). With ``beta`` the updates use momentum (M [.., d, d] updated in
    place, zeros allocated when omitted) and the return is (o, M); else o.
    """
    import torch
    if W.shape[-1] != W.shape[-2]:
        raise LactError(-1, "the linear fast weight is square, [.., d, d]")
    extra = []
    if beta is not None:
        M = torch.zeros_like(W) if M is None else M
        if M.shape != W.shape:
            raise LactError(-1, "M must have W's shape")
        extra = [(beta, "beta"), (M, "M")]
    # W stands in for all three matrices in the shape checks (h = d)
    desc, out, workspace, stream = _marshal(q, k, v, eta, W, W, W, extra, chunk, order, use_muon, ns_steps, out,
                                            workspace, stream, FW_LINEAR)
    wsb = ctypes.c_size_t(workspace.numel() * workspace.element_size())
    if beta is None:
        rc = lib().lact_forward(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(W), ctypes.c_void_p(0),
                                ctypes.c_void_p(0), _ptr(out), _ptr(workspace), wsb, ctypes.c_void_p(stream))
    else:
        rc = lib().lact_forward_momentum(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(beta), _ptr(W),
                                         ctypes.c_void_p(0), ctypes.c_void_p(0), _ptr(M), ctypes.c_void_p(0),
                                         ctypes.c_void_p(0), _ptr(out), _ptr(workspace), wsb, ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return (out, M) if beta is not None else out


def backward_workspace_bytes(desc: LactDesc) -> int:
    err = ctypes.c_int(0)
    n = lib().lact_backward_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    if err.value:
        _raise(err.value)
    return int(n)


def backward_linear(q, k, v, eta, W0, dout, chunk, order=APPLY_THEN_UPDATE, dW_final=None, use_muon=False,
                    ns_steps=5, out=None, workspace=None, stream=None):
    """Backward of forward_linear (lact_backward_linear): the cotangents of q,
    k, v, eta and of the initial fast weight W0 [.., d, d] (fp32, not written)
    given dout (q's shape and dtype) and, optionally, the cotangent of the
    final fast weight. Returns (dq, dk, dv, deta, dW0), written into ``out``
    (a tuple of five tensors of those shapes) when it is given."""
    import torch
    if W0.shape[-1] != W0.shape[-2]:
        raise LactError(-1, "the linear fast weight is square, [.., d, d]")
    extra = [(dout, "dout")] + ([(dW_final, "dW_final")] if dW_final is not None else [])
    if dout.shape != q.shape or dout.dtype != q.dtype:
        raise LactError(-1, "dout must have q's shape and dtype")
    if dW_final is not None and (dW_final.shape != W0.shape or dW_final.dtype != torch.float32):
        raise LactError(-1, "dW_final must have W0's shape, fp32")
    desc, dq, _, stream = _marshal(q, k, v, eta, W0, W0, W0, extra[1:], chunk, order, use_muon, ns_steps,
                                   None if out is None else out[0], None, stream, FW_LINEAR, need_workspace=False)
    if not dout.is_cuda or not dout.is_contiguous():
        raise LactError(-1, "dout must be a contiguous device tensor")
    if workspace is None:
        workspace = torch.empty(max(backward_workspace_bytes(desc), 1), dtype=torch.uint8, device=q.device)
    if out is None:
        dk, dv = torch.empty_like(k), torch.empty_like(v)
        deta = torch.empty_like(eta)
        dW0 = torch.empty_like(W0)
    else:
        _, dk, dv, deta, dW0 = out
        for t, ref, name in ((dq, q, "dq"), (dk, k, "dk"), (dv, v, "dv"), (deta, eta, "deta"), (dW0, W0, "dW0")):
            if t.shape != ref.shape or t.dtype != ref.dtype or not t.is_cuda or not t.is_contiguous():
                raise LactError(-1, f"{name} must be a contiguous device tensor shaped like its input")
    rc = lib().lact_backward_linear(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(W0), _ptr(dout),
                                    _ptr(dW_final), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(deta), _ptr(dW0),
                                    _ptr(workspace), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                    ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return dq, dk, dv, deta, dW0


def backward(q, k, v, eta, W1, W2, W3, dout, chunk, order=APPLY_THEN_UPDATE, dW_final=None, use_muon=False,
             ns_steps=5, out=None, workspace=None, stream=None):
    """Backward of forward() for the SwiGLU fast weight (lact_backward), with
    or without Muon, one rate per token or per matrix, no momentum: the cotangents of q, k, v, eta and of the initial fast
    weights W1, W2, W3 (fp32, not written) given dout (q's shape and dtype)
    and, optionally, dW_final = (dW1, dW2, dW3) of the final fast weights (any
    of them None). Returns (dq, dk, dv, deta, dW1, dW2, dW3), written into
    ``out`` (a tuple of seven tensors of those shapes) when it is given."""
    import torch
    dWf = tuple(dW_final) if dW_final is not None else (None, None, None)
    extra = [(t, name) for t, name in zip(dWf, ("dW1_final", "dW2_final", "dW3_final")) if t is not None]
    if dout.shape != q.shape or dout.dtype != q.dtype:
        raise LactError(-1, "dout must have q's shape and dtype")
    for t, ref in zip(dWf, (W1, W2, W3)):
        if t is not None and (t.shape != ref.shape or t.dtype != torch.float32):
            raise LactError(-1, "dW_final tensors must have the fast weights' shapes, fp32")
    desc, dq, _, stream = _marshal(q, k, v, eta, W1, W2, W3, extra, chunk, order, use_muon, ns_steps,
                                   None if out is None else out[0], None, stream, FW_SWIGLU, need_workspace=False)
    if not dout.is_cuda or not dout.is_contiguous():
        raise LactError(-1, "dout must be a contiguous device tensor")
    if workspace is None:
        workspace = torch.empty(max(backward_workspace_bytes(desc), 1), dtype=torch.uint8, device=q.device)
    if out is None:
        res = (dq, torch.empty_like(k), torch.empty_like(v), torch.empty_like(eta), torch.empty_like(W1),
               torch.empty_like(W2), torch.empty_like(W3))
    else:
        res = tuple(out)
        for t, ref, name in zip(res, (q, k, v, eta, W1, W2, W3), ("dq", "dk", "dv", "deta", "dW1", "dW2", "dW3")):
            if t.shape != ref.shape or t.dtype != ref.dtype or not t.is_cuda or not t.is_contiguous():
                raise LactError(-1, f"{name} must be a contiguous device tensor shaped like its input")
    rc = lib().lact_backward(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(W1), _ptr(W2), _ptr(W3),
                             _ptr(dout), _ptr(dWf[0]), _ptr(dWf[1]), _ptr(dWf[2]), *(_ptr(t) for t in res),
                             _ptr(workspace), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                             ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return res


def backward_momentum_workspace_bytes(desc: LactDesc) -> int:
    err = ctypes.c_int(0)
    n = lib().lact_backward_momentum_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    if err.value:
        _raise(err.value)
    return int(n)


def backward_momentum(q, k, v, eta, beta, W0, M0, dout, chunk, order=APPLY_THEN_UPDATE, dW_final=None,
                      dM_final=None, use_muon=False, ns_steps=5, out=None, workspace=None, stream=None):
    """Backward of the momentum optimizer's path (lact_backward_momentum).

    W0, M0: the fast weights and momentum before the forward (fp32, not
    written): triples (W1, W2, W3), (M1, M2, M3) for SwiGLU, single [.., d, d]
    tensors for the linear fast weight; dW_final, dM_final the same (any of
    them None: zero). Returns (dq, dk, dv, deta, dbeta, dW0, dM0) with dW0,
    dM0 shaped like W0, M0; written into ``out`` (that tuple) when given."""
    import torch
    linear = not isinstance(W0, (tuple, list))
    Ws = (W0,) if linear else tuple(W0)
    Ms = (M0,) if linear else tuple(M0)
    nm = len(Ws)
    if nm not in (1, 3) or len(Ms) != nm:
        raise LactError(-1, "W0 and M0: three tensors (SwiGLU) or one (linear)")
    if linear and W0.shape[-1] != W0.shape[-2]:
        raise LactError(-1, "the linear fast weight is square, [.., d, d]")
    dWf = (None,) * nm if dW_final is None else ((dW_final,) if linear else tuple(dW_final))
    dMf = (None,) * nm if dM_final is None else ((dM_final,) if linear else tuple(dM_final))
    if len(dWf) != nm or len(dMf) != nm:
        raise LactError(-1, "dW_final and dM_final must match W0")
    for t, ref in zip(Ms + dWf + dMf, Ws * 3):
        if t is not None and (t.shape != ref.shape or t.dtype != torch.float32):
            raise LactError(-1, "momentum and final cotangents must have the fast weights' shapes, fp32")
    if dout.shape != q.shape or dout.dtype != q.dtype:
        raise LactError(-1, "dout must have q's shape and dtype")
    if beta.numel() != k.numel() // k.shape[-1] or beta.dtype != torch.float32:
        raise LactError(-1, "beta must be [.., n_kv] fp32")
    extra = [(beta, "beta")] + [(t, "M") for t in Ms] + [(t, "d_final") for t in dWf + dMf if t is not None]
    W1, W2, W3 = (Ws[0],) * 3 if linear else Ws
    desc, dq, _, stream = _marshal(q, k, v, eta, W1, W2, W3, extra, chunk, order, use_muon, ns_steps,
                                   None if out is None else out[0], None, stream,
                                   FW_LINEAR if linear else FW_SWIGLU, need_workspace=False)
    if not dout.is_cuda or not dout.is_contiguous():
        raise LactError(-1, "dout must be a contiguous device tensor")
    if workspace is None:
        workspace = torch.empty(max(backward_momentum_workspace_bytes(desc), 1), dtype=torch.uint8, device=q.device)
    if out is None:
        dW = tuple(torch.empty_like(w) for w in Ws)
        dM = tuple(torch.empty_like(m) for m in Ms)
        head = (dq, torch.empty_like(k), torch.empty_like(v), torch.empty_like(eta), torch.empty_like(beta))
    else:
        head = tuple(out[:5])
        dW = (out[5],) if linear else tuple(out[5])
        dM = (out[6],) if linear else tuple(out[6])
        refs = (q, k, v, eta, beta) + Ws + Ms
        for t, ref in zip(head + dW + dM, refs):
            if t.shape != ref.shape or t.dtype != ref.dtype or not t.is_cuda or not t.is_contiguous():
                raise LactError(-1, "outputs must be contiguous device tensors shaped like their inputs")
    pad = (lambda xs: tuple(xs) + (None,) * (3 - len(xs)))
    args = ([_ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(beta)] + [_ptr(t) for t in pad(Ws)] +
            [_ptr(t) for t in pad(Ms)] + [_ptr(dout)] + [_ptr(t) for t in pad(dWf)] + [_ptr(t) for t in pad(dMf)] +
            [_ptr(t) for t in head[:4]] + [_ptr(head[4])] + [_ptr(t) for t in pad(dW)] + [_ptr(t) for t in pad(dM)])
    rc = lib().lact_backward_momentum(ctypes.byref(desc), *args, _ptr(workspace),
                                      ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                      ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    if linear:
        return head + (dW[0], dM[0])
    return head + (dW, dM)


def forward_schedule(q, k, v, eta, W1, W2, W3, schedule, *, use_muon=False, ns_steps=5, beta=None,
                     M1=None, M2=None, M3=None, chunk=None, out=None, workspace=None, stream=None):
    """The path over a general schedule (lact_forward_schedule): ``schedule`` is a
    sequence of (mode, begin, end) with mode a name of SEG_MODES or its code.
    ``chunk`` (the workspace bound) defaults to the longest update segment.
    With ``beta`` the updates use momentum (M1..M3 updated in place, zeros
    allocated when omitted). Returns o, or (o, (M1, M2, M3)) with beta.
    With W2 and W3 None the fast weight is the linear one (W1 [.., d, d];
    M1 its state, returned alone; M2 and M3 unused).
    """
    import torch
    segs, longest = _segments(schedule)
    linear = W2 is None and W3 is None
    extra = []
    if beta is not None:
        if linear:
            M1 = torch.zeros_like(W1) if M1 is None else M1
            if M1.shape != W1.shape:
                raise LactError(-1, "M1 must have W1's shape")
            extra = [(beta, "beta"), (M1, "M1")]
        else:
            if M1 is None and M2 is None and M3 is None:
                M1, M2, M3 = (torch.zeros_like(w) for w in (W1, W2, W3))
            if M1 is None or M2 is None or M3 is None:
                raise LactError(-1, "pass all three momentum tensors or none")
            extra = [(beta, "beta"), (M1, "M1"), (M2, "M2"), (M3, "M3")]
    if linear and W1.shape[-1] != W1.shape[-2]:
        raise LactError(-1, "the linear fast weight is square, [.., d, d]")
    Wm = (W1, W1, W1) if linear else (W1, W2, W3)
    desc, out, workspace, stream = _marshal(q, k, v, eta, *Wm, extra, chunk or longest, 0, use_muon,
                                            ns_steps, out, workspace, stream, FW_LINEAR if linear else FW_SWIGLU)
    M = (M1, M2, M3) if beta is not None else (None, None, None)
    rc = lib().lact_forward_schedule(ctypes.byref(desc), segs, ctypes.c_int64(len(schedule)), _ptr(q), _ptr(k),
                                     _ptr(v), _ptr(eta), _ptr(beta), _ptr(W1), _ptr(W2), _ptr(W3),
                                     *[_ptr(m) for m in M], _ptr(out), _ptr(workspace),
                                     ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                     ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    if beta is not None:
        return out, (M1 if linear else M)
    return out


def _segments(schedule):
    """ctypes segments of a (mode, begin, end) sequence, and the longest update."""
    segs = (LactSegment * max(len(schedule), 1))()
    longest = 1
    for i, (mode, b, e) in enumerate(schedule):
        m = SEG_MODES[mode] if isinstance(mode, str) else int(mode)
        segs[i] = LactSegment(m, 0, int(b), int(e))
        if m != SEG_APPLY_ONLY:
            longest = max(longest, int(e) - int(b))
    return segs, longest


def backward_schedule_workspace_bytes(desc: LactDesc, schedule, momentum=False) -> int:
    segs, _ = _segments(schedule)
    err = ctypes.c_int(0)
    n = lib().lact_backward_schedule_workspace_bytes(ctypes.byref(desc), segs, ctypes.c_int64(len(schedule)),
                                                     int(bool(momentum)), ctypes.byref(err))
    if err.value:
        _raise(err.value)
    return int(n)


def backward_schedule(q, k, v, eta, W1, W2, W3, dout, schedule, *, dW_final=None, use_muon=False, ns_steps=5,
                      beta=None, M=None, dM_final=None, chunk=None, out=None, workspace=None, stream=None):
    """Backward of forward_schedule (lact_backward_schedule), SwiGLU fast
    weight: the cotangents of q, k, v, eta and of the initial W1, W2, W3 (not
    written) given dout and, optionally, dW_final = (dW1, dW2, dW3). With
    ``beta`` the momentum optimizer (M = (M1, M2, M3) the initial state, zeros
    when omitted; dM_final its final cotangents). Returns (dq, dk, dv, deta,
    (dW1, dW2, dW3)) or, with beta, (dq, dk, dv, deta, dbeta, (dW1, dW2, dW3),
    (dM1, dM2, dM3)); written into ``out`` (that tuple) when given. With W2
    and W3 None the fast weight is the linear one: W1 [.., d, d], and M,
    dW_final, dM_final and the returned dW, dM single tensors."""
    import torch
    segs, longest = _segments(schedule)
    linear = W2 is None and W3 is None
    if linear and W1.shape[-1] != W1.shape[-2]:
        raise LactError(-1, "the linear fast weight is square, [.., d, d]")
    one = lambda t: None if t is None else (t,)
    W = (W1,) if linear else (W1, W2, W3)
    mom = beta is not None
    if linear:
        M, dW_final, dM_final = one(M), one(dW_final), one(dM_final)
        if out is not None:
            out = tuple(out[:-2]) + ((out[-2],), (out[-1],)) if mom else tuple(out[:-1]) + ((out[-1],),)
    if mom and M is None:
        M = tuple(torch.zeros_like(w) for w in W)
    dWf = (None,) * len(W) if dW_final is None else tuple(dW_final)
    dMf = (None,) * len(W) if (dM_final is None or not mom) else tuple(dM_final)
    for t, ref in zip(dWf + dMf + (tuple(M) if mom else ()), W * 3):
        if t is not None and (t.shape != ref.shape or t.dtype != torch.float32):
            raise LactError(-1, "momentum and final cotangents must have the fast weights' shapes, fp32")
    if dout.shape != q.shape or dout.dtype != q.dtype:
        raise LactError(-1, "dout must have q's shape and dtype")
    extra = [(t, "d_final") for t in dWf + dMf if t is not None]
    if mom:
        extra += [(beta, "beta")] + [(m, "M") for m in M]
    Wm = (W1, W1, W1) if linear else W
    desc, dq, _, stream = _marshal(q, k, v, eta, *Wm, extra, chunk or longest, 0, use_muon, ns_steps,
                                   None if out is None else out[0], None, stream,
                                   FW_LINEAR if linear else FW_SWIGLU, need_workspace=False)
    if not dout.is_cuda or not dout.is_contiguous():
        raise LactError(-1, "dout must be a contiguous device tensor")
    if workspace is None:
        nb = backward_schedule_workspace_bytes(desc, schedule, mom)
        workspace = torch.empty(max(nb, 1), dtype=torch.uint8, device=q.device)
    if out is None:
        head = (dq, torch.empty_like(k), torch.empty_like(v), torch.empty_like(eta))
        dW = tuple(torch.empty_like(w) for w in W)
        dbeta = torch.empty_like(beta) if mom else None
        dM = tuple(torch.empty_like(w) for w in W) if mom else (None,) * len(W)
    else:
        head = tuple(out[:4])
        dbeta = out[4] if mom else None
        dW = tuple(out[5] if mom else out[4])
        dM = tuple(out[6]) if mom else (None,) * len(W)
    Ms = tuple(M) if mom else (None,) * len(W)
    pad = lambda t: tuple(t) + (None,) * (3 - len(t))
    args = ([_ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(beta)] + [_ptr(w) for w in pad(W)] +
            [_ptr(m) for m in pad(Ms)] + [_ptr(dout)] + [_ptr(t) for t in pad(dWf)] + [_ptr(t) for t in pad(dMf)] +
            [_ptr(t) for t in head] + [_ptr(dbeta)] + [_ptr(t) for t in pad(dW)] + [_ptr(t) for t in pad(dM)])
    rc = lib().lact_backward_schedule(ctypes.byref(desc), segs, ctypes.c_int64(len(schedule)), *args, _ptr(workspace),
                                      ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                      ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    if linear:
        dW, dM = dW[0], dM[0]
    if mom:
        return head + (dbeta, dW, dM)
    return head + (dW,)


def prologue(qkv, lr_raw, lr_bias, beta_raw=None, n_kv=None, out=None, stream=None):
    """The layer's prologue (lact_prologue): qkv [B, L, 3, H, d] (bf16 or fp32),
    lr_raw [B, L, H] or [B, L, H, 3] fp32, beta_raw [B, L, H] fp32 or None.
    Returns (q [B, H, L, d], k, v [B, H, n_kv, d], eta [B, H, n_kv(, 3)], beta
    [B, H, n_kv] or None); ``out`` may hold preallocated tensors of those shapes.
    """
    import torch
    if qkv.dim() != 5 or qkv.shape[2] != 3:
        raise LactError(-1, "qkv must be [B, L, 3, H, d]")
    B, L, _, H, d = qkv.shape
    n_kv = L if n_kv is None else int(n_kv)
    lr3 = lr_raw.dim() == 4
    if lr_raw.shape[:3] != (B, L, H) or (lr3 and lr_raw.shape[3] != 3):
        raise LactError(-1, "lr_raw must be [B, L, H] or [B, L, H, 3]")
    if beta_raw is not None and beta_raw.shape != (B, L, H):
        raise LactError(-1, "beta_raw must be [B, L, H]")
    for t, name in ((qkv, "qkv"), (lr_raw, "lr_raw"), (beta_raw, "beta_raw")):
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise LactError(-1, f"{name} must be a contiguous device tensor")
    if lr_raw.dtype != torch.float32 or (beta_raw is not None and beta_raw.dtype != torch.float32):
        raise LactError(-1, "lr_raw and beta_raw are fp32")
    io = IO_BF16 if qkv.dtype == torch.bfloat16 else IO_FP32 if qkv.dtype == torch.float32 else None
    if io is None:
        raise LactError(-1, f"unsupported qkv dtype {qkv.dtype}")
    if out is None:
        e = lambda *sh, dt=qkv.dtype: torch.empty(*sh, dtype=dt, device=qkv.device)
        out = (e(B, H, L, d), e(B, H, n_kv, d), e(B, H, n_kv, d),
               e(B, H, n_kv, *((3,) if lr3 else ()), dt=torch.float32),
               e(B, H, n_kv, dt=torch.float32) if beta_raw is not None else None)
    q, k, v, eta, beta = out
    desc = make_desc(B, H, d, d, n_kv, L, 1, 0, False, 0, io, lr3)   # h unused: any valid value
    if stream is None:
        stream = torch.cuda.current_stream(qkv.device).cuda_stream
    rc = lib().lact_prologue(ctypes.byref(desc), _ptr(qkv), _ptr(lr_raw), ctypes.c_float(lr_bias), _ptr(beta_raw),
                             _ptr(q), _ptr(k), _ptr(v), _ptr(eta), _ptr(beta), ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return q, k, v, eta, beta


def rmsnorm_out(o, weight=None, eps=1e-6, out=None, stream=None):
    """Per-head RMSNorm of the path output (lact_rmsnorm_out): o [B, H, L, d]
    -> y [B, L, H, d]; weight [H, d] fp32 or None."""
    import torch
    if o.dim() != 4:
        raise LactError(-1, "o must be [B, H, L, d]")
    B, H, L, d = o.shape
    if not o.is_cuda or not o.is_contiguous():
        raise LactError(-1, "o must be a contiguous device tensor")
    if weight is not None and (weight.shape != (H, d) or weight.dtype != torch.float32 or not weight.is_contiguous()):
        raise LactError(-1, "weight must be a contiguous fp32 [H, d] tensor")
    io = IO_BF16 if o.dtype == torch.bfloat16 else IO_FP32 if o.dtype == torch.float32 else None
    if io is None:
        raise LactError(-1, f"unsupported o dtype {o.dtype}")
    y = torch.empty(B, L, H, d, dtype=o.dtype, device=o.device) if out is None else out
    desc = make_desc(B, H, d, d, 0, L, 1, 0, False, 0, io)
    if stream is None:
        stream = torch.cuda.current_stream(o.device).cuda_stream
    rc = lib().lact_rmsnorm_out(ctypes.byref(desc), _ptr(o), _ptr(weight), ctypes.c_float(eps), _ptr(y),
                                ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return y


def prologue_backward(qkv, lr_raw, lr_bias, beta_raw, dq, dk, dv, deta, dbeta=None, out=None, stream=None):
    """Reverse of prologue() (lact_prologue_backward): the cotangents (dqkv
    [B, L, 3, H, d], dlr_raw like lr_raw, dbeta_raw [B, L, H] or None) of the
    prologue's inputs given those of its outputs (dq [B, H, L, d], dk, dv
    [B, H, n_kv, d], deta like eta, dbeta [B, H, n_kv] or None)."""
    import torch
    if qkv.dim() != 5 or qkv.shape[2] != 3:
        raise LactError(-1, "qkv must be [B, L, 3, H, d]")
    B, L, _, H, d = qkv.shape
    n_kv = dk.shape[-2]
    lr3 = lr_raw.dim() == 4
    if dq.shape != (B, H, L, d) or dk.shape != (B, H, n_kv, d) or dv.shape != dk.shape:
        raise LactError(-1, "dq must be [B, H, L, d], dk and dv [B, H, n_kv, d]")
    if deta.shape != (B, H, n_kv, *((3,) if lr3 else ())):
        raise LactError(-1, "deta must be shaped like eta")
    if (beta_raw is None) != (dbeta is None):
        raise LactError(-1, "pass beta_raw and dbeta together")
    for t in (qkv, lr_raw, beta_raw, dq, dk, dv, deta, dbeta):
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise LactError(-1, "inputs must be contiguous device tensors")
    if any(t.dtype != qkv.dtype for t in (dq, dk, dv)):
        raise LactError(-1, "dq, dk, dv must have qkv's dtype")
    io = IO_BF16 if qkv.dtype == torch.bfloat16 else IO_FP32 if qkv.dtype == torch.float32 else None
    if io is None:
        raise LactError(-1, f"unsupported qkv dtype {qkv.dtype}")
    if out is None:
        out = (torch.empty_like(qkv), torch.empty_like(lr_raw),
               torch.empty_like(beta_raw) if beta_raw is not None else None)
    dqkv, dlr, dbr = out
    desc = make_desc(B, H, d, d, n_kv, L, 1, 0, False, 0, io, lr3)   # h unused: any valid value
    if stream is None:
        stream = torch.cuda.current_stream(qkv.device).cuda_stream
    rc = lib().lact_prologue_backward(ctypes.byref(desc), _ptr(qkv), _ptr(lr_raw), ctypes.c_float(lr_bias),
                                      _ptr(beta_raw), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(deta), _ptr(dbeta),
                                      _ptr(dqkv), _ptr(dlr), _ptr(dbr), ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return dqkv, dlr, dbr


def rmsnorm_out_backward(o, dy, weight=None, eps=1e-6, with_dweight=True, out=None, workspace=None, stream=None):
    """Reverse of rmsnorm_out() (lact_rmsnorm_out_backward): from dy [B, L,
    H, d], returns (d_o [B, H, L, d], dweight [H, d] or None; dweight only
    with a weight and with_dweight)."""
    import torch
    if o.dim() != 4:
        raise LactError(-1, "o must be [B, H, L, d]")
    B, H, L, d = o.shape
    if dy.shape != (B, L, H, d) or dy.dtype != o.dtype:
        raise LactError(-1, "dy must be [B, L, H, d] of o's dtype")
    for t in (o, dy, weight):
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise LactError(-1, "inputs must be contiguous device tensors")
    io = IO_BF16 if o.dtype == torch.bfloat16 else IO_FP32 if o.dtype == torch.float32 else None
    if io is None:
        raise LactError(-1, f"unsupported o dtype {o.dtype}")
    want_dw = weight is not None and with_dweight
    if out is None:
        out = (torch.empty_like(o), torch.empty_like(weight) if want_dw else None)
    d_o, dw = out
    desc = make_desc(B, H, d, d, 0, L, 1, 0, False, 0, io)
    if workspace is None and want_dw:
        err = ctypes.c_int(0)
        nb = lib().lact_rmsnorm_out_backward_workspace_bytes(ctypes.byref(desc), 1, ctypes.byref(err))
        if err.value:
            _raise(err.value)
        workspace = torch.empty(max(int(nb), 1), dtype=torch.uint8, device=o.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if stream is None:
        stream = torch.cuda.current_stream(o.device).cuda_stream
    rc = lib().lact_rmsnorm_out_backward(ctypes.byref(desc), _ptr(o), _ptr(weight), ctypes.c_float(eps), _ptr(dy),
                                         _ptr(d_o), _ptr(dw), _ptr(workspace), ctypes.c_size_t(nbytes),
                                         ctypes.c_void_p(stream))
    if rc:
        _raise(rc)
    return d_o, dw


def timing_enable(on: bool = True):
    lib().lact_timing_enable(int(on))


def timing_reset():
    lib().lact_timing_reset()


def timing_read(kclass: int):
    n, ms, fl = ctypes.c_int64(0), ctypes.c_double(0), ctypes.c_double(0)
    rc = lib().lact_timing_read(int(kclass), ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl))
    if rc:
        _raise(rc)
    return int(n.value), float(ms.value), float(fl.value)
