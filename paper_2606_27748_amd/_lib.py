"""ctypes binding of libflexattn.so (the C ABI declared in include/flex.h).

Argument marshalling only: torch tensors supply device pointers and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no CPU or PyTorch fallback: if the library is missing the
calls raise.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflexattn.so")

FLEX_OK, FLEX_ERR_INVALID_ARG, FLEX_ERR_UNSUPPORTED, FLEX_ERR_WORKSPACE, FLEX_ERR_HIP = range(5)
FLEX_F32, FLEX_BF16 = 0, 1
FLEX_STATIONARY, FLEX_NONSTATIONARY = 0, 1
FLEX_PASS_FEATURE_MAP, FLEX_PASS_FWD, FLEX_PASS_BWD, FLEX_PASS_AWD = 0, 1, 2, 3
EXPORTS = ("flex_abi_version", "flex_status_string", "flex_workspace_size",
           "flex_feature_map", "flex_linattn_fwd", "flex_linattn_prefill", "flex_linattn_fwd_noalloc",
           "flex_linattn_bwd",
           "flex_decode_step",
           "flex_awd_loss", "flex_timing_enable", "flex_timing_read")
KERNELS = {"none": 0, "fwd_state": 1, "fwd_sweep": 2, "scan": 3, "bwd_prepass": 4,
           "bwd_dq": 5, "bwd_dkv": 6, "bwd_reduce": 7, "feature_map": 8, "decode_step": 9,
           "awd_fwd": 10, "awd_bwd_k": 11, "awd_wgrad": 12}


class FlexError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} (status {status})")
        self.status = status


class flex_desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("N", ctypes.c_int32),
                ("d", ctypes.c_int32), ("dv", ctypes.c_int32), ("m", ctypes.c_int32),
                ("variant", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("segments", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("sigma", ctypes.c_float)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(
            f"{path} not found: build it with `python -m paper_2606_27748_amd.build` "
            "or __graft_entry__.build()")
    # The calls take device pointers and streams from torch, so the library must
    # bind to the HIP runtime torch loads (torch ships its own copy): importing
    # torch first makes the dynamic linker reuse that runtime.  Loaded the other
    # way round, torch brings a second runtime whose streams the library's
    # launches reject.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, S, I = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    D = ctypes.POINTER(flex_desc)
    lib.flex_abi_version.restype = I
    lib.flex_abi_version.argtypes = []
    lib.flex_status_string.restype = ctypes.c_char_p
    lib.flex_status_string.argtypes = [I]
    lib.flex_workspace_size.restype = I
    lib.flex_workspace_size.argtypes = [D, I, ctypes.POINTER(S)]
    lib.flex_feature_map.restype = I
    lib.flex_feature_map.argtypes = [D, P, P, P, P, P, P, S, P]
    lib.flex_linattn_fwd.restype = I
    lib.flex_linattn_fwd.argtypes = [D, P, P, P, P, P, P, P, P, P, S, P]
    lib.flex_linattn_prefill.restype = I
    lib.flex_linattn_prefill.argtypes = [D, P, P, P, P, P, P, P, P, P, P, S, P]
    lib.flex_linattn_fwd_noalloc.restype = I
    lib.flex_linattn_fwd_noalloc.argtypes = [D, P, P, P, P, P, P, P, P, P]
    lib.flex_linattn_bwd.restype = I
    lib.flex_linattn_bwd.argtypes = [D] + [P] * 15 + [P, S] + [P, S, P]
    lib.flex_decode_step.restype = I
    lib.flex_decode_step.argtypes = [D] + [P] * 10
    lib.flex_awd_loss.restype = I
    lib.flex_awd_loss.argtypes = [D] + [P] * 10 + [S, P]
    lib.flex_timing_enable.restype = I
    lib.flex_timing_enable.argtypes = [I]
    lib.flex_timing_read.restype = I
    lib.flex_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().flex_status_string(int(status)).decode()


def make_desc(B, H, N, d, m, variant="stationary", causal=False, io="bf16",
              dv=None, sigma=1.0, segments=0, chunk=0) -> flex_desc:
    return flex_desc(B, H, N, d, d if dv is None else dv, m,
                     FLEX_NONSTATIONARY if variant == "nonstationary" else FLEX_STATIONARY,
                     1 if causal else 0, chunk, segments,
                     FLEX_BF16 if io == "bf16" else FLEX_F32, FLEX_F32, float(sigma))


def workspace_size(desc: flex_desc, pass_: int) -> int:
    n = ctypes.c_size_t(0)
    st = load().flex_workspace_size(ctypes.byref(desc), pass_, ctypes.byref(n))
    if st != FLEX_OK:
        raise FlexError(st, "flex_workspace_size")
    return n.value


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(st, what):
    if st != FLEX_OK:
        raise FlexError(st, what)


def _workspace(desc, pass_, ws, device):
    import torch
    need = workspace_size(desc, pass_)
    if ws is None or ws.numel() * ws.element_size() < need:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    return ws


def flex_feature_map(desc: flex_desc, X, W1, W2, tau, Phi=None):
    """phi~(X) -> Phi [B,H,N,2m] (io dtype).  Tensors on the GPU."""
    import torch
    if Phi is None:
        Phi = torch.empty(desc.B, desc.H, desc.N, 2 * desc.m, dtype=X.dtype, device=X.device)
    st = load().flex_feature_map(ctypes.byref(desc), _ptr(X), _ptr(W1), _ptr(W2), _ptr(tau),
                                 _ptr(Phi), None, 0, _stream())
    _check(st, "flex_feature_map")
    return Phi


def flex_linattn_fwd(desc: flex_desc, Q, K, V, W1, W2, tau, O=None, den=None, ws=None,
                     want_den=True):
    """Forward linear attention.  Returns (O, den)."""
    import torch
    dev = Q.device
    if O is None:
        O = torch.empty(desc.B, desc.H, desc.N, desc.dv, dtype=Q.dtype, device=dev)
    if den is None and want_den:
        den = torch.empty(desc.B, desc.H, desc.N, dtype=torch.float32, device=dev)
    ws = _workspace(desc, FLEX_PASS_FWD, ws, dev)
    st = load().flex_linattn_fwd(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(V), _ptr(W1),
                                 _ptr(W2), _ptr(tau), _ptr(O), _ptr(den), _ptr(ws),
                                 ws.numel(), _stream())
    _check(st, "flex_linattn_fwd")
    return O, den


def flex_linattn_prefill(desc: flex_desc, Q, K, V, W1, W2, tau, state=None, O=None, den=None,
                         ws=None, want_den=True):
    """Causal forward that also writes the prefix's state in the decode layout
    (decode_state).  Returns (O, den, state)."""
    import torch
    dev = Q.device
    if O is None:
        O = torch.empty(desc.B, desc.H, desc.N, desc.dv, dtype=Q.dtype, device=dev)
    if den is None and want_den:
        den = torch.empty(desc.B, desc.H, desc.N, dtype=torch.float32, device=dev)
    if state is None:
        state = torch.empty(desc.B, desc.H, 2 * desc.m * (desc.dv + 1), dtype=torch.float32, device=dev)
    if state.numel() != desc.B * desc.H * 2 * desc.m * (desc.dv + 1) or state.dtype != torch.float32:
        raise FlexError(FLEX_ERR_INVALID_ARG, "flex_linattn_prefill: state must hold B*H*2m*(dv+1) fp32")
    ws = _workspace(desc, FLEX_PASS_FWD, ws, dev)
    st = load().flex_linattn_prefill(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(V), _ptr(W1),
                                     _ptr(W2), _ptr(tau), _ptr(O), _ptr(den), _ptr(state), _ptr(ws),
                                     ws.numel(), _stream())
    _check(st, "flex_linattn_prefill")
    return O, den, state


def flex_linattn_fwd_noalloc(desc: flex_desc, Q, K, V, W1, W2, tau, O, den=None):
    """Forward linear attention with the library's static scratch as its
    workspace: O (and den, if given) are caller-allocated, nothing else is.
    Returns (O, den)."""
    st = load().flex_linattn_fwd_noalloc(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(V), _ptr(W1),
                                         _ptr(W2), _ptr(tau), _ptr(O), _ptr(den), _stream())
    _check(st, "flex_linattn_fwd_noalloc")
    return O, den


def flex_linattn_bwd(desc: flex_desc, Q, K, V, W1, W2, tau, O, den, dO, dQ=None, dK=None,
                     dV=None, dW1=None, dW2=None, dtau=None, ws=None, want_dtau=True, fwd_ws=None):
    """Backward linear attention.  Returns dict of fp32 gradients.

    fwd_ws: optionally the workspace tensor of the matching flex_linattn_fwd
    call (same descriptor and inputs, unchanged since): its segment states are
    then reused instead of recomputed."""
    import torch
    dev = Q.device
    f32 = torch.float32
    if dQ is None:
        dQ = torch.empty(desc.B, desc.H, desc.N, desc.d, dtype=f32, device=dev)
    if dK is None:
        dK = torch.empty(desc.B, desc.H, desc.N, desc.d, dtype=f32, device=dev)
    if dV is None:
        dV = torch.empty(desc.B, desc.H, desc.N, desc.dv, dtype=f32, device=dev)
    if dW1 is None:
        dW1 = torch.empty(desc.H, desc.m, desc.d, dtype=f32, device=dev)
    if dW2 is None and desc.variant == FLEX_NONSTATIONARY:
        dW2 = torch.empty(desc.H, desc.m, desc.d, dtype=f32, device=dev)
    if dtau is None and want_dtau:
        dtau = torch.empty(desc.H, dtype=f32, device=dev)
    ws = _workspace(desc, FLEX_PASS_BWD, ws, dev)
    st = load().flex_linattn_bwd(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(V), _ptr(W1),
                                 _ptr(W2), _ptr(tau), _ptr(O), _ptr(den), _ptr(dO), _ptr(dQ),
                                 _ptr(dK), _ptr(dV), _ptr(dW1), _ptr(dW2), _ptr(dtau),
                                 _ptr(fwd_ws), 0 if fwd_ws is None else fwd_ws.numel(),
                                 _ptr(ws), ws.numel(), _stream())
    _check(st, "flex_linattn_bwd")
    return dict(dQ=dQ, dK=dK, dV=dV, dW1=dW1, dW2=dW2, dtau=dtau)


def decode_state(desc: flex_desc, device="cuda"):
    """A zero decode state: fp32 [B,H,2m*dv + 2m], per slice S [2m][dv] then z [2m]."""
    import torch
    F = 2 * desc.m
    return torch.zeros(desc.B, desc.H, F * desc.dv + F, dtype=torch.float32, device=device)


def decode_state_views(desc: flex_desc, state):
    """(S [B,H,2m,dv], z [B,H,2m]) views of a decode state."""
    F = 2 * desc.m
    st = state.reshape(desc.B, desc.H, F * (desc.dv + 1))
    return st[..., :F * desc.dv].unflatten(-1, (F, desc.dv)), st[..., F * desc.dv:]


def flex_decode_step(desc: flex_desc, q, k, v, W1, W2, tau, state, o=None, den=None, want_den=True):
    """One decode step: state (fp32, B*H*2m*(dv+1) floats laid out as in
    decode_state, updated in place) takes the new token k, v; returns (o, den)
    for the new token's query q."""
    import torch
    if state.numel() != desc.B * desc.H * 2 * desc.m * (desc.dv + 1) or state.dtype != torch.float32:
        raise FlexError(FLEX_ERR_INVALID_ARG, "flex_decode_step: state must hold B*H*2m*(dv+1) fp32")
    if o is None:
        o = torch.empty(desc.B, desc.H, desc.dv, dtype=q.dtype, device=q.device)
    if den is None and want_den:
        den = torch.empty(desc.B, desc.H, dtype=torch.float32, device=q.device)
    st = load().flex_decode_step(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(W1), _ptr(W2),
                                 _ptr(tau), _ptr(state), _ptr(o), _ptr(den), _stream())
    _check(st, "flex_decode_step")
    return o, den


def flex_awd_loss(desc: flex_desc, Q, K, W1, W2, tau, grads=True, loss=None, dW1=None, dW2=None,
                  dtau=None, ws=None, want_dtau=True):
    """Attention-weight distillation loss per (b,h) slice and, with grads, the
    gradients of its sum over slices with respect to W1, W2 and tau.
    Returns dict(loss [B,H], dW1, dW2, dtau) (fp32; gradients None without grads)."""
    import torch
    dev = Q.device
    f32 = torch.float32
    if loss is None:
        loss = torch.empty(desc.B, desc.H, dtype=f32, device=dev)
    if grads:
        if dW1 is None:
            dW1 = torch.empty(desc.H, desc.m, desc.d, dtype=f32, device=dev)
        if dW2 is None and desc.variant == FLEX_NONSTATIONARY:
            dW2 = torch.empty(desc.H, desc.m, desc.d, dtype=f32, device=dev)
        if dtau is None and want_dtau:
            dtau = torch.empty(desc.H, dtype=f32, device=dev)
    else:
        dW1 = dW2 = dtau = None
    ws = _workspace(desc, FLEX_PASS_AWD, ws, dev)
    st = load().flex_awd_loss(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(W1), _ptr(W2), _ptr(tau),
                              _ptr(loss), _ptr(dW1), _ptr(dW2), _ptr(dtau), _ptr(ws), ws.numel(),
                              _stream())
    _check(st, "flex_awd_loss")
    return dict(loss=loss, dW1=dW1, dW2=dW2, dtau=dtau)


def flex_timing_enable(kernel: str) -> None:
    """Time every launch of one kernel class with HIP events ("none" disables)."""
    _check(load().flex_timing_enable(KERNELS[kernel]), "flex_timing_enable")


def flex_timing_read():
    """(summed milliseconds, number of launches) since the last enable/read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(load().flex_timing_read(ctypes.byref(ms), ctypes.byref(n)), "flex_timing_read")
    return ms.value, n.value
