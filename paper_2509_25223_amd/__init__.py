"""MI355X (gfx950) RLA / RDN sequence mixing: Python binding of librla_mi355x.so.

The functions here carry the C ABI's names (include/rla.h) and only marshal
arguments: they check torch tensors, allocate outputs and the workspace with
torch, and pass raw device pointers plus the current HIP stream to the
library.  Every step of the computation runs in the library's HIP kernels;
there is no fallback, and importing fails loudly if the library is missing.

Tensor conventions (all on the same CUDA/HIP device, contiguous):
  q, k  [B, T, H, d_k]  v [B, T, H, d_v]   bf16 or fp32 (one dtype for all)
        or [T, H, d] packed with cu_seqlens (int32 [N+1], device)
  alpha_s, beta, alpha_r, gamma  [B, T, H] / [T, H]  fp32 gate values
  S0, R0, states out  [N, H, d_k, d_v]  fp32, stored transposed w.r.t. the
        paper's d_v x d_k states
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librla_mi355x.so")

RLA_OK = 0
RLA_FLAG_SAVE_FOR_BACKWARD, RLA_FLAG_USE_SAVED = 1, 2
# variants (include/rla.h): log-cosh residual, ungated output, decayed residual
RLA_FLAG_RESIDUAL_TANH, RLA_FLAG_UNGATED_OUTPUT, RLA_FLAG_DECAYED_RESIDUAL = 4, 8, 16
# input pre-processing: SiLU + L2 norm of q, k; gates given as pre-activations
RLA_FLAG_QK_SILU_L2NORM, RLA_FLAG_GATE_PREACT = 32, 64
RLA_F32, RLA_BF16 = 0, 1
RLA_OP_RLA_FORWARD, RLA_OP_RDN_FORWARD, RLA_OP_RDN_BACKWARD, RLA_OP_RLA_BACKWARD = 0, 1, 2, 3

SYMBOLS = ("rla_workspace_size", "rla_status_string", "rla_forward", "rdn_forward",
           "rla_backward", "rdn_backward", "rla_set_stage_events", "rla_decode", "rdn_decode",
           "rdn_forward_noalloc")
RLA_ERR_SCRATCH = 8
RLA_NOALLOC_SCRATCH_BYTES = 128 << 20


class rla_problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seq_len", ctypes.c_int64),
                ("num_heads", ctypes.c_int64), ("head_dim_k", ctypes.c_int64),
                ("head_dim_v", ctypes.c_int64), ("num_seqs", ctypes.c_int64),
                ("cu_seqlens", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("clip", ctypes.c_float), ("out_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("decay_param", ctypes.c_void_p),
                ("decay_param_grad", ctypes.c_void_p)]


class RLAError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, status_string(status), status))


_lib = None


def load_library():
    """Loads librla_mi355x.so (built by paper_2509_25223_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("librla_mi355x.so is not built; run `python -m paper_2509_25223_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz, pp = ctypes.c_void_p, ctypes.c_size_t, ctypes.POINTER(rla_problem)
    lib.rla_workspace_size.argtypes = [pp, ctypes.c_int]
    lib.rla_workspace_size.restype = sz
    lib.rla_set_stage_events.argtypes = [ctypes.c_void_p, ctypes.c_int]
    lib.rla_set_stage_events.restype = None
    lib.rla_status_string.argtypes = [ctypes.c_int]
    lib.rla_status_string.restype = ctypes.c_char_p
    fwd_args = [pp] + [vp] * 3 + [vp] * 4 + [vp] * 2 + [vp] * 3 + [vp, sz, vp]
    for name in ("rla_forward", "rdn_forward"):
        f = getattr(lib, name)
        f.argtypes = fwd_args
        f.restype = ctypes.c_int
    for name in ("rla_decode", "rdn_decode", "rdn_forward_noalloc"):
        f = getattr(lib, name)
        f.argtypes = [pp] + [vp] * 3 + [vp] * 4 + [vp] * 2 + [vp] * 3 + [vp]
        f.restype = ctypes.c_int
    for name in ("rla_backward", "rdn_backward"):
        f = getattr(lib, name)
        f.argtypes = ([pp] + [vp] * 3 + [vp] * 4 + [vp] * 2 + [vp] * 3 + [vp] * 3 + [vp] * 4 +
                      [vp] * 2 + [vp, sz, vp])
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().rla_status_string(int(status)).decode()


rla_status_string = status_string


def rla_set_stage_events(events) -> None:
    """Profiling aid: record the given torch.cuda.Event objects at the start of
    the next calls' kernel stages and after each stage (None turns it off)."""
    global _event_handles
    lib = load_library()
    if events is None:
        _event_handles = None
        lib.rla_set_stage_events(None, 0)
        return
    for e in events:
        if not e.cuda_event:   # torch creates its event on the first record
            e.record()
    if not all(e.cuda_event for e in events):
        raise RuntimeError("could not create the HIP events")
    _event_handles = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    lib.rla_set_stage_events(ctypes.cast(_event_handles, ctypes.c_void_p), len(events))


_event_handles = None


def rla_workspace_size(problem: rla_problem, op: int) -> int:
    return int(load_library().rla_workspace_size(ctypes.byref(problem), int(op)))


# ---------------------------------------------------------------------------
# torch-side marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(dt):
    torch = _torch()
    if dt == torch.bfloat16:
        return RLA_BF16
    if dt == torch.float32:
        return RLA_F32
    raise TypeError("dtype must be bfloat16 or float32")


def make_problem(q, v, cu_seqlens=None, clip: float = 1.0, out_dtype=None,
                 flags: int = 0, decay_param=None, decay_param_grad=None) -> rla_problem:
    """rla_problem for q [B,T,H,dk] / [T,H,dk] and v, with optional cu_seqlens.
    out_dtype (dtype of o, dq, dk, dv) defaults to float32."""
    torch = _torch()
    if q.dtype == torch.bfloat16:
        dtype = RLA_BF16
    elif q.dtype == torch.float32:
        dtype = RLA_F32
    else:
        raise TypeError("q, k, v must be bfloat16 or float32")
    if q.dim() == 4:
        B, T, H, dk = q.shape
    elif q.dim() == 3:
        B, (T, H, dk) = 1, q.shape
    else:
        raise ValueError("q must be [B, T, H, d_k] or [T, H, d_k]")
    dv = v.shape[-1]
    N = 0
    if cu_seqlens is not None:
        if B != 1:
            raise ValueError("cu_seqlens requires B == 1")
        if cu_seqlens.dtype != torch.int32 or not cu_seqlens.is_cuda:
            raise TypeError("cu_seqlens must be an int32 device tensor")
        N = cu_seqlens.numel() - 1
    c = math.inf if clip is None else float(clip)
    out = _dtype_code(torch.float32 if out_dtype is None else out_dtype)
    return rla_problem(B, T, H, dk, dv, N, _ptr(cu_seqlens), dtype, c, out, flags,
                       _ptr(decay_param), _ptr(decay_param_grad))


def _check(tensors, device):
    for name, t in tensors.items():
        if t is None:
            continue
        if t.device != device:
            raise ValueError("%s must be on %s" % (name, device))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)


def _expect(name, t, shape, dtype):
    """t (if given) must have exactly this shape and dtype."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))


def _check_operands(problem, q, k, v, gates, states):
    """Shapes and dtypes of the operator's inputs against q: k like q, v with
    q's leading dimensions, fp32 gates [.., H] and fp32 states [N, H, d_k, d_v].
    The library trusts these shapes, so a mismatch must stop here."""
    torch = _torch()
    if v.dim() != q.dim() or tuple(v.shape[:-1]) != tuple(q.shape[:-1]):
        raise ValueError("v must be %s + [d_v], got %s" % (tuple(q.shape[:-1]), tuple(v.shape)))
    _expect("k", k, q.shape, q.dtype)
    _expect("v", v, v.shape, q.dtype)
    for name, t in gates.items():
        if t is None:
            raise ValueError("%s is required" % name)
        _expect(name, t, q.shape[:-1], torch.float32)
    for name, t in states.items():
        _expect(name, t, _state_shape(problem), torch.float32)


def _state_shape(problem):
    N = problem.num_seqs if problem.cu_seqlens else problem.batch
    return (N, problem.num_heads, problem.head_dim_k, problem.head_dim_v)


def _workspace(problem, op, device, workspace):
    """(workspace tensor, its size in bytes): the caller's (checked for device,
    contiguity and size) or a new uint8 tensor of rla_workspace_size bytes."""
    torch = _torch()
    need = rla_workspace_size(problem, op)
    if workspace is not None:
        if workspace.device != device:
            raise ValueError("workspace must be on %s" % device)
        if not workspace.is_contiguous():
            raise ValueError("workspace must be contiguous")
        have = workspace.numel() * workspace.element_size()
        if have < need:
            raise ValueError("workspace too small: need %d bytes" % need)
        return workspace, have
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    return ws, ws.numel()


_VARIANT_MASK = (RLA_FLAG_RESIDUAL_TANH | RLA_FLAG_UNGATED_OUTPUT | RLA_FLAG_DECAYED_RESIDUAL |
                 RLA_FLAG_QK_SILU_L2NORM | RLA_FLAG_GATE_PREACT)


def _variant_bits(variants: int) -> int:
    if variants & ~_VARIANT_MASK:
        raise ValueError("variants must combine RLA_FLAG_RESIDUAL_TANH, RLA_FLAG_UNGATED_OUTPUT, "
                         "RLA_FLAG_DECAYED_RESIDUAL, RLA_FLAG_QK_SILU_L2NORM and RLA_FLAG_GATE_PREACT")
    return int(variants)


def _check_decay_param(variants, decay_param, H, device):
    if variants & RLA_FLAG_GATE_PREACT:
        if decay_param is None:
            raise ValueError("RLA_FLAG_GATE_PREACT needs decay_param [2, H] (a then b)")
        if decay_param.numel() != 2 * H or not decay_param.is_contiguous() or \
                decay_param.device != device or decay_param.dtype != _torch().float32:
            raise ValueError("decay_param must be a contiguous float32 [2, H] tensor on %s" % device)
    return decay_param


def _forward(name, op, q, k, v, alpha_s, beta, alpha_r, gamma, clip, S0, R0, cu_seqlens,
             out, workspace, stream, return_states, out_dtype, save_for_backward, variants=0,
             decay_param=None):
    torch = _torch()
    lib = load_library()
    problem = make_problem(q, v, cu_seqlens, clip, out_dtype,
                           (RLA_FLAG_SAVE_FOR_BACKWARD if save_for_backward else 0) |
                           _variant_bits(variants),
                           _check_decay_param(variants, decay_param, q.shape[-2], q.device))
    if save_for_backward:
        op = RLA_OP_RDN_BACKWARD if op == RLA_OP_RDN_FORWARD else RLA_OP_RLA_BACKWARD
    dev = q.device
    _check(dict(q=q, k=k, v=v, alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma,
                S0=S0, R0=R0, out=out), dev)
    _check_operands(problem, q, k, v, dict(alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma),
                    dict(S0=S0, R0=R0))
    odt = torch.float32 if problem.out_dtype == RLA_F32 else torch.bfloat16
    o = torch.empty(v.shape, dtype=odt, device=dev) if out is None else out
    _expect("out", o, v.shape, odt)
    Sf = Rf = None
    if return_states:
        shape = _state_shape(problem)
        Sf = torch.empty(shape, dtype=torch.float32, device=dev)
        Rf = torch.empty(shape, dtype=torch.float32, device=dev)
    ws, ws_bytes = _workspace(problem, op, dev, workspace)
    st = getattr(lib, name)(ctypes.byref(problem), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha_s),
                            _ptr(beta), _ptr(alpha_r), _ptr(gamma), _ptr(S0), _ptr(R0), _ptr(o),
                            _ptr(Sf), _ptr(Rf), _ptr(ws), ws_bytes, _stream_handle(stream))
    if st != RLA_OK:
        raise RLAError(st, name)
    return o, Sf, Rf


def rla_forward(q, k, v, alpha_s, beta, alpha_r, gamma, clip: float = 1.0, S0=None, R0=None,
                cu_seqlens=None, out=None, workspace=None, stream=None, return_states=True,
                out_dtype=None, save_for_backward=False, variants=0, decay_param=None):
    """RLA forward (Sec. 3.4, left box).  Returns (o, S_final, R_final).
    With save_for_backward the (backward-sized) workspace keeps what the
    matching backward call with use_saved=True reads instead of recomputing.
    variants: RLA_FLAG_RESIDUAL_TANH | RLA_FLAG_UNGATED_OUTPUT |
    RLA_FLAG_DECAYED_RESIDUAL bits (include/rla.h)."""
    return _forward("rla_forward", RLA_OP_RLA_FORWARD, q, k, v, alpha_s, beta, alpha_r, gamma,
                    clip, S0, R0, cu_seqlens, out, workspace, stream, return_states, out_dtype,
                    save_for_backward, variants, decay_param)


def rdn_forward(q, k, v, alpha_s, beta, alpha_r, gamma, clip: float = 1.0, S0=None, R0=None,
                cu_seqlens=None, out=None, workspace=None, stream=None, return_states=True,
                out_dtype=None, save_for_backward=False, variants=0, decay_param=None):
    """RDN forward (Sec. 3.4, right box).  Returns (o, S_final, R_final).
    With save_for_backward the (backward-sized) workspace keeps what the
    matching backward call with use_saved=True reads instead of recomputing."""
    return _forward("rdn_forward", RLA_OP_RDN_FORWARD, q, k, v, alpha_s, beta, alpha_r, gamma,
                    clip, S0, R0, cu_seqlens, out, workspace, stream, return_states, out_dtype,
                    save_for_backward, variants, decay_param)


def rdn_forward_noalloc(q, k, v, alpha_s, beta, alpha_r, gamma, clip: float = 1.0, S0=None,
                        R0=None, cu_seqlens=None, out=None, S_final=None, R_final=None,
                        stream=None, out_dtype=None, variants=0, decay_param=None):
    """RDN forward whose workspace is the library's static per-device scratch
    array (no allocation inside the call; see include/rla.h).  The outputs
    out, S_final, R_final are the caller's (allocated here only when not
    given: pass them to keep the call allocation-free).  Returns (o, S_final,
    R_final)."""
    torch = _torch()
    lib = load_library()
    problem = make_problem(q, v, cu_seqlens, clip, out_dtype, _variant_bits(variants),
                           _check_decay_param(variants, decay_param, q.shape[-2], q.device))
    dev = q.device
    _check(dict(q=q, k=k, v=v, alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma,
                S0=S0, R0=R0, out=out, S_final=S_final, R_final=R_final), dev)
    _check_operands(problem, q, k, v, dict(alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma),
                    dict(S0=S0, R0=R0, S_final=S_final, R_final=R_final))
    odt = torch.float32 if problem.out_dtype == RLA_F32 else torch.bfloat16
    o = torch.empty(v.shape, dtype=odt, device=dev) if out is None else out
    _expect("out", o, v.shape, odt)
    shape = _state_shape(problem)
    Sf = torch.empty(shape, dtype=torch.float32, device=dev) if S_final is None else S_final
    Rf = torch.empty(shape, dtype=torch.float32, device=dev) if R_final is None else R_final
    st = lib.rdn_forward_noalloc(ctypes.byref(problem), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha_s),
                                 _ptr(beta), _ptr(alpha_r), _ptr(gamma), _ptr(S0), _ptr(R0),
                                 _ptr(o), _ptr(Sf), _ptr(Rf), _stream_handle(stream))
    if st != RLA_OK:
        raise RLAError(st, "rdn_forward_noalloc")
    return o, Sf, Rf


def _backward(name, op, q, k, v, alpha_s, beta, alpha_r, gamma, dO, clip: float = 1.0, S0=None,
                 R0=None, dS_final=None, dR_final=None, cu_seqlens=None, workspace=None,
                 stream=None, grads=None, out_dtype=None, use_saved=False, variants=0,
                 decay_param=None):
    torch = _torch()
    lib = load_library()
    if use_saved and workspace is None:
        raise ValueError("use_saved needs the workspace of the saving forward call")
    _check_decay_param(variants, decay_param, q.shape[-2], q.device)
    ddp = None
    if variants & RLA_FLAG_GATE_PREACT:
        ddp = grads.get("ddecay_param") if grads is not None else None
        if ddp is None:
            ddp = torch.empty(2, q.shape[-2], dtype=torch.float32, device=q.device)
    problem = make_problem(q, v, cu_seqlens, clip, out_dtype,
                           (RLA_FLAG_USE_SAVED if use_saved else 0) | _variant_bits(variants),
                           decay_param, ddp)
    dev = q.device
    _check(dict(q=q, k=k, v=v, alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma,
                S0=S0, R0=R0, dO=dO, dS_final=dS_final, dR_final=dR_final), dev)
    _check_operands(problem, q, k, v, dict(alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma),
                    dict(S0=S0, R0=R0, dS_final=dS_final, dR_final=dR_final))
    if dO is None:
        raise ValueError("dO is required")
    _expect("dO", dO, v.shape, q.dtype)
    odt = torch.float32 if problem.out_dtype == RLA_F32 else torch.bfloat16
    shape = _state_shape(problem)
    if grads is None:
        grads = dict(dq=torch.empty(q.shape, dtype=odt, device=dev),
                     dk=torch.empty(k.shape, dtype=odt, device=dev),
                     dv=torch.empty(v.shape, dtype=odt, device=dev),
                     dalpha_s=torch.empty_like(alpha_s), dbeta=torch.empty_like(beta),
                     dalpha_r=torch.empty_like(alpha_r), dgamma=torch.empty_like(gamma),
                     dS0=torch.empty(shape, dtype=torch.float32, device=dev),
                     dR0=torch.empty(shape, dtype=torch.float32, device=dev))
    else:   # caller-supplied gradient buffers: every one is written by the library
        for key in ("dq", "dk", "dv", "dalpha_s", "dbeta", "dalpha_r", "dgamma"):
            if grads.get(key) is None:
                raise ValueError("grads[%r] is required" % key)
    _check({"grads[%s]" % key: t for key, t in grads.items()}, dev)
    gshape = dict(dq=(q.shape, odt), dk=(q.shape, odt), dv=(v.shape, odt),
                  dalpha_s=(q.shape[:-1], torch.float32), dbeta=(q.shape[:-1], torch.float32),
                  dalpha_r=(q.shape[:-1], torch.float32), dgamma=(q.shape[:-1], torch.float32),
                  dS0=(shape, torch.float32), dR0=(shape, torch.float32),
                  ddecay_param=((2, q.shape[-2]), torch.float32))
    for key, t in grads.items():
        if key not in gshape:
            raise ValueError("unknown gradient %r" % key)
        _expect("grads[%s]" % key, t, *gshape[key])
    if ddp is not None:
        grads["ddecay_param"] = ddp
    ws, ws_bytes = _workspace(problem, op, dev, workspace)
    g = grads
    st = getattr(lib, name)(ctypes.byref(problem), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha_s),
                          _ptr(beta), _ptr(alpha_r), _ptr(gamma), _ptr(S0), _ptr(R0), _ptr(dO),
                          _ptr(dS_final), _ptr(dR_final), _ptr(g["dq"]), _ptr(g["dk"]),
                          _ptr(g["dv"]), _ptr(g["dalpha_s"]), _ptr(g["dbeta"]),
                          _ptr(g["dalpha_r"]), _ptr(g["dgamma"]), _ptr(g.get("dS0")),
                          _ptr(g.get("dR0")), _ptr(ws), ws_bytes, _stream_handle(stream))
    if st != RLA_OK:
        raise RLAError(st, name)
    return g


def rdn_backward(q, k, v, alpha_s, beta, alpha_r, gamma, dO, clip: float = 1.0, S0=None,
                 R0=None, dS_final=None, dR_final=None, cu_seqlens=None, workspace=None,
                 stream=None, grads=None, out_dtype=None, use_saved=False, variants=0,
                 decay_param=None):
    """Gradients of <dO,o> + <dS_final,S_T> + <dR_final,R_T> for rdn_forward.
    Returns a dict dq, dk, dv, dalpha_s, dbeta, dalpha_r, dgamma, dS0, dR0.
    use_saved: read what rdn_forward(save_for_backward=True) left in `workspace`."""
    return _backward("rdn_backward", RLA_OP_RDN_BACKWARD, q, k, v, alpha_s, beta, alpha_r, gamma,
                     dO, clip, S0, R0, dS_final, dR_final, cu_seqlens, workspace, stream, grads,
                     out_dtype, use_saved, variants, decay_param)


def rla_backward(q, k, v, alpha_s, beta, alpha_r, gamma, dO, clip: float = 1.0, S0=None,
                 R0=None, dS_final=None, dR_final=None, cu_seqlens=None, workspace=None,
                 stream=None, grads=None, out_dtype=None, use_saved=False, variants=0,
                 decay_param=None):
    """Gradients of <dO,o> + <dS_final,S_T> + <dR_final,R_T> for rla_forward."""
    return _backward("rla_backward", RLA_OP_RLA_BACKWARD, q, k, v, alpha_s, beta, alpha_r, gamma,
                     dO, clip, S0, R0, dS_final, dR_final, cu_seqlens, workspace, stream, grads,
                     out_dtype, use_saved, variants, decay_param)


def _decode(name, q, k, v, alpha_s, beta, alpha_r, gamma, clip, S_in, R_in, S_out, R_out, out,
            stream, out_dtype, variants=0, decay_param=None):
    torch = _torch()
    lib = load_library()
    if q.dim() != 4:
        raise ValueError("decoding takes q, k, v as [B, T, H, d] (T tokens per sequence)")
    problem = make_problem(q, v, None, clip, out_dtype, _variant_bits(variants),
                           _check_decay_param(variants, decay_param, q.shape[-2], q.device))
    dev = q.device
    _check(dict(q=q, k=k, v=v, alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma,
                S_in=S_in, R_in=R_in, S_out=S_out, R_out=R_out, out=out), dev)
    _check_operands(problem, q, k, v, dict(alpha_s=alpha_s, beta=beta, alpha_r=alpha_r, gamma=gamma),
                    dict(S_in=S_in, R_in=R_in, S_out=S_out, R_out=R_out))
    shape = (problem.batch, problem.num_heads, problem.head_dim_k, problem.head_dim_v)
    if S_out is None:
        S_out = torch.empty(shape, dtype=torch.float32, device=dev)
    if R_out is None:
        R_out = torch.empty(shape, dtype=torch.float32, device=dev)
    odt = torch.float32 if problem.out_dtype == RLA_F32 else torch.bfloat16
    o = torch.empty(v.shape, dtype=odt, device=dev) if out is None else out
    _expect("out", o, v.shape, odt)
    st = getattr(lib, name)(ctypes.byref(problem), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha_s),
                            _ptr(beta), _ptr(alpha_r), _ptr(gamma), _ptr(S_in), _ptr(R_in),
                            _ptr(o), _ptr(S_out), _ptr(R_out), _stream_handle(stream))
    if st != RLA_OK:
        raise RLAError(st, name)
    return o, S_out, R_out


def rla_decode(q, k, v, alpha_s, beta, alpha_r, gamma, clip: float = 1.0, S_in=None, R_in=None,
               S_out=None, R_out=None, out=None, stream=None, out_dtype=None, variants=0,
               decay_param=None):
    """RLA recurrent step (Sec. 3.4, left box, evaluated token by token):
    q, k, v [B, T, H, d] with small T, gates [B, T, H].  Returns (o, S_out,
    R_out); pass S_out=S_in, R_out=R_in to update the states in place."""
    return _decode("rla_decode", q, k, v, alpha_s, beta, alpha_r, gamma, clip, S_in, R_in,
                   S_out, R_out, out, stream, out_dtype, variants, decay_param)


def rdn_decode(q, k, v, alpha_s, beta, alpha_r, gamma, clip: float = 1.0, S_in=None, R_in=None,
               S_out=None, R_out=None, out=None, stream=None, out_dtype=None, variants=0,
               decay_param=None):
    """RDN recurrent step (Sec. 3.4, right box); arguments as rla_decode."""
    return _decode("rdn_decode", q, k, v, alpha_s, beta, alpha_r, gamma, clip, S_in, R_in,
                   S_out, R_out, out, stream, out_dtype, variants, decay_param)
