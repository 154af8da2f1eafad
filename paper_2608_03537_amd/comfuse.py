"""Thin Python binding of libcomfuse (ctypes).

Argument marshalling only: every step of every operator runs in the HIP
kernels of ``libcomfuse.so``.  torch supplies device memory and streams.
If the library is missing, every call raises — there is no fallback path.

The raw entry points keep the C names (``cf_gemm_postnorm`` ...) and take the
ctypes structures below; the ``gemm_postnorm`` / ``gemm_subgraph`` / ``b2b_*``
/ ``gemm`` / ``rowop`` helpers build those structures from torch tensors and
allocate the outputs.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcomfuse.so")

# ---------------------------------------------------------------- enums
CF_F32, CF_BF16, CF_FP8_E4M3 = 0, 1, 2
CF_LAYOUT_KN, CF_LAYOUT_NK = 0, 1
(CF_N_SCALE, CF_N_BIAS, CF_N_RESIDUAL, CF_N_LAYERNORM, CF_N_RMSNORM, CF_N_GELU,
 CF_N_GELU_TANH, CF_N_RELU, CF_N_STORE, CF_N_ROWAMAX_QUANT, CF_N_SOFTMAX, CF_N_SOFTCAP) = range(12)
CF_MID_GELU_BIAS, CF_MID_SOFTMAX, CF_MID_RELU_BIAS = 0, 1, 2
CF_OUT_STORE, CF_OUT_BIAS_RESIDUAL_LN, CF_OUT_BIAS_RELU = 0, 1, 2
PATH_AUTO, PATH_WHOLE_ROW, PATH_CLUSTER, PATH_SPLIT = 0, 1, 2, 3
CF_B2B_WS_HEADER_BYTES = 1 << 20   # split-MLP arrival counters at the start of its workspace
STATUS = {0: "CF_OK", 1: "CF_ERR_NULL", 2: "CF_ERR_SHAPE", 3: "CF_ERR_LD", 4: "CF_ERR_ALIGN",
          5: "CF_ERR_DTYPE", 6: "CF_ERR_WORKSPACE", 7: "CF_ERR_UNSUPPORTED", 8: "CF_ERR_ALIAS",
          9: "CF_ERR_HIP", 10: "CF_ERR_STRUCT", 11: "CF_ERR_PEER_TIMEOUT"}

vp, i64, f32p = C.c_void_p, C.c_int64, C.POINTER(C.c_float)


class PostnormArgs(C.Structure):
    _fields_ = [("struct_size", C.c_size_t), ("M", i64), ("N", i64), ("K", i64),
                ("in_dtype", C.c_int), ("out_dtype", C.c_int),
                ("X", vp), ("ldx", i64), ("W", vp), ("ldw", i64), ("w_layout", C.c_int),
                ("bias", vp), ("R", vp), ("ldr", i64), ("gamma", vp), ("beta", vp),
                ("alpha", C.c_float), ("eps", C.c_float), ("Y", vp), ("ldy", i64), ("path", C.c_int)]


class Node(C.Structure):
    _fields_ = [("kind", C.c_int), ("inp", vp), ("out", vp), ("out2", vp), ("ld", i64),
                ("dtype", C.c_int), ("v0", vp), ("v1", vp), ("f0", C.c_float)]


class SubgraphArgs(C.Structure):
    _fields_ = [("struct_size", C.c_size_t), ("M", i64), ("N", i64), ("K", i64), ("in_dtype", C.c_int),
                ("X", vp), ("ldx", i64), ("W", vp), ("ldw", i64), ("w_layout", C.c_int),
                ("nodes", C.POINTER(Node)), ("n_nodes", C.c_int), ("path", C.c_int)]


class B2BArgs(C.Structure):
    _fields_ = [("struct_size", C.c_size_t), ("batch", i64), ("M", i64), ("K", i64), ("N1", i64), ("N2", i64),
                ("dtype", C.c_int),
                ("X", vp), ("ldx", i64), ("sx", i64),
                ("W1", vp), ("ldw1", i64), ("sw1", i64), ("w1_layout", C.c_int), ("b1", vp),
                ("mid", C.c_int), ("mid_scale", C.c_float),
                ("W2", vp), ("ldw2", i64), ("sw2", i64), ("w2_layout", C.c_int),
                ("out", C.c_int), ("b2", vp), ("R", vp), ("ldr", i64), ("sr", i64),
                ("gamma", vp), ("beta", vp), ("eps", C.c_float),
                ("O", vp), ("ldo", i64), ("so", i64)]


class CfError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {detail}")


_lib = None
_lib_lock = threading.Lock()


def lib():
    """Load libcomfuse.so from the package directory (raises if missing)."""
    global _lib
    if _lib is None:
        with _lib_lock:
            if _lib is None:
                if not os.path.exists(LIB_PATH):
                    raise RuntimeError(f"libcomfuse.so not built ({LIB_PATH}); run paper_2608_03537_amd/build.py")
                L = C.CDLL(LIB_PATH)
                L.cf_version.restype = C.c_int
                L.cf_last_error.restype = C.c_char_p
                L.cf_status_string.restype = C.c_char_p
                L.cf_status_string.argtypes = [C.c_int]
                for name, argt in [("cf_gemm_postnorm", C.POINTER(PostnormArgs)),
                                   ("cf_gemm_subgraph", C.POINTER(SubgraphArgs)),
                                   ("cf_b2bgemm", C.POINTER(B2BArgs))]:
                    f = getattr(L, name)
                    f.restype = C.c_int
                    f.argtypes = [argt, vp, C.c_size_t, vp]
                    w = getattr(L, name.replace("cf_b2bgemm", "cf_b2bgemm") + "_workspace")
                    w.restype = C.c_size_t
                    w.argtypes = [argt]
                L.cf_gemm.restype = C.c_int
                L.cf_gemm.argtypes = [i64, i64, i64, i64, C.c_int, C.c_int, vp, i64, i64, vp, i64, i64,
                                      C.c_int, vp, C.c_float, vp, i64, i64, vp]
                L.cf_rowop.restype = C.c_int
                L.cf_rowop.argtypes = [i64, i64, i64, C.c_int, vp, i64, i64, C.POINTER(Node), C.c_int, vp]
                L.cf_gemm_subgraph_noalloc.restype = C.c_int
                L.cf_gemm_subgraph_noalloc.argtypes = [C.POINTER(SubgraphArgs), vp]
                L.cf_workspace_check.restype = C.c_int
                L.cf_workspace_check.argtypes = [vp, C.c_size_t, vp]
                _lib = L
    return _lib


def _check(status):
    if status != 0:
        raise CfError(status, lib().cf_last_error().decode())


# ---------------------------------------------------------------- raw C names
def cf_version():
    return lib().cf_version()


def cf_gemm_postnorm(args, workspace, ws_bytes, stream):
    return lib().cf_gemm_postnorm(C.byref(args), workspace, ws_bytes, stream)


def cf_gemm_postnorm_workspace(args):
    return lib().cf_gemm_postnorm_workspace(C.byref(args))


def cf_gemm_subgraph(args, workspace, ws_bytes, stream):
    return lib().cf_gemm_subgraph(C.byref(args), workspace, ws_bytes, stream)


def cf_gemm_subgraph_workspace(args):
    return lib().cf_gemm_subgraph_workspace(C.byref(args))


def cf_gemm_subgraph_noalloc(args, stream):
    return lib().cf_gemm_subgraph_noalloc(C.byref(args), stream)


def cf_b2bgemm(args, workspace, ws_bytes, stream):
    return lib().cf_b2bgemm(C.byref(args), workspace, ws_bytes, stream)


def cf_b2bgemm_workspace(args):
    return lib().cf_b2bgemm_workspace(C.byref(args))


def cf_gemm(*args):
    return lib().cf_gemm(*args)


def cf_rowop(batch, M, N, dtype, P, ldp, sp, nodes, n_nodes, stream):
    return lib().cf_rowop(batch, M, N, dtype, P, ldp, sp, nodes, n_nodes, stream)


def cf_workspace_check(workspace, ws_bytes, stream):
    return lib().cf_workspace_check(workspace, ws_bytes, stream)


def cf_status_string(s):
    return lib().cf_status_string(s).decode()


def cf_last_error():
    return lib().cf_last_error().decode()


# ---------------------------------------------------------------- torch helpers
def _torch():
    import torch
    return torch


def _dt(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return CF_F32
    if t.dtype == torch.bfloat16:
        return CF_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return None if t is None else t.data_ptr()


def _ld(t):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.stride(0)


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


_ws_cache: dict = {}


def _capturing():
    return _torch().cuda.is_current_stream_capturing()


def workspace(nbytes, device, stream=None, kind="rows"):
    """A zero-initialised workspace of at least nbytes on ``device``, cached per
    (device, stream, kind): calls on one stream run in order, so they may
    share it; calls on different streams get different workspaces (the
    row-cluster round counters live in it).  kind "b2b" is the split MLP's
    (its arrival counters must not meet another entry point's data)."""
    torch = _torch()
    if nbytes == 0:
        return None
    key = (str(device), _stream(stream), kind)
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.zeros(max(nbytes, 1 << 20), dtype=torch.uint8, device=device)
        _ws_cache[key] = ws
    return ws


def check_workspace(ws, stream=None):
    """Raise CfError(CF_ERR_PEER_TIMEOUT) if a row-cluster wait gave up since
    the last check of ``ws`` (synchronises the stream; clears the word)."""
    if ws is not None:
        _check(cf_workspace_check(_ptr(ws), ws.numel(), _stream(stream)))


def _after_call(ws, need, stream, check):
    # The error word exists only when the plan used a workspace; checking
    # synchronises, so it is skipped while a graph is being captured (the
    # caller then checks after replaying, with check_workspace).
    if check and need > 0 and not _capturing():
        check_workspace(ws, stream)


def postnorm_args(X, W, bias=None, R=None, gamma=None, beta=None, Y=None, *, w_layout=CF_LAYOUT_NK,
                  alpha=1.0, eps=1e-5, path=PATH_AUTO):
    M, K = X.shape
    N = W.shape[0] if w_layout == CF_LAYOUT_NK else W.shape[1]
    a = PostnormArgs()
    a.struct_size = C.sizeof(PostnormArgs)
    a.M, a.N, a.K = M, N, K
    a.in_dtype = _dt(X)
    a.out_dtype = _dt(Y)
    a.X, a.ldx = _ptr(X), _ld(X)
    a.W, a.ldw, a.w_layout = _ptr(W), _ld(W), w_layout
    a.bias, a.gamma, a.beta = _ptr(bias), _ptr(gamma), _ptr(beta)
    a.R, a.ldr = _ptr(R), (_ld(R) if R is not None else 0)
    a.alpha, a.eps = alpha, eps
    a.Y, a.ldy = _ptr(Y), _ld(Y)
    a.path = path
    return a


def gemm_postnorm(X, W, bias=None, R=None, gamma=None, beta=None, *, w_layout=CF_LAYOUT_NK, alpha=1.0,
                  eps=1e-5, out_dtype=None, path=PATH_AUTO, out=None, ws=None, stream=None, check=True):
    """Y = LayerNorm(alpha * X.W + bias + R) * gamma + beta, fused.

    check=True reads the workspace's error word after the call (a stream
    synchronisation) and raises if a row-cluster wait gave up; pass
    check=False to keep the call asynchronous and use check_workspace later.
    """
    torch = _torch()
    M = X.shape[0]
    N = W.shape[0] if w_layout == CF_LAYOUT_NK else W.shape[1]
    Y = out if out is not None else torch.empty((M, N), dtype=out_dtype or X.dtype, device=X.device)
    a = postnorm_args(X, W, bias, R, gamma, beta, Y, w_layout=w_layout, alpha=alpha, eps=eps, path=path)
    need = cf_gemm_postnorm_workspace(a)
    if ws is None:
        ws = workspace(need, X.device, stream)
    _check(cf_gemm_postnorm(a, _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))
    _after_call(ws, need, stream, check)
    return Y


def make_nodes(spec):
    """spec: list of dicts {kind, in, out, out2, ld, dtype, v0, v1, f0} (tensors allowed)."""
    arr = (Node * len(spec))()
    for i, d in enumerate(spec):
        n = arr[i]
        n.kind = d["kind"]
        for src, dst in (("in", "inp"), ("out", "out"), ("out2", "out2"), ("v0", "v0"), ("v1", "v1")):
            v = d.get(src)
            setattr(n, dst, v.data_ptr() if hasattr(v, "data_ptr") else v)
        n.ld = d.get("ld", 0)
        n.dtype = d.get("dtype", CF_F32)
        n.f0 = d.get("f0", 0.0)
    return arr


def subgraph_args(X, W, nodes, *, w_layout=CF_LAYOUT_NK, path=PATH_AUTO):
    M, K = X.shape
    N = W.shape[0] if w_layout == CF_LAYOUT_NK else W.shape[1]
    a = SubgraphArgs()
    a.struct_size = C.sizeof(SubgraphArgs)
    a.M, a.N, a.K = M, N, K
    a.in_dtype = _dt(X)
    a.X, a.ldx = _ptr(X), _ld(X)
    a.W, a.ldw, a.w_layout = _ptr(W), _ld(W), w_layout
    a.nodes, a.n_nodes = nodes, len(nodes)
    a.path = path
    return a


def gemm_subgraph(X, W, spec, *, w_layout=CF_LAYOUT_NK, path=PATH_AUTO, ws=None, stream=None, check=True):
    """Run X.W followed by the node list ``spec`` (outputs are given in spec).
    ``check`` as in gemm_postnorm."""
    nodes = make_nodes(spec)
    a = subgraph_args(X, W, nodes, w_layout=w_layout, path=path)
    need = cf_gemm_subgraph_workspace(a)
    if ws is None:
        ws = workspace(need, X.device, stream)
    _check(cf_gemm_subgraph(a, _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))
    _after_call(ws, need, stream, check)


def gemm_subgraph_noalloc(X, W, spec, *, w_layout=CF_LAYOUT_NK, path=PATH_AUTO, stream=None):
    """gemm_subgraph without a workspace: the library's own per-GPU scratch
    array serves the split path (no allocation anywhere; calls on one GPU
    must not overlap)."""
    nodes = make_nodes(spec)
    a = subgraph_args(X, W, nodes, w_layout=w_layout, path=path)
    _check(cf_gemm_subgraph_noalloc(a, _stream(stream)))


def ln_gelu_amax(X, W, bias=None, R=None, *, eps=1e-5, qmax=448.0, z_dtype=None, quant_codes=True,
                 w_layout=CF_LAYOUT_NK, path=PATH_AUTO, ws=None, stream=None, gelu=CF_N_GELU, check=True):
    """Z = GELU(LN(X.W + b + R)); s = rowmax|Z| / qmax; Q = e4m3(Z / s).  Returns (Z, s, Q)."""
    torch = _torch()
    M = X.shape[0]
    N = W.shape[0] if w_layout == CF_LAYOUT_NK else W.shape[1]
    Z = torch.empty((M, N), dtype=z_dtype or X.dtype, device=X.device)
    s = torch.empty((M,), dtype=torch.float32, device=X.device)
    Q = torch.empty((M, N), dtype=torch.uint8, device=X.device) if quant_codes else None
    spec = []
    if bias is not None:
        spec.append(dict(kind=CF_N_BIAS, v0=bias))
    if R is not None:
        spec.append(dict(kind=CF_N_RESIDUAL, **{"in": R}, ld=_ld(R), dtype=_dt(R)))
    spec += [dict(kind=CF_N_LAYERNORM, f0=eps), dict(kind=gelu),
             dict(kind=CF_N_STORE, out=Z, ld=_ld(Z), dtype=_dt(Z)),
             dict(kind=CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=(N if Q is None else _ld(Q)), f0=qmax)]
    gemm_subgraph(X, W, spec, w_layout=w_layout, path=path, ws=ws, stream=stream, check=check)
    return Z, s, Q


def gemm(A, B, *, b_layout=CF_LAYOUT_NK, bias=None, alpha=1.0, out_dtype=None, out=None, stream=None):
    """C = alpha * A.B (+ bias).  A: [M,K] or [b,M,K]; B: [N,K] (NK) or [K,N] (KN), optionally batched."""
    torch = _torch()
    batched = A.dim() == 3
    A3 = A if batched else A.unsqueeze(0)
    B3 = B if B.dim() == 3 else B.unsqueeze(0)
    nb, M, K = A3.shape
    N = B3.shape[1] if b_layout == CF_LAYOUT_NK else B3.shape[2]
    Cm = out if out is not None else torch.empty((nb, M, N), dtype=out_dtype or A.dtype, device=A.device)
    C3 = Cm if Cm.dim() == 3 else Cm.unsqueeze(0)
    sb = B3.stride(0) if B3.shape[0] > 1 else 0
    _check(cf_gemm(nb, M, N, K, _dt(A3), _dt(C3), _ptr(A3), A3.stride(1), A3.stride(0), _ptr(B3), B3.stride(1), sb,
                   b_layout, _ptr(bias), alpha, _ptr(C3), C3.stride(1), C3.stride(0), _stream(stream)))
    return Cm if (batched or out is not None) else Cm[0]


def rowop(P, spec, stream=None):
    """Run a node list over the rows of a materialised matrix P (unfused).

    P is [M, N] or a batch [b, M, N] (any batch stride, unit column stride);
    the node list's matrices then hold the b * M rows one after another."""
    nodes = make_nodes(spec)
    if P.dim() == 3:
        nb, M, N = P.shape
        if P.stride(2) != 1:
            raise ValueError("expected a unit column stride")
        ldp, sp = P.stride(1), P.stride(0)
    else:
        nb, (M, N) = 1, P.shape
        ldp, sp = _ld(P), 0
    _check(cf_rowop(nb, M, N, _dt(P), _ptr(P), ldp, sp, nodes, len(nodes), _stream(stream)))


def _stack(t, batch=None):
    """(batch, rows, cols, ld, batch stride) of a [rows, cols] or [batch, rows,
    cols] operand with unit column stride.  A 2-D operand beside batched ones
    is shared by every batch entry (stride 0)."""
    if t.dim() == 2:
        return (batch or 1), t.shape[0], t.shape[1], _ld(t), 0
    if t.dim() != 3 or t.stride(2) != 1:
        raise ValueError("expected a 2-D or 3-D tensor with unit column stride")
    if batch is not None and t.shape[0] != batch:
        raise ValueError(f"batch {t.shape[0]} != {batch}")
    return t.shape[0], t.shape[1], t.shape[2], t.stride(1), t.stride(0)


def _b2b_args(**kw):
    a = B2BArgs()
    a.struct_size = C.sizeof(B2BArgs)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def b2b_ffn(X, W1t, b1, W2t, b2=None, R=None, gamma=None, beta=None, *, eps=1e-5, layernorm=True, out=None,
            stream=None):
    """Fused FFN block O = LN(GELU(X W1 + b1) W2 + b2 + R) * gamma + beta.

    X [M, K] bf16; W1t = W1^T [N1, K]; W2t = W2^T [N2, N1]; R [M, N2] (pass X
    for the residual FFN block).  With layernorm=False, O = S W2 (+ b2 + R).
    Batched: X [B, M, K] (and R, out [B, M, N2]); a 3-D weight holds one
    matrix per batch entry, a 2-D one is shared; vectors are shared.
    """
    torch = _torch()
    B, M, K, ldx, sx = _stack(X)
    B = B if X.dim() == 3 else None
    _, N1, _, ldw1, sw1 = _stack(W1t, B)
    _, N2, _, ldw2, sw2 = _stack(W2t, B)
    shape = (M, N2) if B is None else (B, M, N2)
    O = out if out is not None else torch.empty(shape, dtype=torch.bfloat16, device=X.device)
    _, _, _, ldo, so = _stack(O, B)
    ldr, sr = _stack(R, B)[3:] if R is not None else (0, 0)
    a = _b2b_args(batch=B or 1, M=M, K=K, N1=N1, N2=N2, dtype=CF_BF16,
                  X=_ptr(X), ldx=ldx, sx=sx, W1=_ptr(W1t), ldw1=ldw1, sw1=sw1, w1_layout=CF_LAYOUT_NK,
                  b1=_ptr(b1), mid=CF_MID_GELU_BIAS, mid_scale=1.0,
                  W2=_ptr(W2t), ldw2=ldw2, sw2=sw2, w2_layout=CF_LAYOUT_NK,
                  out=CF_OUT_BIAS_RESIDUAL_LN if layernorm else CF_OUT_STORE, b2=_ptr(b2),
                  R=_ptr(R), ldr=ldr, sr=sr,
                  gamma=_ptr(gamma), beta=_ptr(beta), eps=eps, O=_ptr(O), ldo=ldo, so=so)
    _check(cf_b2bgemm(a, None, 0, _stream(stream)))
    return O


def b2b_mlp(X, W1t, b1, W2t, b2=None, *, out_relu=False, out=None, ws=None, stream=None):
    """Fused MLP block O = ReLU(X W1 + b1) W2 + b2 (ReLU(O) with out_relu), the
    DLRM bottom-MLP pattern.  X [M, K] bf16; W1t = W1^T [N1, K]; W2t = W2^T
    [N2, N1]; hidden units in chunks of 256, split over workgroups and summed
    through the workspace while that grid fits 256 workgroups, else all run
    by one workgroup per 128-row block.  Batched as b2b_ffn: X, out [B, M, .],
    weights 3-D (per entry) or 2-D (shared)."""
    torch = _torch()
    B, M, K, ldx, sx = _stack(X)
    B = B if X.dim() == 3 else None
    _, N1, _, ldw1, sw1 = _stack(W1t, B)
    _, N2, _, ldw2, sw2 = _stack(W2t, B)
    shape = (M, N2) if B is None else (B, M, N2)
    O = out if out is not None else torch.empty(shape, dtype=torch.bfloat16, device=X.device)
    _, _, _, ldo, so = _stack(O, B)
    a = _b2b_args(batch=B or 1, M=M, K=K, N1=N1, N2=N2, dtype=CF_BF16,
                  X=_ptr(X), ldx=ldx, sx=sx, W1=_ptr(W1t), ldw1=ldw1, sw1=sw1, w1_layout=CF_LAYOUT_NK,
                  b1=_ptr(b1), mid=CF_MID_RELU_BIAS, mid_scale=1.0,
                  W2=_ptr(W2t), ldw2=ldw2, sw2=sw2, w2_layout=CF_LAYOUT_NK,
                  out=CF_OUT_BIAS_RELU if out_relu else CF_OUT_STORE, b2=_ptr(b2),
                  R=None, ldr=0, sr=0, gamma=None, beta=None, eps=0.0, O=_ptr(O), ldo=ldo, so=so)
    need = cf_b2bgemm_workspace(a)
    if ws is None:
        ws = workspace(need, X.device, stream, kind="b2b")
    _check(cf_b2bgemm(a, _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))
    return O


def b2b_attention(Q, K, V, scale=None, out=None, stream=None):
    """O = softmax(scale * Q K^T) V for Q [B, H, Lq, d], K, V [B, H, Lk, d] (bf16, contiguous)."""
    torch = _torch()
    B, H, Lq, d = Q.shape
    Lk = K.shape[2]
    if scale is None:
        scale = d ** -0.5
    for t in (Q, K, V):
        if not t.is_contiguous():
            raise ValueError("attention operands must be contiguous [B, H, L, d]")
    O = out if out is not None else torch.empty((B, H, Lq, d), dtype=torch.bfloat16, device=Q.device)
    a = _b2b_args(batch=B * H, M=Lq, K=d, N1=Lk, N2=d, dtype=CF_BF16,
                  X=_ptr(Q), ldx=d, sx=Lq * d, W1=_ptr(K), ldw1=d, sw1=Lk * d, w1_layout=CF_LAYOUT_NK,
                  b1=None, mid=CF_MID_SOFTMAX, mid_scale=scale,
                  W2=_ptr(V), ldw2=d, sw2=Lk * d, w2_layout=CF_LAYOUT_KN,
                  out=CF_OUT_STORE, b2=None, R=None, ldr=0, sr=0, gamma=None, beta=None, eps=0.0,
                  O=_ptr(O), ldo=d, so=Lq * d)
    _check(cf_b2bgemm(a, None, 0, _stream(stream)))
    return O
