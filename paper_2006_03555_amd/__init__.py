"""FAVOR attention (arXiv 2006.03555) on AMD MI355X: Python binding of libfavor.

Every function here only marshals arguments for the C ABI declared in
``include/favor.h`` (device pointers, sizes, the current HIP stream); all
arithmetic runs in the library's HIP kernels. PyTorch provides device memory
and streams. If ``libfavor.so`` has not been built the calls raise
``FavorLibraryMissing``; there is no fallback.

Tensors: Q, K, V [B, H, L, d] (bfloat16 or float32, contiguous, on the GPU);
W [H, M, d] float32 and b [H, M] float32 from ``orf_draw``.

Keyword options of the feature and attention calls: kernel (KERNEL_SOFTMAX, the
Gaussian-kernel features of softmax attention, or KERNEL_RELU, generalized
attention with ReLU features), renormalize (False returns Q' K'^T V without the
division by D-hat) and kernel_eps (added to every ReLU feature). The attention
calls take row_scale (a [B, H, L] float32 tensor) to save each row's
1 / (D-hat + eps) for the backward calls, which then skip recomputing it.
"""
import ctypes
import functools
import os

from ._lib import (  # noqa: F401
    BF16, F32, RF_IID, RF_ORTHO_CHI, RF_ORTHO_FIXED, RF_HADAMARD, RF_GIVENS, OP_BIDIR, OP_BOTH, OP_CAUSAL, OP_FEATURE_MAP,
    OP_BIDIR_BACKWARD, OP_CAUSAL_BACKWARD, OP_BOTH_BACKWARD, KERNEL_RELU, KERNEL_SOFTMAX, backward_workspace_size,
    FavorDesc, FavorError, FavorLibraryMissing, lib, lib_path, make_desc, status_string,
    validate_desc, workspace_size, last_error, timing_enable, timing_reset, timing_read,
)

__all__ = [
    "orf_draw", "feature_map", "attn_bidir", "attn_causal", "attn_both", "workspace_size",
    "attn_bidir_backward", "attn_causal_backward", "attn_both_backward",
    "backward_workspace_size", "make_desc",
    "attn_both_noalloc", "noalloc_scratch_bytes",
    "validate_desc", "FavorError", "FavorLibraryMissing", "lib", "lib_path",
]


def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t == torch.bfloat16:
        return BF16
    if t == torch.float32:
        return F32
    raise FavorError(1, f"unsupported tensor dtype {t}; use bfloat16 or float32")


def _torch_dtype(code):
    torch = _torch()
    return torch.bfloat16 if code == BF16 else torch.float32


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _on_stream(fn):
    """Run fn with the caller's stream (keyword `stream`) as torch's current
    stream, so that the outputs and the temporary workspace fn allocates belong
    to the stream the kernels run on: the caching allocator then hands a freed
    workspace block only to later work on that same stream, never to another
    stream while the kernels may still use it."""
    @functools.wraps(fn)
    def wrapper(*args, stream=None, **kw):
        # entering a stream context costs microseconds of host time per call:
        # skip it when the caller's stream already is the current one
        if stream is None or stream == _torch().cuda.current_stream():
            return fn(*args, stream=stream, **kw)
        with _torch().cuda.stream(stream):
            return fn(*args, stream=stream, **kw)
    return wrapper


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _check(status):
    if status != 0:
        raise FavorError(status, last_error())


def _require_cuda(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise FavorError(1, "tensors must be contiguous GPU tensors")


@_on_stream
def orf_draw(seed, n_heads, M, d=64, kind=RF_ORTHO_CHI, W=None, b=None, stream=None):
    """Draw W [n_heads, M, d] and b [n_heads, M] on the GPU (favor_orf_draw)."""
    torch = _torch()
    if W is None or b is None:
        dev = torch.device("cuda", torch.cuda.current_device())
    if W is None:
        W = torch.empty((n_heads, M, d), dtype=torch.float32, device=dev)
    if b is None:
        b = torch.empty((n_heads, M), dtype=torch.float32, device=dev)
    _require_features(W, b, n_heads, M, d)
    _require_cuda(W, b)
    _check(lib().favor_orf_draw(ctypes.c_uint64(seed), n_heads, M, d, kind, _ptr(W), _ptr(b),
                                _stream(stream)))
    return W, b


def _require_like(t, shape, dtype, name):
    """A caller-supplied tensor must have exactly the shape and dtype the call
    writes or reads (the kernels trust the descriptor, not the tensor)."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise FavorError(1, f"{name} must be {tuple(shape)} {dtype}, got {tuple(t.shape)} "
                            f"{t.dtype}")


def _require_features(W, b, H, M, d):
    torch = _torch()
    _require_like(W, (H, M, d), torch.float32, "W")
    _require_like(b, (H, M), torch.float32, "b")


def _desc_for(X, W, input_scale, out_dtype, denom_eps=0.0, segment=0, others=(), opts=None):
    """Descriptor for inputs X [B, H, L, d] (and tensors `others` of the same shape
    and dtype) with features W [H, M, d], b [H, M]."""
    if X.dim() != 4:
        raise FavorError(1, f"inputs must be [B, H, L, d], got {tuple(X.shape)}")
    B, H, L, d = X.shape
    for name, t in others:
        _require_like(t, X.shape, X.dtype, name)
    if W.dim() != 3:
        raise FavorError(1, f"W must be [H, M, d], got {tuple(W.shape)}")
    M = W.shape[1]
    in_code = _dtype_code(X.dtype)
    out_code = in_code if out_dtype is None else _dtype_code(out_dtype)
    return make_desc(B, H, L, d, M, in_code, out_code, input_scale, denom_eps, segment,
                     **(opts or {}))


def _opts(kernel, renormalize, kernel_eps):
    return dict(kernel=kernel, renormalize=renormalize, kernel_eps=kernel_eps)


def _out_dtype(out_dtype, out, X):
    """Output dtype: as given, else that of a supplied output tensor, else X's."""
    if out_dtype is not None:
        return out_dtype
    return out.dtype if out is not None else X.dtype


@_on_stream
def feature_map(X, W, b, input_scale, out_dtype=None, out=None, stream=None,
                kernel=KERNEL_SOFTMAX, kernel_eps=1e-3):
    """X' [B, H, L, M] (favor_feature_map): D_X X-hat, or the ReLU features."""
    torch = _torch()
    g = _desc_for(X, W, input_scale, _out_dtype(out_dtype, out, X),
                  opts=_opts(kernel, True, kernel_eps))
    _require_features(W, b, g.H, g.M, g.d)
    shape = (g.B, g.H, g.L, g.M)
    if out is None:
        out = torch.empty(shape, dtype=_torch_dtype(g.out_dtype), device=X.device)
    _require_like(out, shape, _torch_dtype(g.out_dtype), "out")
    _require_cuda(X, W, b, out)
    _check(lib().favor_feature_map(ctypes.byref(g), _ptr(X), _ptr(W), _ptr(b), _ptr(out),
                                   _stream(stream)))
    return out


def _workspace(g, causal, workspace):
    torch = _torch()
    n = workspace_size(g, causal)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8,
                                device=torch.device("cuda", torch.cuda.current_device()))
    return workspace, workspace.numel() * workspace.element_size()


def _require_row_scale(t, g, name):
    torch = _torch()
    _require_like(t, (g.B, g.H, g.L), torch.float32, name)


@_on_stream
def attn_bidir(Q, K, V, W, b, input_scale, denom_eps=0.0, out_dtype=None, out=None,
               workspace=None, stream=None, kernel=KERNEL_SOFTMAX, renormalize=True,
               kernel_eps=1e-3, row_scale=None):
    """Bidirectional FAVOR, Algorithm 1 (favor_attn_bidir). Returns out [B, H, L, d]."""
    torch = _torch()
    g = _desc_for(Q, W, input_scale, _out_dtype(out_dtype, out, Q), denom_eps,
                  others=(("K", K), ("V", V)), opts=_opts(kernel, renormalize, kernel_eps))
    _require_features(W, b, g.H, g.M, g.d)
    if out is None:
        out = torch.empty(Q.shape, dtype=_torch_dtype(g.out_dtype), device=Q.device)
    _require_like(out, Q.shape, _torch_dtype(g.out_dtype), "out")
    _require_row_scale(row_scale, g, "row_scale")
    _require_cuda(Q, K, V, W, b, out, row_scale)
    ws, nbytes = _workspace(g, 0, workspace)
    if row_scale is None:
        _check(lib().favor_attn_bidir(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W),
                                      _ptr(b), _ptr(out), _ptr(ws), ctypes.c_size_t(nbytes),
                                      _stream(stream)))
    else:
        _check(lib().favor_attn_bidir_save(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W),
                                           _ptr(b), _ptr(out), _ptr(row_scale), _ptr(ws),
                                           ctypes.c_size_t(nbytes), _stream(stream)))
    return out


@_on_stream
def attn_causal(Q, K, V, W, b, input_scale, denom_eps=0.0, state_in=None, return_state=False,
                segment=0, out_dtype=None, out=None, state_out=None, workspace=None, stream=None,
                kernel=KERNEL_SOFTMAX, renormalize=True, kernel_eps=1e-3, row_scale=None,
                chunk=0):
    """Unidirectional FAVOR by prefix sums (favor_attn_causal; favor_attn_causal_save
    when row_scale is given). segment: rows per causal segment (0 = library default);
    chunk: tokens per step of the scan (0 = 64; bf16 inputs also take 32).

    Returns out, or (out, state_out [B, H, M, d+1]) when return_state is true.
    """
    torch = _torch()
    g = _desc_for(Q, W, input_scale, _out_dtype(out_dtype, out, Q), denom_eps, segment,
                  others=(("K", K), ("V", V)),
                  opts=dict(_opts(kernel, renormalize, kernel_eps), chunk=chunk))
    _require_features(W, b, g.H, g.M, g.d)
    sshape = (g.B, g.H, g.M, g.d + 1)
    if out is None:
        out = torch.empty(Q.shape, dtype=_torch_dtype(g.out_dtype), device=Q.device)
    if return_state and state_out is None:
        state_out = torch.empty(sshape, dtype=torch.float32, device=Q.device)
    _require_like(out, Q.shape, _torch_dtype(g.out_dtype), "out")
    _require_like(state_in, sshape, torch.float32, "state_in")
    _require_like(state_out, sshape, torch.float32, "state_out")
    _require_row_scale(row_scale, g, "row_scale")
    _require_cuda(Q, K, V, W, b, out, state_in, state_out, row_scale)
    ws, nbytes = _workspace(g, 1, workspace)
    if row_scale is None:
        _check(lib().favor_attn_causal(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W),
                                       _ptr(b), _ptr(out), _ptr(state_in), _ptr(state_out),
                                       _ptr(ws), ctypes.c_size_t(nbytes), _stream(stream)))
    else:
        _check(lib().favor_attn_causal_save(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W),
                                            _ptr(b), _ptr(out), _ptr(state_in), _ptr(state_out),
                                            _ptr(row_scale), _ptr(ws), ctypes.c_size_t(nbytes),
                                            _stream(stream)))
    return (out, state_out) if return_state else out


@_on_stream
def attn_both(Q, K, V, W, b, input_scale, denom_eps=0.0, state_in=None, return_state=False,
              segment=0, out_dtype=None, out_bidir=None, out_causal=None, state_out=None,
              workspace=None, stream=None, kernel=KERNEL_SOFTMAX, renormalize=True,
              kernel_eps=1e-3, row_scale_bidir=None, row_scale_causal=None, chunk=0):
    """Both directions over the same inputs with one key pass (favor_attn_both);
    segment and chunk as for attn_causal.

    Returns (out_bidir, out_causal) or (out_bidir, out_causal, state_out).
    """
    torch = _torch()
    g = _desc_for(Q, W, input_scale, _out_dtype(out_dtype, out_bidir, Q), denom_eps, segment,
                  others=(("K", K), ("V", V)),
                  opts=dict(_opts(kernel, renormalize, kernel_eps), chunk=chunk))
    _require_features(W, b, g.H, g.M, g.d)
    odt = _torch_dtype(g.out_dtype)
    sshape = (g.B, g.H, g.M, g.d + 1)
    if out_bidir is None:
        out_bidir = torch.empty(Q.shape, dtype=odt, device=Q.device)
    if out_causal is None:
        out_causal = torch.empty(Q.shape, dtype=odt, device=Q.device)
    if return_state and state_out is None:
        state_out = torch.empty(sshape, dtype=torch.float32, device=Q.device)
    _require_like(out_bidir, Q.shape, odt, "out_bidir")
    _require_like(out_causal, Q.shape, odt, "out_causal")
    _require_like(state_in, sshape, torch.float32, "state_in")
    _require_like(state_out, sshape, torch.float32, "state_out")
    _require_row_scale(row_scale_bidir, g, "row_scale_bidir")
    _require_row_scale(row_scale_causal, g, "row_scale_causal")
    _require_cuda(Q, K, V, W, b, out_bidir, out_causal, state_in, state_out, row_scale_bidir,
                  row_scale_causal)
    ws, nbytes = _workspace(g, 2, workspace)
    _check(lib().favor_attn_both(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(b),
                                 _ptr(out_bidir), _ptr(out_causal), _ptr(state_in),
                                 _ptr(state_out), _ptr(row_scale_bidir), _ptr(row_scale_causal),
                                 _ptr(ws), ctypes.c_size_t(nbytes), _stream(stream)))
    if return_state:
        return out_bidir, out_causal, state_out
    return out_bidir, out_causal


@_on_stream
def attn_both_noalloc(Q, K, V, W, b, input_scale, denom_eps=0.0, state_in=None,
                      segment=0, out_bidir=None, out_causal=None, state_out=None, stream=None,
                      kernel=KERNEL_SOFTMAX, renormalize=True, kernel_eps=1e-3,
                      row_scale_bidir=None, row_scale_causal=None, chunk=0):
    """attn_both with the library's static scratch as workspace
    (favor_attn_both_noalloc): nothing is allocated when the outputs are given.
    Returns (out_bidir, out_causal)."""
    torch = _torch()
    odt = out_bidir.dtype if out_bidir is not None else Q.dtype
    g = _desc_for(Q, W, input_scale, odt, denom_eps, segment,
                  others=(("K", K), ("V", V)),
                  opts=dict(_opts(kernel, renormalize, kernel_eps), chunk=chunk))
    _require_features(W, b, g.H, g.M, g.d)
    tdt = _torch_dtype(g.out_dtype)
    sshape = (g.B, g.H, g.M, g.d + 1)
    if out_bidir is None:
        out_bidir = torch.empty(Q.shape, dtype=tdt, device=Q.device)
    if out_causal is None:
        out_causal = torch.empty(Q.shape, dtype=tdt, device=Q.device)
    _require_like(out_bidir, Q.shape, tdt, "out_bidir")
    _require_like(out_causal, Q.shape, tdt, "out_causal")
    _require_like(state_in, sshape, torch.float32, "state_in")
    _require_like(state_out, sshape, torch.float32, "state_out")
    _require_row_scale(row_scale_bidir, g, "row_scale_bidir")
    _require_row_scale(row_scale_causal, g, "row_scale_causal")
    _require_cuda(Q, K, V, W, b, out_bidir, out_causal, state_in, state_out, row_scale_bidir,
                  row_scale_causal)
    _check(lib().favor_attn_both_noalloc(
        ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(b), _ptr(out_bidir),
        _ptr(out_causal), _ptr(state_in), _ptr(state_out), _ptr(row_scale_bidir),
        _ptr(row_scale_causal), _stream(stream)))
    return out_bidir, out_causal


def noalloc_scratch_bytes():
    """Size of the static scratch array attn_both_noalloc uses (per GPU)."""
    return lib().favor_noalloc_scratch_bytes()


def _bwd_workspace(g, causal, workspace):
    torch = _torch()
    n = backward_workspace_size(g, causal)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8,
                                device=torch.device("cuda", torch.cuda.current_device()))
    return workspace, workspace.numel() * workspace.element_size()


def _bwd_grads(Q, dQ, dK, dV):
    torch = _torch()
    out = []
    for name, t in (("dQ", dQ), ("dK", dK), ("dV", dV)):
        if t is None:
            t = torch.empty_like(Q)
        _require_like(t, Q.shape, Q.dtype, name)
        out.append(t)
    return out


_FWD_OPS = {"bidir": OP_BIDIR, "causal": OP_CAUSAL, "both": OP_BOTH}


def _forward_ws(forward_workspace, forward_call, allowed):
    """(pointer, op code) of a forward call's workspace offered to a backward call."""
    if forward_workspace is None:
        if forward_call is not None:
            raise FavorError(1, "forward_call without forward_workspace")
        return ctypes.c_void_p(0), 0
    if forward_call not in allowed:
        raise FavorError(1, f"forward_call must be one of {sorted(allowed)}, got {forward_call!r}")
    _require_cuda(forward_workspace)
    return _ptr(forward_workspace), _FWD_OPS[forward_call]


def _saved(out, row_scale, g, Q):
    if (out is None) != (row_scale is None):
        raise FavorError(1, "pass the forward call's out and row_scale together")
    if out is not None:
        _require_like(out, Q.shape, Q.dtype, "out")
        _require_row_scale(row_scale, g, "row_scale")


@_on_stream
def attn_bidir_backward(Q, K, V, W, b, input_scale, dout, denom_eps=0.0, dQ=None, dK=None,
                        dV=None, workspace=None, stream=None, kernel=KERNEL_SOFTMAX,
                        renormalize=True, kernel_eps=1e-3, out=None, row_scale=None,
                        forward_workspace=None, forward_call=None):
    """Gradients (dQ, dK, dV) of attn_bidir for the upstream gradient dout
    (favor_attn_bidir_backward). out and row_scale, from the forward call with
    row_scale, spare recomputing them; forward_workspace, the workspace of the
    forward call forward_call ("bidir" or "both") with the same descriptor and
    inputs, spares recomputing Buf1."""
    g = _desc_for(Q, W, input_scale, Q.dtype, denom_eps,
                  others=(("K", K), ("V", V), ("dout", dout)),
                  opts=_opts(kernel, renormalize, kernel_eps))
    _require_features(W, b, g.H, g.M, g.d)
    dQ, dK, dV = _bwd_grads(Q, dQ, dK, dV)
    _saved(out, row_scale, g, Q)
    _require_cuda(Q, K, V, W, b, dout, dQ, dK, dV, out, row_scale)
    fptr, fop = _forward_ws(forward_workspace, forward_call, ("bidir", "both"))
    ws, nbytes = _bwd_workspace(g, False, workspace)
    _check(lib().favor_attn_bidir_backward(ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W),
                                           _ptr(b), _ptr(dout), _ptr(out), _ptr(row_scale),
                                           fptr, fop, _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws),
                                           ctypes.c_size_t(nbytes), _stream(stream)))
    return dQ, dK, dV


@_on_stream
def attn_causal_backward(Q, K, V, W, b, input_scale, dout, denom_eps=0.0, state_in=None,
                         dstate_out=None, return_state_grad=False, dQ=None, dK=None, dV=None,
                         dstate_in=None, workspace=None, stream=None, kernel=KERNEL_SOFTMAX,
                         renormalize=True, kernel_eps=1e-3, out=None, row_scale=None,
                         forward_workspace=None, forward_call=None, chunk=0):
    """Gradients of attn_causal (favor_attn_causal_backward). Returns (dQ, dK, dV), plus
    dstate_in [B, H, M, d+1] when return_state_grad is true. out and row_scale as for
    attn_bidir_backward; forward_workspace of the forward call forward_call ("causal"
    or "both", same descriptor, inputs and state_in) spares recomputing the segment
    prefixes. chunk: the scan's chunk length for the forward quantities the call
    recomputes (as for attn_causal)."""
    torch = _torch()
    g = _desc_for(Q, W, input_scale, Q.dtype, denom_eps,
                  others=(("K", K), ("V", V), ("dout", dout)),
                  opts=dict(_opts(kernel, renormalize, kernel_eps), chunk=chunk))
    _require_features(W, b, g.H, g.M, g.d)
    dQ, dK, dV = _bwd_grads(Q, dQ, dK, dV)
    sshape = (g.B, g.H, g.M, g.d + 1)
    if return_state_grad and dstate_in is None:
        dstate_in = torch.empty(sshape, dtype=torch.float32, device=Q.device)
    for name, t in (("state_in", state_in), ("dstate_out", dstate_out), ("dstate_in", dstate_in)):
        _require_like(t, sshape, torch.float32, name)
    _saved(out, row_scale, g, Q)
    _require_cuda(Q, K, V, W, b, dout, dQ, dK, dV, state_in, dstate_out, dstate_in, out,
                  row_scale)
    fptr, fop = _forward_ws(forward_workspace, forward_call, ("causal", "both"))
    ws, nbytes = _bwd_workspace(g, True, workspace)
    _check(lib().favor_attn_causal_backward(
        ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(b), _ptr(state_in), _ptr(dout),
        _ptr(out), _ptr(row_scale), fptr, fop, _ptr(dstate_out), _ptr(dQ), _ptr(dK), _ptr(dV),
        _ptr(dstate_in), _ptr(ws), ctypes.c_size_t(nbytes), _stream(stream)))
    return (dQ, dK, dV, dstate_in) if return_state_grad else (dQ, dK, dV)


def attn_both_backward(Q, K, V, W, b, input_scale, dout_bidir, dout_causal, denom_eps=0.0,
                       state_in=None, dstate_out=None, return_state_grad=False, dQ=None,
                       dK=None, dV=None, dstate_in=None, workspace=None, stream=None,
                       kernel=KERNEL_SOFTMAX, renormalize=True, kernel_eps=1e-3,
                       out_bidir=None, row_scale_bidir=None, out_causal=None,
                       row_scale_causal=None, forward_workspace=None, forward_call=None,
                       chunk=0, segment=0):
    """Gradients of attn_both (favor_attn_both_backward): of a loss of both outputs,
    given dout_bidir and dout_causal. Returns (dQ, dK, dV), the sums over the two
    directions, plus the causal state gradient dstate_in when return_state_grad is
    true. out_* and row_scale_* as the forward call saved them (each pair or
    neither); forward_workspace of an attn_both call (forward_call "both", same
    descriptor, inputs and state_in) spares recomputing Buf1 and the segment
    prefixes."""
    torch = _torch()
    g = _desc_for(Q, W, input_scale, Q.dtype, denom_eps, segment,
                  others=(("K", K), ("V", V), ("dout_bidir", dout_bidir),
                          ("dout_causal", dout_causal)),
                  opts=dict(_opts(kernel, renormalize, kernel_eps), chunk=chunk))
    _require_features(W, b, g.H, g.M, g.d)
    dQ, dK, dV = _bwd_grads(Q, dQ, dK, dV)
    sshape = (g.B, g.H, g.M, g.d + 1)
    if return_state_grad and dstate_in is None:
        dstate_in = torch.empty(sshape, dtype=torch.float32, device=Q.device)
    for name, t in (("state_in", state_in), ("dstate_out", dstate_out), ("dstate_in", dstate_in)):
        _require_like(t, sshape, torch.float32, name)
    _saved(out_bidir, row_scale_bidir, g, Q)
    _saved(out_causal, row_scale_causal, g, Q)
    _require_cuda(Q, K, V, W, b, dout_bidir, dout_causal, dQ, dK, dV, state_in, dstate_out,
                  dstate_in, out_bidir, row_scale_bidir, out_causal, row_scale_causal)
    fptr, fop = _forward_ws(forward_workspace, forward_call, ("both",))
    ws, nbytes = _bwd_workspace(g, 2, workspace)
    _check(lib().favor_attn_both_backward(
        ctypes.byref(g), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(b), _ptr(state_in),
        _ptr(dout_bidir), _ptr(dout_causal), _ptr(out_bidir), _ptr(row_scale_bidir),
        _ptr(out_causal), _ptr(row_scale_causal), fptr, fop, _ptr(dstate_out), _ptr(dQ),
        _ptr(dK), _ptr(dV), _ptr(dstate_in), _ptr(ws), ctypes.c_size_t(nbytes),
        _stream(stream)))
    return (dQ, dK, dV, dstate_in) if return_state_grad else (dQ, dK, dV)


def library_loaded_from():
    """Absolute path of the libfavor.so this process uses."""
    return os.path.realpath(lib_path())
