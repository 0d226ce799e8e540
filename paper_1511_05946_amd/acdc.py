"""Python binding of the ACDC / AFDF cascade library.

Argument marshalling only: every step of the computation runs in the HIP
kernels of libacdc.so.  Tensors are torch tensors on a ROCm device; the work
is enqueued on the current torch stream of that device.

Layer (Sec. 4 of arXiv:1511.05946): y = x A C D C^{-1} on row vectors, C the
orthonormal DCT-II; the complex AFDF layer of Sec. 3 uses the DFT.  A cascade
chains K layers with optional fixed permutations and ReLU between them, and
optionally a bias b_k added to each layer's D-domain term (Sec. 6.2):
y = (x A C D + b) C^{-1}.
"""

from __future__ import annotations

import ctypes

import torch

from ._lib import lib, status_string

FLAG_PERM = 1
FLAG_RELU = 2
FLAG_COMPLEX = 4
FLAG_BIAS = 8
FLAG_ACCUMULATE = 16
FLAG_MULTIPASS = 32


class ACDCError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        extra = ""
        if rc == -4:
            extra = f" (hipError {lib().acdc_last_hip_error()})"
        raise ACDCError(f"{what}: {status_string(rc)}{extra}")


def _flags(flags: int, x: torch.Tensor, bias=None) -> int:
    if x.is_complex():
        flags |= FLAG_COMPLEX
    if bias is not None:
        flags |= FLAG_BIAS
    return flags


def _ptr(t):
    if t is None:
        return None
    return t.data_ptr()


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def _dims(x: torch.Tensor, A: torch.Tensor):
    if x.dim() != 2 or A.dim() != 2:
        raise ValueError("x must be [batch, N] and A, D [K, N]")
    if A.shape[1] != x.shape[1]:
        raise ValueError(f"A is {tuple(A.shape)}: its rows must have x's width N = {x.shape[1]}")
    return x.shape[0], x.shape[1], A.shape[0]


def _check_shapes(shapes: dict, B: int, N: int, K: int):
    """Every tensor handed to the library must have exactly the shape its
    pointer is read or written with: rows [B, N], layer vectors [K, N]. The
    library takes raw pointers, so a mismatch here would be an out-of-bounds
    device access there; this runs before any device or dtype check."""
    want = {"row": (B, N), "layer": (K, N)}
    for name, (t, kind) in shapes.items():
        if t is None:
            continue
        if tuple(t.shape) != want[kind]:
            raise ValueError(f"{name} is {tuple(t.shape)}, expected {want[kind]}")


def _validate(tensors, complex_: bool, device):
    for name, t in tensors.items():
        if t is None:
            continue
        if t.device != device:
            raise ValueError(f"{name} is on {t.device}, expected {device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if name == "perm":
            if t.dtype != torch.int32:
                raise ValueError("perm must be int32")
        elif name == "workspace":
            pass
        elif complex_ and t.dtype != torch.complex64:
            raise ValueError(f"{name} must be complex64")
        elif not complex_ and t.dtype != torch.float32:
            raise ValueError(f"{name} must be float32")


def _stream(device):
    return torch.cuda.current_stream(device).cuda_stream


def supported(N: int, flags: int = 0) -> bool:
    return bool(lib().acdc_supported(int(N), int(flags)))


def prepare(N: int, flags: int = 0, device=None):
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        _check(lib().acdc_prepare(int(N), int(flags)), "acdc_prepare")


def sync_timeouts(device=None, clear: bool = False) -> int:
    """Backward row syncs on `device` whose bounded wait ran out (0 when healthy).

    Synchronises the device first; with clear=True the count restarts at 0."""
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        torch.cuda.synchronize()
        n = ctypes.c_int64(0)
        _check(lib().acdc_sync_timeouts(ctypes.byref(n), int(bool(clear))), "acdc_sync_timeouts")
        return int(n.value)


def saved_numel(x: torch.Tensor, K: int, flags: int = 0) -> int:
    """Elements (of x's dtype) of the buffer acdc_forward fills for
    acdc_backward: the layer inputs u_1..u_{K-1}, preceded by u_0 (x gathered
    through perm[0]) with FLAG_PERM."""
    flags = _flags(flags, x)
    nbytes = lib().acdc_saved_bytes(x.shape[0], x.shape[1], K, flags)
    return nbytes // x.element_size()


def alloc_saved(x: torch.Tensor, K: int, flags: int = 0) -> torch.Tensor:
    return torch.empty(saved_numel(x, K, flags), dtype=x.dtype, device=x.device)


def saved_layer_inputs(saved: torch.Tensor, x: torch.Tensor, K: int, flags: int = 0) -> torch.Tensor:
    """View of the layer inputs inside a saved buffer, [slots, batch, N]:
    u_1..u_{K-1} in slots 0..K-2, and with FLAG_PERM u_0 (x gathered through
    perm[0]) in slot K-1."""
    B, N = x.shape
    L = K - 1 + (1 if flags & FLAG_PERM else 0)
    return saved[: L * B * N].view(L, B, N)


def forward_workspace_bytes(x, K: int, flags: int = 0, bias=None) -> int:
    """Bytes of the caller-owned workspace acdc_forward takes for x [B, N]."""
    flags = _flags(flags, x, bias)
    return int(lib().acdc_forward_workspace_size(x.shape[0], x.shape[1], K, flags))


def backward_workspace_bytes(x, K: int, flags: int = 0, have_saved: bool = True, bias=None) -> int:
    """Bytes of the caller-owned workspace acdc_backward takes for x [B, N]
    (more without the forward's saved layer inputs: the stash is rebuilt in
    it)."""
    flags = _flags(flags, x, bias)
    return int(lib().acdc_backward_workspace_size(x.shape[0], x.shape[1], K, flags, 1 if have_saved else 0))


def _workspace(ws, need: int, device):
    if ws is None:
        return torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    if ws.dtype != torch.uint8 or ws.dim() != 1 or ws.numel() < need:
        raise ValueError(f"workspace must be a uint8 vector of at least {need} bytes")
    return ws


def forward(x, A, D, perm=None, flags: int = 0, save: bool = False, out=None, saved=None, bias=None,
            workspace=None):
    """y = cascade(x), with the D-domain biases ``bias`` [K, N] if given.
    Returns (y, saved) where saved holds the layer inputs u_1..u_{K-1} for
    acdc_backward when ``save`` (or a preallocated ``saved``) is given.
    ``workspace``: a uint8 device vector of forward_workspace_bytes() bytes
    (allocated here when not given)."""
    flags = _flags(flags, x, bias)
    cplx = bool(flags & FLAG_COMPLEX)
    B, N, K = _dims(x, A)
    _check_shapes({"D": (D, "layer"), "bias": (bias, "layer"), "y": (out, "row"),
                   "perm": (perm if flags & FLAG_PERM else None, "layer")}, B, N, K)
    if saved is not None and saved.numel() < saved_numel(x, K, flags):
        raise ValueError(f"saved holds {saved.numel()} elements, needs {saved_numel(x, K, flags)}")
    if out is None:
        out = torch.empty_like(x)
    if save and saved is None:
        saved = alloc_saved(x, K, flags)
    _validate({"x": x, "A": A, "D": D, "bias": bias, "y": out, "saved": saved,
               "perm": perm if flags & FLAG_PERM else None}, cplx, x.device)
    L = lib()
    ws_bytes = L.acdc_forward_workspace_size(B, N, K, flags)
    ws = _workspace(workspace, ws_bytes, x.device)
    _validate({"workspace": ws}, cplx, x.device)
    with torch.cuda.device(x.device):
        rc = L.acdc_forward(_ptr(x), _ptr(out), _ptr(A), _ptr(D), _ptr(bias),
                            _ptr(perm) if flags & FLAG_PERM else None, B, N, K, flags,
                            _ptr(saved) if (saved is not None and saved.numel() > 0) else None,
                            _nbytes(saved), _ptr(ws), ws_bytes, _stream(x.device))
    _check(rc, "acdc_forward")
    return out, saved


def backward(x, grad_y, A, D, perm=None, flags: int = 0, saved=None, bias=None, grads=None, out=None,
             workspace=None):
    """(grad_x, grad_A, grad_D), plus grad_bias when ``bias`` is given; the
    parameter gradients are summed over the batch.  Without ``saved`` (from
    ``forward(..., save=True)`` on the same inputs) the forward is recomputed
    inside the call.  ``grads`` = (grad_A, grad_D[, grad_bias]) tensors to
    write into; with FLAG_ACCUMULATE in ``flags`` the sums are added to them.
    ``out``: a tensor to write grad_x into.  ``workspace``: a uint8 device
    vector of backward_workspace_bytes() bytes (allocated when not given)."""
    flags = _flags(flags, x, bias)
    cplx = bool(flags & FLAG_COMPLEX)
    B, N, K = _dims(x, A)
    if grads is None and flags & FLAG_ACCUMULATE:
        raise ValueError("FLAG_ACCUMULATE needs the gradient tensors to add into (grads=...)")
    if grads is not None and len(grads) != (3 if bias is not None else 2):
        raise ValueError("grads must be (grad_A, grad_D) or, with bias, (grad_A, grad_D, grad_bias)")
    _check_shapes({"grad_y": (grad_y, "row"), "grad_x": (out, "row"), "D": (D, "layer"), "bias": (bias, "layer"),
                   "perm": (perm if flags & FLAG_PERM else None, "layer"),
                   "grad_A": (grads[0] if grads is not None else None, "layer"),
                   "grad_D": (grads[1] if grads is not None else None, "layer"),
                   "grad_bias": (grads[2] if grads is not None and bias is not None else None, "layer")}, B, N, K)
    if saved is not None and 0 < saved.numel() < saved_numel(x, K, flags):
        raise ValueError(f"saved holds {saved.numel()} elements, needs {saved_numel(x, K, flags)}")
    gx = torch.empty_like(x) if out is None else out
    if grads is None:
        grads = (torch.empty_like(A), torch.empty_like(D)) + ((torch.empty_like(bias),) if bias is not None else ())
    gA, gD = grads[0], grads[1]
    gB = grads[2] if bias is not None else None
    _validate({"x": x, "grad_y": grad_y, "grad_x": gx, "A": A, "D": D, "bias": bias, "saved": saved, "grad_A": gA,
               "grad_D": gD, "grad_bias": gB, "perm": perm if flags & FLAG_PERM else None}, cplx, x.device)
    L = lib()
    use_saved = saved is not None and saved.numel() > 0
    have_saved = 1 if (use_saved or saved_numel(x, K, flags) == 0) else 0
    ws_bytes = L.acdc_backward_workspace_size(B, N, K, flags, have_saved)
    ws = _workspace(workspace, ws_bytes, x.device)
    _validate({"workspace": ws}, cplx, x.device)
    with torch.cuda.device(x.device):
        rc = L.acdc_backward(_ptr(x), _ptr(grad_y), _ptr(A), _ptr(D), _ptr(bias),
                             _ptr(perm) if flags & FLAG_PERM else None,
                             _ptr(saved) if use_saved else None, _nbytes(saved),
                             _ptr(gx), _ptr(gA), _ptr(gD), _ptr(gB), B, N, K, flags, _ptr(ws), ws_bytes,
                             _stream(x.device))
    _check(rc, "acdc_backward")
    return (gx, gA, gD, gB) if bias is not None else (gx, gA, gD)


class ACDCCascade(torch.autograd.Function):
    """autograd wrapper: stores the layer inputs in the forward pass."""

    @staticmethod
    def forward(ctx, x, A, D, perm, flags, bias=None):
        # the backward gets exactly the (contiguous) tensors the forward used
        x, A, D = x.contiguous(), A.contiguous(), D.contiguous()
        perm = perm.contiguous() if perm is not None else None
        bias = bias.contiguous() if bias is not None else None
        y, saved = forward(x, A, D, perm, flags, save=True, bias=bias)
        ctx.save_for_backward(x, A, D, perm if perm is not None else torch.empty(0),
                              bias if bias is not None else torch.empty(0), saved)
        ctx.flags = flags
        ctx.has_perm = perm is not None
        ctx.has_bias = bias is not None
        return y

    @staticmethod
    def backward(ctx, gy):
        x, A, D, perm, bias, saved = ctx.saved_tensors
        out = backward(x, gy.contiguous(), A, D, perm if ctx.has_perm else None, ctx.flags, saved,
                       bias=bias if ctx.has_bias else None)
        gB = out[3] if ctx.has_bias else None
        return out[0], out[1], out[2], None, None, gB


def acdc_cascade(x, A, D, perm=None, flags: int = 0, bias=None):
    return ACDCCascade.apply(x, A, D, perm, flags, bias)
