"""Python binding of the MI355X GaLore 2 hot-path library (``libgalore.so``).

Argument marshalling only: every step runs in the HIP kernels behind the C ABI
declared in ``include/galore.h``; torch tensors supply device memory and the
current stream. There is no fallback: if the shared object is missing, importing
the binding raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# GALORE_LIB selects another build of the same sources (the tests' host-side
# sanitizer build); by default the in-tree libgalore.so
LIB_PATH = os.environ.get("GALORE_LIB") or os.path.join(_HERE, "libgalore.so")

GALORE_F32 = 0
GALORE_BF16 = 1
GALORE_OK = 0

EXPORTED = (
    "galore_status_string", "galore_version", "galore_sketch", "galore_rsvd_workspace_size",
    "galore_rsvd_update", "galore_rsvd_update_traced", "galore_project_workspace_size", "galore_project",
    "galore_lowrank_adam_step",
    "galore_project_back_workspace_size", "galore_project_back",
    "galore_align_workspace_size", "galore_align_projector",
    "galore_step_workspace_size", "galore_step",
    "galore_quantize_projector", "galore_project_quantized_workspace_size", "galore_project_quantized",
    "galore_project_back_quantized_workspace_size", "galore_project_back_quantized",
    "galore_adam8_scale_count", "galore_lowrank_adam8_step",
    "galore_svd_workspace_size", "galore_svd_update", "galore_probe_mfma_bf16", "galore_probe_copy",
    "galore_project_noalloc_max_bytes", "galore_project_noalloc",
)

GALORE_STEP_ALIGN = 1
GALORE_STEP_REEXPRESS = 2

# galore_stage_t
STAGES = ("sketch", "product_A", "product_At", "gram", "cholesky", "triangular", "jacobi", "projector",
          "other", "operand", "refine")


class GaloreError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))
        self.status = status


def _declare(lib):
    vp, i64, i32, u64, f32, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                  ctypes.c_float, ctypes.c_size_t)
    lib.galore_status_string.argtypes = [ctypes.c_int]
    lib.galore_status_string.restype = ctypes.c_char_p
    lib.galore_version.argtypes = []
    lib.galore_version.restype = ctypes.c_int
    lib.galore_sketch.argtypes = [vp, i64, i64, u64, u64, vp]
    lib.galore_sketch.restype = ctypes.c_int
    lib.galore_rsvd_workspace_size.argtypes = [i64, i64, i32, i32, i32, i32]
    lib.galore_rsvd_workspace_size.restype = sz
    lib.galore_rsvd_update.argtypes = [vp, i32, i64, i64, i64, i64, i32, i32, i32, u64, u64,
                                       vp, i64, i64, vp, i64, vp, i32, vp, sz, vp, vp]
    lib.galore_rsvd_update.restype = ctypes.c_int
    lib.galore_rsvd_update_traced.argtypes = lib.galore_rsvd_update.argtypes + [
        ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_int32), i32, ctypes.POINTER(ctypes.c_int32)]
    lib.galore_rsvd_update_traced.restype = ctypes.c_int
    lib.galore_project_workspace_size.argtypes = [i64, i64, i32, i32, i32]
    lib.galore_project_workspace_size.restype = sz
    lib.galore_project.argtypes = [vp, i64, i64, vp, i32, i64, i64, i64, i64, i32, vp, i64, i64,
                                   i32, vp, sz, vp]
    lib.galore_project.restype = ctypes.c_int
    lib.galore_lowrank_adam_step.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, f32, f32, f32,
                                             i64, vp]
    lib.galore_lowrank_adam_step.restype = ctypes.c_int
    lib.galore_project_back_workspace_size.argtypes = [i64, i64, i32, i32]
    lib.galore_project_back_workspace_size.restype = sz
    lib.galore_project_back.argtypes = [vp, i64, i64, vp, i64, i64, vp, i64, i64, i64, i64, i32,
                                        f32, f32, i32, vp, sz, vp]
    lib.galore_project_back.restype = ctypes.c_int
    lib.galore_align_workspace_size.argtypes = [i32, i32]
    lib.galore_align_workspace_size.restype = sz
    lib.galore_align_projector.argtypes = [vp, i64, i64, vp, i64, i64, i64, i32, vp, vp, vp, i64, i64, i64, i32,
                                           vp, sz, vp]
    lib.galore_align_projector.restype = ctypes.c_int
    lib.galore_step_workspace_size.argtypes = [i64, i64, i32, i32, i32, i32, i32]
    lib.galore_step_workspace_size.restype = sz
    lib.galore_step.argtypes = [vp, i32, i64, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, vp, i64, i64,
                                i32, i32, i32, u64, u64, i64, i32, f32, f32, f32, f32, f32, i32, vp, i32, vp, sz, vp,
                                vp]
    lib.galore_step.restype = ctypes.c_int
    lib.galore_quantize_projector.argtypes = [vp, i64, i64, i64, i32, i32, vp, i64, i64, vp, i64, i32, vp]
    lib.galore_quantize_projector.restype = ctypes.c_int
    lib.galore_project_quantized_workspace_size.argtypes = [i64, i64, i32, i32]
    lib.galore_project_quantized_workspace_size.restype = sz
    lib.galore_project_quantized.argtypes = [vp, i64, i64, vp, i64, i32, vp, i32, i64, i64, i64, i64, i32, vp, i64,
                                             i64, i32, vp, sz, vp]
    lib.galore_project_quantized.restype = ctypes.c_int
    lib.galore_project_back_quantized_workspace_size.argtypes = [i64, i64, i32, i32]
    lib.galore_project_back_quantized_workspace_size.restype = sz
    lib.galore_project_back_quantized.argtypes = [vp, i64, i64, vp, i64, i32, vp, i64, i64, vp, i64, i64, i64, i64,
                                                  i32, f32, f32, i32, vp, sz, vp]
    lib.galore_project_back_quantized.restype = ctypes.c_int
    lib.galore_adam8_scale_count.argtypes = [i64, i64]
    lib.galore_adam8_scale_count.restype = i64
    lib.galore_lowrank_adam8_step.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, i64, i64, i32, f32, f32, f32, i64, vp]
    lib.galore_lowrank_adam8_step.restype = ctypes.c_int
    lib.galore_svd_workspace_size.argtypes = [i64, i64, i32, i32, i32]
    lib.galore_svd_workspace_size.restype = sz
    lib.galore_svd_update.argtypes = [vp, i32, i64, i64, i64, i64, i32, vp, i64, i64, vp, i64, vp, i32, vp, sz, vp,
                                      vp]
    lib.galore_svd_update.restype = ctypes.c_int
    lib.galore_probe_mfma_bf16.argtypes = [i64, i32, vp, ctypes.POINTER(ctypes.c_double), vp]
    lib.galore_probe_mfma_bf16.restype = ctypes.c_int
    lib.galore_probe_copy.argtypes = [vp, vp, sz, vp]
    lib.galore_probe_copy.restype = ctypes.c_int
    lib.galore_project_noalloc_max_bytes.argtypes = []
    lib.galore_project_noalloc_max_bytes.restype = sz
    lib.galore_project_noalloc.argtypes = [vp, i64, i64, vp, i32, i64, i64, i64, i64, i32, vp, i64, i64, i32, vp]
    lib.galore_project_noalloc.restype = ctypes.c_int
    return lib


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("%s is not built (run __graft_entry__.build()); "
                          "there is no fallback path" % LIB_PATH)
    return _declare(ctypes.CDLL(LIB_PATH))


lib = _load()


def status_string(status: int) -> str:
    return lib.galore_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != GALORE_OK:
        raise GaloreError(status, where)


def _torch_stream(stream, device=None):
    """torch stream object for `stream`: None is the current stream of
    `device`; a torch.cuda.Stream is kept; an integer is a raw HIP handle."""
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    if hasattr(stream, "cuda_stream"):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


def _handle(ts):
    return ctypes.c_void_p(ts.cuda_stream if ts is not None else 0)


def _aux(aux_stream, device=None):
    """the optional second stream (None passes NULL: everything on one stream)"""
    return None if aux_stream is None else _torch_stream(aux_stream, device)


def _geom(t: torch.Tensor, name: str):
    """(rows, cols, ld, batch_stride, batch) of a 2-D or 3-D row-major tensor;
    shapes only, no device access (a 2-D tensor is a batch of one)."""
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a tensor" % name)
    if t.dim() == 2:
        if t.stride(1) != 1 and t.shape[1] > 1:
            raise ValueError("%s must be row-major" % name)
        rows, cols = t.shape
        return rows, cols, t.stride(0), rows * t.stride(0), 1
    if t.dim() == 3:
        if t.stride(2) != 1 and t.shape[2] > 1:
            raise ValueError("%s must be row-major" % name)
        b, rows, cols = t.shape
        return rows, cols, t.stride(1), t.stride(0), b
    raise ValueError("%s must be 2-D or 3-D" % name)


def _mat(t: torch.Tensor, name: str):
    """(ptr, rows, cols, ld, batch_stride, batch) of a 2-D or 3-D row-major tensor."""
    rows, cols, ld, st, b = _geom(t, name)
    return t.data_ptr(), rows, cols, ld, st, b


def _expect(t, name, rows, cols, batch, dtype=torch.float32):
    """t must hold `batch` rows x cols matrices of `dtype` (2-D only for a batch of one)."""
    r_, c_, _, _, b_ = _geom(t, name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if (r_, c_, b_) != (rows, cols, batch):
        raise ValueError("%s must hold %d matrices of %d x %d, got shape %s" % (name, batch, rows, cols,
                                                                               tuple(t.shape)))


def _expect_vec(t, name, length, batch, dtype):
    """t: (batch, length) with unit stride in the last dimension, or (length,) for a batch of one"""
    if not isinstance(t, torch.Tensor) or t.dtype != dtype:
        raise ValueError("%s must be a %s tensor" % (name, dtype))
    ok = (t.dim() == 2 and tuple(t.shape) == (batch, length) and (t.stride(1) == 1 or length == 1)) or \
         (t.dim() == 1 and batch == 1 and t.shape[0] == length and (t.stride(0) == 1 or length == 1))
    if not ok:
        raise ValueError("%s must have shape (%d, %d)%s, got %s" % (name, batch, length,
                                                                  " or (%d,)" % length if batch == 1 else "",
                                                                  tuple(t.shape)))


def _on_device(device, **tensors):
    for nm, t in tensors.items():
        if t is None or t is False:
            continue
        if not t.is_cuda:
            raise ValueError("%s must be a device tensor" % nm)
        if device is not None and t.device != device:
            raise ValueError("%s must be on %s" % (nm, device))


def _ws_bytes(ws, name="workspace"):
    if ws.dim() != 1 or not ws.is_contiguous():
        raise ValueError("%s must be a contiguous 1-D tensor" % name)
    return ws.numel() * ws.element_size()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GALORE_F32
    if t.dtype == torch.bfloat16:
        return GALORE_BF16
    raise ValueError("gradient dtype must be float32 or bfloat16")


def galore_version() -> int:
    return lib.galore_version()


def galore_sketch(l: int, k: int, seed: int, sketch_index: int = 0, out=None, stream=None, device="cuda"):
    """Omega (l x k, fp32) as the subspace update draws it."""
    if out is not None:
        _expect(out, "out", l, k, 1)
        if not out.is_contiguous():
            raise ValueError("out must be contiguous")
        _on_device(None, out=out)
        device = out.device
    ts = _torch_stream(stream, torch.device(device))
    with torch.cuda.stream(ts):
        if out is None:
            out = torch.empty((l, k), dtype=torch.float32, device=device)
        _check(lib.galore_sketch(out.data_ptr(), l, k, seed, sketch_index, _handle(ts)), "galore_sketch")
    return out


def galore_rsvd_workspace_size(m: int, n: int, r: int, p: int, batch: int = 1, dtype=torch.float32) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_rsvd_workspace_size(m, n, r, p, batch, code))


def _validate_update(G, r, P, sigma, info, workspace):
    """Shapes, dtypes and devices of a subspace update's tensors (no device access)."""
    m, n, _, _, batch = _geom(G, "G")
    _dtype_code(G)
    s = min(m, n)
    if P is not None:
        _expect(P, "P", s, r, batch)
    if sigma is not None:
        _expect_vec(sigma, "sigma", r, batch, torch.float32)
    if info is not None and (info.dtype != torch.int32 or info.dim() != 1 or info.numel() != batch
                             or not info.is_contiguous()):
        raise ValueError("info must be a contiguous int32 vector of the batch size")
    if workspace is not None:
        _ws_bytes(workspace)
    _on_device(None, G=G)
    _on_device(G.device, P=P, sigma=sigma, info=info, workspace=workspace)


def _update_outputs(G, r, P, sigma, info, workspace, need):
    """P, sigma, info and the workspace of a subspace update of G, allocated on
    the current stream where not given. A workspace allocated here is released
    to torch's caching allocator when the call returns, before the kernels
    have run: the allocator hands that memory out again only to later work on
    the same stream, which runs after them (the second stream's share of the
    work is joined back into that stream before the call returns)."""
    m, n, _, _, batch = _geom(G, "G")
    s, dev = min(m, n), G.device
    if P is None:
        P = torch.empty((batch, s, r) if G.dim() == 3 else (s, r), dtype=torch.float32, device=dev)
    if sigma is None:
        sigma = torch.empty((batch, r) if G.dim() == 3 else (r,), dtype=torch.float32, device=dev)
    if info is None:
        info = torch.empty((batch,), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=dev)
    return P, sigma, info, workspace


def _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, ts, aux):
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    need = galore_rsvd_workspace_size(m, n, r, p, batch, G.dtype)
    P, sigma, info, workspace = _update_outputs(G, r, P, sigma, info, workspace, need)
    pp, _, _, ldp, sp, _ = _mat(P, "P")
    args = (gp, _dtype_code(G), m, n, ldg, sg, r, p, q, seed, sketch_index0, pp, ldp, sp, sigma.data_ptr(),
            sigma.stride(0) if sigma.dim() == 2 else r, info.data_ptr(), batch, workspace.data_ptr(),
            _ws_bytes(workspace), _handle(ts), _handle(aux))
    return args, P, sigma, info, workspace


def galore_rsvd_update(G: torch.Tensor, r: int, p: int, q: int, seed: int, sketch_index0: int = 0,
                       P=None, sigma=None, info=None, workspace=None, stream=None, aux_stream=None):
    """Subspace update of G ((m, n) or (batch, m, n)); returns (P, sigma, info).
    aux_stream (optional): a second stream of the caller that takes the second
    half of the batch's Cholesky and small-SVD launches (same results)."""
    _validate_update(G, r, P, sigma, info, workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        args, P, sigma, info, ws = _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, ts,
                                              _aux(aux_stream, G.device))
        _check(lib.galore_rsvd_update(*args), "galore_rsvd_update")
    return P, sigma, info


def galore_rsvd_update_traced(G: torch.Tensor, r: int, p: int, q: int, seed: int, events, sketch_index0: int = 0,
                              P=None, sigma=None, info=None, workspace=None, stream=None, aux_stream=None):
    """galore_rsvd_update that also records ``events`` (an even-length list of
    torch.cuda.Event with timing enabled) around its stages; returns
    (P, sigma, info, stages) with stages[i] the stage name of the pair
    (events[2 i], events[2 i + 1])."""
    if len(events) % 2:
        raise ValueError("events must come in (start, end) pairs")
    cap = len(events) // 2
    _validate_update(G, r, P, sigma, info, workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        args, P, sigma, info, ws = _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, ts,
                                              _aux(aux_stream, G.device))
        ev = (ctypes.c_void_p * max(1, 2 * cap))(*[e.cuda_event for e in events])
        st = (ctypes.c_int32 * max(1, cap))()
        cnt = ctypes.c_int32(0)
        _check(lib.galore_rsvd_update_traced(*args, ev, st, cap, ctypes.byref(cnt)), "galore_rsvd_update_traced")
    return P, sigma, info, [STAGES[st[i]] for i in range(cnt.value)]


def galore_project_workspace_size(m: int, n: int, r: int, batch: int = 1, dtype=torch.float32) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_project_workspace_size(m, n, r, batch, code))


def galore_project(P: torch.Tensor, G: torch.Tensor, R=None, workspace=None, stream=None):
    """R = P^T A ((r, l) or (batch, r, l)). A bf16 G gets a workspace of
    galore_project_workspace_size bytes unless one is passed; workspace=False
    passes none."""
    m, n, _, _, batch = _geom(G, "G")
    _dtype_code(G)
    s, l = min(m, n), max(m, n)
    r = _geom(P, "P")[1]
    _expect(P, "P", s, r, batch)
    if R is not None:
        _expect(R, "R", r, l, batch)
    if workspace is not None and workspace is not False:
        _ws_bytes(workspace)
    _on_device(None, G=G)
    _on_device(G.device, P=P, R=R, workspace=workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        if R is None:
            R = torch.empty((batch, r, l) if G.dim() == 3 else (r, l), dtype=torch.float32, device=G.device)
        if workspace is None:
            need = galore_project_workspace_size(m, n, r, batch, G.dtype)
            workspace = torch.empty((need,), dtype=torch.uint8, device=G.device) if need > 0 else False
        wp, wb = (None, 0) if workspace is False else (workspace.data_ptr(), _ws_bytes(workspace))
        pp, _, _, ldp, sp, _ = _mat(P, "P")
        gp, _, _, ldg, sg, _ = _mat(G, "G")
        rp, _, _, ldr, sr, _ = _mat(R, "R")
        _check(lib.galore_project(pp, ldp, sp, gp, _dtype_code(G), m, n, ldg, sg, r, rp, ldr, sr, batch, wp, wb,
                                  _handle(ts)), "galore_project")
    return R


def galore_project_noalloc_max_bytes() -> int:
    return int(lib.galore_project_noalloc_max_bytes())


def galore_project_noalloc(P: torch.Tensor, G: torch.Tensor, R: torch.Tensor, stream=None):
    """R = P^T A like galore_project with a workspace, the scratch held in the
    library's own device array (no allocation in the call; R must be given)."""
    m, n, _, _, batch = _geom(G, "G")
    _dtype_code(G)
    s, l = min(m, n), max(m, n)
    r = _geom(P, "P")[1]
    _expect(P, "P", s, r, batch)
    _expect(R, "R", r, l, batch)
    _on_device(None, G=G)
    _on_device(G.device, P=P, R=R)
    ts = _torch_stream(stream, G.device)
    pp, _, _, ldp, sp, _ = _mat(P, "P")
    gp, _, _, ldg, sg, _ = _mat(G, "G")
    rp, _, _, ldr, sr, _ = _mat(R, "R")
    _check(lib.galore_project_noalloc(pp, ldp, sp, gp, _dtype_code(G), m, n, ldg, sg, r, rp, ldr, sr, batch,
                                      _handle(ts)), "galore_project_noalloc")
    return R


def galore_lowrank_adam_step(R: torch.Tensor, M: torch.Tensor, V: torch.Tensor, N=None, beta1=0.9,
                             beta2=0.999, eps=1e-8, t=1, stream=None):
    """In-place M, V; returns N (may be R itself for an in-place update)."""
    rows, cols, ld, st_, batch = _geom(R, "R")
    if R.dtype != torch.float32:
        raise ValueError("R must be float32")
    for x, nm in ((M, "M"), (V, "V"), (N, "N")):
        if x is not None and (x.shape != R.shape or x.stride() != R.stride() or x.dtype != torch.float32):
            raise ValueError("%s must match R in shape, strides and dtype" % nm)
    _on_device(None, R=R)
    _on_device(R.device, M=M, V=V, N=N)
    ts = _torch_stream(stream, R.device)
    with torch.cuda.stream(ts):
        if N is None:
            N = torch.empty_like(R)
        _check(lib.galore_lowrank_adam_step(R.data_ptr(), M.data_ptr(), V.data_ptr(), N.data_ptr(), rows, cols, ld,
                                            st_, batch, beta1, beta2, eps, t, _handle(ts)),
               "galore_lowrank_adam_step")
    return N


def galore_project_back_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_back_workspace_size(m, n, r, batch))


def galore_project_back(P: torch.Tensor, N: torch.Tensor, W: torch.Tensor, lr: float, alpha: float,
                        workspace=None, stream=None):
    """W <- W - lr*alpha*(P N) (m <= n) or its transpose (m > n), in place. A
    workspace of galore_project_back_workspace_size bytes is allocated unless
    one is passed; workspace=False passes none."""
    m, n, _, _, batch = _geom(W, "W")
    s, l = min(m, n), max(m, n)
    r = _geom(P, "P")[1]
    _expect(W, "W", m, n, batch)
    _expect(P, "P", s, r, batch)
    _expect(N, "N", r, l, batch)
    if workspace is not None and workspace is not False:
        _ws_bytes(workspace)
    _on_device(None, W=W)
    _on_device(W.device, P=P, N=N, workspace=workspace)
    ts = _torch_stream(stream, W.device)
    with torch.cuda.stream(ts):
        if workspace is None:
            need = galore_project_back_workspace_size(m, n, r, batch)
            workspace = torch.empty((need,), dtype=torch.uint8, device=W.device) if need > 0 else False
        wsp, wsb = (None, 0) if workspace is False else (workspace.data_ptr(), _ws_bytes(workspace))
        pp, _, _, ldp, sp, _ = _mat(P, "P")
        np_, _, _, ldn, sn, _ = _mat(N, "N")
        wp, _, _, ldw, sw, _ = _mat(W, "W")
        _check(lib.galore_project_back(pp, ldp, sp, np_, ldn, sn, wp, m, n, ldw, sw, r, lr, alpha, batch, wsp, wsb,
                                       _handle(ts)), "galore_project_back")
    return W


def galore_align_workspace_size(r: int, batch: int = 1) -> int:
    return int(lib.galore_align_workspace_size(r, batch))


def galore_align_projector(P_old: torch.Tensor, P_new: torch.Tensor, M=None, M_out=None, flips=None,
                           workspace=None, stream=None):
    """Subspace switch: negate in place the columns of P_new whose overlap with
    P_old is negative; with M (r x l, or batched), also return M re-expressed in
    the new basis, (P_new^T P_old) M, into M_out (allocated unless given).
    Returns (P_new, flips, M_out or None); flips is int32 (r,) or (batch, r)."""
    for t, nm in ((P_old, "P_old"), (P_new, "P_new"), (M, "M"), (M_out, "M_out")):
        if t is not None and t.dtype != torch.float32:
            raise ValueError("%s must be float32" % nm)
    s, r, _, _, batch = _geom(P_old, "P_old")
    _expect(P_new, "P_new", s, r, batch)
    if flips is not None:
        _expect_vec(flips, "flips", r, batch, torch.int32)
    l = 0
    if M is not None:
        _, l, _, _, _ = _geom(M, "M")
        _expect(M, "M", r, l, batch)
        if M_out is not None:
            _expect(M_out, "M_out", r, l, batch)
            if M_out.stride() != M.stride():
                raise ValueError("M_out must match M in shape and strides")
    elif M_out is not None:
        raise ValueError("M_out needs M")
    if workspace is not None:
        _ws_bytes(workspace)
    _on_device(None, P_old=P_old)
    _on_device(P_old.device, P_new=P_new, M=M, M_out=M_out, flips=flips, workspace=workspace)
    ts = _torch_stream(stream, P_old.device)
    with torch.cuda.stream(ts):
        if flips is None:
            flips = torch.empty((batch, r) if P_old.dim() == 3 else (r,), dtype=torch.int32, device=P_old.device)
        po, _, _, ldo, so, _ = _mat(P_old, "P_old")
        pn, _, _, ldn, sn, _ = _mat(P_new, "P_new")
        mi = mo = None
        ldm = sm = 0
        wsp, wsb = None, 0
        if M is not None:
            mi, _, _, ldm, sm, _ = _mat(M, "M")
            if M_out is None:
                M_out = torch.empty_like(M)
            mo = M_out.data_ptr()
            if workspace is None:
                workspace = torch.empty((galore_align_workspace_size(r, batch),), dtype=torch.uint8,
                                        device=M.device)
            wsp, wsb = workspace.data_ptr(), _ws_bytes(workspace)
        _check(lib.galore_align_projector(po, ldo, so, pn, ldn, sn, s, r, flips.data_ptr(), mi, mo, ldm, sm, l,
                                          batch, wsp, wsb, _handle(ts)), "galore_align_projector")
    return P_new, flips, (M_out if M is not None else None)


def galore_step_workspace_size(m: int, n: int, r: int, p: int, batch: int = 1, dtype=torch.float32,
                               flags: int = 0) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_step_workspace_size(m, n, r, p, batch, code, flags))


def galore_step(G: torch.Tensor, W: torch.Tensor, P: torch.Tensor, M: torch.Tensor, V: torch.Tensor, r: int,
                p: int, q: int, seed: int, tau: int, T: int, sketch_index0: int = 0, beta1: float = 0.9,
                beta2: float = 0.999, eps: float = 1e-8, lr: float = 1e-3, alpha: float = 0.25, flags: int = 0,
                info=None, workspace=None, stream=None, aux_stream=None):
    """One scheduled GaLore step (subspace update when tau % T == 0, then
    projection, low-rank Adam and back-projection); W, P, M, V are updated in
    place. Returns info (int32 per matrix, written at update steps)."""
    m, n, _, _, batch = _geom(G, "G")
    _dtype_code(G)
    s, l = min(m, n), max(m, n)
    _expect(W, "W", m, n, batch)
    _expect(P, "P", s, r, batch)
    _expect(M, "M", r, l, batch)
    _expect(V, "V", r, l, batch)
    if V.stride() != M.stride():
        raise ValueError("V must have M's shape and strides")
    if info is not None and (info.dtype != torch.int32 or info.dim() != 1 or info.numel() != batch
                             or not info.is_contiguous()):
        raise ValueError("info must be a contiguous int32 vector of the batch size")
    if workspace is not None:
        _ws_bytes(workspace)
    _on_device(None, G=G)
    _on_device(G.device, W=W, P=P, M=M, V=V, info=info, workspace=workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        if info is None:
            info = torch.zeros((batch,), dtype=torch.int32, device=G.device)
        if workspace is None:
            need = galore_step_workspace_size(m, n, r, p, batch, G.dtype, flags)
            workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=G.device)
        gp, _, _, ldg, sg, _ = _mat(G, "G")
        wp, _, _, ldw, sw, _ = _mat(W, "W")
        pp, _, _, ldp, sp, _ = _mat(P, "P")
        mp, _, _, ldm, sm, _ = _mat(M, "M")
        _check(lib.galore_step(gp, _dtype_code(G), m, n, ldg, sg, wp, ldw, sw, pp, ldp, sp, mp, V.data_ptr(), ldm,
                               sm, r, p, q, seed, sketch_index0, tau, T, beta1, beta2, eps, lr, alpha, flags,
                               info.data_ptr(), batch, workspace.data_ptr(), _ws_bytes(workspace), _handle(ts),
                               _handle(_aux(aux_stream, G.device))), "galore_step")
    return info


class QuantizedProjector:
    """Codes (uint8, (batch,) s x ldq bytes) and scales (fp32, (batch,) r) of a
    low-bit projector, as galore_quantize_projector writes them."""

    def __init__(self, codes: torch.Tensor, scales: torch.Tensor, bits: int, r: int):
        self.codes, self.scales, self.bits, self.r = codes, scales, bits, r

    def batch(self):
        return self.codes.shape[0] if self.codes.dim() == 3 else 1

    def rows(self):
        return self.codes.shape[-2]

    def _validate(self, s, batch):
        ldq = self.r if self.bits == 8 else (self.r + 1) // 2
        c = self.codes
        if c.dtype != torch.uint8 or c.dim() not in (2, 3) or c.shape[-1] < ldq or c.stride(-1) != 1:
            raise ValueError("codes must be uint8 (batch,) s x ldq with ldq >= %d" % ldq)
        if (self.rows(), self.batch()) != (s, batch):
            raise ValueError("the projector's codes hold %d matrices of %d rows; expected %d of %d"
                             % (self.batch(), self.rows(), batch, s))
        _expect_vec(self.scales, "scales", self.r, batch, torch.float32)

    def _args(self):
        c = self.codes
        if c.dim() == 2:
            return c.data_ptr(), c.stride(0), c.shape[0] * c.stride(0), self.scales.data_ptr(), self.r, self.bits
        return c.data_ptr(), c.stride(1), c.stride(0), self.scales.data_ptr(), self.scales.stride(0), self.bits


def galore_quantize_projector(P: torch.Tensor, bits: int = 8, stream=None) -> QuantizedProjector:
    """Symmetric per-column int8 / int4 codes and fp32 scales of the fp32 projector P."""
    if P.dtype != torch.float32:
        raise ValueError("P must be float32")
    s, r, ldp, sp, batch = _geom(P, "P")
    _on_device(None, P=P)
    ts = _torch_stream(stream, P.device)
    with torch.cuda.stream(ts):
        ldq = r if bits == 8 else (r + 1) // 2
        shape = (batch, s, ldq) if P.dim() == 3 else (s, ldq)
        codes = torch.empty(shape, dtype=torch.uint8, device=P.device)
        scales = torch.empty((batch, r) if P.dim() == 3 else (r,), dtype=torch.float32, device=P.device)
        _check(lib.galore_quantize_projector(P.data_ptr(), ldp, sp, s, r, bits, codes.data_ptr(), ldq, s * ldq,
                                             scales.data_ptr(), r, batch, _handle(ts)), "galore_quantize_projector")
    return QuantizedProjector(codes, scales, bits, r)


def galore_project_quantized_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_quantized_workspace_size(m, n, r, batch))


def galore_project_back_quantized_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_back_quantized_workspace_size(m, n, r, batch))


def galore_project_quantized(Pq: QuantizedProjector, G: torch.Tensor, R=None, workspace=None, stream=None):
    """R = Pq^T A with the low-bit projector ((r, l) or (batch, r, l))."""
    m, n, _, _, batch = _geom(G, "G")
    _dtype_code(G)
    s, l, r = min(m, n), max(m, n), Pq.r
    Pq._validate(s, batch)
    if R is not None:
        _expect(R, "R", r, l, batch)
    if workspace is not None:
        _ws_bytes(workspace)
    _on_device(None, G=G)
    _on_device(G.device, codes=Pq.codes, scales=Pq.scales, R=R, workspace=workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        if R is None:
            R = torch.empty((batch, r, l) if G.dim() == 3 else (r, l), dtype=torch.float32, device=G.device)
        if workspace is None:
            workspace = torch.empty((max(galore_project_quantized_workspace_size(m, n, r, batch), 1),),
                                    dtype=torch.uint8, device=G.device)
        gp, _, _, ldg, sg, _ = _mat(G, "G")
        rp, _, _, ldr, sr, _ = _mat(R, "R")
        qp, ldq, sq, scp, ss, bits = Pq._args()
        _check(lib.galore_project_quantized(qp, ldq, sq, scp, ss, bits, gp, _dtype_code(G), m, n, ldg, sg, r, rp,
                                            ldr, sr, batch, workspace.data_ptr(), _ws_bytes(workspace),
                                            _handle(ts)), "galore_project_quantized")
    return R


def galore_project_back_quantized(Pq: QuantizedProjector, N: torch.Tensor, W: torch.Tensor, lr: float, alpha: float,
                                  workspace=None, stream=None):
    """W <- W - lr * alpha * Pq N (transposed for m > n), in place."""
    m, n, _, _, batch = _geom(W, "W")
    s, l, r = min(m, n), max(m, n), Pq.r
    _expect(W, "W", m, n, batch)
    _expect(N, "N", r, l, batch)
    Pq._validate(s, batch)
    if workspace is not None:
        _ws_bytes(workspace)
    _on_device(None, W=W)
    _on_device(W.device, N=N, codes=Pq.codes, scales=Pq.scales, workspace=workspace)
    ts = _torch_stream(stream, W.device)
    with torch.cuda.stream(ts):
        if workspace is None:
            workspace = torch.empty((max(galore_project_back_quantized_workspace_size(m, n, r, batch), 1),),
                                    dtype=torch.uint8, device=W.device)
        np_, _, _, ldn, sn, _ = _mat(N, "N")
        wp, _, _, ldw, sw, _ = _mat(W, "W")
        qp, ldq, sq, scp, ss, bits = Pq._args()
        _check(lib.galore_project_back_quantized(qp, ldq, sq, scp, ss, bits, np_, ldn, sn, wp, m, n, ldw, sw, r, lr,
                                                 alpha, batch, workspace.data_ptr(), _ws_bytes(workspace),
                                                 _handle(ts)), "galore_project_back_quantized")
    return W


def galore_adam8_scale_count(rows: int, cols: int) -> int:
    return int(lib.galore_adam8_scale_count(rows, cols))


class Adam8State:
    """8-bit moments of a batch of rows x cols low-rank states: M8/V8 codes
    (uint8, (batch, rows, cols)) and block scales Ms/Vs (fp32, (batch, nblocks));
    zero-filled = the zero state."""

    def __init__(self, rows: int, cols: int, batch: int = 1, device="cuda"):
        nb = galore_adam8_scale_count(rows, cols)
        self.rows, self.cols, self.batch = rows, cols, batch
        self.M8 = torch.zeros((batch, rows, cols), dtype=torch.uint8, device=device)
        self.V8 = torch.zeros_like(self.M8)
        self.Ms = torch.zeros((batch, nb), dtype=torch.float32, device=device)
        self.Vs = torch.zeros_like(self.Ms)


def galore_lowrank_adam8_step(R: torch.Tensor, state: Adam8State, N=None, beta1=0.9, beta2=0.999, eps=1e-8, t=1,
                              stream=None):
    """8-bit block-wise Adam step on the state (updated in place); returns N (may be R itself)."""
    rows, cols, ld, st_, batch = _geom(R, "R")
    if R.dtype != torch.float32 or (N is not None and (N.shape != R.shape or N.stride() != R.stride()
                                                       or N.dtype != torch.float32)):
        raise ValueError("N must match R in shape, strides and dtype (float32)")
    if (state.rows, state.cols, state.batch) != (rows, cols, batch):
        raise ValueError("state does not match R")
    nb = galore_adam8_scale_count(rows, cols)
    for x, nm, shape, dt in ((state.M8, "M8", (batch, rows, cols), torch.uint8),
                             (state.V8, "V8", (batch, rows, cols), torch.uint8),
                             (state.Ms, "Ms", (batch, nb), torch.float32), (state.Vs, "Vs", (batch, nb), torch.float32)):
        if tuple(x.shape) != shape or x.dtype != dt or not x.is_contiguous():
            raise ValueError("8-bit state %s must be a contiguous %s tensor of shape %s" % (nm, dt, shape))
    _on_device(None, R=R)
    _on_device(R.device, N=N, M8=state.M8, V8=state.V8, Ms=state.Ms, Vs=state.Vs)
    ts = _torch_stream(stream, R.device)
    with torch.cuda.stream(ts):
        if N is None:
            N = torch.empty_like(R)
        _check(lib.galore_lowrank_adam8_step(R.data_ptr(), N.data_ptr(), ld, st_, state.M8.data_ptr(),
                                             state.Ms.data_ptr(), state.V8.data_ptr(), state.Vs.data_ptr(), rows, cols,
                                             batch, beta1, beta2, eps, t, _handle(ts)), "galore_lowrank_adam8_step")
    return N


def galore_svd_workspace_size(m: int, n: int, r: int, batch: int = 1, dtype=torch.float32) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_svd_workspace_size(m, n, r, batch, code))


def galore_svd_update(G: torch.Tensor, r: int, P=None, sigma=None, info=None, workspace=None, stream=None,
                      aux_stream=None):
    """Exact top-r SVD projector of G ((m, n) or (batch, m, n)); returns (P, sigma, info)."""
    m, n, _, _, batch = _geom(G, "G")
    _validate_update(G, r, P, sigma, info, workspace)
    ts = _torch_stream(stream, G.device)
    with torch.cuda.stream(ts):
        need = galore_svd_workspace_size(m, n, r, batch, G.dtype)
        P, sigma, info, workspace = _update_outputs(G, r, P, sigma, info, workspace, need)
        gp, _, _, ldg, sg, _ = _mat(G, "G")
        pp, _, _, ldp, sp, _ = _mat(P, "P")
        _check(lib.galore_svd_update(gp, _dtype_code(G), m, n, ldg, sg, r, pp, ldp, sp, sigma.data_ptr(),
                                     sigma.stride(0) if sigma.dim() == 2 else r, info.data_ptr(), batch,
                                     workspace.data_ptr(), _ws_bytes(workspace), _handle(ts),
                                     _handle(_aux(aux_stream, G.device))), "galore_svd_update")
    return P, sigma, info


def galore_probe_mfma_bf16(iterations: int, blocks: int, sink: torch.Tensor, stream=None) -> float:
    """Enqueue the bf16 matrix-core probe; returns its flops (time it on the stream)."""
    fl = ctypes.c_double(0.0)
    if sink.numel() < blocks * 256 or sink.dtype != torch.float32 or not sink.is_cuda:
        raise ValueError("sink must be a float32 device tensor of blocks * 256 elements")
    ts = _torch_stream(stream, sink.device)
    _check(lib.galore_probe_mfma_bf16(iterations, blocks, sink.data_ptr(), ctypes.byref(fl), _handle(ts)),
           "galore_probe_mfma_bf16")
    return fl.value


def galore_probe_copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    """Enqueue the streaming-copy probe of src into dst (same byte size)."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb or not (src.is_cuda and dst.is_cuda):
        raise ValueError("src and dst must be device tensors of the same byte size")
    ts = _torch_stream(stream, src.device)
    _check(lib.galore_probe_copy(src.data_ptr(), dst.data_ptr(), nb, _handle(ts)), "galore_probe_copy")
