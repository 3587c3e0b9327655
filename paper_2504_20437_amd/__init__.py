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
LIB_PATH = os.path.join(_HERE, "libgalore.so")

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
)

GALORE_STEP_ALIGN = 1
GALORE_STEP_REEXPRESS = 2

# galore_stage_t
STAGES = ("sketch", "product_A", "product_At", "gram", "cholesky", "triangular", "jacobi", "projector",
          "other", "operand")


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
                                       vp, i64, i64, vp, i64, vp, i32, vp, sz, vp]
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
                                i32, i32, i32, u64, u64, i64, i32, f32, f32, f32, f32, f32, i32, vp, i32, vp, sz, vp]
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
    lib.galore_svd_update.argtypes = [vp, i32, i64, i64, i64, i64, i32, vp, i64, i64, vp, i64, vp, i32, vp, sz, vp]
    lib.galore_svd_update.restype = ctypes.c_int
    lib.galore_probe_mfma_bf16.argtypes = [i64, i32, vp, ctypes.POINTER(ctypes.c_double), vp]
    lib.galore_probe_mfma_bf16.restype = ctypes.c_int
    lib.galore_probe_copy.argtypes = [vp, vp, sz, vp]
    lib.galore_probe_copy.restype = ctypes.c_int
    return lib


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libgalore.so is not built (run __graft_entry__.build()); "
                          "there is no fallback path")
    return _declare(ctypes.CDLL(LIB_PATH))


lib = _load()


def status_string(status: int) -> str:
    return lib.galore_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != GALORE_OK:
        raise GaloreError(status, where)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _mat(t: torch.Tensor, name: str):
    """(ptr, rows, cols, ld, batch_stride, batch) of a 2-D or 3-D row-major tensor."""
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dim() == 2:
        if t.stride(1) != 1:
            raise ValueError("%s must be row-major" % name)
        rows, cols = t.shape
        return t.data_ptr(), rows, cols, t.stride(0), rows * t.stride(0), 1
    if t.dim() == 3:
        if t.stride(2) != 1:
            raise ValueError("%s must be row-major" % name)
        b, rows, cols = t.shape
        return t.data_ptr(), rows, cols, t.stride(1), t.stride(0), b
    raise ValueError("%s must be 2-D or 3-D" % name)


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
    if out is None:
        out = torch.empty((l, k), dtype=torch.float32, device=device)
    _check(lib.galore_sketch(out.data_ptr(), l, k, seed, sketch_index, _stream(stream)), "galore_sketch")
    return out


def galore_rsvd_workspace_size(m: int, n: int, r: int, p: int, batch: int = 1, dtype=torch.float32) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_rsvd_workspace_size(m, n, r, p, batch, code))


def _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, stream):
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    s = min(m, n)
    dev = G.device
    if P is None:
        P = torch.empty((batch, s, r) if G.dim() == 3 else (s, r), dtype=torch.float32, device=dev)
    pp, prow, pcol, ldp, sp, pb = _mat(P, "P")
    if sigma is None:
        sigma = torch.empty((batch, r) if G.dim() == 3 else (r,), dtype=torch.float32, device=dev)
    if info is None:
        info = torch.empty((batch,), dtype=torch.int32, device=dev)
    need = galore_rsvd_workspace_size(m, n, r, p, batch, G.dtype)
    if workspace is None:
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=dev)
    args = (gp, _dtype_code(G), m, n, ldg, sg, r, p, q, seed, sketch_index0, pp, ldp, sp, sigma.data_ptr(),
            sigma.stride(0) if sigma.dim() == 2 else r, info.data_ptr(), batch, workspace.data_ptr(),
            workspace.numel(), _stream(stream))
    return args, P, sigma, info


def galore_rsvd_update(G: torch.Tensor, r: int, p: int, q: int, seed: int, sketch_index0: int = 0,
                       P=None, sigma=None, info=None, workspace=None, stream=None):
    """Subspace update of G ((m, n) or (batch, m, n)); returns (P, sigma, info)."""
    args, P, sigma, info = _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, stream)
    _check(lib.galore_rsvd_update(*args), "galore_rsvd_update")
    return P, sigma, info


def galore_rsvd_update_traced(G: torch.Tensor, r: int, p: int, q: int, seed: int, events, sketch_index0: int = 0,
                              P=None, sigma=None, info=None, workspace=None, stream=None):
    """galore_rsvd_update that also records ``events`` (an even-length list of
    torch.cuda.Event with timing enabled) around its stages; returns
    (P, sigma, info, stages) with stages[i] the stage name of the pair
    (events[2 i], events[2 i + 1])."""
    if len(events) % 2:
        raise ValueError("events must come in (start, end) pairs")
    cap = len(events) // 2
    args, P, sigma, info = _rsvd_args(G, r, p, q, seed, sketch_index0, P, sigma, info, workspace, stream)
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
    pp, s, r, ldp, sp, pb = _mat(P, "P")
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    l = max(m, n)
    if R is None:
        R = torch.empty((batch, r, l) if G.dim() == 3 else (r, l), dtype=torch.float32, device=G.device)
    rp, _, _, ldr, sr, _ = _mat(R, "R")
    if workspace is None:
        need = galore_project_workspace_size(m, n, r, batch, G.dtype)
        workspace = torch.empty((need,), dtype=torch.uint8, device=G.device) if need > 0 else False
    wp, wb = (None, 0) if workspace is False else (workspace.data_ptr(), workspace.numel())
    _check(lib.galore_project(pp, ldp, sp, gp, _dtype_code(G), m, n, ldg, sg, r, rp, ldr, sr, batch, wp, wb,
                              _stream(stream)), "galore_project")
    return R


def galore_lowrank_adam_step(R: torch.Tensor, M: torch.Tensor, V: torch.Tensor, N=None, beta1=0.9,
                             beta2=0.999, eps=1e-8, t=1, stream=None):
    """In-place M, V; returns N (may be R itself for an in-place update)."""
    if N is None:
        N = torch.empty_like(R)
    rp, rows, cols, ld, st_, batch = _mat(R, "R")
    for x, nm in ((M, "M"), (V, "V"), (N, "N")):
        if x.shape != R.shape or x.stride() != R.stride() or x.dtype != torch.float32:
            raise ValueError("%s must match R in shape, strides and dtype" % nm)
    _check(lib.galore_lowrank_adam_step(rp, M.data_ptr(), V.data_ptr(), N.data_ptr(), rows, cols, ld,
                                        st_, batch, beta1, beta2, eps, t, _stream(stream)),
           "galore_lowrank_adam_step")
    return N


def galore_project_back_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_back_workspace_size(m, n, r, batch))


def galore_project_back(P: torch.Tensor, N: torch.Tensor, W: torch.Tensor, lr: float, alpha: float,
                        workspace=None, stream=None):
    """W <- W - lr*alpha*(P N) (m <= n) or its transpose (m > n), in place. A
    workspace of galore_project_back_workspace_size bytes is allocated unless
    one is passed; workspace=False passes none."""
    pp, s, r, ldp, sp, _ = _mat(P, "P")
    np_, _, _, ldn, sn, _ = _mat(N, "N")
    wp, m, n, ldw, sw, batch = _mat(W, "W")
    if workspace is None:
        need = galore_project_back_workspace_size(m, n, r, batch)
        workspace = torch.empty((need,), dtype=torch.uint8, device=W.device) if need > 0 else False
    wsp, wsb = (None, 0) if workspace is False else (workspace.data_ptr(), workspace.numel())
    _check(lib.galore_project_back(pp, ldp, sp, np_, ldn, sn, wp, m, n, ldw, sw, r, lr, alpha, batch, wsp, wsb,
                                   _stream(stream)), "galore_project_back")
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
    po, s, r, ldo, so, batch = _mat(P_old, "P_old")
    pn, s2, r2, ldn, sn, batch2 = _mat(P_new, "P_new")
    if (s2, r2, batch2) != (s, r, batch):
        raise ValueError("P_new must match P_old in shape")
    if flips is None:
        flips = torch.empty((batch, r) if P_old.dim() == 3 else (r,), dtype=torch.int32, device=P_old.device)
    mi = mo = None
    ldm = sm = l = 0
    wsp, wsb = None, 0
    if M is not None:
        mi, mr, l, ldm, sm, mb = _mat(M, "M")
        if mr != r or mb != batch:
            raise ValueError("M must be r x l per projector")
        if M_out is None:
            M_out = torch.empty_like(M)
        mo, _, _, ldo2, so2, _ = _mat(M_out, "M_out")
        if M_out.shape != M.shape or (ldo2, so2) != (ldm, sm):
            raise ValueError("M_out must match M in shape and strides")
        if workspace is None:
            workspace = torch.empty((galore_align_workspace_size(r, batch),), dtype=torch.uint8, device=M.device)
        wsp, wsb = workspace.data_ptr(), workspace.numel()
    _check(lib.galore_align_projector(po, ldo, so, pn, ldn, sn, s, r, flips.data_ptr(), mi, mo, ldm, sm, l, batch,
                                      wsp, wsb, _stream(stream)), "galore_align_projector")
    return P_new, flips, (M_out if M is not None else None)


def galore_step_workspace_size(m: int, n: int, r: int, p: int, batch: int = 1, dtype=torch.float32,
                               flags: int = 0) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_step_workspace_size(m, n, r, p, batch, code, flags))


def galore_step(G: torch.Tensor, W: torch.Tensor, P: torch.Tensor, M: torch.Tensor, V: torch.Tensor, r: int,
                p: int, q: int, seed: int, tau: int, T: int, sketch_index0: int = 0, beta1: float = 0.9,
                beta2: float = 0.999, eps: float = 1e-8, lr: float = 1e-3, alpha: float = 0.25, flags: int = 0,
                info=None, workspace=None, stream=None):
    """One scheduled GaLore step (subspace update when tau % T == 0, then
    projection, low-rank Adam and back-projection); W, P, M, V are updated in
    place. Returns info (int32 per matrix, written at update steps)."""
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    for t, nm in ((W, "W"), (P, "P"), (M, "M"), (V, "V")):
        if t.dtype != torch.float32:
            raise ValueError("%s must be float32" % nm)
    wp, wm, wn, ldw, sw, wb = _mat(W, "W")
    pp, ps, pr, ldp, sp, pb = _mat(P, "P")
    mp, mr, ml, ldm, sm, mb = _mat(M, "M")
    vp_, vr, vl, ldv, sv, vb = _mat(V, "V")
    s, l = min(m, n), max(m, n)
    if (wm, wn, wb) != (m, n, batch) or (ps, pr, pb) != (s, r, batch) or (mr, ml, mb) != (r, l, batch):
        raise ValueError("W, P, M must match G in shape (m x n, s x r, r x l)")
    if (vr, vl, vb, ldv, sv) != (mr, ml, mb, ldm, sm):
        raise ValueError("V must have M's shape and strides")
    if info is None:
        info = torch.zeros((batch,), dtype=torch.int32, device=G.device)
    if workspace is None:
        need = galore_step_workspace_size(m, n, r, p, batch, G.dtype, flags)
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=G.device)
    _check(lib.galore_step(gp, _dtype_code(G), m, n, ldg, sg, wp, ldw, sw, pp, ldp, sp, mp, vp_, ldm, sm, r, p, q,
                           seed, sketch_index0, tau, T, beta1, beta2, eps, lr, alpha, flags, info.data_ptr(), batch,
                           workspace.data_ptr(), workspace.numel(), _stream(stream)), "galore_step")
    return info


class QuantizedProjector:
    """Codes (uint8, (batch,) s x ldq bytes) and scales (fp32, (batch,) r) of a
    low-bit projector, as galore_quantize_projector writes them."""

    def __init__(self, codes: torch.Tensor, scales: torch.Tensor, bits: int, r: int):
        self.codes, self.scales, self.bits, self.r = codes, scales, bits, r

    def _args(self):
        c = self.codes
        if c.dim() == 2:
            return c.data_ptr(), c.stride(0), c.shape[0] * c.stride(0), self.scales.data_ptr(), self.r, self.bits
        return c.data_ptr(), c.stride(1), c.stride(0), self.scales.data_ptr(), self.scales.stride(0), self.bits


def galore_quantize_projector(P: torch.Tensor, bits: int = 8, stream=None) -> QuantizedProjector:
    """Symmetric per-column int8 / int4 codes and fp32 scales of the fp32 projector P."""
    if P.dtype != torch.float32:
        raise ValueError("P must be float32")
    pp, s, r, ldp, sp, batch = _mat(P, "P")
    ldq = r if bits == 8 else (r + 1) // 2
    shape = (batch, s, ldq) if P.dim() == 3 else (s, ldq)
    codes = torch.empty(shape, dtype=torch.uint8, device=P.device)
    scales = torch.empty((batch, r) if P.dim() == 3 else (r,), dtype=torch.float32, device=P.device)
    _check(lib.galore_quantize_projector(pp, ldp, sp, s, r, bits, codes.data_ptr(), ldq, s * ldq, scales.data_ptr(),
                                         r, batch, _stream(stream)), "galore_quantize_projector")
    return QuantizedProjector(codes, scales, bits, r)


def galore_project_quantized_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_quantized_workspace_size(m, n, r, batch))


def galore_project_back_quantized_workspace_size(m: int, n: int, r: int, batch: int = 1) -> int:
    return int(lib.galore_project_back_quantized_workspace_size(m, n, r, batch))


def galore_project_quantized(Pq: QuantizedProjector, G: torch.Tensor, R=None, workspace=None, stream=None):
    """R = Pq^T A with the low-bit projector ((r, l) or (batch, r, l))."""
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    l, r = max(m, n), Pq.r
    if R is None:
        R = torch.empty((batch, r, l) if G.dim() == 3 else (r, l), dtype=torch.float32, device=G.device)
    rp, _, _, ldr, sr, _ = _mat(R, "R")
    if workspace is None:
        workspace = torch.empty((max(galore_project_quantized_workspace_size(m, n, r, batch), 1),), dtype=torch.uint8,
                                device=G.device)
    qp, ldq, sq, scp, ss, bits = Pq._args()
    _check(lib.galore_project_quantized(qp, ldq, sq, scp, ss, bits, gp, _dtype_code(G), m, n, ldg, sg, r, rp, ldr,
                                        sr, batch, workspace.data_ptr(), workspace.numel(), _stream(stream)),
           "galore_project_quantized")
    return R


def galore_project_back_quantized(Pq: QuantizedProjector, N: torch.Tensor, W: torch.Tensor, lr: float, alpha: float,
                                  workspace=None, stream=None):
    """W <- W - lr * alpha * Pq N (transposed for m > n), in place."""
    np_, r, l, ldn, sn, batch = _mat(N, "N")
    wp, m, n, ldw, sw, wb = _mat(W, "W")
    if workspace is None:
        workspace = torch.empty((max(galore_project_back_quantized_workspace_size(m, n, r, batch), 1),),
                                dtype=torch.uint8, device=W.device)
    qp, ldq, sq, scp, ss, bits = Pq._args()
    _check(lib.galore_project_back_quantized(qp, ldq, sq, scp, ss, bits, np_, ldn, sn, wp, m, n, ldw, sw, r, lr,
                                             alpha, batch, workspace.data_ptr(), workspace.numel(), _stream(stream)),
           "galore_project_back_quantized")
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
    if N is None:
        N = torch.empty_like(R)
    rp, rows, cols, ld, st_, batch = _mat(R, "R")
    if N.shape != R.shape or N.stride() != R.stride() or N.dtype != torch.float32 or R.dtype != torch.float32:
        raise ValueError("N must match R in shape, strides and dtype (float32)")
    if (state.rows, state.cols, state.batch) != (rows, cols, batch):
        raise ValueError("state does not match R")
    for x in (state.M8, state.V8, state.Ms, state.Vs):
        if not x.is_contiguous():
            raise ValueError("8-bit state must be contiguous")
    _check(lib.galore_lowrank_adam8_step(rp, N.data_ptr(), ld, st_, state.M8.data_ptr(), state.Ms.data_ptr(),
                                         state.V8.data_ptr(), state.Vs.data_ptr(), rows, cols, batch, beta1, beta2,
                                         eps, t, _stream(stream)), "galore_lowrank_adam8_step")
    return N


def galore_svd_workspace_size(m: int, n: int, r: int, batch: int = 1, dtype=torch.float32) -> int:
    code = GALORE_BF16 if dtype in (torch.bfloat16, GALORE_BF16, "bf16") else GALORE_F32
    return int(lib.galore_svd_workspace_size(m, n, r, batch, code))


def galore_svd_update(G: torch.Tensor, r: int, P=None, sigma=None, info=None, workspace=None, stream=None):
    """Exact top-r SVD projector of G ((m, n) or (batch, m, n)); returns (P, sigma, info)."""
    gp, m, n, ldg, sg, batch = _mat(G, "G")
    s = min(m, n)
    dev = G.device
    if P is None:
        P = torch.empty((batch, s, r) if G.dim() == 3 else (s, r), dtype=torch.float32, device=dev)
    pp, _, _, ldp, sp, _ = _mat(P, "P")
    if sigma is None:
        sigma = torch.empty((batch, r) if G.dim() == 3 else (r,), dtype=torch.float32, device=dev)
    if info is None:
        info = torch.empty((batch,), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty((max(galore_svd_workspace_size(m, n, r, batch, G.dtype), 1),), dtype=torch.uint8,
                                device=dev)
    _check(lib.galore_svd_update(gp, _dtype_code(G), m, n, ldg, sg, r, pp, ldp, sp, sigma.data_ptr(),
                                 sigma.stride(0) if sigma.dim() == 2 else r, info.data_ptr(), batch,
                                 workspace.data_ptr(), workspace.numel(), _stream(stream)), "galore_svd_update")
    return P, sigma, info


def galore_probe_mfma_bf16(iterations: int, blocks: int, sink: torch.Tensor, stream=None) -> float:
    """Enqueue the bf16 matrix-core probe; returns its flops (time it on the stream)."""
    fl = ctypes.c_double(0.0)
    if sink.numel() < blocks * 256 or sink.dtype != torch.float32 or not sink.is_cuda:
        raise ValueError("sink must be a float32 device tensor of blocks * 256 elements")
    _check(lib.galore_probe_mfma_bf16(iterations, blocks, sink.data_ptr(), ctypes.byref(fl), _stream(stream)),
           "galore_probe_mfma_bf16")
    return fl.value


def galore_probe_copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    """Enqueue the streaming-copy probe of src into dst (same byte size)."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb or not (src.is_cuda and dst.is_cuda):
        raise ValueError("src and dst must be device tensors of the same byte size")
    _check(lib.galore_probe_copy(src.data_ptr(), dst.data_ptr(), nb, _stream(stream)), "galore_probe_copy")
