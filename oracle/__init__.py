"""CPU oracle for the GaLore 2 hot path -- TEST INFRASTRUCTURE ONLY.

Plain fp64 C (``galore_oracle.c``) behind ctypes. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package; the product library never does.  It shares no code with the HIP
path.  Every function takes and returns float64 numpy arrays; callers widen the
exact stored fp32/bf16 values (and fp32 hyper-parameters) before calling.

What each function follows (paper = "GaLore 2", Su et al. 2025):
  sketch           Gaussian test matrix of Halko, Martinsson & Tropp 2011 (§4),
                   drawn by Philox4x64-10 + Box-Muller
  householder_qr   thin QR, Golub & Van Loan §5.2
  jacobi_left_svd  one-sided (Hestenes) Jacobi SVD, left singular vectors
  rsvd_update      paper §3 / Alg. 1 subspace selection with the randomized SVD
                   of paper §4.1.2 (Halko et al. Alg. 4.4 + Alg. 5.1)
  project          paper §3, R = P^T G
  adam             paper §3 moments + Alg. 1 bias correction
  project_back     paper §3, W <- W + eta alpha P N (applied as W -= lr alpha P N
                   for the autograd gradient)
  align_projector  subspace switch: signs of a new P matched to the previous P
                   (paper §4.1.3 sign indeterminacy, Alg. 1 schedule), optional
                   first-moment re-expression in the new basis
  quantize_projector / pack_codes / dequantize_projector
                   low-bit projector (paper §4.2, after Q-GaLore): symmetric
                   per-column int8 / int4 codes, decisions in binary32, and the
                   byte layout the library stores them in
  fp8_encode / fp8_decode
                   OCP 8-bit floating point E4M3 (fmt 0) and E5M2 (fmt 1),
                   round half to even with saturation
  adam8            8-bit block-wise low-rank Adam (paper §4.2, after the
                   8-bit Adam of Dettmers et al.): M in E4M3, V in E5M2, one
                   binary32 scale per block
  galore_step      one step of paper Alg. 1: a new projector every T steps
                   (optionally followed by the subspace switch), projection,
                   Adam with bias exponent tau + 1, back-projection
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "galore_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "liboracle.so")
# GALORE_ORACLE_LIB selects another build of galore_oracle.c (the tests'
# sanitizer build, see build_sanitized); by default the in-tree liboracle.so
_LIB_PATH = os.environ.get("GALORE_ORACLE_LIB") or _DEFAULT_LIB
_lib = None

_f64p = ctypes.POINTER(ctypes.c_double)
_u64p = ctypes.POINTER(ctypes.c_uint64)


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2 + OpenMP); a build selected by
    GALORE_ORACLE_LIB is used as it is."""
    if _LIB_PATH != _DEFAULT_LIB:
        return _LIB_PATH
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def build_sanitized(out_path: str) -> str:
    """The oracle with AddressSanitizer + UndefinedBehaviorSanitizer (gcc; any
    finding aborts). Load it with GALORE_ORACLE_LIB=out_path in a process that
    preloads gcc's libasan."""
    subprocess.check_call(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fopenmp", "-shared", "-fPIC", "-o", out_path, _SRC, "-lm"])
    return out_path


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = ctypes.c_int
        lib.orc_set_num_threads.argtypes = [ctypes.c_int]
        lib.orc_set_num_threads.restype = None
        lib.orc_philox4x64_10.argtypes = [_u64p, _u64p, _u64p]
        lib.orc_philox4x64_10.restype = None
        lib.orc_normal_from_words.argtypes = [u64, u64]
        lib.orc_normal_from_words.restype = ctypes.c_double
        lib.orc_normal_pair_from_words.argtypes = [u64, u64, _f64p]
        lib.orc_normal_pair_from_words.restype = None
        lib.orc_round_bf16.argtypes = [ctypes.c_double]
        lib.orc_round_bf16.restype = ctypes.c_double
        lib.orc_sketch.argtypes = [i64, i64, u64, u64, _f64p]
        lib.orc_sketch.restype = None
        lib.orc_householder_qr.argtypes = [i64, i64, _f64p, _f64p, _f64p]
        lib.orc_householder_qr.restype = None
        lib.orc_jacobi_left_svd.argtypes = [i64, i64, _f64p, _f64p, _f64p, ctypes.c_int]
        lib.orc_jacobi_left_svd.restype = ctypes.c_int
        lib.orc_canonical_signs.argtypes = [_f64p, i64, i64]
        lib.orc_canonical_signs.restype = None
        lib.orc_rsvd_update.argtypes = [_f64p, i64, i64, i32, i32, i32, u64, u64, _f64p, _f64p]
        lib.orc_rsvd_update.restype = ctypes.c_int
        lib.orc_project.argtypes = [_f64p, _f64p, i64, i64, i32, _f64p]
        lib.orc_project.restype = None
        lib.orc_adam.argtypes = [_f64p, _f64p, _f64p, _f64p, i64, ctypes.c_double, ctypes.c_double,
                                 ctypes.c_double, i64]
        lib.orc_adam.restype = None
        lib.orc_project_back.argtypes = [_f64p, _f64p, _f64p, i64, i64, i32, ctypes.c_double,
                                         ctypes.c_double]
        lib.orc_project_back.restype = None
        lib.orc_align_projector.argtypes = [_f64p, _f64p, i64, i64, ctypes.POINTER(ctypes.c_int32), _f64p, _f64p,
                                            i64]
        lib.orc_align_projector.restype = None
        lib.orc_quantize_projector.argtypes = [_f64p, i64, i64, i32, ctypes.POINTER(ctypes.c_int32),
                                               ctypes.POINTER(ctypes.c_float)]
        lib.orc_quantize_projector.restype = None
        lib.orc_fp8_encode.argtypes = [ctypes.c_float, i32]
        lib.orc_fp8_encode.restype = ctypes.c_uint8
        lib.orc_fp8_decode.argtypes = [ctypes.c_uint8, i32]
        lib.orc_fp8_decode.restype = ctypes.c_double
        u8p, f32p = ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_float)
        lib.orc_adam8.argtypes = [_f64p, u8p, f32p, u8p, f32p, _f64p, i64, i64, ctypes.c_double, ctypes.c_double,
                                  ctypes.c_double, i64, f32p, f32p]
        lib.orc_adam8.restype = None
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_f64p)


def num_threads() -> int:
    """OpenMP threads the oracle's loops run on."""
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the oracle's later OpenMP loops (n > 0)."""
    _load().orc_set_num_threads(int(n))


def philox4x64_10(counter, key) -> np.ndarray:
    lib = _load()
    c = np.ascontiguousarray(np.asarray(counter, dtype=np.uint64).reshape(4))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint64).reshape(2))
    out = np.zeros(4, dtype=np.uint64)
    lib.orc_philox4x64_10(c.ctypes.data_as(_u64p), k.ctypes.data_as(_u64p), out.ctypes.data_as(_u64p))
    return out


def normal_from_words(x0: int, x1: int) -> float:
    return float(_load().orc_normal_from_words(int(x0), int(x1)))


def normal_pair_from_words(x0: int, x1: int):
    """(r cos 2 pi u2, r sin 2 pi u2): both normals of the Box-Muller pair."""
    z = np.zeros(2)
    _load().orc_normal_pair_from_words(x0, x1, _ptr(z))
    return float(z[0]), float(z[1])


def round_bf16(z: float) -> float:
    """The bfloat16 value nearest to the fp64 z (ties to even), rounded once."""
    return float(_load().orc_round_bf16(float(z)))


def sketch(l: int, k: int, seed: int, sketch_index: int = 0) -> np.ndarray:
    """Omega (l x k) as fp64 holding bfloat16-rounded N(0,1) draws (four rows per
    Philox block: two Box-Muller pairs)."""
    out = np.zeros((l, k), dtype=np.float64)
    _load().orc_sketch(l, k, seed, sketch_index, _ptr(out))
    return out


def householder_qr(Y):
    Y = _f64(Y)
    s, k = Y.shape
    assert s >= k
    Q = np.zeros((s, k))
    R = np.zeros((k, k))
    _load().orc_householder_qr(s, k, _ptr(Y), _ptr(Q), _ptr(R))
    return Q, R


def jacobi_left_svd(B, max_sweeps: int = 60):
    """Left singular vectors U (k x k) and sigma (k) of B (k x l, k <= l); sweeps (-1 = no conv.)."""
    B = _f64(B)
    k, l = B.shape
    assert k <= l
    U = np.zeros((k, k))
    sig = np.zeros(k)
    sweeps = _load().orc_jacobi_left_svd(k, l, _ptr(B), _ptr(U), _ptr(sig), max_sweeps)
    return U, sig, sweeps


def canonical_signs(P) -> np.ndarray:
    P = _f64(P).copy()
    _load().orc_canonical_signs(_ptr(P), P.shape[0], P.shape[1])
    return P


def rsvd_update(G, r: int, p: int, q: int, seed: int, sketch_index: int = 0):
    """(P (s x r), sigma (r), sweeps) for the m x n gradient G."""
    G = _f64(G)
    m, n = G.shape
    s = min(m, n)
    P = np.zeros((s, r))
    sig = np.zeros(r)
    sweeps = _load().orc_rsvd_update(_ptr(G), m, n, r, p, q, seed, sketch_index, _ptr(P), _ptr(sig))
    return P, sig, sweeps


def project(P, G) -> np.ndarray:
    P = _f64(P)
    G = _f64(G)
    m, n = G.shape
    r = P.shape[1]
    R = np.zeros((r, max(m, n)))
    _load().orc_project(_ptr(P), _ptr(G), m, n, r, _ptr(R))
    return R


def adam(R, M, V, beta1: float, beta2: float, eps: float, t: int):
    """Returns (M_new, V_new, N); inputs are not modified."""
    R = _f64(R)
    M = _f64(M).copy()
    V = _f64(V).copy()
    N = np.zeros_like(R)
    _load().orc_adam(_ptr(R), _ptr(M), _ptr(V), _ptr(N), R.size, beta1, beta2, eps, t)
    return M, V, N


def project_back(P, N, W, lr: float, alpha: float) -> np.ndarray:
    """Returns the updated W (input not modified)."""
    P = _f64(P)
    N = _f64(N)
    W = _f64(W).copy()
    m, n = W.shape
    r = P.shape[1]
    _load().orc_project_back(_ptr(P), _ptr(N), _ptr(W), m, n, r, lr, alpha)
    return W


def align_projector(P_old, P_new, M=None):
    """Subspace switch: (P_new with each column's sign matched to P_old's,
    flips (r, 1 = negated), M re-expressed in the new basis (P_new^T P_old) M
    or None). Inputs are not modified."""
    P_old = _f64(P_old)
    P_new = _f64(P_new).copy()
    s, r = P_old.shape
    assert P_new.shape == (s, r)
    flips = np.zeros(r, dtype=np.int32)
    fp = flips.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    if M is None:
        _load().orc_align_projector(_ptr(P_old), _ptr(P_new), s, r, fp, None, None, 0)
        return P_new, flips, None
    M = _f64(M)
    assert M.shape[0] == r
    M_out = np.zeros_like(M)
    _load().orc_align_projector(_ptr(P_old), _ptr(P_new), s, r, fp, _ptr(M), _ptr(M_out), M.shape[1])
    return P_new, flips, M_out


def galore_step(G, W, P, M, V, r: int, p: int, q: int, seed: int, tau: int, T: int, sketch_index: int = 0,
                beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, lr: float = 1e-3, alpha: float = 0.25,
                align: bool = False, reexpress: bool = False, P_given=None):
    """One step of paper Alg. 1 at 0-based step tau for one m x n matrix.
    Returns (W, P, M, V) after the step (inputs are not modified). P may be
    None when tau is an update step. P_given, if set, replaces the subspace
    update's raw projector (a test that injects the projector of another
    implementation); alignment and re-expression still apply to it."""
    W = _f64(W).copy()
    M = _f64(M).copy()
    V = _f64(V).copy()
    if tau % T == 0:
        P_new = _f64(P_given) if P_given is not None else rsvd_update(G, r, p, q, seed, sketch_index)[0]
        if align and tau > 0:
            P_new, _, M_re = align_projector(P, P_new, M if reexpress else None)
            if reexpress:
                M = M_re
        P = P_new
    P = _f64(P)
    R = project(P, G)
    M, V, N = adam(R, M, V, beta1, beta2, eps, tau + 1)
    W = project_back(P, N, W, lr, alpha)
    return W, P, M, V


def quantize_projector(P, bits: int):
    """(codes (s x r int32), scales (r float32)) of the fp32 projector P: scale_j
    = max_i |P_ij| / qmax, code = round-half-even(P / scale) clamped to
    [-qmax, qmax], qmax = 2^(bits-1) - 1, every step in binary32."""
    assert bits in (4, 8)
    P = _f64(P)
    s, r = P.shape
    codes = np.zeros((s, r), dtype=np.int32)
    scales = np.zeros(r, dtype=np.float32)
    _load().orc_quantize_projector(_ptr(P), s, r, bits, codes.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                   scales.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
    return codes, scales


def dequantize_projector(codes, scales) -> np.ndarray:
    """code * scale, exact in fp64."""
    return np.asarray(codes, dtype=np.float64) * np.asarray(scales, dtype=np.float64)[None, :]


def pack_codes(codes, bits: int) -> np.ndarray:
    """The bytes of a row-major s x r code matrix as stored: 8 bits -> one
    two's-complement byte per code; 4 bits -> two codes per byte, column 2c in
    the low nibble and 2c + 1 in the high nibble (4-bit two's complement), a
    zero high nibble when r is odd. Shape (s, ceil(r * bits / 8)), uint8."""
    codes = np.asarray(codes, dtype=np.int64)
    s, r = codes.shape
    if bits == 8:
        return (codes & 0xFF).astype(np.uint8)
    out = np.zeros((s, (r + 1) // 2), dtype=np.uint8)
    for c in range(r):
        nib = (codes[:, c] & 0xF).astype(np.uint8)
        out[:, c // 2] |= nib if c % 2 == 0 else (nib << 4).astype(np.uint8)
    return out


E4M3, E5M2 = 0, 1
ADAM8_BLOCK = 2048


def fp8_encode(x, fmt: int) -> np.ndarray:
    """uint8 codes of the binary32 values x (OCP E4M3 or E5M2, RNE, saturating)."""
    x = np.asarray(x, dtype=np.float32)
    lib = _load()
    return np.array([lib.orc_fp8_encode(float(v), fmt) for v in x.ravel()], dtype=np.uint8).reshape(x.shape)


def fp8_decode(c, fmt: int) -> np.ndarray:
    c = np.asarray(c, dtype=np.uint8)
    lib = _load()
    return np.array([lib.orc_fp8_decode(int(v), fmt) for v in c.ravel()], dtype=np.float64).reshape(c.shape)


def adam8(R, M8, Ms, V8, Vs, beta1: float, beta2: float, eps: float, t: int, block: int = ADAM8_BLOCK):
    """One 8-bit block-wise Adam step on the row-major state of one matrix.
    Returns (M8, Ms, V8, Vs, N, M32, V32): the new codes and block scales, the
    update N (fp64), and the binary32 moments that were encoded. Inputs are not
    modified."""
    R = _f64(R)
    count = R.size
    M8 = np.ascontiguousarray(M8, dtype=np.uint8).ravel().copy()
    V8 = np.ascontiguousarray(V8, dtype=np.uint8).ravel().copy()
    Ms = np.ascontiguousarray(Ms, dtype=np.float32).ravel().copy()
    Vs = np.ascontiguousarray(Vs, dtype=np.float32).ravel().copy()
    nb = (count + block - 1) // block
    assert M8.size == count and V8.size == count and Ms.size == nb and Vs.size == nb
    N = np.zeros(count)
    m32 = np.zeros(count, dtype=np.float32)
    v32 = np.zeros(count, dtype=np.float32)
    u8p, f32p = ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_float)
    _load().orc_adam8(_ptr(R), M8.ctypes.data_as(u8p), Ms.ctypes.data_as(f32p), V8.ctypes.data_as(u8p),
                      Vs.ctypes.data_as(f32p), _ptr(N), count, block, beta1, beta2, eps, t, m32.ctypes.data_as(f32p),
                      v32.ctypes.data_as(f32p))
    sh = R.shape
    return (M8.reshape(sh), Ms, V8.reshape(sh), Vs, N.reshape(sh), m32.reshape(sh), v32.reshape(sh))
