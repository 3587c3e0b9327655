"""C-ABI contract checks that need no GPU: the library loads, exports every
function include/galore.h declares, and rejects invalid arguments on the host
before enqueuing anything (each call below has exactly one invalid argument;
the pointers are never dereferenced because validation fails first)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "galore.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(galore_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_four_hot_path_calls():
    names = declared_functions()
    for fn in ("galore_rsvd_update", "galore_project", "galore_lowrank_adam_step", "galore_project_back"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    import paper_2504_20437_amd as gl
    lib = ctypes.CDLL(gl.LIB_PATH)
    for fn in declared_functions():
        assert hasattr(lib, fn), fn
    assert set(gl.EXPORTED) == set(declared_functions())


def test_status_strings_and_version():
    import paper_2504_20437_amd as gl
    assert gl.status_string(0) == "GALORE_OK"
    assert gl.status_string(-3) == "GALORE_ERR_WORKSPACE"
    assert gl.galore_version() >= 100


def test_workspace_size():
    import paper_2504_20437_amd as gl
    one = gl.galore_rsvd_workspace_size(4096, 11008, 1024, 32, 1)
    assert one > 0
    assert gl.galore_rsvd_workspace_size(4096, 11008, 1024, 32, 4) >= 4 * one - 4096
    assert gl.galore_rsvd_workspace_size(11008, 4096, 1024, 32, 1) == one       # orientation
    assert gl.galore_rsvd_workspace_size(10, 20, 11, 0, 1) == 0                  # r > s
    assert gl.galore_rsvd_workspace_size(0, 20, 1, 0, 1) == 0
    assert gl.galore_rsvd_workspace_size(5000, 9000, 4090, 10, 1) == 0           # sketch too wide
    # the exact Gram's digit planes (3 x k x l bytes, padded) must stay below 2^31
    assert gl.galore_rsvd_workspace_size(1056, 600000, 1024, 32, 1) > 0
    assert gl.galore_rsvd_workspace_size(1056, 700000, 1024, 32, 1) == 0
    assert gl.galore_rsvd_workspace_size(300000, 4096, 4000, 96, 1) == 0
    # a bf16 gradient also keeps room for its transposed copy and the split sketch operand
    import torch
    bf = gl.galore_rsvd_workspace_size(4096, 11008, 1024, 32, 1, torch.bfloat16)
    assert bf >= one + 2 * 4096 * 11008 + 3 * 2 * 1056 * 11008
    assert gl.galore_rsvd_workspace_size(11008, 4096, 1024, 32, 1, torch.bfloat16) == bf
    assert gl.lib.galore_rsvd_workspace_size(64, 96, 8, 4, 1, 7) == 0            # bad dtype


FAKE = 0x1000   # never dereferenced: every call below fails validation first
NULL = None


def rsvd(**kw):
    import paper_2504_20437_amd as gl
    a = dict(G=FAKE, g_dtype=0, m=64, n=96, ldg=96, stride_g=64 * 96, r=8, p=4, q=1, seed=1, si=0,
             P=FAKE, ldp=8, stride_p=64 * 8, sigma=FAKE, stride_sigma=8, info=FAKE, batch=1,
             ws=FAKE - FAKE % 256 + 256, ws_bytes=1 << 40, stream=NULL)
    a.update(kw)
    return gl.lib.galore_rsvd_update(a["G"], a["g_dtype"], a["m"], a["n"], a["ldg"], a["stride_g"], a["r"],
                                     a["p"], a["q"], a["seed"], a["si"], a["P"], a["ldp"], a["stride_p"],
                                     a["sigma"], a["stride_sigma"], a["info"], a["batch"], a["ws"],
                                     a["ws_bytes"], a["stream"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(G=NULL), -1), (dict(P=NULL), -1), (dict(ws=NULL), -1), (dict(g_dtype=7), -1),
    (dict(m=0), -2), (dict(n=-3), -2), (dict(r=0), -2), (dict(r=65), -2), (dict(p=-1), -2),
    (dict(q=-1), -2), (dict(ldg=95), -2), (dict(ldp=7), -2), (dict(batch=0), -2),
    (dict(batch=2, stride_g=10), -2), (dict(r=8, p=5000), -2),
    (dict(m=1056, n=700000, ldg=700000, stride_g=0, r=1024, p=32, ldp=1024, stride_p=0, stride_sigma=1024), -2),
    (dict(ws_bytes=1000), -3), (dict(ws=FAKE + 8), -3),
])
def test_rsvd_rejects(kw, code):
    assert rsvd(**kw) == code


def test_project_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_project
    ok = dict(P=FAKE, ldp=8, sp=0, G=FAKE, dt=0, m=64, n=96, ldg=96, sg=0, r=8, R=FAKE, ldr=96, sr=0, b=1)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(a["P"], a["ldp"], a["sp"], a["G"], a["dt"], a["m"], a["n"], a["ldg"], a["sg"], a["r"],
                 a["R"], a["ldr"], a["sr"], a["b"], a.get("ws"), a.get("wb", 0), None)
    assert call(P=NULL) == -1 and call(G=NULL) == -1 and call(R=NULL) == -1 and call(dt=3) == -1
    assert call(r=65) == -2 and call(ldr=95) == -2 and call(ldp=7) == -2 and call(ldg=10) == -2
    assert call(m=0) == -2 and call(b=0) == -2 and call(b=2) == -2
    # right projector: l = m
    assert call(m=200, n=96, ldr=199) == -2
    # bf16 gradient: a workspace, when given, must be aligned and large enough
    need = gl.galore_project_workspace_size(64, 96, 8, 1, "bf16")
    assert call(dt=1, ws=FAKE, wb=need - 1) == -3 and call(dt=1, ws=FAKE + 8, wb=need) == -3


def test_project_workspace_size():
    import paper_2504_20437_amd as gl
    assert gl.galore_project_workspace_size(64, 96, 8, 1, "f32") == 0
    one = gl.galore_project_workspace_size(64, 96, 8, 1, "bf16")
    assert one >= 3 * 8 * 64 * 2 and one % 256 == 0
    assert gl.galore_project_workspace_size(64, 96, 8, 4, "bf16") >= 4 * 3 * 8 * 64 * 2
    # right projector: planes of P^T span s = n
    assert gl.galore_project_workspace_size(96, 64, 8, 1, "bf16") == one
    assert gl.galore_project_workspace_size(64, 96, 65, 1, "bf16") == 0
    assert gl.galore_project_workspace_size(0, 96, 8, 1, "bf16") == 0


def test_adam_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_lowrank_adam_step
    ok = dict(R=FAKE, M=FAKE, V=FAKE, N=FAKE, rows=4, cols=8, ld=8, st=32, b=1, b1=0.9, b2=0.999,
              eps=1e-8, t=1)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(a["R"], a["M"], a["V"], a["N"], a["rows"], a["cols"], a["ld"], a["st"], a["b"],
                 a["b1"], a["b2"], a["eps"], a["t"], None)
    for kw in (dict(R=NULL), dict(M=NULL), dict(V=NULL), dict(N=NULL), dict(b1=1.0), dict(b1=-0.1),
               dict(b2=1.0), dict(eps=0.0), dict(eps=float("nan")), dict(b1=float("inf")), dict(t=0)):
        assert call(**kw) == -1, kw
    for kw in (dict(rows=0), dict(cols=0), dict(ld=7), dict(b=0), dict(b=2, st=31)):
        assert call(**kw) == -2, kw


def test_project_back_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_project_back
    ok = dict(P=FAKE, ldp=8, sp=0, N=FAKE, ldn=96, sn=0, W=FAKE, m=64, n=96, ldw=96, sw=0, r=8,
              lr=1e-3, al=0.25, b=1)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(a["P"], a["ldp"], a["sp"], a["N"], a["ldn"], a["sn"], a["W"], a["m"], a["n"], a["ldw"],
                 a["sw"], a["r"], a["lr"], a["al"], a["b"], a.get("ws"), a.get("wb", 0), None)
    for kw in (dict(P=NULL), dict(N=NULL), dict(W=NULL), dict(lr=float("nan")), dict(al=float("inf"))):
        assert call(**kw) == -1, kw
    for kw in (dict(r=65), dict(ldn=95), dict(ldw=95), dict(ldp=7), dict(m=0), dict(b=0), dict(b=2)):
        assert call(**kw) == -2, kw
    need = gl.galore_project_back_workspace_size(64, 96, 8, 1)
    assert call(ws=FAKE, wb=need - 1) == -3 and call(ws=FAKE + 8, wb=need) == -3


def test_project_back_workspace_size():
    import paper_2504_20437_amd as gl
    one = gl.galore_project_back_workspace_size(64, 96, 8, 1)
    assert one >= 3 * 2 * 8 * (64 + 96) and one % 256 == 0
    assert gl.galore_project_back_workspace_size(96, 64, 8, 1) == one        # orientation
    assert gl.galore_project_back_workspace_size(64, 96, 8, 3) >= 3 * 3 * 2 * 8 * (64 + 96)
    assert gl.galore_project_back_workspace_size(64, 96, 65, 1) == 0        # r > s
    assert gl.galore_project_back_workspace_size(64, 0, 8, 1) == 0


def test_sketch_rejects():
    import paper_2504_20437_amd as gl
    assert gl.lib.galore_sketch(NULL, 10, 4, 1, 0, None) == -1
    assert gl.lib.galore_sketch(FAKE, 0, 4, 1, 0, None) == -2
    assert gl.lib.galore_sketch(FAKE, 10, 0, 1, 0, None) == -2


def test_rsvd_traced_rejects():
    """The traced variant validates its own arguments first, then those of the
    subspace update (capacity 0 records nothing)."""
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_rsvd_update_traced
    base = [FAKE, 0, 64, 96, 96, 64 * 96, 8, 4, 1, 1, 0, FAKE, 8, 64 * 8, FAKE, 8, FAKE, 1,
            FAKE - FAKE % 256 + 256, 1 << 40, None, None]
    cnt = ctypes.c_int32(-1)
    ev = (ctypes.c_void_p * 2)(FAKE, None)          # second handle missing
    st = (ctypes.c_int32 * 1)()
    assert f(*base, ev, st, 1, ctypes.byref(cnt)) == -1
    assert f(*base, None, st, 1, ctypes.byref(cnt)) == -1
    assert f(*base, ev, None, 1, ctypes.byref(cnt)) == -1
    assert f(*base, ev, st, -1, ctypes.byref(cnt)) == -1
    assert f(*base, ev, st, 0, None) == -1
    bad = list(base)
    bad[6] = 65                                      # r > s: rejected by the update itself
    assert f(*bad, None, None, 0, ctypes.byref(cnt)) == -2
    assert cnt.value == 0


def test_align_workspace_size():
    import paper_2504_20437_amd as gl
    one = gl.galore_align_workspace_size(32, 1)
    assert one >= 32 * 32 * 4 and one % 256 == 0
    assert gl.galore_align_workspace_size(32, 5) == 5 * one
    assert gl.galore_align_workspace_size(0, 1) == 0
    assert gl.galore_align_workspace_size(32, 0) == 0


def test_align_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_align_projector
    ws = FAKE - FAKE % 256 + 256
    need = gl.galore_align_workspace_size(8, 1)
    ok = dict(Po=FAKE, ldo=8, so=0, Pn=FAKE + 4096, ldn=8, sn=0, s=64, r=8, fl=None, Mi=FAKE + 8192,
              Mo=FAKE + 65536, ldm=96, sm=0, l=96, b=1, ws=ws, wb=need)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(a["Po"], a["ldo"], a["so"], a["Pn"], a["ldn"], a["sn"], a["s"], a["r"], a["fl"], a["Mi"],
                 a["Mo"], a["ldm"], a["sm"], a["l"], a["b"], a["ws"], a["wb"], None)
    for kw in (dict(Po=NULL), dict(Pn=NULL), dict(Mi=NULL), dict(Mo=NULL),
               dict(Mo=FAKE + 8192 + 4 * 96 * 7)):                            # M_out overlaps M_in
        assert call(**kw) == -1, kw
    for kw in (dict(s=0), dict(r=0), dict(r=65), dict(ldo=7), dict(ldn=7), dict(b=0), dict(b=2),
               dict(b=2, so=64 * 8, sn=64 * 8, sm=8 * 96 - 1), dict(l=0), dict(ldm=95)):
        assert call(**kw) == -2, kw
    for kw in (dict(ws=NULL), dict(ws=ws + 8), dict(wb=need - 1)):
        assert call(**kw) == -3, kw


def test_step_workspace_size():
    import paper_2504_20437_amd as gl
    import torch
    base = gl.galore_step_workspace_size(64, 96, 8, 4, 1)
    rs = gl.galore_rsvd_workspace_size(64, 96, 8, 4, 1)
    assert base >= rs and base % 256 == 0
    al = gl.galore_step_workspace_size(64, 96, 8, 4, 1, flags=1)
    rx = gl.galore_step_workspace_size(64, 96, 8, 4, 1, flags=3)
    assert al >= base + 64 * 8 * 4 and rx >= al + 8 * 96 * 4
    assert gl.galore_step_workspace_size(96, 64, 8, 4, 1, flags=3) == rx            # orientation
    assert gl.galore_step_workspace_size(64, 96, 8, 4, 2, torch.bfloat16) >= gl.galore_rsvd_workspace_size(
        64, 96, 8, 4, 2, torch.bfloat16)
    assert gl.galore_step_workspace_size(64, 96, 8, 4, 1, flags=2) == 0             # REEXPRESS needs ALIGN
    assert gl.galore_step_workspace_size(64, 96, 8, 4, 1, flags=4) == 0
    assert gl.galore_step_workspace_size(64, 96, 65, 0, 1) == 0
    assert gl.galore_step_workspace_size(64, 96, 8, 4, 0) == 0


def test_step_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_step
    ws = FAKE - FAKE % 256 + 256
    need = gl.galore_step_workspace_size(64, 96, 8, 4, 1, flags=3)
    ok = dict(G=FAKE, dt=0, m=64, n=96, ldg=96, sg=0, W=FAKE, ldw=96, sw=0, P=FAKE, ldp=8, sp=0, M=FAKE, V=FAKE,
              ldm=96, sm=0, r=8, p=4, q=1, seed=1, idx=0, tau=0, T=10, b1=0.9, b2=0.999, eps=1e-8, lr=1e-3, al=0.25,
              fl=3, info=None, b=1, ws=ws, wb=need)
    keys = list(ok)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(*[a[k] for k in keys], None, None)
    for kw in (dict(G=NULL), dict(W=NULL), dict(P=NULL), dict(M=NULL), dict(V=NULL), dict(dt=2), dict(tau=-1),
               dict(T=0), dict(fl=2), dict(fl=8), dict(b1=1.0), dict(b2=-0.5), dict(eps=0.0),
               dict(lr=float("nan")), dict(al=float("inf"))):
        assert call(**kw) == -1, kw
    for kw in (dict(m=0), dict(r=0), dict(r=65), dict(p=-1), dict(q=-1), dict(p=4090), dict(ldg=95), dict(ldw=95),
               dict(ldp=7), dict(ldm=95), dict(b=0), dict(b=2), dict(b=2, sg=64 * 96, sw=64 * 96, sp=64 * 8)):
        assert call(**kw) == -2, kw
    for kw in (dict(ws=NULL), dict(ws=ws + 8), dict(wb=need - 1)):
        assert call(**kw) == -3, kw


def test_quantized_workspace_sizes():
    import paper_2504_20437_amd as gl
    pw = gl.galore_project_quantized_workspace_size(64, 96, 8, 1)
    bw = gl.galore_project_back_quantized_workspace_size(64, 96, 8, 1)
    assert pw >= 64 * 8 * 4 and pw % 256 == 0            # holds the fp32 dequantised projector
    assert bw >= 64 * 8 * 2 + 3 * 96 * 8 * 2 and bw % 256 == 0
    assert gl.galore_project_quantized_workspace_size(96, 64, 8, 1) == pw
    assert gl.galore_project_quantized_workspace_size(64, 96, 65, 1) == 0
    assert gl.galore_project_back_quantized_workspace_size(64, 96, 8, 0) == 0


def test_quantize_projector_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_quantize_projector
    ok = dict(P=FAKE, ldp=8, sp=0, s=64, r=8, bits=8, Q=FAKE, ldq=8, sq=0, sc=FAKE, ss=0, b=1)
    keys = list(ok)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(*[a[k] for k in keys], None)
    for kw in (dict(P=NULL), dict(Q=NULL), dict(sc=NULL), dict(bits=2), dict(bits=16)):
        assert call(**kw) == -1, kw
    for kw in (dict(s=0), dict(r=0), dict(r=65), dict(ldp=7), dict(ldq=7), dict(bits=4, ldq=3), dict(b=0), dict(b=2),
               dict(b=2, sp=512, sq=512, ss=7)):
        assert call(**kw) == -2, kw


def test_project_quantized_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_project_quantized
    ws = FAKE - FAKE % 256 + 256
    need = gl.galore_project_quantized_workspace_size(64, 96, 8, 1)
    ok = dict(Q=FAKE, ldq=8, sq=0, sc=FAKE, ss=0, bits=8, G=FAKE, dt=0, m=64, n=96, ldg=96, sg=0, r=8, R=FAKE,
              ldr=96, sr=0, b=1, ws=ws, wb=need)
    keys = list(ok)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(*[a[k] for k in keys], None)
    for kw in (dict(Q=NULL), dict(sc=NULL), dict(G=NULL), dict(R=NULL), dict(bits=3), dict(dt=5)):
        assert call(**kw) == -1, kw
    for kw in (dict(m=0), dict(r=65), dict(ldg=95), dict(ldr=95), dict(ldq=7), dict(bits=4, ldq=3), dict(b=2)):
        assert call(**kw) == -2, kw
    for kw in (dict(ws=NULL), dict(ws=ws + 8), dict(wb=need - 1)):
        assert call(**kw) == -3, kw


def test_project_back_quantized_rejects():
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_project_back_quantized
    ws = FAKE - FAKE % 256 + 256
    need = gl.galore_project_back_quantized_workspace_size(64, 96, 8, 1)
    ok = dict(Q=FAKE, ldq=8, sq=0, sc=FAKE, ss=0, bits=8, N=FAKE, ldn=96, sn=0, W=FAKE, m=64, n=96, ldw=96, sw=0,
              r=8, lr=1e-3, al=0.25, b=1, ws=ws, wb=need)
    keys = list(ok)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(*[a[k] for k in keys], None)
    for kw in (dict(Q=NULL), dict(sc=NULL), dict(N=NULL), dict(W=NULL), dict(bits=1), dict(lr=float("nan")),
               dict(al=float("inf"))):
        assert call(**kw) == -1, kw
    for kw in (dict(m=0), dict(r=65), dict(ldn=95), dict(ldw=95), dict(ldq=7), dict(b=2)):
        assert call(**kw) == -2, kw
    for kw in (dict(ws=NULL), dict(ws=ws + 8), dict(wb=need - 1)):
        assert call(**kw) == -3, kw


def test_adam8_rejects_and_scale_count():
    import paper_2504_20437_amd as gl
    assert gl.galore_adam8_scale_count(1024, 11008) == 5504
    assert gl.galore_adam8_scale_count(3, 700) == 2
    assert gl.galore_adam8_scale_count(0, 5) == 0
    f = gl.lib.galore_lowrank_adam8_step
    ok = dict(R=FAKE, N=FAKE, ld=96, st=0, M8=FAKE, Ms=FAKE, V8=FAKE, Vs=FAKE, rows=8, cols=96, b=1, b1=0.9,
              b2=0.999, eps=1e-8, t=1)
    keys = list(ok)
    def call(**kw):
        a = dict(ok); a.update(kw)
        return f(*[a[k] for k in keys], None)
    for kw in (dict(R=NULL), dict(N=NULL), dict(M8=NULL), dict(Ms=NULL), dict(V8=NULL), dict(Vs=NULL),
               dict(b1=1.0), dict(b2=-0.1), dict(eps=0.0), dict(eps=float("nan")), dict(t=0)):
        assert call(**kw) == -1, kw
    for kw in (dict(rows=0), dict(cols=0), dict(ld=95), dict(b=0), dict(b=2, st=8 * 96 - 1)):
        assert call(**kw) == -2, kw


def test_svd_workspace_and_rejects():
    import paper_2504_20437_amd as gl
    assert gl.galore_svd_workspace_size(64, 96, 8, 1) == gl.galore_rsvd_workspace_size(64, 96, 8, 56, 1)
    assert gl.galore_svd_workspace_size(96, 64, 8, 1) == gl.galore_rsvd_workspace_size(96, 64, 8, 56, 1)
    assert gl.galore_svd_workspace_size(4097, 5000, 8, 1) == 0
    assert gl.galore_svd_workspace_size(64, 96, 65, 1) == 0
    f = gl.lib.galore_svd_update
    args = [FAKE, 0, 64, 96, 96, 0, 8, FAKE, 8, 0, None, 8, None, 1, FAKE - FAKE % 256 + 256, 1 << 40, None, None]
    assert f(*args[:2], 4097, 5000, 5000, *args[5:]) == -2
    assert f(*args[:6], 65, *args[7:]) == -2
    assert f(NULL, *args[1:]) == -1


def test_probe_rejects():
    import ctypes
    import paper_2504_20437_amd as gl
    fl = ctypes.c_double(0.0)
    f = gl.lib.galore_probe_mfma_bf16
    assert f(10, 4, None, ctypes.byref(fl), None) == -1
    assert f(10, 4, FAKE, None, None) == -1
    assert f(0, 4, FAKE, ctypes.byref(fl), None) == -2
    assert f(10, 0, FAKE, ctypes.byref(fl), None) == -2
    g = gl.lib.galore_probe_copy
    assert g(None, FAKE, 256, None) == -1
    assert g(FAKE, FAKE + 8, 256, None) == -1          # misaligned and overlapping
    assert g(FAKE, FAKE + 128, 256, None) == -1        # overlapping
    assert g(FAKE, FAKE + 4096, 0, None) == -2
    assert g(FAKE, FAKE + 4096, 100, None) == -2


# ---------------------------------------------------------------- binding-side validation (no GPU)


def _t(*shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=dtype or torch.float32)


def _raises(fn, match):
    with pytest.raises(ValueError, match=match):
        fn()


def test_binding_rejects_mismatched_tensors():
    """The binding checks every tensor against the shapes derived from G (or W)
    before any pointer reaches the library: a 2-D output with a batched G, a
    sigma of the wrong length, an int64 info, a float64 P, a transposed N or a
    low-bit projector of another batch would otherwise make the kernels write
    past the end of a buffer. Host tensors of the right shapes are rejected as
    not being on the device."""
    import torch
    import paper_2504_20437_amd as gl
    G = _t(3, 64, 96)                                   # batch 3, s = 64, l = 96
    r = 8
    # subspace update
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, P=_t(64, r)), "P must hold 3 matrices")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, P=_t(3, 64, r, dtype=torch.float64)), "P must be")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, sigma=_t(r)), "sigma must have shape")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, sigma=_t(3, r + 1)), "sigma must have shape")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, info=_t(3, dtype=torch.int64)), "info must be")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1, info=_t(2, dtype=torch.int32)), "info must be")
    _raises(lambda: gl.galore_rsvd_update(G.double(), r, 4, 1, 1), "gradient dtype")
    _raises(lambda: gl.galore_rsvd_update(G, r, 4, 1, 1), "device tensor")
    _raises(lambda: gl.galore_svd_update(G, r, P=_t(3, 96, r)), "P must hold")
    _raises(lambda: gl.galore_rsvd_update_traced(G, r, 4, 1, 1, [], sigma=_t(r)), "sigma must have shape")
    # projection
    _raises(lambda: gl.galore_project(_t(3, 64, r), G, R=_t(r, 96)), "R must hold 3 matrices")
    _raises(lambda: gl.galore_project(_t(3, 96, r), G), "P must hold")
    _raises(lambda: gl.galore_project(_t(64, r), G), "P must hold 3 matrices")
    _raises(lambda: gl.galore_project(_t(3, 64, r), G, R=_t(3, r, 96, dtype=torch.float64)), "R must be")
    _raises(lambda: gl.galore_project(_t(3, 64, r), G), "device tensor")
    # back-projection: W (m x n) fixes s, l and the batch
    W = _t(3, 64, 96)
    _raises(lambda: gl.galore_project_back(_t(3, 64, r), _t(r, 96), W, 1e-3, 0.25), "N must hold 3 matrices")
    _raises(lambda: gl.galore_project_back(_t(3, 64, r), _t(3, 96, r), W, 1e-3, 0.25), "N must hold")
    _raises(lambda: gl.galore_project_back(_t(3, 64, r), _t(3, r, 96), _t(3, 64, 96, dtype=torch.float64),
                                           1e-3, 0.25), "W must be")
    _raises(lambda: gl.galore_project_back(_t(3, 64, r), _t(3, r, 96), W, 1e-3, 0.25), "device tensor")
    # Adam
    R = _t(3, r, 96)
    _raises(lambda: gl.galore_lowrank_adam_step(R, _t(3, r, 95), _t(3, r, 96)), "M must match")
    _raises(lambda: gl.galore_lowrank_adam_step(R.double(), R.double(), R.double()), "R must be float32")
    # scheduled step
    Pm, M, V = _t(3, 64, r), _t(3, r, 96), _t(3, r, 96)
    _raises(lambda: gl.galore_step(G, _t(64, 96), Pm, M, V, r, 4, 1, 1, 0, 10), "W must hold 3 matrices")
    _raises(lambda: gl.galore_step(G, W, Pm, M, V, r, 4, 1, 1, 0, 10, info=_t(3, dtype=torch.int64)), "info")
    # subspace switch
    _raises(lambda: gl.galore_align_projector(Pm, _t(3, 64, r + 1)), "P_new must hold")
    _raises(lambda: gl.galore_align_projector(Pm, Pm.clone(), M, M_out=_t(3, r, 97)), "M_out must hold")
    _raises(lambda: gl.galore_align_projector(Pm, Pm.clone(), M_out=M), "M_out needs M")
    # low-bit projector: codes of another batch, scales of another rank
    q = gl.QuantizedProjector(_t(2, 64, r, dtype=torch.uint8), _t(2, r), 8, r)
    _raises(lambda: gl.galore_project_quantized(q, G), "codes hold 2 matrices")
    _raises(lambda: gl.galore_project_back_quantized(q, _t(3, r, 96), W, 1e-3, 0.25), "codes hold 2 matrices")
    q3 = gl.QuantizedProjector(_t(3, 64, r, dtype=torch.uint8), _t(3, r - 1), 8, r)
    _raises(lambda: gl.galore_project_quantized(q3, G), "scales must have shape")
    q3 = gl.QuantizedProjector(_t(3, 64, r, dtype=torch.uint8), _t(3, r), 8, r)
    _raises(lambda: gl.galore_project_back_quantized(q3, _t(3, r + 1, 96), W, 1e-3, 0.25), "N must hold")
    # 8-bit Adam state of another shape
    st = gl.Adam8State.__new__(gl.Adam8State)
    st.rows, st.cols, st.batch = r, 96, 3
    st.M8, st.V8 = _t(3, r, 96, dtype=torch.uint8), _t(3, r, 96, dtype=torch.uint8)
    st.Ms, st.Vs = _t(3, 2), _t(3, 1)
    _raises(lambda: gl.galore_lowrank_adam8_step(R, st), "8-bit state Ms")


def test_project_noalloc_rejects_before_any_device_call():
    """The no-allocation projection validates like galore_project and rejects a
    bf16 workspace need above its fixed scratch (64 MiB) with WORKSPACE, all on
    the host (the pointers below are never dereferenced)."""
    import paper_2504_20437_amd as gl
    f = gl.lib.galore_project_noalloc
    cap = gl.galore_project_noalloc_max_bytes()
    assert cap == 64 << 20
    m, n, r = 4096, 11008, 1024
    one = gl.galore_project_workspace_size(m, n, r, 1, 1)
    assert 2 * one <= cap < 3 * one                      # two bench-shaped matrices fit, three do not
    args = lambda **kw: [kw.get(k, v) for k, v in (("P", FAKE), ("ldp", r), ("sp", m * r), ("G", FAKE), ("dt", 1),
                                                     ("m", m), ("n", n), ("ldg", n), ("sg", m * n), ("r", r),
                                                     ("R", FAKE), ("ldr", n), ("sr", r * n), ("b", 1), ("st", None))]
    assert f(*args(b=3)) == -3
    assert f(*args(P=NULL)) == -1 and f(*args(R=NULL)) == -1 and f(*args(dt=5)) == -1
    assert f(*args(r=4097)) == -2 and f(*args(ldg=n - 1)) == -2 and f(*args(b=2, sg=m * n - 1)) == -2
