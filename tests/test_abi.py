"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2505_23884_amd as P
from paper_2505_23884_amd.binding import make_desc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lact.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(lact_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    L = P.lib()
    names = _declared()
    assert {"lact_forward", "lact_forward_momentum", "lact_forward_schedule", "lact_prologue", "lact_rmsnorm_out",
            "lact_workspace_bytes"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_version():
    assert P.lib().lact_version().decode().startswith("lact-gfx950")


GOOD = dict(B=2, H=2, d=64, h=128, n_kv=1000, n_q=1100, chunk=256, order=0, use_muon=False,
            ns_steps=5, io_dtype=0)


@pytest.mark.parametrize("field,value,code", [
    ("B", 0, -1), ("H", -1, -1), ("d", 0, -1), ("d", 12, -4), ("h", 4100, -4), ("h", 20, -4),
    ("d", 40, -4), ("h", 160 + 8, -4), ("B", 1 << 20, -4),
    ("n_kv", -1, -1), ("n_q", 999, -1), ("chunk", 0, -1), ("order", 2, -1),
    ("ns_steps", 17, -1), ("ns_steps", -1, -1), ("io_dtype", 3, -1),
])
def test_descriptor_validation(field, value, code):
    kw = dict(GOOD)
    kw[field] = value
    d = make_desc(**kw)
    assert P.check_desc(d) == code
    err = ctypes.c_int(0)
    assert P.lib().lact_workspace_bytes(ctypes.byref(d), ctypes.byref(err)) == 0
    assert err.value == code


def test_launch_grids_that_overflow_are_rejected():
    # 2^20 instances of 4096 x 4096 fast weights: the gradient's grid alone
    # would pass 2^31 blocks; the largest realistic shapes stay accepted
    big = dict(GOOD, B=1 << 10, H=1 << 10, d=4096, h=4096, n_kv=1024, n_q=1024)
    assert P.check_desc(make_desc(**big)) == -4
    nvs = dict(GOOD, B=1, H=1, d=768, h=1536, n_kv=1 << 30, n_q=(1 << 30) + 4096, chunk=1 << 30, order=1)
    assert P.check_desc(make_desc(**nvs)) == 0


def test_fp32_envelope_is_multiples_of_8():
    # bf16 I/O needs multiples of 32 (d = 40 is rejected above); fp32 I/O takes 8
    kw = dict(GOOD, d=40, h=24, io_dtype=1)
    assert P.check_desc(make_desc(**kw)) == 0
    kw = dict(GOOD, d=96, h=160)
    assert P.check_desc(make_desc(**kw)) == 0


def test_workspace_grows_with_the_chunk():
    a = P.workspace_bytes(make_desc(**GOOD))
    b = P.workspace_bytes(make_desc(**dict(GOOD, chunk=512)))
    c = P.workspace_bytes(make_desc(**dict(GOOD, io_dtype=1)))
    assert 0 < a < b and a < c and a % 256 == 0


def _fwd(desc, q=0x1000, k=0x2000, v=0x3000, eta=0x4000, w1=0x5000, w2=0x6000, w3=0x7000,
         o=0x8000, ws=0x10000, nbytes=None):
    L = P.lib()
    if nbytes is None:
        nbytes = P.workspace_bytes(desc) if P.check_desc(desc) == 0 else 0
    vp = ctypes.c_void_p
    return L.lact_forward(ctypes.byref(desc), vp(q), vp(k), vp(v), vp(eta), vp(w1), vp(w2), vp(w3),
                          vp(o), vp(ws), ctypes.c_size_t(nbytes), vp(0))


def test_forward_argument_errors_before_any_hip_call():
    d = make_desc(**GOOD)
    assert _fwd(d, q=0) == -1
    assert _fwd(d, w2=0) == -1
    assert _fwd(d, eta=0) == -1
    assert _fwd(d, k=0x2008) == -2          # misaligned tensor
    assert _fwd(d, eta=0x4002) == -2        # eta needs 4-byte alignment
    assert _fwd(d, ws=0x10010) == -2        # workspace needs 256-byte alignment
    assert _fwd(d, ws=0) == -3
    assert _fwd(d, nbytes=P.workspace_bytes(d) - 1) == -3
    bad = make_desc(**dict(GOOD, d=12))
    assert _fwd(bad, nbytes=1 << 30) == -4
    assert ctypes.cast(P.lib().lact_strerror(-3), ctypes.c_char_p).value


def _fwd_mom(desc, beta=0x9000, m1=0xA000, m2=0xB000, m3=0xC000, nbytes=None, **kw):
    L = P.lib()
    a = dict(q=0x1000, k=0x2000, v=0x3000, eta=0x4000, w1=0x5000, w2=0x6000, w3=0x7000, o=0x8000,
             ws=0x10000)
    a.update(kw)
    if nbytes is None:
        nbytes = P.workspace_bytes(desc) if P.check_desc(desc) == 0 else 0
    vp = ctypes.c_void_p
    return L.lact_forward_momentum(ctypes.byref(desc), vp(a["q"]), vp(a["k"]), vp(a["v"]), vp(a["eta"]),
                                   vp(beta), vp(a["w1"]), vp(a["w2"]), vp(a["w3"]), vp(m1), vp(m2), vp(m3),
                                   vp(a["o"]), vp(a["ws"]), ctypes.c_size_t(nbytes), vp(0))


def test_momentum_argument_errors_before_any_hip_call():
    d = make_desc(**GOOD)
    assert _fwd_mom(d, beta=0) == -1        # beta is required when there are key tokens
    assert _fwd_mom(d, m2=0) == -1
    assert _fwd_mom(d, m3=0xC008) == -2     # momentum is read as float4
    assert _fwd_mom(d, beta=0x9002) == -2   # beta needs 4-byte alignment
    assert _fwd_mom(d, q=0) == -1           # the checks of lact_forward apply too
    assert _fwd_mom(d, ws=0) == -3
    assert _fwd_mom(make_desc(**dict(GOOD, d=12)), nbytes=1 << 30) == -4
    # no key tokens: beta may be NULL, the momentum may not
    d0 = make_desc(**dict(GOOD, n_kv=0))
    assert _fwd_mom(d0, m1=0, beta=0) == -1


def _fwd_sched(desc, segs, m1=0, beta=0, nbytes=None, ws=0x10000, q=0x1000):
    from paper_2505_23884_amd.binding import LactSegment
    L = P.lib()
    arr = (LactSegment * max(len(segs), 1))(*[LactSegment(m, r, b, e) for m, r, b, e in segs])
    if nbytes is None:
        nbytes = P.workspace_bytes(desc) if P.check_desc(desc) == 0 else 0
    vp = ctypes.c_void_p
    m = [vp(m1), vp(0xB000 if m1 else 0), vp(0xC000 if m1 else 0)]
    return L.lact_forward_schedule(ctypes.byref(desc), arr, ctypes.c_int64(len(segs)), vp(q), vp(0x2000),
                                   vp(0x3000), vp(0x4000), vp(beta), vp(0x5000), vp(0x6000), vp(0x7000), *m,
                                   vp(0x8000), vp(ws), ctypes.c_size_t(nbytes), vp(0))


def test_schedule_segment_errors_before_any_hip_call():
    d = make_desc(**dict(GOOD, n_kv=256, n_q=300, chunk=64))
    assert _fwd_sched(d, [(4, 0, 0, 8)]) == -1            # unknown mode
    assert _fwd_sched(d, [(0, 1, 0, 8)]) == -1            # reserved field set
    assert _fwd_sched(d, [(3, 5, 5, 0)]) == -1            # empty range
    assert _fwd_sched(d, [(3, 0, -1, 8)]) == -1           # negative begin
    assert _fwd_sched(d, [(2, 0, 200, 265)]) == -1        # update past n_kv
    assert _fwd_sched(d, [(2, 0, 0, 65)]) == -1           # update longer than chunk
    assert _fwd_sched(d, [(3, 0, 0, 301)]) == -1          # apply past n_q
    assert _fwd_sched(d, [(1, 0, 0, 64)], m1=0xA000) == -1   # momentum without beta
    assert _fwd_sched(d, [(1, 0, 0, 64)], ws=0) == -3     # segments fine, workspace missing
    assert _fwd_sched(d, [(3, 0, 0, 300)], q=0x1008, ws=0x10000) == -2
    L = P.lib()
    assert L.lact_forward_schedule(ctypes.byref(d), None, ctypes.c_int64(2), *([ctypes.c_void_p(0x1000)] * 13),
                                   ctypes.c_size_t(1 << 30), ctypes.c_void_p(0)) == -1   # NULL segments


def test_per_matrix_rate_flag_is_validated():
    assert P.check_desc(make_desc(**dict(GOOD, eta_per_matrix=1))) == 0
    bad = make_desc(**GOOD)
    bad.eta_per_matrix = 2
    assert P.check_desc(bad) == -1


def test_prologue_and_norm_errors_before_any_hip_call():
    L = P.lib()
    vp, f = ctypes.c_void_p, ctypes.c_float
    d = make_desc(**GOOD)
    pro = lambda qkv=0x1000, lr=0x2000, bias=0.0, braw=0, q=0x3000, k=0x4000, v=0x5000, eta=0x6000, beta=0: \
        L.lact_prologue(ctypes.byref(d), vp(qkv), vp(lr), f(bias), vp(braw), vp(q), vp(k), vp(v), vp(eta), vp(beta),
                        vp(0))
    assert pro(qkv=0) == -1
    assert pro(eta=0) == -1
    assert pro(braw=0x7000) == -1                 # beta_raw without beta
    assert pro(bias=float("nan")) == -1
    assert pro(bias=float("inf")) == -1
    assert pro(q=0x3008) == -2
    assert pro(lr=0x2002) == -2
    rms = lambda o=0x1000, w=0, eps=1e-6, y=0x2000: L.lact_rmsnorm_out(ctypes.byref(d), vp(o), vp(w), f(eps), vp(y), vp(0))
    assert rms(o=0) == -1
    assert rms(eps=-1.0) == -1
    assert rms(eps=float("nan")) == -1
    assert rms(y=0x2004) == -2
    assert rms(w=0x3001) == -2
    bad = make_desc(**dict(GOOD, d=12))
    assert L.lact_rmsnorm_out(ctypes.byref(bad), vp(0x1000), vp(0), f(1e-6), vp(0x2000), vp(0)) == -4


def test_linear_fast_weight_descriptor():
    ok = make_desc(**dict(GOOD, h=64, fast_weight=1))
    assert P.check_desc(ok) == 0
    assert P.check_desc(make_desc(**dict(GOOD, fast_weight=1))) == -1               # h != d
    assert P.check_desc(make_desc(**dict(GOOD, h=64, fast_weight=1, eta_per_matrix=1))) == -1
    assert P.check_desc(make_desc(**dict(GOOD, fast_weight=2))) == -1
    # W2, W3 may be NULL for the linear weight (validation reaches the workspace)
    assert _fwd(ok, w2=0, w3=0, ws=0) == -3
    assert _fwd(make_desc(**GOOD), w2=0, ws=0) == -1
    assert P.workspace_bytes(ok) < P.workspace_bytes(make_desc(**dict(GOOD, h=64)))


def test_timing_api_without_launches():
    P.timing_reset()
    assert P.timing_read(0) == (0, 0.0, 0.0)
    assert P.lib().lact_timing_read(9, None, None, None) == -1


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(P.LactError):
        P.load_library(str(tmp_path / "missing.so"))


def _fwd_noalloc(desc, q=0x1000, k=0x2000, v=0x3000, eta=0x4000, w1=0x5000, w2=0x6000, w3=0x7000, o=0x8000):
    vp = ctypes.c_void_p
    return P.lib().lact_forward_noalloc(ctypes.byref(desc), vp(q), vp(k), vp(v), vp(eta), vp(w1), vp(w2), vp(w3),
                                        vp(o), vp(0))


def test_noalloc_errors_before_any_hip_call():
    # the binding's constant is the header's
    m = re.search(r"#define LACT_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == P.binding.NOALLOC_SCRATCH_BYTES
    d = make_desc(**GOOD)
    assert _fwd_noalloc(d, q=0) == -1
    assert _fwd_noalloc(d, w2=0) == -1
    assert _fwd_noalloc(d, k=0x2008) == -2
    assert _fwd_noalloc(make_desc(**dict(GOOD, d=12))) == -4
    # a call that needs more than the fixed array: rejected before any HIP call
    lm = dict(GOOD, B=4, H=4, d=512, h=512, n_kv=32768, n_q=32768, chunk=2048)
    assert P.workspace_bytes(make_desc(**lm)) > P.binding.NOALLOC_SCRATCH_BYTES
    assert _fwd_noalloc(make_desc(**lm)) == -6
    assert _fwd_noalloc(make_desc(**lm), q=0) == -1       # argument errors come first
    assert "scratch" in P.lib().lact_strerror(-6).decode()
    # one LM sequence (B = 1, H = 4) fits, with Muon too
    one = make_desc(**dict(lm, B=1, use_muon=True))
    assert P.workspace_bytes(one) <= P.binding.NOALLOC_SCRATCH_BYTES


def _bwd(desc, nbytes=None, **kw):
    a = dict(q=0x1000, k=0x2000, v=0x3000, eta=0x4000, w0=0x5000, do=0x6000, dwf=0, dq=0x7000, dk=0x8000,
             dv=0x9000, deta=0xA000, dw0=0xB000, ws=0x10000)
    a.update(kw)
    if nbytes is None:
        err = ctypes.c_int(0)
        nbytes = P.lib().lact_backward_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    vp = ctypes.c_void_p
    return P.lib().lact_backward_linear(ctypes.byref(desc), *(vp(a[n]) for n in (
        "q", "k", "v", "eta", "w0", "do", "dwf", "dq", "dk", "dv", "deta", "dw0", "ws")), ctypes.c_size_t(nbytes), vp(0))


def test_backward_errors_before_any_hip_call():
    lin = dict(GOOD, h=64, fast_weight=1)
    d = make_desc(**lin)
    assert P.binding.backward_workspace_bytes(d) > P.workspace_bytes(d)
    # the linear entry point: the linear fast weight only; Muon with either I/O type
    muon_fp32 = dict(lin, use_muon=True, io_dtype=1)
    err = ctypes.c_int(0)
    assert P.lib().lact_backward_workspace_bytes(ctypes.byref(make_desc(**muon_fp32)), ctypes.byref(err)) > 0
    assert err.value == 0
    assert _bwd(make_desc(**dict(GOOD)), nbytes=1 << 30) == -4
    # Muon keeps the Newton-Schulz iterates of a chunk: a larger workspace
    assert P.binding.backward_workspace_bytes(make_desc(**dict(lin, use_muon=True))) > P.binding.backward_workspace_bytes(d)
    assert _bwd(make_desc(**dict(lin, d=12, h=12)), nbytes=1 << 30) == -4
    assert _bwd(d, q=0) == -1
    assert _bwd(d, do=0) == -1
    assert _bwd(d, dw0=0) == -1
    assert _bwd(d, deta=0) == -1
    assert _bwd(d, w0=0x5008) == -2
    assert _bwd(d, dwf=0x5008) == -2       # dW_final, when given, is aligned too
    assert _bwd(d, deta=0xA002) == -2
    assert _bwd(d, ws=0) == -3
    assert _bwd(d, nbytes=P.binding.backward_workspace_bytes(d) - 1) == -3
    # no key tokens: k, v, eta and their cotangents may be NULL (reaches the workspace check)
    nk = make_desc(**dict(lin, n_kv=0))
    assert _bwd(nk, k=0, v=0, eta=0, dk=0, dv=0, deta=0, ws=0) == -3
    # the workspace keeps the weights of every chunk boundary: it grows with the chunk count
    more = make_desc(**dict(lin, chunk=128))
    assert P.binding.backward_workspace_bytes(more) > P.binding.backward_workspace_bytes(d)


def _bwd_sw(desc, nbytes=None, **kw):
    a = dict(q=0x1000, k=0x2000, v=0x3000, eta=0x4000, w1=0x5000, w2=0x6000, w3=0x7000, do=0x8000, f1=0, f2=0, f3=0,
             dq=0x9000, dk=0xA000, dv=0xB000, deta=0xC000, d1=0xD000, d2=0xE000, d3=0xF000, ws=0x100000)
    a.update(kw)
    if nbytes is None:
        err = ctypes.c_int(0)
        nbytes = P.lib().lact_backward_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    vp = ctypes.c_void_p
    return P.lib().lact_backward(ctypes.byref(desc), *(vp(a[n]) for n in (
        "q", "k", "v", "eta", "w1", "w2", "w3", "do", "f1", "f2", "f3", "dq", "dk", "dv", "deta", "d1", "d2", "d3",
        "ws")), ctypes.c_size_t(nbytes), vp(0))


def test_swiglu_backward_errors_before_any_hip_call():
    d = make_desc(**GOOD)
    # one workspace query for both fast weights; the SwiGLU backward keeps
    # every chunk's weights and gradient partials, so it grows with the chunk count
    assert P.binding.backward_workspace_bytes(d) > P.workspace_bytes(d)
    assert P.binding.backward_workspace_bytes(make_desc(**dict(GOOD, chunk=128))) > P.binding.backward_workspace_bytes(d)
    # not the linear fast weight; Muon with either I/O type; per-matrix rates accepted
    muon_fp32 = dict(GOOD, use_muon=True, io_dtype=1, d=64, h=64)
    assert _bwd_sw(make_desc(**dict(GOOD, h=64, fast_weight=1)), nbytes=1 << 30) == -4
    assert P.binding.backward_workspace_bytes(make_desc(**dict(GOOD, use_muon=True))) > P.binding.backward_workspace_bytes(d)
    err = ctypes.c_int(0)
    assert P.lib().lact_backward_workspace_bytes(ctypes.byref(make_desc(**muon_fp32)), ctypes.byref(err)) > 0
    assert err.value == 0
    # fp32 operands for the Newton-Schulz reverse: twice the fp16 iterates' bytes
    muon_bf16 = dict(muon_fp32, io_dtype=0)
    assert P.binding.backward_workspace_bytes(make_desc(**muon_fp32)) > P.binding.backward_workspace_bytes(make_desc(**muon_bf16))
    lr3 = make_desc(**dict(GOOD, eta_per_matrix=1))
    assert P.binding.backward_workspace_bytes(lr3) > 0
    assert _bwd_sw(lr3, deta=0) == -1
    assert _bwd_sw(lr3, ws=0) == -3
    assert _bwd_sw(make_desc(**dict(GOOD, d=12)), nbytes=1 << 30) == -4
    assert _bwd_sw(d, q=0) == -1
    assert _bwd_sw(d, do=0) == -1
    assert _bwd_sw(d, w2=0) == -1
    assert _bwd_sw(d, d3=0) == -1
    assert _bwd_sw(d, deta=0) == -1
    assert _bwd_sw(d, w1=0x5008) == -2
    assert _bwd_sw(d, f2=0x5008) == -2     # a final-weight cotangent, when given, is aligned too
    assert _bwd_sw(d, deta=0xC002) == -2
    assert _bwd_sw(d, ws=0) == -3
    assert _bwd_sw(d, ws=0x100010) == -2   # 256-byte workspace alignment
    assert _bwd_sw(d, nbytes=P.binding.backward_workspace_bytes(d) - 1) == -3
    nk = make_desc(**dict(GOOD, n_kv=0))
    assert _bwd_sw(nk, k=0, v=0, eta=0, dk=0, dv=0, deta=0, ws=0) == -3


def _bwd_mom(desc, nbytes=None, **kw):
    names = ("q", "k", "v", "eta", "beta", "w1", "w2", "w3", "m1", "m2", "m3", "do", "f1", "f2", "f3", "g1", "g2",
             "g3", "dq", "dk", "dv", "deta", "dbeta", "d1", "d2", "d3", "e1", "e2", "e3", "ws")
    a = {n: 0x1000 * (i + 1) for i, n in enumerate(names)}
    for n in ("f1", "f2", "f3", "g1", "g2", "g3"):
        a[n] = 0
    a["ws"] = 0x100000
    a.update(kw)
    if nbytes is None:
        err = ctypes.c_int(0)
        nbytes = P.lib().lact_backward_momentum_workspace_bytes(ctypes.byref(desc), ctypes.byref(err))
    vp = ctypes.c_void_p
    return P.lib().lact_backward_momentum(ctypes.byref(desc), *(vp(a[n]) for n in names), ctypes.c_size_t(nbytes),
                                          vp(0))


@pytest.mark.parametrize("fw", [0, 1])
def test_momentum_backward_errors_before_any_hip_call(fw):
    base = dict(GOOD, h=64, fast_weight=1) if fw else dict(GOOD)
    d = make_desc(**base)
    nb = P.binding.backward_momentum_workspace_bytes(d)
    # the plain backward's workspace plus every chunk's state
    assert nb > P.binding.backward_workspace_bytes(d)
    assert P.binding.backward_momentum_workspace_bytes(make_desc(**dict(base, chunk=128))) > nb
    muon_fp32 = dict(base, use_muon=True, io_dtype=1, d=64, h=64)
    err = ctypes.c_int(0)
    assert P.lib().lact_backward_momentum_workspace_bytes(ctypes.byref(make_desc(**muon_fp32)), ctypes.byref(err)) > 0
    assert err.value == 0
    assert _bwd_mom(make_desc(**muon_fp32), ws=0) == -3
    assert _bwd_mom(d, m1=0) == -1
    assert _bwd_mom(d, e1=0) == -1
    assert _bwd_mom(d, beta=0) == -1
    assert _bwd_mom(d, dbeta=0) == -1
    assert _bwd_mom(d, m1=0x9008) == -2
    assert _bwd_mom(d, g1=0x9008) == -2    # a final-state cotangent, when given, is aligned too
    assert _bwd_mom(d, dbeta=0x17002) == -2
    assert _bwd_mom(d, ws=0) == -3
    assert _bwd_mom(d, nbytes=nb - 1) == -3
    if fw == 0:
        assert _bwd_mom(d, m3=0) == -1
        assert _bwd_mom(d, e2=0) == -1
    else:   # the linear fast weight ignores the second and third matrices
        assert _bwd_mom(d, m2=0, m3=0, e2=0, e3=0, w2=0, w3=0, d2=0, d3=0, ws=0) == -3
    # no key tokens: beta and dbeta may be NULL as well
    nk = make_desc(**dict(base, n_kv=0))
    assert _bwd_mom(nk, k=0, v=0, eta=0, beta=0, dk=0, dv=0, deta=0, dbeta=0, ws=0) == -3


def _bwd_sched(desc, segs, nbytes=None, mom=False, **kw):
    names = ("q", "k", "v", "eta", "beta", "w1", "w2", "w3", "m1", "m2", "m3", "do", "f1", "f2", "f3", "g1", "g2",
             "g3", "dq", "dk", "dv", "deta", "dbeta", "d1", "d2", "d3", "e1", "e2", "e3", "ws")
    a = {n: 0x1000 * (i + 1) for i, n in enumerate(names)}
    for n in ("f1", "f2", "f3", "g1", "g2", "g3"):
        a[n] = 0
    if not mom:
        for n in ("beta", "m1", "m2", "m3", "dbeta", "e1", "e2", "e3"):
            a[n] = 0
    a["ws"] = 0x100000
    a.update(kw)
    arr = (P.binding.LactSegment * max(len(segs), 1))()
    for i, (m, b, e) in enumerate(segs):
        arr[i] = P.binding.LactSegment(m, 0, b, e)
    if nbytes is None:
        err = ctypes.c_int(0)
        nbytes = P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(desc), arr, len(segs), int(mom),
                                                                ctypes.byref(err))
    vp = ctypes.c_void_p
    return P.lib().lact_backward_schedule(ctypes.byref(desc), arr, len(segs), *(vp(a[n]) for n in names),
                                          ctypes.c_size_t(nbytes), vp(0))


def test_schedule_backward_errors_before_any_hip_call():
    d = make_desc(**dict(GOOD, n_kv=1000, n_q=1100, chunk=256))
    segs = [(3, 0, 256), (1, 256, 512), (2, 512, 700), (0, 700, 956), (3, 956, 1100)]
    err = ctypes.c_int(0)
    arr = (P.binding.LactSegment * len(segs))(*(P.binding.LactSegment(m, 0, b, e) for m, b, e in segs))
    nb = P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(d), arr, len(segs), 0, ctypes.byref(err))
    assert err.value == 0 and nb > 0
    # three updates: less than the uniform schedule's four chunks; momentum adds the state's trajectory
    assert nb < P.binding.backward_workspace_bytes(d)
    nbm = P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(d), arr, len(segs), 1, ctypes.byref(err))
    assert nbm > nb
    assert _bwd_sched(d, segs, ws=0) == -3
    assert _bwd_sched(d, segs, nbytes=nb - 1) == -3
    assert _bwd_sched(d, segs, mom=True, ws=0) == -3
    assert _bwd_sched(d, segs, mom=True, dbeta=0) == -1
    assert _bwd_sched(d, segs, mom=True, m2=0) == -1
    assert _bwd_sched(d, segs, dq=0) == -1
    assert _bwd_sched(d, [(2, 0, 300)]) == -1          # an update longer than the chunk
    assert _bwd_sched(d, [(4, 0, 10)]) == -1           # an unknown mode
    assert _bwd_sched(d, [(3, 0, 1200)]) == -1         # an apply past n_q
    # overlapping applies, or overlapping updates: not differentiated
    assert _bwd_sched(d, [(3, 0, 100), (3, 50, 150)]) == -4
    assert _bwd_sched(d, [(2, 0, 100), (2, 50, 150)]) == -4
    # the linear fast weight: a workspace of its own size, the same checks
    dl = make_desc(**dict(GOOD, h=64, fast_weight=1))
    nl = P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(dl), arr, len(segs), 0, ctypes.byref(err))
    assert err.value == 0 and nl > 0
    nlm = P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(dl), arr, len(segs), 1, ctypes.byref(err))
    assert err.value == 0 and nlm > nl
    assert _bwd_sched(dl, segs, nbytes=nl - 1) == -3
    assert _bwd_sched(dl, segs, mom=True, nbytes=nlm - 1) == -3
    assert _bwd_sched(dl, segs, mom=True, dbeta=0) == -1
    assert _bwd_sched(dl, segs, mom=True, e1=0) == -1    # the state's cotangent
    assert _bwd_sched(dl, segs, dk=0) == -1
    assert _bwd_sched(dl, [(2, 0, 100), (2, 50, 150)]) == -4
    assert _bwd_sched(dl, [(2, 0, 300)]) == -1
    assert P.lib().lact_backward_schedule_workspace_bytes(ctypes.byref(dl), arr, -1, 0, ctypes.byref(err)) == 0
    assert err.value == -1
    # an empty schedule reaches the workspace check
    assert _bwd_sched(d, [], ws=0) == -3


def test_prologue_and_norm_backward_errors_before_any_hip_call():
    L = P.lib()
    vp = ctypes.c_void_p
    d = make_desc(**dict(GOOD, n_kv=100, n_q=120))
    a = dict(qkv=0x1000, lr=0x2000, br=0, dq=0x3000, dk=0x4000, dv=0x5000, de=0x6000, db=0, dqkv=0x7000,
             dlr=0x8000, dbr=0)

    def pro(**kw):
        x = dict(a)
        x.update(kw)
        return L.lact_prologue_backward(ctypes.byref(d), vp(x["qkv"]), vp(x["lr"]), ctypes.c_float(-1.0),
                                        *(vp(x[n]) for n in ("br", "dq", "dk", "dv", "de", "db", "dqkv", "dlr", "dbr")),
                                        vp(0))
    assert pro(dq=0) == -1
    assert pro(dlr=0) == -1
    assert pro(de=0) == -1
    assert pro(br=0x9000) == -1                 # beta_raw without dbeta_raw
    assert pro(br=0x9000, dbr=0xA000) == -1     # ... and without dbeta
    assert pro(dqkv=0x7008) == -2
    assert pro(dlr=0x8002) == -2
    assert L.lact_prologue_backward(ctypes.byref(d), vp(0x1000), vp(0x2000), ctypes.c_float(float("inf")),
                                    *(vp(a[n]) for n in ("br", "dq", "dk", "dv", "de", "db", "dqkv", "dlr", "dbr")),
                                    vp(0)) == -1

    def rms(w=0x1000, dw=0x2000, ws=0x10000, nbytes=None, eps=1e-6, **kw):
        x = dict(o=0x3000, dy=0x4000, do=0x5000)
        x.update(kw)
        if nbytes is None:
            err = ctypes.c_int(0)
            nbytes = L.lact_rmsnorm_out_backward_workspace_bytes(ctypes.byref(d), int(dw != 0), ctypes.byref(err))
        return L.lact_rmsnorm_out_backward(ctypes.byref(d), vp(x["o"]), vp(w), ctypes.c_float(eps), vp(x["dy"]),
                                           vp(x["do"]), vp(dw), vp(ws), ctypes.c_size_t(nbytes), vp(0))
    err = ctypes.c_int(0)
    assert L.lact_rmsnorm_out_backward_workspace_bytes(ctypes.byref(d), 0, ctypes.byref(err)) == 0 and err.value == 0
    assert L.lact_rmsnorm_out_backward_workspace_bytes(ctypes.byref(d), 1, ctypes.byref(err)) > 0
    assert rms(w=0) == -1                       # dweight needs the weight
    assert rms(do=0) == -1
    assert rms(eps=-1.0) == -1
    assert rms(ws=0) == -3
    assert rms(nbytes=1) == -3
    assert rms(do=0x5008) == -2
    assert rms(ws=0x10010) == -2
