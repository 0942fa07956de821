"""The C ABI on the host: the library loads, exports every function the
header declares, and rejects bad arguments before touching the GPU.  No call
here reaches a kernel launch (every call fails validation or only sizes the
workspace), so these run without a GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pdn.h")

pdn = pytest.importorskip("paper_2604_21100_amd",
                          reason="libpdn.so not built")

A = 1 << 20   # fake, 256-byte aligned addresses; never dereferenced


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pdn_\w+)\s*\(", text)))


def test_header_symbols_exported():
    names = header_functions()
    assert set(names) == set(pdn.EXPORTED)
    lib = ctypes.CDLL(pdn.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    hdr = open(os.path.join(ROOT, "include", "pdn.h")).read()
    ver = int(re.search(r"#define PDN_ABI_VERSION (\d+)", hdr).group(1))
    assert pdn.pdn_abi_version() == ver == pdn.ABI_VERSION


def test_status_strings():
    for st in range(11):
        assert pdn.pdn_status_string(st)
    assert pdn.pdn_status_string(0) == "ok"


def _prob(**kw):
    base = dict(B=2, T=130, H=3, dk=128, dv=64, io="bf16", gate="scalar",
                precond="squash")
    base.update(kw)
    return pdn.make_problem(**base)


def _inputs(**kw):
    names = [f[0] for f in pdn.Inputs._fields_]
    vals = dict(q=A * 1, k=A * 2, v=A * 3, beta=A * 4, g=A * 5, beta_p=A * 6,
                g_p=A * 7, log_a_scale=A * 8, A0=None, S0=None, ktilde=None)
    vals.update(kw)
    return pdn.Inputs(*[vals[n] for n in names])


def _fwd(prob, inp=None, out=None, ws=A * 64, ws_bytes=None):
    if inp is None:
        inp = _inputs()
    if out is None:
        out = pdn.FwdOut(A * 20, A * 21, A * 22)
    if ws_bytes is None:
        try:
            ws_bytes = pdn.pdn_workspace_size(prob) - 1   # always too small
        except pdn.PdnError:
            ws_bytes = 0
    return pdn.pdn_chunk_fwd_raw(prob, inp, out, ws, ws_bytes, 0)


def test_forward_only_modes_validated():
    """DIAG_SM and ATQ need a positive finite ridge; their backward is not
    built (PDN_ERR_UNSUPPORTED, before any HIP call)."""
    for pc in ("diag_sm", "atq"):
        assert pdn.pdn_workspace_size(_prob(precond=pc, ridge=0.5)) > 0
        for bad in (0.0, -1.0, float("nan"), float("inf")):
            with pytest.raises(pdn.PdnError) as e:
                pdn.pdn_workspace_size(_prob(precond=pc, ridge=bad))
            assert e.value.status == pdn.PDN_ERR_VALUE
        with pytest.raises(pdn.PdnError) as e:
            pdn.pdn_workspace_size(_prob(precond=pc, ridge=0.5), True)
        assert e.value.status == pdn.PDN_ERR_UNSUPPORTED
    # the ridge is ignored by the other modes
    assert pdn.pdn_workspace_size(_prob(ridge=0.0)) > 0
    # write-key normalisation: squash only, forward only, and the beta
    # factor needs a scalar (or no) decay
    for kn in ("m", "1pm", "beta"):
        assert pdn.pdn_workspace_size(_prob(knorm=kn)) > 0
        with pytest.raises(pdn.PdnError) as e:
            pdn.pdn_workspace_size(_prob(knorm=kn), True)
        assert e.value.status == pdn.PDN_ERR_UNSUPPORTED
        with pytest.raises(pdn.PdnError) as e:
            pdn.pdn_workspace_size(_prob(knorm=kn, precond="identity"))
        assert e.value.status == pdn.PDN_ERR_VALUE
    with pytest.raises(pdn.PdnError) as e:
        pdn.pdn_workspace_size(_prob(knorm="beta", gate="channel"))
    assert e.value.status == pdn.PDN_ERR_UNSUPPORTED
    with pytest.raises(pdn.PdnError) as e:
        pdn.pdn_workspace_size(_prob(knorm=7))
    assert e.value.status == pdn.PDN_ERR_VALUE
    # ATQ keeps the preconditioned query rows in the workspace
    assert (pdn.pdn_workspace_size(_prob(precond="atq", ridge=1.0))
            > pdn.pdn_workspace_size(_prob(precond="diag_sm", ridge=1.0)))


def test_workspace_size_monotone_and_validated():
    a = pdn.pdn_workspace_size(_prob(T=64))
    b = pdn.pdn_workspace_size(_prob(T=65))
    c = pdn.pdn_workspace_size(_prob(T=130, gate="channel"))
    assert 0 < a < b < c
    assert pdn.pdn_workspace_size(_prob(B=0)) == 0
    with pytest.raises(pdn.PdnError) as e:
        pdn.pdn_workspace_size(_prob(dk=96))
    assert e.value.status == pdn.PDN_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw,code", [
    (dict(dk=96), pdn.PDN_ERR_UNSUPPORTED),
    (dict(dv=256), pdn.PDN_ERR_UNSUPPORTED),
    (dict(chunk=16), pdn.PDN_ERR_UNSUPPORTED),
    (dict(chunk=48), pdn.PDN_ERR_UNSUPPORTED),
    (dict(chunk=128), pdn.PDN_ERR_UNSUPPORTED),
    (dict(B=-1), pdn.PDN_ERR_SHAPE),
    (dict(T=-5), pdn.PDN_ERR_SHAPE),
    (dict(B=1 << 40, T=1 << 30), pdn.PDN_ERR_SHAPE),
    (dict(x=0.9), pdn.PDN_ERR_VALUE),
    (dict(x=float("nan")), pdn.PDN_ERR_VALUE),
    (dict(scale=float("inf")), pdn.PDN_ERR_VALUE),
    (dict(gate=7), pdn.PDN_ERR_VALUE),
    (dict(precond=5), pdn.PDN_ERR_VALUE),
])
def test_problem_validation(kw, code):
    assert _fwd(_prob(**kw)) == code


def test_bad_dtype():
    p = _prob()
    p.io = 9
    assert _fwd(p) == pdn.PDN_ERR_DTYPE


@pytest.mark.parametrize("field", ["q", "k", "v", "beta", "g", "beta_p",
                                   "log_a_scale"])
def test_null_required_pointer(field):
    assert _fwd(_prob(), _inputs(**{field: None})) == pdn.PDN_ERR_NULL


def test_null_pointer_cases():
    assert pdn.pdn_chunk_fwd_raw(_prob(), _inputs(), pdn.FwdOut(None, None, None),
                                 A * 64, 16, 0) == pdn.PDN_ERR_NULL
    assert _fwd(_prob(precond="external")) == pdn.PDN_ERR_NULL   # no ktilde
    # g_p may be NULL (alpha^P = 1): the failure is then the workspace size
    assert _fwd(_prob(), _inputs(g_p=None)) == pdn.PDN_ERR_WORKSPACE


def test_gate_pointer_must_match_kind():
    assert _fwd(_prob(gate="none")) == pdn.PDN_ERR_VALUE   # g given


def test_misaligned():
    assert _fwd(_prob(), _inputs(q=A + 2)) == pdn.PDN_ERR_ALIGN
    assert _fwd(_prob(), out=pdn.FwdOut(A * 20 + 8, None, None)) == pdn.PDN_ERR_ALIGN


def test_workspace_checks():
    p = _prob()
    n = pdn.pdn_workspace_size(p)
    assert _fwd(p, ws=None, ws_bytes=n - 1) == pdn.PDN_ERR_WORKSPACE
    assert _fwd(p, ws_bytes=n - 1) == pdn.PDN_ERR_WORKSPACE
    # a misaligned workspace of sufficient size is only checked on hosts
    # where a launch cannot happen
    if not os.path.exists("/dev/kfd"):
        assert _fwd(p, ws=A * 64 + 16, ws_bytes=n) == pdn.PDN_ERR_WORKSPACE


def test_aliasing():
    # the workspace is one byte short in every call, so even a missed alias
    # could not reach a launch
    p = _prob()
    # o overlaps v
    assert _fwd(p, out=pdn.FwdOut(A * 3 + 256, None, None)) == pdn.PDN_ERR_ALIAS
    # S_T overlaps o
    assert _fwd(p, out=pdn.FwdOut(A * 20, A * 20 + 512, None)) == pdn.PDN_ERR_ALIAS
    # workspace overlaps q
    assert _fwd(p, ws=A * 1 - 256) == pdn.PDN_ERR_ALIAS
    # A_T only exists for the squash preconditioner
    assert _fwd(_prob(precond="identity"), _inputs(beta_p=None)) == pdn.PDN_ERR_VALUE


def test_backward_validates_first():
    p = _prob(dk=96)
    st = pdn.pdn_chunk_bwd_raw(p, _inputs(), A * 30, None,
                               pdn.BwdOut(*([None] * 11)), A * 64, 0, 0)
    assert st == pdn.PDN_ERR_UNSUPPORTED


def test_stage_event_arguments_validated():
    """The event variants reject a missing or wrong-length event array
    before anything else (no HIP call is reached)."""
    vp = ctypes.c_void_p
    p = _prob()
    lib = pdn._lib
    out = pdn.FwdOut(A * 20, A * 21, A * 22)
    ev_f = (vp * pdn.FWD_STAGE_EVENTS)(*([A * 40] * pdn.FWD_STAGE_EVENTS))
    assert lib.pdn_chunk_fwd_events(
        ctypes.byref(p), ctypes.byref(_inputs()), ctypes.byref(out), A * 64, 0,
        None, None, pdn.FWD_STAGE_EVENTS) == pdn.PDN_ERR_NULL
    assert lib.pdn_chunk_fwd_events(
        ctypes.byref(p), ctypes.byref(_inputs()), ctypes.byref(out), A * 64, 0,
        None, ev_f, pdn.FWD_STAGE_EVENTS - 1) == pdn.PDN_ERR_VALUE
    bo = pdn.BwdOut(*([None] * 11))
    ev_b = (vp * pdn.BWD_STAGE_EVENTS)(*([A * 40] * pdn.BWD_STAGE_EVENTS))
    assert lib.pdn_chunk_bwd_events(
        ctypes.byref(p), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, None,
        pdn.BWD_STAGE_EVENTS) == pdn.PDN_ERR_NULL
    assert lib.pdn_chunk_bwd_events(
        ctypes.byref(p), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, ev_b, 6) == pdn.PDN_ERR_VALUE
    # NULL entries are allowed (not recorded): validation then goes on to the
    # problem and reaches the missing workspace
    ev_b[3] = None
    plain = lib.pdn_chunk_bwd(
        ctypes.byref(p), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None)
    assert plain == pdn.PDN_ERR_NULL      # the outputs are missing
    assert lib.pdn_chunk_bwd_events(
        ctypes.byref(p), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, ev_b,
        pdn.BWD_STAGE_EVENTS) == plain
    # with valid event pointers, problem validation still comes first
    ev_b[3] = A * 40
    assert lib.pdn_chunk_bwd_events(
        ctypes.byref(_prob(dk=96)), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, ev_b,
        pdn.BWD_STAGE_EVENTS) == pdn.PDN_ERR_UNSUPPORTED
    assert len(pdn.BWD_STAGES) == pdn.BWD_STAGE_EVENTS - 1
    assert len(pdn.FWD_STAGES) == pdn.FWD_STAGE_EVENTS - 1


def test_one_hip_runtime_in_process():
    """Importing the package first must not map a second HIP runtime when
    torch is imported afterwards (two HSA runtimes in one process break
    every GPU call)."""
    import subprocess
    import sys
    code = ("import paper_2604_21100_amd as p, torch; "
            "print(len(p.loaded_hip_runtimes()))")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "1", r.stdout


def test_training_pair_validation():
    """The training forward needs the backward's workspace and support; no
    call reaches a launch (the workspace is always short)."""
    vp = ctypes.c_void_p
    lib = pdn._lib
    out = pdn.FwdOut(A * 20, A * 21, A * 22)
    p = _prob()
    need_f = pdn.pdn_workspace_size(p, False)
    need_b = pdn.pdn_workspace_size(p, True)
    assert need_b > need_f
    # enough for the plain forward, one byte short for the training forward
    assert lib.pdn_chunk_fwd_train(
        ctypes.byref(p), ctypes.byref(_inputs()), ctypes.byref(out), A * 64,
        need_b - 1, None, None, 0) == pdn.PDN_ERR_WORKSPACE
    # the backward's restriction applies (fp32 io: d = 64 only); a
    # per-channel gate is accepted and then wants the backward's workspace
    pc = _prob(gate="channel")
    assert lib.pdn_chunk_fwd_train(
        ctypes.byref(pc), ctypes.byref(_inputs()), ctypes.byref(out), A * 64,
        pdn.pdn_workspace_size(pc, True) - 1, None, None, 0) == pdn.PDN_ERR_WORKSPACE
    pf = _prob(io="f32", dk=128, dv=64)
    assert lib.pdn_chunk_fwd_train(
        ctypes.byref(pf), ctypes.byref(_inputs()), ctypes.byref(out), A * 64,
        0, None, None, 0) == pdn.PDN_ERR_UNSUPPORTED
    # event arrays: NULL needs n_events 0; a wrong count is rejected
    ev = (vp * 4)(*([A * 40] * 4))
    assert lib.pdn_chunk_fwd_train(
        ctypes.byref(p), ctypes.byref(_inputs()), ctypes.byref(out), A * 64,
        0, None, None, 4) == pdn.PDN_ERR_NULL
    assert lib.pdn_chunk_fwd_train(
        ctypes.byref(p), ctypes.byref(_inputs()), ctypes.byref(out), A * 64,
        0, None, ev, 3) == pdn.PDN_ERR_VALUE
    bo = pdn.BwdOut(*([None] * 11))
    assert lib.pdn_chunk_bwd_train(
        ctypes.byref(p), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, ev, 4) == pdn.PDN_ERR_VALUE
    assert lib.pdn_chunk_bwd_train(
        ctypes.byref(pf), ctypes.byref(_inputs()), A * 30, None,
        ctypes.byref(bo), A * 64, 0, None, None, 0) == pdn.PDN_ERR_UNSUPPORTED


def _fwd_noalloc(prob, inp=None, out=None):
    if inp is None:
        inp = _inputs()
    if out is None:
        out = pdn.FwdOut(A * 20, A * 21, A * 22)
    return pdn.pdn_chunk_fwd_noalloc_raw(prob, inp, out, 0)


def test_noalloc_rejects_problems_beyond_its_scratch():
    """The no-allocation forward holds a fixed 64 MiB scratch per device: a
    problem whose forward workspace is larger is refused with
    PDN_ERR_SCRATCH before any HIP call (the 1B layer, B=4 T=4096 H=16,
    needs about 136 MB)."""
    assert pdn.pdn_noalloc_scratch_bytes() == 64 << 20
    big = pdn.make_problem(4, 4096, 16, 128, 128, gate="scalar")
    assert pdn.pdn_workspace_size(big) > pdn.pdn_noalloc_scratch_bytes()
    assert _fwd_noalloc(big) == pdn.PDN_ERR_SCRATCH
    assert "scratch" in pdn.pdn_status_string(pdn.PDN_ERR_SCRATCH)
    # the largest T that fits, and one chunk more, at B=1 H=14 d=128
    fits = [T for T in range(64, 20000, 64)
            if pdn.pdn_workspace_size(pdn.make_problem(1, T, 14, 128, 128,
                                                       gate="scalar"))
            <= pdn.pdn_noalloc_scratch_bytes()]
    tmax = max(fits)
    assert tmax >= 7680   # (the sequence split's segment states included)
    over = pdn.make_problem(1, tmax + 64, 14, 128, 128, gate="scalar")
    assert _fwd_noalloc(over) == pdn.PDN_ERR_SCRATCH


def test_noalloc_validates_like_the_forward():
    """Every argument check of pdn_chunk_fwd runs first, with its codes."""
    p = _prob()
    assert _fwd_noalloc(pdn.make_problem(2, 130, 3, 96, 64)) == \
        pdn.PDN_ERR_UNSUPPORTED
    assert _fwd_noalloc(p, _inputs(q=None)) == pdn.PDN_ERR_NULL
    assert _fwd_noalloc(p, _inputs(q=A + 2)) == pdn.PDN_ERR_ALIGN
    assert _fwd_noalloc(p, out=pdn.FwdOut(None, None, None)) == pdn.PDN_ERR_NULL
    assert _fwd_noalloc(p, out=pdn.FwdOut(A * 3 + 256, None, None)) == \
        pdn.PDN_ERR_ALIAS
    assert _fwd_noalloc(_prob(precond="identity"), _inputs(beta_p=None)) == \
        pdn.PDN_ERR_VALUE


def test_chunk_sizes():
    """Chunks of 32 and 64 tokens: forward, backward and training-pair
    workspaces size, and argument checks run for both (a one-byte-short
    workspace fails before any HIP call)."""
    p32, p64 = _prob(chunk=32), _prob(chunk=64)
    for with_bwd in (False, True):
        n32 = pdn.pdn_workspace_size(p32, with_bwd)
        n64 = pdn.pdn_workspace_size(p64, with_bwd)
        assert n32 > 0 and n64 > 0
    assert _fwd(p32) == pdn.PDN_ERR_WORKSPACE
    st = pdn.pdn_chunk_bwd_raw(p32, _inputs(), A * 30, None,
                               pdn.BwdOut(A * 40, A * 41, A * 42, A * 43, A * 44,
                                          None, None, None, None, None, None),
                               A * 64, 1, 0)
    assert st == pdn.PDN_ERR_WORKSPACE


def test_scan_segments():
    """The forward scan splits the sequence only when the heads' slabs leave
    most of the 256 compute units idle and segments of ceil(NT / S) >= 4
    chunks remain: the 32K-token 16-head layer runs in 3 segments, the 1B layer
    (64 heads of B x H) in one pass; a single head over 33 chunks takes 9
    segments of 4 (plus one chunk)."""
    mp = pdn.make_problem
    assert pdn.pdn_scan_segments(mp(1, 32768, 16, 128, 128)) == 3
    assert pdn.pdn_scan_segments(mp(4, 4096, 16, 128, 128)) == 1
    assert pdn.pdn_scan_segments(mp(2, 8192, 16, 128, 128)) == 1
    assert pdn.pdn_scan_segments(mp(1, 2112, 1, 128, 128)) == 9
    assert pdn.pdn_scan_segments(mp(1, 700, 2, 64, 64)) == 3
    assert pdn.pdn_scan_segments(mp(1, 704, 2, 64, 64)) == 3
    assert pdn.pdn_scan_segments(mp(1, 640, 2, 64, 64)) == 3   # 10 chunks: 4 + 4 + 2
    assert pdn.pdn_scan_segments(mp(1, 512, 2, 64, 64)) == 1   # 8 chunks: 3 per segment
    assert pdn.pdn_scan_segments(mp(0, 640, 2, 64, 64)) == 1
    # more segments never cost more workspace than their states
    a = pdn.pdn_workspace_size(mp(1, 32768, 16, 128, 128))
    b = pdn.pdn_workspace_size(mp(1, 32768, 16, 128, 128, chunk=32))
    assert a > 0 and b > 0
    with pytest.raises(pdn.PdnError) as e:
        pdn.pdn_scan_segments(mp(1, 64, 2, 96, 64))
    assert e.value.status == pdn.PDN_ERR_UNSUPPORTED
