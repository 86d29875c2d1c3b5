"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before any HIP call (no GPU needed)."""

import ctypes
import os
import re

import pytest

from paper_2608_13578_amd import bcmt as abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bcmt.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(abi.LIB_PATH):
        from paper_2608_13578_amd.build import build
        build()
    return abi.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bcmt_[a-z_]+)\s*\(", text)))


def test_header_declares_the_abi():
    names = declared_functions()
    assert set(names) == set(abi.EXPORTED), names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = os.popen(f"nm -D --defined-only {abi.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}$", out, flags=re.M), name


def test_version_and_strerror(lib):
    assert abi.bcmt_version() >= 100
    for code in (0, -1, -2, -3, -4):
        assert isinstance(abi.bcmt_strerror(code), str) and abi.bcmt_strerror(code)
    assert abi.bcmt_strerror(-99) == "unknown status"


def good(**kw):
    base = dict(B=2, T=256, D=128, H=2, L=64, gamma=0.8, dtype="bf16")
    base.update(kw)
    return abi.make_config(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(), abi.BCMT_OK),
    (dict(dtype="f32"), abi.BCMT_OK),
    (dict(L=10000), abi.BCMT_OK),           # one block
    (dict(T=1000, L=128), abi.BCMT_OK),     # ragged last block
    (dict(gamma=0.0), abi.BCMT_OK),
    (dict(B=0), abi.BCMT_ERR_INVALID),
    (dict(T=0), abi.BCMT_ERR_INVALID),
    (dict(L=0), abi.BCMT_ERR_INVALID),
    (dict(H=3), abi.BCMT_ERR_INVALID),      # D % H != 0
    (dict(gamma=1.0), abi.BCMT_ERR_INVALID),
    (dict(gamma=-0.1), abi.BCMT_ERR_INVALID),
    (dict(gamma=float("nan")), abi.BCMT_ERR_INVALID),
    (dict(D=128, H=8), abi.BCMT_OK),               # head width 16 (the paper's model)
    (dict(D=128, H=4), abi.BCMT_OK),               # head width 32
    (dict(D=96, H=3), abi.BCMT_ERR_UNSUPPORTED),   # D not a multiple of 64
    (dict(D=64, H=8), abi.BCMT_ERR_UNSUPPORTED),   # head width 8
    (dict(D=256, H=2), abi.BCMT_ERR_UNSUPPORTED),  # head width 128
    (dict(D=4096, H=64), abi.BCMT_ERR_UNSUPPORTED),
])
def test_validate(lib, kw, code):
    assert abi.bcmt_validate(good(**kw)) == code


def test_validate_rejects_bad_dtype_and_flags(lib):
    c = good()
    c.dtype = 7
    assert abi.bcmt_validate(c) == abi.BCMT_ERR_INVALID
    c = good()
    c.flags = 8
    assert abi.bcmt_validate(c) == abi.BCMT_ERR_INVALID
    assert lib.bcmt_validate(None) == abi.BCMT_ERR_INVALID


def test_sizes(lib):
    c = good()
    saved = abi.bcmt_saved_bytes(c)
    B, T, D = 2, 256, 128
    assert saved >= (3 + 3) * B * T * D * 2          # qkv, o, h, g in bf16
    assert abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_INFERENCE) == \
        abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_FORWARD) + saved
    assert abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_BACKWARD) > 0
    assert abi.bcmt_workspace_bytes(c, 9) == 0
    f32 = good(dtype="f32")
    assert abi.bcmt_saved_bytes(f32) > saved
    bad = good(B=0)
    assert abi.bcmt_saved_bytes(bad) == 0 and abi.bcmt_workspace_bytes(bad, 0) == 0


# Fake, aligned device addresses: every call below must fail its argument
# checks before touching them.
A = 1 << 40


def _params(**override):
    p = {n: A + 0x100000 * (i + 1) for i, n in enumerate(abi.PARAM_NAMES)}
    p.update(override)
    return abi.bcmt_params(*[p[n] for n in abi.PARAM_NAMES])


def _fwd(cfg, X=A, params=None, Y=A + 0x10000000, saved=A + 0x20000000, ws=A + 0x40000000,
         ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = abi.bcmt_workspace_bytes(cfg, abi.BCMT_PASS_FORWARD)
    return abi.lib().bcmt_layer_forward(ctypes.byref(cfg), X, ctypes.byref(params or _params()),
                                        Y, saved, ws, ws_bytes, None)


def test_forward_argument_errors(lib):
    c = good()
    assert _fwd(good(B=0)) == abi.BCMT_ERR_INVALID
    assert _fwd(good(D=256, H=2)) == abi.BCMT_ERR_UNSUPPORTED
    assert _fwd(c, X=None) == abi.BCMT_ERR_INVALID
    assert _fwd(c, Y=None) == abi.BCMT_ERR_INVALID
    assert _fwd(c, params=_params(Wm=None)) == abi.BCMT_ERR_INVALID
    assert _fwd(c, params=_params(wp=A + 8)) == abi.BCMT_ERR_INVALID      # misaligned
    assert _fwd(c, X=A + 4) == abi.BCMT_ERR_INVALID
    assert _fwd(c, Y=A) == abi.BCMT_ERR_INVALID                            # Y aliases X
    assert _fwd(c, Y=A + 1024) == abi.BCMT_ERR_INVALID                     # Y overlaps X
    assert _fwd(c, ws=None) == abi.BCMT_ERR_INVALID
    need = abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_FORWARD)
    assert _fwd(c, ws_bytes=need - 1) == abi.BCMT_ERR_WORKSPACE
    # inference (no saved) needs the larger workspace
    assert _fwd(c, saved=None, ws_bytes=need) == abi.BCMT_ERR_WORKSPACE
    assert lib.bcmt_layer_forward(None, A, ctypes.byref(_params()), A + 0x10000000, None,
                                  A + 0x40000000, 1 << 30, None) == abi.BCMT_ERR_INVALID


def test_noalloc_forward_argument_errors(lib):
    """The allocation-free forward rejects a pass whose workspace exceeds its
    scratch array, and a missing `saved`, before any HIP call."""
    small = good()
    assert abi.bcmt_workspace_bytes(small, abi.BCMT_PASS_FORWARD) <= abi.BCMT_NOALLOC_SCRATCH_BYTES
    big = good(B=16, T=65536, D=1024, H=16, L=32)
    assert abi.bcmt_workspace_bytes(big, abi.BCMT_PASS_FORWARD) > abi.BCMT_NOALLOC_SCRATCH_BYTES
    p = ctypes.byref(_params())
    f = lib.bcmt_layer_forward_noalloc
    assert f(ctypes.byref(big), A, p, A + 0x10000000, A + 0x20000000, None) == \
        abi.BCMT_ERR_WORKSPACE
    assert f(ctypes.byref(small), A, p, A + 0x10000000, None, None) == abi.BCMT_ERR_INVALID
    assert f(ctypes.byref(good(T=0)), A, p, A + 0x10000000, A + 0x20000000, None) == \
        abi.BCMT_ERR_INVALID
    assert f(None, A, p, A + 0x10000000, A + 0x20000000, None) == abi.BCMT_ERR_INVALID


def _bwd(cfg, X=A, saved=A + 0x20000000, dY=A + 0x30000000, dX=A + 0x38000000, grads=None,
         ws=A + 0x40000000, ws_bytes=None, params=None, side=None):
    if ws_bytes is None:
        ws_bytes = abi.bcmt_workspace_bytes(cfg, abi.BCMT_PASS_BACKWARD)
    g = grads
    return abi.lib().bcmt_layer_backward(ctypes.byref(cfg), X, ctypes.byref(params or _params()),
                                         saved, dY, dX, ctypes.byref(g) if g else None, ws,
                                         ws_bytes, None, ctypes.byref(side) if side else None)


def test_backward_argument_errors(lib):
    c = good()
    assert _bwd(good(T=0)) == abi.BCMT_ERR_INVALID
    assert _bwd(c, saved=None) == abi.BCMT_ERR_INVALID
    assert _bwd(c, dY=None) == abi.BCMT_ERR_INVALID
    assert _bwd(c, X=None) == abi.BCMT_ERR_INVALID
    assert _bwd(c, dX=A + 0x30000000) == abi.BCMT_ERR_INVALID             # dX aliases dY
    assert _bwd(c, dX=A + 2) == abi.BCMT_ERR_INVALID
    assert _bwd(c, ws=None) == abi.BCMT_ERR_INVALID
    need = abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_BACKWARD)
    assert _bwd(c, ws_bytes=need - 256) == abi.BCMT_ERR_WORKSPACE
    g = abi.bcmt_grads(*([A + 0x50000000 + 0x1000000 * i for i in range(7)] + [A + 0x60000002]))
    assert _bwd(c, grads=g) == abi.BCMT_ERR_INVALID                        # dgamma misaligned
    g = abi.bcmt_grads(*([A + 0x50000008] + [None] * 7))
    assert _bwd(c, grads=g) == abi.BCMT_ERR_INVALID                        # dWq misaligned


def test_backward_second_stream_arguments(lib):
    """Without a second stream (NULL) the backward's argument checks are those
    of the one-stream pass; a second stream needs both of its events."""
    c = good()
    need = abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_BACKWARD)
    for side in (None, abi.bcmt_side(0x1000, 0x2000, 0x3000)):
        assert _bwd(c, saved=None, side=side) == abi.BCMT_ERR_INVALID
        assert _bwd(c, ws=None, side=side) == abi.BCMT_ERR_INVALID
        assert _bwd(c, ws_bytes=need - 256, side=side) == abi.BCMT_ERR_WORKSPACE
        assert _bwd(good(D=96, H=1), side=side) == abi.BCMT_ERR_UNSUPPORTED
    for side in (abi.bcmt_side(0x1000, None, 0x3000), abi.bcmt_side(0x1000, 0x2000, None),
                 abi.bcmt_side(None, None, None)):
        assert _bwd(c, side=side) == abi.BCMT_ERR_INVALID
    # the model step passes the same structure to its layers
    mc = abi.make_model_config(V=1000, d=128, H=8, n_layer=1, B=2, T=64, L=32)
    st = lib.bcmt_model_train_step(ctypes.byref(mc), 16, 16, 16, 16, 16, None, None, None, 16, 16,
                                   1 << 40, None, ctypes.byref(abi.bcmt_side(16, None, 16)))
    assert st == abi.BCMT_ERR_INVALID


def test_side_event_helpers_arguments(lib):
    """The event helpers reject a NULL structure; destroying a structure
    whose events are NULL makes no HIP call and succeeds."""
    assert lib.bcmt_side_events_create(None) == abi.BCMT_ERR_INVALID
    assert lib.bcmt_side_events_destroy(None) == abi.BCMT_ERR_INVALID
    s = abi.bcmt_side(0x1000, None, None)
    assert lib.bcmt_side_events_destroy(ctypes.byref(s)) == abi.BCMT_OK
    assert s.stream == 0x1000 and not s.fork and not s.join


def _carry(N, Z):
    return abi.bcmt_carry(N, Z)


def test_chunk_argument_errors(lib):
    """The chunked entry points check their states before anything runs."""
    c = good()
    p = _params()
    ws_f = abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_FORWARD)
    ws_b = abi.bcmt_workspace_bytes(c, abi.BCMT_PASS_BACKWARD)
    ok = _carry(A + 0x70000000, A + 0x71000000)

    def fwd(cin, cout, X=A):
        return lib.bcmt_layer_forward_chunk(
            ctypes.byref(c), X, ctypes.byref(p), ctypes.byref(cin) if cin else None,
            A + 0x10000000, ctypes.byref(cout) if cout else None, A + 0x20000000,
            A + 0x40000000, ws_f, None)

    def bwd(dout, din, saved=A + 0x20000000):
        return lib.bcmt_layer_backward_chunk(
            ctypes.byref(c), A, ctypes.byref(p), saved, A + 0x30000000,
            ctypes.byref(dout) if dout else None, A + 0x38000000,
            ctypes.byref(din) if din else None, None, A + 0x40000000, ws_b, None, None)

    for bad in (_carry(None, A + 0x71000000), _carry(A + 0x70000000, None),
                _carry(A + 0x70000008, A + 0x71000000), _carry(A + 0x70000000, A + 0x71000002)):
        assert fwd(bad, None) == abi.BCMT_ERR_INVALID
        assert fwd(ok, bad) == abi.BCMT_ERR_INVALID
        assert bwd(bad, None) == abi.BCMT_ERR_INVALID
        assert bwd(ok, bad) == abi.BCMT_ERR_INVALID
    assert fwd(ok, ok, X=None) == abi.BCMT_ERR_INVALID
    assert bwd(ok, ok, saved=None) == abi.BCMT_ERR_INVALID
    # the chunked passes use the same workspace sizes
    assert lib.bcmt_layer_forward_chunk(ctypes.byref(c), A, ctypes.byref(p), None, A + 0x10000000,
                                        None, A + 0x20000000, A + 0x40000000, ws_f - 1,
                                        None) == abi.BCMT_ERR_WORKSPACE


def test_decode_sizes_and_argument_errors(lib):
    """Decode sizes follow the config; bad arguments fail before any launch."""
    c = good()
    sb = abi.bcmt_decode_state_bytes(c)
    wb = abi.bcmt_decode_workspace_bytes(c)
    assert sb > 0 and wb > 0
    assert abi.bcmt_decode_state_bytes(good(L=128)) > sb      # caches grow with L
    assert abi.bcmt_decode_state_bytes(good(L=5000)) == 0     # block too long to decode
    assert abi.bcmt_decode_state_bytes(good(B=65)) == 0       # batch too large to decode
    assert abi.bcmt_decode_state_bytes(good(B=0)) == 0
    assert abi.bcmt_decode_state_bytes(good(D=128, H=8)) == 0   # decoding needs 64-wide heads
    p = _params()
    st, ws = A + 0x20000000, A + 0x40000000

    def step(t=0, x=A, y=A + 0x10000000, state=st, w=ws, n=wb, cfg=c):
        return lib.bcmt_decode_step(ctypes.byref(cfg), ctypes.byref(p), t, x, y, state, w, n, None)

    assert step(t=-1) == abi.BCMT_ERR_INVALID
    assert step(x=None) == abi.BCMT_ERR_INVALID
    assert step(y=A) == abi.BCMT_ERR_INVALID                 # y aliases x
    assert step(y=A + 8) == abi.BCMT_ERR_INVALID             # misaligned
    assert step(state=None) == abi.BCMT_ERR_INVALID
    assert step(n=wb - 1) == abi.BCMT_ERR_WORKSPACE
    assert step(cfg=good(L=5000)) == abi.BCMT_ERR_UNSUPPORTED
    assert lib.bcmt_decode_step(ctypes.byref(c), ctypes.byref(_params(Wg=None)), 0, A,
                                A + 0x10000000, st, ws, wb, None) == abi.BCMT_ERR_INVALID
    # reset reads only Wm
    none = abi.bcmt_params(*([None] * 7))
    assert lib.bcmt_decode_reset(ctypes.byref(c), ctypes.byref(none), None, st, ws, wb,
                                 None) == abi.BCMT_ERR_INVALID
    bad = abi.bcmt_carry(A + 0x70000000, None)
    assert lib.bcmt_decode_reset(ctypes.byref(c), ctypes.byref(p), ctypes.byref(bad), st, ws, wb,
                                 None) == abi.BCMT_ERR_INVALID
    assert lib.bcmt_decode_reset(ctypes.byref(c), ctypes.byref(p), None, st, ws, wb - 1,
                                 None) == abi.BCMT_ERR_WORKSPACE


def test_channel_decay_arguments(lib):
    """With BCMT_FLAG_CHANNEL_DECAY the per-channel decay must be given."""
    c = good()
    c.flags |= abi.BCMT_FLAG_CHANNEL_DECAY
    assert abi.bcmt_validate(c) == abi.BCMT_OK
    assert abi.bcmt_saved_bytes(c) == abi.bcmt_saved_bytes(good())
    bad = good()
    bad.flags |= 8
    assert abi.bcmt_validate(bad) == abi.BCMT_ERR_INVALID        # unknown flag
    assert _fwd(c) == abi.BCMT_ERR_INVALID                        # gamma_ch missing
    p = _params()
    p.gamma_ch = A + 0x7000002                                    # misaligned
    assert _fwd(c, params=p) == abi.BCMT_ERR_INVALID
    assert _bwd(c) == abi.BCMT_ERR_INVALID


def test_model_layout_and_argument_errors(lib):
    """The flat parameter vector holds the arrays of model_array_names back
    to back, in order; E has V rounded up to a multiple of 128 rows.
    Invalid configurations size to 0 and the step rejects null pointers
    before touching the GPU."""
    from paper_2608_13578_amd.inputs import make_model_inputs, model_array_names
    V, d, H, nl, B, T, L = 97, 64, 4, 2, 2, 96, 32
    c = abi.make_model_config(V, d, H, nl, B, T, L)
    arrs, _, _ = make_model_inputs(V, d, T, nl, B)
    names = model_array_names(nl)
    off = 0
    for i, (name, a) in enumerate(zip(names, arrs)):
        o, n = abi.bcmt_model_param_array(c, i)
        want = 128 * d if name == "E" else a.size
        assert (o, n) == (off, want), name
        off += n
    assert abi.bcmt_model_param_count(c) == off
    assert abi.bcmt_model_workspace_bytes(c) > 0
    for bad in (dict(V=1), dict(d=96), dict(d=2048), dict(H=3), dict(n_layer=0), dict(L=0),
                dict(V=65537), dict(B=1, T=7)):
        kw = dict(V=V, d=d, H=H, n_layer=nl, B=B, T=T, L=L)
        kw.update(bad)
        cb = abi.make_model_config(**kw)
        assert abi.bcmt_model_param_count(cb) == 0 and abi.bcmt_model_workspace_bytes(cb) == 0, bad
    with pytest.raises(abi.BcmtError) as e:
        abi.bcmt_model_param_array(c, len(names))
    assert e.value.status == abi.BCMT_ERR_INVALID
    for i in range(2):  # null tokens / workspace: rejected on the host
        st = lib.bcmt_model_train_step(ctypes.byref(c), None if i == 0 else 16, 16, 16, 16, 16,
                                       None, None, None, 16, None if i == 1 else 16, 1 << 40,
                                       None, None)
        assert st == abi.BCMT_ERR_INVALID
