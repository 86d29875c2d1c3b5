"""Python binding of libbcmt (the C ABI declared in include/bcmt.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  Tensors are passed as device pointers (``tensor.data_ptr()``); torch
is used by callers for device memory and streams.  The functions have the
names of the C entry points and raise ``BcmtError`` on a negative status.

If the shared library has not been built this module fails loudly on first
use; there is no fallback implementation.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbcmt.so")

BCMT_OK = 0
BCMT_ERR_INVALID = -1
BCMT_ERR_UNSUPPORTED = -2
BCMT_ERR_WORKSPACE = -3
BCMT_ERR_HIP = -4

BCMT_F32 = 0
BCMT_BF16 = 1

BCMT_FLAG_RESIDUAL = 1
BCMT_FLAG_ACCUM_WGRAD = 2
BCMT_FLAG_CHANNEL_DECAY = 4

BCMT_PASS_FORWARD = 0
BCMT_PASS_INFERENCE = 1
BCMT_PASS_BACKWARD = 2

EXPORTED = ("bcmt_validate", "bcmt_saved_bytes", "bcmt_workspace_bytes", "bcmt_layer_forward",
            "bcmt_layer_forward_noalloc",
            "bcmt_layer_backward", "bcmt_layer_forward_chunk", "bcmt_layer_backward_chunk",
            "bcmt_decode_state_bytes", "bcmt_decode_workspace_bytes", "bcmt_decode_reset",
            "bcmt_decode_step", "bcmt_strerror", "bcmt_version", "bcmt_side_events_create",
            "bcmt_side_events_destroy", "bcmt_trace_enable",
            "bcmt_trace_read", "bcmt_model_param_count", "bcmt_model_param_array",
            "bcmt_model_workspace_bytes", "bcmt_model_cast", "bcmt_model_train_step")

PARAM_NAMES = ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")
GRAD_NAMES = ("dWq", "dWk", "dWv", "dWo", "dWm", "dWg", "dwp", "dgamma")
# the per-channel decay and its gradient (read with BCMT_FLAG_CHANNEL_DECAY)
PARAM_FIELDS = PARAM_NAMES + ("gamma_ch",)
GRAD_FIELDS = GRAD_NAMES + ("dgamma_ch",)


class BcmtError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {bcmt_strerror(status)} ({status})")


class bcmt_config(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("D", ctypes.c_int32),
                ("H", ctypes.c_int32), ("L", ctypes.c_int32), ("gamma", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("flags", ctypes.c_int32)]


class bcmt_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS]


class bcmt_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in GRAD_FIELDS]


class bcmt_carry(ctypes.Structure):
    """Memory state between chunks: N [B, D] and Z [B], float32 device pointers."""
    _fields_ = [("N", ctypes.c_void_p), ("Z", ctypes.c_void_p)]


class bcmt_side(ctypes.Structure):
    """A second stream and its fork / join events (hipStream_t, hipEvent_t)."""
    _fields_ = [("stream", ctypes.c_void_p), ("fork", ctypes.c_void_p), ("join", ctypes.c_void_p)]


class bcmt_model_config(ctypes.Structure):
    _fields_ = [("V", ctypes.c_int32), ("d", ctypes.c_int32), ("H", ctypes.c_int32),
                ("n_layer", ctypes.c_int32), ("B", ctypes.c_int32), ("T", ctypes.c_int32),
                ("L", ctypes.c_int32), ("gamma", ctypes.c_float)]


class bcmt_adamw(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("step", ctypes.c_int32)]


class bcmt_trace_entry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("calls", ctypes.c_int32), ("total_ms", ctypes.c_double)]


_lib = None


def lib():
    """The loaded shared library (loaded once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it first with "
                "`python -m paper_2608_13578_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        cfgp = ctypes.POINTER(bcmt_config)
        vp = ctypes.c_void_p
        L.bcmt_validate.argtypes = [cfgp]
        L.bcmt_validate.restype = ctypes.c_int
        L.bcmt_saved_bytes.argtypes = [cfgp]
        L.bcmt_saved_bytes.restype = ctypes.c_size_t
        L.bcmt_workspace_bytes.argtypes = [cfgp, ctypes.c_int]
        L.bcmt_workspace_bytes.restype = ctypes.c_size_t
        L.bcmt_layer_forward.argtypes = [cfgp, vp, ctypes.POINTER(bcmt_params), vp, vp, vp,
                                         ctypes.c_size_t, vp]
        L.bcmt_layer_forward.restype = ctypes.c_int
        L.bcmt_layer_forward_noalloc.argtypes = [cfgp, vp, ctypes.POINTER(bcmt_params), vp, vp, vp]
        L.bcmt_layer_forward_noalloc.restype = ctypes.c_int
        sidep = ctypes.POINTER(bcmt_side)
        L.bcmt_layer_backward.argtypes = [cfgp, vp, ctypes.POINTER(bcmt_params), vp, vp, vp,
                                          ctypes.POINTER(bcmt_grads), vp, ctypes.c_size_t, vp,
                                          sidep]
        L.bcmt_layer_backward.restype = ctypes.c_int
        carryp = ctypes.POINTER(bcmt_carry)
        L.bcmt_layer_forward_chunk.argtypes = [cfgp, vp, ctypes.POINTER(bcmt_params), carryp, vp,
                                               carryp, vp, vp, ctypes.c_size_t, vp]
        L.bcmt_layer_forward_chunk.restype = ctypes.c_int
        L.bcmt_layer_backward_chunk.argtypes = [cfgp, vp, ctypes.POINTER(bcmt_params), vp, vp,
                                                carryp, vp, carryp, ctypes.POINTER(bcmt_grads),
                                                vp, ctypes.c_size_t, vp, sidep]
        L.bcmt_layer_backward_chunk.restype = ctypes.c_int
        L.bcmt_decode_state_bytes.argtypes = [cfgp]
        L.bcmt_decode_state_bytes.restype = ctypes.c_size_t
        L.bcmt_decode_workspace_bytes.argtypes = [cfgp]
        L.bcmt_decode_workspace_bytes.restype = ctypes.c_size_t
        L.bcmt_decode_reset.argtypes = [cfgp, ctypes.POINTER(bcmt_params), carryp, vp, vp,
                                        ctypes.c_size_t, vp]
        L.bcmt_decode_reset.restype = ctypes.c_int
        L.bcmt_decode_step.argtypes = [cfgp, ctypes.POINTER(bcmt_params), ctypes.c_int64, vp, vp,
                                       vp, vp, ctypes.c_size_t, vp]
        L.bcmt_decode_step.restype = ctypes.c_int
        L.bcmt_strerror.argtypes = [ctypes.c_int]
        L.bcmt_strerror.restype = ctypes.c_char_p
        L.bcmt_version.argtypes = []
        L.bcmt_version.restype = ctypes.c_int
        L.bcmt_side_events_create.argtypes = [ctypes.POINTER(bcmt_side)]
        L.bcmt_side_events_create.restype = ctypes.c_int
        L.bcmt_side_events_destroy.argtypes = [ctypes.POINTER(bcmt_side)]
        L.bcmt_side_events_destroy.restype = ctypes.c_int
        L.bcmt_trace_enable.argtypes = [ctypes.c_int]
        L.bcmt_trace_enable.restype = ctypes.c_int
        L.bcmt_trace_read.argtypes = [ctypes.POINTER(bcmt_trace_entry), ctypes.c_int]
        L.bcmt_trace_read.restype = ctypes.c_int
        mcp = ctypes.POINTER(bcmt_model_config)
        L.bcmt_model_param_count.argtypes = [mcp]
        L.bcmt_model_param_count.restype = ctypes.c_size_t
        L.bcmt_model_param_array.argtypes = [mcp, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t),
                                             ctypes.POINTER(ctypes.c_size_t)]
        L.bcmt_model_param_array.restype = ctypes.c_int
        L.bcmt_model_workspace_bytes.argtypes = [mcp]
        L.bcmt_model_workspace_bytes.restype = ctypes.c_size_t
        L.bcmt_model_cast.argtypes = [mcp, vp, vp, vp]
        L.bcmt_model_cast.restype = ctypes.c_int
        L.bcmt_model_train_step.argtypes = [mcp, vp, vp, vp, vp, vp, vp, vp,
                                            ctypes.POINTER(bcmt_adamw), vp, vp, ctypes.c_size_t,
                                            vp, sidep]
        L.bcmt_model_train_step.restype = ctypes.c_int
        _lib = L
    return _lib


def make_config(B, T, D, H, L, gamma=0.8, dtype="bf16", residual=False, accumulate=False,
                channel_decay=False):
    """A bcmt_config from plain values (dtype "bf16" or "f32")."""
    flags = ((BCMT_FLAG_RESIDUAL if residual else 0) | (BCMT_FLAG_ACCUM_WGRAD if accumulate else 0)
             | (BCMT_FLAG_CHANNEL_DECAY if channel_decay else 0))
    dt = {"bf16": BCMT_BF16, "f32": BCMT_F32}[dtype]
    return bcmt_config(int(B), int(T), int(D), int(H), int(L), float(gamma), dt, flags)


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _params(p):
    if isinstance(p, bcmt_params):
        return p
    return bcmt_params(*[_ptr(p[n]) for n in PARAM_NAMES], _ptr(p.get("gamma_ch")))


def _params_partial(p):
    """Like _params, but members missing from a dict are NULL."""
    if isinstance(p, bcmt_params):
        return p
    return bcmt_params(*[_ptr(p.get(n)) for n in PARAM_FIELDS])


def _grads(g):
    if g is None or isinstance(g, bcmt_grads):
        return g
    return bcmt_grads(*[_ptr(g.get(n)) for n in GRAD_FIELDS])


def _carry(c):
    """None, a bcmt_carry, or an (N, Z) pair of tensors / pointers."""
    if c is None or isinstance(c, bcmt_carry):
        return c
    return bcmt_carry(_ptr(c[0]), _ptr(c[1]))


def _side(side):
    """None, a bcmt_side, or an object with .stream, .fork and .join (torch
    stream and events, or raw handles)."""
    if side is None or isinstance(side, bcmt_side):
        return side

    def h(x, attr):
        return x if isinstance(x, int) else getattr(x, attr)
    return bcmt_side(h(side.stream, "cuda_stream"), h(side.fork, "cuda_event"),
                     h(side.join, "cuda_event"))


def _ref(x):
    return ctypes.byref(x) if x is not None else None


def _nbytes(x):
    return x.numel() * x.element_size()


def bcmt_strerror(status):
    return lib().bcmt_strerror(int(status)).decode()


def bcmt_version():
    return lib().bcmt_version()


def bcmt_side_events_create(side):
    """Fills side.fork and side.join (a bcmt_side) with new events."""
    st = lib().bcmt_side_events_create(ctypes.byref(side))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_side_events_create")


def bcmt_side_events_destroy(side):
    st = lib().bcmt_side_events_destroy(ctypes.byref(side))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_side_events_destroy")


def bcmt_validate(cfg):
    return lib().bcmt_validate(ctypes.byref(cfg))


def bcmt_saved_bytes(cfg):
    return lib().bcmt_saved_bytes(ctypes.byref(cfg))


def bcmt_workspace_bytes(cfg, pass_):
    return lib().bcmt_workspace_bytes(ctypes.byref(cfg), int(pass_))


def bcmt_layer_forward(cfg, X, params, Y, saved, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    st = lib().bcmt_layer_forward(ctypes.byref(cfg), _ptr(X), ctypes.byref(_params(params)),
                                  _ptr(Y), _ptr(saved), _ptr(ws), int(ws_bytes), _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_layer_forward")


# bytes of the library's own forward scratch (bcmt_layer_forward_noalloc)
BCMT_NOALLOC_SCRATCH_BYTES = 32 << 20


def bcmt_layer_forward_noalloc(cfg, X, params, Y, saved, stream=None):
    st = lib().bcmt_layer_forward_noalloc(ctypes.byref(cfg), _ptr(X),
                                          ctypes.byref(_params(params)), _ptr(Y), _ptr(saved),
                                          _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_layer_forward_noalloc")


def bcmt_layer_backward(cfg, X, params, saved, dY, dX, grads, ws, ws_bytes=None, stream=None,
                        side=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    g = _grads(grads)
    st = lib().bcmt_layer_backward(ctypes.byref(cfg), _ptr(X), ctypes.byref(_params(params)),
                                   _ptr(saved), _ptr(dY), _ptr(dX),
                                   ctypes.byref(g) if g is not None else None, _ptr(ws),
                                   int(ws_bytes), _stream(stream), _ref(_side(side)))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_layer_backward")


def bcmt_layer_forward_chunk(cfg, X, params, carry_in, Y, carry_out, saved, ws, ws_bytes=None,
                             stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    st = lib().bcmt_layer_forward_chunk(ctypes.byref(cfg), _ptr(X), ctypes.byref(_params(params)),
                                        _ref(_carry(carry_in)), _ptr(Y), _ref(_carry(carry_out)),
                                        _ptr(saved), _ptr(ws), int(ws_bytes), _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_layer_forward_chunk")


def bcmt_layer_backward_chunk(cfg, X, params, saved, dY, dcarry_out, dX, dcarry_in, grads, ws,
                              ws_bytes=None, stream=None, side=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    g = _grads(grads)
    st = lib().bcmt_layer_backward_chunk(ctypes.byref(cfg), _ptr(X), ctypes.byref(_params(params)),
                                         _ptr(saved), _ptr(dY), _ref(_carry(dcarry_out)), _ptr(dX),
                                         _ref(_carry(dcarry_in)), _ref(g), _ptr(ws), int(ws_bytes),
                                         _stream(stream), _ref(_side(side)))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_layer_backward_chunk")


def bcmt_decode_state_bytes(cfg):
    return lib().bcmt_decode_state_bytes(ctypes.byref(cfg))


def bcmt_decode_workspace_bytes(cfg):
    return lib().bcmt_decode_workspace_bytes(ctypes.byref(cfg))


def bcmt_decode_reset(cfg, params, carry_in, state, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    st = lib().bcmt_decode_reset(ctypes.byref(cfg), ctypes.byref(_params_partial(params)),
                                 _ref(_carry(carry_in)), _ptr(state), _ptr(ws), int(ws_bytes),
                                 _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_decode_reset")


def bcmt_decode_step(cfg, params, t, x, y, state, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    st = lib().bcmt_decode_step(ctypes.byref(cfg), ctypes.byref(_params(params)), int(t), _ptr(x),
                                _ptr(y), _ptr(state), _ptr(ws), int(ws_bytes), _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_decode_step")


def bcmt_trace_enable(on):
    return lib().bcmt_trace_enable(1 if on else 0)


def bcmt_trace_read(max_entries=64):
    """Per-stage totals since the last read: list of (name, calls, total_ms)."""
    buf = (bcmt_trace_entry * max_entries)()
    n = lib().bcmt_trace_read(buf, max_entries)
    if n < 0:
        raise BcmtError(n, "bcmt_trace_read")
    return [(buf[i].name.decode(), buf[i].calls, buf[i].total_ms) for i in range(min(n, max_entries))]


# ---- language model built from BCMT layers


def make_model_config(V, d, H, n_layer, B, T, L, gamma=0.8):
    return bcmt_model_config(int(V), int(d), int(H), int(n_layer), int(B), int(T), int(L),
                             float(gamma))


def bcmt_model_param_count(cfg):
    return lib().bcmt_model_param_count(ctypes.byref(cfg))


def bcmt_model_param_array(cfg, index):
    """(offset, count) in elements of array `index` of the flat vector."""
    off, cnt = ctypes.c_size_t(), ctypes.c_size_t()
    st = lib().bcmt_model_param_array(ctypes.byref(cfg), int(index), ctypes.byref(off),
                                      ctypes.byref(cnt))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_model_param_array")
    return off.value, cnt.value


def bcmt_model_workspace_bytes(cfg):
    return lib().bcmt_model_workspace_bytes(ctypes.byref(cfg))


def bcmt_model_cast(cfg, params, params_bf16, stream=None):
    st = lib().bcmt_model_cast(ctypes.byref(cfg), _ptr(params), _ptr(params_bf16),
                               _stream(stream))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_model_cast")


def bcmt_model_train_step(cfg, tokens, targets, params, params_bf16, grads, adam_m, adam_v, opt,
                          loss, ws, ws_bytes=None, stream=None, side=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else _nbytes(ws)
    st = lib().bcmt_model_train_step(ctypes.byref(cfg), _ptr(tokens), _ptr(targets),
                                     _ptr(params), _ptr(params_bf16), _ptr(grads), _ptr(adam_m),
                                     _ptr(adam_v), _ref(opt), _ptr(loss), _ptr(ws),
                                     int(ws_bytes), _stream(stream), _ref(_side(side)))
    if st != BCMT_OK:
        raise BcmtError(st, "bcmt_model_train_step")
