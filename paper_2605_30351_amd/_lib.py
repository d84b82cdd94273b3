"""ctypes binding of libvideomla.so: argument marshalling only.

Every computation runs in the library's HIP kernels; this module converts torch tensors to
device pointers, the current HIP stream to a handle, and return codes to exceptions. It raises
at import time if the shared library has not been built, and never falls back to anything else.

With VIDEOMLA_LIBRARY=stamps in the environment at import, it loads the diagnostic build
libvideomla_stamps.so instead (the same calls, plus phase stamps: include/videomla_stamps.h).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
_VARIANT = os.environ.get("VIDEOMLA_LIBRARY", "")
if _VARIANT not in ("", "stamps"):
    raise ImportError(f"VIDEOMLA_LIBRARY={_VARIANT!r}: only 'stamps' (the diagnostic build) is known")
STAMPS = _VARIANT == "stamps"
LIB_PATH = os.path.join(_PKG, "libvideomla_stamps.so" if STAMPS else "libvideomla.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with "
                      f"`python paper_2605_30351_amd/build.py{' --stamps' if STAMPS else ''}`")

_lib = ctypes.CDLL(LIB_PATH)

OK, EINVAL, EUNSUPPORTED, EALIGN, EWORKSPACE, EHIP = 0, 1, 2, 3, 4, 5

EXPORTED = (
    "videomla_cache_write", "videomla_write_weights_bytes", "videomla_prepare_write_weights",
    "videomla_cache_write_prepared", "videomla_attend_workspace_bytes", "videomla_attend",
    "videomla_attend_workspace_bytes_ex", "videomla_attend_ex", "videomla_attend_noalloc",
    "videomla_window_advance", "videomla_cache_bytes_per_token", "videomla_valid_tokens",
    "videomla_slot_of", "videomla_last_error",
    "videomla_timer_create", "videomla_timer_destroy", "videomla_timer_only",
    "videomla_timer_begin", "videomla_timer_end", "videomla_timer_read",
    "videomla_dense_cache_bytes_per_token", "videomla_dense_cache_write",
    "videomla_dense_attend_workspace_bytes", "videomla_dense_attend",
    "videomla_layer_weights_bytes", "videomla_prepare_layer_weights",
    "videomla_attend_layer_workspace_bytes", "videomla_attend_layer",
)

# the diagnostic build's one extra call (include/videomla_stamps.h)
EXPORTED_STAMPS = ("videomla_stamps_attach",)
STAMP_KERNELS, STAMP_WORKGROUPS, STAMP_WAVES, STAMP_POINTS = 5, 2048, 8, 16
STAMP_KERNEL = {"cache_write_packed": 0, "cache_write_wide": 1, "q_absorb": 2,
                "latent_attend": 3, "out_proj": 4}

PARTITION = {"even": 0, "adaptive": 1, "frozen": 2}
NOALLOC_SCRATCH_BYTES = 64 << 20  # VIDEOMLA_NOALLOC_SCRATCH_BYTES
FORM = {"latent": 0, "materialized": 1, "auto": 2}


class VideomlaDims(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("d_nope", ctypes.c_int32),
        ("d_rope", ctypes.c_int32), ("d_c", ctypes.c_int32), ("d_v", ctypes.c_int32),
        ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
        ("window_frames", ctypes.c_int32), ("chunk_frames", ctypes.c_int32),
        ("rope_pairs", ctypes.c_int32 * 3), ("rope_band_dim", ctypes.c_int32 * 3),
        ("rope_base", ctypes.c_float), ("softmax_scale", ctypes.c_float),
        ("kv_norm_eps", ctypes.c_float), ("sink_frames", ctypes.c_int32),
    ]


class VideomlaWindow(ctypes.Structure):
    _fields_ = [("frame_end", ctypes.c_int64)]


class VideomlaAttendOpts(ctypes.Structure):
    _fields_ = [("n_workgroups", ctypes.c_int32), ("partition", ctypes.c_int32),
                ("form", ctypes.c_int32), ("query_begin", ctypes.c_int32),
                ("query_count", ctypes.c_int32), ("timer", ctypes.c_void_p)]


_P = ctypes.c_void_p
_DP = ctypes.POINTER(VideomlaDims)
_WP = ctypes.POINTER(VideomlaWindow)
_OP = ctypes.POINTER(VideomlaAttendOpts)

_lib.videomla_cache_write.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.videomla_cache_write.restype = ctypes.c_int
_lib.videomla_write_weights_bytes.argtypes = [_DP]
_lib.videomla_write_weights_bytes.restype = ctypes.c_size_t
_lib.videomla_prepare_write_weights.argtypes = [_DP, _P, _P, _P, _P]
_lib.videomla_prepare_write_weights.restype = ctypes.c_int
_lib.videomla_cache_write_prepared.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P]
_lib.videomla_cache_write_prepared.restype = ctypes.c_int
_lib.videomla_attend_workspace_bytes.argtypes = [_DP, ctypes.c_int32]
_lib.videomla_attend_workspace_bytes.restype = ctypes.c_size_t
_lib.videomla_attend.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P,
                                 ctypes.c_size_t, _P]
_lib.videomla_attend.restype = ctypes.c_int
_lib.videomla_attend_workspace_bytes_ex.argtypes = [_DP, ctypes.c_int32, _OP]
_lib.videomla_attend_workspace_bytes_ex.restype = ctypes.c_size_t
_lib.videomla_attend_ex.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P,
                                    ctypes.c_size_t, _OP, _P]
_lib.videomla_attend_ex.restype = ctypes.c_int
_lib.videomla_attend_noalloc.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.videomla_attend_noalloc.restype = ctypes.c_int
_lib.videomla_window_advance.argtypes = [_DP, _WP]
_lib.videomla_window_advance.restype = ctypes.c_int
_lib.videomla_cache_bytes_per_token.argtypes = [_DP]
_lib.videomla_cache_bytes_per_token.restype = ctypes.c_size_t
_lib.videomla_valid_tokens.argtypes = [_DP, _WP]
_lib.videomla_valid_tokens.restype = ctypes.c_int64
_lib.videomla_slot_of.argtypes = [_DP, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32]
_lib.videomla_slot_of.restype = ctypes.c_int64
_lib.videomla_last_error.argtypes = []
_lib.videomla_last_error.restype = ctypes.c_char_p
_lib.videomla_timer_create.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
_lib.videomla_timer_create.restype = ctypes.c_int
_lib.videomla_timer_destroy.argtypes = [_P]
_lib.videomla_timer_destroy.restype = ctypes.c_int
_lib.videomla_timer_only.argtypes = [_P, ctypes.c_char_p]
_lib.videomla_timer_only.restype = ctypes.c_int
_lib.videomla_timer_begin.argtypes = [_P, ctypes.c_char_p, _P]
_lib.videomla_timer_begin.restype = ctypes.c_int
_lib.videomla_timer_end.argtypes = [_P, ctypes.c_char_p, _P]
_lib.videomla_timer_end.restype = ctypes.c_int
_lib.videomla_timer_read.argtypes = [_P, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_double)]
_lib.videomla_timer_read.restype = ctypes.c_int
_lib.videomla_dense_cache_bytes_per_token.argtypes = [_DP]
_lib.videomla_dense_cache_bytes_per_token.restype = ctypes.c_size_t
_lib.videomla_dense_cache_write.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, _P, _P]
_lib.videomla_dense_cache_write.restype = ctypes.c_int
_lib.videomla_dense_attend_workspace_bytes.argtypes = [_DP, ctypes.c_int32, _OP]
_lib.videomla_dense_attend_workspace_bytes.restype = ctypes.c_size_t
_lib.videomla_dense_attend.argtypes = [_DP, _WP, ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t,
                                       _OP, _P]
_lib.videomla_dense_attend.restype = ctypes.c_int
_lib.videomla_layer_weights_bytes.argtypes = [_DP, ctypes.c_int32]
_lib.videomla_layer_weights_bytes.restype = ctypes.c_size_t
_lib.videomla_prepare_layer_weights.argtypes = [_DP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P,
                                                _P, ctypes.c_size_t, _P]
_lib.videomla_prepare_layer_weights.restype = ctypes.c_int
_lib.videomla_attend_layer_workspace_bytes.argtypes = [_DP, ctypes.c_int32, ctypes.c_int32, _OP]
_lib.videomla_attend_layer_workspace_bytes.restype = ctypes.c_size_t
_lib.videomla_attend_layer.argtypes = [_DP, _WP, ctypes.c_int32, ctypes.c_int32, _P, _P,
                                       ctypes.c_size_t, _P, _P, _P, _P, ctypes.c_size_t, _OP, _P]
_lib.videomla_attend_layer.restype = ctypes.c_int
if STAMPS:
    _lib.videomla_stamps_attach.argtypes = [_P, ctypes.c_int64]
    _lib.videomla_stamps_attach.restype = ctypes.c_int


class VideomlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"videomla error {code}: {msg}")
        self.code = code


def _check(code: int):
    if code != OK:
        raise VideomlaError(code, _lib.videomla_last_error().decode())


def make_dims(d) -> VideomlaDims:
    """Build the C struct from any object with the Dims field names."""
    s = VideomlaDims()
    for name in ("d_model", "n_heads", "d_nope", "d_rope", "d_c", "d_v", "grid_h", "grid_w",
                 "window_frames", "chunk_frames"):
        setattr(s, name, int(getattr(d, name)))
    for i in range(3):
        s.rope_pairs[i] = int(d.rope_pairs[i])
        s.rope_band_dim[i] = int(d.rope_band_dim[i])
    s.rope_base = float(d.rope_base)
    s.softmax_scale = float(d.softmax_scale)
    s.kv_norm_eps = float(d.kv_norm_eps)
    s.sink_frames = int(getattr(d, "sink_frames", 0))
    return s


class Timer:
    """A caller-owned videomla_timer: kernels of the attention calls whose options name it are
    bracketed by HIP events on their stream."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(_lib.videomla_timer_create(ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    def only(self, kernel: str | None = None):
        """Bracket only this kernel's launches (None: every kernel)."""
        _check(_lib.videomla_timer_only(self._h, None if kernel is None else kernel.encode()))

    def begin(self, kernel: str, stream=None):
        """videomla_timer_begin on the stream (default: torch's current stream)."""
        _check(_lib.videomla_timer_begin(self._h, kernel.encode(), _stream(stream)))

    def end(self, kernel: str, stream=None):
        """videomla_timer_end on the stream (default: torch's current stream)."""
        _check(_lib.videomla_timer_end(self._h, kernel.encode(), _stream(stream)))

    def read(self, kernel: str) -> tuple[int, float]:
        """(launches, total ms) of the completed launches of `kernel` since the last read."""
        c, t = ctypes.c_int64(0), ctypes.c_double(0.0)
        _check(_lib.videomla_timer_read(self._h, kernel.encode(), ctypes.byref(c),
                                        ctypes.byref(t)))
        return int(c.value), float(t.value)

    def close(self):
        if self._h is not None and self._h.value:
            _lib.videomla_timer_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


@dataclasses.dataclass
class AttendOpts:
    """videomla_attend_opts: workgroups (0 = one per compute unit), partition ("even",
    "adaptive", "frozen"), form ("latent", "materialized", "auto"), the block of query tokens
    [query_begin, query_begin + query_count) of the chunk (query_count 0 = to its end), timer."""

    n_workgroups: int = 0
    partition: str = "even"
    form: str = "latent"
    query_begin: int = 0
    query_count: int = 0
    timer: Timer | None = None

    def struct(self) -> VideomlaAttendOpts:
        o = VideomlaAttendOpts()
        o.n_workgroups = int(self.n_workgroups)
        o.partition = PARTITION[self.partition]
        o.form = FORM[self.form]
        o.query_begin = int(self.query_begin)
        o.query_count = int(self.query_count)
        o.timer = self.timer.handle if self.timer is not None else None
        return o

    def n_queries(self, dims) -> int:
        """Query tokens per batch element of a call with these options."""
        chunk = int(dims.chunk_frames) * int(dims.grid_h) * int(dims.grid_w)
        return int(self.query_count) if self.query_count else chunk - int(self.query_begin)


def _opts(opts: AttendOpts | None):
    return ctypes.byref(opts.struct()) if opts is not None else None


def _nq(dims, opts):
    return (opts or AttendOpts()).n_queries(dims)


def _ptr(t: torch.Tensor | None, name: str, dtypes=(torch.bfloat16, torch.int16, torch.uint16)):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, numel: int):
    if t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")


def cache_write(dims, frame_end: int, batch: int, x, w_dkv, w_kr, gamma, c_kv, k_r, slots=None,
                stream=None):
    """videomla_cache_write on torch tensors (bf16 data, int32 slots)."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    _need(x, "x", batch * d.chunk_frames * hw * d.d_model)
    _need(w_dkv, "w_dkv", d.d_c * d.d_model)
    _need(w_kr, "w_kr", d.d_rope * d.d_model)
    _need(c_kv, "c_kv", batch * d.window_frames * hw * d.d_c)
    _need(k_r, "k_r", batch * d.window_frames * hw * d.d_rope)
    if gamma is not None:
        _need(gamma, "gamma", d.d_c)
    if slots is not None:
        _need(slots, "slots", d.chunk_frames * hw)
    w = VideomlaWindow(int(frame_end))
    _check(_lib.videomla_cache_write(
        ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(x, "x"), _ptr(w_dkv, "w_dkv"),
        _ptr(w_kr, "w_kr"), _ptr(gamma, "gamma"), _ptr(c_kv, "c_kv"), _ptr(k_r, "k_r"),
        _ptr(slots, "slots", (torch.int32,)), _stream(stream)))


def write_weights_bytes(dims) -> int:
    return int(_lib.videomla_write_weights_bytes(ctypes.byref(make_dims(dims))))


def prepare_write_weights(dims, w_dkv, w_kr, w_packed, stream=None):
    """videomla_prepare_write_weights; `w_packed` is a bf16 or uint8 device tensor."""
    d = make_dims(dims)
    _need(w_dkv, "w_dkv", d.d_c * d.d_model)
    _need(w_kr, "w_kr", d.d_rope * d.d_model)
    nbytes = w_packed.numel() * w_packed.element_size()
    if nbytes < write_weights_bytes(dims):
        raise ValueError(f"w_packed holds {nbytes} bytes, needs {write_weights_bytes(dims)}")
    _check(_lib.videomla_prepare_write_weights(
        ctypes.byref(d), _ptr(w_dkv, "w_dkv"), _ptr(w_kr, "w_kr"),
        _ptr(w_packed, "w_packed", (torch.bfloat16, torch.uint8)), _stream(stream)))


def cache_write_prepared(dims, frame_end: int, batch: int, x, w_packed, gamma, c_kv, k_r,
                         slots=None, stream=None):
    """videomla_cache_write_prepared on torch tensors (bf16 data, int32 slots)."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    _need(x, "x", batch * d.chunk_frames * hw * d.d_model)
    _need(c_kv, "c_kv", batch * d.window_frames * hw * d.d_c)
    _need(k_r, "k_r", batch * d.window_frames * hw * d.d_rope)
    nbytes = w_packed.numel() * w_packed.element_size()
    if nbytes < write_weights_bytes(dims):
        raise ValueError(f"w_packed holds {nbytes} bytes, needs {write_weights_bytes(dims)}")
    if gamma is not None:
        _need(gamma, "gamma", d.d_c)
    if slots is not None:
        _need(slots, "slots", d.chunk_frames * hw)
    w = VideomlaWindow(int(frame_end))
    _check(_lib.videomla_cache_write_prepared(
        ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(x, "x"),
        _ptr(w_packed, "w_packed", (torch.bfloat16, torch.uint8)), _ptr(gamma, "gamma"),
        _ptr(c_kv, "c_kv"), _ptr(k_r, "k_r"), _ptr(slots, "slots", (torch.int32,)),
        _stream(stream)))


def attend_workspace_bytes(dims, batch: int, opts: AttendOpts | None = None) -> int:
    """videomla_attend_workspace_bytes, or videomla_attend_workspace_bytes_ex with opts."""
    d = make_dims(dims)
    if opts is None:
        return int(_lib.videomla_attend_workspace_bytes(ctypes.byref(d), int(batch)))
    o = opts.struct()
    return int(_lib.videomla_attend_workspace_bytes_ex(ctypes.byref(d), int(batch), ctypes.byref(o)))


def attend(dims, frame_end: int, batch: int, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, workspace,
           stream=None, opts: AttendOpts | None = None):
    """videomla_attend on torch tensors, or videomla_attend_ex when `opts` is given;
    `workspace` is a uint8 device tensor."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    nq = _nq(dims, opts)
    _need(q_nope, "q_nope", batch * nq * d.n_heads * d.d_nope)
    _need(q_r, "q_r", batch * nq * d.n_heads * d.d_rope)
    _need(w_uk, "w_uk", d.n_heads * d.d_nope * d.d_c)
    _need(w_uv, "w_uv", d.n_heads * d.d_v * d.d_c)
    _need(c_kv, "c_kv", batch * d.window_frames * hw * d.d_c)
    _need(k_r, "k_r", batch * d.window_frames * hw * d.d_rope)
    _need(out, "out", batch * nq * d.n_heads * d.d_v)
    w = VideomlaWindow(int(frame_end))
    ws = _ptr(workspace, "workspace", (torch.uint8,))
    args = [ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(q_nope, "q_nope"), _ptr(q_r, "q_r"),
            _ptr(w_uk, "w_uk"), _ptr(w_uv, "w_uv"), _ptr(c_kv, "c_kv"), _ptr(k_r, "k_r"),
            _ptr(out, "out"), ws, workspace.numel() if workspace is not None else 0]
    if opts is None:
        _check(_lib.videomla_attend(*args, _stream(stream)))
    else:
        o = opts.struct()
        _check(_lib.videomla_attend_ex(*args, ctypes.byref(o), _stream(stream)))


def attend_noalloc(dims, frame_end: int, batch: int, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out,
                   stream=None):
    """videomla_attend_noalloc on torch tensors: videomla_attend with the library's static
    scratch array as its workspace (shapes needing more than NOALLOC_SCRATCH_BYTES raise)."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    nq = d.chunk_frames * hw
    _need(q_nope, "q_nope", batch * nq * d.n_heads * d.d_nope)
    _need(q_r, "q_r", batch * nq * d.n_heads * d.d_rope)
    _need(w_uk, "w_uk", d.n_heads * d.d_nope * d.d_c)
    _need(w_uv, "w_uv", d.n_heads * d.d_v * d.d_c)
    _need(c_kv, "c_kv", batch * d.window_frames * hw * d.d_c)
    _need(k_r, "k_r", batch * d.window_frames * hw * d.d_rope)
    _need(out, "out", batch * nq * d.n_heads * d.d_v)
    w = VideomlaWindow(int(frame_end))
    _check(_lib.videomla_attend_noalloc(
        ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(q_nope, "q_nope"), _ptr(q_r, "q_r"),
        _ptr(w_uk, "w_uk"), _ptr(w_uv, "w_uv"), _ptr(c_kv, "c_kv"), _ptr(k_r, "k_r"),
        _ptr(out, "out"), _stream(stream)))


def dense_cache_bytes_per_token(dims) -> int:
    return int(_lib.videomla_dense_cache_bytes_per_token(ctypes.byref(make_dims(dims))))


def dense_cache_write(dims, frame_end: int, batch: int, x, w_k, w_v, kv, slots=None,
                      stream=None):
    """videomla_dense_cache_write on torch tensors (the dense per-head comparator)."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    _need(x, "x", batch * d.chunk_frames * hw * d.d_model)
    _need(w_k, "w_k", d.n_heads * d.d_v * d.d_model)
    _need(w_v, "w_v", d.n_heads * d.d_v * d.d_model)
    _need(kv, "kv", batch * d.window_frames * hw * d.n_heads * 2 * d.d_v)
    if slots is not None:
        _need(slots, "slots", d.chunk_frames * hw)
    w = VideomlaWindow(int(frame_end))
    _check(_lib.videomla_dense_cache_write(
        ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(x, "x"), _ptr(w_k, "w_k"),
        _ptr(w_v, "w_v"), _ptr(kv, "kv"), _ptr(slots, "slots", (torch.int32,)), _stream(stream)))


def dense_attend_workspace_bytes(dims, batch: int, opts: AttendOpts | None = None) -> int:
    o = opts.struct() if opts is not None else None
    return int(_lib.videomla_dense_attend_workspace_bytes(
        ctypes.byref(make_dims(dims)), int(batch), ctypes.byref(o) if o is not None else None))


def dense_attend(dims, frame_end: int, batch: int, q, kv, out, workspace, stream=None,
                 opts: AttendOpts | None = None):
    """videomla_dense_attend on torch tensors; `workspace` is a uint8 device tensor."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    nq = _nq(dims, opts)
    _need(q, "q", batch * nq * d.n_heads * d.d_v)
    _need(kv, "kv", batch * d.window_frames * hw * d.n_heads * 2 * d.d_v)
    _need(out, "out", batch * nq * d.n_heads * d.d_v)
    w = VideomlaWindow(int(frame_end))
    ws = _ptr(workspace, "workspace", (torch.uint8,))
    o = opts.struct() if opts is not None else None
    _check(_lib.videomla_dense_attend(
        ctypes.byref(d), ctypes.byref(w), int(batch), _ptr(q, "q"), _ptr(kv, "kv"),
        _ptr(out, "out"), ws, workspace.numel() if workspace is not None else 0,
        ctypes.byref(o) if o is not None else None, _stream(stream)))


def layer_weights_bytes(dims, d_q: int) -> int:
    return int(_lib.videomla_layer_weights_bytes(ctypes.byref(make_dims(dims)), int(d_q)))


def prepare_layer_weights(dims, d_q: int, w_dq, gamma_q, w_uq, w_qr, w_uk, w_uv, w_o, weights,
                          stream=None):
    """videomla_prepare_layer_weights; `weights` is a uint8 device tensor."""
    d = make_dims(dims)
    H = d.n_heads
    _need(w_dq, "w_dq", d_q * d.d_model)
    if gamma_q is not None:
        _need(gamma_q, "gamma_q", d_q)
    _need(w_uq, "w_uq", H * d.d_nope * d_q)
    _need(w_qr, "w_qr", H * d.d_rope * d_q)
    _need(w_uk, "w_uk", H * d.d_nope * d.d_c)
    _need(w_uv, "w_uv", H * d.d_v * d.d_c)
    _need(w_o, "w_o", d.d_model * H * d.d_v)
    _check(_lib.videomla_prepare_layer_weights(
        ctypes.byref(d), int(d_q), _ptr(w_dq, "w_dq"), _ptr(gamma_q, "gamma_q"),
        _ptr(w_uq, "w_uq"), _ptr(w_qr, "w_qr"), _ptr(w_uk, "w_uk"), _ptr(w_uv, "w_uv"),
        _ptr(w_o, "w_o"), _ptr(weights, "weights", (torch.uint8,)), weights.numel(),
        _stream(stream)))


def attend_layer_workspace_bytes(dims, d_q: int, batch: int, opts: AttendOpts | None = None) -> int:
    o = opts.struct() if opts is not None else None
    return int(_lib.videomla_attend_layer_workspace_bytes(
        ctypes.byref(make_dims(dims)), int(d_q), int(batch),
        ctypes.byref(o) if o is not None else None))


def attend_layer(dims, frame_end: int, batch: int, d_q: int, x, weights, c_kv, k_r, y, workspace,
                 stream=None, opts: AttendOpts | None = None):
    """videomla_attend_layer on torch tensors; `weights` and `workspace` are uint8 device tensors."""
    d = make_dims(dims)
    hw = d.grid_h * d.grid_w
    nq = _nq(dims, opts)
    _need(x, "x", batch * nq * d.d_model)
    _need(c_kv, "c_kv", batch * d.window_frames * hw * d.d_c)
    _need(k_r, "k_r", batch * d.window_frames * hw * d.d_rope)
    _need(y, "y", batch * nq * d.d_model)
    w = VideomlaWindow(int(frame_end))
    o = opts.struct() if opts is not None else None
    _check(_lib.videomla_attend_layer(
        ctypes.byref(d), ctypes.byref(w), int(batch), int(d_q), _ptr(x, "x"),
        _ptr(weights, "weights", (torch.uint8,)), weights.numel(), _ptr(c_kv, "c_kv"),
        _ptr(k_r, "k_r"), _ptr(y, "y"), _ptr(workspace, "workspace", (torch.uint8,)),
        workspace.numel() if workspace is not None else 0,
        ctypes.byref(o) if o is not None else None, _stream(stream)))


def window_advance(dims, frame_end: int) -> int:
    w = VideomlaWindow(int(frame_end))
    _check(_lib.videomla_window_advance(ctypes.byref(make_dims(dims)), ctypes.byref(w)))
    return int(w.frame_end)


def cache_bytes_per_token(dims) -> int:
    return int(_lib.videomla_cache_bytes_per_token(ctypes.byref(make_dims(dims))))


def valid_tokens(dims, frame_end: int) -> int:
    w = VideomlaWindow(int(frame_end))
    v = int(_lib.videomla_valid_tokens(ctypes.byref(make_dims(dims)), ctypes.byref(w)))
    if v < 0:
        raise VideomlaError(EINVAL, _lib.videomla_last_error().decode())
    return v


def slot_of(dims, f: int, y: int, x: int) -> int:
    v = int(_lib.videomla_slot_of(ctypes.byref(make_dims(dims)), int(f), int(y), int(x)))
    if v < 0:
        raise VideomlaError(EINVAL, _lib.videomla_last_error().decode())
    return v


def raw():
    """The loaded ctypes library (for tests that call the C ABI directly)."""
    return _lib


def stamps_buffer_bytes() -> int:
    """Size of the phase-stamp buffer (VIDEOMLA_STAMP_BUFFER_BYTES)."""
    return STAMP_KERNELS * STAMP_WORKGROUPS * STAMP_WAVES * STAMP_POINTS * 8


def stamps_attach(buf: torch.Tensor | None):
    """Diagnostic build only: record the phase stamps of later calls into `buf`, a device tensor
    of stamps_buffer_bytes() bytes (None detaches). The records are uint64
    [kernel][workgroup][wave][point] (include/videomla_stamps.h)."""
    if not STAMPS:
        raise VideomlaError(EUNSUPPORTED, "phase stamps need VIDEOMLA_LIBRARY=stamps at import")
    if buf is None:
        _check(_lib.videomla_stamps_attach(None, 0))
        return
    if not buf.is_cuda or not buf.is_contiguous():
        raise VideomlaError(EINVAL, "the stamp buffer must be a contiguous device tensor")
    _check(_lib.videomla_stamps_attach(ctypes.c_void_p(buf.data_ptr()),
                                       buf.numel() * buf.element_size()))
