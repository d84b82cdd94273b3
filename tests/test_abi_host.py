"""C-ABI checks that need no GPU: the library loads, exports every declared symbol, and its
host-side validation, window and slot arithmetic behave as documented. No call here reaches a
kernel launch."""
import ctypes
import os
import re

import numpy as np
import pytest

from tests._build_once import ensure_built

ensure_built()

import paper_2605_30351_amd as vm  # noqa: E402
from paper_2605_30351_amd import _lib as L  # noqa: E402
from oracle import videomla_oracle as O  # noqa: E402
from workloads import TINY, WAN, WAN_PAPER  # noqa: E402

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "videomla.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(videomla_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 11
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTED)


STAMPS_HEADER = os.path.join(os.path.dirname(HEADER), "videomla_stamps.h")


def test_stamps_build_exports_the_same_calls_plus_attach():
    """The diagnostic build exports every call of both headers; the product library does not
    export the stamps call."""
    from tests._build_once import ensure_stamps_built
    text = re.sub(r"/\*.*?\*/", "", open(STAMPS_HEADER).read(), flags=re.S)
    extra = sorted(set(re.findall(r"\b(videomla_[a-z_]+)\s*\(", text)))
    assert extra == sorted(L.EXPORTED_STAMPS)
    st = ctypes.CDLL(ensure_stamps_built())
    for n in _declared() + extra:
        assert hasattr(st, n), n
    assert not hasattr(ctypes.CDLL(L.LIB_PATH), "videomla_stamps_attach")
    size = re.search(r"#define VIDEOMLA_STAMP_KERNELS (\d+).*?#define VIDEOMLA_STAMP_WORKGROUPS (\d+)"
                     r".*?#define VIDEOMLA_STAMP_WAVES (\d+).*?#define VIDEOMLA_STAMP_POINTS (\d+)",
                     text, flags=re.S)
    dims = tuple(int(x) for x in size.groups())
    assert dims == (L.STAMP_KERNELS, L.STAMP_WORKGROUPS, L.STAMP_WAVES, L.STAMP_POINTS)
    assert L.stamps_buffer_bytes() == 8 * np.prod(dims)


def test_stamps_attach_validates_without_touching_memory():
    """Attach only stores the pointer: a too small or misaligned buffer is refused, NULL
    detaches. No kernel runs, so the (never dereferenced) addresses need no GPU."""
    from tests._build_once import ensure_stamps_built
    st = ctypes.CDLL(ensure_stamps_built())
    st.videomla_stamps_attach.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    st.videomla_stamps_attach.restype = ctypes.c_int
    st.videomla_last_error.restype = ctypes.c_char_p
    need = L.stamps_buffer_bytes()
    assert st.videomla_stamps_attach(ctypes.c_void_p(0x1000), need - 8) == L.EINVAL
    assert b"bytes" in st.videomla_last_error()
    assert st.videomla_stamps_attach(ctypes.c_void_p(0x1004), need) == L.EALIGN
    assert st.videomla_stamps_attach(None, 0) == L.OK
    assert st.videomla_last_error() == b""


def test_stamps_calls_need_the_stamps_build():
    if L.STAMPS:
        pytest.skip("this process loaded the diagnostic build")
    with pytest.raises(vm.VideomlaError):
        vm.stamps_attach(None)


def test_struct_layout_matches_header():
    # 10 int32 + 2*3 int32 + 3 float + 1 int32 = 20 * 4 bytes, no padding
    assert ctypes.sizeof(L.VideomlaDims) == 80
    assert ctypes.sizeof(L.VideomlaWindow) == 8


def test_cache_bytes_per_token():
    assert vm.cache_bytes_per_token(WAN) == 448
    assert vm.cache_bytes_per_token(WAN_PAPER) == 448
    assert vm.cache_bytes_per_token(TINY) == 48


@pytest.mark.parametrize("dims", [TINY, WAN])
def test_slot_of_matches_oracle(dims):
    rng = np.random.default_rng(0)
    for _ in range(200):
        f = int(rng.integers(0, 500))
        y = int(rng.integers(0, dims.grid_h))
        x = int(rng.integers(0, dims.grid_w))
        assert vm.slot_of(dims, f, y, x) == int(O.ring_slot(f, y, x, dims))


def test_valid_tokens_and_advance():
    fe = 0
    for step in range(10):
        lo, hi = O.window_frame_range(fe, WAN)
        assert vm.valid_tokens(WAN, fe) == (hi - lo) * WAN.hw
        fe = vm.window_advance(WAN, fe)
        assert fe == (step + 1) * WAN.chunk_frames
    assert vm.valid_tokens(TINY, 5) == 48
    assert vm.valid_tokens(TINY, 0) == 16


def _dims_struct(dims, **kw):
    d = L.make_dims(dims)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


FAKE = ctypes.c_void_p(0x1000)       # never dereferenced: validation fails first
MISALIGNED = ctypes.c_void_p(0x1008)


def _write(d, fe=0, batch=1, x=FAKE, gamma=None):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_cache_write(ctypes.byref(d), ctypes.byref(w), batch, x, FAKE, FAKE,
                                        gamma, FAKE, FAKE, None, None)


def _attend(d, fe=0, batch=1, ws=FAKE, ws_bytes=1 << 40, q=FAKE):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_attend(ctypes.byref(d), ctypes.byref(w), batch, q, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, FAKE, ws, ws_bytes, None)


@pytest.mark.parametrize("field,value,code", [
    ("d_rope", 7, L.EINVAL), ("d_model", 0, L.EINVAL), ("n_heads", -1, L.EINVAL),
    ("chunk_frames", 30, L.EINVAL), ("d_model", 1000, L.EUNSUPPORTED), ("d_c", 100, L.EUNSUPPORTED),
])
def test_cache_write_rejects_bad_dims(field, value, code):
    assert _write(_dims_struct(WAN, **{field: value})) == code
    assert L.raw().videomla_last_error().decode() != ""


def test_cache_write_rejects_bad_args():
    d = L.make_dims(WAN)
    assert _write(d, fe=-1) == L.EINVAL
    assert _write(d, batch=0) == L.EINVAL
    assert _write(d, x=None) == L.EINVAL
    assert _write(d, x=MISALIGNED) == L.EALIGN
    d.rope_pairs[0] = 7
    assert _write(d) == L.EINVAL


def _write_prepared(d, fe=0, batch=1, x=FAKE, wp=FAKE):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_cache_write_prepared(ctypes.byref(d), ctypes.byref(w), batch, x, wp,
                                                 None, FAKE, FAKE, None, None)


def test_packed_write_weights_size_and_validation():
    # one 2 KB block per (32-row wave slice, 32-column k-step): 7 x 48 x 2048 for Wan
    assert vm.write_weights_bytes(WAN) == 7 * 48 * 2048
    assert vm.write_weights_bytes(TINY) == 1 * 2 * 2048
    assert L.raw().videomla_write_weights_bytes(ctypes.byref(_dims_struct(WAN, d_model=4096))) == 0
    d = L.make_dims(WAN)
    prep = L.raw().videomla_prepare_write_weights
    assert prep(ctypes.byref(d), FAKE, FAKE, None, None) == L.EINVAL
    assert prep(ctypes.byref(d), FAKE, MISALIGNED, FAKE, None) == L.EALIGN
    assert prep(ctypes.byref(_dims_struct(WAN, d_c=100)), FAKE, FAKE, FAKE, None) == L.EUNSUPPORTED
    assert _write_prepared(d, wp=None) == L.EINVAL
    assert _write_prepared(d, wp=MISALIGNED) == L.EALIGN
    assert _write_prepared(d, x=None) == L.EINVAL
    assert _write_prepared(d, batch=0) == L.EINVAL
    assert _write_prepared(d, fe=-1) == L.EINVAL
    assert _write_prepared(_dims_struct(WAN, d_model=4096)) == L.EUNSUPPORTED
    assert _write(_dims_struct(WAN, d_model=4096)) == L.EUNSUPPORTED


def test_timer_lifecycle_and_names():
    """A timer is a caller-owned object: videomla_timer_only takes the kernel names that
    videomla_timer_read knows, or NULL; reads of a fresh timer are empty."""
    t = vm.Timer()
    t.only("latent_attend")
    t.only(None)
    assert t.read("latent_attend") == (0, 0.0)
    with pytest.raises(vm.VideomlaError):
        t.only("no_such_kernel")
    with pytest.raises(vm.VideomlaError):
        t.read("nope")
    lib = L.raw()
    # an end without its begin, an unknown name (host-side checks: no event is recorded)
    assert lib.videomla_timer_end(t.handle, b"cache_write", None) == L.EINVAL
    assert lib.videomla_timer_begin(t.handle, b"no_such_kernel", None) == L.EINVAL
    t.close()
    lib = L.raw()
    assert lib.videomla_timer_only(None, b"latent_attend") == L.EINVAL
    assert lib.videomla_timer_begin(None, b"cache_write", None) == L.EINVAL
    assert lib.videomla_timer_create(None) == L.EINVAL
    assert lib.videomla_timer_destroy(None) == L.OK


def _opts(**kw):
    o = L.VideomlaAttendOpts()
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def _attend_ex(d, opts, fe=0, batch=1, ws=FAKE, ws_bytes=1 << 40, q=FAKE):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_attend_ex(ctypes.byref(d), ctypes.byref(w), batch, q, FAKE, FAKE,
                                      FAKE, FAKE, FAKE, FAKE, ws, ws_bytes,
                                      ctypes.byref(opts) if opts is not None else None, None)


def test_attend_options_are_validated():
    d = L.make_dims(WAN)
    for bad in (dict(partition=3), dict(partition=-1), dict(form=7), dict(n_workgroups=-1),
                dict(n_workgroups=(1 << 20) + 1), dict(query_begin=-1),
                dict(query_begin=4680), dict(query_begin=4000, query_count=681),
                dict(query_count=-2)):
        assert _attend_ex(d, _opts(**bad)) == L.EINVAL, bad
        assert L.raw().videomla_attend_workspace_bytes_ex(
            ctypes.byref(d), 1, ctypes.byref(_opts(**bad))) == 0, bad
    # the last query range that fits, and NULL options (= videomla_attend)
    assert vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(query_begin=4000, query_count=680)) > 0
    assert (L.raw().videomla_attend_workspace_bytes_ex(ctypes.byref(d), 1, None)
            == vm.attend_workspace_bytes(WAN, 1))
    need = vm.attend_workspace_bytes(WAN, 1)
    assert _attend_ex(d, None, ws_bytes=need - 1) == L.EWORKSPACE
    assert _attend_ex(d, _opts(partition=2), ws_bytes=need - 1) == L.EWORKSPACE


def test_query_range_sizes_the_workspace():
    """A block of the chunk's query rows needs the workspace of that many rows."""
    full = vm.attend_workspace_bytes(WAN, 1)
    part = vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(query_begin=1560, query_count=1560))
    assert part < full
    assert part >= 1560 * 12 * 224 * 2 + 1560 * 12 * 192 * 4
    few = vm.attend_workspace_bytes(WAN, 8, vm.AttendOpts(query_count=16))
    assert 0 < few < full
    assert (vm.dense_attend_workspace_bytes(WAN, 8, vm.AttendOpts(query_count=16))
            < vm.dense_attend_workspace_bytes(WAN, 8))


def test_auto_form_follows_the_cost_model():
    """The cost model picks the materialized form where its cheaper score outweighs the
    reconstruction (a 3-frame Wan chunk), the latent form for few queries, and never the
    materialized form on shapes it is not built for."""
    mat = vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(form="materialized"))
    lat = vm.attend_workspace_bytes(WAN, 1)
    assert mat > lat
    assert vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(form="auto")) == mat
    few = vm.AttendOpts(form="auto", query_count=52)
    assert vm.attend_workspace_bytes(WAN, 1, few) == vm.attend_workspace_bytes(
        WAN, 1, vm.AttendOpts(query_count=52))
    # no materialized kernel is built for d_v = 96: AUTO falls back to the latent form
    d96 = WAN.replace(d_v=96)
    assert (vm.attend_workspace_bytes(d96, 1, vm.AttendOpts(form="auto"))
            == vm.attend_workspace_bytes(d96, 1))
    assert vm.attend_workspace_bytes(d96, 1, vm.AttendOpts(form="materialized")) == 0


def test_two_threads_with_different_options():
    """The library keeps no configuration between calls: two threads asking at the same time
    for the workspace of different options each get their own answer, and each thread reads its
    own last error."""
    import threading
    one = vm.AttendOpts(n_workgroups=1)
    want = {0: vm.attend_workspace_bytes(WAN, 1), 1: vm.attend_workspace_bytes(WAN, 1, one)}
    assert want[0] != want[1]
    bad = {0: _dims_struct(WAN, d_c=100), 1: _dims_struct(WAN, d_nope=100)}
    seen = {0: set(), 1: set()}
    errors = {0: set(), 1: set()}

    def run(k):
        for _ in range(200):
            seen[k].add(vm.attend_workspace_bytes(WAN, 1, one if k else None))
            _attend(bad[k])
            errors[k].add(L.raw().videomla_last_error().decode())
    threads = [threading.Thread(target=run, args=(k,)) for k in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert seen == {0: {want[0]}, 1: {want[1]}}
    assert len(errors[0]) == 1 and len(errors[1]) == 1 and errors[0] != errors[1], errors


def test_dc_sweep_shapes():
    """The paper's Table 5 latent widths 64, 128, 192, 256 and 512 are built (with d_rope = 32).
    d_c + d_rope = 544 exceeds the plain-weight cache write (288 outputs): only the packed-weight
    write takes it; its panel then holds 64 outputs per wave slice."""
    for dc in (64, 128, 192, 256, 512):
        assert vm.attend_workspace_bytes(WAN.replace(d_c=dc), 1) > 0
        assert vm.write_weights_bytes(WAN.replace(d_c=dc)) > 0
    assert vm.write_weights_bytes(WAN.replace(d_c=512)) == 9 * 48 * 4096   # 9 slices of 64 rows
    assert _write(_dims_struct(WAN, d_c=512)) == L.EUNSUPPORTED
    assert _write_prepared(_dims_struct(WAN, d_c=1024)) == L.EUNSUPPORTED
    assert vm.attend_workspace_bytes(WAN.replace(d_c=320), 1) == 0


def test_materialized_attend_validation():
    """The materialized form is built for d_v = 128 with keys of d_nope + d_rope = 128 (the
    paper's 96 + 32) or 160 (128 + 32), no sink."""
    mat = vm.AttendOpts(form="materialized")
    assert vm.attend_workspace_bytes(WAN_PAPER, 1, mat) > 0
    assert vm.attend_workspace_bytes(WAN, 1, mat) > 0
    assert vm.attend_workspace_bytes(WAN.replace(d_nope=112), 1, mat) == 0
    o = _opts(form=1)

    def call(d, ws=FAKE, ws_bytes=1 << 40, q=FAKE):
        return _attend_ex(d, o, ws=ws, ws_bytes=ws_bytes, q=q)
    d = L.make_dims(WAN_PAPER)
    assert call(_dims_struct(WAN, d_nope=112)) == L.EUNSUPPORTED
    assert call(_dims_struct(WAN_PAPER, sink_frames=1, window_frames=7)) == L.EUNSUPPORTED
    assert call(d, q=None) == L.EINVAL
    assert call(d, q=MISALIGNED) == L.EALIGN
    need = vm.attend_workspace_bytes(WAN_PAPER, 1, mat)
    assert call(d, ws=None) == L.EWORKSPACE
    assert call(d, ws_bytes=need - 1) == L.EWORKSPACE
    # the reconstructed rows dominate: ring x heads x (K_h | V_h) in bf16
    assert need >= 32760 * 12 * 256 * 2
    assert vm.attend_workspace_bytes(WAN, 1, mat) >= 32760 * 12 * 288 * 2
    # the partition state sits after the partial results, not over the query rows
    adaptive = vm.AttendOpts(form="materialized", partition="adaptive")
    assert vm.attend_workspace_bytes(WAN, 1, adaptive) == vm.attend_workspace_bytes(WAN, 1, mat)


def test_attend_rejects_bad_args():
    d = L.make_dims(WAN)
    assert _attend(d, q=None) == L.EINVAL
    assert _attend(d, q=MISALIGNED) == L.EALIGN
    need = vm.attend_workspace_bytes(WAN, 1)
    assert need > 0
    assert _attend(d, ws=None) == L.EWORKSPACE
    assert _attend(d, ws_bytes=need - 1) == L.EWORKSPACE
    assert _attend(_dims_struct(WAN, d_c=112)) == L.EUNSUPPORTED
    assert _attend(_dims_struct(WAN, d_v=100)) == L.EUNSUPPORTED
    assert _attend(_dims_struct(WAN, d_nope=100)) == L.EUNSUPPORTED


def test_workspace_tracks_the_work_partition():
    rows = WAN.chunk_tokens * WAN.n_heads
    one_row_block_each = rows * 224 * 2 + rows * 192 * 4 + rows * 8
    # one workgroup walks every row block whole
    single = vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(n_workgroups=1))
    assert single >= one_row_block_each
    # 220 row blocks over 256 workgroups: up to 3 parts each
    assert vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(n_workgroups=256)) > single
    # more workgroups than some windows have tiles
    assert vm.attend_workspace_bytes(WAN, 1, vm.AttendOpts(n_workgroups=5000)) > single
    assert vm.attend_workspace_bytes(WAN, 2) > 0


def test_dense_cache_bytes_per_token():
    # 2 (K and V) * 12 heads * 128 * 2 bytes = 3,072 bf16 scalars per token and layer
    assert vm.dense_cache_bytes_per_token(WAN) == 6144
    assert vm.dense_cache_bytes_per_token(WAN) == 2 * O.dense_scalars_per_token(WAN)
    # the 13.7x memory ratio of the latent cache at the Wan shape
    assert round(vm.dense_cache_bytes_per_token(WAN) / vm.cache_bytes_per_token(WAN), 2) == 13.71


def _dense_write(d, fe=0, batch=1, x=FAKE):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_dense_cache_write(ctypes.byref(d), ctypes.byref(w), batch, x, FAKE,
                                              FAKE, FAKE, None, None)


def _dense_attend(d, fe=0, batch=1, ws=FAKE, ws_bytes=1 << 40, q=FAKE, opts=None):
    w = L.VideomlaWindow(fe)
    return L.raw().videomla_dense_attend(ctypes.byref(d), ctypes.byref(w), batch, q, FAKE, FAKE,
                                         ws, ws_bytes,
                                         ctypes.byref(opts) if opts is not None else None, None)


def test_dense_calls_reject_bad_args():
    d = L.make_dims(WAN)
    assert _dense_write(d, x=None) == L.EINVAL
    assert _dense_write(d, batch=0) == L.EINVAL
    assert _dense_write(d, x=MISALIGNED) == L.EALIGN
    assert _dense_write(_dims_struct(WAN, d_model=1000)) == L.EUNSUPPORTED
    assert _dense_write(_dims_struct(WAN, d_v=130)) == L.EUNSUPPORTED   # more than 64 RoPE pairs
    assert _dense_write(_dims_struct(WAN, d_v=36)) == L.EUNSUPPORTED    # 2 * 12 * 36 % 128 != 0
    assert _dense_attend(d, q=None) == L.EINVAL
    assert _dense_attend(d, q=MISALIGNED) == L.EALIGN
    need = vm.dense_attend_workspace_bytes(WAN, 1)
    assert need > 0
    assert _dense_attend(d, ws=None) == L.EWORKSPACE
    assert _dense_attend(d, ws_bytes=need - 1) == L.EWORKSPACE
    assert _dense_attend(_dims_struct(WAN, d_v=64)) == L.EUNSUPPORTED
    assert vm.dense_attend_workspace_bytes(WAN.replace(d_v=64), 1) == 0
    assert _dense_attend(d, opts=_opts(partition=5)) == L.EINVAL


def test_dense_workspace_covers_padded_rows():
    # q_cat holds every head's rows padded to whole 256-row blocks: 4680 -> 4864 rows per head
    rows = 12 * 4864
    assert vm.dense_attend_workspace_bytes(WAN, 1) >= rows * 128 * 2 + rows * 128 * 4 + rows * 8
    assert vm.dense_attend_workspace_bytes(WAN, 4) >= 4 * (rows * 128 * 2 + rows * 128 * 4 + rows * 8)


def test_sink_slots_and_validation():
    from workloads import TINY_SINK, WAN_SINK
    rng = np.random.default_rng(1)
    for dims in (TINY_SINK, WAN_SINK):
        for _ in range(200):
            f = int(rng.integers(0, 500))
            y = int(rng.integers(0, dims.grid_h))
            x = int(rng.integers(0, dims.grid_w))
            assert vm.slot_of(dims, f, y, x) == int(O.ring_slot(f, y, x, dims))
        for fe in range(0, 30, dims.chunk_frames):
            assert vm.valid_tokens(dims, fe) == len(O.context_frames(fe, dims)) * dims.hw
    # the non-sink slots must hold a whole chunk
    assert _write(_dims_struct(WAN, window_frames=7, sink_frames=5)) == L.EINVAL
    assert _write(_dims_struct(WAN, sink_frames=-1)) == L.EINVAL
    # the workspace also holds the window's rotated keys
    plain = vm.attend_workspace_bytes(WAN_SINK.replace(sink_frames=0), 1)
    assert vm.attend_workspace_bytes(WAN_SINK, 1) >= plain + WAN_SINK.window_tokens * 32 * 2
    # the dense comparator has no sink mode
    assert _dense_write(_dims_struct(WAN, window_frames=7, sink_frames=1)) == L.EUNSUPPORTED
    assert _dense_attend(_dims_struct(WAN, window_frames=7, sink_frames=1)) == L.EUNSUPPORTED


def test_layer_calls_validate_and_size():
    d = L.make_dims(WAN)
    # W_down^Q [768][1536], query matrix [12 * 224][768], B [1536][2304], bf16, 256-aligned
    assert vm.layer_weights_bytes(WAN, 768) == 768 * 1536 * 2 + 2688 * 768 * 2 + 1536 * 2304 * 2
    assert vm.layer_weights_bytes(TINY, 48) >= 64 * 64 * 2 + 48 * 64 * 2 + 64 * 64 * 2  # padded
    assert vm.layer_weights_bytes(WAN, 0) == 0
    ws = vm.attend_layer_workspace_bytes(WAN, 768, 1)
    assert ws >= vm.attend_workspace_bytes(WAN, 1) + 4680 * 768 * 2 + 4680 * 2304 * 2
    w = L.VideomlaWindow(21)
    wb = vm.layer_weights_bytes(WAN, 768)

    def layer(d=d, d_q=768, x=FAKE, weights=FAKE, weights_bytes=wb, ws_ptr=FAKE, ws_bytes=1 << 40):
        return L.raw().videomla_attend_layer(ctypes.byref(d), ctypes.byref(w), 1, d_q, x, weights,
                                             weights_bytes, FAKE, FAKE, FAKE, ws_ptr, ws_bytes,
                                             None, None)
    assert layer(x=None) == L.EINVAL
    assert layer(d_q=0) == L.EINVAL
    assert layer(x=MISALIGNED) == L.EALIGN
    assert layer(weights_bytes=wb - 1) == L.EWORKSPACE
    assert layer(ws_ptr=None) == L.EWORKSPACE
    assert layer(ws_bytes=ws - 1) == L.EWORKSPACE
    assert layer(d=_dims_struct(WAN, d_c=112)) == L.EUNSUPPORTED
    assert layer(d=_dims_struct(WAN, d_model=1000)) == L.EUNSUPPORTED
    # the whole layer runs the latent form only
    assert vm.attend_layer_workspace_bytes(WAN, 768, 1, vm.AttendOpts(form="materialized")) == 0
    assert (vm.attend_layer_workspace_bytes(WAN, 768, 1, vm.AttendOpts(form="auto"))
            == vm.attend_layer_workspace_bytes(WAN, 768, 1))
    prep = L.raw().videomla_prepare_layer_weights
    assert prep(ctypes.byref(d), 768, FAKE, None, FAKE, FAKE, FAKE, FAKE, None, FAKE, wb, None) == L.EINVAL
    assert prep(ctypes.byref(d), 768, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, wb - 1, None) == L.EWORKSPACE
    assert prep(ctypes.byref(d), 768, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, MISALIGNED, wb, None) == L.EALIGN

def test_noalloc_rejects_before_launch():
    """videomla_attend_noalloc: invalid dims are reported as videomla_attend reports them, and a
    shape whose workspace exceeds the static scratch array (the Wan chunk: about 156 MB) is
    rejected with EWORKSPACE; both before any device work."""
    lib = L.raw()

    def call(d, batch=1):
        w = L.VideomlaWindow(21)
        return lib.videomla_attend_noalloc(ctypes.byref(d), ctypes.byref(w), batch, FAKE, FAKE,
                                           FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert vm.attend_workspace_bytes(WAN, 1) > vm.NOALLOC_SCRATCH_BYTES
    assert call(L.make_dims(WAN)) == L.EWORKSPACE
    assert "static scratch" in lib.videomla_last_error().decode()
    assert call(_dims_struct(WAN, d_rope=7)) == L.EINVAL
    assert call(_dims_struct(WAN, d_c=100)) == L.EUNSUPPORTED
    assert call(L.make_dims(TINY), batch=0) == L.EINVAL
