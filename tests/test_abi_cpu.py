"""CPU-side checks of the C-ABI library: it loads without a GPU, exports every
function include/*.h declares, reproduces the paper's state and
conv-state sizes (Appendix A), and rejects bad arguments on the host before
any launch (no device work is started by these calls)."""
import ctypes
import json
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("sr_replay.h", "sr_sidecar.h", "sr_replay_graph.h", "sr_group.h")]
GOLDEN = os.path.join(ROOT, "tests", "golden", "storage_table6.json")

sr = pytest.importorskip("paper_2609_33477_amd.binding",
                         reason="libsr_replay.so not built (run __graft_entry__.build())")
from workloads import Shape, F32, BF16, FP8  # noqa: E402


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    # declarations: "<return type> sr_name(" at the start of a line
    return sorted(set(re.findall(r"^(?:size_t|sr_status|int64_t|void\s*\*|const char\s*\*)\s*(sr_\w+)\s*\(", text, re.M)))


def test_header_declares_and_library_exports_every_function():
    names = declared_functions()
    assert set(names) == {"sr_state_bytes", "sr_conv_tail_bytes", "sr_replay_workspace_size",
                          "sr_replay_state", "sr_replay_state_noalloc", "sr_validate_varlen",
                          "sr_validate_varlen_host", "sr_kernel_timing_enable", "sr_kernel_timing_read",
                          "sr_kernel_timing_kinds", "sr_last_hip_error", "sr_status_str", "sr_anchor_dest_table", "sr_anchor_compact",
                          "sr_anchor_write", "sr_anchor_gather", "sr_replay_graph_create", "sr_replay_graph_anchors",
                          "sr_replay_graph_max_rows", "sr_replay_graph_fetch", "sr_replay_graph_run",
                          "sr_replay_graph_wait", "sr_replay_graph_destroy", "sr_group_workspace_size",
                          "sr_replay_group"}
    lib = ctypes.CDLL(sr.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(sr.EXPORTED_SYMBOLS)


def test_last_hip_error_is_clear_without_a_failed_launch():
    code, kind, msg = sr.last_hip_error()
    assert code == 0 and kind is None and isinstance(msg, str)


def test_size_helpers_match_paper_table():
    tab = json.load(open(GOLDEN))
    for name, m in tab["models"].items():
        shape = Shape(m["d"], m["H_k"], m["H_v"], m["d_k"], m["d_v"], conv_width=tab["conv_width"])
        assert sr.state_bytes(shape) == m["B_rec"], name
        assert sr.conv_tail_bytes(shape, with_q=True) == m["B_conv"], name


def test_status_strings():
    for code in range(7):
        assert isinstance(sr.status_str(code), str) and sr.status_str(code)
    assert sr.status_str(99) == "unknown status"


def test_workspace_size_plan():
    shape = Shape(2560, 16, 32, 128, 128)
    t = 36672
    ws = sr.replay_workspace_size(shape, 1, t)
    # bf16 path: per-row segment info (16 B) + bf16 k|v + fp32 log-alpha/beta,
    # each region 256-byte aligned; the projection itself never reaches HBM
    expect = t * 16 + t * (16 + 32) * 128 * 2 + 2 * t * 32 * 4
    assert expect <= ws <= expect + 5 * 256
    assert sr.replay_workspace_size(shape, 12, t) > 11 * (ws - t * 16)
    # fp32 path keeps the fp32 projection rows in the workspace
    f32 = Shape(256, 2, 2, 32, 32, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    n = (2 + 2) * 32 + 4
    expect32 = 1000 * n * 4 + 1000 * 4 * 32 * 4 + 2 * 1000 * 2 * 4
    assert expect32 <= sr.replay_workspace_size(f32, 1, 1000) <= expect32 + 5 * 256


@pytest.mark.parametrize("bad,code", [
    (dict(d_model=100), 2), (dict(d_model=0), 2), (dict(n_k_heads=0), 2), (dict(n_v_heads=24, n_k_heads=16), 2),
    (dict(d_k=96, d_v=96), 2), (dict(d_k=128, d_v=64), 2), (dict(conv_width=5), 2), (dict(l2_eps=0.0), 2),
    (dict(anchor_dtype=F32, weight_dtype=BF16), 3), (dict(anchor_dtype=FP8), 3), (dict(tail_dtype=FP8), 3),
])
def test_workspace_size_rejects_bad_shapes(bad, code):
    kw = dict(d_model=256, n_k_heads=2, n_v_heads=4, d_k=128, d_v=128)
    kw.update({k: v for k, v in bad.items() if k in kw})
    shape = Shape(**kw)
    for k, v in bad.items():
        setattr(shape, k, v)
    with pytest.raises(sr.SrError) as e:
        sr.replay_workspace_size(shape, 1, 128)
    assert e.value.status == code


def _fake_layer(**over):
    # distinct 256-aligned fake addresses; validation never dereferences them
    base = dict(anchors=0x10000, w_k=0x20000, w_v=0x30000, w_a=0x40000, w_b=0x50000, conv_w=0x60000,
                a_log=0x70000, dt_bias=0x80000, state_out=0x90000)
    base.update(over)
    return sr.LayerTensors(**base)


def _call(layers, shape=None, n_seg=1, t=64, cu=0xA0000, ws=0xB0000, ws_bytes=None, n_layers=None, n_slots=4):
    shape = shape or Shape(256, 2, 4, 128, 128)
    if ws_bytes is None:
        ws_bytes = sr.replay_workspace_size(shape, len(layers), t)
    sh = sr.make_shape(shape)
    arr = sr.make_layer_array(layers)
    return sr.LIB.sr_replay_state(ctypes.byref(sh), len(layers) if n_layers is None else n_layers, arr,
                                  n_seg, t, cu, None, n_slots, None, ws, ws_bytes, None)


def test_replay_state_host_validation():
    assert _call([_fake_layer(w_v=None)]) == 1
    assert _call([_fake_layer(state_out=None)]) == 1
    assert _call([_fake_layer()], cu=None) == 1
    assert _call([_fake_layer(anchors=0x10004)]) == 5
    assert _call([_fake_layer()], ws=0xB0010) == 5
    assert _call([_fake_layer()], ws_bytes=1024) == 4
    assert _call([_fake_layer()], n_seg=-1) == 2
    assert _call([_fake_layer()], n_seg=0, t=64) == 2
    assert _call([_fake_layer()], t=-5, ws_bytes=1 << 30) == 2
    assert _call([_fake_layer()], n_layers=0) == 2
    fp8 = Shape(256, 2, 4, 128, 128, weight_dtype=FP8)
    assert _call([_fake_layer()], shape=fp8) == 1            # fp8 needs scales
    assert _call([_fake_layer(s_k=1 << 20, s_v=1 << 21, s_a=1 << 22, s_b=1 << 23, w_q=1 << 24)], shape=fp8) == 1
    assert sr.LIB.sr_replay_state(None, 1, None, 0, 0, None, None, 0, None, None, 0, None) == 1
    assert _call([_fake_layer()], n_slots=-1) == 2
    assert _call([_fake_layer()], n_slots=(1 << 19) + 1) == 2
    assert _call([_fake_layer()], ws=None) == 1               # a call with segments needs a workspace


def test_replay_state_empty_batch_is_noop():
    # zero segments and zero rows: valid, nothing to launch
    assert _call([_fake_layer(anchors=None)], n_seg=0, t=0, cu=None, ws=None, ws_bytes=0) == 0


def test_kernel_timing_read_without_launches():
    sr.kernel_timing_enable(True)
    out = sr.kernel_timing_read()
    sr.kernel_timing_enable(False)
    assert set(out) == set(sr.KERNEL_KINDS)
    assert all(v == (0.0, 0) for v in out.values())


def test_replay_graph_rejects_bad_arguments_before_allocating():
    import workloads as W
    sh = sr.make_shape(W.Shape(256, 2, 4, 128, 128))
    lay = (sr.SrLayer * 1)()
    h = ctypes.c_void_p()
    rows = (ctypes.c_int64 * 3)(256, 128, 1024)            # not ascending
    assert sr.LIB.sr_replay_graph_create(ctypes.byref(sh), 1, lay, 4, None, 8, rows, 3, None, 0, ctypes.byref(h)) == 2
    rows = (ctypes.c_int64 * 1)(256)
    assert sr.LIB.sr_replay_graph_create(ctypes.byref(sh), 1, lay, 4, None, 0, rows, 1, None, 0, ctypes.byref(h)) == 2
    assert sr.LIB.sr_replay_graph_create(ctypes.byref(sh), 1, lay, -1, None, 8, rows, 1, None, 0, ctypes.byref(h)) == 2
    assert sr.LIB.sr_replay_graph_create(None, 1, lay, 4, None, 8, rows, 1, None, 0, ctypes.byref(h)) == 1
    # a lent workspace below the largest bucket's need, or misaligned
    need = sr.replay_workspace_size(W.Shape(256, 2, 4, 128, 128), 1, 256)
    assert sr.LIB.sr_replay_graph_create(ctypes.byref(sh), 1, lay, 4, None, 8, rows, 1, 4096, need - 1,
                                         ctypes.byref(h)) == 4
    assert sr.LIB.sr_replay_graph_create(ctypes.byref(sh), 1, lay, 4, None, 8, rows, 1, 4096 + 16, need,
                                         ctypes.byref(h)) == 5
    assert sr.LIB.sr_replay_graph_run(None, 1, 10, None, None, None, None, 0, None, None) == 1
    assert sr.LIB.sr_replay_graph_fetch(None, None, 0, None) == 1
    assert sr.LIB.sr_replay_graph_wait(None, None) == 1
    assert sr.LIB.sr_replay_graph_destroy(None) == 0
    assert sr.LIB.sr_replay_graph_anchors(None, 0) is None and sr.LIB.sr_replay_graph_max_rows(None) == 0


def test_noalloc_refuses_oversized_batches_on_the_host():
    """sr_replay_state_noalloc checks its workspace need against the scratch
    before touching the device (this runs without a GPU)."""
    shape = Shape(2560, 16, 32, 128, 128)
    t_big = 16384
    assert sr.replay_workspace_size(shape, 1, t_big) > sr.NOALLOC_SCRATCH_BYTES
    lay = sr.SrLayer()
    arr = (sr.SrLayer * 1)(lay)
    st = sr.LIB.sr_replay_state_noalloc(ctypes.byref(sr.make_shape(shape)), 1, arr, 1, t_big, None, None, 1, None,
                                        None)
    assert st == 4      # SR_ERR_WORKSPACE_TOO_SMALL
    st = sr.LIB.sr_replay_state_noalloc(None, 1, arr, 1, 8, None, None, 1, None, None)
    assert st == 1      # SR_ERR_NULL_ARG


# ------------------------------------------------------- varlen table check
# (Section 5.2, fail-closed: a bad table must become a miss, not a write
# outside a buffer).  The per-segment predicate is the one the device kernel
# runs; here it runs on the host through sr_validate_varlen_host.
VARLEN_CASES = [
    # (name, cu_seqlens, slot_ids, t_total, n_slots, expected mask)
    ("good", [0, 3, 3, 10], [2, -1, 0], 10, 3, 0),
    ("good_identity", [0, 5, 9], None, 9, 2, 0),
    ("good_all_sentinel", [0, 4, 8], [-1, -7], 8, 0, 0),
    ("bad_start", [1, 3, 10], [0, 1], 10, 2, 1),
    ("not_monotone", [0, 6, 4, 10], [0, 1, 2], 10, 3, 2),
    ("total_short", [0, 3, 9], [0, 1], 10, 2, 4),
    ("total_past_end", [0, 3, 12], [0, 1], 10, 2, 4),        # cu[B] > t_total: rows past the buffers
    ("slot_range", [0, 3, 10], [0, 2], 10, 2, 8),
    ("identity_range", [0, 3, 6, 10], None, 10, 2, 8),       # NULL slot ids: segment b writes slot b
    ("slot_duplicate", [0, 3, 6, 10], [1, 0, 1], 10, 2, 16),
    ("duplicate_ignores_sentinels", [0, 3, 6, 10], [-1, 0, -1], 10, 1, 0),
    ("several", [2, 1, 7], [5, 5], 9, 3, 1 | 2 | 4 | 8),
]


@pytest.mark.parametrize("name,cu,slots,t,n_slots,want", VARLEN_CASES, ids=[c[0] for c in VARLEN_CASES])
def test_varlen_check_on_the_host(name, cu, slots, t, n_slots, want):
    assert sr.validate_varlen_host(cu, slots, t, n_slots) == want


def test_varlen_check_many_slots_and_argument_errors():
    import numpy as np
    n = 5000
    cu = np.arange(n + 1, dtype=np.int32) * 2
    slots = np.random.default_rng(0).permutation(n).astype(np.int32)
    assert sr.validate_varlen_host(cu, slots, 2 * n, n) == 0
    slots[4321] = slots[17]
    assert sr.validate_varlen_host(cu, slots, 2 * n, n) == 16
    with pytest.raises(sr.SrError):
        sr.validate_varlen_host([0], None, 0, 1)                  # no segment
    with pytest.raises(sr.SrError):
        sr.validate_varlen_host([0, 1], None, 1, (1 << 19) + 1)   # more slots than the bitmap holds


def test_group_replay_host_checks():
    """sr_replay_group refuses unsupported shapes and bad arguments on the
    host (no device work)."""
    import numpy as np
    g = Shape(2560, 16, 32, 128, 128)
    ws = sr.group_workspace_size(g, 9728, 4096)
    assert ws > 0
    with pytest.raises(sr.SrError) as e:
        sr.group_workspace_size(Shape(2560, 16, 32, 128, 128, weight_dtype=FP8), 9728, 16)
    assert e.value.status == 3
    with pytest.raises(sr.SrError) as e:
        sr.group_workspace_size(Shape(2560, 16, 32, 32, 32), 9728, 16)          # d = 32
    assert e.value.status == 2
    with pytest.raises(sr.SrError) as e:
        sr.group_workspace_size(Shape(2560 + 64, 16, 32, 128, 128), 9728, 16)   # D % 256
    assert e.value.status == 2
    with pytest.raises(sr.SrError) as e:
        sr.group_workspace_size(g, 9728 + 64, 16)                               # d_ff % 128
    assert e.value.status == 2
    fake = dict((n, 0x100000 * (i + 1)) for i, n in enumerate(sr._BLOCK_FIELDS))
    blk = sr.BlockTensors(**fake)
    args = dict(anchors=0x900000, n_segments=1, t_total=64, cu_seqlens=0xA00000, workspace=None,
                workspace_bytes=0, n_slots=1, stream=0)
    with pytest.raises(sr.SrError) as e:                                        # no workspace
        sr.replay_group(g, 9728, 1e-6, [blk], **args)
    assert e.value.status == 4
    with pytest.raises(sr.SrError) as e:
        sr.replay_group(g, 9728, 1e-6, [sr.BlockTensors(**{**fake, "w_o": None})], **args)
    assert e.value.status == 1
    with pytest.raises(sr.SrError) as e:
        sr.replay_group(g, 9728, 0.0, [blk], **args)                            # eps
    assert e.value.status == 2
    with pytest.raises(sr.SrError) as e:
        sr.replay_group(g, 9728, 1e-6, [blk], **{**args, "anchors": 0x900008})
    assert e.value.status == 5


def test_rect_heads_host_checks():
    """OLMo-Hybrid's 96 x 192 heads are accepted for bf16 anchors with the
    Gated DeltaNet recurrence; other rectangles and the other paths refuse."""
    rect = Shape(3840, 30, 30, 96, 192)
    T = 1000
    ws = sr.replay_workspace_size(rect, 1, T)
    # an even number of value heads takes the fused projection: row info,
    # bf16 keys padded to 128 columns, bf16 values, fp32 gates
    assert ws >= T * 16 + T * 30 * (128 + 192) * 2 + 2 * T * 30 * 4
    # an odd number takes the unfused path: fp32 projection rows, bf16 k | v
    odd = Shape(256, 1, 3, 96, 192)
    n = 96 + 3 * 192 + 6
    assert sr.replay_workspace_size(odd, 1, T) >= T * n * 4 + T * (96 + 3 * 192) * 2 + 2 * T * 3 * 4
    for bad in (Shape(256, 2, 2, 96, 96), Shape(256, 2, 2, 64, 192), Shape(256, 2, 2, 192, 96),
                Shape(256, 2, 2, 96, 128)):
        with pytest.raises(sr.SrError) as e:
            sr.replay_workspace_size(bad, 1, T)
        assert e.value.status == 2, bad
    f32 = Shape(256, 2, 2, 96, 192, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    decay = Shape(256, 2, 2, 96, 192, recurrence="decay")
    for bad in (f32, decay):
        with pytest.raises(sr.SrError) as e:
            sr.replay_workspace_size(bad, 1, T)
        assert e.value.status == 3, bad
