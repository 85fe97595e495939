"""ctypes binding of libsr_replay.so (argument marshalling only).

Names mirror the C ABI in include/sr_replay.h: ``state_bytes``,
``conv_tail_bytes``, ``replay_workspace_size``, ``replay_state``.  Tensors are
PyTorch tensors on the current HIP device; only their ``data_ptr()`` values
cross the boundary, and every step of the replay runs in the library's
kernels.  If the library has not been built the import fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsr_replay.so")

SR_F32, SR_BF16, SR_FP8_E4M3 = 0, 1, 2
_DTYPE_CODES = {"f32": SR_F32, "bf16": SR_BF16, "fp8_e4m3": SR_FP8_E4M3,
                SR_F32: SR_F32, SR_BF16: SR_BF16, SR_FP8_E4M3: SR_FP8_E4M3}

STATUS_NAMES = {0: "SR_OK", 1: "SR_ERR_NULL_ARG", 2: "SR_ERR_BAD_SHAPE", 3: "SR_ERR_UNSUPPORTED_DTYPE",
                4: "SR_ERR_WORKSPACE_TOO_SMALL", 5: "SR_ERR_MISALIGNED", 6: "SR_ERR_HIP"}


class SrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class SrShape(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_k_heads", ctypes.c_int32), ("n_v_heads", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("conv_width", ctypes.c_int32),
                ("l2_eps", ctypes.c_float), ("anchor_dtype", ctypes.c_int32), ("weight_dtype", ctypes.c_int32),
                ("conv_dtype", ctypes.c_int32), ("tail_dtype", ctypes.c_int32), ("recurrence", ctypes.c_int32)]


_LAYER_FIELDS = ("anchors", "w_k", "w_v", "w_a", "w_b", "w_q", "s_k", "s_v", "s_a", "s_b", "s_q",
                 "conv_w", "a_log", "dt_bias", "state_in", "state_out", "tail_out")


class SrLayer(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in _LAYER_FIELDS]


def _hip_runtimes_mapped() -> set:
    """Paths of every libamdhip64 mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            return {line.split()[-1] for line in f if "libamdhip64" in line}
    except OSError:  # pragma: no cover
        return set()


class SrHostRange(ctypes.Structure):
    """sr_host_range: `rows` anchor rows at host `src` -> layer `layer`, row `dst_row`."""
    _fields_ = [("src", ctypes.c_void_p), ("layer", ctypes.c_int32), ("dst_row", ctypes.c_int64),
                ("rows", ctypes.c_int64)]


_BLOCK_FIELDS = ("w_q", "w_k", "w_v", "w_z", "w_a", "w_b", "conv_w", "a_log", "dt_bias", "norm_o", "w_o", "ln_in",
                 "ln_post", "w_gate", "w_up", "w_down", "state_out", "tail_out")


class SrBlock(ctypes.Structure):
    """sr_block: one replayed block's device tensors (include/sr_group.h)."""
    _fields_ = [(name, ctypes.c_void_p) for name in _BLOCK_FIELDS]


class SrSidecar(ctypes.Structure):
    """sr_sidecar: the anchor block pool [n_blocks][n_layers][per_page][d]."""
    _fields_ = [("pool", ctypes.c_void_p), ("n_blocks", ctypes.c_int64), ("n_layers", ctypes.c_int32),
                ("per_page", ctypes.c_int32), ("d", ctypes.c_int32), ("elem_bytes", ctypes.c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_33477_amd.build` "
                          "(or __graft_entry__.build())")
    # The library's kernels run on memory and streams that torch owns, so it
    # must use torch's HIP runtime.  torch ships its own libamdhip64 with the
    # same SONAME; loading torch first lets the dynamic linker resolve the
    # library's dependency to that copy.  Loaded the other way round, the
    # process holds two HIP runtimes, and the second one may find no device.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes are mapped into this process ({sorted(runtimes)}); "
                          "libsr_replay.so must share torch's")
    P = ctypes.POINTER
    lib.sr_state_bytes.argtypes = [P(SrShape)]
    lib.sr_state_bytes.restype = ctypes.c_size_t
    lib.sr_conv_tail_bytes.argtypes = [P(SrShape), ctypes.c_int32]
    lib.sr_conv_tail_bytes.restype = ctypes.c_size_t
    lib.sr_replay_workspace_size.argtypes = [P(SrShape), ctypes.c_int32, ctypes.c_int64, P(ctypes.c_size_t)]
    lib.sr_replay_workspace_size.restype = ctypes.c_int
    lib.sr_replay_state.argtypes = [P(SrShape), ctypes.c_int32, P(SrLayer), ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.sr_replay_state.restype = ctypes.c_int
    lib.sr_replay_state_noalloc.argtypes = [P(SrShape), ctypes.c_int32, P(SrLayer), ctypes.c_int32,
                                            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_void_p]
    lib.sr_validate_varlen.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.sr_validate_varlen.restype = ctypes.c_int
    lib.sr_validate_varlen_host.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                            ctypes.c_int32, P(ctypes.c_int32)]
    lib.sr_validate_varlen_host.restype = ctypes.c_int
    lib.sr_replay_state_noalloc.restype = ctypes.c_int
    lib.sr_group_workspace_size.argtypes = [P(SrShape), ctypes.c_int32, ctypes.c_int64, P(ctypes.c_size_t)]
    lib.sr_group_workspace_size.restype = ctypes.c_int
    lib.sr_replay_group.argtypes = [P(SrShape), ctypes.c_int32, ctypes.c_float, ctypes.c_int32, P(SrBlock),
                                    ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_size_t, ctypes.c_void_p]
    lib.sr_replay_group.restype = ctypes.c_int
    lib.sr_kernel_timing_enable.argtypes = [ctypes.c_int32]
    lib.sr_kernel_timing_enable.restype = ctypes.c_int
    lib.sr_kernel_timing_read.argtypes = [P(ctypes.c_double), P(ctypes.c_int64)]
    lib.sr_kernel_timing_read.restype = ctypes.c_int
    lib.sr_kernel_timing_kinds.argtypes = [ctypes.c_uint32]
    lib.sr_kernel_timing_kinds.restype = ctypes.c_int
    lib.sr_last_hip_error.argtypes = [P(ctypes.c_int32), P(ctypes.c_int32), P(ctypes.c_char_p)]
    lib.sr_last_hip_error.restype = ctypes.c_int
    lib.sr_status_str.argtypes = [ctypes.c_int]
    lib.sr_status_str.restype = ctypes.c_char_p
    I32P = ctypes.c_void_p
    lib.sr_anchor_dest_table.argtypes = [I32P, I32P, ctypes.c_int32, I32P, I32P, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_int32, I32P]
    lib.sr_anchor_dest_table.restype = ctypes.c_int
    lib.sr_anchor_compact.argtypes = [I32P, ctypes.c_int32, I32P, I32P, ctypes.c_void_p]
    lib.sr_anchor_compact.restype = ctypes.c_int
    lib.sr_anchor_write.argtypes = [P(SrSidecar), P(ctypes.c_void_p), ctypes.c_int32, I32P, I32P, I32P,
                                    ctypes.c_void_p]
    lib.sr_anchor_write.restype = ctypes.c_int
    lib.sr_anchor_gather.argtypes = [P(SrSidecar), ctypes.c_int32, I32P, I32P, I32P, I32P,
                                     P(ctypes.c_int32), ctypes.c_int32, P(ctypes.c_void_p), ctypes.c_int64,
                                     I32P, ctypes.c_void_p]
    lib.sr_anchor_gather.restype = ctypes.c_int
    lib.sr_replay_graph_create.argtypes = [P(SrShape), ctypes.c_int32, P(SrLayer), ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_int32, P(ctypes.c_int64), ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_size_t, P(ctypes.c_void_p)]
    lib.sr_replay_graph_create.restype = ctypes.c_int
    lib.sr_replay_graph_anchors.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.sr_replay_graph_anchors.restype = ctypes.c_void_p
    lib.sr_replay_graph_max_rows.argtypes = [ctypes.c_void_p]
    lib.sr_replay_graph_max_rows.restype = ctypes.c_int64
    lib.sr_replay_graph_fetch.argtypes = [ctypes.c_void_p, P(SrHostRange), ctypes.c_int32, ctypes.c_void_p]
    lib.sr_replay_graph_fetch.restype = ctypes.c_int
    lib.sr_replay_graph_run.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_void_p, P(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_size_t,
                                        ctypes.c_void_p, P(ctypes.c_int32)]
    lib.sr_replay_graph_run.restype = ctypes.c_int
    lib.sr_replay_graph_wait.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.sr_replay_graph_wait.restype = ctypes.c_int
    lib.sr_replay_graph_destroy.argtypes = [ctypes.c_void_p]
    lib.sr_replay_graph_destroy.restype = ctypes.c_int
    return lib


LIB = _load()

EXPORTED_SYMBOLS = ("sr_state_bytes", "sr_conv_tail_bytes", "sr_replay_workspace_size",
                    "sr_replay_state", "sr_replay_state_noalloc", "sr_validate_varlen",
                    "sr_validate_varlen_host", "sr_kernel_timing_enable", "sr_kernel_timing_read", "sr_kernel_timing_kinds",
                    "sr_last_hip_error",
                    "sr_status_str", "sr_anchor_dest_table", "sr_anchor_compact", "sr_anchor_write",
                    "sr_anchor_gather", "sr_replay_graph_create", "sr_replay_graph_anchors",
                    "sr_replay_graph_max_rows", "sr_replay_graph_fetch", "sr_replay_graph_run",
                    "sr_replay_graph_wait", "sr_replay_graph_destroy", "sr_group_workspace_size",
                    "sr_replay_group")

KERNEL_KINDS = ("proj_gemm", "conv_gate", "tail", "gdn_scan", "proj_conv", "row_info", "anchor_compact",
                "anchor_write", "anchor_seqlens", "anchor_gather", "decay_state", "graph", "validate", "rmsnorm",
                "gdn_output", "gemm_resid", "gemm_swiglu")


_RECURRENCE_CODES = {"gdn": 0, "decay": 1, 0: 0, 1: 1}


def make_shape(shape) -> SrShape:
    """SrShape from any object with the sr_shape field names (dtype fields may
    be the strings 'f32' / 'bf16' / 'fp8_e4m3' or the integer codes)."""
    return SrShape(int(shape.d_model), int(shape.n_k_heads), int(shape.n_v_heads), int(shape.d_k),
                   int(shape.d_v), int(shape.conv_width), float(shape.l2_eps),
                   _DTYPE_CODES[shape.anchor_dtype], _DTYPE_CODES[shape.weight_dtype],
                   _DTYPE_CODES[shape.conv_dtype], _DTYPE_CODES[shape.tail_dtype],
                   _RECURRENCE_CODES[getattr(shape, "recurrence", "gdn")])


def status_str(status: int) -> str:
    return LIB.sr_status_str(int(status)).decode()


def last_hip_error():
    """(hip error code, kernel kind name or None, HIP's message) of this
    thread's most recent failed launch inside replay_state()."""
    code, kind, msg = ctypes.c_int32(0), ctypes.c_int32(-1), ctypes.c_char_p()
    LIB.sr_last_hip_error(ctypes.byref(code), ctypes.byref(kind), ctypes.byref(msg))
    name = KERNEL_KINDS[kind.value] if 0 <= kind.value < len(KERNEL_KINDS) else None
    return int(code.value), name, (msg.value or b"").decode()


def _check(status: int):
    if status != 0:
        detail = status_str(status)
        if status == 6:                          # SR_ERR_HIP
            code, kind, msg = last_hip_error()
            detail += f" (kernel {kind}: hipError {code}, {msg})"
        raise SrError(status, detail)


def state_bytes(shape) -> int:
    return int(LIB.sr_state_bytes(ctypes.byref(make_shape(shape))))


def conv_tail_bytes(shape, with_q: bool = True) -> int:
    return int(LIB.sr_conv_tail_bytes(ctypes.byref(make_shape(shape)), int(bool(with_q))))


def replay_workspace_size(shape, n_layers: int, t_total: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.sr_replay_workspace_size(ctypes.byref(make_shape(shape)), int(n_layers), int(t_total),
                                        ctypes.byref(out)))
    return int(out.value)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


@dataclass
class LayerTensors:
    """Device tensors of one layer; field names and layouts as sr_layer."""
    anchors: object
    w_k: object
    w_v: object
    w_a: object
    w_b: object
    conv_w: object
    a_log: object
    dt_bias: object
    state_out: object
    w_q: object = None
    s_k: object = None
    s_v: object = None
    s_a: object = None
    s_b: object = None
    s_q: object = None
    state_in: object = None
    tail_out: object = None


def make_layer_array(layers: Sequence[LayerTensors]):
    arr = (SrLayer * len(layers))()
    for i, L in enumerate(layers):
        for name in _LAYER_FIELDS:
            setattr(arr[i], name, _ptr(getattr(L, name)))
    return arr


def kernel_timing_enable(enable: bool = True):
    _check(LIB.sr_kernel_timing_enable(int(bool(enable))))


def kernel_timing_kinds(kinds=None):
    """Record only these kernel kinds (names of KERNEL_KINDS) while timing is
    enabled; None: every kind."""
    mask = 0xFFFFFFFF if kinds is None else sum(1 << KERNEL_KINDS.index(k) for k in kinds)
    _check(LIB.sr_kernel_timing_kinds(mask))


def kernel_timing_read():
    """{kind: (total_ms, launches)} of the launches recorded since the last
    read (waits for their events)."""
    ms = (ctypes.c_double * len(KERNEL_KINDS))()
    n = (ctypes.c_int64 * len(KERNEL_KINDS))()
    _check(LIB.sr_kernel_timing_read(ms, n))
    return {k: (ms[i], int(n[i])) for i, k in enumerate(KERNEL_KINDS)}


def _n_slots(layers, n_slots):
    """The slot count sr_replay_state checks slot ids against: given, or the
    leading dimension of the first layer's state_out."""
    return int(layers[0].state_out.shape[0]) if n_slots is None else int(n_slots)


def replay_state(shape, layers: Sequence[LayerTensors], n_segments: int, t_total: int, cu_seqlens,
                 slot_ids=None, workspace=None, workspace_bytes: Optional[int] = None, stream=None,
                 n_slots: Optional[int] = None, varlen_status=None):
    """Enqueue sr_replay_state on `stream` (a torch.cuda.Stream, a raw
    hipStream_t int, or None for torch's current stream).  ``n_slots``
    defaults to state_out's leading dimension; ``varlen_status`` is an
    optional device int32 tensor receiving the table check.  Raises SrError
    on a non-OK status."""
    import torch  # plumbing: device memory and streams

    if stream is None:
        stream_ptr = torch.cuda.current_stream().cuda_stream
    elif isinstance(stream, int):
        stream_ptr = stream
    else:
        stream_ptr = stream.cuda_stream
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    sh = make_shape(shape)
    arr = make_layer_array(layers)
    status = LIB.sr_replay_state(ctypes.byref(sh), len(layers), arr, int(n_segments), int(t_total),
                                 _ptr(cu_seqlens), _ptr(slot_ids), _n_slots(layers, n_slots), _ptr(varlen_status),
                                 _ptr(workspace), int(workspace_bytes), stream_ptr)
    _check(status)


# ---------------------------------------------------- group replay chaining
@dataclass
class BlockTensors:
    """Device tensors of one replayed block; field names and layouts as sr_block."""
    w_q: object
    w_k: object
    w_v: object
    w_z: object
    w_a: object
    w_b: object
    conv_w: object
    a_log: object
    dt_bias: object
    norm_o: object
    w_o: object
    ln_in: object
    ln_post: object
    w_gate: object
    w_up: object
    w_down: object
    state_out: object
    tail_out: object = None


def group_workspace_size(shape, d_ff: int, t_total: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.sr_group_workspace_size(ctypes.byref(make_shape(shape)), int(d_ff), int(t_total), ctypes.byref(out)))
    return int(out.value)


def replay_group(shape, d_ff: int, norm_eps: float, blocks: Sequence[BlockTensors], anchors, n_segments: int,
                 t_total: int, cu_seqlens, slot_ids=None, workspace=None, workspace_bytes: Optional[int] = None,
                 stream=None, n_slots: Optional[int] = None, varlen_status=None):
    """sr_replay_group: every layer of one group rebuilt from its group-entry
    anchors.  ``n_slots`` defaults to the first block's state_out leading
    dimension.  Raises SrError on a non-OK status."""
    arr = (SrBlock * len(blocks))()
    for i, b in enumerate(blocks):
        for name in _BLOCK_FIELDS:
            setattr(arr[i], name, _ptr(getattr(b, name)))
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(LIB.sr_replay_group(ctypes.byref(make_shape(shape)), int(d_ff), float(norm_eps), len(blocks), arr,
                               _ptr(anchors), int(n_segments), int(t_total), _ptr(cu_seqlens), _ptr(slot_ids),
                               _n_slots(blocks, n_slots), _ptr(varlen_status), _ptr(workspace),
                               int(workspace_bytes), _stream_ptr(stream)))


NOALLOC_SCRATCH_BYTES = 128 << 20      # SR_NOALLOC_SCRATCH_BYTES


def replay_state_noalloc(shape, layers: Sequence[LayerTensors], n_segments: int, t_total: int, cu_seqlens,
                         slot_ids=None, stream=None, n_slots: Optional[int] = None, varlen_status=None):
    """sr_replay_state_noalloc: replay_state() on the library's own device
    scratch (no workspace argument).  Raises SrError on a non-OK status
    (SR_ERR_WORKSPACE_TOO_SMALL when the call needs more than
    NOALLOC_SCRATCH_BYTES)."""
    sh = make_shape(shape)
    arr = make_layer_array(layers)
    _check(LIB.sr_replay_state_noalloc(ctypes.byref(sh), len(layers), arr, int(n_segments), int(t_total),
                                       _ptr(cu_seqlens), _ptr(slot_ids), _n_slots(layers, n_slots),
                                       _ptr(varlen_status), _stream_ptr(stream)))


def validate_varlen(cu_seqlens, slot_ids, n_segments: int, t_total: int, n_slots: int, status, stream=None):
    """sr_validate_varlen: the device check of the tables; writes 0 or a mask
    of sr_varlen_error bits into the device int32 tensor ``status``."""
    _check(LIB.sr_validate_varlen(_ptr(cu_seqlens), _ptr(slot_ids), int(n_segments), int(t_total), int(n_slots),
                                  _ptr(status), _stream_ptr(stream)))


def validate_varlen_host(cu_seqlens, slot_ids, t_total: int, n_slots: int) -> int:
    """sr_validate_varlen_host on host int32 arrays; returns the mask."""
    import numpy as np

    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    sl = None if slot_ids is None else np.ascontiguousarray(slot_ids, dtype=np.int32)
    out = ctypes.c_int32(-1)
    _check(LIB.sr_validate_varlen_host(cu.ctypes.data, None if sl is None else sl.ctypes.data, len(cu) - 1,
                                       int(t_total), int(n_slots), ctypes.byref(out)))
    return int(out.value)


VARLEN_BAD_START, VARLEN_NOT_MONOTONE, VARLEN_BAD_TOTAL, VARLEN_SLOT_RANGE, VARLEN_SLOT_DUPLICATE = 1, 2, 4, 8, 16


# ------------------------------------------------------------ anchor sidecar
def _stream_ptr(stream):
    import torch  # plumbing: device memory and streams

    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_sidecar(pool, n_layers: int, per_page: int, d: int) -> SrSidecar:
    """sr_sidecar over a device tensor holding [n_blocks][n_layers][per_page][d]."""
    eb = pool.element_size()
    n_blocks = pool.numel() // (n_layers * per_page * d)
    return SrSidecar(pool.data_ptr(), n_blocks, n_layers, per_page, d, eb)


def anchor_dest_table(positions, token_req, page_table, page_cu, page_size: int, per_page: int):
    """sr_anchor_dest_table on host int32 numpy arrays; returns dest (int32)."""
    import numpy as np

    pos = np.ascontiguousarray(positions, dtype=np.int32)
    req = np.ascontiguousarray(token_req, dtype=np.int32)
    tab = np.ascontiguousarray(page_table, dtype=np.int32)
    cu = np.ascontiguousarray(page_cu, dtype=np.int32)
    dest = np.empty(len(pos), dtype=np.int32)
    _check(LIB.sr_anchor_dest_table(pos.ctypes.data, req.ctypes.data, len(pos), tab.ctypes.data if tab.size else None,
                                    cu.ctypes.data, len(cu) - 1, int(page_size), int(per_page), dest.ctypes.data))
    return dest


def anchor_compact(dest, sel, n_sel, stream=None):
    """sr_anchor_compact: device int32 tensors dest [n], sel [n], n_sel [1]."""
    _check(LIB.sr_anchor_compact(_ptr(dest), int(dest.numel()), _ptr(sel), _ptr(n_sel), _stream_ptr(stream)))


def anchor_write(sidecar: SrSidecar, hidden: Sequence, dest, sel=None, n_sel=None, stream=None):
    """sr_anchor_write: hidden[l] are device tensors [n_tokens][d]."""
    ptrs = (ctypes.c_void_p * len(hidden))(*[_ptr(h) for h in hidden])
    n_tokens = int(dest.numel())
    _check(LIB.sr_anchor_write(ctypes.byref(sidecar), ptrs, n_tokens, _ptr(dest), _ptr(sel), _ptr(n_sel),
                               _stream_ptr(stream)))


def anchor_gather(sidecar: SrSidecar, block_table, block_cu, anchor_first, n_anchors, layers: Sequence[int],
                  out: Sequence, cu_seqlens, stream=None):
    """sr_anchor_gather: device int32 tensors for the tables, out[o] device
    tensors [t_cap][d] receiving layer layers[o]; cu_seqlens [n_req + 1]."""
    lay = (ctypes.c_int32 * len(layers))(*[int(x) for x in layers])
    ptrs = (ctypes.c_void_p * len(out))(*[_ptr(o) for o in out])
    t_cap = min(int(o.shape[0]) for o in out)
    n_req = int(n_anchors.numel())
    _check(LIB.sr_anchor_gather(ctypes.byref(sidecar), n_req, _ptr(block_table), _ptr(block_cu),
                                _ptr(anchor_first), _ptr(n_anchors), lay, len(layers), ptrs, t_cap,
                                _ptr(cu_seqlens), _stream_ptr(stream)))


# ------------------------------------------------------ graph-bucketed replay
class _DevArray:
    """A device buffer the library owns, seen by torch without a copy."""

    def __init__(self, ptr, shape, typestr):
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": typestr, "data": (ptr, False),
                                         "version": 3, "strides": None}


class ReplayGraph:
    """sr_replay_graph: one group of layers replayed from graphs captured at
    creation (one per total-length bucket), with host anchor fetch on a copy
    stream and an eager path for batches no bucket holds."""

    def __init__(self, shape, layers: Sequence[LayerTensors], max_segments: int, bucket_rows: Sequence[int],
                 workspace=None, n_slots: Optional[int] = None, varlen_status=None):
        self.shape = shape
        # The captured graphs hold the raw weight, state and tail pointers, so
        # the tensors behind them must outlive this object: keep references.
        self._tensors = list(layers)
        self._workspace = workspace
        self._status = varlen_status
        self._layers = make_layer_array(layers)
        self._sh = make_shape(shape)
        rows = (ctypes.c_int64 * len(bucket_rows))(*[int(r) for r in bucket_rows])
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        h = ctypes.c_void_p()
        _check(LIB.sr_replay_graph_create(ctypes.byref(self._sh), len(layers), self._layers,
                                          _n_slots(layers, n_slots), _ptr(varlen_status), int(max_segments),
                                          rows, len(bucket_rows), _ptr(workspace), int(ws_bytes), ctypes.byref(h)))
        self._h = h
        self.n_layers = len(layers)
        self.max_rows = int(LIB.sr_replay_graph_max_rows(h))
        self._pending_host = []

    def anchors(self, layer: int):
        """torch view [T_max][d_model] of layer `layer`'s anchor buffer."""
        import torch  # plumbing: device memory

        ptr = LIB.sr_replay_graph_anchors(self._h, int(layer))
        if not ptr:
            raise IndexError(layer)
        typestr = "<f4" if _DTYPE_CODES[self.shape.anchor_dtype] == SR_F32 else "<i2"
        return torch.as_tensor(_DevArray(ptr, (self.max_rows, int(self.shape.d_model)), typestr), device="cuda")

    def fetch(self, ranges, copy_stream):
        """sr_replay_graph_fetch: ranges are (host tensor [rows][d_model] in
        pinned memory, layer, dst_row).  The host tensors are kept referenced
        until the next fetch of this object."""
        arr = (SrHostRange * max(1, len(ranges)))()
        for i, (src, layer, dst_row) in enumerate(ranges):
            arr[i] = SrHostRange(src.data_ptr(), int(layer), int(dst_row), int(src.shape[0]))
        self._pending_host = [r[0] for r in ranges]
        _check(LIB.sr_replay_graph_fetch(self._h, arr, len(ranges), _stream_ptr(copy_stream)))

    def run(self, n_segments: int, t_total: int, cu_seqlens, slot_ids=None, stream=None, eager_anchors=None,
            eager_workspace=None) -> int:
        """Replays the batch; returns the bucket index used (-1: eager)."""
        used = ctypes.c_int32(-2)
        ea = None
        if eager_anchors is not None:
            ea = (ctypes.c_void_p * len(eager_anchors))(*[_ptr(a) for a in eager_anchors])
        ews = 0 if eager_workspace is None else eager_workspace.numel() * eager_workspace.element_size()
        _check(LIB.sr_replay_graph_run(self._h, int(n_segments), int(t_total), _ptr(cu_seqlens), _ptr(slot_ids),
                                       ea, _ptr(eager_workspace), int(ews), _stream_ptr(stream),
                                       ctypes.byref(used)))
        return int(used.value)

    def wait(self, stream=None):
        """sr_replay_graph_wait: `stream` waits for this object's last run."""
        _check(LIB.sr_replay_graph_wait(self._h, _stream_ptr(stream)))

    def close(self):
        if self._h:
            _check(LIB.sr_replay_graph_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
