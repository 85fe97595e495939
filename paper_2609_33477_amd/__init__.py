"""SuffixReplay state reconstruction on MI355X (gfx950).

The replay path lives in libsr_replay.so (hand-written HIP kernels behind the
C ABI of include/sr_replay.h); this package holds the in-tree build script
(``build``) and a thin ctypes binding (``binding``) with the same names as the
C entry points.  The binding, and with it the library, is loaded on first
attribute access so that the build script can run before a library exists.
"""
import importlib

_BINDING_NAMES = {
    "LIB_PATH", "SR_BF16", "SR_F32", "SR_FP8_E4M3", "KERNEL_KINDS", "LayerTensors", "SrError",
    "conv_tail_bytes", "kernel_timing_enable", "kernel_timing_read", "kernel_timing_kinds", "replay_state",
    "replay_workspace_size", "state_bytes", "status_str", "SrSidecar", "make_sidecar", "anchor_dest_table",
    "anchor_compact", "anchor_write", "anchor_gather", "ReplayGraph", "SrHostRange", "replay_state_noalloc",
    "NOALLOC_SCRATCH_BYTES", "validate_varlen", "validate_varlen_host", "VARLEN_BAD_START", "VARLEN_NOT_MONOTONE", "VARLEN_BAD_TOTAL",
    "VARLEN_SLOT_RANGE", "VARLEN_SLOT_DUPLICATE", "BlockTensors", "group_workspace_size", "replay_group",
}


def __getattr__(name):
    if name in _BINDING_NAMES:
        return getattr(importlib.import_module(".binding", __name__), name)
    raise AttributeError(name)
