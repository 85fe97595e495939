"""sr_replay_state_noalloc (the replay on the library's own device scratch)
against sr_replay_state on a caller workspace, through the C ABI: two calls
in a row, the second on a smaller batch, must write exactly what the
workspace entry point writes for the same inputs (same kernels, so bit for
bit), and both must agree with the fp64 oracle.  A call whose workspace need
exceeds the scratch is refused on the host with nothing written."""
import pytest
import torch

import workloads as W
from gpu_harness import TOL_BF16, check_pairs, layer_tensors, log, run, upload

pytestmark = pytest.mark.gpu


def _noalloc(dev):
    import paper_2609_33477_amd as sr
    wl = dev.wl
    sr.replay_state_noalloc(wl.shape, layer_tensors(dev), len(wl.seg_lens), wl.t_total, dev.cu_seqlens,
                            dev.slot_ids)
    torch.cuda.synchronize()


def test_noalloc_matches_workspace_entry_point_twice():
    shape = W.Shape(256, 2, 4, 128, 128)
    cases = [("noalloc_big", [300, 1, 129, 0, 64, 700], [5, 0, 2, 3, -1, 1]),
             ("noalloc_small", [70, 3], [1, 4])]
    for name, seg, slots in cases:
        wl = W.make_workload(name, shape, seg, seed=7, slot_ids=slots, n_slots=6)
        log(f"{name}: T={wl.t_total}, segments {seg}")
        ref = upload(wl)
        run(ref)
        got = upload(wl)                       # outputs NaN-filled: unwritten slots stay visible
        _noalloc(got)
        for li in range(len(wl.layers)):
            assert torch.equal(got.layers[li].state_out.nan_to_num(7.0), ref.layers[li].state_out.nan_to_num(7.0))
            assert torch.equal(got.layers[li].tail_out.float().nan_to_num(7.0),
                               ref.layers[li].tail_out.float().nan_to_num(7.0))
        live = [(0, b) for b, s in enumerate(slots) if s >= 0 and seg[b] > 0]
        check_pairs(got, live, TOL_BF16)


def test_noalloc_refuses_a_batch_beyond_its_scratch():
    import paper_2609_33477_amd as sr
    shape = W.Shape(2560, 16, 32, 128, 128)
    t_big = 16384                              # ~200 MiB of workspace for this shape
    assert sr.replay_workspace_size(shape, 1, t_big) > sr.NOALLOC_SCRATCH_BYTES
    # a real batch of that size (every buffer holds what the call names)
    wl = W.make_workload("noalloc_refuse", shape, [t_big], seed=9)
    dev = upload(wl)
    with pytest.raises(sr.SrError) as e:
        sr.replay_state_noalloc(shape, layer_tensors(dev), 1, t_big, dev.cu_seqlens, dev.slot_ids)
    assert e.value.status == 4                 # SR_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(dev.layers[0].state_out))
