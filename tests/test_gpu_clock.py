"""GPU test of the profiling hooks: the per-workgroup clock (csr_set_workgroup_clock)
changes no output bit and records every unit of the launch plan exactly once, with
sane times and XCD ids, inside the attention kernel's own events
(csr_set_attention_events)."""
import numpy as np
import pytest
import torch

from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, note

pytestmark = pytest.mark.gpu


def test_workgroup_clock_records_every_unit_and_changes_nothing():
    case = dg.config("c2")  # L 8192, n 256: 4 kv heads x 16 row tiles x 4 key splits = 256 units
    dev = Dev(case)
    note("workgroup clock: C2 with and without the hook")
    out0, lse0 = dev.extend()
    for _ in range(3):  # first-call costs (workspace, code objects) stay out of the timed launch below
        dev.extend()
    torch.cuda.synchronize()
    stamps = torch.zeros((1024, 4), dtype=torch.int64, device="cuda")
    # the library's event hook brackets the same attention launch (recording once creates the raw events)
    begin, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    begin.record()
    end.record()
    torch.cuda.synchronize()
    csr.set_workgroup_clock(stamps)
    csr.set_attention_events(begin.cuda_event, end.cuda_event)
    try:
        out1, lse1 = dev.extend()
    finally:
        csr.set_workgroup_clock(None)
        csr.set_attention_events(None, None)
    torch.cuda.synchronize()
    assert torch.equal(out0.view(torch.int16), out1.view(torch.int16))
    assert torch.equal(lse0.view(torch.int32), lse1.view(torch.int32))
    t = csr.workgroup_clock_table(stamps)
    n = len(t["end_us"])
    assert n == 256, n
    assert np.all(t["end_us"] >= t["start_us"]) and np.all(t["start_us"] >= 0)
    assert t["end_us"].max() < 10_000  # one launch, well under 10 ms
    assert set(t["xcd"].tolist()) == set(range(8))
    assert set(t["kv_head"].tolist()) == {0, 1, 2, 3} and set(t["split"].tolist()) == {0, 1, 2, 3}
    assert np.all(t["seq"] == 0) and np.all(t["te"] > t["tb"])
    # the four splits of a row block tile its key range: per kv head, each split's range appears 16 times
    for g in range(4):
        for s in range(4):
            m = (t["kv_head"] == g) & (t["split"] == s)
            assert m.sum() == 16
    # the stamps are counted at 100 MHz (the device's constant wall clock): the span from the first start
    # to the last end lies inside the attention kernel's events and covers most of them (about 0.87 on a
    # warm device; a clock at half or twice the rate would fall outside)
    span_us, event_us = t["end_us"].max(), begin.elapsed_time(end) * 1e3
    ratios = [span_us / event_us]
    assert span_us <= event_us * 1.01 + 1.0, (span_us, event_us)
    for _ in range(2):  # the lower bound is a timing figure: the best of up to three launches
        if max(ratios) > 0.5:
            break
        csr.set_workgroup_clock(stamps)
        csr.set_attention_events(begin.cuda_event, end.cuda_event)
        try:
            dev.extend()
        finally:
            csr.set_workgroup_clock(None)
            csr.set_attention_events(None, None)
        torch.cuda.synchronize()
        sp, ev = csr.workgroup_clock_table(stamps)["end_us"].max(), begin.elapsed_time(end) * 1e3
        assert sp <= ev * 1.01 + 1.0, (sp, ev)
        ratios.append(sp / ev)
    assert max(ratios) > 0.5, ratios
    note(f"workgroup clock: 256 units, ends {t['end_us'].min():.1f}..{t['end_us'].max():.1f} us after the first start, launch {event_us:.1f} us")


def test_workgroup_clock_on_the_fp8_decode_kernel():
    # the 4-wave kernel (two workgroups per CU) of an e4m3 cache at n = 1: one record per unit of the
    # plan, every (kv head, split) pair once, tiles that tile each kv head's key range, outputs unchanged
    case = dg.with_fp8_pools(dg.make_case("clk8", dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128,
                                          cache_len=[20000], seqlen_q=[1], seed=5, cfg_id=312), cfg_id=312)
    dev = Dev(case)
    dev.k_pool = torch.from_numpy(case.k_pool).cuda()
    dev.v_pool = torch.from_numpy(case.v_pool).cuda()
    dev.desc.kv_dtype = csr.CSR_KV_FP8_E4M3
    dev.desc.k_scale, dev.desc.v_scale = 0.0625, 0.0390625
    note("workgroup clock: fp8 decode L=20000 n=1 with and without the hook")
    out0, lse0 = dev.extend()
    stamps = torch.zeros((4096, 4), dtype=torch.int64, device="cuda")
    csr.set_workgroup_clock(stamps)
    try:
        out1, lse1 = dev.extend()
    finally:
        csr.set_workgroup_clock(None)
    torch.cuda.synchronize()
    assert torch.equal(out0.view(torch.int16), out1.view(torch.int16)) and torch.equal(lse0, lse1)
    t = csr.workgroup_clock_table(stamps)
    splits = int(t["split"].max()) + 1
    assert len(t["end_us"]) == 4 * splits  # one row tile per kv head at n = 1
    ntiles = -(-(20000 + 1) // 64)
    for g in range(4):
        m = t["kv_head"] == g
        assert sorted(t["split"][m].tolist()) == list(range(splits))
        order = np.argsort(t["split"][m])
        tb, te = t["tb"][m][order], t["te"][m][order]
        assert tb[0] == 0 and te[-1] == ntiles and np.all(tb[1:] == te[:-1])  # contiguous, complete
    assert np.all(t["end_us"] >= t["start_us"])
    note(f"workgroup clock fp8 decode: {4 * splits} units, last end {t['end_us'].max():.1f} us after the first start")
