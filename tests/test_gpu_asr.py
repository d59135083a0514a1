"""GPU test of asynchronous state reconciliation (Algorithm 1) on one device.

One full reconciliation cycle at a small scale, with the interleaving fixed by
gating when the secondary's work may be observed: tasks served during the
warm-up and a catch-up round, a swap that leaves a remainder, tasks on the new
primary.  Checked against
* the token-level model of Algorithm 1 (which ids every task computes, the
  primary's state after the swap),
* the fp64 oracle (outputs of tasks on the old and on the new primary: RoPE
  attention over the logical token sequence they serve),
* a one-shot prefill of the reconciled sequence (the new primary's cache,
  built by warm-up + catch-up + tasks, holds the same rotated keys and values
  bit for bit: a key's rotation depends only on its token and position).
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from oracle.asr_model import AsrModel
from paper_2605_07325_amd import asr, csr
from tests.gpu_harness import note
from tests.parity import check_bf16

pytestmark = pytest.mark.gpu

HQ, HKV, D, P = 16, 2, 128, 16
PRE, CHUNK, DYN, TAU, NCATCH = 300, 50, 8, 1500, 50
ROPE = (oracle.ROPE_NEOX, 0, 1e6)


def ids(ranges):
    return [t for a, b in ranges for t in range(a, b)]


def host_rows(table, id_list):
    idx = torch.tensor(id_list, dtype=torch.int64, device="cuda")
    conv = lambda t: t.index_select(0, idx).view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
    return conv(table.q), conv(table.k), conv(table.v)


def oracle_task(table, seq_ids, n_rows):
    """fp64 RoPE attention of the last n_rows tokens of seq_ids over the whole sequence."""
    q, k, v = host_rows(table, seq_ids)
    S = len(seq_ids)
    cu = np.array([0, S], np.int32)
    rows = np.arange(S - n_rows, S, dtype=np.int32)
    out, lse, _ = oracle.attention(oracle.BF16, q, k, v, None, None, None, 1, cu, None, rows, HQ, HKV, D, P,
                                   rope=ROPE)
    return out, lse


@pytest.mark.parametrize("partitioned", [True, False], ids=["cu-masked", "two-streams"])
def test_one_reconciliation_cycle(partitioned):
    table = asr.TokenTable.synthetic(6000, HQ, HKV, D, seed=11)
    desc = csr.make_desc(HQ, HKV, D, P, rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e6)
    if partitioned:
        sec_cus = asr.xcd_spread_cus(4)
        ps = asr.cu_masked_stream(sorted(set(range(256)) - set(sec_cus)))
        ss = asr.cu_masked_stream(sec_cus)
    else:
        ps, ss = torch.cuda.Stream(), torch.cuda.Stream()
    allow = {"warmup": False, "catchup": False}
    rec = asr.Reconciler(table, desc, (0, PRE), TAU, NCATCH, 4096, ps, ss, gate=lambda k: allow[k],
                         sync_secondary=True, keep_outputs=True)
    rec.prime()
    model = AsrModel(list(range(PRE)), TAU, NCATCH)
    trigger = (TAU - PRE) // CHUNK - 1  # the chunk that brings |X_static| to tau
    checks = {}
    for i in range(trigger + 9):
        if i == trigger + 4:
            allow["warmup"] = True       # warm-up seen done after 3 buffered chunks -> one catch-up round
        if i == trigger + 5:
            allow["catchup"] = True      # catch-up seen done with one chunk buffered -> swap, remainder 1 chunk
        chunk = (PRE + CHUNK * i, PRE + CHUNK * (i + 1))
        dyn = (5000 + DYN * i, 5000 + DYN * (i + 1))
        seen = len(rec.events)
        note(f"asr task {i} ({'masked' if partitioned else 'streams'}), primary {rec.primary_cache().name}")
        task = rec.step(chunk, dyn)
        for e in rec.events[seen:]:
            if e.kind in ("catchup", "swap") and e.task == i:
                model.secondary_done()
        expect = model.increment(list(range(*chunk)))
        assert ids(task.computed[:-1]) == expect, f"task {i} computed other ids than Algorithm 1"
        assert rec.reconciling == model.reconciling
        if i == trigger + 2:
            checks["old"] = (task, ids(rec.logical_ids()) + list(range(*dyn)))
        if i == trigger + 7:
            checks["new"] = (task, ids(rec.logical_ids()) + list(range(*dyn)))
    torch.cuda.synchronize()
    assert [e.kind for e in rec.events] == ["warmup", "catchup", "swap"]
    assert [e[0] for e in model.log] == ["warmup", "catchup", "swap"]
    assert ids(rec.logical_ids()) == model.x_static()
    swap = rec.events[2]
    assert swap.tokens == CHUNK                       # one chunk left for the new primary
    assert checks["new"][0].cache != checks["old"][0].cache

    # outputs on the old primary (during the warm-up) and on the new one (remainder task + 1)
    for label, (task, seq) in checks.items():
        n = asr.rlen(task.computed)
        ref, ref_lse = oracle_task(table, seq, n)
        got = task.out.float().cpu().numpy().astype(np.float64)
        ok, st = check_bf16(got, None, ref, None)
        note(f"asr {label} primary task: rows={n} {st}")
        assert ok, f"{label}: {st}"

    # the reconciled cache equals a one-shot prefill cache write of the same ids
    prim = rec.primary_cache()
    seq = ids(prim.ids)
    assert seq == model.primary_cached    # warm-up + catch-up + tasks put exactly these ids in the cache
    fresh = asr.Cache("fresh", prim.k_pool.shape[0], P, HKV, D, torch.bfloat16, seed=99)
    qd = table.q.index_select(0, torch.tensor(seq, device="cuda"))
    kd = table.k.index_select(0, torch.tensor(seq, device="cuda"))
    vd = table.v.index_select(0, torch.tensor(seq, device="cuda"))
    cu = torch.tensor([0, len(seq)], dtype=torch.int32, device="cuda")
    csr.prefill(desc, qd, kd, vd, cu, len(seq), k_pool=fresh.k_pool, v_pool=fresh.v_pool,
                block_table=fresh.block_table, bt_stride=fresh.block_table.shape[1], want_lse=False)
    torch.cuda.synchronize()
    pos = torch.arange(len(seq), device="cuda")

    def rows_of(c):
        slot = c.block_table[0, pos // P].long() * P + pos % P
        return (c.k_pool.reshape(-1, HKV, D).index_select(0, slot), c.v_pool.reshape(-1, HKV, D).index_select(0, slot))

    rk, rv = rows_of(prim)
    fk, fv = rows_of(fresh)
    assert torch.equal(rk.view(torch.int16), fk.view(torch.int16))
    assert torch.equal(rv.view(torch.int16), fv.view(torch.int16))
    note(f"asr reconciled cache ({len(seq)} positions) equals a one-shot prefill bit for bit")
    del rec
    asr.destroy_streams(ps, ss)
