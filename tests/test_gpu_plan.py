"""GPU test of the ragged-batch work order (the device-side planner).

The order the planner leaves in the workspace is read back and checked
against what it must be: a permutation of the active units (every unit whose
row tile holds rows runs exactly once), slot w on XCD w % 8, and each XCD's
queue longest first (within the length spread of one subgroup of row tiles).
"""
import math
import numpy as np
import pytest
import torch

from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, compare, note, oracle_rows

pytestmark = pytest.mark.gpu

BM = 256  # packed rows per workgroup of the bf16 kernel (chunks longer than 8 tokens at G = 16)


def subgroup_rows(batch, hkv, mtiles):
    """Row tiles per subgroup: 4, more when batch * Hkv * mtiles exceeds 3072."""
    return max(4, -(-batch * hkv * mtiles // 768))


def check_order(case, dev, nsplit, L, n):
    """Runs the call, reads the order back and checks it; returns the output and LSE."""
    B, Hkv, G = case.batch, case.num_kv_heads, case.num_q_heads // case.num_kv_heads
    ws_bytes = csr.extend_workspace_size(dev.desc, B, case.total_q, case.max_seqlen_q, case.max_cache_len)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    out, lse = dev.extend(workspace=ws)
    torch.cuda.synchronize()
    mtiles = math.ceil(case.max_seqlen_q * G / BM)
    units = B * Hkv * mtiles * nsplit
    slots = (units + 7) // 8 + mtiles * nsplit
    order = ws[ws_bytes - 8 * slots * 4:].cpu().numpy().view(np.int32).reshape(slots, 8)

    def decode(u):  # the attention kernel's unit numbering
        mt = mtiles - 1 - u % mtiles
        rest = u // mtiles
        s = rest % nsplit
        rest //= nsplit
        return rest // Hkv, rest % Hkv, s, mt

    def length(u):  # key tiles the unit scans
        b, _, _, mt = decode(u)
        rows = int(n[b]) * G
        m_last = min(mt * BM + BM, rows) - 1
        return math.ceil(math.ceil((int(L[b]) + m_last // G + 1) / 64) / nsplit)

    active = {u for u in range(units) if decode(u)[3] * BM < int(n[decode(u)[0]]) * G}
    got = order[order >= 0]
    assert len(got) == len(set(got.tolist())), "a unit is scheduled twice"
    assert set(got.tolist()) == active, "scheduled units differ from the active units"
    K = subgroup_rows(B, Hkv, mtiles)
    spread = math.ceil(K * BM / G / 64 / nsplit) + 1  # key tiles between the row tiles of one subgroup
    loads = []
    for x in range(8):
        q = [length(int(u)) for u in order[:, x] if u >= 0]
        loads.append(sum(q))
        for a_, b_ in zip(q, q[1:]):
            assert b_ <= a_ + spread, f"XCD {x}: a longer unit runs after a shorter one ({b_} after {a_})"
    note(f"work order ok: {len(got)} units, XCD loads {loads}")
    longest = max(length(u) for u in active)
    assert max(loads) <= sum(loads) / 8 + 8 * longest, "XCD loads far from balanced"
    return out, lse


@pytest.mark.parametrize("nsplit", [1, 3])
def test_work_order_is_a_longest_first_permutation(nsplit):
    csr.set_plan_overrides(nsplit=nsplit)
    g = np.random.default_rng(17)
    L = g.integers(0, 20000, size=7)
    n = g.integers(9, 700, size=7)
    n[2] = 700
    case = dg.make_case("plan", dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=L.tolist(),
                        seqlen_q=n.tolist(), page_size=16, scale=0.5, seed=4, cfg_id=320, interleave=True)
    note(f"work order: L={L.tolist()} n={n.tolist()} nsplit={nsplit}")
    check_order(case, Dev(case), nsplit, L, n)


def test_work_order_at_the_group_limit_with_wider_subgroups():
    """256 sequences x 4 kv heads = 1024 groups (the most one plan takes) of up to 7 row
    tiles: 10 row tiles per subgroup; the order is checked as above and the outputs of
    five sequences on every row against the oracle."""
    csr.set_plan_overrides(nsplit=1)
    g = np.random.default_rng(23)
    B = 256
    L = g.integers(0, 400, size=B)
    n = g.integers(9, 112, size=B)
    n[5] = 112
    L[7] = 0
    case = dg.make_case("plan1024", dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128,
                        cache_len=L.tolist(), seqlen_q=n.tolist(), page_size=16, scale=0.5, seed=4, cfg_id=321,
                        interleave=True)
    assert subgroup_rows(B, 4, math.ceil(112 * 16 / BM)) == 10
    note(f"work order at 1024 groups: {B} sequences, n {int(n.min())}..{int(n.max())}, L {int(L.min())}..{int(L.max())}")
    out, lse = check_order(case, Dev(case), 1, L, n)
    cu = np.concatenate([[0], np.cumsum(n)])
    rows = np.concatenate([np.arange(cu[b], cu[b + 1]) for b in (0, 5, 7, 128, B - 1)]).astype(np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, "plan1024")
