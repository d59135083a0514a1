"""Constructed gather pins at the headline size (L = 122880 cached keys, n = 512).

At this prefix length attention over random data is nearly uniform, so
random-data parity cannot see a dropped or misplaced 16-key page (eq.
K_cache / V_cache, Sec. II): O moves by ~1e-2 of its size and LSE by ~1e-4.
These tests construct inputs whose answer depends on exactly which cache row
is read, in the launch configuration the benchmark times (the planner's own
choice: two key splits per row tile):

* needles: a chosen row's query equals one key (score ~60 above the rest), so
  its output is that key's value row; needles sit in the first and the last
  prefix page, at the first key of the second split and the last key of the
  first split of the row's workgroup, in the last prefix tile before the
  chunk, and inside the chunk;
* position probe: K = 0 makes every score 0, so o_i is the mean of V over keys
  0 .. L + i and LSE = ln(L + i + 1) exactly; with V[t] = (t mod 251) / 256
  the mean is a closed form, and the LSE counts the visible keys (one page
  more or less moves it by 1.3e-4).
"""
import math

import numpy as np
import pytest
import torch

from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, compare, note, oracle_rows, values

pytestmark = pytest.mark.gpu

L, N, HQ, HKV, D, G, P, BM = 122880, 512, 64, 4, 128, 16, 16, 256


def slot_of(case, t):
    return int(case.block_table[0, t // P]), t % P


def split_start(i):
    """First key of the second of two key splits for chunk row i's workgroup
    (256 packed rows = 16 chunk rows; key tiles of 64 split in halves, the
    larger share first)."""
    m0 = (i * G // BM) * BM
    kv_end = L + (min(m0 + BM, N * G) - 1) // G + 1
    ntiles = -(-kv_end // 64)
    return -(-ntiles // 2) * 64


def test_needles_at_the_page_split_and_chunk_boundaries():
    case = dg.config("c3_512")
    g = np.random.default_rng(31)
    alpha = math.sqrt(60 * math.sqrt(D))
    plan = [  # (chunk row, query head, needle position)
        (3, 1, 0),                              # first prefix page, first slot
        (40, 17, L - 1),                        # last prefix page, last slot
        (77, 33, split_start(77)),              # first key of the second split
        (150, 50, split_start(150) - 1),        # last key of the first split
        (201, 63, L - 64 + 13),                 # last prefix tile before the chunk
        (260, 20, L + 100),                     # inside the chunk (row 260 sees chunk keys 0..260)
        (511, 47, L + 511),                     # the last row's own key
        (333, 9, int(g.integers(1, L - 1))),    # somewhere in the middle
    ]
    targets = []
    for i, h, t in plan:
        assert t <= L + i
        u = g.standard_normal(D)
        u /= np.linalg.norm(u)
        vec = dg.to_bf16_bits((alpha * u).astype(np.float32))
        kv = h // G
        if t < L:
            page, s = slot_of(case, t)
            case.k_pool[page, s, kv] = vec
            want = case.v_pool[page, s, kv]
        else:
            case.k_new[t - L, kv] = vec
            want = case.v_new[t - L, kv]
        case.q[i, h] = vec
        targets.append((i, h, t, dg.bf16_bits_to_f32(want).astype(np.float64)))
    note(f"headline needles at {[t for _, _, t in plan]} (split starts {[split_start(i) for i, _, _ in plan]})")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    got = values(case, out)
    for i, h, t, want in targets:
        err = np.abs(got[i, h] - want).max()
        assert err < 2e-2, f"needle at key {t} for row {i} head {h}: max error {err:.3g}"
    rows = np.array(sorted({i for i, _, _ in plan}), dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, "headline needles")


def test_position_probe_counts_every_visible_key():
    case = dg.config("c3_512")
    t = np.arange(L, dtype=np.int64)
    page = case.block_table[0, t // P].astype(np.int64)
    slots = page * P + t % P
    kflat = case.k_pool.reshape(-1, HKV, D)
    vflat = case.v_pool.reshape(-1, HKV, D)
    kflat[slots] = 0
    val = lambda pos: dg.to_bf16_bits(((pos % 251) / 256.0).astype(np.float32))  # noqa: E731  exact in bf16
    vflat[slots] = val(t)[:, None, None]
    case.k_new[:] = 0
    case.v_new[:] = val(L + np.arange(N, dtype=np.int64))[:, None, None]
    note("headline position probe: K = 0, V[t] = (t mod 251)/256, L=122880 n=512")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    allv = (np.arange(L + N, dtype=np.int64) % 251) / 256.0
    mean = np.cumsum(allv)[L:] / np.arange(L + 1, L + N + 1)       # o_i for every head and column
    want_lse = np.log(np.arange(L + 1, L + N + 1, dtype=np.float64))
    got = values(case, out)
    got_lse = lse.cpu().numpy().astype(np.float64)
    o_err = np.abs(got - mean[:, None, None]).max()
    l_err = np.abs(got_lse - want_lse[:, None]).max()
    note(f"position probe: max |o - mean| {o_err:.3g}, max |lse - ln(L+i+1)| {l_err:.3g}")
    assert o_err <= 2.0 ** -9, o_err      # half a bf16 step at 0.5 plus the accumulation
    assert l_err <= 1e-4, l_err           # one 16-key page more or less: 1.3e-4
