"""Pins for the CPU fp64 oracle, independent of the oracle's own code.

Each test checks the oracle against something the paper or mathematics fixes:
torch's scaled-dot-product attention and logsumexp (library routines) on the
logical, unpaged sequence; closed forms; a hand-derived worked example; and the
paper's invariants (prefix stability, append-only growth, the visible-pair
count of eq. (TTFT_derivation_2)).
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import datagen as dg

HERE = os.path.dirname(os.path.abspath(__file__))


def as_f64(case, a):
    return dg.bf16_bits_to_f32(a).astype(np.float64) if case.dtype == dg.BF16 else a.astype(np.float64)


def run_oracle(case, rows=None, cache_len="case", scale=None):
    if rows is None:
        rows = np.arange(case.total_q, dtype=np.int32)
    cl = case.cache_len if isinstance(cache_len, str) else cache_len
    return oracle.attention(oracle.BF16 if case.dtype == dg.BF16 else oracle.F32, case.q, case.k_new,
                            case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                            case.cu_seqlens_q, cl, rows, case.num_q_heads, case.num_kv_heads,
                            case.head_dim, case.page_size, scale=scale)


def library_reference(case, b, scale=None):
    """torch SDPA (fp64, CPU) on the logical sequence [prefix ; chunk] of sequence b."""
    G = case.num_q_heads // case.num_kv_heads
    lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
    L = int(case.cache_len[b])
    k = np.concatenate([as_f64(case, case.k_prefix[b]), as_f64(case, case.k_new[lo:hi])], axis=0)
    v = np.concatenate([as_f64(case, case.v_prefix[b]), as_f64(case, case.v_new[lo:hi])], axis=0)
    q = torch.from_numpy(as_f64(case, case.q[lo:hi])).permute(1, 0, 2)  # [Hq, n, d]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)  # [Hq, L+n, d]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)
    n = hi - lo
    mask = torch.arange(L + n)[None, :] <= (L + torch.arange(n))[:, None]  # [n, L+n]
    sc = (1.0 / math.sqrt(case.head_dim)) if scale is None else scale
    out = torch.nn.functional.scaled_dot_product_attention(q, kt, vt, attn_mask=mask, scale=sc)
    s = torch.matmul(q, kt.transpose(1, 2)) * sc
    s = s.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    return out.permute(1, 0, 2).numpy(), lse.permute(1, 0).numpy()


SMALL = [
    dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[40], seqlen_q=[9], paged=False),
    dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=2, head_dim=16, cache_len=[37], seqlen_q=[11], page_size=4),
    dict(dtype=dg.BF16, num_q_heads=4, num_kv_heads=4, head_dim=8, cache_len=[0], seqlen_q=[13], page_size=2),
    dict(dtype=dg.BF16, num_q_heads=6, num_kv_heads=3, head_dim=8, cache_len=[5, 0, 33], seqlen_q=[3, 7, 1],
         page_size=4, interleave=True),
    dict(dtype=dg.F32, num_q_heads=2, num_kv_heads=1, head_dim=4, cache_len=[64, 17], seqlen_q=[16, 5],
         page_size=16),
]


@pytest.mark.parametrize("spec", range(len(SMALL)))
def test_oracle_matches_library_sdpa(spec):
    case = dg.make_case(f"small{spec}", scale=0.7, seed=spec, cfg_id=200 + spec, keep_prefix=True,
                        **SMALL[spec])
    out, lse, _ = run_oracle(case)
    for b in range(case.batch):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        if hi == lo:
            continue
        ref, ref_lse = library_reference(case, b)
        np.testing.assert_allclose(out[lo:hi], ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[lo:hi], ref_lse, rtol=0, atol=1e-12)


def test_oracle_custom_scale_matches_library():
    case = dg.make_case("scale", dtype=dg.F32, num_q_heads=4, num_kv_heads=2, head_dim=8, cache_len=[20],
                        seqlen_q=[6], page_size=8, seed=3, cfg_id=230, keep_prefix=True)
    out, lse, _ = run_oracle(case, scale=0.3)
    ref, ref_lse = library_reference(case, 0, scale=0.3)
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, ref_lse, atol=1e-12, rtol=0)


def test_worked_two_key_example():
    vals = {}
    for line in open(os.path.join(HERE, "golden", "two_key_example.txt")):
        if line.startswith("#") or not line.strip():
            continue
        key, *nums = line.split()
        vals[key] = np.array([float(x) for x in nums])
    f = lambda k: vals[k].astype(np.float32).reshape(1, 1, -1)  # noqa: E731
    out, lse, _ = oracle.attention(oracle.F32, f("q"), f("k_new"), f("v_new"), f("k_cache").reshape(1, 1, 1, 2),
                                   f("v_cache").reshape(1, 1, 1, 2), None, 1, np.array([0, 1]), np.array([1]),
                                   np.array([0]), 1, 1, 2, 1, scale=float(vals["scale"][0]))
    np.testing.assert_allclose(out[0, 0], vals["expect_out"], atol=1e-14)
    assert abs(lse[0, 0] - vals["expect_lse"][0]) < 1e-14


def test_zero_keys_give_mean_of_visible_values():
    """K == 0: every score is 0, exp(0) = 1, so o_i = mean of V over keys 0..L+i
    and lse = ln(L+i+1)."""
    case = dg.make_case("k0", dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=16, cache_len=[29],
                        seqlen_q=[7], page_size=4, scale=0.5, seed=4, cfg_id=231, keep_prefix=True)
    case.k_new[:] = 0
    case.k_pool[:] = 0
    out, lse, _ = run_oracle(case)
    v = np.concatenate([as_f64(case, case.v_prefix[0]), as_f64(case, case.v_new)], axis=0)
    L = 29
    for i in range(7):
        for h in range(4):
            expect = v[: L + i + 1, h // 2].mean(axis=0)
            np.testing.assert_allclose(out[i, h], expect, atol=1e-14)
            assert abs(lse[i, h] - math.log(L + i + 1)) < 1e-13


def test_constant_values_pass_through():
    case = dg.make_case("vc", dtype=dg.F32, num_q_heads=2, num_kv_heads=1, head_dim=8, cache_len=[50],
                        seqlen_q=[5], page_size=8, seed=5, cfg_id=232)
    c = np.linspace(-2, 3, 8).astype(np.float32)
    case.v_new[:] = c
    flat = case.v_pool.reshape(-1, 1, 8)
    flat[:] = c
    out, _, _ = run_oracle(case)
    np.testing.assert_allclose(out, np.broadcast_to(c, out.shape), atol=1e-14)


def test_single_token_prefill_returns_its_value():
    case = dg.make_case("one", dtype=dg.BF16, num_q_heads=4, num_kv_heads=1, head_dim=16, cache_len=[0],
                        seqlen_q=[1], seed=6, cfg_id=233)
    out, lse, _ = run_oracle(case)
    np.testing.assert_array_equal(out[0], np.broadcast_to(as_f64(case, case.v_new[0, 0]), (4, 16)))
    q = as_f64(case, case.q[0])
    k = as_f64(case, case.k_new[0, 0])
    np.testing.assert_allclose(lse[0], q @ k / 4.0, atol=1e-14)


def test_needle_selects_its_value():
    """A key aligned with the query (score ~60 above the rest) selects its value."""
    case = dg.make_case("needle", dtype=dg.F32, num_q_heads=1, num_kv_heads=1, head_dim=16, cache_len=[45],
                        seqlen_q=[3], page_size=4, scale=0.05, seed=7, cfg_id=234, keep_prefix=True)
    g = np.random.default_rng(0)
    u = g.standard_normal(16)
    u /= np.linalg.norm(u)
    alpha = math.sqrt(60 * 4)  # alpha^2 * (1/sqrt(16)) = 60
    case.q[1, 0] = (alpha * u).astype(np.float32)
    needle_t = 13  # a prefix key, reached through the block table
    page = case.block_table[0, needle_t // 4]
    case.k_pool[page, needle_t % 4, 0] = (alpha * u).astype(np.float32)
    out, _, _ = run_oracle(case, rows=np.array([1]))
    want = case.v_pool[page, needle_t % 4, 0].astype(np.float64)
    np.testing.assert_allclose(out[0, 0], want, rtol=1e-12, atol=1e-12)


def test_shift_invariance_of_softmax():
    """k_t -> k_t + w for every key: o unchanged, lse shifted by scale * <q, w>."""
    case = dg.make_case("shift", dtype=dg.F32, num_q_heads=2, num_kv_heads=1, head_dim=8, cache_len=[21],
                        seqlen_q=[6], page_size=4, seed=8, cfg_id=235)
    for a in (case.q, case.k_new, case.k_pool, case.v_new, case.v_pool):  # exact in fp32 after shifting
        a[...] = np.round(np.nan_to_num(a) * 8) / 8
    out0, lse0, _ = run_oracle(case)
    w = (np.arange(8) / 4 - 1).astype(np.float32)
    case.k_new += w
    case.k_pool += w
    out1, lse1, _ = run_oracle(case)
    shift = (case.q.astype(np.float64) @ w.astype(np.float64)) / math.sqrt(8)
    np.testing.assert_allclose(out1, out0, atol=1e-13)
    np.testing.assert_allclose(lse1, lse0 + shift, atol=1e-12)


def test_prefix_order_does_not_matter():
    """The whole cached prefix is visible to every chunk row and nothing in the
    definition depends on key position, so permuting prefix tokens keeps o."""
    case = dg.make_case("perm", dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=16, cache_len=[40],
                        seqlen_q=[5], page_size=8, scale=0.5, seed=9, cfg_id=236)
    out0, lse0, _ = run_oracle(case)
    perm = np.random.default_rng(1).permutation(case.block_table[0, :5])
    case.block_table[0, :5] = perm  # whole prefix pages (40 = 5 pages of 8) reordered
    out1, lse1, _ = run_oracle(case)
    np.testing.assert_allclose(out1, out0, atol=1e-13)
    np.testing.assert_allclose(lse1, lse0, atol=1e-13)


def test_causality_future_keys_do_not_matter():
    case = dg.make_case("causal", dtype=dg.BF16, num_q_heads=2, num_kv_heads=1, head_dim=8, cache_len=[10],
                        seqlen_q=[8], page_size=4, seed=10, cfg_id=237)
    out0, _, _ = run_oracle(case)
    case.k_new[5:] = dg.to_bf16_bits(np.full(case.k_new[5:].shape, 3.0, np.float32))
    case.v_new[5:] = dg.to_bf16_bits(np.full(case.v_new[5:].shape, -7.0, np.float32))
    out1, _, _ = run_oracle(case)
    np.testing.assert_array_equal(out1[:5], out0[:5])
    assert np.abs(out1[5:] - out0[5:]).max() > 1e-3


def test_gqa_equals_repeated_kv_heads():
    base = dg.make_case("gqa", dtype=dg.BF16, num_q_heads=4, num_kv_heads=1, head_dim=8, cache_len=[12],
                        seqlen_q=[4], page_size=4, seed=11, cfg_id=238)
    out0, lse0, _ = run_oracle(base)
    rep = dg.make_case("mha", dtype=dg.BF16, num_q_heads=4, num_kv_heads=4, head_dim=8, cache_len=[12],
                       seqlen_q=[4], page_size=4, seed=11, cfg_id=238)
    rep.q[:] = base.q
    for src, dst in ((base.k_new, rep.k_new), (base.v_new, rep.v_new)):
        dst[:] = np.repeat(src, 4, axis=1)
    rep.block_table[:] = base.block_table
    for src, dst in ((base.k_pool, rep.k_pool), (base.v_pool, rep.v_pool)):
        dst[:] = np.repeat(src, 4, axis=2)
    out1, lse1, _ = run_oracle(rep)
    np.testing.assert_array_equal(out1, out0)
    np.testing.assert_array_equal(lse1, lse0)


def test_prefix_stability_extend_equals_prefill_tail():
    """Cached K/V are not altered by later tokens (Sec. II, after eq. (V_cache)):
    extend over the cached prefix equals the last n rows of a full prefill over
    the concatenated history (here given entirely as new tokens, L = 0)."""
    case = dg.make_case("stab", dtype=dg.BF16, num_q_heads=8, num_kv_heads=2, head_dim=16, cache_len=[53],
                        seqlen_q=[10], page_size=4, scale=0.5, seed=12, cfg_id=239, keep_prefix=True)
    out_ext, lse_ext, _ = run_oracle(case)
    full = dg.make_case("stab_full", dtype=dg.BF16, num_q_heads=8, num_kv_heads=2, head_dim=16, cache_len=[0],
                        seqlen_q=[63], page_size=4, seed=13, cfg_id=240)
    full.k_new[:] = np.concatenate([case.k_prefix[0], case.k_new])
    full.v_new[:] = np.concatenate([case.v_prefix[0], case.v_new])
    full.q[53:] = case.q
    out_full, lse_full, _ = run_oracle(full, rows=np.arange(53, 63), cache_len=None)
    np.testing.assert_array_equal(out_full, out_ext)
    np.testing.assert_array_equal(lse_full, lse_ext)


def test_append_then_extend_chunk_split():
    """Incremental extensibility (Theorem 2): appending chunk rows 0..i-1 and
    then extending with the single token i over the longer cache reproduces
    row i of the one-shot extend."""
    case = dg.make_case("split", dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=16, cache_len=[18, 7],
                        seqlen_q=[6, 4], page_size=4, scale=0.5, seed=14, cfg_id=241, interleave=True)
    out_all, lse_all, _ = run_oracle(case)
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table,
                              case.bt_stride, case.cu_seqlens_q, case.cache_len, 2, 16, 4)
    for b in range(2):
        for i in range(int(case.seqlen_q[b])):
            tok = int(case.cu_seqlens_q[b]) + i
            one_q = case.q[tok:tok + 1]
            cu = np.array([0, 1], np.int32)
            bt = case.block_table[b:b + 1]
            L = np.array([case.cache_len[b] + i], np.int32)
            out, lse, _ = oracle.attention(oracle.BF16, one_q, case.k_new[tok:tok + 1], case.v_new[tok:tok + 1],
                                           kp, vp, bt, case.bt_stride, cu, L, np.array([0]), 4, 2, 16, 4)
            np.testing.assert_array_equal(out[0], out_all[tok])
            np.testing.assert_array_equal(lse[0], lse_all[tok])


def test_append_touches_only_empty_slots():
    """Append-only growth: exactly n_b * Hkv * d elements change per pool, all of
    them previously empty (canary) slots; no cached element is modified."""
    case = dg.config("c5", seed=3, cache_len=[70, 3, 0, 45], seqlen_q=[9, 30, 5, 1], num_q_heads=8,
                     num_kv_heads=2, head_dim=16, page_size=8)
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table,
                              case.bt_stride, case.cu_seqlens_q, case.cache_len, 2, 16, 8)
    for before, after, new in ((case.k_pool, kp, case.k_new), (case.v_pool, vp, case.v_new)):
        changed = before != after
        assert changed.sum() == new.size
        assert np.all(before[changed] == dg.CANARY_BF16)
        np.testing.assert_array_equal(np.sort(after[changed]), np.sort(new.reshape(-1)))


def test_visible_pair_count_matches_paper_closed_form():
    """eq. (TTFT_derivation_2): sum_{i=i*}^{|T|} i = (|T| - i* + 1)(|T| + i*) / 2
    with i* = L + 1 (eq. (csr_i_star)) and |T| = L + n."""
    case = dg.make_case("pairs", dtype=dg.BF16, num_q_heads=2, num_kv_heads=1, head_dim=8, cache_len=[100, 0],
                        seqlen_q=[17, 25], page_size=16, seed=15, cfg_id=242)
    _, _, pairs = run_oracle(case)
    for b in range(2):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        T = int(case.cache_len[b]) + (hi - lo)
        istar = int(case.cache_len[b]) + 1
        for h in range(2):
            assert int(pairs[lo:hi, h].sum()) == (T - istar + 1) * (T + istar) // 2
    assert case.flops() == 4 * 8 * 2 * int(pairs[:, 0].sum())


def test_tolerance_gates_reject_zero_output():
    """At long prefixes |o| is small, so the max/mean-abs gates alone would pass
    an all-zero output; the relative Frobenius gate must reject it."""
    from tests.parity import check_bf16

    case = dg.make_case("gate", dtype=dg.BF16, num_q_heads=16, num_kv_heads=1, head_dim=128, cache_len=[122880],
                        seqlen_q=[2], page_size=16, scale=0.5, seed=16, cfg_id=243)
    out, lse, _ = run_oracle(case)
    ok, stats = check_bf16(np.zeros_like(out), lse, out, lse)
    assert stats["max_abs"] < 2e-2 and stats["mean_abs"] < 2e-3  # the plain gates pass...
    assert not ok  # ...the supplementary one does not
    ok2, _ = check_bf16(out.astype(np.float32), lse, out, lse)
    assert ok2
