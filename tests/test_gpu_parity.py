"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Every test feeds identical seeded inputs to both sides.  Small shapes are
checked on every output row (several row tiles, ragged tails, split-K forced);
the full-size workloads on seeded sampled rows.  Appends are compared bit for
bit over the whole pool.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, compare, from_dev, note, oracle_rows

pytestmark = pytest.mark.gpu


SMALL = [
    # (label, kwargs)
    ("f32_g4_d64", dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[300], seqlen_q=[70],
                        page_size=16)),
    ("f32_g2_d128", dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=2, head_dim=128, cache_len=[129],
                         seqlen_q=[33], page_size=8)),
    ("bf16_g16_d128", dict(dtype=dg.BF16, num_q_heads=32, num_kv_heads=2, head_dim=128, cache_len=[1000],
                           seqlen_q=[37], page_size=16, scale=0.5)),
    ("bf16_g8_d64", dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=1, head_dim=64, cache_len=[77],
                         seqlen_q=[100], page_size=4, scale=0.5)),
    ("bf16_g1_mha", dict(dtype=dg.BF16, num_q_heads=3, num_kv_heads=3, head_dim=128, cache_len=[64],
                         seqlen_q=[129], page_size=32, scale=0.5)),
    ("bf16_prefill_L0", dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=4, head_dim=128, cache_len=[0],
                             seqlen_q=[300], page_size=16, scale=0.5)),
    ("bf16_decode_n1", dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=1, head_dim=128, cache_len=[5000],
                            seqlen_q=[1], page_size=16, scale=0.5)),
    ("bf16_page1", dict(dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=128, cache_len=[95],
                        seqlen_q=[20], page_size=1, scale=0.5)),
    ("bf16_ragged", dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, cache_len=[0, 513, 64, 2049],
                         seqlen_q=[17, 1, 200, 64], page_size=16, scale=0.5, interleave=True)),
    ("f32_ragged", dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[31, 0, 200],
                        seqlen_q=[5, 40, 1], page_size=16, interleave=True)),
    # pages larger than a 64-key tile: the tile's offset inside the page is a separate term
    ("bf16_page128", dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, cache_len=[1000, 130],
                          seqlen_q=[50, 77], page_size=128, scale=0.5, interleave=True)),
    ("bf16_page1024_max", dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=1, head_dim=64, cache_len=[3000],
                               seqlen_q=[41], page_size=1024, scale=0.5)),
    # fp32 splits down to one key tile per split: 256 splits of a 20K prefix, merged by the
    # one-workgroup-per-row merge (fp32 output)
    ("f32_decode_long", dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[20000],
                             seqlen_q=[1], page_size=16)),
    ("f32_d128_long_ragged", dict(dtype=dg.F32, num_q_heads=8, num_kv_heads=2, head_dim=128, cache_len=[9000, 0, 3],
                                  seqlen_q=[2, 5, 70], page_size=16, interleave=True)),
]


@pytest.mark.parametrize("label,kw", SMALL, ids=[s[0] for s in SMALL])
@pytest.mark.parametrize("nsplit", [None, 3])
def test_small_shapes_all_rows(label, kw, nsplit):
    if nsplit:
        csr.set_plan_overrides(nsplit=nsplit)
    case = dg.make_case(label, seed=1, cfg_id=300, **kw)
    note(f"{label} nsplit={nsplit} L={case.cache_len.tolist()} n={case.seqlen_q.tolist()}: csr_extend_attention")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, f"{label}/split={nsplit}")


def test_c1_fp32_contiguous():
    case = dg.config("c1")
    note("c1 fp32 4q/1kv d64 L=1024 n=128 contiguous: csr_extend_attention")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, "c1")


def test_c2_bf16_paged_with_append():
    case = dg.config("c2")
    note("c2 bf16 64q/4kv d128 L=8192 n=256 P=16 permuted: csr_extend_attention(APPEND)")
    dev = Dev(case)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, "c2")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size)
    np.testing.assert_array_equal(from_dev(case, dev.k_pool), kp)
    np.testing.assert_array_equal(from_dev(case, dev.v_pool), vp)


@pytest.mark.parametrize("n", [512, 64, 128, 1024])
def test_c3_120k_prefix_sampled_rows(n):
    case = dg.config(f"c3_{n}")
    note(f"c3 bf16 L=122880 n={n}: csr_extend_attention")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 64, cfg_id=3)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, f"c3_{n}")


@pytest.mark.parametrize("n", [512, 1])
def test_tp4_share_of_c3_sampled_rows(n):
    # one GPU's share of C3 under 4-way head parallelism: 16 query heads on one kv head, the same
    # 120K prefix (the planner splits the single kv head's keys 8 ways at n = 512)
    case = dg.config(f"tp4_{n}")
    note(f"tp4 share bf16 16q/1kv L=122880 n={n}: csr_extend_attention(APPEND)")
    dev = Dev(case)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 64, cfg_id=6) if n > 1 else np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, f"tp4_{n}")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size)
    np.testing.assert_array_equal(from_dev(case, dev.k_pool), kp)
    np.testing.assert_array_equal(from_dev(case, dev.v_pool), vp)


@pytest.mark.parametrize("S", [61440, 122880])
def test_c4_reprefill_sampled_rows_and_cache_write(S):
    case = dg.config(f"c4_{S}")
    note(f"c4 bf16 prefill S={S}: csr_prefill (with cache write)")
    dev = Dev(case)
    out, lse = dev.prefill(write_cache=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 64, cfg_id=4)
    ref, ref_lse = oracle_rows(case, rows, prefill=True)
    compare(case, out, lse, rows, ref, ref_lse, f"c4_{S}")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, None, case.num_kv_heads, case.head_dim, case.page_size)
    np.testing.assert_array_equal(from_dev(case, dev.k_pool), kp)
    np.testing.assert_array_equal(from_dev(case, dev.v_pool), vp)


def test_c5_ragged_batch_with_append():
    case = dg.config("c5")
    note(f"c5 ragged L={case.cache_len.tolist()} n={case.seqlen_q.tolist()}: csr_extend_attention(APPEND)")
    dev = Dev(case)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 96, cfg_id=5)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, "c5")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size)
    np.testing.assert_array_equal(from_dev(case, dev.k_pool), kp)
    np.testing.assert_array_equal(from_dev(case, dev.v_pool), vp)


# Short chunks (decode-like: at most 128 packed rows per unit), where most
# waves of a workgroup hold only padding rows and skip the products.
DECODE = [
    ("decode_ragged_append", dict(dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128,
                                  cache_len=[4096, 17, 1000, 333], seqlen_q=[1, 8, 3, 5], page_size=16, scale=0.5,
                                  interleave=True)),
    ("decode_d64_pages4", dict(dtype=dg.BF16, num_q_heads=32, num_kv_heads=4, head_dim=64, cache_len=[2000, 64],
                               seqlen_q=[2, 16], page_size=4, scale=0.5)),
    ("decode_g2_rows40", dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=4, head_dim=128, cache_len=[700, 0, 95],
                              seqlen_q=[20, 7, 1], page_size=8, scale=0.5)),
    # ragged decode batches over small and large pages
    ("decode_d64_ragged", dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=64, cache_len=[3000, 100, 0, 33],
                              seqlen_q=[1, 8, 3, 2], page_size=4, scale=0.5, interleave=True)),
    ("decode_n1_batch4", dict(dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=[9000, 64, 65, 1],
                             seqlen_q=[1, 1, 1, 1], page_size=16, scale=0.5, interleave=True)),
]


@pytest.mark.parametrize("label,kw", DECODE, ids=[d[0] for d in DECODE])
@pytest.mark.parametrize("nsplit", [None, 5, 16])
def test_short_chunks_all_rows(label, kw, nsplit):
    if nsplit:
        csr.set_plan_overrides(nsplit=nsplit)
    case = dg.make_case(label, seed=2, cfg_id=310, **kw)
    note(f"{label} nsplit={nsplit} L={case.cache_len.tolist()} n={case.seqlen_q.tolist()}")
    dev = Dev(case)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, f"{label}/split={nsplit}")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size)
    np.testing.assert_array_equal(from_dev(case, dev.k_pool), kp)
    np.testing.assert_array_equal(from_dev(case, dev.v_pool), vp)


@pytest.mark.parametrize("label,kw", DECODE, ids=[d[0] for d in DECODE])
def test_short_chunks_dma_issuers_do_not_change_results(label, kw):
    """Short chunks load K/V from the waves without rows; the loads land in the
    same places as when every wave loads, so the outputs are identical bits."""
    case = dg.make_case(label, seed=2, cfg_id=311, **kw)
    note(f"{label}: K/V loads from the upper waves vs from every wave")
    outs = []
    for all_waves in (False, True):
        with csr.plan_overrides(dma_all_waves=all_waves):
            out, lse = Dev(case).extend()
            torch.cuda.synchronize()
        outs.append((out.view(torch.int16).cpu(), lse.cpu()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("n", [1, 8])
def test_c3_decode_120k_prefix_all_rows(n):
    case = dg.config(f"c3_{n}")
    note(f"c3 bf16 L=122880 n={n} (decode-like chunk): csr_extend_attention")
    dev = Dev(case)
    out, lse = dev.extend()
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rows(case, rows)
    compare(case, out, lse, rows, ref, ref_lse, f"c3_{n}")
