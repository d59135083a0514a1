"""GPU parity for the FP8 (OCP e4m3) KV cache and the fp8 score products.

The cache holds e4m3 codes with per-tensor scales; the chunk's bf16 keys and
values are quantised by the fused prep launch (and appended); the attention
converts codes to bf16 exactly and computes as the bf16 path does.  The
oracle evaluates the same definition in fp64 (codes decoded exactly, chunk
quantised by its own encoder), so outputs meet the bf16 gates and appended
codes are compared bit for bit (with RoPE both sides rotate in fp64 and
quantise the fp32 rounding of the result).  In the fp8-
product mode (q_scale) the query is quantised by the same rule, on the GPU by
the prep launch and in the oracle by its own encoder, and the scores run on
the fp8 matrix cores; the outputs meet the same gates.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, compare, note, values

pytestmark = pytest.mark.gpu

KS, VS = 0.0625, 0.0390625
QS = 0.015625  # q_scale of the fp8-product runs (|q| / QS stays well inside 448 for these inputs)


class Dev8(Dev):
    """Device copies of an fp8-cache case (uint8 pools) and its descriptor."""

    def __init__(self, case, rope=None, q8=False):
        super().__init__(case)
        self.k_pool = torch.from_numpy(case.k_pool).cuda()
        self.v_pool = torch.from_numpy(case.v_pool).cuda()
        self.desc.kv_dtype = csr.CSR_KV_FP8_E4M3
        self.desc.k_scale, self.desc.v_scale = KS, VS
        if q8:
            self.desc.q_scale = QS
        if rope is not None:
            self.desc.rope_style, self.desc.rope_dim, self.desc.rope_theta = rope


def fp8_case(label, cfg_id, **kw):
    return dg.with_fp8_pools(dg.make_case(label, dtype=dg.BF16, head_dim=128, seed=3, cfg_id=cfg_id, **kw),
                             cfg_id=cfg_id)


def oracle8(case, rows, rope=None, prefill=False, q8=False):
    out, lse, _ = oracle.attention(oracle.BF16, case.q, case.k_new, case.v_new, case.k_pool, case.v_pool,
                                   case.block_table, case.bt_stride, case.cu_seqlens_q,
                                   None if prefill else case.cache_len, rows, case.num_q_heads, case.num_kv_heads,
                                   case.head_dim, case.page_size, rope=rope, fp8=(KS, VS), q_fp8=QS if q8 else None)
    return out, lse


def check_pool8(case, dev, cache_len, rope=None):
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, cache_len, case.num_kv_heads, case.head_dim, case.page_size,
                              rope=rope, fp8=(KS, VS))
    gk, gv = dev.k_pool.cpu().numpy(), dev.v_pool.cpu().numpy()
    assert np.array_equal(gv, vp), "values (and every untouched byte) must match bit for bit"
    differ = int(np.count_nonzero(gk != kp))
    assert differ == 0, f"{differ} key codes differ from the oracle's"
    note(f"fp8 pool{' with RoPE' if rope is not None else ''}: codes bit for bit")


SMALL = [
    ("g16_L1000", dict(num_q_heads=32, num_kv_heads=2, cache_len=[1000], seqlen_q=[37], page_size=16, scale=0.5)),
    ("ragged_empty", dict(num_q_heads=16, num_kv_heads=2, cache_len=[0, 513, 64, 2049, 300], seqlen_q=[17, 1, 0, 64, 9],
                          page_size=16, scale=0.5, interleave=True)),
    ("page4", dict(num_q_heads=8, num_kv_heads=1, cache_len=[777], seqlen_q=[100], page_size=4, scale=0.5)),
    ("prefill_L0", dict(num_q_heads=16, num_kv_heads=4, cache_len=[0], seqlen_q=[300], page_size=16, scale=0.5)),
    ("decode_n1", dict(num_q_heads=16, num_kv_heads=1, cache_len=[5000], seqlen_q=[1], page_size=16, scale=0.5)),
    ("page1024", dict(num_q_heads=16, num_kv_heads=2, cache_len=[2500, 900], seqlen_q=[30, 64], page_size=1024,
                      scale=0.5, interleave=True)),
    # at most 128 packed rows per sequence: the 4-wave workgroups
    ("decode_ragged", dict(num_q_heads=32, num_kv_heads=4, cache_len=[0, 1, 4097, 300, 65], seqlen_q=[16, 1, 3, 0, 7],
                           page_size=16, scale=0.5, interleave=True)),
    ("decode_page4", dict(num_q_heads=16, num_kv_heads=2, cache_len=[777, 64], seqlen_q=[2, 8], page_size=4,
                          scale=0.5)),
    # ragged decode batch, pages smaller than a DMA block
    ("decode_ragged_page4", dict(num_q_heads=16, num_kv_heads=4, cache_len=[5000, 1, 700, 0], seqlen_q=[8, 1, 3, 5],
                          page_size=4, scale=0.5, interleave=True)),
]


@pytest.mark.parametrize("q8", [False, True], ids=["bf16_scores", "fp8_scores"])
@pytest.mark.parametrize("label,kw", SMALL, ids=[s[0] for s in SMALL])
@pytest.mark.parametrize("nsplit", [None, 3])
def test_fp8_extend_append_all_rows(label, kw, nsplit, q8):
    if nsplit:
        csr.set_plan_overrides(nsplit=nsplit)
    case = fp8_case(label, 600, **kw)
    note(f"fp8 {label} nsplit={nsplit} q8={q8} L={case.cache_len.tolist()} n={case.seqlen_q.tolist()}: "
         "csr_extend_attention(APPEND)")
    dev = Dev8(case, q8=q8)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle8(case, rows, q8=q8)
    compare(case, out, lse, rows, ref, ref_lse, f"fp8/{label}/split={nsplit}/q8={q8}")
    check_pool8(case, dev, case.cache_len)


def test_fp8_kv_append_alone():
    case = fp8_case("append", 601, num_q_heads=16, num_kv_heads=2, cache_len=[40, 700], seqlen_q=[70, 5],
                    page_size=16, scale=0.5, interleave=True)
    note("fp8 csr_kv_append")
    dev = Dev8(case)
    dev.append()
    torch.cuda.synchronize()
    check_pool8(case, dev, case.cache_len)


@pytest.mark.parametrize("q8", [False, True], ids=["bf16_scores", "fp8_scores"])
@pytest.mark.parametrize("n", [[90], [1, 2, 1]], ids=["chunk90", "decode"])
@pytest.mark.parametrize("style", [csr.CSR_ROPE_NEOX, csr.CSR_ROPE_INTERLEAVED])
def test_fp8_with_rope(style, n, q8):
    L = [3000] if len(n) == 1 else [3000, 64, 777]
    case = fp8_case("rope8", 602, num_q_heads=16, num_kv_heads=2, cache_len=L, seqlen_q=n, page_size=16,
                    scale=0.5, interleave=len(n) > 1)
    rope = (style, 0, 1e6)
    note(f"fp8 + rope style {style}, L={L} n={n} q8={q8}: csr_extend_attention(APPEND)")
    dev = Dev8(case, rope, q8=q8)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle8(case, rows, rope=rope, q8=q8)
    compare(case, out, lse, rows, ref, ref_lse, f"fp8/rope{style}")
    check_pool8(case, dev, case.cache_len, rope=rope)


@pytest.mark.parametrize("q8", [False, True], ids=["bf16_scores", "fp8_scores"])
@pytest.mark.parametrize("n", [512, 1])
def test_fp8_c3_120k_prefix(n, q8):
    base = dg.config(f"c3_{n}")
    case = dg.with_fp8_pools(base, cfg_id=603)
    note(f"fp8 c3 L=122880 n={n} q8={q8}: csr_extend_attention(APPEND)")
    dev = Dev8(case, q8=q8)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 64, cfg_id=3)
    ref, ref_lse = oracle8(case, rows, q8=q8)
    compare(case, out, lse, rows, ref, ref_lse, f"fp8/c3_{n}/q8={q8}")
    check_pool8(case, dev, case.cache_len)


def test_fp8_chunk_split_on_device():
    """extend(L, n1) + append, then extend(L + n1, n2) over that cache, equals
    extend(L, n1 + n2): a chunk key is quantised once, the same both ways."""
    L, n1, n2 = 2500, 120, 77
    kw = dict(num_q_heads=16, num_kv_heads=2, page_size=16, scale=0.5)
    one = fp8_case("one8", 604, cache_len=[L], seqlen_q=[n1 + n2], **kw)
    note(f"fp8 chunk split L={L} n={n1}+{n2}")
    dev_one = Dev8(one)
    out_one, lse_one = dev_one.extend()
    a = fp8_case("one8", 604, cache_len=[L], seqlen_q=[n1], **kw)
    for f in ("q", "k_new", "v_new"):
        getattr(a, f)[:] = getattr(one, f)[:n1]
    a.k_pool, a.v_pool, a.block_table, a.bt_stride = one.k_pool, one.v_pool, one.block_table, one.bt_stride
    dev_a = Dev8(a)
    out_a, _ = dev_a.extend(append=True)
    b = fp8_case("one8", 604, cache_len=[L + n1], seqlen_q=[n2], **kw)
    for f in ("q", "k_new", "v_new"):
        getattr(b, f)[:] = getattr(one, f)[n1:]
    b.block_table, b.bt_stride = one.block_table, one.bt_stride
    dev_b = Dev8(b)
    dev_b.k_pool, dev_b.v_pool = dev_a.k_pool, dev_a.v_pool
    out_b, lse_b = dev_b.extend()
    torch.cuda.synchronize()
    assert np.abs(values(a, out_a) - values(one, out_one)[:n1]).max() < 1e-2
    assert np.abs(values(b, out_b) - values(one, out_one)[n1:]).max() < 1e-2
    assert np.abs(lse_b.cpu().numpy() - lse_one.cpu().numpy()[n1:]).max() < 1e-4


@pytest.mark.parametrize("q8", [False, True], ids=["bf16_scores", "fp8_scores"])
def test_fp8_prefill_writes_the_quantised_cache(q8):
    case = fp8_case("pf8", 605, num_q_heads=16, num_kv_heads=2, cache_len=[0], seqlen_q=[2600], page_size=16,
                    scale=0.5)
    note(f"fp8 csr_prefill with cache write, q8={q8}")
    dev = Dev8(case, q8=q8)
    out, lse = dev.prefill(write_cache=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 48, cfg_id=6)
    ref, ref_lse = oracle8(case, rows, prefill=True, q8=q8)
    compare(case, out, lse, rows, ref, ref_lse, "fp8/prefill")
    check_pool8(case, dev, None)
