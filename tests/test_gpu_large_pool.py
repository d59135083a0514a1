"""GPU parity with pools larger than 4 GB: the pages a case uses sit at the end
of a 5.4 GB pool, so every K/V address and every appended row lies beyond
32-bit byte offsets.  The oracle runs the same case on its compact pool (the
same tokens under the original block table); outputs meet the parity gates,
appended rows match bit for bit, and canary pages beside the used range stay
untouched."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import compare, note, to_dev

pytestmark = pytest.mark.gpu

KS, VS = 0.0625, 0.0390625
CASES = [("extend", [1500, 700], [40, 9]), ("decode", [3000, 17], [1, 3])]


def _dev_pool(small: np.ndarray, big: int, off: int, fp8: bool) -> torch.Tensor:
    """A device pool of `big` pages holding `small`'s pages at [off, off + len)
    and canary pages at off - 2, off - 1 (the rest is never touched)."""
    if fp8:
        t = torch.empty((big,) + small.shape[1:], dtype=torch.uint8, device="cuda")
        t[off - 2:off].fill_(int(dg.CANARY_FP8))
        t[off:] = torch.from_numpy(small).cuda()
        return t
    t = torch.empty((big,) + small.shape[1:], dtype=torch.bfloat16, device="cuda")
    t[off - 2:off].view(torch.int16).fill_(-1)
    t[off:] = torch.from_numpy(small.view(np.int16)).cuda().view(torch.bfloat16)
    return t


def _host(t: torch.Tensor, fp8: bool) -> np.ndarray:
    return t.cpu().numpy() if fp8 else t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("label,L,n", CASES, ids=[c[0] for c in CASES])
def test_pages_beyond_4gb(kv, label, L, n):
    fp8 = kv == "fp8"
    case = dg.make_case(f"big_{label}", dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, cache_len=L,
                        seqlen_q=n, page_size=16, scale=0.5, seed=5, cfg_id=330, interleave=True)
    if fp8:
        case = dg.with_fp8_pools(case, cfg_id=330)
    pages = case.k_pool.shape[0]
    page_bytes = case.k_pool[0].nbytes
    big = (5 << 30) // page_bytes + pages + 2
    off = big - pages
    note(f"large pool {kv} {label}: {big} pages of {page_bytes} B ({big * page_bytes / 2**30:.2f} GiB per pool), "
         f"used pages at {off}..{big - 1}")
    kb, vb = _dev_pool(case.k_pool, big, off, fp8), _dev_pool(case.v_pool, big, off, fp8)
    bt = case.block_table.copy()
    bt[bt >= 0] += off
    desc = csr.make_desc(case.num_q_heads, case.num_kv_heads, case.head_dim, case.page_size)
    if fp8:
        desc.kv_dtype, desc.k_scale, desc.v_scale = csr.CSR_KV_FP8_E4M3, KS, VS
    q, kn, vn = (to_dev(case, a) for a in (case.q, case.k_new, case.v_new))
    cu = torch.from_numpy(case.cu_seqlens_q).cuda()
    cl = torch.from_numpy(case.cache_len).cuda()
    out, lse = csr.extend_attention(desc, q, kn, vn, kb, vb, torch.from_numpy(bt).cuda(), case.bt_stride, cu, cl,
                                    case.max_seqlen_q, case.max_cache_len, append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    fp8_arg = (KS, VS) if fp8 else None
    ref, ref_lse, _ = oracle.attention(oracle.BF16, case.q, case.k_new, case.v_new, case.k_pool, case.v_pool,
                                       case.block_table, case.bt_stride, case.cu_seqlens_q, case.cache_len, rows,
                                       case.num_q_heads, case.num_kv_heads, case.head_dim, case.page_size, fp8=fp8_arg)
    compare(case, out, lse, rows, ref, ref_lse, f"large pool {kv} {label}")
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size,
                              fp8=fp8_arg)
    assert np.array_equal(_host(kb[off:], fp8), kp), "appended keys (or untouched bytes) differ"
    assert np.array_equal(_host(vb[off:], fp8), vp), "appended values (or untouched bytes) differ"
    canary = dg.CANARY_FP8 if fp8 else dg.CANARY_BF16
    assert np.all(_host(kb[off - 2:off], fp8) == canary) and np.all(_host(vb[off - 2:off], fp8) == canary)
