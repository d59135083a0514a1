"""GPU test of csr_extend_attention_noalloc, the entry point for callers that
cannot allocate: through the C ABI, its outputs (and, with CSR_APPEND, the
cache) must equal csr_extend_attention's bit for bit on the same inputs, on
two calls in a row (the second smaller, so the shared scratch array holds the
first call's leftovers), and a call needing more scratch than the array holds
must be refused."""
import numpy as np
import pytest
import torch

from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, note

pytestmark = pytest.mark.gpu


def run_both(case, append):
    a, b = Dev(case), Dev(case)
    c = case
    note(f"no-alloc vs workspace: L={c.cache_len.tolist()} n={c.seqlen_q.tolist()} append={append}")
    out_ws, lse_ws = a.extend(append=append)
    out_na, lse_na = csr.extend_attention_noalloc(b.desc, b.q, b.k_new, b.v_new, b.k_pool, b.v_pool, b.bt,
                                                  c.bt_stride, b.cu, b.cache_len, c.max_seqlen_q, c.max_cache_len,
                                                  append=append)
    torch.cuda.synchronize()
    assert torch.equal(out_ws.view(torch.int16), out_na.view(torch.int16))
    assert torch.equal(lse_ws.view(torch.int32), lse_na.view(torch.int32))
    assert torch.equal(a.k_pool.view(torch.int16), b.k_pool.view(torch.int16))
    assert torch.equal(a.v_pool.view(torch.int16), b.v_pool.view(torch.int16))


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    big = dg.make_case("noalloc_big", dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128,
                       cache_len=[8192], seqlen_q=[256], page_size=16, scale=0.5, seed=7, cfg_id=700)
    need = csr.extend_workspace_size(Dev(big).desc, 1, big.total_q, big.max_seqlen_q, big.max_cache_len)
    assert 0 < need <= csr.CSR_NOALLOC_SCRATCH_BYTES
    run_both(big, append=True)
    small = dg.make_case("noalloc_small", dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128,
                         cache_len=[3000, 513], seqlen_q=[3, 1], page_size=16, scale=0.5, seed=8, cfg_id=701,
                         interleave=True)
    run_both(small, append=True)


def test_noalloc_refuses_calls_beyond_its_scratch():
    """With RoPE the workspace also holds the rotated q of every chunk token: 4096 tokens x 64
    heads x 128 bf16 alone are 64 MiB, more than the array."""
    case = dg.make_case("noalloc_over", dtype=dg.BF16, num_q_heads=64, num_kv_heads=4, head_dim=128,
                        cache_len=[64], seqlen_q=[16], page_size=16, scale=0.5, seed=9, cfg_id=702)
    dev = Dev(case)
    dev.desc.rope_style, dev.desc.rope_theta = csr.CSR_ROPE_NEOX, 1e6
    total = 4096
    need = csr.extend_workspace_size(dev.desc, 2, total, 2048, 64)
    assert need > csr.CSR_NOALLOC_SCRATCH_BYTES
    cu = torch.tensor([0, 2048, total], dtype=torch.int32, device="cuda")
    q = torch.zeros((total, 64, 128), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((total, 4, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(csr.CsrError) as err:
        csr.extend_attention_noalloc(dev.desc, q, kv, kv, dev.k_pool, dev.v_pool, dev.bt, case.bt_stride, cu,
                                     torch.zeros(2, dtype=torch.int32, device="cuda"), 2048, 64)
    assert err.value.status == csr.CSR_E_WORKSPACE
    note(f"no-alloc refuses a call needing {need} bytes of scratch")
