"""Glue between seeded cases, the HIP library (through the C ABI) and the oracle.

Nothing here computes attention: it uploads inputs, calls the binding, calls
the oracle on the same inputs and hands both results to the parity gates.
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

from oracle import oracle
from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.parity import check_bf16, check_f32


def note(msg: str) -> None:
    print(f"[gpu-test {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def to_dev(case: dg.Case, a: np.ndarray) -> torch.Tensor:
    if case.dtype == dg.BF16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def from_dev(case: dg.Case, t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy in the storage format the oracle reads."""
    if case.dtype == dg.BF16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def values(case: dg.Case, t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class Dev:
    """Device copies of a case."""

    def __init__(self, case: dg.Case):
        self.case = case
        self.q = to_dev(case, case.q)
        self.k_new = to_dev(case, case.k_new)
        self.v_new = to_dev(case, case.v_new)
        self.k_pool = to_dev(case, case.k_pool)
        self.v_pool = to_dev(case, case.v_pool)
        self.bt = None if case.block_table is None else torch.from_numpy(case.block_table).cuda()
        self.cu = torch.from_numpy(case.cu_seqlens_q).cuda()
        self.cache_len = torch.from_numpy(case.cache_len).cuda()
        self.desc = csr.make_desc(case.num_q_heads, case.num_kv_heads, case.head_dim, case.page_size,
                                  torch.bfloat16 if case.dtype == dg.BF16 else torch.float32)

    def extend(self, append: bool = False, **kw):
        c = self.case
        return csr.extend_attention(self.desc, self.q, self.k_new, self.v_new, self.k_pool, self.v_pool, self.bt,
                                    c.bt_stride, self.cu, self.cache_len, c.max_seqlen_q, c.max_cache_len,
                                    append=append, **kw)

    def prefill(self, write_cache: bool = True, **kw):
        c = self.case
        if write_cache:
            return csr.prefill(self.desc, self.q, self.k_new, self.v_new, self.cu, c.max_seqlen_q,
                               k_pool=self.k_pool, v_pool=self.v_pool, block_table=self.bt, bt_stride=c.bt_stride,
                               **kw)
        return csr.prefill(self.desc, self.q, self.k_new, self.v_new, self.cu, c.max_seqlen_q, **kw)

    def append(self):
        c = self.case
        csr.kv_append(self.desc, self.k_new, self.v_new, self.k_pool, self.v_pool, self.bt, c.bt_stride, self.cu,
                      self.cache_len)


def oracle_rows(case: dg.Case, rows: np.ndarray, prefill: bool = False):
    out, lse, _ = oracle.attention(oracle.BF16 if case.dtype == dg.BF16 else oracle.F32, case.q, case.k_new,
                                   case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                                   case.cu_seqlens_q, None if prefill else case.cache_len, rows, case.num_q_heads,
                                   case.num_kv_heads, case.head_dim, case.page_size)
    return out, lse


def compare(case: dg.Case, out: torch.Tensor, lse: torch.Tensor, rows: np.ndarray, ref, ref_lse, label: str):
    idx = torch.from_numpy(rows.astype(np.int64)).cuda()
    got = values(case, out.index_select(0, idx))
    got_lse = None if lse is None else lse.index_select(0, idx).cpu().numpy().astype(np.float64)
    check = check_bf16 if case.dtype == dg.BF16 else check_f32
    ok, st = check(got, got_lse, ref, ref_lse)
    note(f"{label}: rows={len(rows)} {st}")
    assert ok, f"{label}: parity failed {st}"
    return st
