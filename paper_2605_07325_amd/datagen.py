"""Seeded synthetic inputs for the extend-attention path.

This module holds no attention arithmetic: it draws random numbers, rounds them
to the storage type, and lays the cached prefix out in the paged pool the way
the library's contract defines (pool[num_pages][P][Hkv][d]; position t of
sequence b lives in slot block_table[b][t // P] * P + t % P).  Both the GPU
tests and the CPU oracle consume exactly these arrays.

Shapes follow the paper's workloads: a static prefix of N cached tokens reused
across tasks and a freshly computed dynamic part of M tokens (Sec. IV-A, prompt
construction; N up to 120K and M up to 8192 in the latency sweep), plus the
eviction-time re-prefill of the compacted history (Algorithm 1, warm-up; the
experiments evict the oldest half at 110K tokens).  Values are i.i.d. normal,
scaled, then rounded to bf16 with round-to-nearest-even.  One more family holds
one GPU's share of the 120K-prefix workload when its kv heads are split over
four GPUs (16 query heads on one kv head).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

BF16, F32 = "bf16", "f32"

# bf16 NaN with all payload bits set: marks pool slots that hold no token yet.
CANARY_BF16 = np.uint16(0xFFFF)
CANARY_F32 = np.uint32(0xFFFFFFFF)


# e4m3 NaN (S.1111.111): marks slots of an fp8 pool that hold no token yet.
CANARY_FP8 = np.uint8(0xFF)


def fp8_codes(g: np.random.Generator, shape, exp_lo: int = 3, exp_hi: int = 9) -> np.ndarray:
    """Random OCP e4m3 bit patterns (uint8): random sign and mantissa, biased
    exponent field uniform in [exp_lo, exp_hi], so magnitudes lie in
    [2^(exp_lo-7), 2^(exp_hi-6)) before the pool's scale; never NaN."""
    sign = g.integers(0, 2, size=shape, dtype=np.uint8) << 7
    expo = g.integers(exp_lo, exp_hi + 1, size=shape, dtype=np.uint8) << 3
    mant = g.integers(0, 8, size=shape, dtype=np.uint8)
    return (sign | expo | mant).astype(np.uint8)


def with_fp8_pools(case: "Case", cfg_id: int = 0) -> "Case":
    """The same workload with e4m3 pools: every slot that holds a prefix
    token gets random codes (``fp8_codes``), every other slot the NaN canary.
    The chunk's K/V stay in the case's input type."""
    import dataclasses
    P = case.page_size
    shape = case.k_pool.shape
    k8 = np.full(shape, CANARY_FP8, np.uint8)
    v8 = np.full(shape, CANARY_FP8, np.uint8)
    for b in range(case.batch):
        L = int(case.cache_len[b])
        if L == 0:
            continue
        t = np.arange(L, dtype=np.int64)
        page = (case.block_table[b, t // P].astype(np.int64) if case.block_table is not None
                else b * case.bt_stride + t // P)
        slots = page * P + t % P
        k8.reshape(-1, shape[2], shape[3])[slots] = fp8_codes(rng(case.seed, cfg_id, 300 + 2 * b), (L, shape[2], shape[3]))
        v8.reshape(-1, shape[2], shape[3])[slots] = fp8_codes(rng(case.seed, cfg_id, 301 + 2 * b), (L, shape[2], shape[3]))
    return dataclasses.replace(case, k_pool=k8, v_pool=v8, k_prefix=None, v_prefix=None)


def rng(seed: int, cfg_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, cfg_id, tensor_id])))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even (torch's CPU cast)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def normal(g: np.random.Generator, shape, scale: float, dtype: str) -> np.ndarray:
    x = g.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return to_bf16_bits(x) if dtype == BF16 else x


@dataclasses.dataclass
class Case:
    name: str
    dtype: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    cache_len: np.ndarray  # int32 [B]
    seqlen_q: np.ndarray  # int32 [B]
    cu_seqlens_q: np.ndarray  # int32 [B+1]
    q: np.ndarray  # [T_q, Hq, d]  (uint16 bf16 bits or float32)
    k_new: np.ndarray  # [T_q, Hkv, d]
    v_new: np.ndarray
    k_pool: np.ndarray  # [num_pages, P, Hkv, d]
    v_pool: np.ndarray
    block_table: Optional[np.ndarray]  # int32 [B, bt_stride], -1 = unused; None = identity
    bt_stride: int
    seed: int = 0
    # logical (unpaged) prefixes [L_b, Hkv, d] per sequence, kept only on request
    k_prefix: Optional[list] = None
    v_prefix: Optional[list] = None

    @property
    def batch(self) -> int:
        return int(self.cache_len.shape[0])

    @property
    def total_q(self) -> int:
        return int(self.cu_seqlens_q[-1])

    @property
    def max_seqlen_q(self) -> int:
        return int(self.seqlen_q.max()) if self.batch else 0

    @property
    def max_cache_len(self) -> int:
        return int(self.cache_len.max()) if self.batch else 0

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == BF16 else 4

    def flops(self) -> int:
        """4 d Hq per visible (query, key) pair: QK^T and PV multiply-adds."""
        n = self.seqlen_q.astype(np.int64)
        L = self.cache_len.astype(np.int64)
        pairs = int(np.sum(n * L + n * (n + 1) // 2))
        return 4 * self.head_dim * self.num_q_heads * pairs

    def algorithmic_bytes(self, append: bool = True, kv_bytes: Optional[int] = None) -> int:
        """K/V read once, Q read, O written, chunk K/V appended (K/V elements
        of ``kv_bytes`` each, default the input type's)."""
        e, d, hq, hkv = self.elem_bytes, self.head_dim, self.num_q_heads, self.num_kv_heads
        ekv = e if kv_bytes is None else kv_bytes
        n = self.seqlen_q.astype(np.int64)
        L = self.cache_len.astype(np.int64)
        kv = int(np.sum(2 * hkv * d * ekv * (L + n)))
        qo = int(np.sum(2 * hq * d * e * n))
        ap = int(np.sum(2 * hkv * d * ekv * n)) if append else 0
        return kv + qo + ap


def _place_prefix(pool: np.ndarray, prefix: np.ndarray, table_row: Optional[np.ndarray], b: int,
                  bt_stride: int, P: int) -> None:
    L = prefix.shape[0]
    if L == 0:
        return
    t = np.arange(L, dtype=np.int64)
    page = table_row[t // P].astype(np.int64) if table_row is not None else b * bt_stride + t // P
    slots = page * P + t % P
    flat = pool.reshape(-1, pool.shape[2], pool.shape[3])
    flat[slots] = prefix


def make_case(name: str, *, dtype: str, num_q_heads: int, num_kv_heads: int, head_dim: int,
              cache_len, seqlen_q, page_size: int = 16, scale: float = 1.0, seed: int = 0,
              cfg_id: int = 0, paged: bool = True, interleave: bool = False,
              spare_pages: int = 0, keep_prefix: bool = False, fill: bool = True) -> Case:
    """Build one workload.

    ``paged=False`` gives the contiguous cache (identity table: sequence b owns
    pages b*bt_stride .. ).  With ``paged=True`` every sequence gets
    ceil((L_b + n_b) / P) pages; ``interleave`` deals page ids round-robin over
    (page index, sequence) before a seeded permutation of the pool, otherwise
    one seeded permutation is drawn per table.  Slots that hold no prefix token
    carry a NaN canary.  ``fill=False`` draws the layout only (lengths, page
    table): the value arrays are then read-only zero-stride views of the right
    shapes, for callers that draw the values elsewhere.
    """
    L = np.asarray(cache_len, dtype=np.int32).reshape(-1)
    n = np.asarray(seqlen_q, dtype=np.int32).reshape(-1)
    assert L.shape == n.shape
    B = int(L.shape[0])
    P = page_size
    hq, hkv, d = num_q_heads, num_kv_heads, head_dim
    cu = np.zeros(B + 1, np.int32)
    cu[1:] = np.cumsum(n)
    T = int(cu[-1])
    pages_per_seq = [int(math.ceil((int(L[b]) + int(n[b])) / P)) for b in range(B)]
    bt_stride = max(1, max(pages_per_seq) if B else 1)
    if paged:
        num_pages = sum(pages_per_seq) + spare_pages
        table = np.full((B, bt_stride), -1, np.int32)
        if interleave:
            ids = []
            for j in range(bt_stride):
                for b in range(B):
                    if j < pages_per_seq[b]:
                        ids.append((b, j))
            perm = rng(seed, cfg_id, 90).permutation(num_pages)
            for k, (b, j) in enumerate(ids):
                table[b, j] = perm[k]
        else:
            perm = rng(seed, cfg_id, 90).permutation(num_pages)
            k = 0
            for b in range(B):
                table[b, : pages_per_seq[b]] = perm[k:k + pages_per_seq[b]]
                k += pages_per_seq[b]
    else:
        num_pages = B * bt_stride
        table = None
    store = np.uint16 if dtype == BF16 else np.float32
    if not fill:
        def shaped(shape):
            return np.broadcast_to(np.zeros((), store), shape)
        return Case(name, dtype, hq, hkv, d, P, L, n, cu, shaped((T, hq, d)), shaped((T, hkv, d)),
                    shaped((T, hkv, d)), shaped((num_pages, P, hkv, d)), shaped((num_pages, P, hkv, d)), table,
                    bt_stride, seed)
    canary = CANARY_BF16 if dtype == BF16 else CANARY_F32.view(np.float32)
    k_pool = np.full((num_pages, P, hkv, d), canary, dtype=store)
    v_pool = np.full((num_pages, P, hkv, d), canary, dtype=store)
    kept_k, kept_v = ([], []) if keep_prefix else (None, None)
    for b in range(B):
        kp = normal(rng(seed, cfg_id, 100 + 2 * b), (int(L[b]), hkv, d), scale, dtype)
        vp = normal(rng(seed, cfg_id, 101 + 2 * b), (int(L[b]), hkv, d), scale, dtype)
        row = table[b] if table is not None else None
        _place_prefix(k_pool, kp, row, b, bt_stride, P)
        _place_prefix(v_pool, vp, row, b, bt_stride, P)
        if keep_prefix:
            kept_k.append(kp)
            kept_v.append(vp)
    q = normal(rng(seed, cfg_id, 1), (T, hq, d), scale, dtype)
    k_new = normal(rng(seed, cfg_id, 2), (T, hkv, d), scale, dtype)
    v_new = normal(rng(seed, cfg_id, 3), (T, hkv, d), scale, dtype)
    return Case(name, dtype, hq, hkv, d, P, L, n, cu, q, k_new, v_new, k_pool, v_pool, table,
                bt_stride, seed, kept_k, kept_v)


def sample_rows(case: Case, count: int, seed: int = 0, cfg_id: int = 0) -> np.ndarray:
    """Seeded query tokens to check: the first and last token of every sequence
    plus random ones, ``count`` in total (or every token if there are fewer)."""
    T = case.total_q
    if count >= T:
        return np.arange(T, dtype=np.int32)
    must = set()
    for b in range(case.batch):
        if case.seqlen_q[b] > 0:
            must.add(int(case.cu_seqlens_q[b]))
            must.add(int(case.cu_seqlens_q[b + 1]) - 1)
    g = rng(seed, cfg_id, 77)
    rest = [int(x) for x in g.permutation(T) if int(x) not in must]
    chosen = sorted(must | set(rest[: max(0, count - len(must))]))
    return np.asarray(chosen, dtype=np.int32)


# The workload families (sizes from the paper's sweeps; see module doc).
def config(cfg: str, seed: int = 0, **over) -> Case:
    if cfg == "c1":  # fp32 single layer, contiguous cache
        kw = dict(dtype=F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[1024],
                  seqlen_q=[128], scale=1.0, paged=False, cfg_id=1)
    elif cfg == "c2":  # bf16 GQA 64/4, 8K prefix, 256-token chunk, paged
        kw = dict(dtype=BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=[8192],
                  seqlen_q=[256], scale=0.5, cfg_id=2)
    elif cfg.startswith("c3"):  # 120K prefix; chunk n from the name, default 512
        nq = int(cfg.split("_")[1]) if "_" in cfg else 512
        kw = dict(dtype=BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=[122880],
                  seqlen_q=[nq], scale=0.5, cfg_id=3)
    elif cfg.startswith("tp4"):  # one GPU's share of C3 under 4-way head parallelism: 16q / 1kv, chunk n from the name
        nq = int(cfg.split("_")[1]) if "_" in cfg else 512
        kw = dict(dtype=BF16, num_q_heads=16, num_kv_heads=1, head_dim=128, cache_len=[122880],
                  seqlen_q=[nq], scale=0.5, cfg_id=6)
    elif cfg.startswith("c4"):  # re-prefill of the compacted history, L = 0
        S = int(cfg.split("_")[1]) if "_" in cfg else 61440
        kw = dict(dtype=BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=[0],
                  seqlen_q=[S], scale=0.5, cfg_id=4)
    elif cfg == "c5":  # ragged batch of 8, interleaved pages
        g = rng(seed, 5, 50)
        L = g.integers(4096, 122880 + 1, size=8)
        n = g.integers(64, 1024 + 1, size=8)
        kw = dict(dtype=BF16, num_q_heads=64, num_kv_heads=4, head_dim=128, cache_len=L,
                  seqlen_q=n, scale=0.5, cfg_id=5, interleave=True)
    else:
        raise KeyError(cfg)
    kw.update(over)
    return make_case(cfg, seed=seed, **kw)
