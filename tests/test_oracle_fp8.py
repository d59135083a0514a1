"""Pins for the oracle's FP8 (OCP e4m3) KV cache.

The paper's model is served in FP8; a cache of e4m3 codes with one
dequantisation scale per tensor is the storage convention here.  Independent
pins: torch's float8_e4m3fn conversions (a library routine) for every code and
for rounding, closed forms of the format, torch SDPA over values dequantised
by torch for the attention oracle, and the chunk-split identity (a chunk key
enters the attention exactly as it is cached).
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import datagen as dg


def torch_encode(x32):
    """torch's e4m3 conversion of fp32 values after the saturation the format convention adds."""
    t = torch.from_numpy(np.clip(np.asarray(x32, np.float32), -448, 448))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_torch_for_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ours = oracle.e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan) and nan.sum() == 2   # 0x7f and 0xff
    assert np.array_equal(ours[~nan], ref[~nan])


def test_format_closed_forms():
    dec = oracle.e4m3_decode(np.array([0x7E, 0xFE, 0x01, 0x08, 0x38, 0x00, 0x80, 0x07], np.uint8))
    assert list(dec[:2]) == [448.0, -448.0]
    assert dec[2] == 2.0 ** -9 and dec[3] == 2.0 ** -6 and dec[4] == 1.0
    assert dec[5] == 0.0 and math.copysign(1, dec[6]) == -1 and dec[7] == 7 * 2.0 ** -9
    enc = oracle.e4m3_encode(np.array([1e6, -1e6, 449.0, float("nan"), 0.0, -0.0], np.float32))
    assert list(enc) == [0x7E, 0xFE, 0x7E, 0x7F, 0x00, 0x80]


def test_encode_matches_torch():
    g = np.random.default_rng(0)
    mags = np.exp2(g.uniform(-14, 9.5, size=20000)).astype(np.float32)
    x = mags * np.where(g.random(20000) < 0.5, -1, 1).astype(np.float32)
    # exact midpoints between neighbouring codes (ties go to the even code)
    vals = oracle.e4m3_decode(np.arange(0, 0x7E, dtype=np.uint8))
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids, np.float32([2.0 ** -10, 3 * 2.0 ** -11, 2.0 ** -12])])
    assert np.array_equal(oracle.e4m3_encode(x), torch_encode(x))


SCALES = (0.0625, 0.0390625)


def torch_quant_dequant(x_bf16_bits, scale):
    """bf16 inputs -> fp32 product with fp32(1/scale) -> torch e4m3 -> exact value * scale."""
    x = dg.bf16_bits_to_f32(x_bf16_bits).astype(np.float32)
    inv = np.float32(1.0) / np.float32(scale)
    codes = torch_encode(x * inv)
    return torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy() * float(np.float32(scale))


QS = 0.015625  # q_scale of the fp8-product mode in these pins


@pytest.mark.parametrize("q_fp8", [None, QS], ids=["bf16_q", "fp8_q"])
@pytest.mark.parametrize("kw", [
    dict(num_q_heads=8, num_kv_heads=2, head_dim=32, cache_len=[37], seqlen_q=[11], page_size=4),
    dict(num_q_heads=6, num_kv_heads=3, head_dim=16, cache_len=[5, 0, 33], seqlen_q=[3, 7, 1], page_size=2,
         interleave=True),
])
def test_attention_over_an_fp8_cache_matches_sdpa(kw, q_fp8):
    case = dg.with_fp8_pools(dg.make_case("fp8", dtype=dg.BF16, scale=0.5, cfg_id=80, **kw), cfg_id=80)
    ks, vs = SCALES
    out, lse, _ = oracle.attention(oracle.BF16, case.q, case.k_new, case.v_new, case.k_pool, case.v_pool,
                                   case.block_table, case.bt_stride, case.cu_seqlens_q, case.cache_len,
                                   np.arange(case.total_q, dtype=np.int32), case.num_q_heads, case.num_kv_heads,
                                   case.head_dim, case.page_size, fp8=(ks, vs), q_fp8=q_fp8)
    G = case.num_q_heads // case.num_kv_heads
    P = case.page_size
    deq = lambda c, s: torch.from_numpy(c).view(torch.float8_e4m3fn).to(torch.float64).numpy() * float(np.float32(s))  # noqa: E731
    for b in range(case.batch):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        L, n = int(case.cache_len[b]), hi - lo
        if n == 0:
            continue
        t = np.arange(L)
        page = case.block_table[b, t // P].astype(np.int64)
        kp = case.k_pool[page, t % P]
        vp = case.v_pool[page, t % P]
        k = np.concatenate([deq(kp, ks), torch_quant_dequant(case.k_new[lo:hi], ks)], axis=0)
        v = np.concatenate([deq(vp, vs), torch_quant_dequant(case.v_new[lo:hi], vs)], axis=0)
        q = (dg.bf16_bits_to_f32(case.q[lo:hi]).astype(np.float64) if q_fp8 is None
             else torch_quant_dequant(case.q[lo:hi], q_fp8))
        qt = torch.from_numpy(q).permute(1, 0, 2)
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)
        mask = torch.arange(L + n)[None, :] <= (L + torch.arange(n))[:, None]
        sc = 1.0 / math.sqrt(case.head_dim)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=sc)
        s = (torch.matmul(qt, kt.transpose(1, 2)) * sc).masked_fill(~mask, float("-inf"))
        np.testing.assert_allclose(out[lo:hi], ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[lo:hi], torch.logsumexp(s, -1).permute(1, 0).numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("rope", [None, (oracle.ROPE_NEOX, 0, 1e4)])
def test_fp8_append_stores_the_quantised_chunk(rope):
    case = dg.with_fp8_pools(dg.make_case("fp8a", dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=32,
                                          cache_len=[20, 3], seqlen_q=[9, 14], page_size=4, scale=0.5, cfg_id=81),
                             cfg_id=81)
    ks, vs = SCALES
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim, case.page_size,
                              rope=rope, fp8=(ks, vs))
    touched = np.zeros(kp.shape[:2], bool)
    inv_k, inv_v = np.float32(1) / np.float32(ks), np.float32(1) / np.float32(vs)
    for b in range(case.batch):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        pos = int(case.cache_len[b]) + np.arange(hi - lo)
        slots = (case.block_table[b, pos // 4], pos % 4)
        touched[slots] = True
        k = dg.bf16_bits_to_f32(case.k_new[lo:hi]).astype(np.float64)
        if rope is not None:
            k = oracle.rope(k, pos, *rope)
        assert np.array_equal(kp[slots], torch_encode(k.astype(np.float32) * inv_k))
        assert np.array_equal(vp[slots], torch_encode(dg.bf16_bits_to_f32(case.v_new[lo:hi]) * inv_v))
    assert np.array_equal(kp[~touched], case.k_pool[~touched]) and np.array_equal(vp[~touched], case.v_pool[~touched])


@pytest.mark.parametrize("rope", [None, (oracle.ROPE_INTERLEAVED, 16, 1e4)])
def test_fp8_chunk_split_is_exact(rope):
    """A chunk key is quantised identically whether the attention reads it from
    the chunk or, after an append, from the cache: the split is bit for bit."""
    L, n1, n2 = 23, 6, 9
    kw = dict(dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=32, page_size=4, scale=0.5, cfg_id=82)
    whole = dg.with_fp8_pools(dg.make_case("w", cache_len=[L], seqlen_q=[n1 + n2], **kw), cfg_id=82)
    fp8 = SCALES
    args = (whole.num_q_heads, whole.num_kv_heads, whole.head_dim, whole.page_size)
    one, one_lse, _ = oracle.attention(oracle.BF16, whole.q, whole.k_new, whole.v_new, whole.k_pool, whole.v_pool,
                                       whole.block_table, whole.bt_stride, whole.cu_seqlens_q, whole.cache_len,
                                       np.arange(n1 + n2, dtype=np.int32), *args, rope=rope, fp8=fp8)
    cu1 = np.array([0, n1], np.int32)
    kp, vp = oracle.kv_append(whole.k_new[:n1], whole.v_new[:n1], whole.k_pool, whole.v_pool, whole.block_table,
                              whole.bt_stride, cu1, whole.cache_len, whole.num_kv_heads, whole.head_dim,
                              whole.page_size, rope=rope, fp8=fp8)
    second, second_lse, _ = oracle.attention(oracle.BF16, whole.q[n1:], whole.k_new[n1:], whole.v_new[n1:], kp, vp,
                                             whole.block_table, whole.bt_stride, np.array([0, n2], np.int32),
                                             np.array([L + n1], np.int32), np.arange(n2, dtype=np.int32), *args,
                                             rope=rope, fp8=fp8)
    assert np.array_equal(second, one[n1:]) and np.array_equal(second_lse, one_lse[n1:])


def test_fp8_products_quantise_the_rotated_query():
    """With RoPE the query is rotated first (fp64, then fp32 as the quantiser
    reads it) and then quantised like a key: the result equals SDPA over
    torch-quantised rotated queries and an unrotated-cache, rotated-chunk key set."""
    case = dg.with_fp8_pools(dg.make_case("fp8qr", dtype=dg.BF16, num_q_heads=4, num_kv_heads=2, head_dim=32,
                                          cache_len=[19], seqlen_q=[6], page_size=4, scale=0.5, cfg_id=83),
                             cfg_id=83)
    ks, vs = SCALES
    rope = (oracle.ROPE_NEOX, 0, 1e4)
    rows = np.arange(case.total_q, dtype=np.int32)
    args = (case.q, case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
            case.cu_seqlens_q, case.cache_len, rows, case.num_q_heads, case.num_kv_heads, case.head_dim,
            case.page_size)
    out, lse, _ = oracle.attention(oracle.BF16, *args, rope=rope, fp8=(ks, vs), q_fp8=QS)
    L, n, P, G = 19, 6, 4, 2
    pos = L + np.arange(n)
    q = oracle.rope(dg.bf16_bits_to_f32(case.q).astype(np.float64), pos, *rope)
    qd = torch.from_numpy(torch_encode(q.astype(np.float32) * (np.float32(1) / np.float32(QS)))).view(
        torch.float8_e4m3fn).to(torch.float64).numpy() * QS
    t = np.arange(L)
    page = case.block_table[0, t // P].astype(np.int64)
    deq = lambda c, sc: torch.from_numpy(c).view(torch.float8_e4m3fn).to(torch.float64).numpy() * float(np.float32(sc))  # noqa: E731
    kc = oracle.rope(dg.bf16_bits_to_f32(case.k_new).astype(np.float64), pos, *rope)
    kq = deq(torch_encode(kc.astype(np.float32) * (np.float32(1) / np.float32(ks))), ks)
    k = np.concatenate([deq(case.k_pool[page, t % P], ks), kq], axis=0)
    v = np.concatenate([deq(case.v_pool[page, t % P], vs), torch_quant_dequant(case.v_new, vs)], axis=0)
    qt = torch.from_numpy(qd).permute(1, 0, 2)
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)
    mask = torch.arange(L + n)[None, :] <= (L + torch.arange(n))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=1 / math.sqrt(32))
    np.testing.assert_allclose(out, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)
    # and quantising the query changes the result (the pin is not vacuous)
    out_bf16, _, _ = oracle.attention(oracle.BF16, *args, rope=rope, fp8=(ks, vs))
    assert np.abs(out - out_bf16).max() > 1e-4
