"""Pins for the oracle's rotary position embedding (RoFormer, Su et al. 2021).

The paper's attention (Sec. II) takes q_n and k_n as plain projections of the
token at position n; models of the family it deploys rotate both at their
absolute position before the product and the cache.  Keeping those positions
fixed is what prefix stability (Theorem 1) needs once RoPE is in play: a key
is rotated once, when it is appended at position L_b + i, and never again.

Independent pins: transformers' Qwen2 rotary embedding and
``apply_rotary_pos_emb`` (a library routine, the "neox" pairing), the
de-interleaving permutation that maps the interleaved pairing onto it, closed
forms (position 0, the unit-frequency pair), invariants (norms, relative
positions, geometric frequencies), torch SDPA on rotated inputs for the
attention oracle, and the chunk-split / prefix-stability identities.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import datagen as dg

NEOX, INTER = oracle.ROPE_NEOX, oracle.ROPE_INTERLEAVED


def hf_rope_neox(x, positions, r, base):
    """transformers' Qwen2 rotary embedding on the first r dims of x [R, H, d]
    (fp64 data; the library forms its angles in fp32, so keep positions small)."""
    from transformers import Qwen2Config
    from transformers.models.qwen2.modeling_qwen2 import Qwen2RotaryEmbedding, apply_rotary_pos_emb
    R, H, d = x.shape
    cfg = Qwen2Config(hidden_size=r * 2, num_attention_heads=2, num_key_value_heads=2, rope_theta=float(base))
    emb = Qwen2RotaryEmbedding(cfg)
    xt = torch.from_numpy(np.ascontiguousarray(x[:, :, :r])).permute(1, 0, 2).unsqueeze(0)  # [1, H, R, r]
    pos = torch.as_tensor(np.asarray(positions, dtype=np.int64)).reshape(1, R)
    cos, sin = emb(xt, pos)
    rot, _ = apply_rotary_pos_emb(xt, xt, cos, sin)
    y = np.array(x, copy=True)
    y[:, :, :r] = rot.squeeze(0).permute(1, 0, 2).numpy()
    return y


def deinterleave(r, d):
    """Permutation taking the interleaved pairing (2i, 2i+1) onto the neox
    pairing (i, i + r/2) of the first r dims; dims >= r stay in place."""
    return np.concatenate([np.arange(0, r, 2), np.arange(1, r, 2), np.arange(r, d)])


@pytest.mark.parametrize("d,r,base", [(128, 128, 10000.0), (128, 64, 1e6), (64, 64, 500000.0), (64, 32, 10000.0)])
def test_rope_neox_matches_transformers(d, r, base):
    g = np.random.default_rng(1)
    x = g.standard_normal((37, 3, d))
    pos = g.integers(0, 48, size=37)
    y = oracle.rope(x, pos, NEOX, r, base)
    ref = hf_rope_neox(x, pos, r, base)
    np.testing.assert_allclose(y, ref, rtol=0, atol=2e-5)
    assert np.array_equal(y[:, :, r:], x[:, :, r:])


@pytest.mark.parametrize("d,r", [(128, 128), (64, 48)])
def test_rope_interleaved_is_deinterleaved_neox(d, r):
    g = np.random.default_rng(2)
    x = g.standard_normal((29, 2, d))
    pos = g.integers(0, 40, size=29)
    perm = deinterleave(r, d)
    y = oracle.rope(x, pos, INTER, r, 10000.0)
    via_neox = hf_rope_neox(x[:, :, perm], pos, r, 10000.0)
    back = np.empty_like(via_neox)
    back[:, :, perm] = via_neox
    np.testing.assert_allclose(y, back, rtol=0, atol=2e-5)


@pytest.mark.parametrize("style", [NEOX, INTER])
def test_rope_closed_forms(style):
    d, r = 64, 64
    g = np.random.default_rng(3)
    x = g.standard_normal((5, d))
    # position 0: the identity, bit for bit
    assert np.array_equal(oracle.rope(x, np.zeros(5, np.int64), style, r, 1e4), x)
    # pair 0 has unit frequency for every base: it turns by exactly `pos` radians
    a, b = (0, r // 2) if style == NEOX else (0, 1)
    for pos in (1, 7, 1000, 122879):
        e = np.zeros((1, d))
        e[0, a] = 1.0
        y = oracle.rope(e, np.array([pos]), style, r, 1e6)[0]
        assert abs(y[a] - math.cos(pos)) < 1e-12 and abs(y[b] - math.sin(pos)) < 1e-12
    # each pair keeps its length
    pos = g.integers(0, 200000, size=5)
    y = oracle.rope(x, pos, style, r, 1e4)
    pa = np.arange(r // 2) if style == NEOX else np.arange(0, r, 2)
    pb = pa + r // 2 if style == NEOX else pa + 1
    np.testing.assert_allclose(y[:, pa] ** 2 + y[:, pb] ** 2, x[:, pa] ** 2 + x[:, pb] ** 2, rtol=1e-12)


@pytest.mark.parametrize("style", [NEOX, INTER])
def test_rope_scores_depend_on_relative_position_only(style):
    d = 128
    g = np.random.default_rng(4)
    q = g.standard_normal((1, d))
    k = g.standard_normal((1, d))
    m, n = 700, 650
    base_score = float(oracle.rope(q, [m], style, d, 1e4)[0] @ oracle.rope(k, [n], style, d, 1e4)[0])
    for s in (1, 1000, 60000, 122000):
        sc = float(oracle.rope(q, [m + s], style, d, 1e4)[0] @ oracle.rope(k, [n + s], style, d, 1e4)[0])
        assert abs(sc - base_score) < 1e-9
    # and it does depend on the offset itself
    other = float(oracle.rope(q, [m + 1], style, d, 1e4)[0] @ oracle.rope(k, [n], style, d, 1e4)[0])
    assert abs(other - base_score) > 1e-3


def test_rope_frequencies_form_a_geometric_progression():
    d, r, base = 128, 128, 1e6
    eye = np.eye(d)[: r // 2]  # unit vector in the first dim of each pair
    y = oracle.rope(eye, np.ones(r // 2, np.int64), NEOX, r, base)
    phi = np.array([math.atan2(y[i, i + r // 2], y[i, i]) for i in range(r // 2)])  # all in (0, 1]
    assert abs(phi[0] - 1.0) < 1e-15
    ratio = phi[1:] / phi[:-1]
    np.testing.assert_allclose(ratio, ratio[0], rtol=1e-12)
    assert abs(ratio[0] ** (r // 2) - 1.0 / base) < 1e-12 / base


SMALL_ROPE = [
    dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64, cache_len=[40], seqlen_q=[9], paged=False),
    dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=2, head_dim=32, cache_len=[23, 0, 5], seqlen_q=[11, 6, 1],
         page_size=4),
]


def as_f64(case, a):
    return dg.bf16_bits_to_f32(a).astype(np.float64) if case.dtype == dg.BF16 else a.astype(np.float64)


@pytest.mark.parametrize("idx", range(len(SMALL_ROPE)))
@pytest.mark.parametrize("style,rdiv", [(NEOX, 1), (INTER, 2)])
def test_oracle_attention_with_rope_matches_sdpa(idx, style, rdiv):
    """Query rows and chunk keys rotated at L_b + i by transformers' routine,
    cached keys as stored, then torch SDPA in fp64."""
    case = dg.make_case(f"rope{idx}", keep_prefix=True, cfg_id=60 + idx, **SMALL_ROPE[idx])
    d = case.head_dim
    r = d // rdiv
    base = 10000.0
    perm = deinterleave(r, d) if style == INTER else np.arange(d)

    def rot(x, pos):  # x [n, H, d] fp64
        y = hf_rope_neox(x[:, :, perm], pos, r, base)
        out = np.empty_like(y)
        out[:, :, perm] = y
        return out

    out, lse, _ = oracle.attention(oracle.BF16 if case.dtype == dg.BF16 else oracle.F32, case.q, case.k_new,
                                   case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                                   case.cu_seqlens_q, case.cache_len, np.arange(case.total_q, dtype=np.int32),
                                   case.num_q_heads, case.num_kv_heads, d, case.page_size,
                                   rope=(style, r, base))
    G = case.num_q_heads // case.num_kv_heads
    for b in range(case.batch):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        L, n = int(case.cache_len[b]), hi - lo
        if n == 0:
            continue
        pos = L + np.arange(n)
        q = rot(as_f64(case, case.q[lo:hi]), pos)
        kc = rot(as_f64(case, case.k_new[lo:hi]), pos)
        k = np.concatenate([as_f64(case, case.k_prefix[b]), kc], axis=0)
        v = np.concatenate([as_f64(case, case.v_prefix[b]), as_f64(case, case.v_new[lo:hi])], axis=0)
        qt = torch.from_numpy(q).permute(1, 0, 2)
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)
        mask = torch.arange(L + n)[None, :] <= (L + torch.arange(n))[:, None]
        sc = 1.0 / math.sqrt(d)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=sc)
        s = (torch.matmul(qt, kt.transpose(1, 2)) * sc).masked_fill(~mask, float("-inf"))
        np.testing.assert_allclose(out[lo:hi], ref.permute(1, 0, 2).numpy(), rtol=0, atol=2e-5)
        np.testing.assert_allclose(lse[lo:hi], torch.logsumexp(s, -1).permute(1, 0).numpy(), rtol=0, atol=2e-5)


def half_ulp_bf16(y):
    a = np.abs(y)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


@pytest.mark.parametrize("dtype", [dg.BF16, dg.F32])
@pytest.mark.parametrize("style", [NEOX, INTER])
def test_oracle_append_with_rope_rounds_the_rotation(dtype, style):
    case = dg.make_case("rope_app", dtype=dtype, num_q_heads=4, num_kv_heads=2, head_dim=64, cache_len=[30, 3],
                        seqlen_q=[9, 20], page_size=4, cfg_id=70)
    rope = (style, 32, 10000.0)
    kp, vp = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                              case.cu_seqlens_q, case.cache_len, case.num_kv_heads, case.head_dim,
                              case.page_size, rope=rope)
    plain_k, plain_v = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table,
                                        case.bt_stride, case.cu_seqlens_q, case.cache_len, case.num_kv_heads,
                                        case.head_dim, case.page_size)
    assert np.array_equal(vp.view(np.uint8), plain_v.view(np.uint8))  # values: bit copies
    touched = np.zeros(kp.shape[:2], bool)
    for b in range(case.batch):
        lo, hi = int(case.cu_seqlens_q[b]), int(case.cu_seqlens_q[b + 1])
        L = int(case.cache_len[b])
        pos = L + np.arange(hi - lo)
        y = oracle.rope(as_f64(case, case.k_new[lo:hi]), pos, *rope)
        pages = case.block_table[b, pos // case.page_size]
        slots = (pages, pos % case.page_size)
        touched[slots] = True
        got = as_f64(case, kp[slots])
        if dtype == dg.F32:
            assert np.array_equal(kp[slots], y.astype(np.float32))  # numpy's nearest-even cast
        else:
            assert np.all(np.abs(got - y) <= half_ulp_bf16(y) * (1 + 1e-12))
        assert np.array_equal(got[:, :, 32:], y[:, :, 32:])  # unrotated tail is a bit copy
    # every other slot is untouched
    assert np.array_equal(kp[~touched].view(np.uint8), case.k_pool[~touched].view(np.uint8))


@pytest.mark.parametrize("style", [NEOX, INTER])
def test_oracle_chunk_split_and_prefix_stability_with_rope(style):
    """Absolute positions make the rotation compose with append-only growth:
    extend(L, n1); append; extend(L + n1, n2) gives the rows of extend(L, n1 + n2),
    and extend over a rope-appended prefix gives the tail rows of a rope prefill."""
    rope = (style, 64, 10000.0)
    L, n1, n2 = 21, 7, 12
    whole = dg.make_case("split", dtype=dg.F32, num_q_heads=4, num_kv_heads=2, head_dim=64, cache_len=[L],
                         seqlen_q=[n1 + n2], page_size=4, cfg_id=71)
    args = (whole.num_q_heads, whole.num_kv_heads, whole.head_dim, whole.page_size)
    one, one_lse, _ = oracle.attention(oracle.F32, whole.q, whole.k_new, whole.v_new, whole.k_pool, whole.v_pool,
                                       whole.block_table, whole.bt_stride, whole.cu_seqlens_q, whole.cache_len,
                                       np.arange(n1 + n2, dtype=np.int32), *args, rope=rope)
    cu1 = np.array([0, n1], np.int32)
    first, _, _ = oracle.attention(oracle.F32, whole.q[:n1], whole.k_new[:n1], whole.v_new[:n1], whole.k_pool,
                                   whole.v_pool, whole.block_table, whole.bt_stride, cu1, whole.cache_len,
                                   np.arange(n1, dtype=np.int32), *args, rope=rope)
    kp, vp = oracle.kv_append(whole.k_new[:n1], whole.v_new[:n1], whole.k_pool, whole.v_pool, whole.block_table,
                              whole.bt_stride, cu1, whole.cache_len, whole.num_kv_heads, whole.head_dim,
                              whole.page_size, rope=rope)
    second, second_lse, _ = oracle.attention(oracle.F32, whole.q[n1:], whole.k_new[n1:], whole.v_new[n1:], kp, vp,
                                             whole.block_table, whole.bt_stride, np.array([0, n2], np.int32),
                                             np.array([L + n1], np.int32), np.arange(n2, dtype=np.int32), *args,
                                             rope=rope)
    np.testing.assert_array_equal(first, one[:n1])  # same keys, same positions: identical arithmetic
    np.testing.assert_allclose(second, one[n1:], rtol=0, atol=2e-6)  # cached keys rounded to fp32
    np.testing.assert_allclose(second_lse, one_lse[n1:], rtol=0, atol=2e-6)

    # prefix stability: a rope prefill of the whole history, its tail rows ...
    S = L + n1 + n2
    hist = dg.make_case("hist", dtype=dg.F32, num_q_heads=4, num_kv_heads=2, head_dim=64, cache_len=[0],
                        seqlen_q=[S], page_size=4, cfg_id=72)
    full, full_lse, _ = oracle.attention(oracle.F32, hist.q, hist.k_new, hist.v_new, None, None, None, 1,
                                         hist.cu_seqlens_q, None, np.arange(L, S, dtype=np.int32), *args, rope=rope)
    # ... equal extend(L, S - L) over a cache built by rope-appending the first L tokens
    pool_k = np.zeros((S // 4 + 1, 4, 2, 64), np.float32)
    pool_v = np.zeros_like(pool_k)
    table = np.arange(pool_k.shape[0], dtype=np.int32)[None, ::-1].copy()
    kp, vp = oracle.kv_append(hist.k_new[:L], hist.v_new[:L], pool_k, pool_v, table, table.shape[1],
                              np.array([0, L], np.int32), None, 2, 64, 4, rope=rope)
    ext, ext_lse, _ = oracle.attention(oracle.F32, hist.q[L:], hist.k_new[L:], hist.v_new[L:], kp, vp, table,
                                       table.shape[1], np.array([0, S - L], np.int32), np.array([L], np.int32),
                                       np.arange(S - L, dtype=np.int32), *args, rope=rope)
    np.testing.assert_allclose(ext, full, rtol=0, atol=2e-6)
    np.testing.assert_allclose(ext_lse, full_lse, rtol=0, atol=2e-6)


def test_oracle_rope_rejects_malformed_arguments():
    x = np.zeros((1, 8))
    for style, r in ((NEOX, 7), (NEOX, 10), (5, 8), (INTER, 0)):
        with pytest.raises(ValueError):
            oracle.rope(x, [0], style, r if r else -2, 1e4)
