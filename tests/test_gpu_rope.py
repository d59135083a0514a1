"""GPU parity for rotary position embedding at absolute cache positions.

The HIP path rotates q and k_new at L_b + i (one fused launch that also
appends) and runs the attention on the rotated copies; the oracle rotates in
fp64 inside its attention and append.  Both rotate in fp64 and round each key
once, so the whole pool after the append (rotated keys, copied values,
untouched canaries) is compared bit for bit.  Outputs use the same gates as
every other attention test.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_07325_amd import csr
from paper_2605_07325_amd import datagen as dg
from tests.gpu_harness import Dev, compare, from_dev, note, values

pytestmark = pytest.mark.gpu

NEOX, INTER = csr.CSR_ROPE_NEOX, csr.CSR_ROPE_INTERLEAVED


def rope_dev(case, style, r, theta):
    dev = Dev(case)
    dev.desc.rope_style = style
    dev.desc.rope_dim = r
    dev.desc.rope_theta = theta
    return dev


def oracle_rope_rows(case, rows, rope, prefill=False):
    out, lse, _ = oracle.attention(oracle.BF16 if case.dtype == dg.BF16 else oracle.F32, case.q, case.k_new,
                                   case.v_new, case.k_pool, case.v_pool, case.block_table, case.bt_stride,
                                   case.cu_seqlens_q, None if prefill else case.cache_len, rows, case.num_q_heads,
                                   case.num_kv_heads, case.head_dim, case.page_size, rope=rope)
    return out, lse


def as_f64(case, a):
    return dg.bf16_bits_to_f32(a).astype(np.float64) if case.dtype == dg.BF16 else a.astype(np.float64)


def check_rope_pool(case, dev, rope, cache_len):
    """Pool after a rope append equals the append oracle bit for bit: values
    copied, each key rotated in fp64 at its position and rounded once to the
    element type (the library's rotation is fp64 too), untouched slots keep
    their canaries."""
    kp_ref, vp_ref = oracle.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table,
                                      case.bt_stride, case.cu_seqlens_q, cache_len, case.num_kv_heads,
                                      case.head_dim, case.page_size, rope=rope)
    kp, vp = from_dev(case, dev.k_pool), from_dev(case, dev.v_pool)
    bits = lambda a: a.view(np.uint32) if a.dtype == np.float32 else a  # noqa: E731  (NaN canaries compare by bits)
    np.testing.assert_array_equal(bits(vp), bits(vp_ref))
    differ = int(np.count_nonzero(bits(kp) != bits(kp_ref)))
    assert differ == 0, f"{differ} rotated key elements differ from the oracle's"
    note(f"rope pool: {kp.size} key elements bit for bit")


SMALL = [
    ("bf16_neox_d128", NEOX, 0, 1e6, dict(dtype=dg.BF16, num_q_heads=32, num_kv_heads=2, head_dim=128,
                                          cache_len=[1000], seqlen_q=[37], page_size=16, scale=0.5)),
    ("bf16_inter_d64_r32", INTER, 32, 1e4, dict(dtype=dg.BF16, num_q_heads=8, num_kv_heads=1, head_dim=64,
                                                cache_len=[77], seqlen_q=[100], page_size=4, scale=0.5)),
    ("bf16_neox_ragged", NEOX, 64, 5e5, dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128,
                                             cache_len=[0, 513, 64, 2049], seqlen_q=[17, 1, 200, 64], page_size=16,
                                             scale=0.5, interleave=True)),
    ("f32_neox_d64_r48", NEOX, 48, 1e4, dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=1, head_dim=64,
                                             cache_len=[300], seqlen_q=[70], page_size=16)),
    ("f32_inter_d128", INTER, 0, 1e4, dict(dtype=dg.F32, num_q_heads=4, num_kv_heads=2, head_dim=128,
                                           cache_len=[31, 0, 200], seqlen_q=[5, 40, 1], page_size=8,
                                           interleave=True)),
]


@pytest.mark.parametrize("label,style,r,theta,kw", SMALL, ids=[s[0] for s in SMALL])
@pytest.mark.parametrize("nsplit", [None, 3])
def test_rope_extend_append_all_rows(label, style, r, theta, kw, nsplit):
    if nsplit:
        csr.set_plan_overrides(nsplit=nsplit)
    case = dg.make_case(label, seed=2, cfg_id=500, **kw)
    rope = (style, r, theta)
    note(f"rope {label} nsplit={nsplit} L={case.cache_len.tolist()} n={case.seqlen_q.tolist()}: "
         f"csr_extend_attention(APPEND)")
    dev = rope_dev(case, style, r, theta)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = np.arange(case.total_q, dtype=np.int32)
    ref, ref_lse = oracle_rope_rows(case, rows, rope)
    compare(case, out, lse, rows, ref, ref_lse, f"rope/{label}/split={nsplit}")
    check_rope_pool(case, dev, rope, case.cache_len)


@pytest.mark.parametrize("label,style,r,theta,kw", SMALL[:3], ids=[s[0] for s in SMALL[:3]])
def test_rope_kv_append_alone(label, style, r, theta, kw):
    case = dg.make_case(label, seed=3, cfg_id=501, **kw)
    note(f"rope {label}: csr_kv_append")
    dev = rope_dev(case, style, r, theta)
    dev.append()
    torch.cuda.synchronize()
    check_rope_pool(case, dev, (style, r, theta), case.cache_len)


@pytest.mark.parametrize("where", ["subnormal", "overflow", "nan_inf"])
def test_rope_append_rounding_at_the_range_ends(where):
    """Keys in bf16's subnormal range (N(0,1) x 2^-128), and keys of magnitude 2.5e38 - 3.3e38
    with random signs, whose rotations pass bf16's largest value at most angles (those round to
    infinity): the single rounding from fp64 holds there too."""
    case = dg.make_case("rope_range", dtype=dg.BF16, num_q_heads=8, num_kv_heads=2, head_dim=128,
                        cache_len=[40], seqlen_q=[300], page_size=16, seed=4, cfg_id=502,
                        scale=2.0 ** -128 if where == "subnormal" else 1.0 if where == "overflow" else 0.5)
    if where == "overflow":
        g = dg.rng(4, 502, 7)
        mag = g.uniform(2.5e38, 3.3e38, size=case.k_new.shape).astype(np.float32)
        case.k_new = dg.to_bf16_bits(np.where(g.integers(0, 2, size=mag.shape) == 1, mag, -mag))
    elif where == "nan_inf":  # a sprinkling of NaNs (two payloads) and infinities: NaN results are 0x7fc0
        g = dg.rng(4, 502, 8)
        k = case.k_new.copy()
        special = np.array([0x7fc0, 0xffc1, 0x7f80, 0xff80], dtype=np.uint16)
        hit = g.random(k.shape) < 0.01
        k[hit] = special[g.integers(0, 4, size=int(hit.sum()))]
        case.k_new = k
    note(f"rope bf16 keys, {where}: csr_kv_append")
    dev = rope_dev(case, NEOX, 0, 1e4)
    dev.append()
    torch.cuda.synchronize()
    check_rope_pool(case, dev, (NEOX, 0, 1e4), case.cache_len)


@pytest.mark.parametrize("n", [512, 1])
def test_rope_c3_120k_positions(n):
    """Positions 122880 .. 122880 + n - 1: the angle reduction in fp64 keeps the
    rotation exact to fp32 even where pos * theta_0 is ~1.2e5 rad."""
    case = dg.config(f"c3_{n}")
    rope = (NEOX, 0, 1e6)
    note(f"rope c3 bf16 L=122880 n={n}: csr_extend_attention(APPEND)")
    dev = rope_dev(case, *rope)
    out, lse = dev.extend(append=True)
    torch.cuda.synchronize()
    rows = dg.sample_rows(case, 64, cfg_id=3)
    ref, ref_lse = oracle_rope_rows(case, rows, rope)
    compare(case, out, lse, rows, ref, ref_lse, f"rope/c3_{n}")
    check_rope_pool(case, dev, rope, case.cache_len)


@pytest.mark.parametrize("style", [NEOX, INTER])
def test_rope_chunk_split_on_device(style):
    """extend(L, n1) with append, then extend(L + n1, n2) over that cache, gives
    the rows of one extend(L, n1 + n2): the positions are absolute."""
    L, n1, n2 = 3000, 150, 90
    kw = dict(dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, page_size=16, scale=0.5)
    one = dg.make_case("rope_one", cache_len=[L], seqlen_q=[n1 + n2], seed=4, cfg_id=502, **kw)
    rope = (style, 0, 1e4)
    note(f"rope chunk split style={style} L={L} n={n1}+{n2}")
    dev_one = rope_dev(one, *rope)
    out_one, lse_one = dev_one.extend()
    a = dg.make_case("rope_a", cache_len=[L], seqlen_q=[n1], seed=4, cfg_id=502, **kw)
    for f in ("q", "k_new", "v_new"):
        getattr(a, f)[:] = getattr(one, f)[:n1]
    a.k_pool, a.v_pool, a.block_table, a.bt_stride = one.k_pool, one.v_pool, one.block_table, one.bt_stride
    dev_a = rope_dev(a, *rope)
    out_a, _ = dev_a.extend(append=True)
    b = dg.make_case("rope_b", cache_len=[L + n1], seqlen_q=[n2], seed=4, cfg_id=502, **kw)
    for f in ("q", "k_new", "v_new"):
        getattr(b, f)[:] = getattr(one, f)[n1:]
    b.block_table, b.bt_stride = one.block_table, one.bt_stride
    dev_b = rope_dev(b, *rope)
    dev_b.k_pool, dev_b.v_pool = dev_a.k_pool, dev_a.v_pool  # the cache after A's rope append
    out_b, lse_b = dev_b.extend()
    torch.cuda.synchronize()
    assert np.abs(values(a, out_a) - values(one, out_one)[:n1]).max() < 1e-2
    assert np.abs(values(b, out_b) - values(one, out_one)[n1:]).max() < 1e-2
    assert np.abs(lse_b.cpu().numpy() - lse_one.cpu().numpy()[n1:]).max() < 1e-4
    rows = np.arange(n2, dtype=np.int32)
    b_ref = dg.make_case("rope_b", cache_len=[L + n1], seqlen_q=[n2], seed=4, cfg_id=502, **kw)
    for f in ("q", "k_new", "v_new"):
        getattr(b_ref, f)[:] = getattr(one, f)[n1:]
    kp, vp = oracle.kv_append(a.k_new, a.v_new, one.k_pool, one.v_pool, one.block_table, one.bt_stride,
                              a.cu_seqlens_q, a.cache_len, 2, 128, 16, rope=rope)
    b_ref.k_pool, b_ref.v_pool, b_ref.block_table, b_ref.bt_stride = kp, vp, one.block_table, one.bt_stride
    ref, ref_lse = oracle_rope_rows(b_ref, rows, rope)
    compare(b, out_b, lse_b, rows, ref, ref_lse, f"rope/chunk-split/{style}")


def test_rope_prefix_stability_on_device():
    """A rope prefill of S tokens writes the rotated cache; an extend over its
    first L positions with the last S - L tokens reproduces the prefill's rows."""
    S, L = 2600, 2000
    case = dg.make_case("rope_hist", dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, cache_len=[0],
                        seqlen_q=[S], page_size=16, scale=0.5, seed=5, cfg_id=503)
    rope = (NEOX, 0, 1e6)
    note(f"rope prefix stability S={S} L={L}: csr_prefill(cache write) then csr_extend_attention")
    dev = rope_dev(case, *rope)
    out_p, lse_p = dev.prefill(write_cache=True)
    torch.cuda.synchronize()
    check_rope_pool(case, dev, rope, None)
    rows = dg.sample_rows(case, 48, cfg_id=6)
    ref, ref_lse = oracle_rope_rows(case, rows, rope, prefill=True)
    compare(case, out_p, lse_p, rows, ref, ref_lse, "rope/prefill")
    ext = dg.make_case("rope_tail", dtype=dg.BF16, num_q_heads=16, num_kv_heads=2, head_dim=128, cache_len=[L],
                       seqlen_q=[S - L], page_size=16, scale=0.5, seed=5, cfg_id=503)
    for f in ("q", "k_new", "v_new"):
        getattr(ext, f)[:] = getattr(case, f)[L:]
    ext.block_table, ext.bt_stride = case.block_table, case.bt_stride
    dev_e = rope_dev(ext, *rope)
    dev_e.k_pool, dev_e.v_pool = dev.k_pool, dev.v_pool
    out_e, lse_e = dev_e.extend()
    torch.cuda.synchronize()
    assert np.abs(values(ext, out_e) - values(case, out_p)[L:]).max() < 1e-2
    assert np.abs(lse_e.cpu().numpy() - lse_p.cpu().numpy()[L:]).max() < 1e-4
