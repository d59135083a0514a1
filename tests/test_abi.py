"""C-ABI checks that need no GPU: the library loads, exports every function
include/csr.h declares, and rejects malformed arguments on the host before
any HIP runtime call (no argument below would be valid on a device either)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2605_07325_amd import csr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "csr.h")

FAKE = 0x100000  # 16-byte aligned, never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(csr_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = csr.lib()
    names = declared_functions()
    assert set(names) == set(csr.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    lib = csr.lib()
    for code, name in [(0, "CSR_OK"), (1, "CSR_E_INVAL"), (2, "CSR_E_UNSUPPORTED"), (3, "CSR_E_WORKSPACE"),
                       (4, "CSR_E_HIP")]:
        assert lib.csr_status_string(code).decode() == name
    assert lib.csr_status_string(99).decode() == "CSR_E_UNKNOWN"


def call_extend(desc, batch=1, q=FAKE, kn=FAKE, vn=FAKE, kp=FAKE, vp=FAKE, num_pages=64, bt=FAKE, bt_stride=8,
                cu=FAKE, cl=FAKE, total_q=16, max_q=16, max_l=100, flags=0, out=FAKE, lse=None, ws=None, ws_bytes=0):
    lib = csr.lib()
    p = lambda x: None if x is None else ctypes.c_void_p(x)  # noqa: E731
    return lib.csr_extend_attention(None if desc is None else ctypes.byref(desc), batch, p(q), p(kn), p(vn), p(kp),
                                    p(vp), num_pages, p(bt), bt_stride, p(cu), p(cl), total_q, max_q, max_l, flags,
                                    p(out), p(lse), p(ws), ws_bytes, None)


def good_desc(**over):
    kw = dict(num_q_heads=16, num_kv_heads=2, head_dim=128, page_size=16)
    kw.update(over)
    return csr.make_desc(**kw)


@pytest.mark.parametrize("desc,code", [
    (None, csr.CSR_E_INVAL),
    (csr.AttnDesc(16, 3, 128, 16, 0.0, csr.CSR_BF16), csr.CSR_E_INVAL),   # Hq % Hkv
    (csr.AttnDesc(0, 1, 128, 16, 0.0, csr.CSR_BF16), csr.CSR_E_INVAL),    # no heads
    (csr.AttnDesc(16, 2, 96, 16, 0.0, csr.CSR_BF16), csr.CSR_E_UNSUPPORTED),  # head_dim
    (csr.AttnDesc(16, 2, 128, 16, 0.0, 7), csr.CSR_E_UNSUPPORTED),        # dtype
    (csr.AttnDesc(16, 2, 128, 12, 0.0, csr.CSR_BF16), csr.CSR_E_INVAL),   # page size not a power of two
    (csr.AttnDesc(16, 2, 128, 2048, 0.0, csr.CSR_BF16), csr.CSR_E_INVAL),  # page size too large
    (csr.AttnDesc(16, 2, 128, 16, -1.0, csr.CSR_BF16), csr.CSR_E_INVAL),  # negative scale
    (csr.AttnDesc(16, 2, 128, 16, float("nan"), csr.CSR_BF16), csr.CSR_E_INVAL),
])
def test_descriptor_validation(desc, code):
    assert call_extend(desc) == code
    assert csr.lib().csr_last_error().decode()


@pytest.mark.parametrize("over,code", [
    (dict(q=FAKE + 8), csr.CSR_E_INVAL),           # misaligned q
    (dict(out=None), csr.CSR_E_INVAL),             # no output
    (dict(cu=None), csr.CSR_E_INVAL),              # no cu_seqlens
    (dict(kp=None), csr.CSR_E_INVAL),              # prefix but no pool
    (dict(cl=None), csr.CSR_E_INVAL),              # prefix lengths missing
    (dict(max_q=17), csr.CSR_E_INVAL),             # max_seqlen_q > total_q
    (dict(max_q=0), csr.CSR_E_INVAL),
    (dict(batch=-1), csr.CSR_E_INVAL),
    (dict(bt_stride=0), csr.CSR_E_INVAL),
    (dict(bt_stride=4), csr.CSR_E_INVAL),          # 4 pages of 16 cannot hold 100 cached positions
    (dict(num_pages=0), csr.CSR_E_INVAL),
    (dict(flags=2), csr.CSR_E_INVAL),              # unknown flag
    (dict(lse=FAKE + 2), csr.CSR_E_INVAL),         # misaligned lse
    (dict(batch=0, total_q=3), csr.CSR_E_INVAL),
])
def test_argument_validation(over, code):
    assert call_extend(good_desc(), **over) == code


def test_empty_call_is_a_noop():
    assert call_extend(good_desc(), total_q=0, max_q=0) == csr.CSR_OK


def test_missing_workspace_is_reported():
    desc = good_desc(num_q_heads=64, num_kv_heads=4)
    need = csr.extend_workspace_size(desc, 1, 512, 512, 122880)
    assert need > 0  # 120K prefix with a 512-token chunk splits the key range
    st = call_extend(desc, total_q=512, max_q=512, max_l=122880, bt_stride=7712, num_pages=7712, ws=None)
    assert st == csr.CSR_E_WORKSPACE
    st = call_extend(desc, total_q=512, max_q=512, max_l=122880, bt_stride=7712, num_pages=7712, ws=FAKE,
                     ws_bytes=need - 16)
    assert st == csr.CSR_E_WORKSPACE


def test_workspace_query_rejects_bad_sizes():
    d = good_desc()
    assert csr.extend_workspace_size(d, 0, 16, 16, 100) == 0
    assert csr.extend_workspace_size(csr.AttnDesc(16, 3, 128, 16, 0.0, csr.CSR_BF16), 1, 16, 16, 100) == 0


def test_kv_append_validation():
    lib = csr.lib()
    p = ctypes.c_void_p
    d = good_desc()
    args = lambda **o: dict(dict(batch=1, kn=FAKE, vn=FAKE, kp=FAKE, vp=FAKE, pages=8, bt=FAKE, bts=4, cu=FAKE,  # noqa: E731
                                 cl=FAKE, total=8), **o)
    def run(**o):
        a = args(**o)
        return lib.csr_kv_append(ctypes.byref(d), a["batch"], p(a["kn"]) if a["kn"] else None, p(a["vn"]) if a["vn"] else None,
                                 p(a["kp"]) if a["kp"] else None, p(a["vp"]) if a["vp"] else None, a["pages"],
                                 p(a["bt"]), a["bts"], p(a["cu"]) if a["cu"] else None, p(a["cl"]), a["total"], None)
    assert run(kp=None) == csr.CSR_E_INVAL
    assert run(kn=FAKE + 4) == csr.CSR_E_INVAL
    assert run(pages=0) == csr.CSR_E_INVAL
    assert run(cu=None) == csr.CSR_E_INVAL
    assert run(total=0) == csr.CSR_OK


def test_prefill_validation():
    lib = csr.lib()
    p = ctypes.c_void_p
    d = good_desc()
    # max_seqlen above total
    assert lib.csr_prefill(ctypes.byref(d), 1, p(FAKE), p(FAKE), p(FAKE), None, None, 0, None, 1, p(FAKE), 8, 9,
                           p(FAKE), None, None, 0, None) == csr.CSR_E_INVAL
    # only one pool given
    assert lib.csr_prefill(ctypes.byref(d), 1, p(FAKE), p(FAKE), p(FAKE), p(FAKE), None, 4, None, 1, p(FAKE), 8, 8,
                           p(FAKE), None, None, 0, None) == csr.CSR_E_INVAL


def test_event_hook_requires_both_events():
    lib = csr.lib()
    assert lib.csr_set_attention_events(ctypes.c_void_p(FAKE), None) == csr.CSR_E_INVAL
    assert lib.csr_set_attention_events(None, None) == csr.CSR_OK


def test_workgroup_clock_hook_validation():
    lib = csr.lib()
    assert lib.csr_set_workgroup_clock(None, 5) == csr.CSR_E_INVAL
    assert lib.csr_set_workgroup_clock(ctypes.c_void_p(FAKE), 0) == csr.CSR_E_INVAL
    assert lib.csr_set_workgroup_clock(ctypes.c_void_p(FAKE), -1) == csr.CSR_E_INVAL
    assert lib.csr_set_workgroup_clock(ctypes.c_void_p(FAKE + 4), 8) == csr.CSR_E_INVAL   # misaligned
    assert lib.csr_set_workgroup_clock(ctypes.c_void_p(FAKE), 8) == csr.CSR_OK
    assert lib.csr_set_workgroup_clock(None, 0) == csr.CSR_OK


@pytest.mark.parametrize("over,code", [
    (dict(rope_style=3, rope_theta=1e4), csr.CSR_E_INVAL),                 # unknown pairing
    (dict(rope_style=csr.CSR_ROPE_NEOX, rope_theta=0.0), csr.CSR_E_INVAL),  # no base
    (dict(rope_style=csr.CSR_ROPE_NEOX, rope_theta=float("inf")), csr.CSR_E_INVAL),
    (dict(rope_style=csr.CSR_ROPE_NEOX, rope_theta=float("nan")), csr.CSR_E_INVAL),
    (dict(rope_style=csr.CSR_ROPE_NEOX, rope_dim=24, rope_theta=1e4), csr.CSR_E_UNSUPPORTED),   # not a multiple of 16
    (dict(rope_style=csr.CSR_ROPE_INTERLEAVED, rope_dim=144, rope_theta=1e4), csr.CSR_E_UNSUPPORTED),  # > d
])
def test_rope_descriptor_validation(over, code):
    assert call_extend(good_desc(**over)) == code
    assert csr.lib().csr_last_error().decode()


def test_rope_workspace_holds_rotated_q_and_k():
    plain = good_desc(num_q_heads=64, num_kv_heads=4)
    rope = good_desc(num_q_heads=64, num_kv_heads=4, rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e6)
    for T, L in ((512, 122880), (8, 0), (3, 100)):
        extra = csr.extend_workspace_size(rope, 1, T, T, L) - csr.extend_workspace_size(plain, 1, T, T, L)
        align = lambda x: (x + 255) // 256 * 256  # noqa: E731
        assert extra == align(T * 64 * 128 * 2) + align(T * 4 * 128 * 2)
    # prefill needs them too, and a call with too small a workspace is refused before any launch
    assert csr.prefill_workspace_size(rope, 1, 8, 8) >= align(8 * 64 * 128 * 2) + align(8 * 4 * 128 * 2)
    need = csr.extend_workspace_size(rope, 1, 16, 16, 100)
    st = call_extend(good_desc(rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e4), ws=FAKE,
                     ws_bytes=csr.extend_workspace_size(good_desc(rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e4), 1, 16,
                                                        16, 100) - 16)
    assert need > 0 and st == csr.CSR_E_WORKSPACE
    assert call_extend(good_desc(rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e4), ws=None) == csr.CSR_E_WORKSPACE


@pytest.mark.parametrize("over,code", [
    (dict(kv_dtype=7, k_scale=1.0, v_scale=1.0), csr.CSR_E_INVAL),                        # unknown cache type
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=0.0, v_scale=1.0), csr.CSR_E_INVAL),       # no key scale
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=1.0, v_scale=float("nan")), csr.CSR_E_INVAL),
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=1.0, v_scale=1.0, head_dim=64), csr.CSR_E_UNSUPPORTED),
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=1.0, v_scale=1.0, dtype=torch.float32), csr.CSR_E_UNSUPPORTED),
    (dict(q_scale=0.5), csr.CSR_E_UNSUPPORTED),                                            # fp8 products, bf16 cache
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=1.0, v_scale=1.0, q_scale=-1.0), csr.CSR_E_INVAL),
    (dict(kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=1.0, v_scale=1.0, q_scale=float("inf")), csr.CSR_E_INVAL),
])
def test_fp8_cache_descriptor_validation(over, code):
    assert call_extend(good_desc(**over)) == code
    assert csr.lib().csr_last_error().decode()


def test_fp8_cache_workspace_holds_quantised_chunk():
    plain = good_desc(num_q_heads=64, num_kv_heads=4)
    fp8 = good_desc(num_q_heads=64, num_kv_heads=4, kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=0.05, v_scale=0.05)
    both = good_desc(num_q_heads=64, num_kv_heads=4, kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=0.05, v_scale=0.05,
                     rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e6)
    align = lambda x: (x + 255) // 256 * 256  # noqa: E731
    # split partials (fp32 O and LSE per split); with no device the plan assumes 256 CUs
    partials = lambda T, ns: align(ns * T * 64 * 128 * 4) + ns * T * 64 * 4 if ns > 1 else 0  # noqa: E731
    # (T, L, key splits over a bf16 cache, over an fp8 cache): a decode step over
    # an fp8 cache runs 4-wave workgroups, two per CU, and doubles its splits
    for T, L, ns, ns8 in ((512, 122880, 2, 2), (1, 122880, 64, 128), (7, 0, 1, 1)):
        base = csr.extend_workspace_size(plain, 1, T, T, L)
        assert base == partials(T, ns)
        extra = partials(T, ns8) - partials(T, ns)
        assert csr.extend_workspace_size(fp8, 1, T, T, L) - base == extra + 2 * align(T * 4 * 128)
        assert (csr.extend_workspace_size(both, 1, T, T, L) - base
                == extra + align(T * 64 * 128 * 2) + 2 * align(T * 4 * 128))
        # fp8 score products: the query as e4m3 codes (one byte), with or without RoPE
        for over in (dict(), dict(rope_style=csr.CSR_ROPE_NEOX, rope_theta=1e6)):
            q8 = good_desc(num_q_heads=64, num_kv_heads=4, kv_dtype=csr.CSR_KV_FP8_E4M3, k_scale=0.05, v_scale=0.05,
                           q_scale=0.015625, **over)
            assert (csr.extend_workspace_size(q8, 1, T, T, L) - base
                    == extra + align(T * 64 * 128) + 2 * align(T * 4 * 128))


def test_plan_overrides_validation():
    lib = csr.lib()
    assert lib.csr_set_plan_overrides(-1, 0, 0) == csr.CSR_E_INVAL
    assert lib.csr_set_plan_overrides(0, 2, 0) == csr.CSR_E_INVAL
    assert lib.csr_set_plan_overrides(0, 0, -1) == csr.CSR_E_INVAL
    assert lib.csr_set_plan_overrides(0, 0, 0) == csr.CSR_OK


def test_plan_overrides_steer_the_split_and_the_environment_does_not():
    """Forcing 4 key splits sizes the split-K partials for 4; the planner's own choice
    comes back afterwards, and an environment variable of the old override names
    changes nothing."""
    d = good_desc(num_q_heads=64, num_kv_heads=4)
    args = (1, 512, 512, 122880)
    base = csr.extend_workspace_size(d, *args)
    with csr.plan_overrides(nsplit=4):
        forced = csr.extend_workspace_size(d, *args)
    rows = 512 * 64
    want = ((4 * rows * 128 * 4 + 255) // 256) * 256 + 4 * rows * 4
    assert forced == want
    assert csr.extend_workspace_size(d, *args) == base
    os.environ["CSR_NSPLIT"] = "7"
    try:
        assert csr.extend_workspace_size(d, *args) == base
    finally:
        os.environ.pop("CSR_NSPLIT", None)


def test_binding_rejects_pools_of_another_layout():
    """num_pages bounds every page id the kernels read, so the binding accepts only
    [num_pages][P][Hkv][d] pools of the descriptor's element type."""
    d = good_desc()
    flat = torch.zeros((64 * 16, 2, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        csr._pool_pages(d, flat, flat)
    wrong_type = torch.zeros((64, 16, 2, 128), dtype=torch.float32)
    with pytest.raises(ValueError):
        csr._pool_pages(d, wrong_type, wrong_type)
    ok = torch.zeros((64, 16, 2, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):  # right layout, but a host tensor
        csr._pool_pages(d, ok, ok)
    with pytest.raises(ValueError):
        csr._pool_pages(d, None, ok)
