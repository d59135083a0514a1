"""ctypes front end of the C fp64 oracle (``csr_oracle.c``) plus its build step.

Test infrastructure only (see ``oracle/__init__.py``).  Each function names the
passage of the paper it follows; the arithmetic lives in ``csr_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csr_oracle.c")
# CSR_ORACLE_LIBRARY: a separately built copy of the same source (e.g. with
# host sanitizers); default: the in-tree build.
LIB = os.environ.get("CSR_ORACLE_LIBRARY") or os.path.join(HERE, "liboracle.so")

F32, BF16 = 0, 1
ROPE_NONE, ROPE_NEOX, ROPE_INTERLEAVED = 0, 1, 2

_lib = None


def build() -> str:
    """Compile the oracle with gcc (plain C, OpenMP)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", SRC, "-o", LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.environ.get("CSR_ORACLE_LIBRARY") and (
                not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC)):
            build()
        lib = ctypes.CDLL(LIB)
        p, i, d = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
        f = ctypes.c_float
        lib.csr_oracle_attention.argtypes = [i, i, i, i, i, d, i, i, d, i, f, f, f, i, p, p, p, p, p, p, i, p, p, i,
                                             p, p, p, p, i]
        lib.csr_oracle_attention.restype = i
        lib.csr_oracle_kv_append.argtypes = [i, i, i, i, i, i, d, i, f, f, i, p, p, p, p, p, i, p, p]
        lib.csr_oracle_e4m3_encode.argtypes = [p, p, ctypes.c_int64]
        lib.csr_oracle_e4m3_encode.restype = i
        lib.csr_oracle_e4m3_decode.argtypes = [p, p, ctypes.c_int64]
        lib.csr_oracle_e4m3_decode.restype = i
        lib.csr_oracle_kv_append.restype = i
        lib.csr_oracle_rope.argtypes = [p, p, ctypes.c_int64, i, i, i, d, p]
        lib.csr_oracle_rope.restype = i
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def default_threads() -> int:
    return len(os.sched_getaffinity(0))


def _rope_args(rope, head_dim):
    """``rope`` = None or ``(style, rotary_dims, base)``; rotary_dims 0 means all."""
    if rope is None or rope[0] == ROPE_NONE:
        return ROPE_NONE, 0, 0.0
    style, r, base = rope
    return int(style), int(r or head_dim), float(base)


def _fp8_args(fp8):
    """``fp8`` = None (pools in the input type) or ``(k_scale, v_scale)``:
    pools of OCP e4m3 codes (uint8) with those dequantisation scales."""
    if fp8 is None:
        return 0, 1.0, 1.0
    return 1, float(fp8[0]), float(fp8[1])


def e4m3_encode(x):
    """OCP e4m3 codes of fp32 values: saturate to +-448, nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint8)
    _load().csr_oracle_e4m3_encode(_ptr(x), _ptr(out), x.size)
    return out


def e4m3_decode(codes):
    """Exact values (float64) of OCP e4m3 codes."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(c.shape, np.float64)
    _load().csr_oracle_e4m3_decode(_ptr(c), _ptr(out), c.size)
    return out


def rope(x, positions, style, rotary_dims, base):
    """RoFormer's rotary position embedding (Su et al., 2021) of fp64 rows
    ``x [R, d]`` (or ``[R, H, d]``, one position per leading row) at
    ``positions [R]``: pair i of the first ``rotary_dims`` dims turns by
    ``position * base**(-2i/rotary_dims)``; ``style`` picks the pairing
    (ROPE_NEOX: i with i + r/2, ROPE_INTERLEAVED: 2i with 2i + 1)."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float64)
    R = x.shape[0]
    d = x.shape[-1]
    per = int(np.prod(x.shape[1:-1])) if x.ndim > 2 else 1
    pos = np.repeat(np.ascontiguousarray(positions, dtype=np.int64).reshape(R), per)
    y = np.empty_like(x)
    rc = lib.csr_oracle_rope(_ptr(x), _ptr(y), R * per, d, int(rotary_dims or d), int(style), float(base),
                             _ptr(pos))
    if rc != 0:
        raise ValueError("malformed rotary embedding arguments")
    return y


def attention(dtype, q, k_new, v_new, k_pool, v_pool, block_table, bt_stride, cu_seqlens_q,
              cache_len, rows, num_q_heads, num_kv_heads, head_dim, page_size, scale=None,
              nthreads=None, rope=None, fp8=None, q_fp8=None):
    """Extend attention for the query tokens in ``rows`` (all heads).

    Paper Sec. II, eq. (causal_attention_1)-(causal_attention_3) over the
    cached concatenation of eq. (K_cache)-(V_cache); prefix length L_b = i* - 1
    (eq. (csr_i_star)).  ``cache_len=None`` is the L_b = 0 full re-prefill
    (warm-up of Algorithm 1).  Arrays: bf16 as uint16 bit patterns, fp32 as
    float32.  ``rope=(style, rotary_dims, base)`` first rotates every query
    row and every chunk key at its absolute position (see ``rope``); cached
    keys are used as stored.  ``fp8=(k_scale, v_scale)``: the pools hold e4m3
    codes (uint8) and chunk keys/values enter quantised exactly as the append
    stores them.  ``q_fp8=q_scale`` (with ``fp8``): fp8 products, every
    (rotated) query element enters as e4m3(x * fp32(1/q_scale)) * q_scale, the
    keys' quantiser.  Returns ``(out [R,Hq,d] f64, lse [R,Hq] f64, pairs
    [R,Hq] i64)``.
    """
    lib = _load()
    if q_fp8 is not None and fp8 is None:
        raise ValueError("fp8 products (q_fp8) need an fp8 cache (fp8)")
    G = num_q_heads // num_kv_heads
    if G > 64 or num_q_heads % num_kv_heads:
        raise ValueError("oracle supports Hq % Hkv == 0 and G <= 64")
    rows = _i32(rows)
    R = int(rows.shape[0])
    out = np.zeros((R, num_q_heads, head_dim), np.float64)
    lse = np.zeros((R, num_q_heads), np.float64)
    pairs = np.zeros((R, num_q_heads), np.int64)
    arrs = [np.ascontiguousarray(a) if a is not None else None for a in (q, k_new, v_new, k_pool, v_pool)]
    bt = _i32(block_table)
    cu = _i32(cu_seqlens_q)
    cl = _i32(cache_len)
    rc = lib.csr_oracle_attention(
        dtype, num_q_heads, num_kv_heads, head_dim, page_size, 0.0 if scale is None else float(scale),
        *_rope_args(rope, head_dim), *_fp8_args(fp8), 0.0 if q_fp8 is None else float(q_fp8), int(cu.shape[0] - 1),
        *[_ptr(a) for a in arrs], _ptr(bt), int(bt_stride), _ptr(cu), _ptr(cl),
        R, _ptr(rows), _ptr(out), _ptr(lse), _ptr(pairs), int(nthreads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle attention failed ({rc})")
    return out, lse, pairs


def kv_append(k_new, v_new, k_pool, v_pool, block_table, bt_stride, cu_seqlens_q, cache_len,
              num_kv_heads, head_dim, page_size, rope=None, fp8=None):
    """Append oracle, in place on copies: Theorem 2's T (+) dX as a bit copy of
    each chunk row into cache position L_b + i.  With ``rope`` the key rows are
    rotated at that position and rounded to the pool's type (nearest, ties to
    even) instead.  ``fp8=(k_scale, v_scale)``: the pools hold e4m3 codes and
    both keys and values are quantised.  bf16 as uint16 bit patterns.  Returns
    the new pools."""
    lib = _load()
    kp = np.array(k_pool, copy=True)
    vp = np.array(v_pool, copy=True)
    kn = np.ascontiguousarray(k_new)
    vn = np.ascontiguousarray(v_new)
    bt = _i32(block_table)
    cu = _i32(cu_seqlens_q)
    cl = _i32(cache_len)
    dt = {np.dtype(np.uint16): BF16, np.dtype(np.float32): F32}[kn.dtype]
    rc = lib.csr_oracle_kv_append(dt, num_kv_heads, head_dim, page_size, *_rope_args(rope, head_dim),
                                  *_fp8_args(fp8), int(cu.shape[0] - 1),
                                  _ptr(kn), _ptr(vn), _ptr(kp), _ptr(vp), _ptr(bt), int(bt_stride),
                                  _ptr(cu), _ptr(cl))
    if rc != 0:
        raise RuntimeError("oracle append failed")
    return kp, vp
