// Rotary position embedding (RoFormer, Su et al. 2021) at absolute cache
// positions and FP8 (OCP e4m3) quantisation of the K/V cache, fused with the
// paged KV append.
//
// With an fp8 cache each key (after its rotation) and value is stored as
// e4m3(clamp(x * inv_scale, +-448)), nearest even, inv_scale = fp32(1/scale);
// the quantised chunk rows also go to the workspace, so the attention reads a
// chunk key exactly as later calls will read it from the cache.  In the
// fp8-product mode the (rotated) query rows are quantised the same way into
// the workspace (without RoPE they are only quantised: no pair is rotated).
//
// Chunk row i of sequence b sits at position pos = L_b + i, fixed for as long
// as the row stays cached (prefix stability, Theorem 1), so its query and key
// are rotated once, here, and the rotated key is what the cache keeps
// (append-only growth, Theorem 2).
//
// Grid: x = token, y = slices of that token's 8-element pieces.  Short chunks
// (decode) spread one token over several workgroups, one piece per thread;
// long ones use one workgroup per token that loops over its pieces, so the
// angles are formed once per token.  The token's sequence and position are
// uniform over the workgroup.  The first r/2 threads form (cos, sin) of each
// pair angle pos * theta_i into LDS in fp64 (theta_i comes from the host as
// the double pow(theta, -2i/r)).  Every thread then takes 8-element pieces of
// the token's rows: a neox piece rotates elements [e, e+8) against
// [e + r/2, e + r/2 + 8), an interleaved piece rotates the four pairs inside
// [e, e+8), tail pieces (dims >= r) and value rows are copied bit for bit.
// The result is the fp64 rotation (x cos - x' sin, each product rounded, no
// fused multiply-add) rounded once to the element type: fp32 by the plain
// conversion; an fp8 code from the fp32 value; bf16 nearest even.  For bf16
// results an fp32 rotation is used wherever it provably rounds to the same
// bf16 (almost every element), and the fp64 rotation, rounded to odd in fp32,
// elsewhere.  The rotated values therefore depend on the inputs and
// on how closely cos and sin are evaluated, not on any fp32 intermediate.
// Loads and stores are 16 bytes per lane, and consecutive lanes take
// consecutive pieces of a row.
#include "kernels.h"

namespace csr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int token_sequence(const int32_t* __restrict__ cu, int batch, int tok) {
  int lo = 0, hi = batch - 1;  // largest b with cu[b] <= tok
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= tok) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));  // nearest, ties to even
}

// 8 consecutive elements as floats (BF16: one 16-byte load; fp32: two).
template <bool BF16>
__device__ __forceinline__ void load8(const void* base, int64_t e, float (&x)[8]) {
  if constexpr (BF16) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + e);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[2 * j] = lo_bf16(w[j]);
      x[2 * j + 1] = hi_bf16(w[j]);
    }
  } else {
    // Loaded as float vectors: a bit cast of one element of an integer vector
    // would read element 0 (clang lowers it through the vector's address).
    const f32x4* p = reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + e);
    const f32x4 a = p[0], b = p[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = a[j];
      x[4 + j] = b[j];
    }
  }
}

// fp32 value of v rounded to odd: toward zero, with the lowest bit set when
// inexact.  fp32 keeps 16 more bits than bf16 in the normal and the subnormal
// range, so rounding this value to bf16 (nearest, ties to even) rounds v
// itself once.  From 2^-126 up (and for zeros, infinities and NaNs) the low
// 29 fraction bits of the fp64 pattern are folded into one sticky bit at the
// fp32 unit, after which the conversion to fp32 is exact (or overflows to
// infinity, as v's own rounding to bf16 does); below 2^-126 fp32 steps are
// coarser and a compare against the nearest-even conversion decides.
__device__ __forceinline__ float f32_round_odd(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t hi = (uint32_t)(b >> 32);
  uint32_t lo = (uint32_t)b;
  if (((hi >> 20) & 0x7FFu) >= 897u || (b << 1) == 0) {
    lo = (lo & 0xE0000000u) | ((lo & 0x1FFFFFFFu) != 0u ? 0x20000000u : 0u);
    return (float)__longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
  }
  const float t = (float)v;  // nearest even
  const double back = (double)t;
  uint32_t tb = __float_as_uint(t);
  if (back != v) {
    if (fabs(back) > fabs(v)) tb -= 1;  // rounded away from zero: one step back
    tb |= 1u;
  }
  return __uint_as_float(tb);
}

// bf16 bit patterns of the nearest bf16 values to v0, v1 (ties to even),
// rounded once from fp64; a NaN gives the quiet NaN 0x7fc0.
__device__ __forceinline__ uint32_t bf16x2_bits_of(double v0, double v1) {
  uint32_t w = pack_bf16x2(f32_round_odd(v0), f32_round_odd(v1));
  if ((w & 0x7fffu) > 0x7f80u) w = (w & 0xffff0000u) | 0x7fc0u;
  if ((w & 0x7fff0000u) > 0x7f800000u) w = (w & 0x0000ffffu) | 0x7fc00000u;
  return w;
}

// The fp32 rotation of a bf16 pair decides the bf16 result when it lies far
// enough from every bf16 rounding midpoint.  With c32 = fp32(c), s32 = fp32(s),
// y = fma(u0, c32, -fp32(u1 s32)) differs from the fp64 rotation
// fl(fl(u0 c) - fl(u1 s)) by at most 2^-22 (|u0| + |u1|) (three fp32
// roundings of terms bounded by |u0| + |u1|, plus the fp64 ones); in fp32
// units of y that is at most 4 m / |y|, m = |u0| + |u1|.  All bf16 midpoints
// of y's binade sit where the low 16 bits of y are 0x8000 (the nearest ones
// outside it are 2^14 units away), so a normal, finite y whose low half is
// more than that bound (with margins for this test's own roundings) from
// 0x8000 rounds to the same bf16 as the fp64 value.
__device__ __forceinline__ bool bf16_decided(float y, float m) {
#pragma clang fp contract(off)
  const uint32_t bits = __float_as_uint(y) & 0x7fffffffu;
  const uint32_t ex = bits >> 23;                  // biased exponent: 1 .. 254 for normal, finite y
  const uint32_t low = bits & 0xffffu;
  const uint32_t dist = low > 0x8000u ? low - 0x8000u : 0x8000u - low;
  // the bound in fp32 units of y: 2^-22 m / 2^(e - 23) = m 2^(1 - e), e = ex - 127
  const float bound = __builtin_ldexpf(m, 128 - (int)ex);
  // bitwise, not short-circuit: no branches on the common path
  return (ex - 1u < 254u) & ((float)dist > bound * 1.01f + 2.f) & (bound < 8000.f);
}

// Rotated bf16 pair (u0 c - u1 s, u1 c + u0 s) as fp32 values whose nearest-even
// bf16 is the fp64 rotation rounded once: the fp32 rotation where it decides
// the result, else the fp64 rotation rounded to odd.
__device__ __forceinline__ void rotate_bf16_pair(float u0, float u1, f32x2 t32, f64x2 t64, float& ya, float& yb) {
#pragma clang fp contract(off)
  const float q1 = u1 * t32[1], q0 = u0 * t32[1];
  ya = fmaf(u0, t32[0], -q1);
  yb = fmaf(u1, t32[0], q0);
  const float m = fabsf(u0) + fabsf(u1);
  if (!(bf16_decided(ya, m) & bf16_decided(yb, m))) {
    const double d0 = u0, d1 = u1;
    ya = f32_round_odd(d0 * t64[0] - d1 * t64[1]);
    yb = f32_round_odd(d1 * t64[0] + d0 * t64[1]);
    // NaNs as the quiet NaN whose bf16 is 0x7fc0
    if (ya != ya) ya = __uint_as_float(0x7fc00000u);
    if (yb != yb) yb = __uint_as_float(0x7fc00000u);
  }
}

template <bool BF16>
__device__ __forceinline__ void store8d(void* base, int64_t e, const double (&y)[8]) {
  if constexpr (BF16) {
    const u32x4 w = {bf16x2_bits_of(y[0], y[1]), bf16x2_bits_of(y[2], y[3]), bf16x2_bits_of(y[4], y[5]),
                     bf16x2_bits_of(y[6], y[7])};
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(base) + e) = w;
  } else {
    f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(base) + e);
    p[0] = f32x4{(float)y[0], (float)y[1], (float)y[2], (float)y[3]};
    p[1] = f32x4{(float)y[4], (float)y[5], (float)y[6], (float)y[7]};
  }
}

template <bool BF16>
__device__ __forceinline__ void store8(void* base, int64_t e, const float (&y)[8]) {
  if constexpr (BF16) {
    const u32x4 w = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                     pack_bf16x2(y[6], y[7])};
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(base) + e) = w;
  } else {
    f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(base) + e);
    p[0] = f32x4{y[0], y[1], y[2], y[3]};
    p[1] = f32x4{y[4], y[5], y[6], y[7]};
  }
}

// OCP e4m3 code of x: saturate to +-448, round to nearest even (subnormal
// steps of 2^-9), NaN to 0x7f.  Rounds the fp32 bit pattern at the 3-bit
// mantissa (a carry moves the exponent up, which is the correct result).
__device__ __forceinline__ uint32_t e4m3_code(float x) {
  if (x != x) return 0x7f;
  const uint32_t sign = (__float_as_uint(x) >> 24) & 0x80;
  const float a = fminf(fabsf(x), 448.f);
  if (a < 0.015625f) return sign | (uint32_t)rintf(a * 512.f);  // exact scaling; 8 = smallest normal
  const uint32_t b = __float_as_uint(a);
  const uint32_t r = b + 0x7FFFFu + ((b >> 20) & 1u);
  return sign | (((r >> 23) - 120u) << 3) | ((r >> 20) & 7u);
}

// 8 values scaled by inv and quantised, stored as 8 bytes.
__device__ __forceinline__ void store8q(void* base, int64_t e, const float (&y)[8], float inv) {
  uint32_t w[2] = {0, 0};
#pragma unroll
  for (int j = 0; j < 8; ++j) w[j >> 2] |= e4m3_code(y[j] * inv) << (8 * (j & 3));
  *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(base) + e) = u32x2{w[0], w[1]};
}

// 8 fp64 values, each rounded to fp32, scaled by inv and quantised.
__device__ __forceinline__ void store8qd(void* base, int64_t e, const double (&y)[8], float inv) {
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)y[j];
  store8q(base, e, f, inv);
}

// Bit copy of 8 elements (tail dims, value rows).
template <bool BF16>
__device__ __forceinline__ void copy8(void* dst, const void* src, int64_t de, int64_t se) {
  constexpr int kWords = BF16 ? 1 : 2;
  const u32x4* s = reinterpret_cast<const u32x4*>(static_cast<const char*>(src) + se * (BF16 ? 2 : 4));
  u32x4* d = reinterpret_cast<u32x4*>(static_cast<char*>(dst) + de * (BF16 ? 2 : 4));
#pragma unroll
  for (int j = 0; j < kWords; ++j) d[j] = s[j];
}

template <bool BF16, bool KV8>
__device__ __forceinline__ void rotate_piece(const RopeArgs& a, const f64x2* cs, const f32x2* cs32, int tok,
                                             int64_t slot, int u,
                                             int rot_units, int per_row, int n_rot, int nq, bool neox) {
#pragma clang fp contract(off)
  const int d = a.d;
  const int half = a.rdim >> 1;
  if (u >= rot_units) {  // value row piece: into the cache (and, quantised, the workspace)
    const int w = u - rot_units;
    const int g = w / (d >> 3), e = (w - g * (d >> 3)) << 3;
    const int64_t src = ((int64_t)tok * a.Hkv + g) * d + e;
    if constexpr (KV8) {
      float x[8];
      load8<BF16>(a.v, src, x);
      if (a.v_out) store8q(a.v_out, src, x, a.inv_v);
      if (slot >= 0) store8q(a.v_pool, (slot * a.Hkv + g) * d + e, x, a.inv_v);
    } else {
      copy8<BF16>(a.v_pool, a.v, (slot * a.Hkv + g) * d + e, src);
    }
    return;
  }
  const int r = u / per_row, piece = u - r * per_row;
  const bool is_q = r < nq;
  const int h = is_q ? r : r - nq;
  const void* src = is_q ? a.q : a.k;
  const int64_t row = ((int64_t)tok * (is_q ? a.Hq : a.Hkv) + h) * d;
  void* out = is_q ? a.q_out : a.k_out;
  void* pool = is_q ? nullptr : (slot >= 0 ? a.k_pool : nullptr);
  const int64_t prow = is_q ? 0 : (slot * a.Hkv + h) * d;
  // Keys of an fp8 cache are stored as codes; so are queries in the fp8-product mode.
  const bool quant = KV8 && (!is_q || a.q8);
  const float inv = is_q ? a.inv_q : a.inv_k;
  auto put = [&](void* base, int64_t e, const float (&y)[8]) {
    if (quant) store8q(base, e, y, inv);
    else store8<BF16>(base, e, y);
  };
  auto putd = [&](void* base, int64_t e, const double (&y)[8]) {
    if (quant) store8qd(base, e, y, inv);
    else store8d<BF16>(base, e, y);
  };
  if (piece >= n_rot) {  // dims >= r: unchanged (quantised for an fp8 cache)
    const int e = a.rdim + ((piece - n_rot) << 3);
    if (quant) {
      float x[8];
      load8<BF16>(src, row + e, x);
      if (out) put(out, row + e, x);
      if (pool) put(pool, prow + e, x);
    } else {
      if (out) copy8<BF16>(out, src, row + e, row + e);
      if (pool) copy8<BF16>(pool, src, prow + e, row + e);
    }
    return;
  }
  // x cos - x' sin and x' cos + x sin in fp64, each product rounded separately
  // (no contraction into fused multiply-adds: see the pragma at the top).
  if (neox) {
    const int e0 = piece << 3, e1 = e0 + half;
    float x0[8], x1[8];
    double y0[8], y1[8];
    load8<BF16>(src, row + e0, x0);
    load8<BF16>(src, row + e1, x1);
    if (BF16 && !quant) {  // bf16 results: fp32 rotation, fp64 where it does not decide the rounding
      float z0[8], z1[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) rotate_bf16_pair(x0[j], x1[j], cs32[e0 + j], cs[e0 + j], z0[j], z1[j]);
      if (out) {
        store8<true>(out, row + e0, z0);
        store8<true>(out, row + e1, z1);
      }
      if (pool) {
        store8<true>(pool, prow + e0, z0);
        store8<true>(pool, prow + e1, z1);
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const f64x2 t = cs[e0 + j];
      const double u0 = x0[j], u1 = x1[j];
      y0[j] = u0 * t[0] - u1 * t[1];
      y1[j] = u1 * t[0] + u0 * t[1];
    }
    if (out) {
      putd(out, row + e0, y0);
      putd(out, row + e1, y1);
    }
    if (pool) {
      putd(pool, prow + e0, y0);
      putd(pool, prow + e1, y1);
    }
  } else {
    const int e0 = piece << 3;
    float x[8];
    double y[8];
    load8<BF16>(src, row + e0, x);
    if (BF16 && !quant) {
      float z[8];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        rotate_bf16_pair(x[2 * j], x[2 * j + 1], cs32[(e0 >> 1) + j], cs[(e0 >> 1) + j], z[2 * j], z[2 * j + 1]);
      if (out) store8<true>(out, row + e0, z);
      if (pool) store8<true>(pool, prow + e0, z);
      return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f64x2 t = cs[(e0 >> 1) + j];
      const double u0 = x[2 * j], u1 = x[2 * j + 1];
      y[2 * j] = u0 * t[0] - u1 * t[1];
      y[2 * j + 1] = u1 * t[0] + u0 * t[1];
    }
    if (out) putd(out, row + e0, y);
    if (pool) putd(pool, prow + e0, y);
  }
}

template <bool BF16, bool KV8>
__global__ void __launch_bounds__(256) rope_append_kernel(RopeArgs a) {
  __shared__ f64x2 cs[64];
  __shared__ f32x2 cs32[64];
  const int tok = blockIdx.x;
  const int b = token_sequence(a.cu_q, a.batch, tok);
  const int64_t pos = (int64_t)(a.cache_len ? a.cache_len[b] : 0) + (tok - a.cu_q[b]);
  const int half = a.rdim >> 1;
  if ((int)threadIdx.x < half) {
    const double angle = (double)pos * a.inv_freq[threadIdx.x];
    double s, c;
    sincos(angle, &s, &c);
    cs[threadIdx.x] = f64x2{c, s};
    cs32[threadIdx.x] = f32x2{(float)c, (float)s};
  }

  // Cache slot of this token (pool writes only); an invalid page drops them.
  int64_t slot = -1;
  if (a.k_pool) {
    const int64_t pidx = pos >> a.log2P;
    const int64_t page = a.block_table ? (int64_t)a.block_table[(int64_t)b * a.bt_stride + pidx]
                                       : (int64_t)b * a.bt_stride + pidx;
    if (page >= 0 && page < a.num_pages) slot = (page << a.log2P) + (pos & ((1 << a.log2P) - 1));
  }
  __syncthreads();

  const int d = a.d;
  const bool neox = a.style == 1;
  const int n_rot = neox ? a.rdim >> 4 : a.rdim >> 3;  // rotating pieces per row
  const int per_row = n_rot + ((d - a.rdim) >> 3);      // + tail pieces
  const int nq = a.q ? a.Hq : 0;
  const int rows = nq + a.Hkv;
  const int rot_units = rows * per_row;
  const int v_units = (slot >= 0 || (KV8 && a.v_out)) ? a.Hkv * (d >> 3) : 0;

  for (int u = blockIdx.y * blockDim.x + threadIdx.x; u < rot_units + v_units; u += gridDim.y * blockDim.x)
    rotate_piece<BF16, KV8>(a, cs, cs32, tok, slot, u, rot_units, per_row, n_rot, nq, neox);
}

}  // namespace

hipError_t launch_rope_append(const RopeArgs& a, int dtype_bf16, hipStream_t stream) {
  if (a.total_q == 0) return hipSuccess;
  // Upper bound of the pieces one token has (rows * pieces per row + value pieces).
  const int pieces_per_row = (a.style == 1 ? a.rdim / 16 : a.rdim / 8) + (a.d - a.rdim) / 8;
  const bool v_rows = a.k_pool || (a.kv8 && a.v_out);
  const int units = ((a.q ? a.Hq : 0) + a.Hkv) * pieces_per_row + (v_rows ? a.Hkv * (a.d / 8) : 0);
  // Slices per token: enough workgroups (~2048) to spread a short chunk over
  // the chip, one when the chunk alone provides them.
  const int max_slices = (units + 255) / 256;
  int slices = (2048 + a.total_q - 1) / a.total_q;
  if (slices > max_slices) slices = max_slices;
  const dim3 grid((unsigned)a.total_q, (unsigned)slices);
  if (a.kv8) hipLaunchKernelGGL((rope_append_kernel<true, true>), grid, dim3(256), 0, stream, a);
  else if (dtype_bf16) hipLaunchKernelGGL((rope_append_kernel<true, false>), grid, dim3(256), 0, stream, a);
  else hipLaunchKernelGGL((rope_append_kernel<false, false>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace csr
