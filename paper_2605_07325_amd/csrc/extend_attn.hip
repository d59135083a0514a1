// Cached-prefix extend attention for gfx950 (MI355X).
//
// Definition (paper Sec. II, eq. (causal_attention_1)-(causal_attention_3)):
// chunk row i of sequence b attends to keys 0 .. L_b + i; keys below L_b come
// from the paged cache, the rest from the chunk's own K/V rows.
//
// Work decomposition
//   * Grouped-query packing: the G = Hq/Hkv query heads that share kv head g
//     are packed into the M dimension, packed row m = i * G + j (chunk row i,
//     head g*G + j).  One workgroup owns BM packed rows of one (sequence, kv
//     head), so every K/V tile it stages in LDS feeds G query heads.
//   * A unit is (sequence, kv head, key split, row tile).  Split-K cuts the key
//     range of long prefixes when there are too few row tiles to fill 256 CUs;
//     partial (o, lse) go to the workspace and a merge kernel combines them.
//   * XCD-aware order: workgroup ids are dealt round-robin over the 8 XCDs, so
//     the unit index is remapped to give each XCD a contiguous range of units;
//     units sharing a K/V stream then share that XCD's L2.
//
// Per-tile math (one wave = NB blocks of 32 packed rows; 64 keys per tile)
//   S^T = K Q^T with v_mfma_f32_32x32x16_bf16: A = K tile from LDS, B = Q^T in
//   registers.  The accumulator layout gives each lane one packed row (lane
//   mod 32) and 16 keys, so the softmax row statistics are lane-local except
//   for one exchange between lanes l and l^32.
//   O^T += V^T P^T: the probabilities stay in registers and are exactly the B
//   operand (row = lane mod 32, 8 keys per lane); V^T comes from LDS with
//   ds_read_b64_tr_b16, which transposes 4x16 bf16 blocks on the way out.  The
//   key order inside each 16-key contraction step is permuted consistently on
//   both operands.  O^T keeps each lane on its own row, so the online-softmax
//   rescale is lane-local too.
//   Softmax runs in the log2 domain: scores are scaled by scale*log2(e) and
//   exponentiated with v_exp_f32.
//
// LDS: K and V tiles (64 keys x d) double-buffered; 16-byte chunks of each key
// row are XOR-swizzled by row so both the 16-byte K reads (32 rows, one chunk)
// and the transposing V reads (4 rows x 32 bytes) spread over the banks.
//
// An fp32 instance uses v_mfma_f32_32x32x2f32 with the same layout scheme and
// never rounds through bf16.
#include "kernels.h"

namespace csr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int KT = 64;        // keys per tile
constexpr int NTHREADS = 256;  // 4 waves
constexpr int NWAVES = 4;
constexpr float LN2 = 0.693147180559945309f;

// XOR swizzle of the 16-byte chunk index within a key row (NCH chunks per row).
template <int NCH>
__device__ __forceinline__ int swz(int row) {
  if constexpr (NCH >= 16) return ((row & 7) << 1) | ((row >> 3) & 1);
  else return ((row & 3) << 1) | ((row >> 2) & 1);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  bf16x2 v = __builtin_convertvector(f, bf16x2);  // v_cvt_pk_bf16_f32, round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Everything a workgroup needs about its unit.
struct Unit {
  int b, g, s;
  int cuq, n, L;
  int rows_total;  // n * G packed rows in this sequence
  int m0;          // first packed row of the tile
  int kv_end;      // keys [0, kv_end) can be visible to some row of the tile
  int tb, te;      // key tiles [tb, te) of this split
};

template <int BM>
__device__ __forceinline__ bool decode_unit(const AttnArgs& a, Unit& u) {
  const int w = blockIdx.x;
  int r = w;
  if (a.xcd_remap) {
    const int q8 = gridDim.x >> 3;  // grid is padded to a multiple of 8
    r = (w & 7) * q8 + (w >> 3);
  }
  if (r >= a.n_units) return false;
  int mt = r % a.mtiles;
  int rest = r / a.mtiles;
  u.s = rest % a.nsplit;
  rest /= a.nsplit;
  u.g = rest % a.Hkv;
  u.b = rest / a.Hkv;
  mt = a.mtiles - 1 - mt;  // later rows see more keys: issue them first
  u.cuq = a.cu_q[u.b];
  u.n = a.cu_q[u.b + 1] - u.cuq;
  u.L = a.cache_len ? a.cache_len[u.b] : 0;
  u.rows_total = u.n * a.G;
  u.m0 = mt * BM;
  if (u.m0 >= u.rows_total) return false;
  const int m_last = min(u.m0 + BM, u.rows_total) - 1;
  u.kv_end = u.L + m_last / a.G + 1;
  const int ntiles = (u.kv_end + KT - 1) / KT;
  const int per = (ntiles + a.nsplit - 1) / a.nsplit;
  u.tb = u.s * per;
  u.te = min(ntiles, u.tb + per);
  return true;
}

// Global -> register -> LDS staging of one K tile and one V tile (64 keys).
template <int D, int ESZ>
struct TileLoader {
  static constexpr int ROWB = D * ESZ;
  static constexpr int NCH = ROWB / 16;
  static constexpr int PER_THREAD = KT * NCH / NTHREADS;
  static constexpr int ROWS_PER_PASS = NTHREADS / NCH;
  u32x4 kr[PER_THREAD], vr[PER_THREAD];

  __device__ __forceinline__ void load(const AttnArgs& a, const Unit& u, int t0) {
    const int chunk = threadIdx.x % NCH;
    const int row0 = threadIdx.x / NCH;
#pragma unroll
    for (int j = 0; j < PER_THREAD; ++j) {
      const int t = t0 + row0 + j * ROWS_PER_PASS;
      kr[j] = u32x4{0, 0, 0, 0};
      vr[j] = u32x4{0, 0, 0, 0};
      if (t < u.kv_end) {
        const char* kb;
        const char* vb;
        int64_t row;
        bool ok = true;
        if (t < u.L) {
          const int pidx = t >> a.log2P;
          const int64_t page = a.block_table ? (int64_t)a.block_table[(int64_t)u.b * a.bt_stride + pidx]
                                             : (int64_t)u.b * a.bt_stride + pidx;
          ok = page >= 0 && page < a.num_pages;
          row = ((page << a.log2P) + (t & ((1 << a.log2P) - 1))) * a.Hkv + u.g;
          kb = static_cast<const char*>(a.k_pool);
          vb = static_cast<const char*>(a.v_pool);
        } else {
          row = (int64_t)(u.cuq + t - u.L) * a.Hkv + u.g;
          kb = static_cast<const char*>(a.k_new);
          vb = static_cast<const char*>(a.v_new);
        }
        if (ok) {
          const int64_t off = row * ROWB + chunk * 16;
          kr[j] = *reinterpret_cast<const u32x4*>(kb + off);
          vr[j] = *reinterpret_cast<const u32x4*>(vb + off);
        }
      }
    }
  }

  __device__ __forceinline__ void store(char* kl, char* vl) const {
    const int chunk = threadIdx.x % NCH;
    const int row0 = threadIdx.x / NCH;
#pragma unroll
    for (int j = 0; j < PER_THREAD; ++j) {
      const int row = row0 + j * ROWS_PER_PASS;
      const int off = row * ROWB + ((chunk ^ swz<NCH>(row)) << 4);
      *reinterpret_cast<u32x4*>(kl + off) = kr[j];
      *reinterpret_cast<u32x4*>(vl + off) = vr[j];
    }
  }
};

// ---------------------------------------------------------------------------
// bf16 inputs, fp32 accumulation.
template <int D, int NB>
__global__ void __launch_bounds__(NTHREADS, 1) attn_bf16_kernel(AttnArgs a) {
  constexpr int BM = NWAVES * 32 * NB;
  constexpr int ROWB = D * 2;
  constexpr int NCH = ROWB / 16;
  constexpr int DS = D / 16;  // QK^T contraction steps
  constexpr int DB = D / 32;  // 32-wide d blocks of the output
  __shared__ __attribute__((aligned(16))) char lds[2][2][KT * ROWB];

  Unit u;
  if (!decode_unit<BM>(a, u)) return;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int G = a.G;

  // Q^T fragments: lane holds packed row (l32) of each 32-row block, d = ds*16 + 8h .. +7.
  u32x4 qf[NB][DS];
  int tok[NB];
  bool valid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int m = u.m0 + (wave * NB + nb) * 32 + l32;
    valid[nb] = m < u.rows_total;
    const int i = m / G, j = m - (m / G) * G;
    tok[nb] = i;
    const char* qrow = static_cast<const char*>(a.q) +
                       (((int64_t)(u.cuq + i) * a.Hq + u.g * G + j) * D + h * 8) * 2;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      qf[nb][ds] = valid[nb] ? *reinterpret_cast<const u32x4*>(qrow + ds * 32) : u32x4{0, 0, 0, 0};
  }
  const int wave_first_tok = (u.m0 + wave * NB * 32) / G;

  f32x16 o[NB][DB];
  float mrow[NB], lrow[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    mrow[nb] = -INFINITY;
    lrow[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[nb][db] = f32x16{};
  }

  TileLoader<D, 2> ld;
  if (u.tb < u.te) {
    ld.load(a, u, u.tb * KT);
    ld.store(lds[0][0], lds[0][1]);
  }
  __syncthreads();

  // Per-lane constants of the transposing V read: group of 16 lanes, row r within 4, column quad q.
  const int grp = lane >> 4;
  const int rr = (lane & 15) >> 2;
  const int qq = lane & 3;
  const int hh = grp >> 1;

  for (int it = u.tb; it < u.te; ++it) {
    const int cur = (it - u.tb) & 1;
    const bool has_next = it + 1 < u.te;
    if (has_next) ld.load(a, u, (it + 1) * KT);
    const char* kl = lds[cur][0];
    const char* vl = lds[cur][1];
    const int t0 = it * KT;

    // S^T = K Q^T for two 32-key blocks.
    f32x16 sacc[NB][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) sacc[nb][kb] = f32x16{};
      const int row = kb * 32 + l32;
      const char* kp = kl + row * ROWB;
      const int sw = swz<NCH>(row);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const u32x4 kf = *reinterpret_cast<const u32x4*>(kp + (((ds * 2 + h) ^ sw) << 4));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          sacc[nb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, kf), __builtin_bit_cast(bf16x8, qf[nb][ds]), sacc[nb][kb], 0, 0, 0);
      }
    }

    // Online softmax (log2 domain).
    const bool need_mask = t0 + KT - 1 > u.L + wave_first_tok;
    u32x4 pf[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float sv[2][16];
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = sacc[nb][kb][v] * a.scale_log2;
          if (need_mask) {
            const int t = t0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (t > u.L + tok[nb]) x = -INFINITY;
          }
          sv[kb][v] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(mrow[nb], mx);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = fast_exp2(mrow[nb] - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float p = fast_exp2(sv[kb][v] - m_use);
          sv[kb][v] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 32);
      lrow[nb] = lrow[nb] * alpha + rs;
      mrow[nb] = m_new;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[nb][db] *= alpha;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int kb = ks >> 1, v0 = (ks & 1) * 8;
        pf[nb][ks] = u32x4{pack_bf16x2(sv[kb][v0 + 0], sv[kb][v0 + 1]), pack_bf16x2(sv[kb][v0 + 2], sv[kb][v0 + 3]),
                           pack_bf16x2(sv[kb][v0 + 4], sv[kb][v0 + 5]), pack_bf16x2(sv[kb][v0 + 6], sv[kb][v0 + 7])};
      }
    }

    // O^T += V^T P^T.  Contraction slot 8h+s of step ks is key
    // kb*32 + 16*(ks&1) + 8*(s/4) + 4h + s%4 (kb = ks/2), matching pf.
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kb = ks >> 1, half = ks & 1;
      const int row_a = kb * 32 + 16 * half + 4 * hh + rr;
      const int row_b = row_a + 8;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int dcol = db * 32 + 16 * (grp & 1) + 4 * qq;
        const int chunk = dcol >> 3, within = (dcol & 7) * 2;
        const char* pa = vl + row_a * ROWB + ((chunk ^ swz<NCH>(row_a)) << 4) + within;
        const char* pb = vl + row_b * ROWB + ((chunk ^ swz<NCH>(row_b)) << 4) + within;
        const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(pa));
        const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(pb));
        const u32x2 wa = __builtin_bit_cast(u32x2, va);
        const u32x2 wb = __builtin_bit_cast(u32x2, vb);
        const u32x4 vf = u32x4{wa[0], wa[1], wb[0], wb[1]};
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          o[nb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, vf), __builtin_bit_cast(bf16x8, pf[nb][ks]), o[nb][db], 0, 0, 0);
      }
    }

    if (has_next) ld.store(lds[cur ^ 1][0], lds[cur ^ 1][1]);
    __syncthreads();
  }

  // Epilogue: normalise and write o (bf16) and lse, or the split partials.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (!valid[nb]) continue;
    const int m = u.m0 + (wave * NB + nb) * 32 + l32;
    const int i = tok[nb], j = m - i * G;
    const int64_t qrow = (int64_t)(u.cuq + i) * a.Hq + u.g * G + j;
    const float inv = lrow[nb] > 0.f ? 1.f / lrow[nb] : 0.f;
    const float lse = lrow[nb] > 0.f ? (mrow[nb] + __log2f(lrow[nb])) * LN2 : -INFINITY;
    if (a.nsplit == 1) {
      char* orow = static_cast<char*>(a.out) + qrow * D * 2;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int vg = 0; vg < 4; ++vg) {
          const int d0 = db * 32 + 8 * vg + 4 * h;
          const u32x2 w = {pack_bf16x2(o[nb][db][4 * vg + 0] * inv, o[nb][db][4 * vg + 1] * inv),
                           pack_bf16x2(o[nb][db][4 * vg + 2] * inv, o[nb][db][4 * vg + 3] * inv)};
          *reinterpret_cast<u32x2*>(orow + d0 * 2) = w;
        }
      if (h == 0 && a.lse) a.lse[qrow] = lse;
    } else {
      const int64_t prow = (int64_t)u.s * a.total_q * a.Hq + qrow;
      float* orow = a.part_o + prow * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int vg = 0; vg < 4; ++vg) {
          const int d0 = db * 32 + 8 * vg + 4 * h;
          const f32x4 w = {o[nb][db][4 * vg + 0] * inv, o[nb][db][4 * vg + 1] * inv, o[nb][db][4 * vg + 2] * inv,
                           o[nb][db][4 * vg + 3] * inv};
          *reinterpret_cast<f32x4*>(orow + d0) = w;
        }
      if (h == 0) a.part_lse[prow] = lse;
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 inputs and accumulation: v_mfma_f32_32x32x2f32, one 32-row block per wave.
template <int D>
__global__ void __launch_bounds__(NTHREADS, 1) attn_f32_kernel(AttnArgs a) {
  constexpr int BM = NWAVES * 32;
  constexpr int ROWB = D * 4;
  constexpr int NCH = ROWB / 16;
  constexpr int DS = D / 2;
  constexpr int DB = D / 32;
  __shared__ __attribute__((aligned(16))) char lds[2][2][KT * ROWB];

  Unit u;
  if (!decode_unit<BM>(a, u)) return;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int G = a.G;

  const int m = u.m0 + wave * 32 + l32;
  const bool valid = m < u.rows_total;
  const int tok = m / G, jh = m - (m / G) * G;
  float qf[DS];
  {
    const float* qrow = static_cast<const float*>(a.q) + ((int64_t)(u.cuq + tok) * a.Hq + u.g * G + jh) * D;
#pragma unroll
    for (int st = 0; st < DS; ++st) qf[st] = valid ? qrow[2 * st + h] : 0.f;
  }
  const int wave_first_tok = (u.m0 + wave * 32) / G;

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};
  float mrow = -INFINITY, lrow = 0.f;

  TileLoader<D, 4> ld;
  if (u.tb < u.te) {
    ld.load(a, u, u.tb * KT);
    ld.store(lds[0][0], lds[0][1]);
  }
  __syncthreads();

  for (int it = u.tb; it < u.te; ++it) {
    const int cur = (it - u.tb) & 1;
    const bool has_next = it + 1 < u.te;
    if (has_next) ld.load(a, u, (it + 1) * KT);
    const char* kl = lds[cur][0];
    const char* vl = lds[cur][1];
    const int t0 = it * KT;

    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
      const int row = kb * 32 + l32;
      const char* kp = kl + row * ROWB;
      const int sw = swz<NCH>(row);
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        const int dd = 2 * st + h;
        const float kf = *reinterpret_cast<const float*>(kp + ((((dd >> 2) ^ sw)) << 4) + (dd & 3) * 4);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf, qf[st], sacc[kb], 0, 0, 0);
      }
    }

    const bool need_mask = t0 + KT - 1 > u.L + wave_first_tok;
    float sv[2][16];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = sacc[kb][v] * a.scale_log2;
        if (need_mask) {
          const int t = t0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
          if (t > u.L + tok) x = -INFINITY;
        }
        sv[kb][v] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(mrow, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = fast_exp2(mrow - m_use);
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = fast_exp2(sv[kb][v] - m_use);
        sv[kb][v] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32);
    lrow = lrow * alpha + rs;
    mrow = m_new;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] *= alpha;

    // O^T += V^T P^T, two keys per step: slot h of step (kb, v) is key kb*32 + 8*(v/4) + 4h + v%4.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const char* vp = vl + row * ROWB;
        const int sw = swz<NCH>(row);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int dd = db * 32 + l32;
          const float vv = *reinterpret_cast<const float*>(vp + (((dd >> 2) ^ sw) << 4) + (dd & 3) * 4);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(vv, sv[kb][v], o[db], 0, 0, 0);
        }
      }

    if (has_next) ld.store(lds[cur ^ 1][0], lds[cur ^ 1][1]);
    __syncthreads();
  }

  if (!valid) return;
  const int64_t qrow = (int64_t)(u.cuq + tok) * a.Hq + u.g * G + jh;
  const float inv = lrow > 0.f ? 1.f / lrow : 0.f;
  const float lse = lrow > 0.f ? (mrow + __log2f(lrow)) * LN2 : -INFINITY;
  float* orow = a.nsplit == 1 ? static_cast<float*>(a.out) + qrow * D
                              : a.part_o + ((int64_t)u.s * a.total_q * a.Hq + qrow) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int vg = 0; vg < 4; ++vg) {
      const int d0 = db * 32 + 8 * vg + 4 * h;
      const f32x4 w = {o[db][4 * vg + 0] * inv, o[db][4 * vg + 1] * inv, o[db][4 * vg + 2] * inv,
                       o[db][4 * vg + 3] * inv};
      *reinterpret_cast<f32x4*>(orow + d0) = w;
    }
  if (h == 0) {
    if (a.nsplit == 1) {
      if (a.lse) a.lse[qrow] = lse;
    } else {
      a.part_lse[(int64_t)u.s * a.total_q * a.Hq + qrow] = lse;
    }
  }
}

constexpr int BF16_NB = 2;

}  // namespace

int attn_block_m(int dtype_bf16, int d) {
  (void)d;
  return dtype_bf16 ? NWAVES * 32 * BF16_NB : NWAVES * 32;
}

hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, hipStream_t stream) {
  if (a.n_units == 0) return hipSuccess;
  unsigned grid = (unsigned)a.n_units;
  if (a.xcd_remap) grid = (grid + 7u) & ~7u;
  if (dtype_bf16) {
    if (a.d == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, BF16_NB>), dim3(grid), dim3(NTHREADS), 0, stream, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<64, BF16_NB>), dim3(grid), dim3(NTHREADS), 0, stream, a);
  } else {
    if (a.d == 128) hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(grid), dim3(NTHREADS), 0, stream, a);
    else hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(grid), dim3(NTHREADS), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace csr
