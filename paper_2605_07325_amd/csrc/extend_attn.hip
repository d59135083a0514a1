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
#include <stdlib.h>

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
//
// K/V tiles move HBM -> LDS with global_load_lds_dwordx4 (no register
// staging): wave w's j-th instruction fills one 1 KB block of the tile, lane i
// writing bytes [16i, 16i+16) of it, so each lane fetches the global chunk that
// the swizzle places in its slot.  Page ids for tile it+1 are loaded while tile
// it is computed.  Keys at or beyond the tile's last visible key are clamped
// to it: they are masked for every row of the tile, and a finite value times a
// zero probability contributes nothing.
//
// Online softmax keeps a per-row reference max and rescales O only when a new
// score exceeds it by more than 2^8 (wave-uniform branch), so the rescale of
// the fp32 accumulators is rare; probabilities stay below 2^8 and the final
// normalisation is exact whatever reference was used.
template <int D, int NB, int NW>
__global__ void __launch_bounds__(NW * 64, 1) attn_bf16_kernel(const AttnArgs a) {
  constexpr int NWAVES = NW;
  constexpr int BM = NWAVES * 32 * NB;
  constexpr int ROWB = D * 2;
  constexpr int NCH = ROWB / 16;
  constexpr int DS = D / 16;  // QK^T contraction steps
  constexpr int DB = D / 32;  // 32-wide d blocks of the output
  constexpr int TILEB = KT * ROWB;
  constexpr int ROWS_PER_KB = 1024 / ROWB;
  constexpr int NDMA = TILEB / (NWAVES * 1024);  // DMA instructions per wave per tensor
  constexpr float THRESH = 8.f;                  // lazy-rescale threshold (log2 units)
  __shared__ __attribute__((aligned(1024))) char lds[2 * 2 * TILEB];  // [buf][K|V]

  Unit u;
  if (!decode_unit<BM>(a, u)) return;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int G = a.G;
  const float c = a.scale_log2;
  const char* __restrict__ kpool = static_cast<const char*>(a.k_pool);
  const char* __restrict__ vpool = static_cast<const char*>(a.v_pool);
  const char* __restrict__ knew = static_cast<const char*>(a.k_new);
  const char* __restrict__ vnew = static_cast<const char*>(a.v_new);
  const int32_t* __restrict__ bt = a.block_table ? a.block_table + (int64_t)u.b * a.bt_stride : nullptr;
  const int64_t bt_base = (int64_t)u.b * a.bt_stride;
  const int log2P = a.log2P, Pmask = (1 << a.log2P) - 1, Hkv = a.Hkv, num_pages = a.num_pages;

  // Q^T fragments: lane holds packed row (l32) of each 32-row block, d = ds*16 + 8h .. +7.
  u32x4 qf[NB][DS];
  int lim[NB];  // last visible key of the lane's row
  bool valid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int m = u.m0 + (wave * NB + nb) * 32 + l32;
    valid[nb] = m < u.rows_total;
    const int i = m / G, j = m - i * G;
    lim[nb] = u.L + i;
    const char* qrow = static_cast<const char*>(a.q) + (((int64_t)(u.cuq + i) * a.Hq + u.g * G + j) * D + h * 8) * 2;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      qf[nb][ds] = valid[nb] ? *reinterpret_cast<const u32x4*>(qrow + ds * 32) : u32x4{0, 0, 0, 0};
  }
  const int wave_first_lim = u.L + (u.m0 + wave * NB * 32) / G;

  // DMA geometry: lane's row within each 1 KB block and its swizzled source chunk.
  int dma_row[NDMA], dma_chunk[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int blk = j * NWAVES + wave;
    dma_row[j] = blk * ROWS_PER_KB + lane / NCH;
    dma_chunk[j] = (lane % NCH) ^ swz<NCH>(dma_row[j]);
  }
  const int last_key = u.kv_end - 1;

  // Byte offset of key row t's chunk for this lane (pool or chunk source).
  auto row_src = [&](int t, int pg, const char*& kb, const char*& vb) -> int64_t {
    t = min(t, last_key);
    if (t < u.L) {
      if (pg >= 0 && pg < num_pages) {
        kb = kpool;
        vb = vpool;
        return ((((int64_t)pg << log2P) + (t & Pmask)) * Hkv + u.g) * ROWB;
      }
      t = u.L;  // invalid page id: never dereferenced, read another valid row instead
    }
    kb = knew;
    vb = vnew;
    return ((int64_t)(u.cuq + t - u.L) * Hkv + u.g) * ROWB;
  };
  auto page_of = [&](int t) -> int {
    t = min(t, last_key);
    if (t >= u.L) return 0;
    const int pidx = t >> log2P;
    return bt ? __ldg(bt + pidx) : (int)(bt_base + pidx);
  };
  auto issue_tile = [&](int tile, const int* pg, int buf) {
    char* kl = lds + buf * 2 * TILEB;
    char* vl = kl + TILEB;
#pragma unroll
    for (int j = 0; j < NDMA; ++j) {
      const char* kb;
      const char* vb;
      const int64_t off = row_src(tile * KT + dma_row[j], pg[j], kb, vb) + dma_chunk[j] * 16;
      const int blk = j * NWAVES + wave;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(kb + off),
                                       (__attribute__((address_space(3))) void*)(kl + blk * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(vb + off),
                                       (__attribute__((address_space(3))) void*)(vl + blk * 1024), 16, 0, 0);
    }
  };

  // Per-lane LDS offsets (buffer and 32-key block offsets are immediates).
  int koff[DS];
  {
    const int sw = swz<NCH>(l32);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) koff[ds] = l32 * ROWB + (((ds * 2 + h) ^ sw) << 4);
  }
  const int grp = lane >> 4, rr = (lane & 15) >> 2, qq = lane & 3, hh = grp >> 1;
  int voff_a[DB], voff_b[DB];
  {
    const int ra = 4 * hh + rr, rb = ra + 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int dcol = db * 32 + 16 * (grp & 1) + 4 * qq;
      const int chunk = dcol >> 3, within = (dcol & 7) * 2;
      voff_a[db] = ra * ROWB + ((chunk ^ swz<NCH>(ra)) << 4) + within;
      voff_b[db] = rb * ROWB + ((chunk ^ swz<NCH>(rb)) << 4) + within;
    }
  }

  f32x16 o[NB][DB];
  float mref[NB], lrow[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    mref[nb] = -INFINITY;
    lrow[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[nb][db] = f32x16{};
  }

  auto compute_tile = [&](const char* kl, int t0, bool masked) {
    const char* vl = kl + TILEB;
    // S^T = K Q^T for two 32-key blocks.
    f32x16 sacc[NB][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) sacc[nb][kb] = f32x16{};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const u32x4 kf = *reinterpret_cast<const u32x4*>(kl + kb * 32 * ROWB + koff[ds]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          sacc[nb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, kf), __builtin_bit_cast(bf16x8, qf[nb][ds]), sacc[nb][kb], 0, 0, 0);
      }
    }
    // Online softmax in the log2 domain with a lazily moved reference max.
    float mxs[NB];
    bool grow = false;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (masked) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int t = t0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (t > lim[nb]) sacc[nb][kb][v] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; v += 2) mx = fmaxf(mx, fmaxf(sacc[nb][kb][v], sacc[nb][kb][v + 1]));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      mxs[nb] = mx * c;
      grow |= mxs[nb] > mref[nb] + THRESH;
    }
    if (__any(grow)) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const float mnew = fmaxf(mref[nb], mxs[nb]);
        const float alpha = fast_exp2((mref[nb] == -INFINITY ? 0.f : mref[nb]) - (mnew == -INFINITY ? 0.f : mnew));
        lrow[nb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[nb][db] *= alpha;
        mref[nb] = mnew;
      }
    }
    u32x4 pf[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const float neg_m = mref[nb] == -INFINITY ? 0.f : -mref[nb];
      float p[2][16];
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          p[kb][v] = fast_exp2(__builtin_fmaf(sacc[nb][kb][v], c, neg_m));
          rs += p[kb][v];
        }
      lrow[nb] += rs;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int kb = ks >> 1, v0 = (ks & 1) * 8;
        pf[nb][ks] = u32x4{pack_bf16x2(p[kb][v0 + 0], p[kb][v0 + 1]), pack_bf16x2(p[kb][v0 + 2], p[kb][v0 + 3]),
                           pack_bf16x2(p[kb][v0 + 4], p[kb][v0 + 5]), pack_bf16x2(p[kb][v0 + 6], p[kb][v0 + 7])};
      }
    }
    // O^T += V^T P^T.  Contraction slot 8h+s of step ks is key
    // kb*32 + 16*(ks&1) + 8*(s/4) + 4h + s%4 (kb = ks/2), matching pf.
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kb = ks >> 1, half = ks & 1;
      const char* vbase = vl + (kb * 32 + 16 * half) * ROWB;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vbase + voff_a[db]));
        const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vbase + voff_b[db]));
        const u32x2 wa = __builtin_bit_cast(u32x2, va);
        const u32x2 wb = __builtin_bit_cast(u32x2, vb);
        const u32x4 vf = u32x4{wa[0], wa[1], wb[0], wb[1]};
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          o[nb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, vf), __builtin_bit_cast(bf16x8, pf[nb][ks]), o[nb][db], 0, 0, 0);
      }
    }
  };

  // Tiles below first_masked need no causal mask for any row of this wave.
  int first_masked = (wave_first_lim + 1) / KT;  // first tile containing a key > wave_first_lim
  first_masked = max(first_masked, u.tb);
  int pg[NDMA], pg_next[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) pg_next[j] = 0;
  if (u.tb < u.te) {
#pragma unroll
    for (int j = 0; j < NDMA; ++j) pg[j] = page_of(u.tb * KT + dma_row[j]);
    issue_tile(u.tb, pg, 0);
    if (u.tb + 1 < u.te) {
#pragma unroll
      for (int j = 0; j < NDMA; ++j) pg[j] = page_of((u.tb + 1) * KT + dma_row[j]);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  __syncthreads();

  for (int it = u.tb; it < u.te; ++it) {
    const int cur = (it - u.tb) & 1;
    if (it + 1 < u.te) {
      issue_tile(it + 1, pg, cur ^ 1);
      if (it + 2 < u.te) {
#pragma unroll
        for (int j = 0; j < NDMA; ++j) pg_next[j] = page_of((it + 2) * KT + dma_row[j]);
      }
    }
    compute_tile(lds + cur * 2 * TILEB, it * KT, it >= first_masked);
#pragma unroll
    for (int j = 0; j < NDMA; ++j) pg[j] = pg_next[j];
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // Epilogue: combine the two half-rows' sums, normalise, write o and lse (or split partials).
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float lsum = lrow[nb] + __shfl_xor(lrow[nb], 32);
    if (!valid[nb]) continue;
    const int m = u.m0 + (wave * NB + nb) * 32 + l32;
    const int i = m / G, j = m - i * G;
    const int64_t qrow = (int64_t)(u.cuq + i) * a.Hq + u.g * G + j;
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    const float lse = lsum > 0.f ? (mref[nb] + __log2f(lsum)) * LN2 : -INFINITY;
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

// bf16 launch shapes: 4 waves x 64 rows (one wave per SIMD) or 8 waves x 32
// rows (two waves per SIMD, so one wave's softmax overlaps the other's MFMAs).
// Both cover 256 packed rows per workgroup.
constexpr int BF16_BM = 256;

int bf16_variant() {
  static int v = -1;
  if (v < 0) {
    const char* e = getenv("CSR_ATTN_VARIANT");  // tuning override
    v = (e && atoi(e) == 0) ? 0 : 1;
  }
  return v;
}

}  // namespace

int attn_block_m(int dtype_bf16, int d) {
  (void)d;
  return dtype_bf16 ? BF16_BM : NWAVES * 32;
}

hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, hipStream_t stream) {
  if (a.n_units == 0) return hipSuccess;
  unsigned grid = (unsigned)a.n_units;
  if (a.xcd_remap) grid = (grid + 7u) & ~7u;
  if (dtype_bf16) {
    if (bf16_variant() == 1) {
      if (a.d == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, 1, 8>), dim3(grid), dim3(512), 0, stream, a);
      else hipLaunchKernelGGL((attn_bf16_kernel<64, 1, 8>), dim3(grid), dim3(512), 0, stream, a);
    } else {
      if (a.d == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, 2, 4>), dim3(grid), dim3(256), 0, stream, a);
      else hipLaunchKernelGGL((attn_bf16_kernel<64, 2, 4>), dim3(grid), dim3(256), 0, stream, a);
    }
  } else {
    if (a.d == 128) hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(grid), dim3(NTHREADS), 0, stream, a);
    else hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(grid), dim3(NTHREADS), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace csr
