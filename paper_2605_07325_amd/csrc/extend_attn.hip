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
// Per-tile math (one wave = 32 packed rows; 64 keys per tile)
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
// LDS: K and V tiles (64 keys x d) stream through 4-stage rings filled by LDS
// DMA in the bf16 / fp8 kernel and through double buffers in the fp32 one;
// 16-byte chunks of each key row are XOR-swizzled by row so both the 16-byte K
// reads (32 rows, one chunk) and the transposing V reads (4 rows x 32 bytes)
// spread over the banks.
//
// An fp32 instance uses v_mfma_f32_32x32x2f32 with the same layout scheme and
// never rounds through bf16.
#include <stdlib.h>

#include <type_traits>

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
typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;


constexpr int KT = 64;        // keys per tile
constexpr int NTHREADS = 256;  // 4 waves
constexpr int NWAVES = 4;
constexpr float LN2 = 0.693147180559945309f;

// Key rows one page lookup of the bf16-Q kernel covers (a run of one or two
// 1 KB DMA blocks of one wave); the scalar page path needs pages at least this long.
constexpr int dma_rows_per_lookup(int d, bool kv8, int nw, bool dma_upper) {
  const int rowb = d * (kv8 ? 1 : 2);
  const int ndma = KT * rowb / ((dma_upper ? nw / 2 : nw) * 1024);
  return (ndma >= 2 ? 2 : 1) * (1024 / rowb);
}

// XOR swizzle of the 16-byte chunk index within a key row (NCH chunks per row).
template <int NCH>
__device__ __forceinline__ int swz(int row) {
  if constexpr (NCH >= 16) return ((row & 7) << 1) | ((row >> 3) & 1);
  else return ((row & 3) << 1) | ((row >> 2) & 1);
}

// Rows of fp8 keys (128 bytes at d = 128): each 16-lane group of a transposing
// V read touches the 8 key rows {a, a+1, a+2, a+3, a+8, .., a+11}, which
// differ in row bits 0, 1 and 3; the XOR uses exactly those bits (bit 2 folded
// in) so the 8 rows land in 8 different chunk slots.
__device__ __forceinline__ int swz8(int row) {
  return ((row & 3) | ((row >> 1) & 4)) ^ ((row >> 2) & 1);
}

// Slot of 16-byte chunk c in key row `row` of an LDS tile: the row XOR plus,
// for 256-byte rows, a swap of chunk bit 1 into bit 3 so the two 16-lane
// groups of a transposing V read fall into opposite halves of the 64 banks.
// A bijection on the chunks of each row; chunk_of_slot is its inverse.
template <int NCH, bool B8 = false>
__device__ __forceinline__ int slot(int row, int c) {
  if constexpr (B8) return c ^ swz8(row);
  int s = c ^ swz<NCH>(row);
  if constexpr (NCH == 16) s ^= ((c >> 1) & 1) << 3;
  return s;
}
template <int NCH, bool B8 = false>
__device__ __forceinline__ int chunk_of_slot(int row, int s) {
  if constexpr (B8) return s ^ swz8(row);
  int c = s ^ swz<NCH>(row);
  if constexpr (NCH == 16) c ^= ((c >> 1) & 1) << 3;
  return c;
}

// Eight OCP e4m3 codes (bytes in memory order) as eight bf16 values: every
// e4m3 value is exactly a bf16 value, so the conversion is exact.
__device__ __forceinline__ u32x4 e4m3x8_to_bf16(u32x2 w) {
  return u32x4{__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, false)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, true)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, false)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, true))};
}

// A K fragment as the MFMA's eight bf16 values: bf16 fragments as read, fp8
// fragments (8 codes) converted.
__device__ __forceinline__ u32x4 kfrag(u32x4 x) { return x; }
__device__ __forceinline__ u32x4 kfrag(u32x2 x) { return e4m3x8_to_bf16(x); }
template <bool B8> struct KFragT { typedef u32x4 type; };
template <> struct KFragT<true> { typedef u32x2 type; };

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  bf16x2 v = __builtin_convertvector(f, bf16x2);  // v_cvt_pk_bf16_f32, round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS DMA (global_load_lds_dwordx4: 16 bytes per lane, 1 KB per wave) written
// as inline assembly, so that the compiler neither merges the address paths
// nor waits for these loads before unrelated LDS reads; every wait on them is
// explicit.  M0 holds the LDS address; the instruction offset moves the LDS
// and the global address alike, so run member i (LDS m0 + 1024 i) takes a
// per-lane offset that already carries -1024 i.  NT sets the non-temporal
// hint: for K/V that no other workgroup reads again it streams ~15 % faster
// (a 252 MB K/V stream through the same LDS ring: 44.6 -> 38.4 us).
#define CSR_DMA1(NTS) "s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" NTS
#define CSR_DMA2(NTS)                                                                                   \
  "s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %3" NTS "\n\tglobal_load_lds_dwordx4 %2, %3 " \
  "offset:1024" NTS
#define CSR_DMAV(NTS) "s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" NTS
template <int N, bool NT>
__device__ __forceinline__ void dma_sbase(const char* base, uint32_t m0, const uint32_t* voff) {
  static_assert(N == 1 || N == 2, "runs of one or two DMA blocks");
  if constexpr (N == 1 && NT)
    asm volatile(CSR_DMA1(" nt") : : "s"(m0), "v"(voff[0]), "s"(base) : "memory");
  else if constexpr (N == 1)
    asm volatile(CSR_DMA1("") : : "s"(m0), "v"(voff[0]), "s"(base) : "memory");
  else if constexpr (NT)
    asm volatile(CSR_DMA2(" nt") : : "s"(m0), "v"(voff[0]), "v"(voff[1]), "s"(base) : "memory");
  else
    asm volatile(CSR_DMA2("") : : "s"(m0), "v"(voff[0]), "v"(voff[1]), "s"(base) : "memory");
}
template <bool NT>
__device__ __forceinline__ void dma_vaddr(const char* src, uint32_t m0) {
  if constexpr (NT)
    asm volatile(CSR_DMAV(" nt") : : "s"(m0), "v"(src) : "memory");
  else
    asm volatile(CSR_DMAV("") : : "s"(m0), "v"(src) : "memory");
}
#undef CSR_DMA1
#undef CSR_DMA2
#undef CSR_DMAV

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
  // The unit's description is read through the constant address space
  // (scalar loads): every field is then wave-uniform by construction.
  typedef const __attribute__((address_space(4))) int32_t* cptr;
  const int w = blockIdx.x;
  int r = w;
  if (a.order) {
    r = ((cptr)a.order)[w];  // planned on the device (ragged batches): -1 = no unit
    if (r < 0) return false;
  } else if (a.xcd_remap) {
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
  u.cuq = ((cptr)a.cu_q)[u.b];
  u.n = ((cptr)a.cu_q)[u.b + 1] - u.cuq;
  u.L = a.cache_len ? ((cptr)a.cache_len)[u.b] : 0;
  u.rows_total = u.n * a.G;
  u.m0 = mt * BM;
  if (u.m0 >= u.rows_total) return false;
  const int m_last = min(u.m0 + BM, u.rows_total) - 1;
  u.kv_end = u.L + m_last / a.G + 1;
  const int ntiles = (u.kv_end + KT - 1) / KT;
  // Split sizes differ by at most one tile, the larger ones first: the last
  // split holds the diagonal (masked, unpipelined) tiles and gets the smaller share.
  const int q = ntiles / a.nsplit, rem = ntiles - q * a.nsplit;
  u.tb = u.s * q + min(u.s, rem);
  u.te = u.tb + q + (u.s < rem ? 1 : 0);
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
// One workgroup = 8 waves x 32 packed rows; two waves share each SIMD.
//
// K/V tiles (64 keys) move HBM -> LDS with global_load_lds_dwordx4 (no
// register staging) through 4-stage rings: wave w's j-th DMA instruction fills
// one 1 KB block of a tile, lane i writing bytes [16i, 16i+16), so each lane
// fetches the global chunk that lives in its LDS slot.  Tile t is issued three
// tiles before it is processed; each tile waits only for loads older than the
// previous tile's.  When a page holds at least the 4 (d=128) or 8 (d=64) keys
// of one DMA block, the page id is wave-uniform, comes through the scalar
// cache, and the source address is a scalar base plus a per-lane constant.
//
// Main loop (tiles no row of the workgroup needs masked), software-pipelined
// per 32-key block b inside every wave: the exponentials of block b are
// computed while the MFMA pipe works on the scores of block b+1, then the
// block's overflow check and P(b) V(b).  The loop is unrolled over the ring so
// every LDS address is a per-lane register plus an immediate.  The diagonal
// tiles run afterwards, unpipelined, with the causal mask.
//
// Online softmax keeps a per-row reference max.  In the main loop the
// probabilities are formed against it and summed per 16-key half-block; a row
// whose sum passes 2^16 (or is NaN) takes a divergent branch that forms the
// exact row max, moves the reference and rescales O and the row sum.  The first
// tile and the diagonal tiles move the reference when a score exceeds it by
// more than 2^8 (wave-uniform test).  Either way every probability stays below
// 2^16 and the final normalisation is exact whatever reference was used.
// NW waves per workgroup, 2 waves per SIMD either way: 8 (one workgroup per
// CU) or, for an fp8 cache whose 64 KB of rings let two workgroups share a
// CU, 4 -- decode steps then run two computing waves per CU instead of one.
//
// DMA_UPPER (short chunks: every packed row of a unit falls in the lower
// half of the waves): the upper half, which has no rows, issues all of the
// K/V DMA and the computing waves none, so the DMA issue stalls stay off the
// computing waves' per-tile dependency chain.
//
// QK8 (fp8 score products, with KV8): q arrives as e4m3 codes and the scores
// of a 32-key block are two v_mfma_f32_32x32x64_f8f6f4 (d 0..63, 64..127).
// In that instruction lane r + 32h of either operand holds 32 bytes, and A
// and B pair the same byte slots (probed), so both take d = 64i + 32h + b:
// two 16-byte chunks of the key row in LDS, two of the query row.
template <int D, bool SCALAR_PAGES, bool KV8 = false, int NW = 8, bool DMA_UPPER = false, bool QK8 = false>
__global__ void __launch_bounds__(NW * 64, 8 / NW) attn_bf16_kernel(const AttnArgs a) {
  // Profiling hook: the 100 MHz constant clock at the start, stored at once
  // (nothing stays live for it); the end fields follow in the epilogue.
  if (a.wg_clock && threadIdx.x == 0 && (int)blockIdx.x < a.wg_clock_cap)
    a.wg_clock[4 * (size_t)blockIdx.x] = __builtin_amdgcn_s_memrealtime();
  static_assert(!KV8 || D == 128, "fp8 K/V rows are laid out for d = 128");
  static_assert(NW == 8 || (NW == 4 && KV8), "4-wave workgroups only with the 64 KB fp8 rings");
  static_assert(!QK8 || KV8, "fp8 score products need the fp8 cache");
  typedef typename KFragT<KV8 && !QK8>::type KF;  // one K fragment as read from LDS
  constexpr int BM = NW * 32;
  constexpr int ROWB = D * (KV8 ? 1 : 2);  // bytes per key row (bf16 or e4m3 codes)
  constexpr int NCH = ROWB / 16;
  constexpr int DS = D / 16;  // QK^T contraction steps
  constexpr int DB = D / 32;  // 32-wide d blocks of the output
  constexpr int TILEB = KT * ROWB;
  constexpr int ROWS_PER_KB = 1024 / ROWB;
  constexpr int DW = DMA_UPPER ? NW / 2 : NW;  // waves that issue the K/V DMA
  constexpr int NDMA = TILEB / (DW * 1024);    // DMA instructions per issuing wave per tensor tile
  static_assert(NDMA >= 1, "a tile must give every wave at least one DMA block");
  constexpr int PB = NDMA >= 2 ? 2 : 1;        // consecutive blocks per run (one page, one M0)
  constexpr int PG = SCALAR_PAGES ? PB : 1;    // blocks per page lookup
  constexpr int NPG = NDMA / PG;               // page lookups per issuing wave per tile
  constexpr int NG0 = (NPG + 1) / 2;           // lookup groups issued in a tile's first step
  static_assert(!SCALAR_PAGES || PB * ROWS_PER_KB == dma_rows_per_lookup(D, KV8, NW, DMA_UPPER),
                "scalar page lookups cover the rows the launcher checks against the page size");
  // With every row of a unit in one workgroup, no other workgroup reads the
  // unit's K/V tiles: stream them with the non-temporal hint.
  constexpr bool NT_KV = DMA_UPPER;
  constexpr int ST = 4;                      // ring stages (K and V each)
  constexpr float THRESH = 8.f;              // first / diagonal tiles: reference moves past +2^8 (log2 units)
  __shared__ __attribute__((aligned(1024))) char lds[2 * ST * TILEB];

  Unit u;
  if (!decode_unit<BM>(a, u)) return;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // DMA slot of this wave (clamped to 0 for the computing waves when only the
  // upper half loads, so that their unused addresses stay in range too)
  const bool dma_wave = !DMA_UPPER || wave >= NW / 2;
  const int dw = DMA_UPPER ? max(wave - NW / 2, 0) : wave;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int G = a.G;
  const float c = a.scale_log2;
  const char* __restrict__ kpool = static_cast<const char*>(a.k_pool);
  const char* __restrict__ vpool = static_cast<const char*>(a.v_pool);
  const char* __restrict__ knew = static_cast<const char*>(a.k_new);
  const char* __restrict__ vnew = static_cast<const char*>(a.v_new);
  // The block table is read-only for the kernel's lifetime: reading it through
  // the constant address space lets wave-uniform lookups use scalar loads,
  // which the scalar cache serves without queueing behind the K/V DMA.
  typedef const __attribute__((address_space(4))) int32_t* const_i32p;
  const_i32p bt = a.block_table ? (const_i32p)(a.block_table + (int64_t)u.b * a.bt_stride) : nullptr;
  const int bt_base = u.b * a.bt_stride;
  const int log2P = a.log2P, Pmask = (1 << a.log2P) - 1, num_pages = a.num_pages;
  const int kv_stride = a.Hkv * ROWB;  // bytes between consecutive tokens of one kv head
  const int last_key = u.kv_end - 1;

  // Q^T fragment: lane holds packed row (l32), d = ds*16 + 8h .. +7 (bf16);
  // QK8: e4m3 codes of d = 64i + 32h + 16j .. +15 in qf[2i + j].
  constexpr int NQF = QK8 ? 4 : DS;
  u32x4 qf[NQF];
  const int m_row = u.m0 + wave * 32 + l32;
  const bool valid = m_row < u.rows_total;
  // A wave whose 32 rows are all padding (short chunks: n*G < BM) skips the
  // products and exponentials but still issues its share of every K/V DMA
  // and joins every barrier.
  const bool wave_active =
      __builtin_amdgcn_readfirstlane((!DMA_UPPER || wave < NW / 2) && u.m0 + wave * 32 < u.rows_total ? 1 : 0) != 0;
  const int tok = m_row / G;
  const int lim = u.L + tok;  // last key this lane's row sees
  {
    const int j = m_row - tok * G;
    if constexpr (QK8) {
      const char* qrow = static_cast<const char*>(a.q) + ((int64_t)(u.cuq + tok) * a.Hq + u.g * G + j) * D + h * 32;
#pragma unroll
      for (int x = 0; x < 4; ++x)
        qf[x] = valid ? *reinterpret_cast<const u32x4*>(qrow + 64 * (x >> 1) + 16 * (x & 1)) : u32x4{0, 0, 0, 0};
    } else {
      const char* qrow =
          static_cast<const char*>(a.q) + (((int64_t)(u.cuq + tok) * a.Hq + u.g * G + j) * D + h * 8) * 2;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
        qf[ds] = valid ? *reinterpret_cast<const u32x4*>(qrow + ds * 32) : u32x4{0, 0, 0, 0};
    }
    // Take delivery of q here, on every path: the K/V DMA below is invisible
    // to the compiler, which would otherwise wait for "the q loads" with a
    // vmcnt(0) inside the key loop, i.e. for every DMA in flight.
#pragma unroll
    for (int x = 0; x < NQF; ++x) asm volatile("" : "+v"(qf[x]));
  }

  // ---- DMA.  Wave dw loads the 1 KB blocks blk(j) of every K and V tile, j < NDMA: runs of PB
  // consecutive blocks (PB * ROWS_PER_KB consecutive key rows), so that with pages of at least
  // that many keys one page lookup serves a run and one LDS address (M0) with instruction
  // offsets 0 / 1024 serves its DMAs.  Lane's key row within the tile for block j, and its byte
  // offset inside a token row:
  auto blk = [&](int j) { return ((j / PB) * DW + dw) * PB + (j % PB); };
  int drow[NDMA], dchunk[NDMA];
  // Byte offsets of the lane's row inside a page (pool tiles) and inside the
  // chunk's K/V rows (chunk tiles): with 64-key tiles aligned to 64, a page of
  // P <= 64 keys starts the lane's in-page index at drow & (P-1); for P > 64
  // the tile start inside the page is a scalar added separately.  The _v
  // copies carry -1024 (j % PB): the instruction offset of the run's j-th DMA
  // moves the global address by as much as the LDS one.
  uint32_t pool_off[NDMA], new_off[NDMA], pool_v[NDMA], new_v[NDMA];
  const int in_page_mask = min((1 << a.log2P) - 1, KT - 1);
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    drow[j] = blk(j) * ROWS_PER_KB + lane / NCH;
    dchunk[j] = u.g * ROWB + (chunk_of_slot<NCH, KV8>(drow[j], lane % NCH) << 4);
    pool_off[j] = (drow[j] & in_page_mask) * (a.Hkv * ROWB) + dchunk[j];
    new_off[j] = drow[j] * (a.Hkv * ROWB) + dchunk[j];
    pool_v[j] = pool_off[j] - 1024u * (j % PB);
    new_v[j] = new_off[j] - 1024u * (j % PB);
  }
  // Byte offset, from the pool base, of the 64-key-aligned stretch of the page
  // that holds lookup group g of `tile` (PG blocks; wave-uniform in scalar
  // mode, per lane otherwise; unused for chunk keys).  Page ids outside
  // [0, num_pages) read page 0 instead, so a bad table cannot send a load out
  // of bounds.
  const int64_t page_bytes = (int64_t)kv_stride << log2P;
  auto block_key = [&](int tile, int g) -> int {
    if constexpr (SCALAR_PAGES)
      return min(tile * KT + blk(g * PB) * ROWS_PER_KB, last_key);
    else
      return min(tile * KT + drow[g], last_key);
  };
  // Split in two so that the block-table load can be issued well before the
  // offset is needed: page_id loads, page_off does the arithmetic.
  auto page_id = [&](int tile, int g) -> int {
    const int t = block_key(tile, g);
    if (t >= u.L) return 0;
    const int pidx = t >> log2P;
    return bt ? bt[pidx] : bt_base + pidx;
  };
  // Page ids of the prefix loop, with no test or branch: the table entry is
  // loaded (for the contiguous cache, with no table, the first word of
  // cu_seqlens instead) into `raw` and the contiguous cache's page id goes
  // to `alt`; page_pick chooses once the load has landed.
  const_i32p bt_row = bt ? bt : (const_i32p)a.cu_q;
  const int bt_any = bt ? -1 : 0;
  auto page_pick = [&](int raw, int alt) -> int { return bt_any ? raw : alt; };
  // Prefix loop (pages of at most 64 keys, so a tile starts a page): the page
  // index of lookup group g of tile t is (t << pidx_sh) + pidx_g[g], clamped
  // to the row's last page; the page's byte offset is a 32 x 32-bit product.
  const int pidx_sh = log2P <= 6 ? 6 - log2P : 0;
  const int last_pidx = last_key >> log2P;
  const uint32_t page_bytes32 = (uint32_t)page_bytes;
  int pidx_g[NPG];
#pragma unroll
  for (int g = 0; g < NPG; ++g) pidx_g[g] = SCALAR_PAGES ? (blk(g * PB) * ROWS_PER_KB) >> log2P : 0;
  // The load is inline assembly (a scalar load with a register byte offset):
  // it is issued whether or not a table is present, and its result is only
  // read after the tile-start wait, which covers it.
  auto page_id_pfx = [&](int tile, int g, int& raw, int& alt) {
    const int pidx = min((tile << pidx_sh) + pidx_g[g], last_pidx);
    const uint32_t off = (uint32_t)(pidx & bt_any) << 2;
    asm volatile("s_load_dword %0, %1, %2" : "=s"(raw) : "s"(bt_row), "s"(off));
    alt = bt_base + pidx;
  };
  auto page_off_pfx = [&](int pg) -> int64_t {
    return (int64_t)((uint64_t)((uint32_t)pg < (uint32_t)num_pages ? (uint32_t)pg : 0u) * page_bytes32);
  };
  auto page_off = [&](int tile, int g, int pg) -> int64_t {
    const int t = block_key(tile, g);
    pg = (uint32_t)pg < (uint32_t)num_pages ? pg : 0;
    return (int64_t)(uint32_t)pg * page_bytes + (int64_t)((t & Pmask & ~(KT - 1)) * kv_stride);
  };
  auto page_of = [&](int tile, int g) -> int64_t { return page_off(tile, g, page_id(tile, g)); };
  auto lds_addr = [](const char* p) -> uint32_t {
    return (uint32_t)(size_t)((const __attribute__((address_space(3))) char*)p);
  };
  // The DMA of lookup group g of a K or V tile into `dst`.  A tile wholly
  // inside the prefix or wholly inside the chunk takes a scalar base plus the
  // lanes' constant 32-bit offsets; a tile straddling L or ending the key
  // range selects per lane.
  auto issue_group = [&](int tile, int g, int64_t pgoff, char* dst, const char* pool_base, const char* new_base,
                         auto pfx) {
    const int t0 = tile * KT;
    if constexpr (SCALAR_PAGES) {
      const uint32_t m0 = lds_addr(dst) + blk(g * PB) * 1024;
      if constexpr (decltype(pfx)::value) {  // caller guarantees a wholly cached tile
        dma_sbase<PB, NT_KV>(pool_base + pgoff, m0, &pool_v[g * PB]);
        return;
      }
      if (t0 + KT - 1 < u.L) {
        dma_sbase<PB, NT_KV>(pool_base + pgoff, m0, &pool_v[g * PB]);
        return;
      }
      if (t0 >= u.L && t0 + KT - 1 <= last_key) {
        dma_sbase<PB, NT_KV>(new_base + (int64_t)(u.cuq + t0 - u.L) * kv_stride, m0, &new_v[g * PB]);
        return;
      }
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        const int j = g * PB + i;
        const int t = min(t0 + drow[j], last_key);
        const char* src = t < u.L ? pool_base + pgoff + pool_off[j]
                                  : new_base + (int64_t)(u.cuq + t - u.L) * kv_stride + dchunk[j];
        dma_vaddr<NT_KV>(src, m0 + 1024u * i);
      }
    } else {
      const int t = min(t0 + drow[g], last_key);
      const char* src = t < u.L ? pool_base + pgoff + pool_off[g]
                                : new_base + (int64_t)(u.cuq + t - u.L) * kv_stride + dchunk[g];
      dma_vaddr<NT_KV>(src, lds_addr(dst) + blk(g) * 1024);
    }
  };
  auto issue = [&](int tile, const int64_t* pg, char* dst, const char* pool_base, const char* new_base) {
    if (!dma_wave) return;
#pragma unroll
    for (int g = 0; g < NPG; ++g) issue_group(tile, g, pg[g], dst, pool_base, new_base, std::false_type{});
  };
  // K ring first: its stage and block offsets then fit the 16-bit DS offset
  // field; the V ring's base is folded into the per-lane V read addresses.
  char* const kring = lds;
  char* const vring = lds + ST * TILEB;
  const uint32_t vring_addr = (uint32_t)(size_t)((__attribute__((address_space(3))) char*)vring);

  // Per-lane LDS read offsets (stage and 32-key block offsets are added as immediates).
  // QK8: koff[2i + j] = 16-byte chunk 4i + 2h + j of the key row (d = 64i + 32h + 16j ..).
  int koff[QK8 ? 4 : DS];
  if constexpr (QK8) {
#pragma unroll
    for (int x = 0; x < 4; ++x) koff[x] = l32 * ROWB + (slot<NCH, true>(l32, 4 * (x >> 1) + 2 * h + (x & 1)) << 4);
  } else {
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      koff[ds] = KV8 ? l32 * ROWB + (slot<NCH, true>(l32, ds) << 4) + 8 * h  // 8 codes: d = 16 ds + 8h ..
                     : l32 * ROWB + (slot<NCH>(l32, ds * 2 + h) << 4);
  }
  const int grp = lane >> 4, rr = (lane & 15) >> 2, qq = lane & 3, hh = grp >> 1;
  int voff_a[DB], voff_b[DB];
  {
    const int ra = 4 * hh + rr, rb = ra + 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int dcol = db * 32 + 16 * (grp & 1) + 4 * qq;
      const int chunk = dcol >> 3, within = (dcol & 7) * 2;
      voff_a[db] = ra * ROWB + (slot<NCH>(ra, chunk) << 4) + within;
      voff_b[db] = rb * ROWB + (slot<NCH>(rb, chunk) << 4) + within;
    }
  }

  // fp8 V: one transposing byte read per (16-key half, 32-wide d block).  In a
  // 16-lane group g, output lane i receives byte i % 8 of the reads of lanes
  // 2k + i / 8 (k = 0 .. 7), so lane 2k + p points at key 8(k/4) + 4(g/2) + k%4
  // (the probabilities' key order) and d column 16(g%2) + 8p of the block.
  int voff8[DB];
  if constexpr (KV8) {
    const int g = lane >> 4, kk = (lane & 15) >> 1, p8 = lane & 1;
    const int row = 8 * (kk >> 2) + 4 * (g >> 1) + (kk & 3);
#pragma unroll
    for (int db = 0; db < DB; ++db) voff8[db] = row * ROWB + (slot<NCH, true>(row, 2 * db + (g & 1)) << 4) + 8 * p8;
  }

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};
  float mref = -INFINITY, lrow = 0.f;
  // -mref (0 while no key has been seen), and the per-lane score above which
  // the reference must move: (mref + THRESH) / c.
  float neg_m = 0.f, thr = -INFINITY;

  // Scores of 32-key block kb of a K tile: S^T[key][row] (contraction steps [d0, d1)).
  // K fragments of k-steps [d0, d0 + DS/2) of block kb, and the score MFMAs over them.
  // QK8: one fp8 product over d = 64i .. 64i + 63 from the two key chunks k0, k1.
  auto mfma8 = [&](const u32x4& k0, const u32x4& k1, int i, f32x16& s) {
    if constexpr (QK8) {
      const i32x8 kv = {(int)k0[0], (int)k0[1], (int)k0[2], (int)k0[3],
                        (int)k1[0], (int)k1[1], (int)k1[2], (int)k1[3]};
      const u32x4 q0 = qf[2 * i], q1 = qf[2 * i + 1];
      const i32x8 qv = {(int)q0[0], (int)q0[1], (int)q0[2], (int)q0[3],
                        (int)q1[0], (int)q1[1], (int)q1[2], (int)q1[3]};
      // operand formats 0, 0: e4m3 x e4m3; no block scales
      s = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kv, qv, s, 0, 0, 0, 0, 0, 0);
    }
  };
  // K fragments of k-steps [d0, d0 + DS/2) of block kb (QK8: the two chunks of
  // product d0 == 0 ? 0 : 1), and the score MFMAs over them.
  auto load_k = [&](const char* kl, int kb, int d0, KF* kf) {
    if constexpr (QK8) {
      const int i = d0 ? 1 : 0;
      kf[0] = *reinterpret_cast<const KF*>(kl + kb * 32 * ROWB + koff[2 * i]);
      kf[1] = *reinterpret_cast<const KF*>(kl + kb * 32 * ROWB + koff[2 * i + 1]);
    } else {
#pragma unroll
      for (int i = 0; i < DS / 2; ++i) kf[i] = *reinterpret_cast<const KF*>(kl + kb * 32 * ROWB + koff[d0 + i]);
    }
  };
  auto mfma_k = [&](const KF* kf, int d0, f32x16& s) {
    if constexpr (QK8) {
      mfma8(kf[0], kf[1], d0 ? 1 : 0, s);
    } else {
#pragma unroll
      for (int i = 0; i < DS / 2; ++i)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kfrag(kf[i])),
                                                    __builtin_bit_cast(bf16x8, qf[d0 + i]), s, 0, 0, 0);
    }
  };
  auto qk = [&](const char* kl, int kb, f32x16& s) {
    s = f32x16{};
    if constexpr (QK8) {
      KF kf[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) kf[x] = *reinterpret_cast<const KF*>(kl + kb * 32 * ROWB + koff[x]);
      mfma8(kf[0], kf[1], 0, s);
      mfma8(kf[2], kf[3], 1, s);
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const KF kf = *reinterpret_cast<const KF*>(kl + kb * 32 * ROWB + koff[ds]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kfrag(kf)),
                                                    __builtin_bit_cast(bf16x8, qf[ds]), s, 0, 0, 0);
      }
    }
  };
  // O^T += V^T P^T for 32-key block kb.  Contraction slot 8h+s of half hf is
  // key kb*32 + 16*hf + 8*(s/4) + 4h + s%4, matching the probabilities' order.
  auto pv = [&](const char* vl, int kb, const u32x4* pf) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const char* vb = vl + (kb * 32 + 16 * hf) * ROWB;
      if constexpr (KV8) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const u32x2 w = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(vb + voff8[db])));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, e4m3x8_to_bf16(w)),
                                                          __builtin_bit_cast(bf16x8, pf[hf]), o[db], 0, 0, 0);
        }
        continue;
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const u32x2 wa = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb + voff_a[db])));
        const u32x2 wb = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb + voff_b[db])));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u32x4{wa[0], wa[1], wb[0], wb[1]}),
                                                        __builtin_bit_cast(bf16x8, pf[hf]), o[db], 0, 0, 0);
      }
    }
  };
  // Same product with the transposing reads issued as inline assembly and a
  // single explicit LDS wait.  The compiler cannot tell these reads from the
  // in-flight global->LDS DMA of later tiles and would otherwise wait for all
  // of that DMA (vmcnt(0)) before each read; the ring protocol already
  // guarantees the stage was filled (vmcnt + barrier at the tile start).
  // VOFF is the compile-time LDS byte offset of the 32-key block.
  auto pv_asm = [&](auto voff_c, const u32x4* pf) {
    constexpr int VOFF = decltype(voff_c)::value;
    static_assert(VOFF + 16 * ROWB < 65536, "DS immediate offset range");
    if constexpr (KV8) {
      static_assert(DB == 4, "fp8 V path is laid out for d = 128");
      u32x2 w8[2][DB];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int db = 0; db < DB; ++db)
          asm volatile("ds_read_b64_tr_b8 %0, %1 offset:%2" : "=v"(w8[hf][db]) : "v"(vring_addr + voff8[db]), "i"(VOFF + hf * 16 * ROWB));
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(w8[0][0]), "+v"(w8[0][1]), "+v"(w8[0][2]), "+v"(w8[0][3]), "+v"(w8[1][0]), "+v"(w8[1][1]),
                     "+v"(w8[1][2]), "+v"(w8[1][3]));
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int db = 0; db < DB; ++db)
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, e4m3x8_to_bf16(w8[hf][db])),
                                                          __builtin_bit_cast(bf16x8, pf[hf]), o[db], 0, 0, 0);
      return;
    }
    u32x2 w[2][DB][2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(w[hf][db][0]) : "v"(vring_addr + voff_a[db]), "i"(VOFF + hf * 16 * ROWB));
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(w[hf][db][1]) : "v"(vring_addr + voff_b[db]), "i"(VOFF + hf * 16 * ROWB));
      }
    if constexpr (DB == 4) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(w[0][0][0]), "+v"(w[0][0][1]), "+v"(w[0][1][0]), "+v"(w[0][1][1]), "+v"(w[0][2][0]),
                     "+v"(w[0][2][1]), "+v"(w[0][3][0]), "+v"(w[0][3][1]), "+v"(w[1][0][0]), "+v"(w[1][0][1]),
                     "+v"(w[1][1][0]), "+v"(w[1][1][1]), "+v"(w[1][2][0]), "+v"(w[1][2][1]), "+v"(w[1][3][0]),
                     "+v"(w[1][3][1]));
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(w[0][0][0]), "+v"(w[0][0][1]), "+v"(w[0][1][0]), "+v"(w[0][1][1]), "+v"(w[1][0][0]),
                     "+v"(w[1][0][1]), "+v"(w[1][1][0]), "+v"(w[1][1][1]));
    }
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, u32x4{w[hf][db][0][0], w[hf][db][0][1], w[hf][db][1][0], w[hf][db][1][1]}),
            __builtin_bit_cast(bf16x8, pf[hf]), o[db], 0, 0, 0);
  };
  // exp2(s*c - m) packed to bf16 for contraction half hf (8 keys), and their
  // sum (a tree: no dependent chain through all eight).
  auto exp_half = [&](const f32x16& s, int hf, float& bs) -> u32x4 {
    float p[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) p[e] = fast_exp2(__builtin_fmaf(s[8 * hf + e], c, neg_m));
    bs = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
    return u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
  };
  auto softmax_exp = [&](const f32x16& s, u32x4* pf) {
    float b0, b1;
    pf[0] = exp_half(s, 0, b0);
    pf[1] = exp_half(s, 1, b1);
    lrow += b0 + b1;
  };
  // Pins a value at this point of the program: IR-level sinking would
  // otherwise move the exponentials past the DMA branches to their use by the
  // PV products, leaving them no score MFMAs to overlap with.
  auto pin = [](u32x4& x) { asm volatile("" : "+v"(x)); };
  // Maximum of the lane's 16 raw scores (half of its row's 32 keys).
  auto row_max = [&](const f32x16& s) -> float {
    auto mx3 = [](float a, float b, float c) {
      return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
    };
    const float u0 = mx3(mx3(s[0], s[1], s[2]), mx3(s[3], s[4], s[5]), mx3(s[6], s[7], s[8]));
    const float u1 = mx3(mx3(s[9], s[10], s[11]), mx3(s[12], s[13], s[14]), s[15]);
    return __builtin_elementwise_maximum(u0, u1);
  };
  // Move the reference max if any lane's scores grew past the threshold; only
  // then is the exact row max (both half-rows) formed.
  auto update_ref = [&](float mx) {
    if (__any(mx > thr)) {
      const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      const float mxs = __builtin_elementwise_maximum(__uint_as_float(pr[0]), __uint_as_float(pr[1])) * c;
      const float mnew = fmaxf(mref, mxs);
      // With no reference yet (mref = -inf) nothing has been accumulated: the
      // factor is 0, not exp2(-mnew), which overflows for very low scores.
      const float alpha = mref == -INFINITY ? 0.f : fast_exp2(mref - mnew);
      lrow *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
      mref = mnew;
      neg_m = mnew == -INFINITY ? 0.f : -mnew;
      thr = (mnew + THRESH) / c;
    }
  };
  // Main-loop check of a block's probabilities instead of its row max: if in
  // either lane of a row the 16 of them (formed against the current
  // reference) sum past 2^16, or to NaN, form the block's exact row max, move
  // the reference, rescale the row sum and recompute the probabilities;
  // alpha then rescales O.
  // Every probability used stays below 2^16, and as with the lazily moved
  // maximum the final normalisation is exact whatever reference was used.
  auto reexp = [&](const f32x16& s, u32x4* pf, float& bsum, float& alpha) {
    const float mx = row_max(s);
    const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    const float mxs = __builtin_elementwise_maximum(__uint_as_float(pr[0]), __uint_as_float(pr[1])) * c;
    const float mnew = fmaxf(mref, mxs);
    alpha = mref == -INFINITY ? 0.f : fast_exp2(mref - mnew);
    lrow *= alpha;
    mref = mnew;
    neg_m = mnew == -INFINITY ? 0.f : -mnew;
    thr = (mnew + THRESH) / c;
    float b0, b1;
    pf[0] = exp_half(s, 0, b0);
    pf[1] = exp_half(s, 1, b1);
    bsum = b0 + b1;
  };
  // One pipelined block step: the probabilities of s_cur (block kb of V tile
  // vl) are formed while the MFMA pipe works on the scores of the next block
  // (block kb_next of K tile kl_next); then the block's check, the next K
  // fragments' reads and P V.  dma_a / dma_b issue this wave's DMA runs of
  // the step (one tensor per step) and, after the second step's, the page
  // ids of the tile after next.  The compiler schedules the step freely; the
  // empty asm markers (pin) keep each half's probabilities next to the score
  // products they overlap.  K fragments of the first half of the next step's
  // score block are read one group of products ahead, so that their LDS
  // latency hides behind MFMAs.
  KF kpre[DS / 2];
  auto step = [&](f32x16& s_cur, f32x16& s_next, auto voff_c, const char* kl_next, int kb_next,
                  const char* kl_after, int kb_after, auto dma_a, auto dma_b) {
    u32x4 pf[2];
    KF kh1[DS / 2];
    float b0, b1;
    s_next = f32x16{};
    load_k(kl_next, kb_next, DS / 2, kh1);
    pf[0] = exp_half(s_cur, 0, b0);
    mfma_k(kpre, 0, s_next);
    pin(pf[0]);
    dma_a();
    pf[1] = exp_half(s_cur, 1, b1);
    mfma_k(kh1, DS / 2, s_next);
    pin(pf[1]);
    float bsum = b0 + b1;
    {
      // Per row (lanes l and l^32 hold its two halves), as a divergent
      // branch: the rare path then writes the fast path's registers under
      // the exec mask instead of leaving copies on the fast path.
      const uint32_t ov = !(bsum <= 65536.f) ? 1u : 0u;
      const auto pr = __builtin_amdgcn_permlane32_swap(ov, ov, false, false);
      if ((pr[0] | pr[1]) != 0u) {
        float alpha;
        reexp(s_cur, pf, bsum, alpha);
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;
      }
    }
    lrow += bsum;
    dma_b();
    load_k(kl_after, kb_after, 0, kpre);
    pv_asm(voff_c, pf);
    s_cur = s_next;
  };

  // ---- main loop: tiles [tb, main_end) are unmasked for every row of the workgroup
  const int wg_first_lim = u.L + u.m0 / G;
  const int main_end = max(u.tb, min(u.te, (wg_first_lim + 1) / KT));
  const int n_main = main_end - u.tb;
  if (n_main > 0) {
    // K(tb+k) and V(tb+k) live in stage k % 4.  Every tile issues exactly
    // 2*NDMA DMA instructions per wave (tiles past the end are clamped to the
    // last one and land in a stage nobody reads again), so "all but the
    // previous tile's loads" is the constant vmcnt(2*NDMA).
    auto clampt = [&](int t) { return min(t, main_end - 1); };
    int64_t pgn[NPG];  // page offsets of tile tb+k+3, issued at tile k
    int pgi[NPG];      // their page ids (raw table words), loaded half a tile earlier
    int pga[NPG];      // ... and the contiguous cache's ids (used when there is no table)
    {
      int64_t pg[NPG];
      if (dma_wave) {
#pragma unroll
        for (int i = 0; i < 3; ++i) {
#pragma unroll
          for (int g = 0; g < NPG; ++g) pg[g] = page_of(clampt(u.tb + i), g);
          issue(clampt(u.tb + i), pg, kring + i * TILEB, kpool, knew);
          issue(clampt(u.tb + i), pg, vring + i * TILEB, vpool, vnew);
        }
      }
#pragma unroll
      for (int g = 0; g < NPG; ++g) pgi[g] = pga[g] = dma_wave ? page_id(clampt(u.tb + 3), g) : 0;
    }
    // Only tile 0's K must have landed (the first scores below); the loop's
    // first tile waits for the rest.  Each DMA wave issued 6 * NDMA loads,
    // K(0) first, and loads complete in order.
    static_assert(5 * NDMA <= 63, "vmcnt field");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(5 * NDMA) : "memory");
    __builtin_amdgcn_s_barrier();
    f32x16 s_a, s_b;
    if (wave_active) {
      qk(kring, 0, s_a);
      update_ref(row_max(s_a));
      load_k(kring, 1, 0, kpre);
    }
    // Tile k with ring stage S = k % 4 known at compile time; ACT: the wave
    // holds rows (else it only issues its share of the DMA and joins the
    // barriers).  Active and row-less waves run separate copies of the loop, so
    // the compiler's wait counting in the active loop never merges with the
    // row-less path's scalar loads.
    // PFX: the tile whose DMA this tile issues (tb+k+3) lies wholly in the
    // cached prefix, so is the one whose page id it loads (tb+k+4) inside the
    // table row: neither needs a test.
    // CLS: 1 / 2 when the caller knows the wave is in the lower / upper half
    // (its issue-priority turns then need no branch), 0 otherwise.
    auto tile = [&](int k, auto stage, auto act, auto pfx, auto cls) {
      constexpr int S = decltype(stage)::value;
      constexpr bool ACT = decltype(act)::value;
      constexpr int CLS = decltype(cls)::value;
      auto prio = [&](bool first) {
        if constexpr (CLS == 1) {
          if (first) __builtin_amdgcn_s_setprio(1); else __builtin_amdgcn_s_setprio(0);
        } else if constexpr (CLS == 2) {
          if (first) __builtin_amdgcn_s_setprio(0); else __builtin_amdgcn_s_setprio(1);
        } else {
          if ((wave < NW / 2) == first) __builtin_amdgcn_s_setprio(1); else __builtin_amdgcn_s_setprio(0);
        }
      };
      // Tiles k and k+1 have landed in LDS (only the previous tile's DMA may
      // still be in flight) and this wave's LDS reads of tile k-1 are done.
      // A plain s_barrier: __syncthreads() would also fence, i.e. wait for the
      // DMA of later tiles too.
      if constexpr (SCALAR_PAGES) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(2 * NDMA) : "memory");
      else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      // The page ids loaded during the previous tile have arrived (the wait
      // above); passing them through an empty asm tells the compiler so, which
      // keeps it from waiting for them, and with them for every LDS read
      // issued meanwhile, at their first use.
#pragma unroll
      for (int g = 0; g < NPG; ++g) {
        if constexpr (SCALAR_PAGES) asm volatile("" : "+s"(pgi[g]));
        else asm volatile("" : "+v"(pgi[g]));
      }
      // K/V(tb+k+3) replace K/V(tb+k-1), last read during tile k-1; their
      // DMA blocks are spread over the tile's two steps.
      const int nt = clampt(u.tb + k + 3);
      if (dma_wave) {
#pragma unroll
        for (int g = 0; g < NPG; ++g) {
          if constexpr (SCALAR_PAGES && decltype(pfx)::value) pgn[g] = page_off_pfx(page_pick(pgi[g], pga[g]));
          else pgn[g] = page_off(nt, g, page_pick(pgi[g], pga[g]));
        }
      }
      char* kdst = kring + ((S + 3) % ST) * TILEB;
      char* vdst = vring + ((S + 3) % ST) * TILEB;
      const char* kl = kring + S * TILEB;
      auto kd0 = [&] {
        if (!dma_wave) return;
#pragma unroll
        for (int g = 0; g < NG0; ++g) issue_group(nt, g, pgn[g], kdst, kpool, knew, pfx);
      };
      auto kd1 = [&] {
        if (!dma_wave) return;
#pragma unroll
        for (int g = NG0; g < NPG; ++g) issue_group(nt, g, pgn[g], kdst, kpool, knew, pfx);
      };
      auto vd0 = [&] {
        if (!dma_wave) return;
#pragma unroll
        for (int g = 0; g < NG0; ++g) issue_group(nt, g, pgn[g], vdst, vpool, vnew, pfx);
      };
      auto vd1 = [&] {
        if (!dma_wave) return;
#pragma unroll
        for (int g = NG0; g < NPG; ++g) issue_group(nt, g, pgn[g], vdst, vpool, vnew, pfx);
#pragma unroll
        for (int g = 0; g < NPG; ++g) {
          if constexpr (SCALAR_PAGES && decltype(pfx)::value) page_id_pfx(u.tb + k + 4, g, pgi[g], pga[g]);
          else pgi[g] = pga[g] = page_id(clampt(u.tb + k + 4), g);
        }
      };
      // The two waves of a SIMD take turns at the higher issue priority, one
      // step each, so that neither lags the other into the tile barrier.
      prio(true);
      // block 0 || scores of block 1, then block 1 || scores of the next tile's block 0
      if constexpr (!ACT) {
        kd0(); kd1(); vd0(); vd1();
        return;
      }
      step(s_a, s_b, std::integral_constant<int, S * TILEB>{}, kl, 1, kring + ((S + 1) % ST) * TILEB, 0, kd0, kd1);
      prio(false);
      step(s_a, s_b, std::integral_constant<int, S * TILEB + 32 * ROWB>{}, kring + ((S + 1) % ST) * TILEB, 0,
           kring + ((S + 1) % ST) * TILEB, 1, vd0, vd1);
    };
    // Iterations whose DMA target tile (tb+k+3, clamped) lies wholly in the
    // cached prefix run first, in whole rounds of the ring, without the
    // per-tile classification; the rest take the general path.
    const int pfx_tiles = u.L / KT;  // tiles [0, pfx_tiles) are wholly cached
    const int k_pfx = log2P > 6 ? 0 : main_end - 1 < pfx_tiles ? n_main : max(0, min(n_main, pfx_tiles - u.tb - 3));
    auto prefix_tiles = [&](int& k, auto act, auto cls) {
      for (; k + 4 <= k_pfx; k += 4) {
        tile(k, std::integral_constant<int, 0>{}, act, std::true_type{}, cls);
        tile(k + 1, std::integral_constant<int, 1>{}, act, std::true_type{}, cls);
        tile(k + 2, std::integral_constant<int, 2>{}, act, std::true_type{}, cls);
        tile(k + 3, std::integral_constant<int, 3>{}, act, std::true_type{}, cls);
      }
    };
    auto tiles = [&](auto act) {
      int k = 0;
      if constexpr (SCALAR_PAGES) {
        // computing waves: one copy of the loop per half, for branch-free priority turns
        if constexpr (decltype(act)::value) {
          if (wave < NW / 2) prefix_tiles(k, act, std::integral_constant<int, 1>{});
          else prefix_tiles(k, act, std::integral_constant<int, 2>{});
        } else {
          prefix_tiles(k, act, std::integral_constant<int, 0>{});
        }
      }
      for (; k < n_main; k += 4) {
        tile(k, std::integral_constant<int, 0>{}, act, std::false_type{}, std::integral_constant<int, 0>{});
        if (k + 1 >= n_main) break;
        tile(k + 1, std::integral_constant<int, 1>{}, act, std::false_type{}, std::integral_constant<int, 0>{});
        if (k + 2 >= n_main) break;
        tile(k + 2, std::integral_constant<int, 2>{}, act, std::false_type{}, std::integral_constant<int, 0>{});
        if (k + 3 >= n_main) break;
        tile(k + 3, std::integral_constant<int, 3>{}, act, std::false_type{}, std::integral_constant<int, 0>{});
      }
    };
    if (wave_active) tiles(std::true_type{});
    else tiles(std::false_type{});
    __builtin_amdgcn_s_setprio(0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();  // every wave is done with the rings before the tail reuses them
  }

  // ---- tail: tiles [main_end, te) with the causal mask, one tile at a time
  for (int it = max(main_end, u.tb); it < u.te; ++it) {
    int64_t pg[NPG];
#pragma unroll
    for (int g = 0; g < NPG; ++g) pg[g] = dma_wave ? page_of(it, g) : 0;
    issue(it, pg, kring, kpool, knew);
    issue(it, pg, vring, vpool, vnew);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const int t0 = it * KT;
#pragma unroll
    for (int kb = 0; kb < 2 && wave_active; ++kb) {
      f32x16 s;
      qk(kring, kb, s);
      if (t0 + kb * 32 + 31 > lim) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (t0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3) > lim) s[v] = -INFINITY;
      }
      update_ref(row_max(s));
      u32x4 pf[2];
      softmax_exp(s, pf);
      pv(vring, kb, pf);
    }
    __syncthreads();
  }

  // Profiling hook: end of this workgroup's key tiles on the 100 MHz
  // constant clock, the tiles, and its unit and XCD.
  if (a.wg_clock && threadIdx.x == 0 && (int)blockIdx.x < a.wg_clock_cap) {
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    uint64_t* w = a.wg_clock + 4 * (size_t)blockIdx.x;
    w[1] = __builtin_amdgcn_s_memrealtime();
    w[2] = ((uint64_t)(uint32_t)u.tb << 32) | (uint32_t)u.te;
    w[3] = ((uint64_t)(uint32_t)u.b << 32) | ((uint64_t)(u.s & 0xffff) << 16) | ((uint64_t)(u.g & 0xff) << 8) |
           (xcc & 0xffu);
  }
  // Epilogue: combine the two half-rows' sums, normalise, write o and lse (or split partials).
  const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(lrow), __float_as_uint(lrow), false, false);
  const float lsum = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
  if (!valid) return;
  const int64_t qrow = (int64_t)(u.cuq + tok) * a.Hq + u.g * G + (m_row - tok * G);
  // (an fp8 cache stores V / v_scale: the scale comes back here)
  const float inv = (lsum > 0.f ? 1.f / lsum : 0.f) * a.v_scale;
  const float lse = lsum > 0.f ? (mref + __log2f(lsum)) * LN2 : -INFINITY;
  if (a.nsplit == 1) {
    char* orow = static_cast<char*>(a.out) + qrow * D * 2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int vg = 0; vg < 4; ++vg) {
        const int d0 = db * 32 + 8 * vg + 4 * h;
        const u32x2 w = {pack_bf16x2(o[db][4 * vg + 0] * inv, o[db][4 * vg + 1] * inv),
                         pack_bf16x2(o[db][4 * vg + 2] * inv, o[db][4 * vg + 3] * inv)};
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
        const f32x4 w = {o[db][4 * vg + 0] * inv, o[db][4 * vg + 1] * inv, o[db][4 * vg + 2] * inv,
                         o[db][4 * vg + 3] * inv};
        *reinterpret_cast<f32x4*>(orow + d0) = w;
      }
    if (h == 0) a.part_lse[prow] = lse;
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

constexpr int BF16_BM = 256;  // 8 waves x 32 packed rows

}  // namespace

int attn_block_m(int dtype_bf16, int d, int four_waves) {
  (void)d;
  if (four_waves) return 128;
  return dtype_bf16 ? BF16_BM : NWAVES * 32;
}

namespace {

// One bf16-Q kernel variant: the DMA issued by every wave or by the upper half
// only, and the scalar page path when every page lookup run fits in a page.
template <int D, bool KV8, int NW, bool QK8 = false>
void launch_bf16(const AttnArgs& a, unsigned grid, hipStream_t stream) {
  const bool up = a.dma_upper != 0;
  const bool sp = a.P >= dma_rows_per_lookup(D, KV8, NW, up);
  const dim3 g(grid), b(NW * 64);
  if (up) {
    if (sp) hipLaunchKernelGGL((attn_bf16_kernel<D, true, KV8, NW, true, QK8>), g, b, 0, stream, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<D, false, KV8, NW, true, QK8>), g, b, 0, stream, a);
  } else {
    if (sp) hipLaunchKernelGGL((attn_bf16_kernel<D, true, KV8, NW, false, QK8>), g, b, 0, stream, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<D, false, KV8, NW, false, QK8>), g, b, 0, stream, a);
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, hipStream_t stream) {
  if (a.n_units == 0) return hipSuccess;
  unsigned grid = (unsigned)a.n_units;
  if (a.order) grid = 8u * (unsigned)a.order_slots;
  else if (a.xcd_remap) grid = (grid + 7u) & ~7u;
  if (dtype_bf16 && a.kv_fp8) {
    // fp8 rows (d = 128); 4-wave workgroups of 128 rows for short chunks
    if (a.four_waves) {
      if (a.qk8) launch_bf16<128, true, 4, true>(a, grid, stream);
      else launch_bf16<128, true, 4>(a, grid, stream);
    } else {
      if (a.qk8) launch_bf16<128, true, 8, true>(a, grid, stream);
      else launch_bf16<128, true, 8>(a, grid, stream);
    }
  } else if (dtype_bf16) {
    if (a.d == 128) launch_bf16<128, false, 8>(a, grid, stream);
    else launch_bf16<64, false, 8>(a, grid, stream);
  } else {
    if (a.d == 128) hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(grid), dim3(NTHREADS), 0, stream, a);
    else hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(grid), dim3(NTHREADS), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace csr
