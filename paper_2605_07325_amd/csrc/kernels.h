// Internal launch interface between the C ABI (csr_api.cpp) and the HIP
// kernels.  Not installed; the public interface is include/csr.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace csr {

// Everything one attention launch needs.  Sizes are validated by the caller.
struct AttnArgs {
  const void* q;
  const void* k_new;
  const void* v_new;
  const void* k_pool;
  const void* v_pool;
  const int32_t* block_table;
  const int32_t* cu_q;
  const int32_t* cache_len;  // nullptr: every L_b = 0
  void* out;                 // final output (nsplit == 1)
  float* lse;                // final lse or nullptr (nsplit == 1)
  float* part_o;             // [nsplit][T_q][Hq][d] partial outputs (nsplit > 1)
  float* part_lse;           // [nsplit][T_q][Hq]
  int32_t num_pages;
  int32_t bt_stride;
  int32_t Hq, Hkv, G, d, P, log2P;
  float scale_log2;          // softmax scale * log2(e) (times k_scale for an fp8 cache)
  float v_scale;             // output multiplier: 1, or v_scale for an fp8 cache
  int32_t kv_fp8;            // K/V (pool and chunk) are OCP e4m3 codes (bf16 q, d = 128)
  int32_t four_waves;        // fp8 only: 4-wave workgroups of 128 rows, two per CU
  int32_t qk8;               // fp8 only: q holds e4m3 codes, Q K^T on the fp8 MFMA
  int32_t dma_upper;         // bf16 Q: all rows in the lower half of the waves; the upper half loads K/V
  int32_t batch, total_q;
  int32_t mtiles;            // packed-row tiles per (sequence, kv head)
  int32_t nsplit;            // key-range splits per tile
  int32_t n_units;           // batch * Hkv * nsplit * mtiles
  int32_t xcd_remap;         // 1: keep units that share K/V on one XCD
  const int32_t* order;      // unit of each workgroup (-1: none), or nullptr for the fixed order
  int32_t order_slots;       // with `order`: the grid is 8 * order_slots workgroups
  uint64_t* wg_clock;        // profiling: 4 words per workgroup (start, end, key tiles, unit and XCD), or nullptr
  int32_t wg_clock_cap;      // workgroups that record (workgroup id < cap)
};

// Packed rows (query token x head-in-group) per workgroup for each kernel.
int attn_block_m(int dtype_bf16, int d, int four_waves);
hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, hipStream_t stream);

// Longest-first work order for ragged batches (see plan.hip).
struct PlanArgs {
  const int32_t* cu_q;
  const int32_t* cache_len;  // nullptr: every L_b = 0
  int32_t* order;            // [8 * slots]
  int32_t batch, Hkv, G, bm, mtiles, nsplit, slots;
  int32_t rt_per_sub;        // row tiles per subgroup (the XCD-assignment granule)
};
int plan_subgroup_rows(int batch, int Hkv, int mtiles);
int plan_smem_bytes(int batch, int Hkv, int mtiles, int rt_per_sub);
hipError_t launch_plan(const PlanArgs& p, hipStream_t stream);

struct AppendArgs {
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* block_table;
  const int32_t* cu_q;
  const int32_t* cache_len;  // nullptr: every L_b = 0
  int32_t num_pages, bt_stride, batch, total_q, Hkv, P, log2P;
  int32_t row_chunks;        // 16-byte chunks per (token, kv head) row = d * elem / 16
};
hipError_t launch_append(const AppendArgs& a, hipStream_t stream);

struct MergeArgs {
  const float* part_o;
  const float* part_lse;
  void* out;
  float* lse;
  int32_t nsplit, total_q, Hq, d;
  // An append carried by the same launch (extra workgroups after the merge's;
  // append.total_q == 0: none).  It writes only cache slots [L_b, L_b + n_b),
  // which the attention of the same call never reads.
  AppendArgs append;
};
hipError_t launch_merge(const MergeArgs& a, int dtype_bf16, hipStream_t stream);

// Rotary embedding at absolute positions L_b + i and/or fp8 quantisation of
// K/V, fused with the append.
struct RopeArgs {
  const void* q;             // [T_q][Hq][d] or nullptr (keys only)
  const void* k;             // [T_q][Hkv][d]
  const void* v;             // [T_q][Hkv][d], read only when k_pool is set
  void* q_out;               // rotated q, or nullptr
  void* k_out;               // rotated (and, kv8, quantised) k, or nullptr
  void* v_out;               // kv8: quantised v, or nullptr
  void* k_pool;              // nullptr: no cache write
  void* v_pool;
  const int32_t* block_table;
  const int32_t* cu_q;
  const int32_t* cache_len;  // nullptr: every L_b = 0
  int32_t num_pages, bt_stride, batch, total_q, Hq, Hkv, d, log2P;
  int32_t rdim;              // rotated dims, multiple of 16, <= d (0: no rotation)
  int32_t style;             // 0 none, 1 neox (i, i + r/2), 2 interleaved (2i, 2i + 1)
  int32_t kv8;               // keys/values (outputs and cache) are e4m3 codes; bf16 inputs
  int32_t q8;                // kv8 only: q rows are quantised too (q_out holds e4m3 codes)
  float inv_k, inv_v, inv_q;  // fp32(1 / k_scale), fp32(1 / v_scale), fp32(1 / q_scale)
  double inv_freq[64];       // theta_i = pow(theta, -2i / rdim) in fp64, i < rdim / 2 (pair i turns by pos * theta_i)
};
hipError_t launch_rope_append(const RopeArgs& a, int dtype_bf16, hipStream_t stream);

}  // namespace csr
