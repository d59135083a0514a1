// C ABI of libcsr (declared in include/csr.h): host-side validation, launch
// planning and kernel launches on the caller's stream.
//
// Argument validation runs entirely on the host before any work is enqueued:
// the only runtime queries before the last check (the workspace size, which
// depends on the plan) are hipGetDevice and, once per device, its CU count.
#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <atomic>
#include <mutex>
#include <string>

#include "../../include/csr.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_ev_begin = nullptr, g_ev_end = nullptr;  // csr_set_attention_events
thread_local uint64_t* g_wg_clock = nullptr;                         // csr_set_workgroup_clock
thread_local int32_t g_wg_clock_cap = 0;
// csr_set_plan_overrides (testing and A/B measurement): 0 = the planner's choice.
struct PlanOverrides {
  int nsplit = 0;         // > 0: key-range splits per unit
  int fixed_order = 0;    // 1: ragged batches keep the index order of their units
  int dma_all_waves = 0;  // 1: short chunks load K/V from every wave
};
thread_local PlanOverrides g_ovr;

csr_status fail(csr_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
csr_status fail(csr_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int ilog2(int x) {
  int r = 0;
  while ((1 << r) < x) ++r;
  return r;
}

csr_status check_desc(const csr_attn_desc* d) {
  if (!d) return fail(CSR_E_INVAL, "desc is NULL");
  if (d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(CSR_E_INVAL, "head counts must be >= 1 (Hq=%d, Hkv=%d)", d->num_q_heads, d->num_kv_heads);
  if (d->num_q_heads % d->num_kv_heads)
    return fail(CSR_E_INVAL, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)", d->num_q_heads,
                d->num_kv_heads);
  if (d->dtype != CSR_BF16 && d->dtype != CSR_F32) return fail(CSR_E_UNSUPPORTED, "unsupported dtype %d", d->dtype);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(CSR_E_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", d->head_dim);
  if (d->page_size < 1 || d->page_size > 1024 || (d->page_size & (d->page_size - 1)))
    return fail(CSR_E_INVAL, "page_size %d must be a power of two in [1, 1024]", d->page_size);
  if (!(d->softmax_scale >= 0.f) || isinf(d->softmax_scale))
    return fail(CSR_E_INVAL, "softmax_scale must be finite and >= 0 (0 = 1/sqrt(d))");
  if (d->rope_style != CSR_ROPE_NONE) {
    if (d->rope_style != CSR_ROPE_NEOX && d->rope_style != CSR_ROPE_INTERLEAVED)
      return fail(CSR_E_INVAL, "unknown rope_style %d", d->rope_style);
    const int r = d->rope_dim ? d->rope_dim : d->head_dim;
    if (r < 16 || r > d->head_dim || r % 16)
      return fail(CSR_E_UNSUPPORTED, "rope_dim %d must be a multiple of 16 in [16, head_dim=%d]", d->rope_dim,
                  d->head_dim);
    if (!(d->rope_theta > 0.f) || isinf(d->rope_theta))
      return fail(CSR_E_INVAL, "rope_theta must be finite and > 0");
  }
  if (d->kv_dtype != CSR_KV_SAME) {
    if (d->kv_dtype != CSR_KV_FP8_E4M3) return fail(CSR_E_INVAL, "unknown kv_dtype %d", d->kv_dtype);
    if (d->dtype != CSR_BF16 || d->head_dim != 128)
      return fail(CSR_E_UNSUPPORTED, "an fp8 cache needs bf16 inputs and head_dim 128");
    if (!(d->k_scale > 0.f) || isinf(d->k_scale) || !(d->v_scale > 0.f) || isinf(d->v_scale))
      return fail(CSR_E_INVAL, "k_scale and v_scale must be finite and > 0");
  }
  if (d->q_scale != 0.f) {
    if (d->kv_dtype != CSR_KV_FP8_E4M3)
      return fail(CSR_E_UNSUPPORTED, "fp8 score products (q_scale) need an fp8 cache");
    if (!(d->q_scale > 0.f) || isinf(d->q_scale)) return fail(CSR_E_INVAL, "q_scale must be 0, or finite and > 0");
  }
  return CSR_OK;
}

bool has_rope(const csr_attn_desc* d) { return d->rope_style != CSR_ROPE_NONE; }
bool kv_fp8(const csr_attn_desc* d) { return d->kv_dtype == CSR_KV_FP8_E4M3; }
// fp8 score products: q quantised like the keys, Q K^T on the fp8 matrix cores.
bool qk_fp8(const csr_attn_desc* d) { return kv_fp8(d) && d->q_scale > 0.f; }
// The attention reads q from the workspace: rotated (RoPE) and/or quantised (fp8 products).
bool prep_q(const csr_attn_desc* d) { return has_rope(d) || qk_fp8(d); }
// RoPE or an fp8 cache: one launch prepares q/k/v (and appends) before the attention.
bool needs_prep(const csr_attn_desc* d) { return has_rope(d) || kv_fp8(d); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int elem_bytes(const csr_attn_desc* d) { return d->dtype == CSR_BF16 ? 2 : 4; }

// Workspace head written by the prep launch, each part 256-aligned: prepared q
// (rotated with RoPE, e4m3 codes with fp8 products), prepared k (rotated
// and/or quantised), quantised v (fp8 only).
struct PrepLayout {
  size_t q_off, k_off, v_off, bytes;
};
PrepLayout prep_layout(const csr_attn_desc* d, int total) {
  PrepLayout l{0, 0, 0, 0};
  if (!needs_prep(d)) return l;
  const size_t rows = (size_t)total * d->head_dim;
  const size_t qb = prep_q(d) ? align256(rows * d->num_q_heads * (qk_fp8(d) ? 1 : elem_bytes(d))) : 0;
  const size_t kb = align256(rows * d->num_kv_heads * (kv_fp8(d) ? 1 : elem_bytes(d)));
  const size_t vb = kv_fp8(d) ? align256(rows * d->num_kv_heads) : 0;
  l.q_off = 0;
  l.k_off = qb;
  l.v_off = qb + kb;
  l.bytes = qb + kb + vb;
  return l;
}

// q / q_out may be NULL (keys only), k_out / v_out NULL (no workspace copy),
// k_pool NULL (no cache write).
csr::RopeArgs rope_args(const csr_attn_desc* d, int batch, const void* q, const void* k, const void* v, void* q_out,
                        void* k_out, void* v_out, void* k_pool, void* v_pool, int num_pages, const int32_t* bt,
                        int bt_stride, const int32_t* cu, const int32_t* cache_len, int total) {
  csr::RopeArgs a;
  a.q = prep_q(d) ? q : nullptr;
  a.k = k;
  a.v = v;
  a.q_out = prep_q(d) ? q_out : nullptr;
  a.q8 = qk_fp8(d) ? 1 : 0;
  a.inv_q = qk_fp8(d) ? 1.f / d->q_scale : 1.f;
  a.k_out = k_out;
  a.v_out = kv_fp8(d) ? v_out : nullptr;
  a.kv8 = kv_fp8(d) ? 1 : 0;
  a.inv_k = kv_fp8(d) ? 1.f / d->k_scale : 1.f;
  a.inv_v = kv_fp8(d) ? 1.f / d->v_scale : 1.f;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.block_table = bt;
  a.cu_q = cu;
  a.cache_len = cache_len;
  a.num_pages = num_pages;
  a.bt_stride = bt_stride;
  a.batch = batch;
  a.total_q = total;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.d = d->head_dim;
  a.log2P = ilog2(d->page_size);
  a.rdim = has_rope(d) ? (d->rope_dim ? d->rope_dim : d->head_dim) : 0;
  a.style = d->rope_style;
  // Pair i turns by pos * theta^(-2i/r) radians (theta: the descriptor's float, widened).
  for (int i = 0; i < 64; ++i) a.inv_freq[i] = i < a.rdim / 2 ? pow((double)d->rope_theta, -2.0 * i / a.rdim) : 0.0;
  return a;
}

// Launch plan: row tiles, key splits, workspace.  Pure function of the host
// integers and the device's CU count, so the size query and the call agree.
struct Plan {
  int bm, mtiles, nsplit, n_units, xcd_remap;
  int four_waves;   // fp8 cache, at most 128 packed rows per sequence: 4-wave workgroups
  int dma_upper;    // bf16 Q, rows of every unit in the lower half of the waves: the upper half loads K/V
  int order_slots;  // > 0: a device-side longest-first order (ragged batches)
  size_t ws_o, ws_lse, ws_order_off, ws_bytes;
};

// CU count of the current device, queried once per device (256 on MI355X).
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];
int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return 256;
  }
  if (dev < kMaxDevices) {
    const int c = g_cus[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
    (void)hipGetLastError();
    cus = 256;
  }
  if (dev < kMaxDevices) g_cus[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

csr_status make_plan(const csr_attn_desc* d, int batch, int total_q, int max_q, int max_L, Plan& p) {
  const int G = d->num_q_heads / d->num_kv_heads;
  // Short chunks over an fp8 cache (decode): one 128-row tile holds every
  // row of a sequence, and 4-wave workgroups (64 KB of LDS) run two per CU.
  p.four_waves = kv_fp8(d) && (int64_t)max_q * G <= 128 ? 1 : 0;
  p.bm = csr::attn_block_m(d->dtype == CSR_BF16, d->head_dim, p.four_waves);
  const int64_t rows = (int64_t)max_q * G;
  if (rows >= (1ll << 30) || (int64_t)max_L + max_q >= (1ll << 30))
    return fail(CSR_E_UNSUPPORTED, "sequence too long (max_seqlen_q*G=%lld, max_cache_len+max_seqlen_q=%lld)",
                (long long)rows, (long long)max_L + max_q);
  p.mtiles = (int)((rows + p.bm - 1) / p.bm);
  // Short chunks leave the upper half of the waves without rows: they then
  // issue all of the K/V DMA, off the computing waves' critical path.
  p.dma_upper = d->dtype == CSR_BF16 && rows <= p.bm / 2 && !g_ovr.dma_all_waves ? 1 : 0;
  const int64_t base = (int64_t)batch * d->num_kv_heads * p.mtiles;
  const int ntiles = (max_L + max_q + 63) / 64;
  int nsplit = 1;
  if (g_ovr.nsplit > 0) {
    nsplit = g_ovr.nsplit;
  } else {
    const int cus = device_cus() * (p.four_waves ? 2 : 1);  // resident workgroups
    if (base > 0 && base < cus) {
      nsplit = (int)((cus + base - 1) / base);
      // bf16: keep >= 8 key tiles per split (its 4-stage DMA pipeline takes
      // 3 tiles to fill); the fp32 kernel stages one tile ahead and splits
      // down to a tile per split
      const int min_tiles = d->dtype == CSR_BF16 ? 8 : 1;
      const int cap = ntiles / min_tiles > 1 ? ntiles / min_tiles : 1;
      if (nsplit > cap) nsplit = cap;
    }
  }
  if (nsplit > ntiles) nsplit = ntiles > 0 ? ntiles : 1;
  if (nsplit < 1) nsplit = 1;
  p.nsplit = nsplit;
  const int64_t units = base * nsplit;
  if (units >= (1ll << 31) - 8) return fail(CSR_E_UNSUPPORTED, "too many work units (%lld)", (long long)units);
  p.n_units = (int)units;
  p.xcd_remap = max_L >= max_q ? 1 : 0;
  if (nsplit > 1) {
    const size_t rows_all = (size_t)total_q * d->num_q_heads;
    p.ws_o = (size_t)nsplit * rows_all * d->head_dim * sizeof(float);
    p.ws_lse = (size_t)nsplit * rows_all * sizeof(float);
    p.ws_bytes = ((p.ws_o + 255) & ~(size_t)255) + p.ws_lse;
  } else {
    p.ws_o = p.ws_lse = p.ws_bytes = 0;
  }
  // Ragged batches: units differ in length by up to the ratio of the longest
  // to the shortest sequence, so a device-side plan orders them longest first
  // per XCD.  Slots per XCD: an eighth of all units plus one whole group (no
  // subgroup is larger), so the plan's greedy assignment always finds an XCD
  // with room.
  p.order_slots = 0;
  p.ws_order_off = 0;
  if (!g_ovr.fixed_order && batch > 1 && (int64_t)batch * d->num_kv_heads <= 1024) {
    p.order_slots = (int)((units + 7) / 8 + (int64_t)p.mtiles * nsplit);
    p.ws_order_off = align256(p.ws_bytes);
    p.ws_bytes = p.ws_order_off + (size_t)8 * p.order_slots * sizeof(int32_t);
  }
  return CSR_OK;
}

csr_status check_common(const csr_attn_desc* d, int batch, int total, const void* q, const void* k,
                        const void* v, void* out, float* lse, const int32_t* cu) {
  csr_status st = check_desc(d);
  if (st != CSR_OK) return st;
  if (batch < 0 || total < 0) return fail(CSR_E_INVAL, "negative batch (%d) or token count (%d)", batch, total);
  if (batch == 0 && total != 0) return fail(CSR_E_INVAL, "batch 0 with %d tokens", total);
  if (total == 0) return CSR_OK;
  if (!q || !k || !v || !out || !cu) return fail(CSR_E_INVAL, "q, k, v, out and cu_seqlens must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(CSR_E_INVAL, "q, k, v and out must be 16-byte aligned");
  if (lse && !aligned4(lse)) return fail(CSR_E_INVAL, "lse must be 4-byte aligned");
  if (!aligned4(cu)) return fail(CSR_E_INVAL, "cu_seqlens must be 4-byte aligned");
  return CSR_OK;
}

csr_status check_pool(const csr_attn_desc* d, const void* k_pool, const void* v_pool, int num_pages,
                      const int32_t* block_table, int bt_stride, int max_len, const char* what) {
  (void)d;
  if (!k_pool || !v_pool) return fail(CSR_E_INVAL, "%s: k_pool and v_pool must be non-NULL", what);
  if (!aligned16(k_pool) || !aligned16(v_pool)) return fail(CSR_E_INVAL, "%s: pools must be 16-byte aligned", what);
  if (num_pages < 1) return fail(CSR_E_INVAL, "%s: num_pages must be >= 1", what);
  if (bt_stride < 1) return fail(CSR_E_INVAL, "%s: bt_stride must be >= 1", what);
  if ((int64_t)bt_stride * d->page_size < max_len)
    return fail(CSR_E_INVAL, "%s: bt_stride %d pages of %d cannot hold %d positions", what, bt_stride,
                d->page_size, max_len);
  if (block_table && !aligned4(block_table)) return fail(CSR_E_INVAL, "%s: block_table must be 4-byte aligned", what);
  return CSR_OK;
}

csr_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(CSR_E_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return CSR_OK;
}

csr::AppendArgs append_args(const csr_attn_desc* d, int batch, const void* k_new, const void* v_new, void* k_pool,
                            void* v_pool, int num_pages, const int32_t* bt, int bt_stride, const int32_t* cu,
                            const int32_t* cache_len, int total_q) {
  csr::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.block_table = bt;
  a.cu_q = cu;
  a.cache_len = cache_len;
  a.num_pages = num_pages;
  a.bt_stride = bt_stride;
  a.batch = batch;
  a.total_q = total_q;
  a.Hkv = d->num_kv_heads;
  a.P = d->page_size;
  a.log2P = ilog2(d->page_size);
  a.row_chunks = d->head_dim * elem_bytes(d) / 16;
  return a;
}

// Shared body of extend attention and prefill (cache_len == NULL, max_L == 0).
csr_status run_attention(const csr_attn_desc* d, int batch, const void* q, const void* k_new, const void* v_new,
                         const void* k_pool, const void* v_pool, int num_pages, const int32_t* bt, int bt_stride,
                         const int32_t* cu, const int32_t* cache_len, int total_q, int max_q, int max_L, void* out,
                         float* lse, void* ws, size_t ws_bytes, hipStream_t stream,
                         const csr::AppendArgs* app = nullptr) {
  Plan p;
  csr_status st = make_plan(d, batch, total_q, max_q, max_L, p);
  if (st != CSR_OK) return st;
  if (p.ws_bytes > 0) {
    if (!ws) return fail(CSR_E_WORKSPACE, "workspace of %zu bytes required, got NULL", p.ws_bytes);
    if (ws_bytes < p.ws_bytes)
      return fail(CSR_E_WORKSPACE, "workspace of %zu bytes required, got %zu", p.ws_bytes, ws_bytes);
    if (!aligned16(ws)) return fail(CSR_E_INVAL, "workspace must be 16-byte aligned");
  }
  // The append writes only slots [L_b, L_b + n_b), which this attention
  // never reads: with a merge launch it rides along in that launch, else it
  // is a launch of its own.
  if (app && p.nsplit == 1) {
    st = launched(csr::launch_append(*app, stream), "kv_append");
    if (st != CSR_OK) return st;
  }
  const int G = d->num_q_heads / d->num_kv_heads;
  const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.f / sqrtf((float)d->head_dim);
  csr::AttnArgs a{};
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.block_table = bt;
  a.cu_q = cu;
  a.cache_len = cache_len;
  a.out = out;
  a.lse = lse;
  a.part_o = p.nsplit > 1 ? static_cast<float*>(ws) : nullptr;
  a.part_lse = p.nsplit > 1 ? reinterpret_cast<float*>(static_cast<char*>(ws) + ((p.ws_o + 255) & ~(size_t)255))
                            : nullptr;
  a.num_pages = num_pages;
  a.bt_stride = bt_stride;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.G = G;
  a.d = d->head_dim;
  a.P = d->page_size;
  a.log2P = ilog2(d->page_size);
  // an fp8 cache holds K / k_scale and V / v_scale: the scales come back in the
  // score scale and in the output
  a.scale_log2 = scale * 1.4426950408889634f * (kv_fp8(d) ? d->k_scale : 1.f) * (qk_fp8(d) ? d->q_scale : 1.f);
  a.v_scale = kv_fp8(d) ? d->v_scale : 1.f;
  a.qk8 = qk_fp8(d) ? 1 : 0;
  a.kv_fp8 = kv_fp8(d) ? 1 : 0;
  a.four_waves = p.four_waves;
  a.dma_upper = p.dma_upper;
  a.batch = batch;
  a.total_q = total_q;
  a.mtiles = p.mtiles;
  a.nsplit = p.nsplit;
  a.n_units = p.n_units;
  a.xcd_remap = p.xcd_remap;
  a.order = nullptr;
  a.order_slots = 0;
  a.wg_clock = g_wg_clock;
  a.wg_clock_cap = g_wg_clock_cap;
  if (p.order_slots > 0) {
    csr::PlanArgs pa;
    pa.cu_q = cu;
    pa.cache_len = cache_len;
    pa.order = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + p.ws_order_off);
    pa.batch = batch;
    pa.Hkv = d->num_kv_heads;
    pa.G = G;
    pa.bm = p.bm;
    pa.mtiles = p.mtiles;
    pa.nsplit = p.nsplit;
    pa.slots = p.order_slots;
    pa.rt_per_sub = csr::plan_subgroup_rows(batch, d->num_kv_heads, p.mtiles);
    st = launched(csr::launch_plan(pa, stream), "work order");
    if (st != CSR_OK) return st;
    a.order = pa.order;
    a.order_slots = p.order_slots;
  }
  if (g_ev_begin && hipEventRecord(g_ev_begin, stream) != hipSuccess)
    return fail(CSR_E_HIP, "hipEventRecord(begin) failed");
  st = launched(csr::launch_attention(a, d->dtype == CSR_BF16, stream), "attention");
  if (st != CSR_OK) return st;
  if (g_ev_end && hipEventRecord(g_ev_end, stream) != hipSuccess) return fail(CSR_E_HIP, "hipEventRecord(end) failed");
  if (p.nsplit == 1) return st;
  csr::MergeArgs m{};
  if (app) m.append = *app;
  m.part_o = a.part_o;
  m.part_lse = a.part_lse;
  m.out = out;
  m.lse = lse;
  m.nsplit = p.nsplit;
  m.total_q = total_q;
  m.Hq = d->num_q_heads;
  m.d = d->head_dim;
  return launched(csr::launch_merge(m, d->dtype == CSR_BF16, stream), "split-K merge");
}


// ---- Scratch of csr_extend_attention_noalloc: one array per device, in the
// library's code object, holding what the workspace holds for
// csr_extend_attention.  Host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (the array's name in
// host code is a host-side stand-in, not a device address).
constexpr size_t kNoAllocScratchBytes = (size_t)CSR_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device, looked up on the first
// call for that device (with the device current) and kept for the process.
csr_status scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CSR_E_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(CSR_E_UNSUPPORTED, "device %d beyond the %d the library tracks", dev,
                                                 kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(CSR_E_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CSR_OK;
}

}  // namespace

extern "C" {

const char* csr_status_string(int32_t s) {
  switch (s) {
    case CSR_OK: return "CSR_OK";
    case CSR_E_INVAL: return "CSR_E_INVAL";
    case CSR_E_UNSUPPORTED: return "CSR_E_UNSUPPORTED";
    case CSR_E_WORKSPACE: return "CSR_E_WORKSPACE";
    case CSR_E_HIP: return "CSR_E_HIP";
  }
  return "CSR_E_UNKNOWN";
}

const char* csr_last_error(void) { return g_last_error.c_str(); }

csr_status csr_set_attention_events(void* begin_event, void* end_event) {
  if ((begin_event == nullptr) != (end_event == nullptr))
    return fail(CSR_E_INVAL, "set both events or neither");
  g_ev_begin = static_cast<hipEvent_t>(begin_event);
  g_ev_end = static_cast<hipEvent_t>(end_event);
  return CSR_OK;
}

csr_status csr_set_workgroup_clock(void* stamps, int32_t capacity) {
  if ((stamps == nullptr) != (capacity == 0) || capacity < 0)
    return fail(CSR_E_INVAL, "workgroup clock: a buffer and a positive capacity, or NULL and 0 (got %p, %d)", stamps,
                capacity);
  if (reinterpret_cast<uintptr_t>(stamps) % 8 != 0) return fail(CSR_E_INVAL, "workgroup clock buffer not 8-byte aligned");
  g_wg_clock = static_cast<uint64_t*>(stamps);
  g_wg_clock_cap = capacity;
  return CSR_OK;
}

csr_status csr_set_plan_overrides(int32_t nsplit, int32_t fixed_order, int32_t dma_all_waves) {
  if (nsplit < 0 || (fixed_order != 0 && fixed_order != 1) || (dma_all_waves != 0 && dma_all_waves != 1))
    return fail(CSR_E_INVAL, "plan overrides: nsplit >= 0, flags 0 or 1 (got %d, %d, %d)", nsplit, fixed_order,
                dma_all_waves);
  g_ovr.nsplit = nsplit;
  g_ovr.fixed_order = fixed_order;
  g_ovr.dma_all_waves = dma_all_waves;
  return CSR_OK;
}

csr_status csr_kv_append(const csr_attn_desc* desc, int32_t batch, const void* k_new, const void* v_new,
                         void* k_pool, void* v_pool, int32_t num_pages, const int32_t* block_table,
                         int32_t bt_stride, const int32_t* cu_seqlens_q, const int32_t* cache_seqlens,
                         int32_t total_q, void* stream) {
  g_last_error.clear();
  csr_status st = check_desc(desc);
  if (st != CSR_OK) return st;
  if (batch < 0 || total_q < 0) return fail(CSR_E_INVAL, "negative batch or total_q");
  if (total_q == 0) return CSR_OK;
  if (batch == 0) return fail(CSR_E_INVAL, "batch 0 with %d tokens", total_q);
  if (!k_new || !v_new || !cu_seqlens_q) return fail(CSR_E_INVAL, "k_new, v_new and cu_seqlens_q must be non-NULL");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(CSR_E_INVAL, "k_new and v_new must be 16-byte aligned");
  st = check_pool(desc, k_pool, v_pool, num_pages, block_table, bt_stride, 0, "kv_append");
  if (st != CSR_OK) return st;
  if (cache_seqlens && !aligned4(cache_seqlens)) return fail(CSR_E_INVAL, "cache_seqlens must be 4-byte aligned");
  if (needs_prep(desc)) {
    const csr::RopeArgs r = rope_args(desc, batch, nullptr, k_new, v_new, nullptr, nullptr, nullptr, k_pool, v_pool,
                                      num_pages, block_table, bt_stride, cu_seqlens_q, cache_seqlens, total_q);
    return launched(csr::launch_rope_append(r, desc->dtype == CSR_BF16, static_cast<hipStream_t>(stream)),
                    "prepared kv_append");
  }
  const csr::AppendArgs a = append_args(desc, batch, k_new, v_new, k_pool, v_pool, num_pages, block_table, bt_stride,
                                        cu_seqlens_q, cache_seqlens, total_q);
  return launched(csr::launch_append(a, static_cast<hipStream_t>(stream)), "kv_append");
}

size_t csr_extend_workspace_size(const csr_attn_desc* desc, int32_t batch, int32_t total_q, int32_t max_seqlen_q,
                                 int32_t max_cache_len) {
  if (check_desc(desc) != CSR_OK || batch < 1 || total_q < 1 || max_seqlen_q < 1 || max_cache_len < 0) return 0;
  Plan p;
  if (make_plan(desc, batch, total_q, max_seqlen_q, max_cache_len, p) != CSR_OK) return 0;
  return prep_layout(desc, total_q).bytes + p.ws_bytes;
}

size_t csr_prefill_workspace_size(const csr_attn_desc* desc, int32_t batch, int32_t total, int32_t max_seqlen) {
  return csr_extend_workspace_size(desc, batch, total, max_seqlen, 0);
}

csr_status csr_extend_attention(const csr_attn_desc* desc, int32_t batch, const void* q, const void* k_new,
                                const void* v_new, void* k_pool, void* v_pool, int32_t num_pages,
                                const int32_t* block_table, int32_t bt_stride, const int32_t* cu_seqlens_q,
                                const int32_t* cache_seqlens, int32_t total_q, int32_t max_seqlen_q,
                                int32_t max_cache_len, uint32_t flags, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  csr_status st = check_common(desc, batch, total_q, q, k_new, v_new, out, lse, cu_seqlens_q);
  if (st != CSR_OK || total_q == 0) return st;
  if (flags & ~CSR_APPEND) return fail(CSR_E_INVAL, "unknown flags 0x%x", flags);
  if (max_seqlen_q < 1 || max_cache_len < 0)
    return fail(CSR_E_INVAL, "max_seqlen_q must be >= 1 and max_cache_len >= 0");
  if (max_seqlen_q > total_q) return fail(CSR_E_INVAL, "max_seqlen_q %d exceeds total_q %d", max_seqlen_q, total_q);
  const bool need_pool = max_cache_len > 0 || (flags & CSR_APPEND);
  if (need_pool) {
    // Each of L_b and n_b must fit a table row; their per-sequence sum is a
    // caller contract (the host does not see the device-side lengths).
    st = check_pool(desc, k_pool, v_pool, num_pages, block_table, bt_stride,
                    max_cache_len > max_seqlen_q ? max_cache_len : max_seqlen_q, "extend_attention");
    if (st != CSR_OK) return st;
  }
  if (max_cache_len > 0 && !cache_seqlens)
    return fail(CSR_E_INVAL, "cache_seqlens must be non-NULL when max_cache_len > 0");
  if (cache_seqlens && !aligned4(cache_seqlens)) return fail(CSR_E_INVAL, "cache_seqlens must be 4-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Validate the plan (workspace) before enqueuing anything.
  Plan p;
  st = make_plan(desc, batch, total_q, max_seqlen_q, max_cache_len, p);
  if (st != CSR_OK) return st;
  const PrepLayout pl = prep_layout(desc, total_q);
  if (pl.bytes + p.ws_bytes > 0) {
    if (!workspace || workspace_bytes < pl.bytes + p.ws_bytes)
      return fail(CSR_E_WORKSPACE, "workspace of %zu bytes required, got %zu", pl.bytes + p.ws_bytes,
                  workspace ? workspace_bytes : (size_t)0);
    if (!aligned16(workspace)) return fail(CSR_E_INVAL, "workspace must be 16-byte aligned");
  }
  const bool append = (flags & CSR_APPEND) != 0;
  if (pl.bytes > 0) {
    // One launch rotates q and k_new at L_b + i and/or quantises k_new and
    // v_new into the workspace (and appends); the attention then reads the
    // prepared copies.
    char* ws = static_cast<char*>(workspace);
    const bool pq = prep_q(desc), fp8 = kv_fp8(desc);
    const csr::RopeArgs r = rope_args(desc, batch, q, k_new, v_new, ws + pl.q_off, ws + pl.k_off, ws + pl.v_off,
                                      append ? k_pool : nullptr, append ? v_pool : nullptr, num_pages, block_table,
                                      bt_stride, cu_seqlens_q, cache_seqlens, total_q);
    st = launched(csr::launch_rope_append(r, desc->dtype == CSR_BF16, s), "prep");
    if (st != CSR_OK) return st;
    return run_attention(desc, batch, pq ? ws + pl.q_off : q, ws + pl.k_off, fp8 ? ws + pl.v_off : v_new, k_pool,
                         v_pool, num_pages, block_table, bt_stride, cu_seqlens_q,
                         max_cache_len > 0 ? cache_seqlens : nullptr, total_q, max_seqlen_q, max_cache_len, out, lse,
                         p.ws_bytes ? ws + pl.bytes : nullptr, workspace_bytes - pl.bytes, s);
  }
  const csr::AppendArgs app = append_args(desc, batch, k_new, v_new, k_pool, v_pool, num_pages, block_table,
                                          bt_stride, cu_seqlens_q, cache_seqlens, total_q);
  return run_attention(desc, batch, q, k_new, v_new, k_pool, v_pool, num_pages, block_table, bt_stride, cu_seqlens_q,
                       max_cache_len > 0 ? cache_seqlens : nullptr, total_q, max_seqlen_q, max_cache_len, out, lse,
                       workspace, workspace_bytes, s, append ? &app : nullptr);
}

csr_status csr_extend_attention_noalloc(const csr_attn_desc* desc, int32_t batch, const void* q, const void* k_new,
                                        const void* v_new, void* k_pool, void* v_pool, int32_t num_pages,
                                        const int32_t* block_table, int32_t bt_stride, const int32_t* cu_seqlens_q,
                                        const int32_t* cache_seqlens, int32_t total_q, int32_t max_seqlen_q,
                                        int32_t max_cache_len, uint32_t flags, void* out, float* lse, void* stream) {
  g_last_error.clear();
  const size_t need =
      total_q > 0 ? csr_extend_workspace_size(desc, batch, total_q, max_seqlen_q, max_cache_len) : (size_t)0;
  if (need > kNoAllocScratchBytes)
    return fail(CSR_E_WORKSPACE, "this call needs %zu bytes of scratch; the no-allocation entry point has %zu",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    const csr_status st = scratch_of_current_device(&ws);
    if (st != CSR_OK) return st;
  }
  return csr_extend_attention(desc, batch, q, k_new, v_new, k_pool, v_pool, num_pages, block_table, bt_stride,
                              cu_seqlens_q, cache_seqlens, total_q, max_seqlen_q, max_cache_len, flags, out, lse, ws,
                              need > 0 ? kNoAllocScratchBytes : 0, stream);
}

csr_status csr_prefill(const csr_attn_desc* desc, int32_t batch, const void* q, const void* k, const void* v,
                       void* k_pool, void* v_pool, int32_t num_pages, const int32_t* block_table, int32_t bt_stride,
                       const int32_t* cu_seqlens, int32_t total, int32_t max_seqlen, void* out, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  csr_status st = check_common(desc, batch, total, q, k, v, out, lse, cu_seqlens);
  if (st != CSR_OK || total == 0) return st;
  if (max_seqlen < 1 || max_seqlen > total) return fail(CSR_E_INVAL, "max_seqlen must be in [1, total]");
  const bool write_cache = k_pool != nullptr || v_pool != nullptr;
  if (write_cache) {
    st = check_pool(desc, k_pool, v_pool, num_pages, block_table, bt_stride, max_seqlen, "prefill");
    if (st != CSR_OK) return st;
  }
  Plan p;
  st = make_plan(desc, batch, total, max_seqlen, 0, p);
  if (st != CSR_OK) return st;
  const PrepLayout pl = prep_layout(desc, total);
  if (pl.bytes + p.ws_bytes > 0) {
    if (!workspace || workspace_bytes < pl.bytes + p.ws_bytes)
      return fail(CSR_E_WORKSPACE, "workspace of %zu bytes required, got %zu", pl.bytes + p.ws_bytes,
                  workspace ? workspace_bytes : (size_t)0);
    if (!aligned16(workspace)) return fail(CSR_E_INVAL, "workspace must be 16-byte aligned");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (pl.bytes > 0) {
    char* ws = static_cast<char*>(workspace);
    const bool pq = prep_q(desc), fp8 = kv_fp8(desc);
    const csr::RopeArgs r = rope_args(desc, batch, q, k, v, ws + pl.q_off, ws + pl.k_off, ws + pl.v_off,
                                      write_cache ? k_pool : nullptr, write_cache ? v_pool : nullptr, num_pages,
                                      block_table, bt_stride, cu_seqlens, nullptr, total);
    st = launched(csr::launch_rope_append(r, desc->dtype == CSR_BF16, s), "prep");
    if (st != CSR_OK) return st;
    return run_attention(desc, batch, pq ? ws + pl.q_off : q, ws + pl.k_off, fp8 ? ws + pl.v_off : v, nullptr,
                         nullptr, 0, nullptr, 1, cu_seqlens, nullptr, total, max_seqlen, 0, out, lse,
                         p.ws_bytes ? ws + pl.bytes : nullptr, workspace_bytes - pl.bytes, s);
  }
  if (write_cache) {
    const csr::AppendArgs a = append_args(desc, batch, k, v, k_pool, v_pool, num_pages, block_table, bt_stride,
                                          cu_seqlens, nullptr, total);
    st = launched(csr::launch_append(a, s), "prefill cache write");
    if (st != CSR_OK) return st;
  }
  return run_attention(desc, batch, q, k, v, nullptr, nullptr, 0, nullptr, 1, cu_seqlens, nullptr, total, max_seqlen,
                       0, out, lse, workspace, workspace_bytes, s);
}

}  // extern "C"
