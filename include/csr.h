/*
 * csr.h - C ABI of libcsr: cached-prefix extend attention for Cached State
 * Representations (CSR) on AMD MI355X (gfx950).
 *
 * The operation (paper Sec. II, eq. (causal_attention_1)-(causal_attention_3),
 * with the KV cache of eq. (K_cache)-(V_cache)): a chunk of n_b new query tokens
 * of sequence b sits at absolute positions L_b .. L_b + n_b - 1 behind a cached
 * prefix of L_b tokens.  For chunk row i, query head h and kv head
 * g = h / (Hq / Hkv):
 *     keys t = 0 .. L_b + i (inclusive; prefix fully visible, causal inside
 *     the chunk), k_t / v_t from the paged cache for t < L_b and from the
 *     chunk's own K/V rows for t >= L_b;
 *     o = softmax(scale * q K^T) V,  lse = ln sum_t exp(scale * <q, k_t>).
 * L_b is the reused-prefix length of the paper's CSR structure: i* = L_b + 1
 * (eq. (csr_i_star)), i.e. the static part X_static is cached and the chunk is
 * the new state chunk plus the dynamic suffix X_dyn.  L_b = 0 is the full
 * re-prefill that asynchronous state reconciliation runs at eviction
 * (Algorithm 1, warm-up; Theorem 4).
 *
 * Rotary position embedding (optional, csr_attn_desc.rope_style): the paper's
 * q_n and k_n are the projections of the token at position n; models of the
 * family it deploys rotate both at that position first (RoFormer, Su et al.
 * 2021).  With rope_style set, the library applies the rotation itself at the
 * absolute cache position L_b + i of each chunk row, to q and k_new, before the
 * attention and before the append, so a cached key is rotated exactly once and
 * never moves again (prefix stability, Theorem 1).  The first r = rope_dim dims
 * form r/2 pairs; pair i turns by pos * rope_theta^(-2i/r); CSR_ROPE_NEOX pairs
 * dim i with dim i + r/2, CSR_ROPE_INTERLEAVED pairs dim 2i with dim 2i + 1;
 * dims >= r pass through.  Rotated q and k values are the fp64 rotation
 * (x cos - x' sin with cos and sin of the fp64 angle, each product rounded, no
 * fused multiply-add) rounded once to the element type (nearest, ties to
 * even; with an fp8 cache the key's code is taken from that value rounded to
 * fp32).  Keys that are already in the cache are read as stored.
 *
 * FP8 KV cache (optional, csr_attn_desc.kv_dtype = CSR_KV_FP8_E4M3): the pools
 * hold OCP e4m3 codes (1 byte: sign, 4 exponent bits with bias 7, 3 mantissa
 * bits, no infinities, S.1111.111 = NaN, largest finite 448), one byte per
 * element, with one dequantisation scale per tensor: a cached key is
 * code * k_scale, a value code * v_scale.  The chunk's keys (after RoPE) and
 * values arrive in bf16 and are stored as
 * e4m3_nearest_even(clamp(x * fp32(1 / scale), -448, 448)); the attention
 * reads the chunk through that same quantisation, so a key is identical
 * whether it comes from the chunk or, on a later call, from the cache.  The
 * attention converts codes to bf16 exactly and computes as for bf16 (fp32
 * accumulation); q and the output stay bf16.  Needs dtype CSR_BF16, d = 128.
 * FP8 score products (q_scale > 0): each (rotated) query element is
 * quantised by the same rule under q_scale, e4m3_nearest_even(clamp(
 * x * fp32(1 / q_scale), -448, 448)), and the scores are q_scale * k_scale *
 * sum of code products, evaluated on the fp8 matrix cores with fp32
 * accumulation; the probabilities and values stay bf16.  The caller picks
 * q_scale so that |q| / q_scale stays within 448.
 *
 * Memory layout (all row-major, element type per csr_attn_desc.dtype):
 *   q                 [T_q][Hq][d]        T_q = cu_seqlens_q[batch]
 *   k_new, v_new      [T_q][Hkv][d]
 *   out               [T_q][Hq][d]        same element type as q
 *   lse               [T_q][Hq]           float (natural log), optional
 *   k_pool, v_pool    [num_pages][P][Hkv][d]   (uint8 codes with an fp8 cache)
 *   block_table       [batch][bt_stride]  int32 page ids
 * Position t of sequence b lives in pool slot page * P + t % P with
 * page = block_table[b * bt_stride + t / P].  A NULL block_table means the
 * contiguous cache page = b * bt_stride + t / P.
 *
 * Ownership: every pointer belongs to the caller.  Array arguments are device
 * pointers (HIP device memory) unless stated otherwise; integers passed by
 * value are host values, so no call synchronises with the device.  The library
 * allocates no memory; split-K partials live in the caller's workspace.
 *
 * Streams: every call enqueues its kernels on `stream` (a hipStream_t passed
 * as void*, NULL = the default stream) and returns without waiting.
 *
 * Errors: every argument is validated on the host before any work is
 * enqueued; a failed check returns CSR_E_INVAL / CSR_E_UNSUPPORTED /
 * CSR_E_WORKSPACE and enqueues nothing.  The only HIP runtime calls made
 * before the checks end are two queries the launch plan (and with it the
 * workspace size) depends on: hipGetDevice, and on the first call for a
 * device its CU count (cached for the process).  A launch error returns
 * CSR_E_HIP.  csr_last_error() gives a thread-local description of the last
 * failure.  Block-table contents are a caller contract: every page a call
 * touches must be a valid id in [0, num_pages); ids outside that range are
 * never dereferenced (attention reads some other in-bounds key row in its
 * place, the append row is dropped) so a bad table cannot fault the GPU, but
 * the result is then unspecified.
 *
 * Nothing in the environment changes what a call computes; the plan can be
 * steered only through csr_set_plan_overrides (testing and A/B measurement).
 */
#ifndef CSR_H
#define CSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CSR_OK = 0,
  CSR_E_INVAL = 1,        /* malformed argument (null pointer, bad size, misalignment) */
  CSR_E_UNSUPPORTED = 2,  /* well-formed but not implemented (head_dim, dtype) */
  CSR_E_WORKSPACE = 3,    /* workspace missing or smaller than the query says */
  CSR_E_HIP = 4           /* HIP runtime reported an error at launch */
} csr_status;

typedef enum { CSR_F32 = 0, CSR_BF16 = 1 } csr_dtype;

/* csr_extend_attention flags */
#define CSR_APPEND 1u /* also append the chunk's K/V to the cache (csr_kv_append) */

/* csr_attn_desc.kv_dtype */
typedef enum {
  CSR_KV_SAME = 0,      /* the cache holds the input type (csr_attn_desc.dtype) */
  CSR_KV_FP8_E4M3 = 1   /* OCP e4m3 codes with per-tensor scales k_scale, v_scale */
} csr_kv_dtype;

/* csr_attn_desc.rope_style */
typedef enum {
  CSR_ROPE_NONE = 0,        /* q and k arrive already carrying their positions */
  CSR_ROPE_NEOX = 1,        /* pairs (i, i + r/2) */
  CSR_ROPE_INTERLEAVED = 2  /* pairs (2i, 2i + 1) */
} csr_rope_style;

/* Attention geometry shared by every call. */
typedef struct {
  int32_t num_q_heads;   /* Hq >= 1 */
  int32_t num_kv_heads;  /* Hkv >= 1, Hq % Hkv == 0 (grouped-query attention, G = Hq/Hkv) */
  int32_t head_dim;      /* d: 64 or 128 */
  int32_t page_size;     /* P: power of two, 1 .. 1024 */
  float softmax_scale;   /* > 0, or 0 for 1/sqrt(d) (the paper's 1/sqrt(d_k)) */
  int32_t dtype;         /* csr_dtype: CSR_BF16 (fp32 accumulate) or CSR_F32 */
  int32_t rope_style;    /* csr_rope_style; 0 (all fields zero) = no rotation */
  int32_t rope_dim;      /* r: rotated leading dims, a multiple of 16 in [16, d]; 0 = d */
  float rope_theta;      /* base of the pair frequencies, finite and > 0 (e.g. 1e4, 1e6) */
  int32_t kv_dtype;      /* csr_kv_dtype; 0 = the cache holds the input type */
  float k_scale;         /* fp8 cache: key dequantisation scale, finite and > 0 */
  float v_scale;         /* fp8 cache: value dequantisation scale, finite and > 0 */
  float q_scale;         /* fp8 cache only: > 0 selects fp8 score products (q quantised under
                            this scale like the keys); 0 = bf16 q */
} csr_attn_desc;

/*
 * Append the chunk's keys and values to the paged cache: the paper's
 * append-only growth T_{t+1} = T_t (+) dX_t (Theorem 2, eq.
 * (incremental_extensibility)).  Chunk row i of sequence b (row
 * cu_seqlens_q[b] + i of k_new / v_new) is copied bit for bit to cache
 * position L_b + i, for every kv head.  No other byte of either pool changes,
 * so every cached position < L_b stays as it was.  With desc->rope_style set,
 * each key row is rotated at its position L_b + i and rounded to the element
 * type instead of copied (values are still copied bit for bit); the pass is
 * fused into the same launch.  With an fp8 cache (desc->kv_dtype) keys and
 * values are quantised as the file comment defines.  Committing the appended
 * rows (advancing L_b) is the caller's choice: rows of the dynamic suffix are
 * simply overwritten by the next call.
 *   cu_seqlens_q   [batch+1] device int32 prefix sums of n_b
 *   cache_seqlens  [batch] device int32 L_b, or NULL for all zero
 *   total_q        host copy of cu_seqlens_q[batch]
 *   num_pages      number of pages in each pool (bounds the writes)
 * Pointers must be 16-byte aligned.
 */
csr_status csr_kv_append(const csr_attn_desc* desc, int32_t batch, const void* k_new,
                         const void* v_new, void* k_pool, void* v_pool, int32_t num_pages,
                         const int32_t* block_table, int32_t bt_stride,
                         const int32_t* cu_seqlens_q, const int32_t* cache_seqlens,
                         int32_t total_q, void* stream);

/*
 * Workspace bytes csr_extend_attention needs for these sizes: split-K
 * partials when the plan splits the key range, plus the prepared chunk when
 * RoPE or an fp8 cache is set (each part 256-byte aligned): rotated q
 * [T_q][Hq][d] (RoPE), prepared k [T_q][Hkv][d] (rotated and/or e4m3), e4m3
 * v [T_q][Hkv][d] (fp8 cache); 0 when none applies.  The same host integers
 * must be passed to the call.
 */
size_t csr_extend_workspace_size(const csr_attn_desc* desc, int32_t batch, int32_t total_q,
                                 int32_t max_seqlen_q, int32_t max_cache_len);

/*
 * Cached-prefix extend attention (see the file comment for the definition).
 *   q, k_new, v_new   the chunk's projections, layouts above
 *   k_pool, v_pool    the paged cache holding positions 0 .. L_b - 1; may be
 *                     NULL only if max_cache_len == 0 and CSR_APPEND is unset
 *   max_seqlen_q      host upper bound of n_b; max_cache_len host upper bound
 *                     of L_b (they size the launch; exceeding them is an error
 *                     the library cannot detect)
 *   flags             CSR_APPEND: also append the chunk exactly as
 *                     csr_kv_append does, within this call's stream work
 *                     (before the attention, or in the split-K merge launch
 *                     after it: the attention reads chunk keys from k_new /
 *                     v_new, or from their prepared workspace copies, and
 *                     never reads the slots being appended)
 *   q, k_new          with desc->rope_style set: unrotated projections; one
 *                     fused launch writes their rotations at L_b + i to the
 *                     workspace (and, with CSR_APPEND, the rotated keys and
 *                     the values to the cache) before the attention; with an
 *                     fp8 cache the same launch quantises k_new and v_new
 *   out               [T_q][Hq][d], element type of q
 *   lse               [T_q][Hq] float or NULL
 *   workspace         device scratch of >= csr_extend_workspace_size() bytes
 *                     (may be NULL when that size is 0); contents on entry
 *                     are ignored
 * Results are bitwise deterministic for a fixed set of host arguments.
 */
csr_status csr_extend_attention(const csr_attn_desc* desc, int32_t batch, const void* q,
                                const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                                int32_t num_pages, const int32_t* block_table, int32_t bt_stride,
                                const int32_t* cu_seqlens_q, const int32_t* cache_seqlens,
                                int32_t total_q, int32_t max_seqlen_q, int32_t max_cache_len,
                                uint32_t flags, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation as csr_extend_attention, with the same arguments except the
 * workspace.  The workspace lives in a scratch array of
 * CSR_NOALLOC_SCRATCH_BYTES that the library's code object holds on each
 * device it runs on, for as long as the process lives; the call allocates and
 * frees nothing.  Calls whose csr_extend_workspace_size exceeds that size
 * return CSR_E_WORKSPACE.  Every call on a device shares that device's array
 * (which keeps the last call's contents; nothing in it needs clearing), so
 * calls that overlap on one device - on different streams, or from different
 * threads without ordering - race and give undefined results.  On its first
 * call on a device (with that device current) the entry point looks the
 * array's address up with hipGetSymbolAddress, a HIP runtime call made before
 * the argument checks end; otherwise as csr_extend_attention.
 */
#define CSR_NOALLOC_SCRATCH_BYTES (64u << 20)
csr_status csr_extend_attention_noalloc(const csr_attn_desc* desc, int32_t batch, const void* q,
                                        const void* k_new, const void* v_new, void* k_pool,
                                        void* v_pool, int32_t num_pages,
                                        const int32_t* block_table, int32_t bt_stride,
                                        const int32_t* cu_seqlens_q, const int32_t* cache_seqlens,
                                        int32_t total_q, int32_t max_seqlen_q,
                                        int32_t max_cache_len, uint32_t flags, void* out,
                                        float* lse, void* stream);

/* Workspace bytes csr_prefill needs (split-K partials, rotated q/k with RoPE; 0 if neither). */
size_t csr_prefill_workspace_size(const csr_attn_desc* desc, int32_t batch, int32_t total,
                                  int32_t max_seqlen);

/*
 * Full causal re-prefill, L_b = 0 for every sequence: the warm-up that
 * recomputes the KV cache of the evicted state from scratch (i* = 1) in
 * asynchronous state reconciliation (Algorithm 1; Theorem 4, warm-up time).
 * Same computation as csr_extend_attention with no cached prefix.  If k_pool
 * is non-NULL the sequence's K/V are also written to the cache at positions
 * 0 .. n_b - 1 (the warmed-up cache), exactly as csr_kv_append with L_b = 0.
 * With desc->rope_style set, q and k are rotated at positions 0 .. n_b - 1
 * (the workspace then also holds the rotated copies, as for extend).
 */
csr_status csr_prefill(const csr_attn_desc* desc, int32_t batch, const void* q, const void* k,
                       const void* v, void* k_pool, void* v_pool, int32_t num_pages,
                       const int32_t* block_table, int32_t bt_stride, const int32_t* cu_seqlens,
                       int32_t total, int32_t max_seqlen, void* out, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Timing hook for profilers and benchmarks.  While set, every later
 * csr_extend_attention / csr_prefill call made on this thread enqueues
 * hipEventRecord(begin_event) immediately before its attention kernel and
 * hipEventRecord(end_event) immediately after it, on the call's stream, so the
 * caller can read that kernel's duration with hipEventElapsedTime.  The events
 * are hipEvent_t handles owned by the caller; pass NULL, NULL to switch the
 * hook off.  Returns CSR_E_INVAL if exactly one of them is NULL.
 */
csr_status csr_set_attention_events(void* begin_event, void* end_event);

/*
 * Profiling hook.  While set, the bf16 / fp8 attention kernel of every later
 * csr_extend_attention / csr_prefill call made on this thread records, for
 * each workgroup with id < capacity, four 64-bit words at stamps[4 * id]:
 * the constant 100 MHz clock (s_memrealtime; the rate HIP reports as
 * hipDeviceAttributeWallClockRate) when the workgroup started and
 * when it finished its key tiles, its key tiles (first << 32 | end), and
 * (sequence << 32 | split << 16 | kv head << 8 | XCD).  Workgroups without a
 * unit write nothing.  stamps is device memory owned by the caller (8-byte
 * aligned, 32 * capacity bytes); pass NULL, 0 to switch the hook off.
 * Results are unchanged.  Returns CSR_E_INVAL for a buffer without a
 * positive capacity or the reverse, or a misaligned buffer.
 */
csr_status csr_set_workgroup_clock(void* stamps, int32_t capacity);

/*
 * Testing and A/B measurement only: steer the launch plan of later
 * csr_extend_attention / csr_prefill calls and workspace queries made on this
 * thread (a workspace query and the call it sizes must see the same values).
 *   nsplit          > 0: split the key range of every unit into nsplit parts
 *                   (changes the summation order: results move within
 *                   rounding); 0: the planner's choice
 *   fixed_order     1: ragged batches run their units in index order instead
 *                   of the device-side longest-first order (identical results)
 *   dma_all_waves   1: short chunks load K/V from every wave instead of only
 *                   the waves without rows (identical results)
 * All zero restores the planner.  Returns CSR_E_INVAL for a negative nsplit or
 * flags other than 0 and 1.
 */
csr_status csr_set_plan_overrides(int32_t nsplit, int32_t fixed_order, int32_t dma_all_waves);

/* Static name of a status code (any int: values outside csr_status give "CSR_E_UNKNOWN"). */
const char* csr_status_string(int32_t status);

/* Thread-local description of the last failure on this thread ("" if none). */
const char* csr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CSR_H */
