/*
 * kvpattn.h — prefix-shared paged-KV attention for mixed RL rollout sessions, on AMD MI355X (gfx950).
 *
 * The operations follow the serving model of "Scheduling Mixed RL Rollouts Beyond Prefix Locality"
 * (MISA-T, arXiv 2608.11152):
 *   - KV state is held in fixed-size blocks of a paged pool, and each session retains a growing set of
 *     blocks (Sec. 2.3 on PagedAttention KV management; Sec. 3.2, the retained blocks k_s(t) of Eq. 2);
 *   - a prompt fans out into grouped samples that share the prompt prefix (Sec. 3.1, group id g_r), and
 *     prefix reuse is block-granular (Sec. 4.4: a request reuses the leading whole prompt blocks whose
 *     hashes are cached), so a group shares whole pages;
 *   - a later agentic turn prefills only its L - H new tokens over the cached history H (Eq. 1).
 * The attention itself is scaled dot-product softmax attention with grouped-query heads: query head h
 * reads KV head h / (num_q_heads / num_kv_heads).
 *
 * Conventions for every entry point
 *   - Return value: KVP_OK (0) or a negative kvp_status.  On a negative return nothing has been enqueued
 *     and no output has been touched; kvp_last_error() then holds a human-readable detail (thread-local).
 *   - "device" pointers are HIP device allocations owned by the caller; they must stay valid until the
 *     work enqueued on `stream` has completed.  "host" arrays are read during the call only; the library
 *     keeps no reference to them after it returns.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call is asynchronous on it.
 *   - Page ids read from device block tables are range-checked on the device.  An id outside
 *     [0, num_pages) is never dereferenced: the kernels skip that page and record KVP_ERANGE in the
 *     pool's device error word, which kv_pool_device_error() returns.  Such device-side errors are
 *     reported after the launch: the call has already returned KVP_OK and the outputs are written (a
 *     skipped page contributes nothing).  kvp_check_tables() validates a host copy of the tables before
 *     any launch, for callers that need the error up front.
 *   - There is no strided-tensor view of a pool layer (its layout below is not a plain strided array):
 *     kv_pool_layer_ptr() returns the raw layer instead.  Workspace sizes are queried per operation
 *     (paged_decode_workspace_size, prefix_chunk_prefill_workspace_size) rather than through one query
 *     taking an operation code.
 *   - Queries are bf16; outputs may be bf16 or fp32.  KV pages are bf16 (KVP_BF16) or OCP FP8 E4M3
 *     (KVP_FP8_E4M3, one byte per element with a per-layer K scale and V scale, see kv_pool_set_scales).
 *   - page_size is 16 tokens; head_dim is 64 or 128; num_q_heads / num_kv_heads is 1, 2, 4, 8 or 16.
 *
 * Pool layout in HBM (one layer):  bf16 [num_pages][num_kv_heads][2][16 * head_dim]
 *   Each (page, kv head) holds a K block then a V block of 16 * head_dim elements each.  Within them,
 *   token t (0..15 within the page) and dimension c are stored at
 *     K block:  ((c / 8) * 16 + t) * 8 + (c % 8)                       chunk-major rows of 8 dims
 *     V block:  (((c / 16) * 2 + s / 8) * 16 + (c % 16)) * 8 + (s % 8)  with slot s = pi(t)
 *   where pi(t) swaps bits 2 and 3 of t (an involution: V slots 0..7 hold tokens 0-3 and 8-11, slots
 *   8..15 hold tokens 4-7 and 12-15).  This order makes every operand load of the attention kernels a
 *   16-byte, fully used, contiguous access.  kv_pool_layer_ptr() exposes the raw layer for inspection.
 *
 * FP8 pools (KVP_FP8_E4M3): uint8 [num_pages][num_kv_heads][2][16 * head_dim], with byte positions
 *     K block:  (X * 16 + t) * 16 + ((c / 32) % 2) * 8 + (c % 8),   X = (c / 64) * 4 + (c % 32) / 8
 *     V block:  ((Y * 2 + s / 8) * 16 + (c % 16)) * 16 + ((c / 16) % 2) * 8 + (s % 8),   Y = c / 32
 *   (s = pi(t) as above), so one 16-byte load carries the operands of two matrix-core steps.  An element
 *   x is stored as the E4M3 code of y = fp32(x) * fp32(1 / scale), rounded to nearest with ties to the
 *   even mantissa and saturated to +-448 (NaN stays NaN); it reads back as code value * scale.
 */
#ifndef KVPATTN_H
#define KVPATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvp_pool* kvp_pool_t; /* opaque; created by kv_pool_create, owned by the library */

typedef enum kvp_status {
  KVP_OK = 0,
  KVP_EINVAL = -1,      /* null pointer, bad count, inconsistent shape or dtype                      */
  KVP_ERANGE = -2,      /* length beyond the block table (maxp * 16), or page id outside the pool    */
  KVP_EGROUP = -3,      /* bad group id, shared prefix longer than a member, or members' tables differ */
  KVP_ESHARED = -4,     /* kv_append would write into a page shared by a rollout group               */
  KVP_EWORKSPACE = -5,  /* workspace smaller than the size query returned                            */
  KVP_EUNSUPPORTED = -6,/* head_dim, page size, dtype or GQA ratio not supported                     */
  KVP_EHIP = -7,        /* HIP runtime error (detail in kvp_last_error)                              */
  KVP_ENOMEM = -8       /* device or pinned-host allocation failed                                   */
} kvp_status;

typedef enum kvp_dtype { KVP_BF16 = 0, KVP_F32 = 1, KVP_FP8_E4M3 = 2 } kvp_dtype;

/* Rollout-group prefix sharing (Sec. 3.1 group id g_r; Sec. 4.4 block-granular reuse).
 *   group_id[i]      host int32 [num_seqs]: group of sequence i, or -1 if ungrouped.
 *   shared_pages[g]  host int32 [num_groups]: the first shared_pages[g] entries of every member's block
 *                    table are the same physical pages (the group's whole prompt pages).
 * For decode it is an optimisation hint: the shared prefix is read once per group (once per 16 query
 * columns instead, for wide groups whose prompt is at most about 1% of the call's pages, which keeps the
 * launch on its fastest form) and merged with each member's private suffix by a log-sum-exp combine;
 * the result equals the ungrouped result.  The members that read the shared pages together (a group,
 * or a subgroup of a wide group) read them through the table row of their first decoding member, the
 * representative.  Because block tables are device-resident, the promise that the other members' first
 * shared_pages[g] entries equal the representative's is checked on the device: a member whose entries
 * differ makes the kernels record KVP_EGROUP in the pool's device error word (kv_pool_device_error), and
 * its output is then attention over the representative's pages for the shared range. */
typedef struct kvp_group_prefix {
  const int32_t* group_id;
  const int32_t* shared_pages;
  int32_t num_groups;
} kvp_group_prefix;

/* ---------------------------------------------------------------------------------------------------
 * Pool (Sec. 3.2: sessions retain KV blocks of a fixed-capacity instance pool)
 * ------------------------------------------------------------------------------------------------- */

/* Allocate a zero-filled pool of num_layers x num_pages pages on the current HIP device.
 * page_size must be 16, head_dim 64 or 128, dtype KVP_BF16 or KVP_FP8_E4M3.  *out receives the handle. */
int kv_pool_create(kvp_pool_t* out, int num_layers, int num_pages, int page_size, int num_kv_heads,
                   int head_dim, int dtype);

/* Free the pool and its device memory (synchronises the device first).  NULL is accepted. */
int kv_pool_destroy(kvp_pool_t pool);

/* Zero every page and clear the device error word, enqueued on `stream` (the weight-sync cache reset
 * of Sec. 5.2: cached prefixes become invalid after new weights are loaded). */
int kv_pool_reset(kvp_pool_t pool, void* stream);

/* Device address and byte size of one layer of the pool (layout in the file header). */
int kv_pool_layer_ptr(kvp_pool_t pool, int layer, void** dev_ptr, size_t* bytes);

/* Pool geometry: any output pointer may be NULL. */
int kv_pool_info(kvp_pool_t pool, int* num_layers, int* num_pages, int* num_kv_heads, int* head_dim);

/* KV element type of the pool (KVP_BF16 or KVP_FP8_E4M3). */
int kv_pool_dtype(kvp_pool_t pool, int* dtype);

/* Per-layer quantisation scales of an FP8 pool (both 1.0 when created): K elements are stored as
 * E4M3(k / k_scale) and V as E4M3(v / v_scale) by kv_append, and read back multiplied by the scale.
 * Set them before the layer's first append.  Errors: KVP_EINVAL for a scale that is not finite and
 * positive; KVP_EUNSUPPORTED for a bf16 pool. */
int kv_pool_set_scales(kvp_pool_t pool, int layer, float k_scale, float v_scale);

/* Synchronise the device, then return (in *code) and clear the first device-side error recorded by
 * kernels using this pool (KVP_OK if none). */
int kv_pool_device_error(kvp_pool_t pool, int* code);

/* ---------------------------------------------------------------------------------------------------
 * kv_append — write new tokens' K/V into their paged slots (a session's retained blocks grow, Sec. 3.2)
 * ------------------------------------------------------------------------------------------------- */

/* Sequence i appends the tokens k[cu_new[i] .. cu_new[i+1]) at logical positions start_pos[i] + j; the
 * token at position p goes to page block_tables[i * maxp + p / 16], slot p % 16, of every KV head.
 *   k, v          device bf16 [cu_new[num_seqs], num_kv_heads, head_dim] (token-major)
 *   block_tables  device int32 [num_seqs, maxp]
 *   start_pos     host int32 [num_seqs];  cu_new host int32 [num_seqs + 1], non-decreasing, cu_new[0]=0
 *   gp            host, nullable.  When given, a write into any of a member's first shared_pages[g]
 *                 pages is refused with KVP_ESHARED (shared prompt pages are written once, before the
 *                 group is formed, by an append without gp).
 * Errors: KVP_ERANGE if start_pos[i] + count > maxp * 16.  The copy is bit-exact (bf16 pools) or the
 * quantisation defined in the file header (FP8 pools). */
int kv_append(kvp_pool_t pool, int layer, const void* k, const void* v, const int32_t* block_tables,
              int maxp, const int32_t* start_pos, const int32_t* cu_new, int num_seqs,
              const kvp_group_prefix* gp, void* stream);

/* Read back tokens [0, lens[i]) of every sequence in logical order (inverse of kv_append), for
 * inspection and tests.  k_out, v_out: device bf16 [sum(lens), num_kv_heads, head_dim] (an FP8 pool
 * returns bf16(fp32(code value) * fp32(scale)), both roundings to nearest even);
 * block_tables device int32 [num_seqs, maxp]; lens host int32 [num_seqs]. */
int kv_gather(kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp, const int32_t* lens,
              int num_seqs, void* k_out, void* v_out, void* stream);

/* ---------------------------------------------------------------------------------------------------
 * paged_decode_attn — one query token per sequence over its paged KV (Sec. 3.1 groups, Sec. 4.4 reuse)
 * ------------------------------------------------------------------------------------------------- */

/* Workspace bytes paged_decode_attn needs for these lengths / groups (host arrays as below). */
int paged_decode_workspace_size(kvp_pool_t pool, const int32_t* seq_lens, int num_seqs,
                                const kvp_group_prefix* group_prefix, int num_q_heads, size_t* bytes);

/* out[i, h, :] = softmax(scale * q[i,h,:] . K_i[t, g(h), :]) over t < seq_lens[i], applied to V_i,
 * where K_i / V_i are read through block_tables row i and g(h) = h / (num_q_heads / num_kv_heads).
 *   q             device bf16 [num_seqs, num_q_heads, head_dim]
 *   block_tables  device int32 [num_seqs, maxp]
 *   seq_lens      host int32 [num_seqs]: cached tokens including the current one (0 = zero output)
 *   group_prefix  host, nullable: members' shared prompt pages are read once per group (see above)
 *   out           device [num_seqs, num_q_heads, head_dim], out_dtype KVP_BF16 or KVP_F32
 *   ws            device workspace of ws_bytes >= paged_decode_workspace_size(...)
 *   scale         softmax scale applied to q . k (finite, > 0; usually 1 / sqrt(head_dim))
 * Errors: KVP_ERANGE if seq_lens[i] > maxp * 16; KVP_EGROUP if a group id is out of range or a member's
 * seq_len is shorter than its group's shared pages; KVP_EWORKSPACE if ws_bytes is too small; KVP_EINVAL
 * if scale is not finite and positive.  After the launch (kv_pool_device_error): KVP_ERANGE for a page
 * id outside the pool, KVP_EGROUP for a member whose shared table entries differ from its group's
 * representative (see kvp_group_prefix). */
int paged_decode_attn(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp,
                      const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* group_prefix,
                      int num_q_heads, float scale, void* out, int out_dtype, void* ws, size_t ws_bytes,
                      void* stream);

/* paged_decode_attn without any allocation, for callers that cannot allocate memory during the call
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same arguments,
 * results and errors as paged_decode_attn, bitwise-identical outputs, but no workspace argument: the work
 * list and the split-KV partial states live in a scratch array of KVP_NOALLOC_SCRATCH_BYTES that the
 * library's code object holds in device memory (one copy per GPU, kept until the process ends), and the
 * work list reaches it through kernel launch arguments, so the call allocates neither device nor pinned
 * host memory.  The pool must live on the current device (else KVP_EINVAL).  A call whose work list plus
 * partials exceed the scratch returns KVP_EWORKSPACE before anything is enqueued (the RLVR batch of 512
 * sequences over 1k-16k tokens needs about 37 MiB).  Every call on one GPU shares that GPU's scratch, and
 * nothing in it needs clearing between calls: calls on one stream are ordered, but calls that overlap on
 * one GPU (concurrent streams, or host threads) race on the scratch and must be serialised by the
 * caller. */
#define KVP_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int paged_decode_attn_noalloc(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp,
                              const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* group_prefix,
                              int num_q_heads, float scale, void* out, int out_dtype, void* stream);

/* ---------------------------------------------------------------------------------------------------
 * prefix_chunk_prefill_attn — a new chunk attends to its cached history plus itself (Eq. 1: only the
 * L - H uncached tokens are prefilled over the reusable prefix H)
 * ------------------------------------------------------------------------------------------------- */

/* Workspace bytes prefix_chunk_prefill_attn needs. */
int prefix_chunk_prefill_workspace_size(kvp_pool_t pool, const int32_t* ctx_lens, const int32_t* cu_q,
                                        int num_seqs, int num_q_heads, size_t* bytes);

/* Session i's chunk queries q[cu_q[i] + j] sit at positions ctx_lens[i] + j, and row j attends keys
 * [0, ctx_lens[i] + j] of its sequence (bottom-right causal).  The chunk's own K/V must already have
 * been appended.
 *   q             device bf16 [cu_q[num_seqs], num_q_heads, head_dim]
 *   block_tables  device int32 [num_seqs, maxp] (row i = session i)
 *   ctx_lens      host int32 [num_seqs];  cu_q host int32 [num_seqs + 1]
 *   out           device [cu_q[num_seqs], num_q_heads, head_dim], out_dtype KVP_BF16 or KVP_F32
 *   scale         softmax scale applied to q . k (finite, > 0)
 * Errors: KVP_ERANGE if ctx_lens[i] + chunk > maxp * 16; KVP_EWORKSPACE if ws_bytes is too small;
 * KVP_EINVAL if scale is not finite and positive. */
int prefix_chunk_prefill_attn(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables,
                              int maxp, const int32_t* ctx_lens, const int32_t* cu_q, int num_seqs,
                              int num_q_heads, float scale, void* out, int out_dtype, void* ws,
                              size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------------
 * mixed_step_attn — one launch for a serving step that decodes some sequences and prefills chunks of
 * others on the same pool (Sec. 2.4 and Table 1: the rollout classes share one inference instance; the
 * decode of Sec. 3.1 groups and the chunk prefill of Eq. 1 run side by side)
 * ------------------------------------------------------------------------------------------------- */

/* Workspace bytes mixed_step_attn needs (host arrays as below; either part may be empty). */
int mixed_step_workspace_size(kvp_pool_t pool, const int32_t* seq_lens, int num_dec,
                              const kvp_group_prefix* group_prefix, const int32_t* ctx_lens, const int32_t* cu_q,
                              int num_pf, int num_q_heads, size_t* bytes);

/* paged_decode_attn(q_dec, pool, layer, block_tables_dec, maxp_dec, seq_lens, num_dec, group_prefix,
 * num_q_heads, scale, out_dec, out_dtype, ...) and prefix_chunk_prefill_attn(q_pf, pool, layer,
 * block_tables_pf, maxp_pf, ctx_lens, cu_q, num_pf, num_q_heads, scale, out_pf, out_dtype, ...) in one
 * kernel launch: the decode work is dispatched first and the prefill workgroups take the compute units as
 * the decode's retire, so neither the decode's tail nor a launch boundary idles the GPU.  Split-KV
 * partials of either part are merged by a second, small launch; shared-prefix ranges that the plan stages
 * through LDS (wide groups over long prompts) run in a launch of their own ahead of the fused one; a call
 * with one part empty makes that part's call.  Arguments, layouts and errors are those
 * of the two calls (num_dec = 0 or num_pf = 0 leaves that part out); both parts read one pool and layer,
 * and the prefill chunks' K/V must already have been appended.  Outputs are bitwise identical to the two
 * calls.  ws: device workspace of ws_bytes >= mixed_step_workspace_size(...). */
int mixed_step_attn(kvp_pool_t pool, int layer, int num_q_heads, float scale, int out_dtype, const void* q_dec,
                    const int32_t* block_tables_dec, int maxp_dec, const int32_t* seq_lens, int num_dec,
                    const kvp_group_prefix* group_prefix, void* out_dec, const void* q_pf,
                    const int32_t* block_tables_pf, int maxp_pf, const int32_t* ctx_lens, const int32_t* cu_q,
                    int num_pf, void* out_pf, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------------
 * CPU KV tier (Sec. 5.5: a host-memory tier keeps a backup copy of GPU-resident KV, so the GPU pool can
 * run close to capacity and pages evicted from it come back without recomputation)
 * ------------------------------------------------------------------------------------------------- */

/* Bytes of one pool page of one layer (all KV heads, K and V blocks): num_kv_heads * 32 * head_dim
 * bytes per element byte (64 * head_dim * num_kv_heads for bf16, half of that for FP8). */
int kv_pool_page_bytes(kvp_pool_t pool, size_t* bytes);

/* Copy pool pages page_ids[0 .. n) of `layer` to the host tier: page i goes to host_dst + i * page_bytes,
 * in the pool's page layout (file header), bit-exact.
 *   page_ids  host int32 [n] (ids may repeat)
 *   host_dst  pinned host memory (hipHostMalloc, or a torch tensor created with pin_memory=True) of
 *             n * page_bytes bytes; the GPU writes it directly, in one launch for all n pages.  It is
 *             complete once the work enqueued on `stream` has finished.
 * Errors: KVP_ERANGE if an id is outside [0, num_pages); KVP_EINVAL if host_dst is not pinned host
 * memory. */
int kv_offload(kvp_pool_t pool, int layer, const int32_t* page_ids, int n, void* host_dst, void* stream);

/* Copy host-tier page i (as kv_offload wrote it) into pool page page_ids[i] of `layer`, bit-exact, in
 * one launch.  When block_tables is not NULL, block_tables[rows[i] * maxp + lpages[i]] is also set to
 * page_ids[i] on the stream, so the restored page becomes logical page lpages[i] of table row rows[i].
 *   host_src      pinned host memory of n * page_bytes bytes
 *   page_ids      host int32 [n], distinct
 *   block_tables  device int32 [num_rows, maxp], nullable;  rows, lpages host int32 [n] (used with it)
 * Errors: KVP_ERANGE for a page id outside [0, num_pages) or lpages[i] outside [0, maxp); KVP_EINVAL if
 * a page id repeats, rows[i] is outside [0, num_rows), or host_src is not pinned host memory. */
int kv_restore(kvp_pool_t pool, int layer, const void* host_src, const int32_t* page_ids, int n,
               int32_t* block_tables, int num_rows, int maxp, const int32_t* rows, const int32_t* lpages,
               void* stream);

/* ---------------------------------------------------------------------------------------------------
 * Prompt-block hashing and prefix lookup (Sec. 4.4: the engine keys every full prompt block by a hash;
 * a request's reusable prefix H of Eq. 1 is the longest run of its leading blocks whose hashes are cached)
 *
 * Block hash (the paper does not specify one; this is the library's definition, all arithmetic mod 2^64):
 *   mix(z)   = SplitMix64 output function: z += 0x9E3779B97F4A7C15; z = (z ^ z>>30) * 0xBF58476D1CE4E5B9;
 *              z = (z ^ z>>27) * 0x94D049BB133111EB; z ^= z>>31
 *   local(k) = x after x = mix(x ^ (t[16k+2j] | t[16k+2j+1] << 32)) for j = 0..7, from x = 0
 *              (token ids as uint32)
 *   h(-1) = seed;  h(k) = h(k-1) * 0x9E3779B97F4A7C15 + local(k);  hash(k) = mix(h(k))
 * so hash(k) names the tokens [0, 16(k+1)) of a sequence: equal prefixes give equal hashes.  Only full
 * pages are hashed.  Hash slots are laid out per sequence: sequence i's floor(len_i / 16) hashes start
 * at sum_{j<i} floor(len_j / 16), with len_i = cu_tokens[i+1] - cu_tokens[i].
 * ------------------------------------------------------------------------------------------------- */

/* Block hashes of every full page of every sequence.
 *   tokens     device int32 [cu_tokens[num_seqs]] (token ids, sequences concatenated)
 *   cu_tokens  host int32 [num_seqs + 1], non-decreasing, cu_tokens[0] = 0
 *   hashes     device uint64 [total full pages] (layout above) */
int kvp_block_hashes(const int32_t* tokens, const int32_t* cu_tokens, int num_seqs, uint64_t seed,
                     uint64_t* hashes, void* stream);

/* Rollout-group shared prefix from block hashes: shared_pages[g] (device int32 [num_groups]) = the
 * number of leading full pages on which every member of group g has the same hash as its first member,
 * capped by the shortest member (0 for a group without members).  With the groups' prompt tokens this is
 * the kvp_group_prefix.shared_pages of decode (whole pages only).
 *   hashes, cu_tokens  as written by kvp_block_hashes;  group_id host int32 [num_seqs], -1 = ungrouped.
 * Errors: KVP_EGROUP for a group id outside [-1, num_groups). */
int kvp_group_shared_pages(const uint64_t* hashes, const int32_t* cu_tokens, int num_seqs,
                           const int32_t* group_id, int num_groups, int32_t* shared_pages, void* stream);

typedef struct kvp_prefix_table* kvp_prefix_table_t; /* device hash table: block hash -> pool page */

/* An empty table of 2^capacity_log2 slots (4..30) in device memory, 12 bytes per slot.
 * Open addressing with linear probing; a slot's page is the largest page id inserted for its hash, or
 * -1 after that page was erased.  A block hash of 0 is stored as 1. */
int kvp_prefix_table_create(kvp_prefix_table_t* out, int capacity_log2);
int kvp_prefix_table_destroy(kvp_prefix_table_t table);

/* Empty the table on `stream` (the cache reset after a weight sync, Sec. 5.2). */
int kvp_prefix_table_clear(kvp_prefix_table_t table, void* stream);

/* Record that pool page page_ids[i] holds the block named hashes[i] (device arrays of n entries).  When
 * the table is full an entry is dropped and kvp_prefix_table_error reports KVP_ENOMEM. */
int kvp_prefix_table_insert(kvp_prefix_table_t table, const uint64_t* hashes, const int32_t* page_ids,
                            int64_t n, void* stream);

/* Forget that page page_ids[i] holds block hashes[i] (a page evicted from the pool); entries that map
 * the hash to another page are left alone. */
int kvp_prefix_table_erase(kvp_prefix_table_t table, const uint64_t* hashes, const int32_t* page_ids,
                           int64_t n, void* stream);

/* Reusable prefix of each sequence: matched_pages[i] (device int32 [num_seqs]) = the number of leading
 * full pages whose hash the table maps to a page; page_ids (device int32 [total full pages], layout above)
 * receives those pages and -1 after the first miss.  H = 16 * matched_pages[i] tokens need no prefill. */
int kvp_prefix_lookup(kvp_prefix_table_t table, const uint64_t* hashes, const int32_t* cu_tokens,
                      int num_seqs, int32_t* matched_pages, int32_t* page_ids, void* stream);

/* Synchronise the device, then return (in *code) and clear the table's device error word. */
int kvp_prefix_table_error(kvp_prefix_table_t table, int* code);

/* ---------------------------------------------------------------------------------------------------
 * Host-side checks and diagnostics
 * ------------------------------------------------------------------------------------------------- */

/* Full host validation of a host copy of the block tables: every entry a sequence of length lens[i]
 * uses is in [0, num_pages) (else KVP_ERANGE), and every group member's first shared_pages[g] entries
 * equal those of the group's first member (else KVP_EGROUP).  gp may be NULL. */
int kvp_check_tables(const int32_t* block_tables_host, int maxp, const int32_t* lens, int num_seqs,
                     int num_pages, const kvp_group_prefix* gp);

/* Decode work plan, for inspection and tests (pure host computation, no device needed): the plan
 * paged_decode_attn uses for a bf16 pool (an FP8 pool's segments charge each chunk start more pages,
 * so their cut can differ).  Writes up to cap items of 8 int32 each into items_out:
 *   {kind (0 = private, 1 = shared prefix), table row, page_lo, page_hi, token_end, first member,
 *    member count, partial slot (-1 = writes the final output)}
 * and returns the item count in *n_items (which may exceed cap), the number of partial slots in
 * *n_partials, and the chosen pages per split in *pages_per_split. */
int kvp_plan_decode(const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* gp, int num_q_heads,
                    int num_kv_heads, int32_t* items_out, int cap, int* n_items, int* n_partials,
                    int* pages_per_split);

const char* kvp_strerror(int code);
const char* kvp_last_error(void);
const char* kvp_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KVPATTN_H */
