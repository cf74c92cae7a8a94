/*
 * lazy_attn.h - C ABI of the LazyAttention hot path for AMD Instinct MI355X (gfx950).
 *
 * LazyAttention (arXiv 2606.04302) keeps the KV cache free of positional encoding and applies RoPE inside the
 * attention kernel, at the position each retrieved chunk takes in the current request (Sec. 3.1 "Deferred
 * encoding"; Sec. 3.2 "Efficient Rotation with Tiling").  One stored copy of a chunk can therefore serve any number
 * of requests at different offsets, in the same batch, without writing a re-rotated copy (problem statement at the
 * start of Sec. 3).
 *
 * Conventions shared by every entry point
 *  - All tensors live in device memory and are owned by the caller.  The library allocates no device memory,
 *    never synchronises the device, and enqueues all work asynchronously on `stream` (a hipStream_t; NULL = the
 *    null stream).  Inputs are read-only; in particular the chunk store is never written, so concurrent requests
 *    that share a chunk cannot race (Sec. 1: in-place re-encoding races when two prompts share data).
 *  - Element type of q, k, v and out is bfloat16 (raw 16-bit storage, passed as void*); accumulation is fp32.
 *  - head_dim D is 64 or 128.  RoPE pairs dimension t with t + D/2 by default (half-split, the K1/K2 halves of
 *    Sec. 3.2 "Prefilling"; params->rope_style selects the interleaved pairs (2t, 2t+1) instead):
 *    x1' = x1 cos(p theta_t) - x2 sin(p theta_t), x2' = x1 sin(p theta_t) + x2 cos(p theta_t),
 *    theta_t = rope_base^(-2t/D) unless params->inv_freq supplies the D/2 frequencies (RoPE variants, Sec. 3.5).
 *  - GQA: query head h reads KV head h / (num_q_heads / num_kv_heads) (Sec. 3.5).
 *  - Causal rule: a key at position pk is visible to a query at position pq iff pk <= pq (positions, not table
 *    indices, decide, so chunks may sit at arbitrary offsets).  A query that sees no key yields out = 0 and
 *    lse = -inf.
 *  - Return value: LAZY_OK (0) on success, a negative LAZY_E* code otherwise.  Scalar arguments are checked on
 *    every call; the contents of device tables are only checked by lazy_attn_validate (host copies).  Errors
 *    never cross the ABI as exceptions.
 */
#ifndef LAZY_ATTN_H
#define LAZY_ATTN_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define LAZY_API __attribute__((visibility("default")))
#else
#define LAZY_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define LAZY_OK 0
#define LAZY_EINVAL (-1)       /* bad scalar argument or null pointer */
#define LAZY_EUNSUPPORTED (-2) /* valid request outside what the kernels implement (e.g. head_dim not 64/128) */
#define LAZY_EWORKSPACE (-3)   /* workspace missing or smaller than the *_workspace_size query returned */
#define LAZY_EHIP (-4)         /* the HIP runtime reported an error at launch */
#define LAZY_EDATA (-5)        /* lazy_attn_validate: a table entry breaks the layout contract */

/* Largest position (exclusive) a key or query may take. */
#define LAZY_MAX_POS (1 << 24)

/*
 * One use of a stored chunk by one request (the paper's per-document offset, Sec. 3.2 "Prefilling": a single
 * offset for the whole document).  The chunk's keys j = 0..len-1 take positions pos_offset + j in this request.
 * Storage is position-free and head-major: key j of KV head g is the D contiguous elements at
 *     k_pool + k_offset + (g * k_stride + j) * D
 * and its value at v_pool + v_offset + (g * v_stride + j) * D (offsets and strides in elements / tokens; a
 * stride is the chunk's capacity, >= len, so a growing decode tail can be appended in place).
 * Requirements: len >= 1, pos_offset >= 0, pos_offset + len <= LAZY_MAX_POS, k_stride >= len, v_stride >= len,
 * offsets >= 0 and multiples of 8 (16-byte alignment).  32 bytes, no padding.
 */
typedef struct lazy_chunk {
  int64_t k_offset;
  int64_t v_offset;
  int32_t len;
  int32_t pos_offset;
  int32_t k_stride;
  int32_t v_stride;
} lazy_chunk_t;

typedef struct lazy_attn_params {
  int32_t num_q_heads;   /* Hq */
  int32_t num_kv_heads;  /* Hkv, divides Hq */
  int32_t head_dim;      /* D: 64 or 128 */
  int32_t causal;        /* 1: position-based causal rule; 0: every key visible */
  float rope_base;       /* theta_t = rope_base^(-2t/D); ignored if inv_freq != NULL */
  float softmax_scale;   /* 0 => 1/sqrt(D) (Eqn. standard attention) */
  const float* inv_freq; /* optional device array of D/2 fp32 frequencies theta_t (scaled / NTK tables);
                            with LAZY_ALIBI: optional device array of Hq slopes */
  int32_t num_splits;    /* 0 => chosen by the library; otherwise the number of KV splits per request */
  int32_t key_positions; /* LAZY_KEYS_NOPE or LAZY_KEYS_LOCAL: how the chunk store holds its keys (below) */
  int32_t rope_style;    /* LAZY_ROPE_HALF, LAZY_ROPE_INTERLEAVED or LAZY_ALIBI: the positional method (below) */
  int32_t q_prerotated;  /* 0: q is position-free and the kernels rotate it; 1: q arrives already rotated (below) */
  int32_t cache_hint;    /* LAZY_CACHE_DEFAULT or LAZY_CACHE_STREAM: how the decode reads K and V (below) */
} lazy_attn_params_t;

/*
 * Rotation pairs (params->rope_style; Sec. 3.5 "RoPE-family variants").  Pair t (0 <= t < D/2) is rotated by
 * p * theta_t in both styles:
 *  LAZY_ROPE_HALF        (0): pair t = dimensions (t, t + D/2), the K1/K2 halves of Sec. 3.2 "Prefilling".
 *  LAZY_ROPE_INTERLEAVED (1): pair t = dimensions (2t, 2t + 1), as in Llama's reference implementation.
 * Q, K and the materialised copy follow the style; V and the output are not affected.
 *  LAZY_ALIBI            (2): no rotation at all; slope_h * (pos_k - pos_q) is added to every scaled score of query
 *                             head h (ALiBi, Sec. 3.5 "Score-space positional methods"), with positions taken from
 *                             the chunk table exactly as for RoPE.  slope_h = 2^(-8 (h+1) / Hq) unless params->inv_freq
 *                             points to a device table of Hq fp32 slopes (that field has no other use here).  Requires
 *                             key_positions = LAZY_KEYS_NOPE; rope_base is ignored; the materialise-then-attend
 *                             entry points return LAZY_EUNSUPPORTED (there is nothing to re-encode).
 *
 * Pre-rotated queries (params->q_prerotated = 1): q holds R(q_pos) q in the chosen pairing, as the paper's prefill
 * assumes (Sec. 3.2, tiling figure panel (b): only keys are rotated inside the kernel).  The kernels then leave the
 * query as it is where they would rotate it at q_pos, and where they rotate it by a relative offset q_pos - pos_offset
 * (decode over local-position keys, the chunk-major shared decode) they rotate it by -pos_offset instead, since
 * R(q_pos - pos_offset) q = R(-pos_offset) R(q_pos) q.  Positions still come from q_pos0 / q_pos for the causal rule.
 * No effect with LAZY_ALIBI (nothing is rotated).  Any value other than 0 or 1 is LAZY_EINVAL.
 */
#define LAZY_ROPE_HALF 0
#define LAZY_ROPE_INTERLEAVED 1
#define LAZY_ALIBI 2

/*
 * Cache hint for K and V (params->cache_hint; a performance choice only, results are bit-identical).
 *  LAZY_CACHE_DEFAULT (0): ordinary loads.  Right whenever the call's chunks are shared between its requests, or are
 *                          read again soon enough to still be in the last-level cache (a pool that fits in it).
 *  LAZY_CACHE_STREAM  (1): the decode entry points (lazy_attn_decode, lazy_plain_attn_decode,
 *                          lazy_attn_decode_noalloc, lazy_attn_decode_shared) read K and V with non-temporal loads,
 *                          which stream faster from HBM but give up the cache reuse above: for requests whose
 *                          contexts are private and larger than the last-level cache, read once per decode step.  In
 *                          the shared decode an item holds at most 16 / G users, so a chunk with more users is read
 *                          by several workgroups: there too the hint only pays for private contexts.  Other entry
 *                          points ignore it.
 * Any other value is LAZY_EINVAL.
 */
#define LAZY_CACHE_DEFAULT 0
#define LAZY_CACHE_STREAM 1

/*
 * Key-store conventions (params->key_positions).  Values and the causal rule are the same in both; only the
 * encoding of the stored keys differs.
 *  LAZY_KEYS_NOPE  (0): keys are stored without positional encoding.  Key j of a record is rotated inside the
 *                       kernels at pos_offset + j (prefill and decode rotate every key tile; the per-key angle is
 *                       built from one base row per 32 keys and a 32-row table of offsets).
 *  LAZY_KEYS_LOCAL (1): the paper's own convention (Sec. 3.2 "Prefilling": each document's cache keeps local
 *                       positions from 0 and is reused at offset Delta with one fixed rotation).  Key j is stored
 *                       already encoded at position j; using it at pos_offset + j needs the single rotation
 *                       R(pos_offset), the same for every key of the record.  Prefill rotates each key tile by that
 *                       one angle row; decode instead rotates the query by q_pos - pos_offset whenever the record
 *                       changes (Sec. 3.2 "Decoding") and reads the keys as stored.
 */
#define LAZY_KEYS_NOPE 0
#define LAZY_KEYS_LOCAL 1

/*
 * Prefill (Sec. 3.2 "Prefilling"; Fig. 3(b)): every request's new query tokens attend over all keys of its chunk
 * table, each key rotated inside the kernel at pos_offset + j, queries rotated at their own positions.
 *   q            [total_q][Hq][D] bf16, NoPE queries; rows of request r are q_start[r] .. q_start[r+1]-1
 *   q_start      [batch+1] int32 device, non-decreasing, q_start[0] = 0
 *   q_pos0       [batch] int32 device: token i of request r sits at position q_pos0[r] + i
 *   k_pool,v_pool bf16 device base pointers of the chunk store (may be the same pointer)
 *   chunks       device array of lazy_chunk_t, all requests back to back; request r owns
 *                chunks[chunk_start[r] .. chunk_start[r+1]-1].  The request's own new K/V (if it attends to
 *                itself) is simply one of its records, usually the last, at pos_offset = q_pos0[r].
 *   chunk_start  [batch+1] int32 device prefix sums
 *   max_q_len    upper bound of any request's query count (sizes the grid)
 *   max_kv_len   upper bound of any request's total key count (sizes the KV split)
 *   out          [total_q][Hq][D] bf16, fully overwritten
 *   lse          [total_q][Hq] fp32 natural-log sum-exp of the scaled scores, or NULL
 *   workspace    device scratch of at least lazy_attn_prefill_workspace_size(...) bytes (may be NULL if 0)
 */
LAZY_API int lazy_attn_prefill(const lazy_attn_params_t* params, const void* q, const int32_t* q_start,
                      const int32_t* q_pos0, const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                      const int32_t* chunk_start, int32_t batch, int32_t total_q, int32_t max_q_len,
                      int32_t max_kv_len, void* out, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream);

LAZY_API size_t lazy_attn_prefill_workspace_size(const lazy_attn_params_t* params, int32_t batch, int32_t total_q,
                                        int32_t max_q_len, int32_t max_kv_len);

/*
 * Decode (Sec. 3.2 "Decoding"; Fig. 3(c)): one new query token per request at q_pos[r] attends over its chunk
 * table; the token's own K/V must already be appended to one of the request's chunks.  KV is split across
 * workgroups (split-KV) and the partial softmax states are merged by lazy_attn_combine's kernel.
 *   q [batch][Hq][D] bf16, q_pos [batch] int32 device, out [batch][Hq][D] bf16, lse [batch][Hq] fp32 or NULL.
 *   Other arguments as for prefill.
 */
LAZY_API int lazy_attn_decode(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos, const void* k_pool,
                     const void* v_pool, const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
                     int32_t max_kv_len, void* out, float* lse, void* workspace, size_t workspace_bytes,
                     void* stream);

LAZY_API size_t lazy_attn_decode_workspace_size(const lazy_attn_params_t* params, int32_t batch, int32_t max_kv_len);

/*
 * Decode that allocates nothing and takes no workspace, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation).  Same arguments, kernels and results
 * as lazy_attn_decode; the split-KV partial results go to a fixed device array of LAZY_NOALLOC_SCRATCH_BYTES inside
 * the library instead of a caller workspace (each device the library runs on holds its own copy until the process
 * ends).
 *  - The first call on a device looks up that device's copy (hipGetSymbolAddress, which may make the HIP runtime
 *    load the library's code object on that device); later calls only launch.  The library itself calls no
 *    allocating routine.
 *  - `stream` (NULL = the null stream) must belong to the calling thread's current device: LAZY_EINVAL otherwise.
 *  - LAZY_EWORKSPACE if the launch needs more than LAZY_NOALLOC_SCRATCH_BYTES, i.e. if
 *    lazy_attn_decode_workspace_size(params, batch, max_kv_len) exceeds it; nothing is launched then.  Every launch
 *    with the library's own split count (params->num_splits = 0) fits: it needs less than
 *    1024 * min(G, 16) * (2 D + 4) bytes (4.3 MB at D = 128).
 *  - Every call on one device shares the array, which keeps the last call's contents.  Each launch writes every
 *    partial result it later reads, so nothing needs clearing between calls, but calls that overlap on one device
 *    (on different streams, or from different host threads without ordering) race on it and give wrong results.
 */
#define LAZY_NOALLOC_SCRATCH_BYTES (8 << 20)
LAZY_API int lazy_attn_decode_noalloc(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos,
                                      const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                                      const int32_t* chunk_start, int32_t batch, int32_t max_kv_len, void* out,
                                      float* lse, void* stream);

/*
 * Split-KV merge (standard log-sum-exp combination of partial softmax results over disjoint key sets): each split s
 * holds its own normalised output o[s][row] and the log-sum-exp lse[s][row] of its scaled scores (natural log);
 * with M = max_s lse[s][row] and w_s = exp(lse[s][row] - M):
 *     out[row] = sum_s w_s o[s][row][:] / sum_s w_s,   lse[row] = M + ln(sum_s w_s).
 *   part_o [splits][rows][D] bf16, part_lse [splits][rows] fp32 (-inf for a split that saw no key; its o is
 *   ignored).  out [rows][D] bf16; lse [rows] fp32 or NULL.  Rows whose every split is empty get out = 0,
 *   lse = -inf.  The prefill / decode workspaces hold exactly these two arrays (part_o first, then part_lse).
 */
LAZY_API int lazy_attn_combine(const void* part_o, const float* part_lse, int32_t splits, int32_t rows,
                               int32_t head_dim, void* out, float* lse, void* stream);

/*
 * Materialise-then-attend baseline, step 1 (the re-encoding copy that LazyAttention avoids; Block-Attention's
 * rotate-and-copy path described in the appendix "Experiments Details"): for every record i of every request,
 * write R(pos_offset + j) k_j into k_out, request after request, so that each request's rotated keys form one
 * contiguous region: record i's block [Hkv][len_i][D] starts at element sum_{i' < i} Hkv * len_{i'} * D.
 * chunks_out (device, same count) receives the records that describe the copy: k_offset into k_out,
 * k_stride = len, v_offset / v_stride / len / pos_offset unchanged (values are read in place).
 *   num_records = chunk_start[batch]; total_kv = sum of all len (k_out holds Hkv * total_kv * D elements).
 */
LAZY_API int lazy_materialize_k(const lazy_attn_params_t* params, const void* k_pool, const lazy_chunk_t* chunks,
                       int32_t num_records, int32_t max_chunk_len, int64_t total_kv, void* k_out,
                       lazy_chunk_t* chunks_out, void* stream);

/*
 * Materialise-then-attend baseline, step 2: ordinary attention over keys that already carry their positions
 * (k_pool / chunks as produced by lazy_materialize_k); queries are still rotated at their positions.  Same
 * arguments and workspace sizes as lazy_attn_prefill / lazy_attn_decode.
 */
LAZY_API int lazy_plain_attn_prefill(const lazy_attn_params_t* params, const void* q, const int32_t* q_start,
                            const int32_t* q_pos0, const void* k_pool, const void* v_pool,
                            const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch, int32_t total_q,
                            int32_t max_q_len, int32_t max_kv_len, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream);

LAZY_API int lazy_plain_attn_decode(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos,
                           const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                           const int32_t* chunk_start, int32_t batch, int32_t max_kv_len, void* out, float* lse,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * Chunk-major shared decode.  Position-free storage lets one stored chunk serve several requests of a batch at
 * different offsets (the problem statement at the start of Sec. 3).  In decode, where reading K/V dominates
 * (Sec. 3.2 "Decoding"), such a batch can read every shared chunk once per step for all of its users instead of
 * once per user.  A work item is a run of stored keys (one or more ranges of records, read back to back) together
 * with up to floor(16 / G) of its users (G = num_q_heads / num_kv_heads <= 16); its workgroups (one per KV head) read
 * the run once and score it against every (user, query head) pair.  Key j of the run (j counted from 0 over its
 * ranges) sits at position pos_offset_u + j in user u's request.  User u's query is rotated by the relative offset
 * q_pos[r_u] - pos_offset_u (the query-side rotation of Sec. 3.2 "Decoding") and keys are rotated by R(j) for a
 * NoPE store, since (R(q_pos) q).(R(pos_offset + j) k) = (R(q_pos - pos_offset) q).(R(j) k) (the relative-rotation
 * Fact of Sec. 3.2).  A local-position store holds keys already encoded at their index in the record, so its items
 * are single ranges, the keys are used as stored and the query is rotated by the record's own offset,
 * q_pos[r_u] - (pos_offset_u - key_begin).  The causal rule is applied per user (key j visible iff
 * pos_offset_u + j <= q_pos[r_u]).  Every (user, item) writes one partial result into its request's slot; the
 * request's slots are then merged as in lazy_attn_combine.
 */
typedef struct lazy_shared_range {
  int64_t k_offset;   /* a stored record, as in lazy_chunk_t */
  int64_t v_offset;
  int32_t k_stride;
  int32_t v_stride;
  int32_t key_begin;  /* this range is the record's keys key_begin .. key_end - 1 */
  int32_t key_end;
} lazy_shared_range_t; /* 32 bytes */

typedef struct lazy_shared_item {
  int32_t range_begin; /* its keys: ranges[range_begin .. range_begin + num_ranges - 1], back to back */
  int32_t num_ranges;  /* 1 .. LAZY_SHARED_MAX_RANGES */
  int32_t range_keys;  /* keys in every range but the last, a multiple of 32 when num_ranges > 1; the last range
                          has 1 .. range_keys keys */
  int32_t user_begin;  /* its users are users[user_begin .. user_begin + num_users - 1] */
  int32_t num_users;   /* 1 .. floor(16 / G) */
  int32_t reserved;    /* 0 */
} lazy_shared_item_t; /* 24 bytes */

#define LAZY_SHARED_MAX_RANGES 64

typedef struct lazy_shared_user {
  int32_t request;    /* the request: row block of q, q_pos and out */
  int32_t pos_offset; /* position of the item's first key in that request */
  int32_t slot;       /* partial-result slot within the request, 0 .. (slot_start[r+1] - slot_start[r]) - 1 */
  int32_t reserved;   /* 0 */
} lazy_shared_user_t; /* 16 bytes */

/*
 * Host planner (CPU only, on HOST copies of the decode tables).
 *  1. Groups the records that read the same stored keys (same k_offset, v_offset, k_stride, v_stride) and cuts
 *     each record into pieces of at most max_keys_per_item keys (0 = 1024); pieces with the same bounds share a
 *     group, whose users are the (request, piece) pairs.
 *  2. With a NoPE store (key_positions = LAZY_KEYS_NOPE, any rope_style), chains groups into runs: group B follows
 *     group A when both cover whole records, A holds a multiple of 32 keys, B at most as many, and every user of A
 *     continues, in its own table, with the next record in B at the next position (so a chunk held as a sequence of
 *     blocks, e.g. a paged store, is read as one run).  A run stops at max_keys_per_item keys or
 *     LAZY_SHARED_MAX_RANGES ranges.
 *  3. Every (request, run) gets one slot; runs become items of up to floor(16 / G) users, longest first.
 * Writes *num_items items, *num_ranges ranges, *num_users users and slot_start[batch+1] (prefix sums of the slots
 * per request).  Returns LAZY_EINVAL if a capacity is too small (the counts needed are still written),
 * LAZY_EUNSUPPORTED if G > 16, LAZY_EDATA for a negative length.
 */
LAZY_API int lazy_shared_decode_plan(const lazy_attn_params_t* params, const lazy_chunk_t* chunks,
                                     const int32_t* chunk_start, int32_t batch, int32_t max_keys_per_item,
                                     lazy_shared_item_t* items, int32_t item_capacity, lazy_shared_range_t* ranges,
                                     int32_t range_capacity, lazy_shared_user_t* users, int32_t user_capacity,
                                     int32_t* num_items, int32_t* num_ranges, int32_t* num_users,
                                     int32_t* slot_start);

/*
 * Chunk table in storage order (host only, on HOST copies): out receives the records of chunks with each request's
 * records stably sorted by k_offset (out may be chunks itself; otherwise the two must not overlap).  A request's
 * attention is set by its records' positions, not by their order in the table (Sec. 3.2: chunks at any offsets), so
 * a table in either order gives the same result up to the order of the floating-point sums.  Why a caller would want
 * it: the per-request kernels walk a request's keys in table order, and the decode's workgroups for one (split, KV
 * head) of all requests are placed on one XCD when splits x ceil(G / 16) x Hkv is a multiple of 8 (always with 8 KV
 * heads), all running at once when the grid fits the chip (two workgroups per CU); requests whose tables list the
 * chunks they share in the same order then read those chunks together, through one L2, instead of each from memory.  The chunk-major shared decode's planner wants tables in
 * position order instead (it chains the blocks a request reads back to back).  Returns LAZY_EINVAL for a bad
 * chunk_start (not starting at 0, decreasing) or missing arrays.
 */
LAZY_API int lazy_chunk_table_storage_order(const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
                                            lazy_chunk_t* out);

/*
 * Shared decode over a plan (all arrays in device memory): q [batch][Hq][D] bf16, q_pos [batch] int32, items /
 * ranges / users / slot_start as written by lazy_shared_decode_plan, max_slots >= the largest slot count of a
 * request.  out [batch][Hq][D] bf16 and lse [batch][Hq] (or NULL) as for lazy_attn_decode.  workspace: at least
 * lazy_attn_decode_shared_workspace_size(params, batch, max_slots) bytes, holding the partial results
 * [max_slots][batch * Hq] (bf16 outputs, then fp32 log-sum-exps).  Requests with no slot get out = 0, lse = -inf.
 */
LAZY_API int lazy_attn_decode_shared(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos,
                                     const void* k_pool, const void* v_pool, const lazy_shared_item_t* items,
                                     int32_t num_items, const lazy_shared_range_t* ranges,
                                     const lazy_shared_user_t* users, const int32_t* slot_start, int32_t batch,
                                     int32_t max_slots, void* out, float* lse, void* workspace,
                                     size_t workspace_bytes, void* stream);

LAZY_API size_t lazy_attn_decode_shared_workspace_size(const lazy_attn_params_t* params, int32_t batch,
                                                       int32_t max_slots);

/*
 * Position-agnostic chunk pool (host only).  A serving system keeps reusable chunks in a device KV region of
 * `capacity_slots` equal-size slots; this LRU directory maps a 64-bit id to its slot.  With position-free storage
 * the id is the document alone, so one slot serves every request at every offset (Sec. 2 "Hit-ratio impact under
 * limited cache capacity": a position-aware cache spends its capacity on positional variants; such a cache would
 * key by (document, position)).  The caller fills a slot on a miss and builds lazy_chunk_t records from slot
 * numbers.  Not thread-safe: one owner per pool.
 *   lazy_pool_create      NULL on a non-positive capacity or allocation failure.
 *   lazy_pool_acquire     *hit = 1 and the slot of `key` (now most recent), or *hit = 0 and a slot for it: a free
 *                         one, else the least recently used one, whose key is reported (*evicted = 1).
 *   lazy_pool_stats       counters since creation; any output may be NULL.
 */
typedef struct lazy_pool lazy_pool_t;
LAZY_API lazy_pool_t* lazy_pool_create(int32_t capacity_slots);
LAZY_API void lazy_pool_destroy(lazy_pool_t* pool);
LAZY_API int lazy_pool_acquire(lazy_pool_t* pool, uint64_t key, int32_t* slot, int32_t* hit, uint64_t* evicted_key,
                               int32_t* evicted);
LAZY_API int lazy_pool_stats(const lazy_pool_t* pool, int64_t* lookups, int64_t* hits, int64_t* evictions,
                             int32_t* resident);

/*
 * Host-side check of the table contents against the layout contract, on HOST copies of the tables (CPU only, no
 * device access).  k_pool_elems / v_pool_elems are the pool sizes in elements.  Returns LAZY_OK or LAZY_EDATA and
 * writes the offending record / request index and a reason to *bad_index / reason (either may be NULL).
 * q_start / q_pos0 may be NULL to skip query checks (decode passes q_start = NULL and q_pos as q_pos0).
 * Checks: prefix sums monotone and starting at 0; every record as required by lazy_chunk_t; K/V ranges inside
 * the pools; positions below LAZY_MAX_POS; with the causal rule, every query sees at least one key.
 */
LAZY_API int lazy_attn_validate(const lazy_attn_params_t* params, const int32_t* q_start, const int32_t* q_pos0,
                       const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch, int64_t k_pool_elems,
                       int64_t v_pool_elems, int64_t* bad_index, const char** reason);

/*
 * Host-side check of a shared-decode plan (HOST copies of what lazy_attn_decode_shared would read; CPU only).  The
 * kernel trusts these tables, so a plan built by hand rather than by lazy_shared_decode_plan should pass this first.
 * Checks: slot_start starts at 0, is non-decreasing and no request has more than max_slots slots; every range has
 * non-negative 16-byte-aligned offsets, 0 <= key_begin < key_end <= both strides and its K / V inside the pools
 * (pool sizes in elements); every item has 1..LAZY_SHARED_MAX_RANGES ranges inside the range table (exactly one
 * with LAZY_KEYS_LOCAL), all but the last of range_keys keys (a multiple of 32 when there are several), the last
 * 1..range_keys keys, 1..floor(16 / G) users inside the user table and reserved = 0; every user names a request of
 * the batch, one of its slots and key positions in 0..LAZY_MAX_POS; every slot of every request is written by
 * exactly one (item, user) pair.  q_pos (nullable) must lie in 0..LAZY_MAX_POS - 1.  Returns LAZY_OK, LAZY_EDATA
 * (with the offending item / range / request index in *bad_index and a reason), LAZY_EINVAL for bad arguments or
 * LAZY_EUNSUPPORTED for a head layout the shared decode does not take.
 */
LAZY_API int lazy_shared_decode_validate(const lazy_attn_params_t* params, const lazy_shared_item_t* items,
                                         int32_t num_items, const lazy_shared_range_t* ranges, int32_t num_ranges,
                                         const lazy_shared_user_t* users, int32_t num_users,
                                         const int32_t* slot_start, int32_t batch, int32_t max_slots,
                                         const int32_t* q_pos, int64_t k_pool_elems, int64_t v_pool_elems,
                                         int64_t* bad_index, const char** reason);

/* Static text for a LAZY_* code. */
LAZY_API const char* lazy_attn_strerror(int code);

/* Library version (major * 10000 + minor * 100 + patch). */
LAZY_API int lazy_attn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LAZY_ATTN_H */
