// C ABI of the LazyAttention hot path: argument checks, launch configuration and dispatch to the HIP kernels.
// The library never allocates device memory and never synchronises; every launch goes to the caller's stream.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>

#include "lazy_attn.h"
#include "lazy_attn_internal.h"

namespace {

constexpr int kNumCUs = 256;              // MI355X compute units

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int check_params(const lazy_attn_params_t* p) {
  if (!p) return LAZY_EINVAL;
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_q_heads % p->num_kv_heads != 0) return LAZY_EINVAL;
  if (p->causal != 0 && p->causal != 1) return LAZY_EINVAL;
  if (!isfinite(p->softmax_scale) || p->softmax_scale < 0.f) return LAZY_EINVAL;
  if (p->rope_style != LAZY_ALIBI && !p->inv_freq && !(isfinite(p->rope_base) && p->rope_base > 0.f)) return LAZY_EINVAL;
  if (p->num_splits < 0) return LAZY_EINVAL;
  if (p->key_positions != LAZY_KEYS_NOPE && p->key_positions != LAZY_KEYS_LOCAL) return LAZY_EINVAL;
  if (p->rope_style != LAZY_ROPE_HALF && p->rope_style != LAZY_ROPE_INTERLEAVED && p->rope_style != LAZY_ALIBI)
    return LAZY_EINVAL;
  if (p->rope_style == LAZY_ALIBI && p->key_positions != LAZY_KEYS_NOPE) return LAZY_EINVAL;
  if (p->q_prerotated != 0 && p->q_prerotated != 1) return LAZY_EINVAL;
  if (p->cache_hint != LAZY_CACHE_DEFAULT && p->cache_hint != LAZY_CACHE_STREAM) return LAZY_EINVAL;
  if (p->head_dim != 64 && p->head_dim != 128) return LAZY_EUNSUPPORTED;
  return LAZY_OK;
}

float scale_log2(const lazy_attn_params_t* p) {
  const float s = p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / sqrtf((float)p->head_dim);
  return s * 1.4426950408889634f;
}

// 256 packed rows per workgroup (eight waves, one workgroup per CU; head_dim 128 only) once a request has enough
// rows; otherwise 128 rows (four waves, two workgroups per CU).  Must match the kernel chosen in launch_prefill.
int prefill_row_blocks(const lazy_attn_params_t* p, int32_t max_q_len) {
  const int64_t g = p->num_q_heads / p->num_kv_heads;
  return p->head_dim == 128 && (int64_t)max_q_len * g >= 2 * lazy::kPrefillRowsPerBlock ? 2 : 1;
}

int prefill_q_tiles(const lazy_attn_params_t* p, int32_t max_q_len) {
  const int64_t g = p->num_q_heads / p->num_kv_heads;
  return (int)ceil_div((int64_t)max_q_len * g, (int64_t)lazy::kPrefillRowsPerBlock * prefill_row_blocks(p, max_q_len));
}

// A batch is ragged when its mean query length is below 3/4 of the maximum.
bool prefill_ragged(int32_t batch, int32_t total_q, int32_t max_q_len) {
  return 4 * (int64_t)total_q < 3 * (int64_t)batch * max_q_len;
}

// KV splits per request.  Workgroups are (query tile, KV head, request, split); those of a query tile past the end
// of a shorter request exit at once, so the busy ones number about Hkv * ceil(total_q G / rows per tile) per split.
// Equal requests: one round of workgroups over the chip.  Ragged query lengths (mean below 3/4 of the maximum)
// usually come with ragged key lengths, and one round then leaves CUs idle behind the longest requests: aim for
// about three rounds so that the dispatcher can even out the load.
int prefill_splits(const lazy_attn_params_t* p, int32_t batch, int32_t total_q, int32_t max_q_len,
                   int32_t max_kv_len) {
  if (p->num_splits > 0) return p->num_splits;
  const int64_t g = p->num_q_heads / p->num_kv_heads;
  const int64_t rows_per_tile = (int64_t)lazy::kPrefillRowsPerBlock * prefill_row_blocks(p, max_q_len);
  const int64_t busy = (int64_t)p->num_kv_heads * ceil_div((int64_t)total_q * g, rows_per_tile);
  const int64_t tiles = ceil_div(max_kv_len, lazy::kPrefillTileKeys);
  // 256-row workgroups occupy a whole CU (LDS), 128-row ones leave room for two per CU.
  const int64_t slots = prefill_row_blocks(p, max_q_len) == 2 ? kNumCUs : 2 * kNumCUs;
  const int64_t target = prefill_ragged(batch, total_q, max_q_len) ? 3 * slots : slots;
  int64_t s = busy > 0 ? ceil_div(target, busy) : 1;
  const int64_t cap = tiles / 4 > 1 ? tiles / 4 : 1;  // keep at least ~4 key tiles per split
  if (s > cap) s = cap;
  if (s > 64) s = 64;
  return s < 1 ? 1 : (int)s;
}

int decode_head_groups(const lazy_attn_params_t* p) {
  const int g = p->num_q_heads / p->num_kv_heads;
  return (g + lazy::kDecodeHeadsPerGroup - 1) / lazy::kDecodeHeadsPerGroup;
}

int decode_splits(const lazy_attn_params_t* p, int32_t batch, int32_t max_kv_len) {
  if (p->num_splits > 0) return p->num_splits;
  // Two streaming workgroups per CU; split only when the batch alone cannot fill the chip.
  const int64_t base = (int64_t)batch * p->num_kv_heads * decode_head_groups(p);
  const int64_t tiles = ceil_div(max_kv_len, lazy::kDecodeTileKeys);
  int64_t s = base > 0 ? ceil_div(2 * kNumCUs, base) : 1;
  const int64_t cap = tiles / 2 > 1 ? tiles / 2 : 1;
  if (s > cap) s = cap;
  if (s > 64) s = 64;
  return s < 1 ? 1 : (int)s;
}

// Split-KV workspace: bf16 normalised partial outputs [splits][rows][d], then fp32 partial lse [splits][rows]
// (16-byte aligned because d is a multiple of 8).
size_t split_workspace(int splits, int64_t rows, int d) {
  if (splits <= 1) return 0;
  return (size_t)splits * (size_t)rows * ((size_t)d * sizeof(uint16_t) + sizeof(float));
}

int status(hipError_t e) { return e == hipSuccess ? LAZY_OK : LAZY_EHIP; }

int run_prefill(bool rotate_k, const lazy_attn_params_t* p, const void* q, const int32_t* q_start,
                const int32_t* q_pos0, const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                const int32_t* chunk_start, int32_t batch, int32_t total_q, int32_t max_q_len, int32_t max_kv_len,
                void* out, float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  int e = check_params(p);
  if (e != LAZY_OK) return e;
  if (!rotate_k && p->rope_style == LAZY_ALIBI) return LAZY_EUNSUPPORTED;  // no materialised copy for ALiBi
  if (batch < 0 || total_q < 0 || max_q_len < 0 || max_kv_len < 0) return LAZY_EINVAL;
  if (batch == 0 || total_q == 0) return LAZY_OK;
  if (max_q_len == 0) return LAZY_EINVAL;
  if (!q || !q_start || !q_pos0 || !k_pool || !v_pool || !chunks || !chunk_start || !out) return LAZY_EINVAL;
  const int splits = prefill_splits(p, batch, total_q, max_q_len, max_kv_len);
  const int q_tiles = prefill_q_tiles(p, max_q_len);
  if ((int64_t)batch * splits > 65535 || p->num_kv_heads > 65535) return LAZY_EUNSUPPORTED;
  const int64_t rows = (int64_t)total_q * p->num_q_heads;
  const size_t need = split_workspace(splits, rows, p->head_dim);
  if (need > 0 && (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 15u))) return LAZY_EWORKSPACE;

  lazy::AttnArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.q_start = q_start;
  a.q_pos0 = q_pos0;
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.chunks = chunks;
  a.chunk_start = chunk_start;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.ws_o = need ? static_cast<uint16_t*>(workspace) : nullptr;
  a.ws_lse = need ? reinterpret_cast<float*>(static_cast<uint16_t*>(workspace) + (size_t)splits * rows * p->head_dim)
                  : nullptr;
  a.inv_freq = p->inv_freq;
  a.batch = batch;
  a.total_q = total_q;
  a.hq = p->num_q_heads;
  a.hkv = p->num_kv_heads;
  a.group = p->num_q_heads / p->num_kv_heads;
  a.causal = p->causal;
  a.splits = splits;
  a.q_tiles = q_tiles;
  a.row_blocks = prefill_row_blocks(p, max_q_len);
  // Ragged batches spread their (request, split) units over the XCDs; alike requests keep whole requests per XCD.
  a.xcd_interleave = prefill_ragged(batch, total_q, max_q_len);
  a.head_groups = 1;
  a.rope_log2_base = p->inv_freq || p->rope_style == LAZY_ALIBI ? 0.0 : log2((double)p->rope_base);
  a.scale_log2 = scale_log2(p);
  a.local_keys = p->key_positions == LAZY_KEYS_LOCAL;
  a.interleaved = p->rope_style == LAZY_ROPE_INTERLEAVED;
  a.alibi = p->rope_style == LAZY_ALIBI;
  a.q_prerot = p->q_prerotated && p->rope_style != LAZY_ALIBI;
  return status(lazy::launch_prefill(a, p->head_dim, rotate_k, static_cast<hipStream_t>(stream)));
}

int run_decode(bool rotate_k, const lazy_attn_params_t* p, const void* q, const int32_t* q_pos, const void* k_pool,
               const void* v_pool, const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
               int32_t max_kv_len, void* out, float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  int e = check_params(p);
  if (e != LAZY_OK) return e;
  if (!rotate_k && p->rope_style == LAZY_ALIBI) return LAZY_EUNSUPPORTED;
  if (batch < 0 || max_kv_len < 0) return LAZY_EINVAL;
  if (batch == 0) return LAZY_OK;
  if (!q || !q_pos || !k_pool || !v_pool || !chunks || !chunk_start || !out) return LAZY_EINVAL;
  const int splits = decode_splits(p, batch, max_kv_len);
  const int hg = decode_head_groups(p);
  if (batch > 65535 || (int64_t)p->num_kv_heads * hg > 65535) return LAZY_EUNSUPPORTED;
  const int64_t rows = (int64_t)batch * p->num_q_heads;
  const size_t need = split_workspace(splits, rows, p->head_dim);
  if (need > 0 && (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 15u))) return LAZY_EWORKSPACE;

  lazy::AttnArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.q_start = nullptr;
  a.q_pos0 = q_pos;
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.chunks = chunks;
  a.chunk_start = chunk_start;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.ws_o = need ? static_cast<uint16_t*>(workspace) : nullptr;
  a.ws_lse = need ? reinterpret_cast<float*>(static_cast<uint16_t*>(workspace) + (size_t)splits * rows * p->head_dim)
                  : nullptr;
  a.inv_freq = p->inv_freq;
  a.batch = batch;
  a.total_q = batch;
  a.hq = p->num_q_heads;
  a.hkv = p->num_kv_heads;
  a.group = p->num_q_heads / p->num_kv_heads;
  a.causal = p->causal;
  a.splits = splits;
  a.q_tiles = 1;
  a.row_blocks = 1;
  a.head_groups = hg;
  a.rope_log2_base = p->inv_freq || p->rope_style == LAZY_ALIBI ? 0.0 : log2((double)p->rope_base);
  a.scale_log2 = scale_log2(p);
  a.local_keys = p->key_positions == LAZY_KEYS_LOCAL;
  a.interleaved = p->rope_style == LAZY_ROPE_INTERLEAVED;
  a.alibi = p->rope_style == LAZY_ALIBI;
  a.q_prerot = p->q_prerotated && p->rope_style != LAZY_ALIBI;
  a.stream_kv = p->cache_hint == LAZY_CACHE_STREAM;
  return status(lazy::launch_decode(a, p->head_dim, rotate_k, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

size_t lazy_attn_prefill_workspace_size(const lazy_attn_params_t* params, int32_t batch, int32_t total_q,
                                        int32_t max_q_len, int32_t max_kv_len) {
  if (check_params(params) != LAZY_OK || batch <= 0 || total_q <= 0 || max_q_len <= 0 || max_kv_len < 0) return 0;
  const int splits = prefill_splits(params, batch, total_q, max_q_len, max_kv_len);
  return split_workspace(splits, (int64_t)total_q * params->num_q_heads, params->head_dim);
}

size_t lazy_attn_decode_workspace_size(const lazy_attn_params_t* params, int32_t batch, int32_t max_kv_len) {
  if (check_params(params) != LAZY_OK || batch <= 0 || max_kv_len < 0) return 0;
  const int splits = decode_splits(params, batch, max_kv_len);
  return split_workspace(splits, (int64_t)batch * params->num_q_heads, params->head_dim);
}

int lazy_attn_prefill(const lazy_attn_params_t* params, const void* q, const int32_t* q_start,
                      const int32_t* q_pos0, const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                      const int32_t* chunk_start, int32_t batch, int32_t total_q, int32_t max_q_len,
                      int32_t max_kv_len, void* out, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream) {
  return run_prefill(true, params, q, q_start, q_pos0, k_pool, v_pool, chunks, chunk_start, batch, total_q,
                     max_q_len, max_kv_len, out, lse, workspace, workspace_bytes, stream);
}

int lazy_plain_attn_prefill(const lazy_attn_params_t* params, const void* q, const int32_t* q_start,
                            const int32_t* q_pos0, const void* k_pool, const void* v_pool,
                            const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch, int32_t total_q,
                            int32_t max_q_len, int32_t max_kv_len, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return run_prefill(false, params, q, q_start, q_pos0, k_pool, v_pool, chunks, chunk_start, batch, total_q,
                     max_q_len, max_kv_len, out, lse, workspace, workspace_bytes, stream);
}

int lazy_attn_decode(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos, const void* k_pool,
                     const void* v_pool, const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
                     int32_t max_kv_len, void* out, float* lse, void* workspace, size_t workspace_bytes,
                     void* stream) {
  return run_decode(true, params, q, q_pos, k_pool, v_pool, chunks, chunk_start, batch, max_kv_len, out, lse,
                    workspace, workspace_bytes, stream);
}

int lazy_plain_attn_decode(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos,
                           const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                           const int32_t* chunk_start, int32_t batch, int32_t max_kv_len, void* out, float* lse,
                           void* workspace, size_t workspace_bytes, void* stream) {
  return run_decode(false, params, q, q_pos, k_pool, v_pool, chunks, chunk_start, batch, max_kv_len, out, lse,
                    workspace, workspace_bytes, stream);
}

int lazy_attn_decode_noalloc(const lazy_attn_params_t* params, const void* q, const int32_t* q_pos,
                             const void* k_pool, const void* v_pool, const lazy_chunk_t* chunks,
                             const int32_t* chunk_start, int32_t batch, int32_t max_kv_len, void* out, float* lse,
                             void* stream) {
  const int e = check_params(params);
  if (e != LAZY_OK) return e;
  if (batch < 0 || max_kv_len < 0) return LAZY_EINVAL;
  if (batch == 0) return LAZY_OK;
  const size_t need = lazy_attn_decode_workspace_size(params, batch, max_kv_len);
  if (need > (size_t)LAZY_NOALLOC_SCRATCH_BYTES) return LAZY_EWORKSPACE;
  int device = -1;
  if (hipGetDevice(&device) != hipSuccess) return LAZY_EHIP;
  if (stream) {
    hipDevice_t sd = -1;
    if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sd) != hipSuccess) return LAZY_EHIP;
    if (sd != device) return LAZY_EINVAL;
  }
  void* ws = nullptr;
  if (lazy::noalloc_scratch(device, &ws) != hipSuccess) return LAZY_EHIP;
  return run_decode(true, params, q, q_pos, k_pool, v_pool, chunks, chunk_start, batch, max_kv_len, out, lse, ws,
                    (size_t)LAZY_NOALLOC_SCRATCH_BYTES, stream);
}

int lazy_attn_combine(const void* part_o, const float* part_lse, int32_t splits, int32_t rows, int32_t head_dim,
                      void* out, float* lse, void* stream) {
  if (head_dim != 64 && head_dim != 128) return LAZY_EUNSUPPORTED;
  if (splits <= 0 || rows < 0) return LAZY_EINVAL;
  if (rows == 0) return LAZY_OK;
  if (!part_o || !part_lse || !out || ((uintptr_t)part_o & 15u)) return LAZY_EINVAL;
  return status(lazy::launch_combine(static_cast<const uint16_t*>(part_o), part_lse, splits, rows, head_dim,
                                     static_cast<uint16_t*>(out), lse, static_cast<hipStream_t>(stream)));
}

int lazy_materialize_k(const lazy_attn_params_t* params, const void* k_pool, const lazy_chunk_t* chunks,
                       int32_t num_records, int32_t max_chunk_len, int64_t total_kv, void* k_out,
                       lazy_chunk_t* chunks_out, void* stream) {
  int e = check_params(params);
  if (e != LAZY_OK) return e;
  if (params->rope_style == LAZY_ALIBI) return LAZY_EUNSUPPORTED;
  if (num_records < 0 || max_chunk_len < 0 || total_kv < 0) return LAZY_EINVAL;
  if (num_records == 0) return LAZY_OK;
  if (!k_pool || !chunks || !chunks_out || (total_kv > 0 && !k_out)) return LAZY_EINVAL;
  if (num_records > 65535 || params->num_kv_heads > 65535) return LAZY_EUNSUPPORTED;
  return status(lazy::launch_materialize(static_cast<const uint16_t*>(k_pool), chunks, num_records, max_chunk_len,
                                         params->num_kv_heads, params->head_dim,
                                         params->inv_freq ? 0.0 : log2((double)params->rope_base),
                                         params->inv_freq, params->key_positions == LAZY_KEYS_LOCAL,
                                         params->rope_style == LAZY_ROPE_INTERLEAVED,
                                         static_cast<uint16_t*>(k_out), chunks_out,
                                         static_cast<hipStream_t>(stream)));
}

size_t lazy_attn_decode_shared_workspace_size(const lazy_attn_params_t* params, int32_t batch, int32_t max_slots) {
  if (check_params(params) != LAZY_OK || batch <= 0 || max_slots <= 0) return 0;
  return (size_t)max_slots * (size_t)batch * params->num_q_heads *
         ((size_t)params->head_dim * sizeof(uint16_t) + sizeof(float));
}

int lazy_attn_decode_shared(const lazy_attn_params_t* p, const void* q, const int32_t* q_pos, const void* k_pool,
                            const void* v_pool, const lazy_shared_item_t* items, int32_t num_items,
                            const lazy_shared_range_t* ranges, const lazy_shared_user_t* users,
                            const int32_t* slot_start, int32_t batch, int32_t max_slots, void* out, float* lse,
                            void* workspace, size_t workspace_bytes, void* stream) {
  int e = check_params(p);
  if (e != LAZY_OK) return e;
  if (p->num_q_heads / p->num_kv_heads > 16) return LAZY_EUNSUPPORTED;
  if (batch < 0 || num_items < 0 || max_slots < 0 || (num_items > 0 && max_slots == 0)) return LAZY_EINVAL;
  if (batch == 0) return LAZY_OK;
  if (!q || !q_pos || !k_pool || !v_pool || !slot_start || !out || (num_items > 0 && (!items || !ranges || !users)))
    return LAZY_EINVAL;
  if (p->num_kv_heads > 65535) return LAZY_EUNSUPPORTED;
  const size_t need = lazy_attn_decode_shared_workspace_size(p, batch, max_slots);
  if (need > 0 && (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 15u))) return LAZY_EWORKSPACE;
  lazy::SharedArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.q_pos = q_pos;
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.items = items;
  a.ranges = ranges;
  a.users = users;
  const int64_t rows = (int64_t)batch * p->num_q_heads;
  a.ws_o = need ? static_cast<uint16_t*>(workspace) : nullptr;
  a.ws_lse = need ? reinterpret_cast<float*>(static_cast<uint16_t*>(workspace) + (size_t)max_slots * rows * p->head_dim)
                  : nullptr;
  a.inv_freq = p->inv_freq;
  a.batch = batch;
  a.hq = p->num_q_heads;
  a.hkv = p->num_kv_heads;
  a.group = p->num_q_heads / p->num_kv_heads;
  a.causal = p->causal;
  a.local_keys = p->key_positions == LAZY_KEYS_LOCAL;
  a.interleaved = p->rope_style == LAZY_ROPE_INTERLEAVED;
  a.alibi = p->rope_style == LAZY_ALIBI;
  a.q_prerot = p->q_prerotated && p->rope_style != LAZY_ALIBI;
  a.stream_kv = p->cache_hint == LAZY_CACHE_STREAM;
  a.rope_log2_base = p->inv_freq || p->rope_style == LAZY_ALIBI ? 0.0 : log2((double)p->rope_base);
  a.scale_log2 = scale_log2(p);
  return status(lazy::launch_decode_shared(a, num_items, max_slots, slot_start, p->head_dim,
                                           static_cast<uint16_t*>(out), lse, static_cast<hipStream_t>(stream)));
}

const char* lazy_attn_strerror(int code) {
  switch (code) {
    case LAZY_OK: return "success";
    case LAZY_EINVAL: return "invalid argument";
    case LAZY_EUNSUPPORTED: return "unsupported configuration";
    case LAZY_EWORKSPACE: return "workspace missing, too small or misaligned";
    case LAZY_EHIP: return "HIP runtime error at launch";
    case LAZY_EDATA: return "chunk or query table violates the layout contract";
    default: return "unknown error";
  }
}

int lazy_attn_version(void) { return 100; }

}  // extern "C"
