// Internal interface between the C ABI (lazy_attn_api.cpp) and the HIP kernels (lazy_attn_kernels.hip).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "lazy_attn.h"

namespace lazy {

// Everything one attention launch needs.  Pointers are device pointers.
struct AttnArgs {
  const uint16_t* q;          // [total_q][hq][D] bf16 bits
  const int32_t* q_start;     // [batch+1]
  const int32_t* q_pos0;      // [batch]
  const uint16_t* k_pool;     // bf16 bits
  const uint16_t* v_pool;
  const lazy_chunk_t* chunks;
  const int32_t* chunk_start; // [batch+1]
  uint16_t* out;              // [total_q][hq][D] bf16 bits
  float* lse;                 // [total_q][hq] or null
  uint16_t* ws_o;             // [splits][total_q*hq][D] bf16 normalised partial outputs, null when splits == 1
  float* ws_lse;              // [splits][total_q*hq] fp32 partial log-sum-exp, null when splits == 1
  const float* inv_freq;      // [D/2] or null
  int32_t batch;
  int32_t total_q;
  int32_t hq;
  int32_t hkv;
  int32_t group;              // hq / hkv
  int32_t causal;
  int32_t splits;
  int32_t q_tiles;            // prefill: row tiles per (request, kv head)
  int32_t row_blocks;         // prefill: a workgroup covers 128 * row_blocks packed rows (2 = eight-wave kernel)
  int32_t xcd_interleave;     // prefill: 1 spreads (request, split) units over the XCDs (ragged batches)
  int32_t head_groups;        // decode: ceil(group / 16)
  int32_t local_keys;         // 1: the store holds keys encoded at local positions (LAZY_KEYS_LOCAL)
  int32_t interleaved;        // 1: RoPE pairs (2t, 2t+1) (LAZY_ROPE_INTERLEAVED)
  int32_t alibi;              // 1: no rotation, ALiBi bias (LAZY_ALIBI); inv_freq then holds optional slopes
  int32_t q_prerot;           // 1: q arrives rotated at its own positions (rotations use -pos_offset / none)
  int32_t stream_kv;          // decode: 1 reads K / V with non-temporal loads (LAZY_CACHE_STREAM)
  double rope_log2_base;      // log2(rope_base), computed on the host (unused with inv_freq)
  float scale_log2;           // softmax scale * log2(e)
};

// Arguments of the chunk-major shared decode kernel.
struct SharedArgs {
  const uint16_t* q;                 // [batch][hq][D]
  const int32_t* q_pos;              // [batch]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const lazy_shared_item_t* items;   // [num_items]
  const lazy_shared_range_t* ranges; // key ranges of the items' runs
  const lazy_shared_user_t* users;
  uint16_t* ws_o;                    // [max_slots][batch*hq][D] bf16 partial outputs
  float* ws_lse;                     // [max_slots][batch*hq]
  const float* inv_freq;             // [D/2] or null
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t causal;
  int32_t local_keys;
  int32_t interleaved;
  int32_t alibi;
  int32_t q_prerot;
  int32_t stream_kv;                 // 1 reads K / V with non-temporal loads (LAZY_CACHE_STREAM)
  double rope_log2_base;
  float scale_log2;
};

// Packed rows (token, head in group) handled by one prefill workgroup, and keys per decode tile.
constexpr int kPrefillRowsPerBlock = 128;  // packed rows of a prefill workgroup per row block
constexpr int kPrefillTileKeys = 64;
constexpr int kDecodeTileKeys = 128;  // keys a decode workgroup consumes per step (4 waves x 32)
constexpr int kDecodeHeadsPerGroup = 16;

hipError_t launch_prefill(const AttnArgs& a, int head_dim, bool rotate_k, hipStream_t stream);
hipError_t launch_decode(const AttnArgs& a, int head_dim, bool rotate_k, hipStream_t stream);
hipError_t launch_decode_shared(const SharedArgs& a, int num_items, int max_slots, const int32_t* slot_start,
                                int head_dim, uint16_t* out, float* lse, hipStream_t stream);
// Device address of the fixed scratch array of lazy_attn_decode_noalloc on `device`, which must be the calling
// thread's current device; looked up once per device and cached.
hipError_t noalloc_scratch(int device, void** ptr);
hipError_t launch_combine(const uint16_t* part_o, const float* part_lse, int splits, int rows, int head_dim,
                          uint16_t* out, float* lse, hipStream_t stream);
hipError_t launch_materialize(const uint16_t* k_pool, const lazy_chunk_t* chunks, int num_records,
                              int max_chunk_len, int hkv, int head_dim, double rope_log2_base, const float* inv_freq,
                              bool local_keys, bool interleaved,
                              uint16_t* k_out, lazy_chunk_t* chunks_out, hipStream_t stream);

}  // namespace lazy
