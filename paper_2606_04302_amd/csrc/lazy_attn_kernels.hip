// HIP kernels of the LazyAttention hot path for gfx950 (MI355X / CDNA4).
//
// The chunk store holds K and V without positional encoding (Sec. 3.1 "Deferred encoding").  Every kernel that
// reads K rotates it on the way from HBM into LDS, at position pos_offset + j of the chunk in the current request
// (Sec. 3.2 "Prefilling": one rotation of the two half-dimensions per key, never "back to zero then forward").
// Variants selected per kernel instance: keys stored at local positions (one rotation by the record offset in
// prefill, the query rotated per record in decode), interleaved pairs (2t, 2t+1), and ALiBi (no rotation, a bias
// on every score); see the key-mode constants below.
//
// Data path of one key tile (64 keys per sub-tile, shared by the waves of a workgroup):
//   global K rows (bf16, natural layout) --16 B loads--> registers --fp32 rotation--> bf16 --> LDS K tile
//   global V rows --16 B loads--> registers --> LDS V tile (row-major), read back transposed by ds_read_b64_tr_b16
// The rotation is done once per workgroup and tile (not once per wave), which matters on gfx950 where the bf16
// MFMA rate is 16x the fp32 VALU rate: the relative cost of rotating K is 3/(4M) in FLOPs (eq. prefilling) but
// paid at VALU speed.
//
// Rotation angles are stateless (Appendix "Long-Context Scalability and Numerical Stability": absolute indices,
// no recurrence).  theta_t is held in revolutions per position in fp64; for a tile whose row 0 sits at position b
// the workgroup computes cos/sin(b theta_t) once per t (per 32-row half), and each loader thread keeps
// cos/sin(delta theta_t) for its fixed row delta (from a 32-row LDS table written once per workgroup, held in
// registers by the eight-wave kernel); the angle of row b + delta follows by one angle addition.
//
// Operand layouts (verified for v_mfma_f32_32x32x16_bf16 and v_mfma_f32_16x16x32_bf16):
//   32x32x16: A[i][k] in lane i%32 ... k = 8*(lane/32)+e; B[k][j] in lane j%32, k = 8*(lane/32)+e;
//             C[8*(r/4) + 4*(lane/32) + r%4][lane%32] in register r.
//   16x16x32: A[i][k] lane i%16, k = 8*(lane/16)+e; B[k][j] lane j%16, same k; C[4*(lane/16)+r][lane%16].
// Both attention products are computed transposed (S^T = K Q^T and O^T = V^T P^T) so that every lane owns whole
// query rows (prefill) or query heads (decode): softmax statistics and the O rescale stay inside a lane.
// The head dimension inside the K tile and in the Q fragments is stored in a permuted "virtual" order that puts
// each rotation pair (t, t + D/2) into the same 16-byte group: for pair t, the low half goes to virtual column
// 16*(t/8) + 8*((t%8)/4) + t%4 and the high half four columns later.  Any permutation applied to both Q and K
// leaves Q K^T unchanged.  V fragments are gathered with transposing LDS reads whose rows follow the key order
// in which P leaves the S^T accumulators, so P needs no shuffling.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "lazy_attn_internal.h"

namespace lazy {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kSub = 64;  // keys of one loader sub-tile; tile row 0 of a sub-tile is a multiple of 64 in its chunk
constexpr int kPad = 8;   // bf16 elements of padding per LDS row
constexpr float kLn2 = 0.69314718055994530942f;
// The softmax reference max only moves when a tile's max exceeds it by more than this (log2 units): unnormalised
// probabilities stay below 2^8, far inside fp32 and bf16 range, and the O accumulator is rescaled rarely.
constexpr float kRescaleSlack = 8.0f;
constexpr float kRescaleBound = 256.0f;  // 2^kRescaleSlack
constexpr double kInvTwoPi = 0.15915494309189533577;

static_assert(kPrefillTileKeys == kSub, "prefill tiles are one loader sub-tile");

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// A value that is the same in every lane of the wave, marked as such.  The compiler cannot prove it for values
// derived from threadIdx (the wave index) or computed with the vector integer-division expansion; without the mark
// the chunk-table walk that depends on them runs as divergent vector code, its record loads become vector loads,
// and their waits drain the vector-memory queue that holds the next tile's prefetched K / V.
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Inclusive prefix sum over the 64 lanes of a wave (all lanes active), with DPP lane moves instead of LDS
// permutes: shifts by 1, 2, 4, 8 within each 16-lane row (lanes shifted in from outside the row read 0), then the
// last lane of row 0 is added to row 1 and that of row 2 to row 3 (row_bcast:15), then the last lane of row 1
// (the total of rows 0-1) to rows 2 and 3 (row_bcast:31).  Rows left out by the row mask keep their value.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2 and 3
  return x;
}
// Reductions over lane pairs (l, l ^ 32) with v_permlane32_swap (one VALU op, no LDS round trip).  Swapping a
// register with itself yields x[l % 32] in one result and x[l % 32 + 32] in the other, in every lane, so both
// lanes of a pair combine the same two values in the same order.
__device__ __forceinline__ float xor32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// acc + (lo + hi) of a packed bf16 pair (v_dot2c_f32_bf16 with weights 1): the softmax denominator is summed over
// the same bf16-rounded probabilities that enter the P V product.
__device__ __forceinline__ float add_pair(uint32_t pair, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), bf16x2{(__bf16)1.0f, (__bf16)1.0f}, acc,
                                         false);
}

// theta_t / (2 pi): RoPE frequency of pair t in revolutions per position (original RoPE: base^(-2t/D), evaluated as
// exp2(-(2t/D) log2(base)) with log2(base) from the host, far cheaper than a double pow; RoPE variants pass their own
// table, Sec. 3.5).
__device__ __forceinline__ double theta_rev(int t, int d, double log2_base, const float* inv_freq) {
  const double th = inv_freq ? (double)inv_freq[t] : exp2(-2.0 * (double)t / (double)d * log2_base);
  return th * kInvTwoPi;
}

// (cos, sin) of the angle p * theta for theta given in revolutions: the product and its fractional part in fp64
// (exact range reduction for any position below 2^24), then the hardware sine and cosine, which take the angle in
// revolutions (v_sin_f32 / v_cos_f32; on [0, 1) within 1.3e-7 of the exact values, measured on an MI355X against
// fp64, about twice the error of a libm-style sincospi at a tenth of the instructions).
__device__ __forceinline__ float2 rope_cs(int p, double rev) {
  const float r = (float)__builtin_amdgcn_fract((double)p * rev);
  return make_float2(__builtin_amdgcn_cosf(r), __builtin_amdgcn_sinf(r));
}

// Rotate one pair (x1, x2) = (k[t], k[t + D/2]) by the angle base + delta, given (cos, sin) of each part.
// Written with explicit fmaf so that every kernel that rotates keys rounds identically.
__device__ __forceinline__ void rotate_pair(float x1, float x2, float2 cb, float2 cd, float& y1, float& y2) {
  const float c = fmaf(cb.x, cd.x, -(cb.y * cd.y));
  const float s = fmaf(cb.y, cd.x, cb.x * cd.y);
  y1 = fmaf(x1, c, -(x2 * s));
  y2 = fmaf(x1, s, x2 * c);
}

// Rotate one pair by a single angle given its (cos, sin): the one rotation of a local-position key by its record's
// offset.  Same fmaf form in every kernel that uses it.
__device__ __forceinline__ void rotate_by(float x1, float x2, float2 cs, float& y1, float& y2) {
  y1 = fmaf(x1, cs.x, -(x2 * cs.y));
  y2 = fmaf(x1, cs.y, x2 * cs.x);
}

// Key handling of a kernel instance: keys already encoded at their positions (the plain kernels of the
// materialise-then-attend baseline), NoPE keys rotated at pos_offset + j, or local-position keys (stored encoded at
// j) rotated by the record's pos_offset.
constexpr int kKeysPlain = 0, kKeysNope = 1, kKeysLocal = 2;
// Score-space positions (ALiBi): keys and queries are used as stored and slope_h (k_pos - q_pos) is added to every
// scaled score (Sec. 3.5 "Score-space positional methods").
constexpr int kKeysAlibi = 3;

// ALiBi slope of query head h: table[h], or 2^(-8 (h+1) / Hq); returned divided by the softmax scale (times
// log2 e over scale_log2), so that adding slope' (k_pos - q_pos) to the raw dot product adds the bias to the scaled
// score.
__device__ __forceinline__ float alibi_slope(int h, int hq, const float* table, float scale_log2) {
  const float sl = table ? table[h] : exp2f(-8.0f * (float)(h + 1) / (float)hq);
  return sl * 1.4426950408889634f / scale_log2;
}
// Bit 2 of a kernel's key-mode argument selects the interleaved pairing (pairs (2t, 2t+1)).  Interleaved RoPE on
// (q, k) is the half-split rotation of (P q, P k) for the permutation P: 2t -> t, 2t+1 -> t + D/2 (V unchanged), so
// the kernels only change their Q and K loads: 16 consecutive elements are split into the pairs' first and second
// halves, the layout a half-split load produces, and everything after the load is shared.
constexpr int kInterleaved = 4;
constexpr int keys_of(int km) { return km & 3; }
constexpr bool interleaved_of(int km) { return (km & kInterleaved) != 0; }
// Bit 3 of a decode kernel's key-mode argument: K and V are read with non-temporal loads (LAZY_CACHE_STREAM).
constexpr int kStreamKV = 8;
constexpr bool stream_of(int km) { return (km & kStreamKV) != 0; }

// 16 bf16 = pairs t0..t0+7 of an interleaved vector (w0: pairs t0..t0+3, one pair per 32-bit word, first element
// in the low half; w1: pairs t0+4..t0+7) -> the first elements (lo) and second elements (hi) in pair order.
__device__ __forceinline__ void deinterleave8(u32x4 w0, u32x4 w1, u32x4& lo, u32x4& hi) {
  lo = u32x4{(w0[0] & 0xffffu) | (w0[1] << 16), (w0[2] & 0xffffu) | (w0[3] << 16), (w1[0] & 0xffffu) | (w1[1] << 16),
             (w1[2] & 0xffffu) | (w1[3] << 16)};
  hi = u32x4{(w0[0] >> 16) | (w0[1] & 0xffff0000u), (w0[2] >> 16) | (w0[3] & 0xffff0000u),
             (w1[0] >> 16) | (w1[1] & 0xffff0000u), (w1[2] >> 16) | (w1[3] & 0xffff0000u)};
}
// Four pairs: 8 bf16 of an interleaved vector -> first and second elements.
__device__ __forceinline__ void deinterleave4(u32x4 w, u32x2& lo, u32x2& hi) {
  lo = u32x2{(w[0] & 0xffffu) | (w[1] << 16), (w[2] & 0xffffu) | (w[3] << 16)};
  hi = u32x2{(w[0] >> 16) | (w[1] & 0xffff0000u), (w[2] >> 16) | (w[3] & 0xffff0000u)};
}

// Rotate a query pair at position p (accurate angle per pair).
__device__ __forceinline__ void rotate_q_pair(float x1, float x2, int p, double rev, float& y1, float& y2) {
  const float2 cs = rope_cs(p, rev);
  y1 = fmaf(x1, cs.x, -(x2 * cs.y));
  y2 = fmaf(x1, cs.y, x2 * cs.x);
}

struct Rec {
  int64_t koff, voff;
  int len, pos, kst, vst;
};

// Read-only tables are read through the constant address space: uniform loads from it become scalar loads, whose
// waits (lgkmcnt) do not drain the vector-memory queue that holds the next tile's prefetched K / V.
template <typename T>
using cptr = const T __attribute__((address_space(4)))*;
template <typename T>
__device__ __forceinline__ cptr<T> as_const(const T* p) {
  return (cptr<T>)p;
}

__device__ __forceinline__ Rec load_rec(cptr<lazy_chunk_t> c) {
  Rec r;
  r.koff = c->k_offset;
  r.voff = c->v_offset;
  r.len = c->len;
  r.pos = c->pos_offset;
  r.kst = c->k_stride;
  r.vst = c->v_stride;
  return r;
}

// Walks the key tiles of one request that belong to one KV split: tiles never straddle chunks; the request's
// tiles (chunk after chunk, TK keys each, the last one of a chunk possibly partial) are numbered and split
// evenly.  With the causal rule, tiles whose first key lies after the last query of the workgroup are skipped.
template <int TK>
struct TileIter {
  cptr<lazy_chunk_t> recs;
  int i, end, j0, left;
  Rec cur, nxt;  // records i and i + 1 (nxt only while i + 1 < end): the next record is always loaded ahead

  // The tile counts are taken one record per lane, 64 records at a time, with a wave-wide prefix sum, so that a long
  // chunk table costs a few parallel loads rather than a chain of dependent ones.  Must be called by whole waves
  // with wave-uniform arguments; every member ends up wave-uniform.
  //
  // The loads of the first 256 records come first and on their own (first_block), so that a caller can issue other
  // loads while they are in flight: record c0 + lane whole (the record holding the split's first tile and the one
  // after it then come from a lane instead of one more dependent load), and the lengths of records
  // c0 + 64 (u + 1) + lane.  Indexes past the table's end read its last record and are ignored afterwards, so no
  // load sits behind a per-lane branch.
  struct First {
    lazy_chunk_t mine;
    int len[3];
  };
  __device__ static First first_block(const lazy_chunk_t* table, int c0, int c1) {
    First f = {};
    if (c1 > c0) {
      const int k = c0 + (threadIdx.x & 63);
      f.mine = table[min(k, c1 - 1)];
#pragma unroll
      for (int u = 0; u < 3; ++u) f.len[u] = table[min(k + 64 * (u + 1), c1 - 1)].len;
    }
    return f;
  }
  __device__ void init(const lazy_chunk_t* table, int c0, int c1, int split, int splits) {
    init(table, c0, c1, split, splits, first_block(table, c0, c1));
  }
  __device__ void init(const lazy_chunk_t* table, int c0, int c1, int split, int splits, const First& first) {
    recs = as_const(table);
    end = c1;
    const int lane = threadIdx.x & 63;
    const lazy_chunk_t& mine = first.mine;
    // Pass 1: the request's tile count, four blocks of 64 records at a time; the first four blocks' counts stay in
    // registers for pass 2.
    int ntiles = 0, ntb[4];
    for (int k0 = c0; k0 < c1; k0 += 256) {
      int nt[4], sum = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = k0 + 64 * u + lane;
        const int len = k0 != c0 ? (k < c1 ? table[k].len : 0) : u == 0 ? mine.len : first.len[u - 1];
        nt[u] = k < c1 ? (len + TK - 1) / TK : 0;
        if (k0 == c0) ntb[u] = nt[u];
        sum += nt[u];
      }
      ntiles += __builtin_amdgcn_readlane(wave_incl_scan(sum), 63);
    }
    const int lo = (int)((int64_t)ntiles * split / splits);
    const int hi = (int)((int64_t)ntiles * (split + 1) / splits);
    left = hi - lo;
    i = c1;
    j0 = 0;
    if (left <= 0) return;
    // Pass 2: the record holding tile lo, the first whose inclusive tile count exceeds lo.
    int acc = 0;
    for (int k0 = c0; k0 < c1; k0 += 64) {
      const int k = k0 + lane;
      const int b = (k0 - c0) >> 6;
      const int nt = b < 4 ? (b == 0 ? ntb[0] : b == 1 ? ntb[1] : b == 2 ? ntb[2] : ntb[3])
                           : (k < c1 ? (table[k].len + TK - 1) / TK : 0);
      const int incl = acc + wave_incl_scan(nt);
      const uint64_t hit = __ballot(k < c1 && incl > lo);
      if (hit) {
        const int f = __builtin_ctzll(hit);
        i = k0 + f;
        j0 = (lo - __builtin_amdgcn_readlane(incl - nt, f)) * TK;
        break;
      }
      acc = __builtin_amdgcn_readlane(incl, 63);
    }
    const int f = i - c0;
    if (f < 64) {
      cur = lane_rec(mine, f);
      if (i + 1 < end) nxt = f + 1 < 64 ? lane_rec(mine, f + 1) : load_rec(recs + i + 1);
    } else {
      cur = load_rec(recs + i);
      if (i + 1 < end) nxt = load_rec(recs + i + 1);
    }
  }
  // Lane f's record as a wave-uniform value.
  __device__ static Rec lane_rec(const lazy_chunk_t& r, int f) {
    Rec x;
    x.koff = ((int64_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)r.k_offset >> 32), f) << 32) |
             (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)r.k_offset, f);
    x.voff = ((int64_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)r.v_offset >> 32), f) << 32) |
             (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)r.v_offset, f);
    x.len = __builtin_amdgcn_readlane(r.len, f);
    x.pos = __builtin_amdgcn_readlane(r.pos_offset, f);
    x.kst = __builtin_amdgcn_readlane(r.k_stride, f);
    x.vst = __builtin_amdgcn_readlane(r.v_stride, f);
    return x;
  }
  __device__ void step() {
    --left;
    j0 += TK;
    // Zero-length records own no tile, so while tiles are left a record with keys lies ahead.
    while (left > 0 && j0 >= cur.len) {
      ++i;
      j0 = 0;
      cur = nxt;
      if (i + 1 < end) nxt = load_rec(recs + i + 1);
    }
  }
  // Move to the next tile that some query of the workgroup can see (the current one included).
  __device__ bool seek(bool causal, int qmax) {
    while (left > 0) {
      if (!causal || cur.pos + j0 <= qmax) return true;
      step();
    }
    return false;
  }
  // Advance by `n` tiles (fewer if the split ends first).
  __device__ void skip(int n) {
    for (int k = 0; k < n && left > 0; ++k) step();
  }
  // seek() for a walker that owns every stride-th tile of the split (the decode waves): invisible tiles are passed
  // over `stride` at a time, so the walker stays on its own residue class of tiles.  Positions need not increase
  // along the table, so a tile after the query may precede visible ones.
  __device__ bool seek_strided(bool causal, int qmax, int stride) {
    while (left > 0) {
      if (!causal || cur.pos + j0 <= qmax) return true;
      skip(stride);
    }
    return false;
  }
};

// Angles: the rotation of key j of a chunk (position pos + j) uses one decomposition everywhere (lazy kernels and
// the materialising copy), so every path produces bit-identical rotated keys:
//     angle(pos + j) = base(pos + 32 * floor(j / 32)) + row(j mod 32)
// with cos/sin of each part from rope_cs and one angle addition (rotate_pair).
constexpr int kAngleRows = 32;

// LDS layout constants of a 64-key prefill tile.  Bank-conflict notes: gfx950 LDS has 64 banks of 4 bytes and
// serves a 16-byte read for 16 lanes per pass (8-byte reads: 32 lanes per pass; writes: 8 lanes per pass, half
// the read rate); a pattern is conflict free when the lanes of one pass that read distinct addresses cover
// distinct banks.
//  - K tile rows are D + 8 elements apart (a 4-bank shift per row, so 16 consecutive rows of one 16-byte column
//    tile the 64 banks); the 16-byte blocks of a row are permuted by kblk_t().
//  - The V tile is row-major (key, dimension) with rows D + 32 elements apart (a 16-bank shift per row): the
//    transposing reads (ds_read_b64_tr_b16: 32 lanes read 4 rows x 64 bytes per pass) hit 4 disjoint 16-bank
//    groups.  With rows D + 16 apart they conflict two ways.
//  - cos/sin rows interleave (c, s) with a 4-float gap after every 32 pairs (cs_idx), and the per-row table has a
//    row stride of 8 (mod 64) floats for D = 128 and 4 for D = 64: the 16-byte reads of the loader threads of
//    one pass (4 or 8 threads per key row) hit distinct banks.
template <int D>
struct TileLayout {
  static constexpr int KLD = D + kPad;                    // K tile: [64][KLD], head dimension in virtual order
  static constexpr int VLD = D + 32;                      // V tile: [64][VLD], natural layout
  static constexpr int CSW = D + 4 * ((D / 2 - 1) / 32);  // floats per cos/sin row: (c, s) of pair t at cs_idx(t)
  static constexpr int CSD_LD = CSW + 4;                  // row stride of the per-row table
};

// Transposing LDS read (gfx950 ds_read_b64_tr_b16).  Within each group of 16 lanes, lane i supplies the address
// of 4 consecutive 16-bit elements M[i][0..3]; lane j receives M[4e + j/4][j%4] for e = 0..3.  With lane i pointing
// at row (base + i/4) and column (4 * (i%4)) of a row-major tile, lane j gets column j of rows base..base+3, which is
// an MFMA operand fragment of four consecutive keys for one dimension.
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 tr_read(const uint16_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}
template <int D>
__device__ __forceinline__ int cs_idx(int t) { return 2 * t + 4 * (t / 32); }

// Four query pairs (t0..t0+3 with their partners t0+D/2..) of one query row (raw bf16: lo = elements t0..t0+3,
// hi = t0+D/2..t0+D/2+3), rotated at position p, as one 8-element
// MFMA fragment in virtual order [low t0..t0+3, high t0..t0+3].  The angles follow the decomposition used for the
// keys: cos/sin(p theta_t) from the query block
// base (qb: position 32 (p / 32)) and the per-row delta table (qd: row p % 32), one angle addition per pair.
template <int D>
__device__ __forceinline__ bf16x8 q_fragment_tab(u32x2 lo, u32x2 hi, int t0, const float* qb, const float* qd,
                                                 bool valid) {
  // Rows past the end are computed like the others and zeroed at the end: no per-lane branch, so the waits for the
  // raw Q loads stay exact (a branch makes the compiler wait for every load in flight, the first tile's included).
  const f32x4 b01 = reinterpret_cast<const f32x4*>(qb + cs_idx<D>(t0))[0];
  const f32x4 b23 = reinterpret_cast<const f32x4*>(qb + cs_idx<D>(t0))[1];
  const f32x4 d01 = reinterpret_cast<const f32x4*>(qd + cs_idx<D>(t0))[0];
  const f32x4 d23 = reinterpret_cast<const f32x4*>(qd + cs_idx<D>(t0))[1];
  float y1[4], y2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x1 = (e & 1) ? bf_hi(lo[e >> 1]) : bf_lo(lo[e >> 1]);
    const float x2 = (e & 1) ? bf_hi(hi[e >> 1]) : bf_lo(hi[e >> 1]);
    const f32x4& bq = e < 2 ? b01 : b23;
    const f32x4& dq = e < 2 ? d01 : d23;
    const int o2 = 2 * (e & 1);
    rotate_pair(x1, x2, make_float2(bq[o2], bq[o2 + 1]), make_float2(dq[o2], dq[o2 + 1]), y1[e], y2[e]);
  }
  const u32x4 w = {pack2(y1[0], y1[1]), pack2(y1[2], y1[3]), pack2(y2[0], y2[1]), pack2(y2[2], y2[3])};
  return as_bf16x8(valid ? w : u32x4{0, 0, 0, 0});
}

__device__ __forceinline__ const uint16_t* k_ptr(const uint16_t* pool, const Rec& r, int g, int j0, int d) {
  return pool + r.koff + ((int64_t)g * r.kst + j0) * d;
}
__device__ __forceinline__ const uint16_t* v_ptr(const uint16_t* pool, const Rec& r, int g, int j0, int d) {
  return pool + r.voff + ((int64_t)g * r.vst + j0) * d;
}

// ---------------------------------------------------------------------------------------------------------------
// Prefill: workgroup = (row tile of 32*NW*RB packed query rows, KV head, request x split).  Packed row =
// token * G + g (the G query heads sharing one KV head, Sec. 3.5).  NW waves; each wave owns RB blocks of 32 rows,
// one row per lane pair (lane, lane+32).  The launch uses eight waves x one block (256 rows, the K rotation of a
// tile shared by all of them) or four waves x one block (128 rows); RB = 2 (every K / V fragment read from LDS
// feeding two MFMAs) exists as a compile-time option but needs more registers than a wave has.  NBUF = 2
// double-buffers the LDS tiles (one barrier per tile, the next tile's global loads in flight during the current
// tile's MFMAs); NBUF = 1 keeps the LDS small enough for two workgroups per CU.
// ---------------------------------------------------------------------------------------------------------------
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2): linear id L runs on XCD L % 8.  Two
// maps from L to the logical workgroup:
//  - contiguous (uniform batches): XCD k takes the k-th eighth of the logical ids, i.e. whole requests with all of
//    their heads and splits, which measured fastest when requests are alike;
//  - interleaved (ragged batches): the nx row tiles and ny heads of one (request, split) unit z stay on one XCD,
//    and unit z runs on XCD z % 8 (its XCD's m-th workgroup is tile m % (nx ny) of unit z = L % 8 + 8 (m / (nx ny))),
//    so requests of different lengths are spread evenly over the XCDs instead of piling onto some of them.
// Both fall back to the identity where the counts do not divide by 8.
// Both maps are evaluated and one is selected, with no branch: the kernel's first loads then issue together.
__device__ __forceinline__ int xcd_remap(int id, int n, int inner, int units, bool interleave) {
  const int m = id >> 3;
  const int spread = (units & 7) ? id : m % inner + inner * ((id & 7) + 8 * (m / inner));
  const int per = n >> 3;
  const int whole = id < (per << 3) ? (id & 7) * per + m : id;
  return interleave ? spread : whole;
}

// Query positions of a workgroup of at most 256 rows span at most 256 consecutive positions: at most 9 blocks of 32.
constexpr int kQueryBases = 9;

template <int D, int NBUF>
struct PrefillSmem {
  using S = TileLayout<D>;
  uint16_t k[NBUF][kSub * S::KLD] __attribute__((aligned(16)));
  uint16_t v[NBUF][kSub * S::VLD] __attribute__((aligned(16)));
  float csd[kAngleRows * S::CSD_LD] __attribute__((aligned(16)));  // cos/sin(delta theta_t), delta < 32
  float csb[2][2][S::CSW] __attribute__((aligned(16)));            // [tile parity][half]: cos/sin(base theta_t)
  float qb[kQueryBases][S::CSW] __attribute__((aligned(16)));      // cos/sin(32 a theta_t) for the query blocks
  double freq[D / 2];
};

// Physical 16-byte block of a K tile row for a loader with TPR threads per row: the TPR threads of one row write
// blocks 16 pairs apart (TPR = 4) or 8 pairs apart (TPR = 8); both swizzles send them to distinct bank groups.
template <int TPR>
__device__ __forceinline__ int kblk_t(int b) {
  return TPR == 8 ? (b ^ ((b >> 3) & 1)) : (b ^ (((b >> 3) & 1) << 1));
}

// Cooperative loader of one 64-key tile for the prefill kernel with NT threads: TPR = NT / 64 threads per key row,
// each rotating PP = D / (2 TPR) pairs of its row; V copied row-major in 16-byte chunks (VC per thread, of the same
// row, so that a thread's share of K and V is one key row: threads 0..NT/2-1 hold rows 0..31).
// The per-row cos/sin constants are written to a private LDS slice once per workgroup and read per tile.
template <int D, int KMI, int NT, bool CSD_REGS = false>
struct PLoader {
  using S = TileLayout<D>;
  static constexpr int KM = keys_of(KMI);
  static constexpr bool ROT = KM == kKeysNope || KM == kKeysLocal, LOCAL = KM == kKeysLocal,
                        IL = interleaved_of(KMI);
  static constexpr int TPR = NT / kSub;
  static constexpr int PP = D / (2 * TPR);
  static constexpr int NV = PP / 8;
  static constexpr int VC = kSub * (D / 8) / NT;
  static_assert(PP % 8 == 0, "each loader thread rotates whole groups of 8 pairs");
  static_assert(VC * TPR == D / 8, "a row's V chunks are shared by its TPR threads");
  u32x4 klo[NV], khi[NV];
  u32x4 vr[VC];
  float2 cdr[CSD_REGS && KM == kKeysNope ? PP : 1];
  int tid, row, part;

  __device__ void init(int t) {
    tid = t;
    row = t / TPR;
    part = t % TPR;
  }
  // With CSD_REGS, after that barrier: keep this thread's per-row constants in registers (the loop writes LDS, so
  // they cannot be re-derived inside it).
  __device__ void load_constants(const float* csd) {
    if (KM == kKeysNope && CSD_REGS) {
      const float* cd = csd + (row & (kAngleRows - 1)) * S::CSD_LD;
#pragma unroll
      for (int e = 0; e < PP; ++e) cdr[e] = *reinterpret_cast<const float2*>(cd + cs_idx<D>(part * PP + e));
    }
  }

  __device__ void fetch(const uint16_t* kbase, const uint16_t* vbase, int nvalid) {
    const u32x4 zero = {0, 0, 0, 0};
    if (nvalid >= kSub) {
      if (IL) {
        const u32x4* src = reinterpret_cast<const u32x4*>(kbase + (size_t)row * D + 2 * part * PP);
#pragma unroll
        for (int v = 0; v < NV; ++v) deinterleave8(src[2 * v], src[2 * v + 1], klo[v], khi[v]);
      } else {
        const uint16_t* src = kbase + (size_t)row * D + part * PP;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          klo[v] = reinterpret_cast<const u32x4*>(src)[v];
          khi[v] = reinterpret_cast<const u32x4*>(src + D / 2)[v];
        }
      }
#pragma unroll
      for (int i = 0; i < VC; ++i)
        vr[i] = *reinterpret_cast<const u32x4*>(vbase + (size_t)row * D + 8 * (part + TPR * i));
      return;
    }
    const bool ok = row < nvalid;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      u32x4 lo, hi;
      if (IL) {
        const u32x4* src = reinterpret_cast<const u32x4*>(kbase + (size_t)(ok ? row : 0) * D + 2 * part * PP);
        deinterleave8(src[2 * v], src[2 * v + 1], lo, hi);
      } else {
        const uint16_t* src = kbase + (size_t)(ok ? row : 0) * D + part * PP;
        lo = reinterpret_cast<const u32x4*>(src)[v];
        hi = reinterpret_cast<const u32x4*>(src + D / 2)[v];
      }
      klo[v] = ok ? lo : zero;
      khi[v] = ok ? hi : zero;
    }
#pragma unroll
    for (int i = 0; i < VC; ++i) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(vbase + (size_t)(ok ? row : 0) * D + 8 * (part + TPR * i));
      vr[i] = ok ? x : zero;
    }
  }

  // cb: the tile's two base tables [2][CSW] (rows 0..31 and 32..63; for local-position keys both hold the record
  // offset's angles and the per-row table is not used).
  __device__ void store(uint16_t* kbuf, uint16_t* vtbuf, const float* cb2, const float* csd) {
    uint16_t* krow = kbuf + row * S::KLD;
    const float* cb = cb2 + (row / kAngleRows) * S::CSW;
    const float* cd = csd + (row & (kAngleRows - 1)) * S::CSD_LD;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int t0 = part * PP + 8 * v;
      u32x4 w0, w1;
      if (ROT) {
        float yl[8], yh[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x1 = (e & 1) ? bf_hi(klo[v][e >> 1]) : bf_lo(klo[v][e >> 1]);
          const float x2 = (e & 1) ? bf_hi(khi[v][e >> 1]) : bf_lo(khi[v][e >> 1]);
          const int ci = cs_idx<D>(t0 + e);
          if (LOCAL) {
            rotate_by(x1, x2, *reinterpret_cast<const float2*>(cb + ci), yl[e], yh[e]);
          } else {
            const float2 d = CSD_REGS ? cdr[8 * v + e] : *reinterpret_cast<const float2*>(cd + ci);
            rotate_pair(x1, x2, *reinterpret_cast<const float2*>(cb + ci), d, yl[e], yh[e]);
          }
        }
        w0 = u32x4{pack2(yl[0], yl[1]), pack2(yl[2], yl[3]), pack2(yh[0], yh[1]), pack2(yh[2], yh[3])};
        w1 = u32x4{pack2(yl[4], yl[5]), pack2(yl[6], yl[7]), pack2(yh[4], yh[5]), pack2(yh[6], yh[7])};
      } else {
        w0 = u32x4{klo[v][0], klo[v][1], khi[v][0], khi[v][1]};
        w1 = u32x4{klo[v][2], klo[v][3], khi[v][2], khi[v][3]};
      }
      *reinterpret_cast<u32x4*>(krow + 8 * kblk_t<TPR>(t0 / 4)) = w0;
      *reinterpret_cast<u32x4*>(krow + 8 * kblk_t<TPR>(t0 / 4 + 1)) = w1;
    }
#pragma unroll
    for (int i = 0; i < VC; ++i) *reinterpret_cast<u32x4*>(vtbuf + row * S::VLD + 8 * (part + TPR * i)) = vr[i];
  }
};

// Base tables of a 64-key tile whose first key sits at position b0: [0] for rows 0..31, [1] for rows 32..63.
// For local-position keys b0 is the record offset and both halves get its angles.
template <int D, bool LOCAL>
__device__ __forceinline__ void prefill_base(float* csb2, const double* freq, int tid, int b0) {
  if (tid < D) {
    const int h = tid / (D / 2), t = tid % (D / 2);
    *reinterpret_cast<float2*>(csb2 + h * TileLayout<D>::CSW + cs_idx<D>(t)) =
        rope_cs(LOCAL ? b0 : b0 + kAngleRows * h, freq[t]);
  }
}

// V^T fragments of 16-key step s2 for the four 32-dimension blocks (two transposing reads each).
template <int D>
__device__ __forceinline__ void v_fragments(const uint16_t* vlane, int s2, u32x4 (&vv)[D / 32]) {
  using S = TileLayout<D>;
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    const u32x2 lo = tr_read(vlane + (16 * s2) * S::VLD + 32 * db);
    const u32x2 hi = tr_read(vlane + (16 * s2 + 8) * S::VLD + 32 * db);
    vv[db] = u32x4{lo[0], lo[1], hi[0], hi[1]};
  }
}

// One 64-key tile for one wave's RB blocks of 32 query rows: S^T = K Q^T on the matrix cores, the key mask (tile
// tail and position-based causal rule), the online-softmax update with lazy rescaling, and O^T += V^T P^T.
// kb / vt: the tile's rotated K and row-major V in LDS; b0: position of the tile's first key; nvalid: keys in the
// tile; qmin: smallest query position of the workgroup (tiles entirely at or before it need no causal mask).
// ab: per row block the ALiBi slope over the scale (only with ALIBI).
template <int D, int NT, int RB, bool ALIBI>
__device__ __forceinline__ void attend_tile(const uint16_t* kb, const uint16_t* vt, int lane,
                                            const bf16x8 (&qf)[RB][D / 16], f32x16 (&o)[RB][D / 32],
                                            float (&m2)[RB], float (&lsum)[RB], const int (&qpos)[RB], int b0,
                                            int nvalid, int qmin, int causal, float c, const float (&ab)[RB]) {
  using S = TileLayout<D>;
  const int h2 = lane >> 5;
  // Transposing-read address of this lane in the V tile: row 4*(g/2) + i/4 (+ 16 per key step, + 8 for the
  // second half of the fragment), column 16*(g%2) + 4*(i%4) (+ 32 per dimension block); g = lane/16, i = lane%16.
  const uint16_t* vlane = vt + (4 * ((lane >> 4) >> 1) + ((lane & 15) >> 2)) * S::VLD +
                          16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // S^T = K Q^T: two 32-key blocks per row block; each K fragment feeds RB MFMAs.  Fragments are read one
  // k-step ahead and the scheduler is fenced per k-step, which bounds the registers held by in-flight reads.
  f32x16 sa[RB][2];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) sa[rb][0] = sa[rb][1] = f32x16{};
  // Waves raise their issue priority while they feed the matrix cores, so that the MFMA blocks of one wave run
  // ahead and the other wave's softmax / rotation VALU work fills the gaps.
  __builtin_amdgcn_s_setprio(1);
  {
    const uint16_t* kl = kb + (lane & 31) * S::KLD;
    u32x4 kv[2][2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
      kv[0][blk] = *reinterpret_cast<const u32x4*>(kl + 32 * blk * S::KLD + 8 * kblk_t<NT / kSub>(h2));
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      if (s + 1 < D / 16) {
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
          kv[(s + 1) & 1][blk] = *reinterpret_cast<const u32x4*>(kl + 32 * blk * S::KLD +
                                                                 8 * kblk_t<NT / kSub>(2 * (s + 1) + h2));
      }
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          sa[rb][blk] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv[s & 1][blk]), qf[rb][s], sa[rb][blk], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __builtin_amdgcn_s_setprio(0);
  if (ALIBI) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // key 32 blk + 8 (i / 4) + 4 h2 + i % 4: the lane's 4 h2 goes into the base, the rest is a constant
      const float base = ab[rb] * (float)(b0 + 4 * h2 - qpos[rb]);
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          sa[rb][blk][i] = fmaf(ab[rb], (float)(32 * blk + 8 * (i >> 2) + (i & 3)), sa[rb][blk][i] + base);
    }
  }
  if (nvalid < kSub || (causal && b0 + kSub - 1 > qmin)) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kk = 32 * blk + 8 * (i >> 2) + 4 * h2 + (i & 3);
          const bool ok = kk < nvalid && (!causal || b0 + kk <= qpos[rb]);
          if (!ok) sa[rb][blk][i] = -INFINITY;
        }
  }
  uint32_t pk[RB][16];  // bf16 pairs of P: block blk, keys 8 (i / 4) + 4 h2 + i % 4 for i = 2 j, 2 j + 1
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    // Lazy rescale: the reference max only moves when this tile's max exceeds it by more than kRescaleSlack.  The
    // probabilities are first formed against the current reference; if this lane's sum of them is at most
    // 2^kRescaleSlack, none of them exceeds 2^kRescaleSlack, so the tile's max cannot exceed the reference by more
    // than the slack and the maximum need not be taken.  Otherwise (and before any reference exists) the maximum
    // decides as usual and the probabilities are formed again if the reference moved.
    auto form = [&](float muse, float& ps) {
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint32_t pp = pack2(fast_exp2(fmaf(sa[rb][blk][2 * j], c, -muse)),
                                    fast_exp2(fmaf(sa[rb][blk][2 * j + 1], c, -muse)));
          pk[rb][8 * blk + j] = pp;
          if (j & 1)
            ps1 = add_pair(pp, ps1);
          else
            ps0 = add_pair(pp, ps0);
        }
      ps = ps0 + ps1;
    };
    float ps;
    if constexpr (ALIBI) {
      // ALiBi scores grow tile by tile towards the query, so the reference moves on most tiles: the maximum is
      // taken first and the probabilities are formed once.
      float mx = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sa[rb][blk][i]);
      mx = xor32_max(mx);
      const float mt = mx * c;
      if (__any(mt > m2[rb] + kRescaleSlack)) {
        const float mnew = fmaxf(m2[rb], mt);
        const float alpha = m2[rb] == -INFINITY ? 0.f : fast_exp2(m2[rb] - mnew);
        lsum[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) o[rb][db] *= alpha;
        m2[rb] = mnew;
      }
      form(m2[rb] == -INFINITY ? 0.f : m2[rb], ps);
      lsum[rb] += ps;
      continue;
    }
    form(m2[rb] == -INFINITY ? 0.f : m2[rb], ps);
    if (__any(!(ps <= kRescaleBound) || m2[rb] == -INFINITY)) {
      float mx = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sa[rb][blk][i]);
      mx = xor32_max(mx);
      const float mt = mx * c;
      if (__any(mt > m2[rb] + kRescaleSlack)) {
        const float mnew = fmaxf(m2[rb], mt);
        const float alpha = m2[rb] == -INFINITY ? 0.f : fast_exp2(m2[rb] - mnew);
        lsum[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) o[rb][db] *= alpha;
        m2[rb] = mnew;
        form(m2[rb] == -INFINITY ? 0.f : m2[rb], ps);
      }
    }
    lsum[rb] += ps;
  }

  // O^T += V^T P^T: four 16-key steps; each V fragment feeds RB MFMAs (same bounded read-ahead).
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int s2 = 0; s2 < 4; ++s2) {
    bf16x8 pb[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int j0 = 8 * (s2 >> 1) + 4 * (s2 & 1);
      pb[rb] = as_bf16x8(u32x4{pk[rb][j0], pk[rb][j0 + 1], pk[rb][j0 + 2], pk[rb][j0 + 3]});
    }
    u32x4 vv[D / 32];
    v_fragments<D>(vlane, s2, vv);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        o[rb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv[db]), pb[rb], o[rb][db], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }

  __builtin_amdgcn_s_setprio(0);
}

template <int D, int KMI, int NW, int NBUF, int RB>
__global__ __launch_bounds__(NW * 64)
__attribute__((amdgpu_waves_per_eu(RB == 1 ? 2 : 1, RB == 1 ? 2 : 1))) void prefill_kernel(AttnArgs a) {
  __shared__ PrefillSmem<D, NBUF> sm;
  constexpr int KM = keys_of(KMI);
  constexpr bool ALIBI = KM == kKeysAlibi;
  constexpr bool ROT = KM == kKeysNope || KM == kKeysLocal, LOCAL = KM == kKeysLocal, IL = interleaved_of(KMI);
  using S = TileLayout<D>;
  constexpr int NT = NW * 64;
  constexpr int BM = 32 * NW * RB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nx = gridDim.x, ny = gridDim.y;
  // The argument block's lines are fetched in one round trip: the index arithmetic below needs the grid constants and
  // the split count, and right after it the index-array pointers (otherwise loaded one round trip later).
  asm volatile("" ::"s"(a.q_start), "s"(a.chunk_start), "s"(a.splits), "s"(a.xcd_interleave), "s"(nx), "s"(ny),
               "s"(gridDim.z));
  const int lid = uniform(xcd_remap(blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z), nx * ny * gridDim.z, nx * ny,
                                    gridDim.z, a.xcd_interleave != 0));
  const int qtile = lid % nx;
  const int g = (lid / nx) % ny;
  const int zz = lid / (nx * ny);
  const int r = zz / a.splits, split = zz % a.splits;
  // The request's index entries are loaded together, before the exit test that needs only q_start (the empty asm
  // keeps the compiler from sinking the other loads below the test, which would cost two more round trips).
  const int qs = as_const(a.q_start)[r], qe = as_const(a.q_start)[r + 1], qp0 = as_const(a.q_pos0)[r];
  const int c0 = as_const(a.chunk_start)[r], c1 = as_const(a.chunk_start)[r + 1];
  asm volatile("" ::"s"(qp0), "s"(c0), "s"(c1));
  const int G = a.group;
  const int nrows = (qe - qs) * G;
  const int row0 = qtile * BM;
  if (row0 >= nrows) return;

  const int h2 = lane >> 5;
  bool rvalid[RB];
  int tok[RB], head[RB], qpos[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int prow = row0 + wave * 32 * RB + 32 * rb + (lane & 31);
    rvalid[rb] = prow < nrows;
    tok[rb] = rvalid[rb] ? prow / G : 0;
    head[rb] = g * G + (rvalid[rb] ? prow % G : 0);
    qpos[rb] = qp0 + tok[rb];
  }
  const int last = min(row0 + BM, nrows) - 1;
  const int qmin = uniform(qp0 + row0 / G), qmax = uniform(qp0 + last / G);

  // Loads first: the first block of the chunk table and raw Q.  The angle tables below need neither and are computed
  // while they are in flight.
  const TileIter<kSub>::First first = TileIter<kSub>::first_block(a.chunks, c0, c1);
  u32x2 qraw[RB][D / 16][2];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const uint16_t* qrow = a.q + ((int64_t)(qs + tok[rb]) * a.hq + head[rb]) * D;
    // Rows past the request's end read its first query row (tok 0, head g G: always present, since the request
    // has a row here) and give zero fragments below; the loads sit behind no per-lane branch.
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      const int t0 = 8 * s + 4 * h2;
      if (IL) {
        deinterleave4(*reinterpret_cast<const u32x4*>(qrow + 2 * t0), qraw[rb][s][0], qraw[rb][s][1]);
      } else {
        qraw[rb][s][0] = *reinterpret_cast<const u32x2*>(qrow + t0);
        qraw[rb][s][1] = *reinterpret_cast<const u32x2*>(qrow + D / 2 + t0);
      }
    }
  }
  // Every table entry this thread computes below is for pair t = tid % (D/2) (the block size is a multiple of D/2):
  // each thread evaluates its own frequency, with no barrier before the tables.  The per-tile bases in the loop read
  // the frequencies from LDS (fewer registers held across the loop); the tables' barrier publishes them.
  const double rev = ALIBI ? 0.0 : theta_rev(tid % (D / 2), D, a.rope_log2_base, a.inv_freq);
  if (tid < D / 2) sm.freq[tid] = rev;

  // Angle tables: per-row deltas cos/sin(delta theta_t), delta < 32 (queries and keys), and the query block bases
  // cos/sin(32 a theta_t), a = qmin / 32 .. qmax / 32.
  const int qa0 = qmin / kAngleRows, nqb = qmax / kAngleRows - qa0 + 1;
  static_assert(NT % (D / 2) == 0, "a thread's table entries share one pair index");
  for (int e = tid; e < (ALIBI ? 0 : (kAngleRows + nqb) * (D / 2)); e += NT) {
    const int trow = e / (D / 2), t = e % (D / 2);
    float* dst = trow < kAngleRows ? sm.csd + trow * S::CSD_LD : sm.qb[trow - kAngleRows];
    const int p = trow < kAngleRows ? trow : kAngleRows * (qa0 + trow - kAngleRows);
    *reinterpret_cast<float2*>(dst + cs_idx<D>(t)) = rope_cs(p, rev);
  }
  __syncthreads();

  // The chunk-table walk (its loads have been in flight during the tables) and the first tile's K / V, whose
  // latency the Q rotation below covers.
  // Eight-wave and two-block workgroups keep the loader's per-row angle constants in registers.
  PLoader<D, KMI, NT, RB == 2 || NW == 8> ld;
  ld.init(tid);
  TileIter<kSub> it;
  it.init(a.chunks, c0, c1, split, a.splits, first);
  bool have = it.seek(a.causal, qmax);
  if (have)
    ld.fetch(k_ptr(a.k_pool, it.cur, g, it.j0, D), v_ptr(a.v_pool, it.cur, g, it.j0, D),
             min(kSub, it.cur.len - it.j0));

  // Pre-rotated queries take the angle row of position 0 (cos 1, sin 0) for both parts, which leaves them exactly
  // as given without a second code path.
  bf16x8 qf[RB][D / 16];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float* qbr = a.q_prerot ? sm.csd : sm.qb[qpos[rb] / kAngleRows - qa0];
    const float* qdr = sm.csd + (a.q_prerot ? 0 : qpos[rb] & (kAngleRows - 1)) * S::CSD_LD;
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
      qf[rb][s] = ALIBI ? as_bf16x8(rvalid[rb] ? u32x4{qraw[rb][s][0][0], qraw[rb][s][0][1], qraw[rb][s][1][0],
                                                       qraw[rb][s][1][1]}
                                             : u32x4{0, 0, 0, 0})
                        : q_fragment_tab<D>(qraw[rb][s][0], qraw[rb][s][1], 8 * s + 4 * h2, qbr, qdr, rvalid[rb]);
  }

  f32x16 o[RB][D / 32];
  float m2[RB], lsum[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[rb][db] = f32x16{};
    m2[rb] = -INFINITY;
    lsum[rb] = 0.f;
  }
  const float c = a.scale_log2;
  float ab[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) ab[rb] = ALIBI ? alibi_slope(head[rb], a.hq, a.inv_freq, c) : 0.f;

  ld.load_constants(sm.csd);

  // Tile "ahead" state for NBUF == 2: position of the tile after the current one.
  // Eight-wave workgroups: waves w and w + 4 share a SIMD, and the tile barrier would keep them in the same phase
  // (both feeding the matrix core, then both on the vector ALU).  The upper four waves therefore store their share
  // of the next tile at the start of the interval and fetch theirs one tile further ahead, while the lower four
  // store theirs at the end: the two waves on a SIMD alternate between MFMA and VALU phases.  Both halves of a tile
  // are in LDS by the barrier that ends the interval before it is read; the buffer they overwrite was last read in
  // the interval before (double buffering is enough).
  const bool early = NBUF == 2 && NW == 8 && uniform(wave) >= NW / 2;
  TileIter<kSub> ahead = it;
  bool have_ahead = false;
  if (have && NBUF == 2) {
    if (ROT) prefill_base<D, LOCAL>(sm.csb[0][0], sm.freq, tid, it.cur.pos + (LOCAL ? 0 : it.j0));
    ahead.step();
    have_ahead = ahead.seek(a.causal, qmax);
    if (ROT && have_ahead)
      prefill_base<D, LOCAL>(sm.csb[1][0], sm.freq, tid, ahead.cur.pos + (LOCAL ? 0 : ahead.j0));
    __syncthreads();
    ld.store(sm.k[0], sm.v[0], sm.csb[0][0], sm.csd);
    if (early && have_ahead)
      ld.fetch(k_ptr(a.k_pool, ahead.cur, g, ahead.j0, D), v_ptr(a.v_pool, ahead.cur, g, ahead.j0, D),
               min(kSub, ahead.cur.len - ahead.j0));
    __syncthreads();
  }
  int parity = 0;
  while (have) {
    const int nvalid = min(kSub, it.cur.len - it.j0);
    const int b0 = it.cur.pos + it.j0, rec_pos = it.cur.pos;
    int cur_buf = 0;
    bool have_next;
    if (NBUF == 1) {
      it.step();
      have_next = it.seek(a.causal, qmax);
      if (ROT) prefill_base<D, LOCAL>(sm.csb[0][0], sm.freq, tid, LOCAL ? rec_pos : b0);
      __syncthreads();
      ld.store(sm.k[0], sm.v[0], sm.csb[0][0], sm.csd);
      __syncthreads();
      if (have_next)
        ld.fetch(k_ptr(a.k_pool, it.cur, g, it.j0, D), v_ptr(a.v_pool, it.cur, g, it.j0, D),
                 min(kSub, it.cur.len - it.j0));
    } else {
      cur_buf = parity;
      it = ahead;  // the next tile
      have_next = have_ahead;
      if (early && have_next) ld.store(sm.k[parity ^ 1], sm.v[parity ^ 1], sm.csb[parity ^ 1][0], sm.csd);
      if (have_next) {
        if (!early)
          ld.fetch(k_ptr(a.k_pool, it.cur, g, it.j0, D), v_ptr(a.v_pool, it.cur, g, it.j0, D),
                   min(kSub, it.cur.len - it.j0));
        ahead.step();
        have_ahead = ahead.seek(a.causal, qmax);
        if (early && have_ahead)
          ld.fetch(k_ptr(a.k_pool, ahead.cur, g, ahead.j0, D), v_ptr(a.v_pool, ahead.cur, g, ahead.j0, D),
                   min(kSub, ahead.cur.len - ahead.j0));
      }
    }
    attend_tile<D, NT, RB, ALIBI>(sm.k[cur_buf], sm.v[cur_buf], lane, qf, o, m2, lsum, qpos, b0, nvalid, qmin,
                                  a.causal, c, ab);
    if (NBUF == 2) {
      // Base angles two tiles ahead go to the table slot this tile used; the next tile goes to the other buffer.
      if (ROT && have_ahead)
        prefill_base<D, LOCAL>(sm.csb[parity][0], sm.freq, tid, ahead.cur.pos + (LOCAL ? 0 : ahead.j0));
      if (!early && have_next) ld.store(sm.k[parity ^ 1], sm.v[parity ^ 1], sm.csb[parity ^ 1][0], sm.csd);
      __syncthreads();
      parity ^= 1;
    }
    have = have_next;
  }

  if constexpr (NBUF == 2 && RB == 1) {
    // Normalised output and log-sum-exp: the final result, or with several splits this split's partial result.
    // The output goes through LDS (the tile buffers are free after the loop's last barrier): each wave stages its 32
    // rows, then writes whole 256-byte rows, 16 bytes per lane, so that one store instruction covers four rows
    // instead of 16 bytes in each of 32 rows.
    constexpr int OLD = D + 8;
    using SM = PrefillSmem<D, NBUF>;
    static_assert(offsetof(SM, v) == sizeof(sm.k) &&
                      sizeof(sm.k) + sizeof(sm.v) >= sizeof(uint16_t) * NW * 32 * OLD,
                  "the output stage spans the K and V tile buffers");
    uint16_t* stage = &sm.k[0][0] + wave * 32 * OLD;
    const float ltot = xor32_sum(lsum[0]);
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<u32x2*>(stage + (lane & 31) * OLD + 32 * db + 8 * q4 + 4 * h2) =
            u32x2{pack2(o[0][db][4 * q4] * inv, o[0][db][4 * q4 + 1] * inv),
                  pack2(o[0][db][4 * q4 + 2] * inv, o[0][db][4 * q4 + 3] * inv)};
    if (rvalid[0] && h2 == 0) {
      const int64_t orow = (int64_t)(qs + tok[0]) * a.hq + head[0];
      float* lse_dst = a.splits == 1 ? (a.lse ? a.lse + orow : nullptr) : a.ws_lse + (int64_t)split * a.total_q * a.hq + orow;
      if (lse_dst) *lse_dst = ltot > 0.f ? (m2[0] + log2f(ltot)) * kLn2 : -INFINITY;
    }
    __syncthreads();
    uint16_t* base = a.splits == 1 ? a.out : a.ws_o + (int64_t)split * a.total_q * a.hq * D;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int lrow = 4 * i + (lane >> 4);
      const int prow = row0 + 32 * wave + lrow;
      if (prow < nrows) {
        const int64_t orow = (int64_t)(qs + prow / G) * a.hq + g * G + prow % G;
        *reinterpret_cast<u32x4*>(base + orow * D + 8 * (lane & 15)) =
            *reinterpret_cast<const u32x4*>(stage + lrow * OLD + 8 * (lane & 15));
      }
    }
    return;
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float ltot = xor32_sum(lsum[rb]);
    if (!rvalid[rb]) continue;
    // Normalised output and log-sum-exp: the final result, or with several splits this split's partial result.
    const int64_t orow = (int64_t)(qs + tok[rb]) * a.hq + head[rb];
    const int64_t wrow = (int64_t)split * a.total_q * a.hq + orow;
    uint16_t* dst = a.splits == 1 ? a.out + orow * D : a.ws_o + wrow * D;
    float* lse_dst = a.splits == 1 ? (a.lse ? a.lse + orow : nullptr) : a.ws_lse + wrow;
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int dim = 32 * db + 8 * q4 + 4 * h2;
        *reinterpret_cast<u32x2*>(dst + dim) = u32x2{pack2(o[rb][db][4 * q4] * inv, o[rb][db][4 * q4 + 1] * inv),
                                                     pack2(o[rb][db][4 * q4 + 2] * inv, o[rb][db][4 * q4 + 3] * inv)};
      }
    if (lse_dst && h2 == 0) *lse_dst = ltot > 0.f ? (m2[rb] + log2f(ltot)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Decode: workgroup = (KV split, KV head x head group, request), four waves that stream independently.  The split's
// keys are cut into 32-key tiles (never straddling chunks); wave w takes tiles w, w+4, w+8, ... and keeps its own
// softmax state for up to 16 query heads (one head per MFMA column), with the next tile's K / V already in flight
// in registers while the current one is processed.  No barrier is needed until the four states are merged.
//  - K goes straight from global memory into the A-operand layout of v_mfma_f32_16x16x32_bf16 and is rotated in
//    registers.  Decode uses its own head-dimension order: k-step 2s+h holds, in lane (row, kq), the 8 dims
//    h*D/2 + 32s + 8kq .. +7, so the two halves of every rotation pair sit in the same lane (two k-steps apart)
//    and each half is one 16-byte load.
//  - Block b (0/1) row r of S^T is tile key kappa(b, r) = 16*(r/8) + r%8 + 8b, so a lane's four probabilities of a
//    block are four consecutive keys: exactly what one transposing read of the row-major V slice delivers.
//  - Angles: cos/sin((b0 + kappa) theta_t) = base (per tile, one table per wave, computed one tile ahead) x
//    per-row constants (a 32-row table shared by the workgroup).
// ---------------------------------------------------------------------------------------------------------------
__device__ __forceinline__ int kappa(int b, int r) { return 16 * (r >> 3) + (r & 7) + 8 * b; }

constexpr int kDecWaveKeys = 32;

template <int D>
struct DecodeSmem {
  static constexpr int VLD = D + 16;                 // V slice row stride (elements)
  static constexpr int CSD_LD = D + 4;               // per-row cos/sin row stride (floats): 4 banks per row
  static constexpr int CSB = D + D / 4;              // per-tile base table: (c, s) of pair t at 2t + 4*(t/8)
  uint16_t v[4][kDecWaveKeys * VLD] __attribute__((aligned(16)));
  float csd[kDecWaveKeys * CSD_LD + 32] __attribute__((aligned(16)));  // row r at dec_row(r)
  float csb[4][2][CSB] __attribute__((aligned(16)));
  u32x4 qsave[D / 64][2][64];                       // raw Q fragments [s][half][lane] (local-position keys)
  double freq[D / 2];
};
template <int D>
__device__ __forceinline__ int csb_idx(int t) { return 2 * t + 4 * (t >> 3); }
// Start of row r of the per-row cos/sin table.  The 16 lanes of one 16-byte read pass take rows kappa(b, 0..15) =
// {0..7, 16..23} + 8b at one column; rows 16 apart would share banks (16 x 4-bank shift = 64 banks), so rows
// 16..31 are moved 32 banks further.
template <int D>
__device__ __forceinline__ int dec_row(int r) { return r * DecodeSmem<D>::CSD_LD + 32 * (r >> 4); }

// Raw K / V of one wave tile in registers.
template <int D>
struct DecTile {
  static constexpr int SP = D / 64;          // 16-byte groups per half row per lane
  static constexpr int VC = kDecWaveKeys * (D / 8) / 64;
  u32x4 k[2][SP][2];                         // [block][s][half]
  u32x4 v[VC];
};

// One key row's k-step pair s for this lane (pairs 32 s + 8 kq .. +7): first elements in lo, second in hi for
// the half-split pairing; for the interleaved pairing the raw 16 elements (pairs_of splits them where they are
// used, so that tiles in flight hold no extra registers).
// A 16-byte load of K / V; NT: non-temporal (streamed from HBM without being kept for reuse).
template <bool NT>
__device__ __forceinline__ u32x4 kv_load(const uint16_t* p) {
  if (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return *reinterpret_cast<const u32x4*>(p);
}
template <int D, bool IL, bool NT>
__device__ __forceinline__ void dec_k_pairs(const uint16_t* krow, int s, int kq, u32x4& lo, u32x4& hi) {
  if (IL) {
    lo = kv_load<NT>(krow + 2 * (32 * s + 8 * kq));
    hi = kv_load<NT>(krow + 2 * (32 * s + 8 * kq) + 8);
  } else {
    lo = kv_load<NT>(krow + 32 * s + 8 * kq);
    hi = kv_load<NT>(krow + D / 2 + 32 * s + 8 * kq);
  }
}

template <bool IL>
__device__ __forceinline__ void pairs_of(u32x4 a, u32x4 b, u32x4& lo, u32x4& hi) {
  if (IL) {
    deinterleave8(a, b, lo, hi);
  } else {
    lo = a;
    hi = b;
  }
}

template <int D, bool IL, bool NT>
__device__ __forceinline__ void dec_fetch(DecTile<D>& t, const uint16_t* kbase, const uint16_t* vbase, int nvalid,
                                          int lane) {
  const int r = lane & 15, kq = lane >> 4;
  const u32x4 zero = {0, 0, 0, 0};
  if (nvalid >= kDecWaveKeys) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const uint16_t* row = kbase + (size_t)kappa(b, r) * D;
#pragma unroll
      for (int s = 0; s < DecTile<D>::SP; ++s) dec_k_pairs<D, IL, NT>(row, s, kq, t.k[b][s][0], t.k[b][s][1]);
    }
#pragma unroll
    for (int i = 0; i < DecTile<D>::VC; ++i) {
      const int c = lane + 64 * i;
      t.v[i] = kv_load<NT>(vbase + (size_t)(c / (D / 8)) * D + 8 * (c % (D / 8)));
    }
    return;
  }
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int key = kappa(b, r);
    const bool ok = key < nvalid;
    const uint16_t* row = kbase + (size_t)(ok ? key : 0) * D;
#pragma unroll
    for (int s = 0; s < DecTile<D>::SP; ++s) {
      u32x4 lo, hi;
      dec_k_pairs<D, IL, NT>(row, s, kq, lo, hi);
      t.k[b][s][0] = ok ? lo : zero;
      t.k[b][s][1] = ok ? hi : zero;
    }
  }
#pragma unroll
  for (int i = 0; i < DecTile<D>::VC; ++i) {
    const int c = lane + 64 * i;
    const int key = c / (D / 8);
    const bool ok = key < nvalid;
    const u32x4 x = kv_load<NT>(vbase + (size_t)(ok ? key : 0) * D + 8 * (c % (D / 8)));
    t.v[i] = ok ? x : zero;
  }
}

// One 32-key tile of one decode wave: V into the wave's LDS slice, K rotated in registers (NoPE store: base row cb
// of the tile, per-row rows cd0 / cd1 of blocks 0 / 1) and S^T = K Q^T, the key mask, the online-softmax update
// and O^T += V^T P^T.  lim: this lane's visible keys are the tile keys kk < lim (tile tail and causal rule; it may
// differ between the lanes' columns).
// ALIBI: ab = this lane's column slope over the scale, abase = ab (first key position - query position).
template <int D, bool ROT, bool IL, bool ALIBI>
__device__ __forceinline__ void dec_tile(const DecTile<D>& cur, uint16_t* vw, const uint16_t* vlane, const float* cb,
                                         const float* cd0, const float* cd1, const bf16x8 (&qf)[D / 32],
                                         f32x4 (&o)[D / 16], float& m2, float& lsum, int lim, float c, int lane,
                                         float ab, float abase) {
  using S = DecodeSmem<D>;
  constexpr int SP = DecTile<D>::SP;
  const int kq = lane >> 4;
  // V of this tile into the wave's LDS slice (row-major).
#pragma unroll
  for (int i = 0; i < DecTile<D>::VC; ++i) {
    const int cc = lane + 64 * i;
    *reinterpret_cast<u32x4*>(vw + (cc / (D / 8)) * S::VLD + 8 * (cc % (D / 8))) = cur.v[i];
  }

  // Rotate K in registers and form S^T = K Q^T, one pair of k-steps (low / high halves) at a time.
  f32x4 sa[2] = {f32x4{}, f32x4{}};
#pragma unroll
  for (int s = 0; s < SP; ++s) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      u32x4 wl, wh;
      pairs_of<IL>(cur.k[b][s][0], cur.k[b][s][1], wl, wh);
      u32x4 klo, khi;
      if (ROT) {
        const float* cdb = b ? cd1 : cd0;
        float y1[8], y2[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int t = 32 * s + 8 * kq + e;
          const float x1 = (e & 1) ? bf_hi(wl[e >> 1]) : bf_lo(wl[e >> 1]);
          const float x2 = (e & 1) ? bf_hi(wh[e >> 1]) : bf_lo(wh[e >> 1]);
          rotate_pair(x1, x2, *reinterpret_cast<const float2*>(cb + csb_idx<D>(t)),
                      *reinterpret_cast<const float2*>(cdb + 2 * t), y1[e], y2[e]);
        }
        klo = u32x4{pack2(y1[0], y1[1]), pack2(y1[2], y1[3]), pack2(y1[4], y1[5]), pack2(y1[6], y1[7])};
        khi = u32x4{pack2(y2[0], y2[1]), pack2(y2[2], y2[3]), pack2(y2[4], y2[5]), pack2(y2[6], y2[7])};
      } else {
        klo = wl;
        khi = wh;
      }
      sa[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(klo), qf[2 * s], sa[b], 0, 0, 0);
      sa[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(khi), qf[2 * s + 1], sa[b], 0, 0, 0);
    }
  }
  if (ALIBI) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) sa[b][i] = fmaf(ab, (float)kappa(b, 4 * kq + i), sa[b][i] + abase);
  }
  if (__any(lim < kDecWaveKeys)) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (kappa(b, 4 * kq + i) >= lim) sa[b][i] = -INFINITY;
  }
  // Lazy rescale as in the prefill tile: probabilities against the current reference first; the maximum is only
  // taken when some lane's sum exceeds 2^kRescaleSlack (or no reference exists yet).
  float pr[2][4];
  auto form = [&](float muse) {
    float ps = 0.f;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[b][i] = fast_exp2(fmaf(sa[b][i], c, -muse));
        ps += pr[b][i];
      }
    return ps;
  };
  float ps = form(m2 == -INFINITY ? 0.f : m2);
  if (__any(!(ps <= kRescaleBound) || m2 == -INFINITY)) {
    float mx = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sa[b][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mt = mx * c;
    if (__any(mt > m2 + kRescaleSlack)) {
      const float mnew = fmaxf(m2, mt);
      const float alpha = m2 == -INFINITY ? 0.f : fast_exp2(m2 - mnew);
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) o[db] *= alpha;
      m2 = mnew;
      ps = form(m2 == -INFINITY ? 0.f : m2);
    }
  }
  lsum += ps;
  const bf16x8 pb = as_bf16x8(u32x4{pack2(pr[0][0], pr[0][1]), pack2(pr[0][2], pr[0][3]),
                                    pack2(pr[1][0], pr[1][1]), pack2(pr[1][2], pr[1][3])});
  // O^T += V^T P^T from the wave's V slice (same-wave LDS ordering: written above, read here).
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const u32x2 lo = tr_read(vlane + 16 * db);
    const u32x2 hi = tr_read(vlane + 8 * S::VLD + 16 * db);
    o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]}), pb, o[db], 0,
                                                    0, 0);
  }
}

template <int D, int KMI>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void decode_kernel(AttnArgs a) {
  __shared__ DecodeSmem<D> sm;
  constexpr int KM = keys_of(KMI);
  constexpr bool IL = interleaved_of(KMI), ALIBI = KM == kKeysAlibi, NT = stream_of(KMI);
  // Keys are rotated in registers only for a NoPE store; with local-position keys the query is rotated by the
  // relative offset q_pos - pos_offset whenever the record changes (Sec. 3.2 "Decoding") and the keys are used as
  // stored.
  constexpr bool ROT = KM == kKeysNope, LOCAL = KM == kKeysLocal;
  using S = DecodeSmem<D>;
  constexpr int SP = DecTile<D>::SP;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int split = blockIdx.x;
  const int g = blockIdx.y / a.head_groups, hg = blockIdx.y % a.head_groups;
  const int r = blockIdx.z;
  const int G = a.group;
  const int hcount = min(kDecodeHeadsPerGroup, G - kDecodeHeadsPerGroup * hg);
  const int col = lane & 15, kq = lane >> 4;
  const int qpos = as_const(a.q_pos0)[r];
  const int c0 = as_const(a.chunk_start)[r], c1 = as_const(a.chunk_start)[r + 1];
  asm volatile("" ::"s"(qpos), "s"(c0), "s"(c1));  // one round trip for the three (the compiler would sink qpos)

  const bool hvalid = col < hcount;
  const int head = g * G + kDecodeHeadsPerGroup * hg + (hvalid ? col : 0);
  // Loads first: the first chunk-table block and the raw Q (columns past the group's heads read a valid head and
  // are zeroed once Q is needed; no load sits behind a per-lane branch, which would make the compiler wait for
  // every load in flight at its first use).  The frequency and per-row tables are built while they are in flight,
  // then the table walk issues this wave's first tile.
  const TileIter<kDecWaveKeys>::First first = TileIter<kDecWaveKeys>::first_block(a.chunks, c0, c1);
  u32x4 qraw[SP][2];
  {
    const uint16_t* qrow = a.q + ((int64_t)r * a.hq + head) * D;
#pragma unroll
    for (int s = 0; s < SP; ++s) dec_k_pairs<D, IL, false>(qrow, s, kq, qraw[s][0], qraw[s][1]);
  }
  if (!ALIBI && tid < D / 2) sm.freq[tid] = theta_rev(tid, D, a.rope_log2_base, a.inv_freq);
  __syncthreads();
  // This wave's tiles: every fourth tile of the split, starting at tile `wave`.
  TileIter<kDecWaveKeys> it;
  it.init(a.chunks, c0, c1, split, a.splits, first);
  it.skip(wave);
  bool have = it.seek_strided(a.causal, qpos, 4);
  DecTile<D> cur, nxt;
  if (have)
    dec_fetch<D, IL, NT>(cur, k_ptr(a.k_pool, it.cur, g, it.j0, D), v_ptr(a.v_pool, it.cur, g, it.j0, D),
                 min(kDecWaveKeys, it.cur.len - it.j0), lane);
  if (ROT) {
    // Per-row constants cos/sin(delta theta_t), delta < 32: 16 per thread, while the first tile is in flight.
    for (int e = tid; e < kDecWaveKeys * (D / 2); e += kThreads) {
      const int dr = e / (D / 2), t = e % (D / 2);
      *reinterpret_cast<float2*>(sm.csd + dec_row<D>(dr) + 2 * t) = rope_cs(dr, sm.freq[t]);
    }
  }
  if (ROT && have && lane < D / 2)
    *reinterpret_cast<float2*>(sm.csb[wave][0] + csb_idx<D>(lane)) = rope_cs(it.cur.pos + it.j0, sm.freq[lane]);
#pragma unroll
  for (int s = 0; s < SP; ++s) {
    const u32x4 zero = {0, 0, 0, 0};
    qraw[s][0] = hvalid ? qraw[s][0] : zero;
    qraw[s][1] = hvalid ? qraw[s][1] : zero;
  }
  // Q fragments in the decode head-dimension order, rotated at the query position.  With local-position keys they
  // are built per record instead (below), from the raw query.
  bf16x8 qf[D / 32];
  if (ALIBI) {  // no rotation: the raw query
#pragma unroll
    for (int s = 0; s < SP; ++s) {
      u32x4 ql, qh;
      pairs_of<IL>(qraw[s][0], qraw[s][1], ql, qh);
      qf[2 * s] = as_bf16x8(ql);
      qf[2 * s + 1] = as_bf16x8(qh);
    }
  } else if (!LOCAL) {
#pragma unroll
    for (int s = 0; s < SP; ++s) {
      float y1[8], y2[8];
      const int t0 = 32 * s + 8 * kq;
      u32x4 ql, qh;
      pairs_of<IL>(qraw[s][0], qraw[s][1], ql, qh);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x1 = (e & 1) ? bf_hi(ql[e >> 1]) : bf_lo(ql[e >> 1]);
        const float x2 = (e & 1) ? bf_hi(qh[e >> 1]) : bf_lo(qh[e >> 1]);
        rotate_q_pair(x1, x2, a.q_prerot ? 0 : qpos, sm.freq[t0 + e], y1[e], y2[e]);  // position 0: identity
      }
      qf[2 * s] =
          as_bf16x8(u32x4{pack2(y1[0], y1[1]), pack2(y1[2], y1[3]), pack2(y1[4], y1[5]), pack2(y1[6], y1[7])});
      qf[2 * s + 1] =
          as_bf16x8(u32x4{pack2(y2[0], y2[1]), pack2(y2[2], y2[3]), pack2(y2[4], y2[5]), pack2(y2[6], y2[7])});
    }
  }
  if (LOCAL && wave == 0) {
#pragma unroll
    for (int s = 0; s < SP; ++s) {
      sm.qsave[s][0][lane] = qraw[s][0];
      sm.qsave[s][1][lane] = qraw[s][1];
    }
  }
  int qdelta = -1;  // record offset the fragments are rotated for (local-position keys; offsets are >= 0)
  __syncthreads();  // per-row table and saved Q complete

  f32x4 o[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) o[db] = f32x4{};
  float m2 = -INFINITY, lsum = 0.f;
  const float c = a.scale_log2;
  const float ab = ALIBI ? alibi_slope(head, a.hq, a.inv_freq, c) : 0.f;

  uint16_t* vw = sm.v[wave];
  // Transposing-read address of this lane in its V slice: row 16*(kq/2) + 4*(kq%2) + i/4 (+ 8 for the second
  // half), column 4*(i%4) (+ 16 per dimension block); i = lane % 16.
  const uint16_t* vlane = vw + (16 * (kq >> 1) + 4 * (kq & 1) + ((lane & 15) >> 2)) * S::VLD + 4 * (lane & 3);
  const float* cd0 = sm.csd + dec_row<D>(kappa(0, col));
  const float* cd1 = sm.csd + dec_row<D>(kappa(1, col));
  int buf = 0;
  while (have) {
    const int nvalid = min(kDecWaveKeys, it.cur.len - it.j0);
    const int b0 = it.cur.pos + it.j0;
    if (LOCAL && it.cur.pos != qdelta) {
      // New record: q' = R(q_pos - pos_offset) q, one rotation by the relative offset.  One lane per pair writes the
      // angle row to this wave's table (same-wave LDS ordering: written here, read just below).
      qdelta = it.cur.pos;
      if (lane < D / 2)
        *reinterpret_cast<float2*>(sm.csb[wave][0] + csb_idx<D>(lane)) =
            rope_cs((a.q_prerot ? 0 : qpos) - qdelta, sm.freq[lane]);
#pragma unroll
      for (int s = 0; s < SP; ++s) {
        float y1[8], y2[8];
        u32x4 ql, qh;
        pairs_of<IL>(sm.qsave[s][0][lane], sm.qsave[s][1][lane], ql, qh);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x1 = (e & 1) ? bf_hi(ql[e >> 1]) : bf_lo(ql[e >> 1]);
          const float x2 = (e & 1) ? bf_hi(qh[e >> 1]) : bf_lo(qh[e >> 1]);
          rotate_by(x1, x2, *reinterpret_cast<const float2*>(sm.csb[wave][0] + csb_idx<D>(32 * s + 8 * kq + e)),
                    y1[e], y2[e]);
        }
        qf[2 * s] =
            as_bf16x8(u32x4{pack2(y1[0], y1[1]), pack2(y1[2], y1[3]), pack2(y1[4], y1[5]), pack2(y1[6], y1[7])});
        qf[2 * s + 1] =
            as_bf16x8(u32x4{pack2(y2[0], y2[1]), pack2(y2[2], y2[3]), pack2(y2[4], y2[5]), pack2(y2[6], y2[7])});
      }
    }
    it.skip(4);
    const bool have_next = it.seek_strided(a.causal, qpos, 4);
    if (have_next) {
      dec_fetch<D, IL, NT>(nxt, k_ptr(a.k_pool, it.cur, g, it.j0, D), v_ptr(a.v_pool, it.cur, g, it.j0, D),
                   min(kDecWaveKeys, it.cur.len - it.j0), lane);
      if (ROT && lane < D / 2)
        *reinterpret_cast<float2*>(sm.csb[wave][buf ^ 1] + csb_idx<D>(lane)) =
            rope_cs(it.cur.pos + it.j0, sm.freq[lane]);
    }

    const int lim = min(nvalid, a.causal ? qpos - b0 + 1 : kDecWaveKeys);
    dec_tile<D, ROT, IL, ALIBI>(cur, vw, vlane, sm.csb[wave][buf], cd0, cd1, qf, o, m2, lsum, lim, c, lane, ab,
                                ab * (float)(b0 - qpos));
    cur = nxt;
    buf ^= 1;
    have = have_next;
  }

  // Merge the four waves' states through LDS (the V slices are free once every wave is here).
  float ltot = lsum + __shfl_xor(lsum, 16);
  ltot += __shfl_xor(ltot, 32);
  __syncthreads();
  float* macc = reinterpret_cast<float*>(sm.v[0]);  // [4][D][16]
  float* mm = macc + 4 * D * 16;                    // [4][16]
  float* ml = mm + 4 * 16;                          // [4][16]
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) macc[(wave * D + 16 * db + 4 * kq + i) * 16 + col] = o[db][i];
  if (kq == 0) {
    mm[wave * 16 + col] = m2;
    ml[wave * 16 + col] = ltot;
  }
  __syncthreads();
  for (int idx = tid; idx < 16 * (D / 4); idx += kThreads) {
    const int hc = idx & 15, d4 = idx >> 4;
    if (hc >= hcount) continue;
    float mw[4], mmax = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      mw[w] = mm[w * 16 + hc];
      mmax = fmaxf(mmax, mw[w]);
    }
    float l = 0.f;
    f32x4 acc = f32x4{};
    if (mmax != -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float sc = fast_exp2(mw[w] - mmax);
        l = fmaf(ml[w * 16 + hc], sc, l);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = fmaf(macc[(w * D + 4 * d4 + e) * 16 + hc], sc, acc[e]);
      }
    }
    const int hh = g * G + kDecodeHeadsPerGroup * hg + hc;
    // Normalised output and log-sum-exp: the final result, or with several splits this split's partial result.
    const int64_t orow = (int64_t)r * a.hq + hh;
    const int64_t wrow = (int64_t)split * a.total_q * a.hq + orow;
    uint16_t* dst = a.splits == 1 ? a.out + orow * D : a.ws_o + wrow * D;
    float* lse_dst = a.splits == 1 ? (a.lse ? a.lse + orow : nullptr) : a.ws_lse + wrow;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    *reinterpret_cast<u32x2*>(dst + 4 * d4) = u32x2{pack2(acc[0] * inv, acc[1] * inv), pack2(acc[2] * inv, acc[3] * inv)};
    if (lse_dst && d4 == 0) *lse_dst = l > 0.f ? (mmax + log2f(l)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Chunk-major shared decode: workgroup = (work item, KV head).  A work item is a run of stored keys (one or more
// ranges of records, read back to back) with up to 16 / G users (requests that read the run, each at its own
// offset); MFMA column c is the pair (user c / G, query head c % G).  The run's K / V are read once for all users.
// Key j of the run is at position pos_offset + j for a user.  Column c's query is rotated by its user's relative
// offset rel = q_pos - pos_offset and the keys are rotated by R(j) in registers (NoPE store), or used as stored
// with the query rotated by the record's own offset (local-position store, single-range items); key j is visible to
// the column iff j <= rel under the causal rule.  Waves take the run's 32-key tiles w, w + 4, ... with the next tile
// in flight, as in decode_kernel; tile t lies in range 32 t / range_keys (every range but the last holds a multiple
// of 32 keys).  Every (user, item) writes one partial result into its request's slot.
// ---------------------------------------------------------------------------------------------------------------
// K / V address of key j (within the run) of KV head g: range j / rk of the run, whose ranges are staged in LDS.
__device__ __forceinline__ void run_key(const lazy_shared_range_t* rg, int nr, int rk, int g, int j, int d,
                                        int64_t& koff, int64_t& voff) {
  const int r = nr == 1 ? 0 : min(j / rk, nr - 1);
  const int jr = j - r * rk + rg[r].key_begin;
  koff = rg[r].k_offset + ((int64_t)g * rg[r].k_stride + jr) * d;
  voff = rg[r].v_offset + ((int64_t)g * rg[r].v_stride + jr) * d;
}

template <int D, int KMI>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void decode_shared_kernel(
    SharedArgs a) {
  constexpr int KM = keys_of(KMI);
  constexpr bool IL = interleaved_of(KMI), ALIBI = KM == kKeysAlibi, NT = stream_of(KMI);
  __shared__ DecodeSmem<D> sm;
  __shared__ float ucs[16][DecodeSmem<D>::CSB];  // per user: cos/sin(rel theta_t) at csb_idx(t)
  __shared__ int uang[16];                         // per user: (q_pos, or 0 for pre-rotated queries) - pos_offset
  using S = DecodeSmem<D>;
  constexpr int SP = DecTile<D>::SP;
  constexpr bool ROT = KM == kKeysNope;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  __shared__ lazy_shared_range_t srg[LAZY_SHARED_MAX_RANGES];
  // Workgroup (item, KV head) = the logical id under the contiguous map of xcd_remap: XCD k takes the k-th eighth of
  // the item-major ids (one KV head's items in plan order), so the items of one run (a chunk with more users than an
  // item holds) run together on one XCD and read its keys through one L2.
  const int lid = uniform(xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y, gridDim.x,
                                    gridDim.y, false));
  const cptr<lazy_shared_item_t> item = as_const(a.items) + lid % gridDim.x;
  const int g = lid / gridDim.x;
  // Item fields come from the planner (lazy_shared_decode_validate checks a plan on the host).  The clamps keep
  // every LDS index in bounds whatever the item holds: the range table (at most LAZY_SHARED_MAX_RANGES entries) and
  // the per-user angle rows (at most floor(16 / G) users, one MFMA column per (user, query head)).
  const int G = a.group;
  const int rb = item->range_begin, nr = max(1, min(item->num_ranges, LAZY_SHARED_MAX_RANGES));
  const int rk = max(1, item->range_keys);
  const int u0 = item->user_begin, nu = max(0, min(item->num_users, 16 / G));
  if (nu == 0) return;  // no user: nothing to score or write (the whole workgroup leaves before any barrier)
  const cptr<lazy_shared_range_t> rgs = as_const(a.ranges) + rb;
  const int nk = (nr - 1) * rk + (rgs[nr - 1].key_end - rgs[nr - 1].key_begin);  // keys of the run
  if (tid < nr) srg[tid] = a.ranges[rb + tid];
  const int col = lane & 15, kq = lane >> 4;
  const int cu = col / G;
  const bool cvalid = cu < nu;
  const int cuser = cvalid ? cu : 0;
  const lazy_shared_user_t usr = a.users[u0 + cuser];
  const int rel = a.q_pos[usr.request] - usr.pos_offset;
  // The lane of each user's first column publishes its query angle offset, so that the per-user angle rows below
  // need no second round of user and position loads.
  if (wave == 0 && kq == 0 && cvalid && col % G == 0) uang[cu] = a.q_prerot ? -usr.pos_offset : rel;

  // Raw Q of this lane's column and the first tile's K / V before the tables (as in decode_kernel).
  u32x4 qraw[SP][2];
  {
    const uint16_t* qrow = a.q + ((int64_t)usr.request * a.hq + g * G + col % G) * D;
#pragma unroll
    for (int s = 0; s < SP; ++s) {
      qraw[s][0] = qraw[s][1] = u32x4{0, 0, 0, 0};
      if (cvalid) dec_k_pairs<D, IL, false>(qrow, s, kq, qraw[s][0], qraw[s][1]);
    }
  }
  const int ntiles = (nk + kDecWaveKeys - 1) / kDecWaveKeys;
  int tile = wave;
  DecTile<D> cur, nxt;
  if (tile < ntiles) {  // the first tile straight from the range table (the LDS copy is not ready yet)
    const int j0 = kDecWaveKeys * tile;
    const int r = nr == 1 ? 0 : min(j0 / rk, nr - 1);
    const int jr = j0 - r * rk + rgs[r].key_begin;
    dec_fetch<D, IL, NT>(cur, a.k_pool + rgs[r].k_offset + ((int64_t)g * rgs[r].k_stride + jr) * D,
                     a.v_pool + rgs[r].v_offset + ((int64_t)g * rgs[r].v_stride + jr) * D,
                     min(kDecWaveKeys, nk - j0), lane);
  }

  if (!ALIBI && tid < D / 2) sm.freq[tid] = theta_rev(tid, D, a.rope_log2_base, a.inv_freq);
  __syncthreads();
  if (ROT) {
    for (int e = tid; e < kDecWaveKeys * (D / 2); e += kThreads) {
      const int dr = e / (D / 2), t = e % (D / 2);
      *reinterpret_cast<float2*>(sm.csd + dec_row<D>(dr) + 2 * t) = rope_cs(dr, sm.freq[t]);
    }
    if (tile < ntiles && lane < D / 2)
      *reinterpret_cast<float2*>(sm.csb[wave][0] + csb_idx<D>(lane)) = rope_cs(kDecWaveKeys * tile, sm.freq[lane]);
  }
  // Per user: the query rotation q_pos - pos_offset (NoPE), or by the record's own offset (local-position keys are
  // encoded at their index in the record, key_begin for the run's first key).
  const int qrot_shift = KM == kKeysLocal ? rgs[0].key_begin : 0;
  for (int e = tid; e < (ALIBI ? 0 : nu * (D / 2)); e += kThreads) {
    const int u = e / (D / 2), t = e % (D / 2);
    *reinterpret_cast<float2*>(&ucs[u][csb_idx<D>(t)]) = rope_cs(uang[u] + qrot_shift, sm.freq[t]);
  }
  __syncthreads();

  // Q fragments: R(rel) q for this lane's column.
  bf16x8 qf[D / 32];
#pragma unroll
  for (int s = 0; s < SP; ++s) {
    float y1[8], y2[8];
    u32x4 ql, qh;
    pairs_of<IL>(qraw[s][0], qraw[s][1], ql, qh);
    if (ALIBI) {  // no rotation: the raw query
      qf[2 * s] = as_bf16x8(ql);
      qf[2 * s + 1] = as_bf16x8(qh);
      continue;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x1 = (e & 1) ? bf_hi(ql[e >> 1]) : bf_lo(ql[e >> 1]);
      const float x2 = (e & 1) ? bf_hi(qh[e >> 1]) : bf_lo(qh[e >> 1]);
      rotate_by(x1, x2, *reinterpret_cast<const float2*>(&ucs[cuser][csb_idx<D>(32 * s + 8 * kq + e)]), y1[e],
                y2[e]);
    }
    qf[2 * s] = as_bf16x8(u32x4{pack2(y1[0], y1[1]), pack2(y1[2], y1[3]), pack2(y1[4], y1[5]), pack2(y1[6], y1[7])});
    qf[2 * s + 1] =
        as_bf16x8(u32x4{pack2(y2[0], y2[1]), pack2(y2[2], y2[3]), pack2(y2[4], y2[5]), pack2(y2[6], y2[7])});
  }

  f32x4 o[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) o[db] = f32x4{};
  float m2 = -INFINITY, lsum = 0.f;
  const float c = a.scale_log2;
  const float ab = ALIBI ? alibi_slope(g * G + col % G, a.hq, a.inv_freq, c) : 0.f;
  uint16_t* vw = sm.v[wave];
  const uint16_t* vlane = vw + (16 * (kq >> 1) + 4 * (kq & 1) + ((lane & 15) >> 2)) * S::VLD + 4 * (lane & 3);
  const float* cd0 = sm.csd + dec_row<D>(kappa(0, col));
  const float* cd1 = sm.csd + dec_row<D>(kappa(1, col));
  int buf = 0;
  while (tile < ntiles) {
    const int j0 = kDecWaveKeys * tile;
    const int nvalid = min(kDecWaveKeys, nk - j0);
    const int next = tile + 4;
    if (next < ntiles) {
      const int j1 = kDecWaveKeys * next;
      int64_t k1, v1;
      run_key(srg, nr, rk, g, j1, D, k1, v1);
      dec_fetch<D, IL, NT>(nxt, a.k_pool + k1, a.v_pool + v1, min(kDecWaveKeys, nk - j1), lane);
      if (ROT && lane < D / 2)
        *reinterpret_cast<float2*>(sm.csb[wave][buf ^ 1] + csb_idx<D>(lane)) = rope_cs(j1, sm.freq[lane]);
    }
    const int lim = min(nvalid, a.causal ? rel - j0 + 1 : kDecWaveKeys);
    dec_tile<D, ROT, IL, ALIBI>(cur, vw, vlane, sm.csb[wave][buf], cd0, cd1, qf, o, m2, lsum, lim, c, lane, ab,
                                ab * (float)(j0 - rel));
    cur = nxt;
    buf ^= 1;
    tile = next;
  }

  // Merge the four waves' states through LDS, then one partial result per (user, query head).
  float ltot = lsum + __shfl_xor(lsum, 16);
  ltot += __shfl_xor(ltot, 32);
  __syncthreads();
  float* macc = reinterpret_cast<float*>(sm.v[0]);  // [4][D][16]
  float* mm = macc + 4 * D * 16;                    // [4][16]
  float* ml = mm + 4 * 16;                          // [4][16]
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) macc[(wave * D + 16 * db + 4 * kq + i) * 16 + col] = o[db][i];
  if (kq == 0) {
    mm[wave * 16 + col] = m2;
    ml[wave * 16 + col] = ltot;
  }
  __syncthreads();
  const int64_t rows = (int64_t)a.batch * a.hq;
  for (int idx = tid; idx < 16 * (D / 4); idx += kThreads) {
    const int hc = idx & 15, d4 = idx >> 4;
    if (hc / G >= nu) continue;
    float mw[4], mmax = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      mw[w] = mm[w * 16 + hc];
      mmax = fmaxf(mmax, mw[w]);
    }
    float l = 0.f;
    f32x4 acc = f32x4{};
    if (mmax != -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float sc = fast_exp2(mw[w] - mmax);
        l = fmaf(ml[w * 16 + hc], sc, l);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = fmaf(macc[(w * D + 4 * d4 + e) * 16 + hc], sc, acc[e]);
      }
    }
    const lazy_shared_user_t uu = a.users[u0 + hc / G];
    const int64_t wrow = (int64_t)uu.slot * rows + (int64_t)uu.request * a.hq + g * G + hc % G;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    *reinterpret_cast<u32x2*>(a.ws_o + wrow * D + 4 * d4) =
        u32x2{pack2(acc[0] * inv, acc[1] * inv), pack2(acc[2] * inv, acc[3] * inv)};
    if (d4 == 0) a.ws_lse[wrow] = l > 0.f ? (mmax + log2f(l)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Split-KV merge: per row, the splits' normalised outputs weighted by exp(lse_s - max lse), divided by the sum of
// the weights.  A row is served by CG x D / 8 lanes of one wave: lane (g, d8) loads 8 dims (16 bytes) of the
// splits g, g + CG, ... together with their log-sum-exps, U splits per memory round trip, and keeps a running
// maximum, weight sum and weighted sum (rescaled when the maximum grows); with CG > 1 the groups' states are then
// merged across lanes.  A merge of up to U x CG splits thus costs one memory round trip: CG = 1, U = 4 for up to 4
// splits; CG = 4 with U = 8 (32 per round trip) up to 32, U = 16 (64 per round trip) beyond.
// ---------------------------------------------------------------------------------------------------------------
template <int D, int CG, int U>
__global__ __launch_bounds__(kThreads) void combine_kernel(const uint16_t* __restrict__ part_o,
                                                           const float* __restrict__ part_lse, int splits, int rows,
                                                           const int32_t* __restrict__ slot_start, int hq,
                                                           uint16_t* __restrict__ out, float* __restrict__ lse) {
  constexpr int TPR = D / 8;
  constexpr int LPR = TPR * CG;        // lanes per row
  static_assert(LPR <= 64 && 64 % LPR == 0, "a row's lanes lie in one wave");
  const int row = blockIdx.x * (kThreads / LPR) + threadIdx.x / LPR;
  const int d8 = threadIdx.x % TPR;
  const int grp = (threadIdx.x / TPR) % CG;
  // Rows past the end take part in the shuffles with no memory access (the whole wave stays converged).
  const bool live = row < rows;
  // With slot_start (shared decode), row r * hq + h of request r merges that request's own slot count.
  if (live && slot_start) splits = slot_start[row / hq + 1] - slot_start[row / hq];
  float m = -INFINITY, den = 0.f, sum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (live) {
    for (int s0 = grp; s0 < splits; s0 += U * CG) {
      float ls[U];
      u32x4 v[U];
#pragma unroll
      for (int e = 0; e < U; ++e) {
        const int sp = s0 + e * CG;
        const int64_t w = (int64_t)(sp < splits ? sp : s0) * rows + row;
        ls[e] = sp < splits ? part_lse[w] : -INFINITY;
        v[e] = *reinterpret_cast<const u32x4*>(part_o + w * D + 8 * d8);
      }
      float mb = ls[0];
#pragma unroll
      for (int e = 1; e < U; ++e) mb = fmaxf(mb, ls[e]);
      if (mb == -INFINITY) continue;  // every split here is empty
      if (mb > m) {
        const float c = expf(m - mb);  // 0 while nothing has been added (m = -inf)
        den *= c;
#pragma unroll
        for (int k = 0; k < 8; ++k) sum[k] *= c;
        m = mb;
      }
#pragma unroll
      for (int e = 0; e < U; ++e) {
        if (ls[e] == -INFINITY) continue;  // an empty split contributes nothing, whatever its output holds
        const float sc = expf(ls[e] - m);
        den += sc;
#pragma unroll
        for (int k = 0; k < 8; ++k) sum[k] = fmaf((k & 1) ? bf_hi(v[e][k >> 1]) : bf_lo(v[e][k >> 1]), sc, sum[k]);
      }
    }
  }
#pragma unroll
  for (int off = TPR; off < LPR; off *= 2) {
    const float mo = __shfl_xor(m, off);
    const float mn = fmaxf(m, mo);
    const float c0 = m == -INFINITY ? 0.f : expf(m - mn), c1 = mo == -INFINITY ? 0.f : expf(mo - mn);
    den = den * c0 + __shfl_xor(den, off) * c1;
#pragma unroll
    for (int k = 0; k < 8; ++k) sum[k] = sum[k] * c0 + __shfl_xor(sum[k], off) * c1;
    m = mn;
  }
  if (!live || grp != 0) return;
  const float inv = den > 0.f ? 1.f / den : 0.f;
  *reinterpret_cast<u32x4*>(out + (int64_t)row * D + 8 * d8) =
      u32x4{pack2(sum[0] * inv, sum[1] * inv), pack2(sum[2] * inv, sum[3] * inv), pack2(sum[4] * inv, sum[5] * inv),
            pack2(sum[6] * inv, sum[7] * inv)};
  if (lse && d8 == 0) lse[row] = den > 0.f ? m + logf(den) : -INFINITY;
}

// ---------------------------------------------------------------------------------------------------------------
// Materialise-then-attend baseline.
// ---------------------------------------------------------------------------------------------------------------
// Plan: exclusive prefix sum of record lengths -> records describing the contiguous rotated copy.
__global__ __launch_bounds__(kThreads) void materialize_plan_kernel(const lazy_chunk_t* in, int n, int hkv, int d,
                                                                    lazy_chunk_t* out) {
  __shared__ int64_t scan[kThreads];
  const int tid = threadIdx.x;
  int64_t carry = 0;
  for (int base = 0; base < n; base += kThreads) {
    const int i = base + tid;
    const int64_t len = i < n ? in[i].len : 0;
    scan[tid] = len;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
      const int64_t add = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += add;
      __syncthreads();
    }
    if (i < n) {
      lazy_chunk_t rec = in[i];
      rec.k_offset = (scan[tid] - len + carry) * hkv * d;
      rec.k_stride = rec.len;
      out[i] = rec;
    }
    carry += scan[kThreads - 1];
    __syncthreads();
  }
}

// Rotate-and-copy: workgroup = (64-key sub-tile, KV head, record).  Same angle decomposition and rounding as the
// lazy loader, written back in the natural head-dimension order.
template <int D, bool LOCAL, bool IL>
__global__ __launch_bounds__(kThreads) void materialize_rotate_kernel(const uint16_t* __restrict__ k_pool,
                                                                      const lazy_chunk_t* __restrict__ in,
                                                                      const lazy_chunk_t* __restrict__ plan,
                                                                      double log2_base, const float* inv_freq,
                                                                      uint16_t* __restrict__ k_out) {
  constexpr int PP = D / 8, NV = PP / 8;
  __shared__ double freq[D / 2];
  __shared__ float2 cs[2][D / 2];  // base angles of rows 0..31 and 32..63 of this 64-key block
  const int tid = threadIdx.x;
  const Rec rc = load_rec(as_const(in) + blockIdx.z);
  const int g = blockIdx.y, j0 = blockIdx.x * kSub;
  if (j0 >= rc.len) return;
  if (tid < D / 2) freq[tid] = theta_rev(tid, D, log2_base, inv_freq);
  __syncthreads();
  // NoPE keys: base angles of the two 32-row halves (key j at rc.pos + j); local-position keys: the record offset.
  if (tid < D)
    cs[tid / (D / 2)][tid % (D / 2)] =
        rope_cs(LOCAL ? rc.pos : rc.pos + j0 + kAngleRows * (tid / (D / 2)), freq[tid % (D / 2)]);
  __syncthreads();
  const int row = tid >> 2, quarter = tid & 3;
  if (j0 + row >= rc.len) return;
  const uint16_t* src = k_ptr(k_pool, rc, g, j0 + row, D);
  uint16_t* dst = k_out + plan[blockIdx.z].k_offset + ((int64_t)g * rc.len + j0 + row) * D;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int t0 = quarter * PP + 8 * v;
    u32x4 wl, wh;
    if (IL) {
      deinterleave8(reinterpret_cast<const u32x4*>(src + 2 * t0)[0], reinterpret_cast<const u32x4*>(src + 2 * t0)[1],
                    wl, wh);
    } else {
      wl = *reinterpret_cast<const u32x4*>(src + t0);
      wh = *reinterpret_cast<const u32x4*>(src + D / 2 + t0);
    }
    float yl[8], yh[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x1 = (e & 1) ? bf_hi(wl[e >> 1]) : bf_lo(wl[e >> 1]);
      const float x2 = (e & 1) ? bf_hi(wh[e >> 1]) : bf_lo(wh[e >> 1]);
      if (LOCAL)
        rotate_by(x1, x2, cs[0][t0 + e], yl[e], yh[e]);
      else
        rotate_pair(x1, x2, cs[row / kAngleRows][t0 + e], rope_cs(row % kAngleRows, freq[t0 + e]), yl[e], yh[e]);
    }
    if (IL) {  // written back interleaved: pair t0 + e at elements 2 (t0 + e), 2 (t0 + e) + 1
      *reinterpret_cast<u32x4*>(dst + 2 * t0) =
          u32x4{pack2(yl[0], yh[0]), pack2(yl[1], yh[1]), pack2(yl[2], yh[2]), pack2(yl[3], yh[3])};
      *reinterpret_cast<u32x4*>(dst + 2 * t0 + 8) =
          u32x4{pack2(yl[4], yh[4]), pack2(yl[5], yh[5]), pack2(yl[6], yh[6]), pack2(yl[7], yh[7])};
    } else {
      *reinterpret_cast<u32x4*>(dst + t0) =
          u32x4{pack2(yl[0], yl[1]), pack2(yl[2], yl[3]), pack2(yl[4], yl[5]), pack2(yl[6], yl[7])};
      *reinterpret_cast<u32x4*>(dst + D / 2 + t0) =
          u32x4{pack2(yh[0], yh[1]), pack2(yh[2], yh[3]), pack2(yh[4], yh[5]), pack2(yh[6], yh[7])};
    }
  }
}

// 256-row prefill workgroups: eight waves x one 32-row block, or four waves x two blocks.
#ifndef LAZY_PREFILL_BIG_WAVES
#define LAZY_PREFILL_BIG_WAVES 8
#endif
template <int D, int KM>
hipError_t prefill_d(const AttnArgs& a, hipStream_t st) {
  const dim3 grid(a.q_tiles, a.hkv, a.batch * a.splits);
  if constexpr (D == 128) {
    if (a.row_blocks == 2) {
      hipLaunchKernelGGL((prefill_kernel<D, KM, LAZY_PREFILL_BIG_WAVES, 2, 8 / LAZY_PREFILL_BIG_WAVES>), grid,
                         dim3(64 * LAZY_PREFILL_BIG_WAVES), 0, st, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((prefill_kernel<D, KM, 4, 1, 1>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <int D, int KM>
hipError_t decode_d(const AttnArgs& a, hipStream_t st) {
  const dim3 grid(a.splits, a.hkv * a.head_groups, a.batch);
  if (a.stream_kv)
    hipLaunchKernelGGL((decode_kernel<D, KM | kStreamKV>), grid, dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((decode_kernel<D, KM>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

int key_mode(const AttnArgs& a, bool rotate_k) {
  if (a.alibi) return kKeysAlibi;
  return (!rotate_k ? kKeysPlain : a.local_keys ? kKeysLocal : kKeysNope) | (a.interleaved ? kInterleaved : 0);
}

template <int D>
hipError_t prefill_dk(const AttnArgs& a, int km, hipStream_t st) {
  switch (km) {
    case kKeysPlain: return prefill_d<D, kKeysPlain>(a, st);
    case kKeysNope: return prefill_d<D, kKeysNope>(a, st);
    case kKeysLocal: return prefill_d<D, kKeysLocal>(a, st);
    case kKeysPlain | kInterleaved: return prefill_d<D, kKeysPlain | kInterleaved>(a, st);
    case kKeysNope | kInterleaved: return prefill_d<D, kKeysNope | kInterleaved>(a, st);
    case kKeysAlibi: return prefill_d<D, kKeysAlibi>(a, st);
    default: return prefill_d<D, kKeysLocal | kInterleaved>(a, st);
  }
}
template <int D>
hipError_t decode_dk(const AttnArgs& a, int km, hipStream_t st) {
  switch (km) {
    case kKeysPlain: return decode_d<D, kKeysPlain>(a, st);
    case kKeysNope: return decode_d<D, kKeysNope>(a, st);
    case kKeysLocal: return decode_d<D, kKeysLocal>(a, st);
    case kKeysPlain | kInterleaved: return decode_d<D, kKeysPlain | kInterleaved>(a, st);
    case kKeysNope | kInterleaved: return decode_d<D, kKeysNope | kInterleaved>(a, st);
    case kKeysAlibi: return decode_d<D, kKeysAlibi>(a, st);
    default: return decode_d<D, kKeysLocal | kInterleaved>(a, st);
  }
}
template <int D, int NT>
void shared_dk_nt(const SharedArgs& a, int km, dim3 grid, hipStream_t st) {
  switch (km) {
    case kKeysAlibi:
      hipLaunchKernelGGL((decode_shared_kernel<D, kKeysAlibi | NT>), grid, dim3(kThreads), 0, st, a);
      break;
    case kKeysNope: hipLaunchKernelGGL((decode_shared_kernel<D, kKeysNope | NT>), grid, dim3(kThreads), 0, st, a); break;
    case kKeysLocal:
      hipLaunchKernelGGL((decode_shared_kernel<D, kKeysLocal | NT>), grid, dim3(kThreads), 0, st, a);
      break;
    case kKeysNope | kInterleaved:
      hipLaunchKernelGGL((decode_shared_kernel<D, kKeysNope | kInterleaved | NT>), grid, dim3(kThreads), 0, st, a);
      break;
    default:
      hipLaunchKernelGGL((decode_shared_kernel<D, kKeysLocal | kInterleaved | NT>), grid, dim3(kThreads), 0, st, a);
  }
}
template <int D>
void shared_dk(const SharedArgs& a, dim3 grid, hipStream_t st) {
  const int km = a.alibi ? kKeysAlibi : (a.local_keys ? kKeysLocal : kKeysNope) | (a.interleaved ? kInterleaved : 0);
  if (a.stream_kv)
    shared_dk_nt<D, kStreamKV>(a, km, grid, st);
  else
    shared_dk_nt<D, 0>(a, km, grid, st);
}
template <int D>
void materialize_dk(bool local, bool il, dim3 grid, hipStream_t st, const uint16_t* k_pool, const lazy_chunk_t* in,
                    const lazy_chunk_t* plan, double log2_base, const float* inv_freq, uint16_t* k_out) {
  if (local) {
    if (il)
      hipLaunchKernelGGL((materialize_rotate_kernel<D, true, true>), grid, dim3(kThreads), 0, st, k_pool, in, plan,
                         log2_base, inv_freq, k_out);
    else
      hipLaunchKernelGGL((materialize_rotate_kernel<D, true, false>), grid, dim3(kThreads), 0, st, k_pool, in, plan,
                         log2_base, inv_freq, k_out);
  } else {
    if (il)
      hipLaunchKernelGGL((materialize_rotate_kernel<D, false, true>), grid, dim3(kThreads), 0, st, k_pool, in, plan,
                         log2_base, inv_freq, k_out);
    else
      hipLaunchKernelGGL((materialize_rotate_kernel<D, false, false>), grid, dim3(kThreads), 0, st, k_pool, in, plan,
                         log2_base, inv_freq, k_out);
  }
}

template <int D, int CG, int U>
hipError_t combine_d(const uint16_t* part_o, const float* part_lse, int splits, int rows, const int32_t* slot_start,
                     int hq, uint16_t* out, float* lse, hipStream_t st) {
  constexpr int per_block = kThreads / (D / 8 * CG);
  const dim3 grid((rows + per_block - 1) / per_block);
  hipLaunchKernelGGL((combine_kernel<D, CG, U>), grid, dim3(kThreads), 0, st, part_o, part_lse, splits, rows,
                     slot_start, hq, out, lse);
  return hipGetLastError();
}

// splits: the (largest) number of partial results per row.
hipError_t combine_dispatch(const uint16_t* part_o, const float* part_lse, int splits, int rows,
                            const int32_t* slot_start, int hq, int head_dim, uint16_t* out, float* lse,
                            hipStream_t st) {
  if (head_dim == 128) {
    if (splits <= 4) return combine_d<128, 1, 4>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
    if (splits <= 32) return combine_d<128, 4, 8>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
    return combine_d<128, 4, 16>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
  }
  if (splits <= 4) return combine_d<64, 1, 4>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
  if (splits <= 32) return combine_d<64, 4, 8>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
  return combine_d<64, 4, 16>(part_o, part_lse, splits, rows, slot_start, hq, out, lse, st);
}

}  // namespace

// Split-KV partial results of lazy_attn_decode_noalloc: a fixed device array that every call on a device shares,
// for callers that cannot allocate.  Each device holds its own copy for the life of the process.  Host code never
// uses this name as an address: its device address comes from hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) unsigned char scratch[LAZY_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(int device, void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* per_device[kMaxDevices] = {};
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!per_device[device]) {
    // The calling thread's current device is `device` (checked by the caller): the address is that device's copy.
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    per_device[device] = p;
  }
  *ptr = per_device[device];
  return hipSuccess;
}

hipError_t launch_combine(const uint16_t* part_o, const float* part_lse, int splits, int rows, int head_dim,
                          uint16_t* out, float* lse, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  return combine_dispatch(part_o, part_lse, splits, rows, nullptr, 1, head_dim, out, lse, st);
}

hipError_t launch_prefill(const AttnArgs& a, int head_dim, bool rotate_k, hipStream_t st) {
  const int km = key_mode(a, rotate_k);
  const hipError_t e = head_dim == 128 ? prefill_dk<128>(a, km, st) : prefill_dk<64>(a, km, st);
  if (e != hipSuccess || a.splits == 1) return e;
  return launch_combine(a.ws_o, a.ws_lse, a.splits, a.total_q * a.hq, head_dim, a.out, a.lse, st);
}

hipError_t launch_decode(const AttnArgs& a, int head_dim, bool rotate_k, hipStream_t st) {
  const int km = key_mode(a, rotate_k);
  const hipError_t e = head_dim == 128 ? decode_dk<128>(a, km, st) : decode_dk<64>(a, km, st);
  if (e != hipSuccess || a.splits == 1) return e;
  return launch_combine(a.ws_o, a.ws_lse, a.splits, a.total_q * a.hq, head_dim, a.out, a.lse, st);
}

hipError_t launch_decode_shared(const SharedArgs& a, int num_items, int max_slots, const int32_t* slot_start,
                                int head_dim, uint16_t* out, float* lse, hipStream_t st) {
  const int rows = a.batch * a.hq;
  if (num_items > 0) {
    const dim3 grid(num_items, a.hkv);
    if (head_dim == 128)
      shared_dk<128>(a, grid, st);
    else
      shared_dk<64>(a, grid, st);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // Ragged merge of every request's slots (a request without slots gets out = 0, lse = -inf).
  return combine_dispatch(a.ws_o, a.ws_lse, max_slots, rows, slot_start, a.hq, head_dim, out, lse, st);
}

hipError_t launch_materialize(const uint16_t* k_pool, const lazy_chunk_t* chunks, int num_records,
                              int max_chunk_len, int hkv, int head_dim, double rope_log2_base, const float* inv_freq,
                              bool local_keys, bool interleaved, uint16_t* k_out, lazy_chunk_t* chunks_out,
                              hipStream_t st) {
  if (num_records <= 0) return hipSuccess;
  hipLaunchKernelGGL(materialize_plan_kernel, dim3(1), dim3(kThreads), 0, st, chunks, num_records, hkv, head_dim,
                     chunks_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_chunk_len <= 0) return e;
  const dim3 grid((max_chunk_len + kSub - 1) / kSub, hkv, num_records);
  if (head_dim == 128)
    materialize_dk<128>(local_keys, interleaved, grid, st, k_pool, chunks, chunks_out, rope_log2_base, inv_freq,
                        k_out);
  else
    materialize_dk<64>(local_keys, interleaved, grid, st, k_pool, chunks, chunks_out, rope_log2_base, inv_freq,
                       k_out);
  return hipGetLastError();
}

}  // namespace lazy
