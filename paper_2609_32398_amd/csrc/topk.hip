// Router Top-K, signature packing and the co-occurrence Gram of the DO-loss
// path, in one pass over the scores.
//
// Paper: Sec. 3.1.1, Eq. (1) -- f_it = 1 iff expert i is in the Top-K of
// token t; the binary load signature F_i collects f_it over the batch.
// Sec. 3.1.3, Eq. (6) and App. C.3 -- ||F_i - F_j||_1 = c_ii + c_jj - 2 c_ij
// with c_ij = sum_t f_it f_jt, which is what the Gram part accumulates.
//
// Work layout.  A block of 8 wavefronts owns 8 consecutive signature words
// (512 output bit positions) per step; lane l of wave w ranks token
// 64*(word) + l - tok_off.  Score rows stream through LDS in 128-byte column
// chunks so the global loads are fully coalesced; the next chunk's loads are
// issued before the current chunk is ranked, so each wave keeps one chunk in
// flight at all times.  The 8 signature words of a step land in an LDS tile
// (double-buffered) from which, during the next step, the block writes them
// out and feeds the Gram.  Signatures are stored unit-major (sig_off): a
// step's 8 words of every expert are one contiguous block of E * 64 bytes.
//
// Exact Top-K with composite 32-bit keys.  Each element becomes one signed
// integer whose high bits order the score and whose low byte is (255 - expert
// index), so larger keys rank first and equal scores fall to the lower index.
// "Positive" keys use the raw bit pattern (one instruction, exact whenever the
// k-th score is a positive number); "general" keys first map the pattern to
// an order-preserving integer (exact for all non-NaN values except that -0
// sorts one step below +0).  An fp32 wave starts with positive keys and
// switches to general keys for the rest of its tiles after meeting a
// non-positive threshold; bf16 waves use general keys throughout.  bf16 keys keep all 16 value bits; fp32 keys keep 24, so a token
// whose k-th and (k+1)-th keys share a 24-bit bucket is settled by the whole
// wave from the full values of that bucket.  A token whose threshold lands on
// +-0, +-inf or NaN, or is not positive under positive keys, is re-ranked by
// an exact per-lane fallback on 64-bit keys.
//
// Gram.  Default: scaled fp4 (e2m1) MFMA, v_mfma_scale_f32_32x32x64_f8f6f4 at
// 256 experts and v_mfma_scale_f32_16x16x128_f8f6f4 below, on operands
// expanded from the signature words (one nibble per token, 0.5 or 0, block
// scale 2^1 on both sides so that every co-occurrence adds exactly 1.0); up
// to five expert tile pairs per wave, fp32 accumulators in registers, exact
// while a count stays below 2^24 (a block flushes at the latest every 32,767
// units of 512 tokens).  Alternative (do_set_option DO_OPT_GRAM = 1): VALU
// popcount(a & b) on 4x4 micro-tiles per thread.  Either way a block adds its
// integer partial counts into the accumulator matrix when the layer changes
// and at the end (order-independent).
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <mutex>

#include <hip/hip_ext.h>

#include "common.h"

namespace dol {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef short v2s __attribute__((ext_vector_type(2)));

// Per wave, two 8 KiB stage buffers of 64 rows x 128 bytes.  Piece q of row r
// lives at slot q ^ swz(r), swz(r) = (r & 7) ^ ((r >> 3) & 1): the per-lane row
// reads are then bank-conflict free and each direct-to-LDS load instruction
// still reads whole 128-byte row segments.
constexpr int kChunkBytes = 64 * 128;
constexpr int kStageBytes = kFusedWaves * 2 * kChunkBytes;

__device__ __forceinline__ int row_swizzle(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// The signature word of expert e in slot s of the bit tile lives at index
// e ^ bt_swz(s): the 8 words of one expert then sit in 8 different banks
// (the signature output reads them together), and 4-aligned groups and
// 32-expert tiles stay intact for the Gram readers.
__device__ __forceinline__ int bt_swz(int s) { return (s & 7) << 2; }

// Cache policy of the score loads: non-temporal (the "slc" bit, nt on gfx950), so
// the read-once stream ages out of L2 before the partially written signature
// lines, which then merge there into whole lines before eviction.
constexpr int kStreamPolicy = 2;
// Fourth word of a raw buffer resource on gfx9-family GPUs (no format
// conversion, no swizzle; offsets in bytes).
constexpr int kBufWord3 = 0x00020000;
// Units of signature stores held in registers (see batch_flush), and the
// (expert, word pair) items a lane holds per unit: 4 * E/8 items per wave.
template <int EPW>
struct StoreBatch {
  static constexpr int kUnits = EPW > 128 ? 4 : 2;
  static constexpr int kItems = EPW > 128 ? 2 : 1;
};

// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left at their maxima)
#define DOL_WAIT_VMEM() __builtin_amdgcn_s_waitcnt(0x0F70)

constexpr int kGramNone = 0, kGramPopc = 1, kGramMfma = 2;

constexpr int kCompPosInf = 0x7F800000;          // key >= this: +inf or NaN
constexpr int kCompNegInfMax = (int)0x807FFFFF;  // general key <= this: -inf or NaN

template <typename T>
struct Traits;
template <>
struct Traits<float> {
  static constexpr int kVec = 4;                       // elements per 16-byte vector
  static constexpr bool kExact = false;                // 24 value bits kept
  static constexpr int kPosMin = 0x100;                // positive keys: threshold must be >= this
  static constexpr int kZeroLo = -256, kZeroHi = 255;  // general keys of the -0 / +0 buckets
};
template <>
struct Traits<uint16_t> {
  static constexpr int kVec = 8;
  static constexpr bool kExact = true;
  static constexpr int kPosMin = 0x10000;
  static constexpr int kZeroLo = -65536, kZeroHi = 65535;
};

// Median of three in one instruction (the compiler does not form it from
// min/max of non-constant operands).
__device__ __forceinline__ int med3(int a, int b, int c) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Insert key x into the descending list top[0..7], dropping the smallest of
// the nine.  New entry i is x clamped to [old top[i], old top[i-1]].  With
// TRACK, rej <- max(rej, dropped key), i.e. the running 9th largest, which is
// again a clamp because rej <= top[7].
template <bool TRACK>
__device__ __forceinline__ void insert8(int (&top)[8], int x, int& rej) {
  if (TRACK) rej = med3(rej, top[7], x);
#pragma unroll
  for (int i = 7; i > 0; --i) top[i] = med3(top[i], top[i - 1], x);
  top[0] = max(top[0], x);
}

// The index part of the composite keys: byte b of word w is 255 - (4w + b),
// the complemented expert index of expert 4w + b.  A chunk's index bytes are
// read with one scalar load and each key takes its byte with one v_perm_b32,
// so building a key costs no scalar instruction for its index constant.
struct IdxTab {
  uint32_t w[kFastMaxE / 4];
};
constexpr IdxTab make_idx_tab() {
  IdxTab t{};
  for (int i = 0; i < kFastMaxE / 4; ++i) {
    uint32_t v = 0;
    for (int b = 0; b < 4; ++b) v |= (uint32_t)(255 - (4 * i + b)) << (8 * b);
    t.w[i] = v;
  }
  return t;
}
__constant__ IdxTab kIdxTab = make_idx_tab();

// v_perm_b32: byte i of the result is byte sel.byte[i] of {x (bytes 4-7),
// sidx (bytes 0-3)}, 12 selects 0x00.  sidx is a scalar (the index bytes),
// sel a loop-invariant VGPR.
__device__ __forceinline__ uint32_t perm(uint32_t x, uint32_t sidx, uint32_t sel) {
  uint32_t r;
  asm("v_perm_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(sidx), "v"(sel));
  return r;
}

// Byte selectors of the composite keys (VGPRs set once per kernel).
//   f32[j]: [index byte j, x.b1, x.b2, x.b3]                 -> value bits 8..31, index
//   lo[j]:  [index byte j, 0, x.b0, x.b1] (bf16 in the low half)
//   hi[j]:  [index byte j, 0, x.b2, x.b3] (bf16 in the high half)
struct KeySel {
  uint32_t f32[4];
  uint32_t lo[2];  // index bytes 0 and 2
  uint32_t hi[2];  // index bytes 1 and 3
};

// Composite keys.  idx: scalar holding the index bytes of 4 consecutive experts.
template <bool GEN>
__device__ __forceinline__ int key_f32(uint32_t u, uint32_t idx, uint32_t sel) {
  if (GEN) u ^= (uint32_t)((int32_t)u >> 31) & 0x7FFFFF00u;
  return (int)perm(u, idx, sel);
}

// Two bf16 scores packed in x (the even expert in the low half), their index
// bytes in bytes 2h and 2h + 1 of idx.
template <bool GEN>
__device__ __forceinline__ void key_bf16x2(uint32_t x, uint32_t idx, int h, const KeySel& ks, int& lo, int& hi) {
  if (GEN) {
    const v2s s = __builtin_bit_cast(v2s, x) >> (short)15;
    x ^= __builtin_bit_cast(uint32_t, s) & 0x7FFF7FFFu;
  }
  lo = (int)perm(x, idx, ks.lo[h]);
  hi = (int)perm(x, idx, ks.hi[h]);
}

// Rank one staged 128-byte chunk (vectors cv0..cv0+7 of the lane's row) into top/rej.
template <typename T, bool GEN>
__device__ __forceinline__ void rank_chunk(const unsigned char* sbuf, int lane, int cv0, const KeySel& ks,
                                           int (&top)[8], int& rej) {
  const unsigned char* row = sbuf + lane * 128;
  const int sw = row_swizzle(lane);
  auto piece = [&](int q) { return *reinterpret_cast<const v4u*>(row + ((q ^ sw) << 4)); };
  // index bytes of the chunk's experts (one scalar load: the chunk index is uniform)
  constexpr int kWords = Traits<T>::kVec * 8 / 4;
  const uint32_t* iw = kIdxTab.w + cv0 * (Traits<T>::kVec / 4);
  uint32_t idx[kWords];
#pragma unroll
  for (int i = 0; i < kWords; ++i) idx[i] = __builtin_amdgcn_readfirstlane(iw[i]);
  if (Traits<T>::kVec == 4) {
    // the next piece's read is issued before the current piece is ranked, and
    // a piece's four keys are built before any is inserted
    v4u x = piece(0);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const v4u xn = piece(q + 1 < 8 ? q + 1 : q);
      int g[4];
      g[0] = key_f32<GEN>(x.x, idx[q], ks.f32[0]);
      g[1] = key_f32<GEN>(x.y, idx[q], ks.f32[1]);
      g[2] = key_f32<GEN>(x.z, idx[q], ks.f32[2]);
      g[3] = key_f32<GEN>(x.w, idx[q], ks.f32[3]);
#pragma unroll
      for (int i = 0; i < 4; ++i) insert8<!Traits<T>::kExact>(top, g[i], rej);
      x = xn;
    }
  } else {
    // all eight reads issued up front: their latency overlaps the ranking of
    // the earlier pieces instead of stalling the wave every two pieces
    v4u xs[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) xs[v] = piece(v);
    __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the ranking
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      int g[8];
      const v4u x = xs[v];
      key_bf16x2<GEN>(x.x, idx[2 * v], 0, ks, g[0], g[1]);
      key_bf16x2<GEN>(x.y, idx[2 * v], 1, ks, g[2], g[3]);
      key_bf16x2<GEN>(x.z, idx[2 * v + 1], 0, ks, g[4], g[5]);
      key_bf16x2<GEN>(x.w, idx[2 * v + 1], 1, ks, g[6], g[7]);
#pragma unroll
      for (int i = 0; i < 8; ++i) insert8<false>(top, g[i], rej);
    }
  }
}

template <typename T>
__device__ __forceinline__ uint32_t elem_bits(const T* row, int e);
template <>
__device__ __forceinline__ uint32_t elem_bits<float>(const float* row, int e) {
  return reinterpret_cast<const uint32_t*>(row)[e];
}
template <>
__device__ __forceinline__ uint32_t elem_bits<uint16_t>(const uint16_t* row, int e) {
  return (uint32_t)row[e] << 16;
}

// Exact order key: larger = ranks first.  NaN -> 0 (below -inf), -0 -> +0.
__device__ __forceinline__ uint32_t exact_key(uint32_t u) {
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ u64 exact_key64(uint32_t bits, int e) {
  return ((u64)exact_key(bits) << 32) | (u64)(0xFFFFFFFFu - (uint32_t)e);
}

// Exact Top-k (k <= KL) of one row in a single pass: insertion of unique
// 64-bit keys (value key, then the complemented index) into a sorted list of
// KL entries.  The row is read 16 elements at a time so that the loads of a
// batch are in flight together instead of one memory round trip per element.
template <typename T, int KL>
__device__ void exact_topk_list_lane(const T* row, int E, int k, u64* bt, int swz, u64 bit) {
  u64 lst[KL];
#pragma unroll
  for (int i = 0; i < KL; ++i) lst[i] = 0ull;  // every real key is > 0
  for (int e0 = 0; e0 < E; e0 += 16) {
    // all 16 loads issued unconditionally (positions past E re-read element
    // E - 1 and are skipped below): a branch per load would make each load
    // wait for its data before the next one is issued
    uint32_t v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = elem_bits<T>(row, min(e0 + j, E - 1));
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (e0 + j >= E) break;
      const u64 key = exact_key64(v[j], e0 + j);
      if (key <= lst[KL - 1]) continue;
#pragma unroll
      for (int i = KL - 1; i > 0; --i) lst[i] = max(lst[i], min(lst[i - 1], key));
      lst[0] = max(lst[0], key);
    }
  }
#pragma unroll
  for (int i = 0; i < KL; ++i)
    if (i < k) atomicOr(&bt[(int)(0xFFFFFFFFu - (uint32_t)(lst[i] & 0xFFFFFFFFull)) ^ swz], bit);
}

// Exact Top-k for any k: k selection passes, each taking the largest key
// below the previous one (rows read 16 elements per batch).
template <typename T>
__device__ void exact_topk_passes_lane(const T* row, int E, int k, u64* bt, int swz, u64 bit) {
  u64 prev = ~0ull;
  for (int r = 0; r < k; ++r) {
    u64 best = 0;
    for (int e0 = 0; e0 < E; e0 += 16) {
      uint32_t v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] = elem_bits<T>(row, min(e0 + j, E - 1));  // unconditional, as above
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if (e0 + j >= E) break;
        const u64 key = exact_key64(v[j], e0 + j);
        if (key < prev && key > best) best = key;
      }
    }
    atomicOr(&bt[(int)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFull)) ^ swz], bit);
    prev = best;
  }
}

// Exact selection of one lane's token (the paths above), kept out of line:
// inlined into the Top-K kernel, its registers and live ranges cost the
// kernel's common path spills although it runs for few tokens.
template <typename T>
__device__ __attribute__((noinline)) void exact_select_lane(const T* row, int E, int k, u64* bt, int swz, u64 bit) {
  if (k <= 8)
    exact_topk_list_lane<T, 8>(row, E, k, bt, swz, bit);
  else if (k <= 16)
    exact_topk_list_lane<T, 16>(row, E, k, bt, swz, bit);
  else
    exact_topk_passes_lane<T>(row, E, k, bt, swz, bit);
}

// Tokens whose k-th and (k+1)-th fp32 keys share a 24-bit value bucket
// (bit L of tie_mask; B = bucket of sk, need = picks still missing; row0 =
// the row of lane 0's token; swz = the wave's bit-tile swizzle).  For each,
// the whole wave loads the token's row (16 bytes per lane, one round trip),
// marks the elements of the bucket with a 16-bit sub-key (low 8 value bits,
// then the complemented index) and takes the `need` largest across the wave:
// by full value, ties to the lower index.  Out of line for the same reason as
// exact_select_lane; every lane of the wave must be active.
__device__ __attribute__((noinline)) void resolve_ties(u64 tie_mask, int sk_v, int need_v, bool gen_keys, u64* mybt,
                                                      const unsigned char* row0, int rowB, int swz) {
  const int lane = (int)__lane_id();
  while (tie_mask != 0ull) {
    const int L = __builtin_ctzll(tie_mask);
    tie_mask &= tie_mask - 1;
    const int B = __builtin_amdgcn_readlane(sk_v, L) >> 8;
    const int need_l = __builtin_amdgcn_readlane(need_v, L);
    const unsigned char* row = row0 + (int64_t)L * rowB;
    const bool has = lane * 16 < rowB;
    const v4u x = has ? *reinterpret_cast<const v4u*>(row + lane * 16) : v4u{0u, 0u, 0u, 0u};
    int sub[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t u = x[j];
      if (gen_keys) u ^= (uint32_t)((int32_t)u >> 31) & 0x7FFFFFFFu;
      const int e = lane * 4 + j;
      sub[j] = (has && ((int32_t)u >> 8) == B) ? (int)(((u & 0xFFu) << 8) | (uint32_t)(255 - e)) : -1;
    }
    for (int r = 0; r < need_l; ++r) {
      int m = max(max(sub[0], sub[1]), max(sub[2], sub[3]));
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) m = max(m, __shfl_xor(m, d));
      if (m < 0) break;
      if (lane == 0) atomicOr(&mybt[(255 - (m & 255)) ^ swz], 1ull << L);
#pragma unroll
      for (int j = 0; j < 4; ++j) sub[j] = (sub[j] == m) ? -1 : sub[j];
    }
  }
}

// ---------------------------------------------------------------------------
// Popcount Gram held in registers across a block: thread `tid` owns up to MTQ
// 4x4 micro-tiles (a, b), a <= b, of the upper triangle of c.
// ---------------------------------------------------------------------------
template <int EP, int NTHREADS, bool ON>
struct PopcGram {
  static constexpr int NB = EP / 4;
  static constexpr int NMT = NB * (NB + 1) / 2;
  static constexpr int MTQ = ON ? (NMT + NTHREADS - 1) / NTHREADS : 1;
  uint32_t acc[MTQ][16];
  int ra[MTQ], rb[MTQ];

  __device__ __forceinline__ void init(int tid, int E) {
#pragma unroll
    for (int q = 0; q < MTQ; ++q) {
      int mt = tid + q * NTHREADS;
      int a = -1, b = -1;
      if (ON && mt < NMT) {
        a = 0;
        while (mt >= NB - a) {
          mt -= NB - a;
          ++a;
        }
        b = a + mt;
        if (4 * b >= E) a = b = -1;  // b >= a, so this also drops blocks with a >= E/4
      }
      ra[q] = a;
      rb[q] = b;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[q][i] = 0;
    }
  }

  // bt: signature words per expert, slot-major with `stride` words per slot; slots [s0, s1)
  __device__ __forceinline__ void accumulate(const u64* bt, int s0, int s1, int stride) {
    for (int s = s0; s < s1; ++s) {
      const u64* w = bt + s * stride;
#pragma unroll
      for (int q = 0; q < MTQ; ++q) {
        if (ra[q] < 0) continue;
        const int ga = (4 * ra[q]) ^ bt_swz(s), gb = (4 * rb[q]) ^ bt_swz(s);
        const ulonglong2 a01 = *reinterpret_cast<const ulonglong2*>(w + ga);
        const ulonglong2 a23 = *reinterpret_cast<const ulonglong2*>(w + ga + 2);
        const ulonglong2 b01 = *reinterpret_cast<const ulonglong2*>(w + gb);
        const ulonglong2 b23 = *reinterpret_cast<const ulonglong2*>(w + gb + 2);
        const u64 A[4] = {a01.x, a01.y, a23.x, a23.y};
        const u64 B[4] = {b01.x, b01.y, b23.x, b23.y};
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[q][i * 4 + j] += (uint32_t)__popcll(A[i] & B[j]);
      }
    }
  }

  __device__ __forceinline__ void flush(uint32_t* c, int E) {
#pragma unroll
    for (int q = 0; q < MTQ; ++q) {
      if (ra[q] < 0) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int gi = 4 * ra[q] + i, gj = 4 * rb[q] + j;
          const uint32_t v = acc[q][i * 4 + j];
          if (gi <= gj && gj < E && v) atomicAdd(&c[(int64_t)gi * E + gj], v);
        }
    }
  }
};

// ---------------------------------------------------------------------------
// MFMA Gram.  The upper triangle of c is split into T x T tile pairs (T <= 8
// tiles of TS experts).  Every wave runs the same code: it owns four local
// tiles L0..L3 and five pair slots (L0,L0) (L0,L1) (L1,L2) (L0,L2) (L0,L3),
// each enabled by a bit of `act`.  For T = 8 wave w takes L = (w, w+1, w+3,
// w+4) mod 8: slot 0..3 then hold the tile pairs at cyclic distance 0, 1, 2
// and 3 (8 each), and slot 4 of waves 0-3 those at distance 4 (4) -- every
// one of the 36 pairs exactly once, with 3-4 distinct tiles per wave.
// ---------------------------------------------------------------------------
constexpr int kGP = 5;  // pair slots per wave
__device__ __forceinline__ int slot_a(int p) { return p == 2 ? 1 : 0; }
__device__ __forceinline__ int slot_b(int p) { return p == 0 ? 0 : p == 1 ? 1 : p == 4 ? 3 : 2; }

struct WaveTiles {
  int tile[4];
  int act;  // bit p: slot p accumulates a pair of its own
};

__device__ __forceinline__ WaveTiles wave_tiles(int T, int w) {
  WaveTiles t;
  if (T == 8) {
    t.tile[0] = w;
    t.tile[1] = (w + 1) & 7;
    t.tile[2] = (w + 3) & 7;
    t.tile[3] = (w + 4) & 7;
    t.act = 0xF | (w < 4 ? 0x10 : 0);
  } else if (T == 4) {  // distances 0, 1 (slots 0, 1) and 2 (slot 3, waves 0-1)
    t.tile[0] = w & 3;
    t.tile[1] = (w + 1) & 3;
    t.tile[2] = (w + 2) & 3;
    t.tile[3] = w & 3;
    t.act = w < 4 ? (0x3 | (w < 2 ? 0x8 : 0)) : 0;
  } else if (T == 2) {
    t.tile[0] = w & 1;
    t.tile[1] = (w + 1) & 1;
    t.tile[2] = t.tile[3] = w & 1;
    t.act = w == 0 ? 0x3 : w == 1 ? 0x1 : 0;
  } else {
    t.tile[0] = t.tile[1] = t.tile[2] = t.tile[3] = 0;
    t.act = w == 0 ? 0x1 : 0;
  }
  return t;
}

// 32 signature bits -> 32 fp4 (e2m1) operands of an MFMA: register d holds
// bits d, d+4, ..., d+28 as nibbles 0..7, each 0b0001 (0.5) or 0b0000 (0.0).
// Every bit lands in exactly one nibble; the token order along k does not
// matter because the A and B fragments of a Gram come from the same mapping.
__device__ __forceinline__ v8i expand32_fp4(uint32_t b) {
  v8i r;
  r[0] = (int)(b & 0x11111111u);
  r[1] = (int)((b >> 1) & 0x11111111u);
  r[2] = (int)((b >> 2) & 0x11111111u);
  r[3] = (int)((b >> 3) & 0x11111111u);
  r[4] = r[5] = r[6] = r[7] = 0;  // fp4 operands use the low four registers
  return r;
}

// MFMA shapes for TS-expert tiles, fp4 operands with block scale 2^1 on both
// sides, so that every co-occurring token adds 0.5 * 2 * 0.5 * 2 = 1.0 to the
// fp32 accumulator (exact while a count stays below 2^24).  A and B operands
// of lane l hold the same k indices, so one expanded fragment serves as both
// operands of a Gram.
//   TS = 32: v_mfma_scale_f32_32x32x64_f8f6f4, one signature word per
//            instruction; lane l = expert l%32, bits 32*(l/32) .. +31 of the word;
//            C row 8*(r/4)+4*(l/32)+r%4, col l%32
//   TS = 16: v_mfma_scale_f32_16x16x128_f8f6f4, two words per instruction;
//            lane l = expert l%16, 32-bit quarter l/16 of the word pair;
//            C row 4*(l/16)+r, col l%16
constexpr int kFp4 = 4;        // cbsz / blgp operand format code of e2m1
constexpr int kScaleTwo = 128; // E8M0 block scale 2^(128-127)
template <int TS>
struct Mfma;
template <>
struct Mfma<32> {
  typedef v16f Acc;
  static constexpr int kWords = 1, kRegs = 16;
  __device__ static __forceinline__ int expert(int tile, int lane) { return tile * 32 + (lane & 31); }
  __device__ static __forceinline__ int quarter(int lane) { return lane >> 5; }
  __device__ static __forceinline__ Acc mac(v8i a, v8i b, Acc c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, kFp4, kFp4, 0, kScaleTwo, 0, kScaleTwo);
  }
  __device__ static __forceinline__ int row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
  __device__ static __forceinline__ int col(int lane) { return lane & 31; }
};
template <>
struct Mfma<16> {
  typedef v4f Acc;
  static constexpr int kWords = 2, kRegs = 4;
  __device__ static __forceinline__ int expert(int tile, int lane) { return tile * 16 + (lane & 15); }
  __device__ static __forceinline__ int quarter(int lane) { return lane >> 4; }
  __device__ static __forceinline__ Acc mac(v8i a, v8i b, Acc c) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, kFp4, kFp4, 0, kScaleTwo, 0, kScaleTwo);
  }
  __device__ static __forceinline__ int row(int r, int lane) { return 4 * (lane >> 4) + r; }
  __device__ static __forceinline__ int col(int lane) { return lane & 15; }
};

// Tile shape for a padded expert count: 32-wide tiles at 256 experts,
// 16-wide below (8 tiles at 128 experts spread 36 pairs over all 8 waves).
template <int EPW>
struct GramShape {
  static constexpr int TS = EPW >= 256 ? 32 : 16;
  static constexpr int T = EPW / TS;
};

// Accumulate the wave's pair slots over slots [s0, s1) of the bit tile; s0
// and s1 are multiples of Mfma<TS>::kWords.
template <int TS>
__device__ __forceinline__ void mfma_slots(typename Mfma<TS>::Acc (&acc)[kGP], const WaveTiles& wt, const u64* bt,
                                           int stride, int s0, int s1, int lane) {
  if (wt.act == 0) return;
  const bool need[4] = {(wt.act & 0x1B) != 0, (wt.act & 0x6) != 0, (wt.act & 0xC) != 0, (wt.act & 0x10) != 0};
  const int q = Mfma<TS>::quarter(lane);
#pragma unroll 1
  for (int s = s0; s < s1; s += Mfma<TS>::kWords) {  // not unrolled: keeps the fragment registers to one step's worth
    const int ws = s + (q >> 1);                      // the word this lane reads
    const uint32_t* w32 = reinterpret_cast<const uint32_t*>(bt + ws * stride);
    // a fragment no active pair slot reads is left unset (the MFMAs below
    // run only for active slots, whose tiles are all in need)
    v8i f[4];
#pragma unroll
    for (int l = 0; l < 4; ++l)
      if (need[l]) f[l] = expand32_fp4(w32[(Mfma<TS>::expert(wt.tile[l], lane) ^ bt_swz(ws)) * 2 + (q & 1)]);
#pragma unroll
    for (int p = 0; p < kGP; ++p)
      if (wt.act & (1 << p)) acc[p] = Mfma<TS>::mac(f[slot_a(p)], f[slot_b(p)], acc[p]);
  }
}

// Add the counts of one pair slot (row tile I, column tile J) into c (upper
// triangle).  With pair64, two neighbouring counters go in one 64-bit atomic
// add: their sum never carries across the halves because every count of a
// layer stays below 2^32.  Direct entries (I <= J) pair neighbouring
// columns, held by lanes l and l ^ 1; transposed entries (I > J, stored at
// c[col][row]) pair neighbouring rows, held by registers r and r + 1 of one
// lane.  A diagonal tile pair holds every pair of its experts twice; the
// entries below the diagonal are dropped.
template <int TS>
__device__ __forceinline__ void flush_slot(const typename Mfma<TS>::Acc& acc, int I, int J, uint32_t* c, int E,
                                           int lane, bool pair64) {
  const int gj = TS * J + Mfma<TS>::col(lane);
  if (!pair64) {
#pragma unroll
    for (int r = 0; r < Mfma<TS>::kRegs; ++r) {
      const int gi = TS * I + Mfma<TS>::row(r, lane);
      const uint32_t v = (uint32_t)acc[r];  // an exact integer count
      const bool keep = (I != J || gi <= gj) && gi < E && gj < E && v != 0u;
      if (keep) atomicAdd(&c[(int64_t)min(gi, gj) * E + max(gi, gj)], v);
    }
    return;
  }
  u64* c64 = reinterpret_cast<u64*>(c);
  if (I > J) {
#pragma unroll
    for (int r = 0; r < Mfma<TS>::kRegs; r += 2) {
      const int gi = TS * I + Mfma<TS>::row(r, lane);  // even; row(r + 1) = gi + 1
      const u64 v = (u64)(uint32_t)acc[r] | ((u64)(uint32_t)acc[r + 1] << 32);
      if (gi < E && gj < E && v != 0ull) atomicAdd(&c64[((int64_t)gj * E + gi) >> 1], v);
    }
  } else {
    const bool even = (lane & 1) == 0;
#pragma unroll
    for (int r = 0; r < Mfma<TS>::kRegs; ++r) {
      const int gi = TS * I + Mfma<TS>::row(r, lane);
      uint32_t v = (uint32_t)acc[r];
      if (I == J && gi > gj) v = 0u;
      const uint32_t w = (uint32_t)__shfl_xor((int)v, 1);  // column gj ^ 1
      const u64 pv = even ? ((u64)v | ((u64)w << 32)) : 0ull;
      if (gi < E && gj < E && pv != 0ull) atomicAdd(&c64[((int64_t)gi * E + gj) >> 1], pv);
    }
  }
}

// Add the wave's partial counts into c.  Blocks start at different pair
// slots (rot), so that at the end of a launch, when every block flushes at
// once, fewer of them add into the same counters at the same time.  The
// lane index is passed through an empty asm statement so that the compiler
// cannot hoist the addresses of all the atomics out of the unit loop (it
// would keep them live in registers for the whole kernel).
template <int TS>
__device__ __forceinline__ void mfma_flush(const typename Mfma<TS>::Acc (&acc)[kGP], const WaveTiles& wt, uint32_t* c,
                                           int E, int lane_in, int rot, bool pair64) {
  int lane = lane_in;
  asm volatile("" : "+v"(lane));
  for (int t = 0; t < kGP; ++t) {
    int p = t + rot;
    p = p >= kGP ? p - kGP : p;
    if (!(wt.act & (1 << p))) continue;
    const int I = wt.tile[slot_a(p)], J = wt.tile[slot_b(p)];
    switch (p) {  // wave-uniform: static register indices in every case
      case 0: flush_slot<TS>(acc[0], I, J, c, E, lane, pair64); break;
      case 1: flush_slot<TS>(acc[1], I, J, c, E, lane, pair64); break;
      case 2: flush_slot<TS>(acc[2], I, J, c, E, lane, pair64); break;
      case 3: flush_slot<TS>(acc[3], I, J, c, E, lane, pair64); break;
      default: flush_slot<TS>(acc[4], I, J, c, E, lane, pair64); break;
    }
  }
}

// The flush of the Top-K kernel, out of line: it runs a few times per block,
// and inlined, its address arithmetic and atomics cost the kernel's unit loop
// registers (SGPR and VGPR spills).  The accumulators travel by value.
template <int TS>
__device__ __attribute__((noinline)) void mfma_flush_ool(typename Mfma<TS>::Acc a0, typename Mfma<TS>::Acc a1,
                                                         typename Mfma<TS>::Acc a2, typename Mfma<TS>::Acc a3,
                                                         typename Mfma<TS>::Acc a4, WaveTiles wt, uint32_t* c, int E,
                                                         int rot, bool pair64) {
  const typename Mfma<TS>::Acc acc[kGP] = {a0, a1, a2, a3, a4};
  mfma_flush<TS>(acc, wt, c, E, (int)__lane_id(), rot, pair64);
}

#define DOL_WAVE_FENCE() asm volatile("" ::: "memory")

// One segment as the kernel sees it (all values wave-uniform).  Counts fit
// 32 bits: a segment holds fewer than 2^32 tokens and its bit positions stay
// below 2^32, so word indices are below 2^26 and unit indices below 2^29.
// Row r of local word wl holds token wl*64 + r - sh; base points at the
// (virtual) token -sh, so the row pointer of a word is base + wl*64*rowB.
struct Seg {
  const unsigned char* base;  // scores of token -sh
  uint32_t n;                 // tokens
  uint32_t sh;                // bit position of token 0 within its first word
  uint32_t w_first;           // first signature word it touches
  uint32_t words;             // signature words it touches
  uint32_t full_lo, full_hi;  // local words [full_lo, full_hi) hold 64 of its tokens
  uint32_t u_begin;           // its first global unit
  int layer;
};

// The segment table is read in place from the kernel-argument segment with
// scalar loads: indexing the by-value argument with a runtime index would make
// the compiler copy the whole table to private memory first.
typedef const __attribute__((address_space(4))) SegTable* SegTablePtr;

__device__ __forceinline__ Seg load_seg(SegTablePtr tab, int i, int rowB) {
  Seg v;
  const uint64_t off = (uint64_t)tab->s[i].tok_off;
  const uint64_t n = (uint64_t)tab->s[i].n;
  v.n = (uint32_t)n;
  v.sh = (uint32_t)(off & 63);
  v.base = reinterpret_cast<const unsigned char*>(tab->s[i].scores) - (uint64_t)v.sh * (uint64_t)rowB;
  v.w_first = (uint32_t)(off >> 6);
  v.words = n > 0 ? (uint32_t)(((off & 63) + n + 63) >> 6) : 0u;
  v.full_lo = v.sh != 0 ? 1u : 0u;
  v.full_hi = (uint32_t)(((off & 63) + n) >> 6);
  v.u_begin = (uint32_t)tab->tile_start[i];
  v.layer = tab->s[i].layer;
  return v;
}

// Segment holding global unit u (segments with no units are skipped).
__device__ __forceinline__ int seg_of(SegTablePtr tab, uint32_t u, int from) {
  int i = from;
  while (i + 1 < tab->nseg && u >= (uint32_t)tab->tile_start[i + 1]) ++i;
  return i;
}

// Row pointer of local word wl of segment sg.
__device__ __forceinline__ const unsigned char* word_rows(const Seg& sg, uint32_t wl, int rowB) {
  return sg.base + (uint64_t)(wl << 6) * (uint64_t)rowB;
}

// ---------------------------------------------------------------------------
// Top-K (+ Gram) kernel.  Work unit: 8 consecutive signature words (512
// output positions) of one segment, starting 8-aligned within it; one unit
// per block step, one word (64 tokens) per wave.  The grid is persistent
// (one block per CU slot); each block walks the units of its schedule: either
// one contiguous range, or interleaved groups of consecutive units (see
// next_unit and launch_one).
//
// Software pipeline: the signature stores and the Gram of a unit run during
// the next unit (stores right after its first chunk arrives, one Gram slot
// after each ranked chunk), so they overlap other waves' ranking instead of
// following every barrier at once.  Gram accumulators are flushed when the
// layer changes and at the end.  flags bit 0: fast path allowed (16-byte
// rows, k <= 8, E <= 256); bit 1: XCD-partitioned schedule.  gu: units per
// schedule group.
// ---------------------------------------------------------------------------
template <typename T, int EP, int GM, bool AL>
__global__ __launch_bounds__(kFusedThreads) void k_topk(const SegTable tab_arg, const PathArgs a, int flags, uint32_t gu) {
  // AL: every segment starts and ends on a unit boundary (token offset and
  // count multiples of 512) and rows are whole 128-byte chunks, so every word
  // is full, every unit has 8 words, no word is shared between segments and
  // every row of a chunk lies inside its segment.  The edge handling then
  // compiles away, with the registers it holds.
  (void)tab_arg;  // read through `tab` below (it is the first kernel argument)
  const SegTablePtr tab = (SegTablePtr)__builtin_amdgcn_kernarg_segment_ptr();
  constexpr int EPW = EP < 32 ? 32 : EP;  // signature words per slot of the bit tile
  typedef GramShape<EPW> GS;
  typedef typename Mfma<GS::TS>::Acc Acc;
  extern __shared__ __align__(16) unsigned char smem[];
  const bool fast = (flags & 1) != 0;
  u64* bt_all = reinterpret_cast<u64*>(smem + (fast ? kStageBytes : 0));  // [2][kFusedWaves][EPW]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: keeps per-wave control scalar
  const int E = a.E, k = a.k;
  const int rowB = E * (int)sizeof(T);
  const int rowv = rowB >> 4;
  const int nch = (rowv + 7) >> 3;
  unsigned char* st = smem + wave * 2 * kChunkBytes;  // this wave's two stage buffers

  // Unit schedule: the unit range [lo, hi) of a block's partition is cut into
  // groups of `gu` consecutive units, and the Gs blocks of the partition take
  // groups pos, pos + Gs, pos + 2 Gs, ...  Contiguous ranges are the case of
  // one group per block.  flags bit 1 selects the partition:
  //   0: one partition [0, U), pos = b
  //   1: eight partitions, one per XCD (blocks are dispatched round-robin,
  //      so block b runs on XCD b mod 8), of U/8 units each; the XCD's
  //      blocks work on adjacent groups of its partition, so their signature
  //      stores land side by side while each block stays in few layers (few
  //      Gram flushes, and those of different XCDs go to different layers)
  // All unit counts are below 2^29 (64 segments of fewer than 2^32 tokens).
  const uint32_t U = (uint32_t)tab->tile_start[tab->nseg];
  const uint32_t G = gridDim.x;
  const uint32_t b = blockIdx.x;
  const bool xcd = (G & 7) == 0 && (flags & 2) != 0;
  const uint32_t lo = xcd ? (uint32_t)(((uint64_t)(b & 7) * U) >> 3) : 0u;
  const uint32_t hi = xcd ? (uint32_t)(((uint64_t)((b & 7) + 1) * U) >> 3) : U;
  const uint32_t Gs = xcd ? G >> 3 : G;
  const uint32_t pos = xcd ? b >> 3 : b;
  const uint32_t ug = lo + pos * gu;
  if (ug >= hi) return;
  // The unit after u in this block's schedule (U when there is none), from
  // the bounds of the current group: called once per unit, in order.
  uint32_t g_start = ug, g_end = min(ug + gu, hi);
  auto next_unit = [&](uint32_t u_) -> uint32_t {
    if (u_ + 1 < g_end) return u_ + 1;
    g_start += Gs * gu;
    if (g_start >= hi) return U;
    g_end = min(g_start + gu, hi);
    return g_start;
  };

  PopcGram<EPW, kFusedThreads, GM == kGramPopc> pg;
  if (GM == kGramPopc) pg.init(tid, E);
  const WaveTiles wt = wave_tiles(GS::T, wave);
  Acc acc[kGP];
  auto zero_acc = [&]() {
#pragma unroll
    for (int p = 0; p < kGP; ++p)
#pragma unroll
      for (int r = 0; r < Mfma<GS::TS>::kRegs; ++r) acc[p][r] = 0.0f;
  };
  zero_acc();

  // Lane offsets inside a chunk: instruction j fills rows 8j..8j+7; lane i
  // fills slot (i & 7) of row 8j + i/8, which holds piece
  // q = (i & 7) ^ swz(8j + i/8) = (i & 7) ^ (i >> 3) ^ (j & 1).
  const int q_even = (lane & 7) ^ (lane >> 3);
  const uint32_t off_even = (uint32_t)((lane >> 3) * rowB + q_even * 16);        // bytes from the chunk's row 0
  const uint32_t off_odd = (uint32_t)((lane >> 3) * rowB + (q_even ^ 1) * 16);  // odd j: piece q_even ^ 1
  // Up to 128 experts the lane offsets of the eight loads of a full chunk are
  // kept in VGPRs: as scalar offsets they are spilled and read back (with
  // hazard waits) per load (-1 % at the stream workload).  At 256 experts the
  // VGPRs are full and the scalar offsets measured faster.
  constexpr bool kVoff = EP <= 128;
  uint32_t voff[8] = {};
  if constexpr (kVoff) {
#pragma unroll
    for (int j = 0; j < 8; ++j) voff[j] = ((j & 1) ? off_odd : off_even) + (uint32_t)(j * 8 * rowB);
    asm volatile("" : "+v"(voff[0]), "+v"(voff[1]), "+v"(voff[2]), "+v"(voff[3]), "+v"(voff[4]), "+v"(voff[5]),
                 "+v"(voff[6]), "+v"(voff[7]));
  }

  // Rows [r_lo, r_hi) of local word wl of segment sg hold its tokens
  // (wave-uniform; 64-bit only where sh + n may reach 2^32).
  const int row_in_j0 = lane >> 3;
  auto row_bounds = [&](const Seg& sg, uint32_t wl, int& r_lo, int& r_hi) {
    r_lo = wl == 0 ? (int)sg.sh : 0;
    const int64_t rem = (int64_t)sg.sh + (int64_t)sg.n - ((int64_t)wl << 6);
    r_hi = (int)max((int64_t)0, min((int64_t)64, rem));
  };
  // Direct-to-LDS load of full 128-byte chunk c_ of the 64 rows of local word
  // wl of segment sg (asynchronous; the consumer waits with DOL_WAIT_VMEM).
  // When every row lies inside the segment the loads go through a buffer
  // resource based at the chunk's row 0: the row offsets are scalar and the
  // lane offset is one 32-bit register, so issuing a load costs no vector
  // instruction.
  auto dma = [&](const Seg& sg, uint32_t wl, int c_, unsigned char* sbuf) {
    if (c_ * 8 + 8 > rowv) return;
    const unsigned char* cbase = word_rows(sg, wl, rowB) + c_ * 128;  // row 0 of the chunk (uniform)
    if (AL || (wl >= sg.full_lo && wl < sg.full_hi)) {  // every row inside the segment
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(cbase), (short)0, 0x7FFFFFFF, kBufWord3);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if constexpr (kVoff)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(sbuf + j * 1024), 16,
                                                   voff[j], 0, 0, kStreamPolicy);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(sbuf + j * 1024), 16,
                                                   (j & 1) ? off_odd : off_even, (uint32_t)(j * 8 * rowB), 0,
                                                   kStreamPolicy);
    } else {
      int r_lo, r_hi;
      row_bounds(sg, wl, r_lo, r_hi);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = 8 * j + row_in_j0;
        if (r >= r_lo && r < r_hi)
          __builtin_amdgcn_global_load_lds(cbase + (uint32_t)(j * 8 * rowB) + ((j & 1) ? off_odd : off_even),
                                           (__attribute__((address_space(3))) void*)(sbuf + j * 1024), 16, 0, kStreamPolicy);
      }
    }
  };
  // Synchronous fill of a partial chunk (the row ends inside it): missing
  // vectors read as all-ones (a NaN), ranked last and never selected on the fast path.
  auto fill_partial = [&](const Seg& sg, uint32_t wl, int c_, unsigned char* sbuf) {
    const int cvn = rowv - c_ * 8;
    const unsigned char* cbase = word_rows(sg, wl, rowB) + c_ * 128;
    int r_lo, r_hi;
    row_bounds(sg, wl, r_lo, r_hi);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int r = 8 * j + row_in_j0;
      const int q = q_even ^ (j & 1);
      v4u val = v4u{~0u, ~0u, ~0u, ~0u};
      if (q < cvn && r >= r_lo && r < r_hi)
        val = *reinterpret_cast<const v4u*>(cbase + (uint32_t)(j * 8 * rowB) + ((j & 1) ? off_odd : off_even));
      *reinterpret_cast<v4u*>(sbuf + j * 1024 + lane * 16) = val;
    }
  };

  constexpr int kGramStep = GM == kGramMfma ? Mfma<GS::TS>::kWords : 1;  // slots per Gram step
  constexpr int kMaxAccUnits = ((1 << 24) / 512) - 1;  // units per flush at most (counts < 2^24)
  int acc_units = 0;

  // The unit whose bit tile is complete and whose stores and Gram are pending.
  struct Pending {
    u64* lb;          // bits of its layer (null: no signature output)
    uint32_t w0;      // its first signature word
    int cnt;          // words in it
    int layer;
    int shared_lo;    // slot 0 holds a word shared with the previous segment (OR it in)
    int shared_hi;    // slot holding a word shared with the next segment, or -1
  };
  Pending pend{};
  bool have_pend = false;
  typedef StoreBatch<EPW> SB;
  v2u64 sreg[SB::kUnits][SB::kItems];  // batched signature stores (see batch_flush)
  u64* sb_lb = nullptr;
  uint32_t sb_w0 = 0;
  int sb_n = 0;
  // This wave's share of the pending unit's signature stores: experts
  // [wave*E/8, (wave+1)*E/8), 64 bytes (8 words) per expert as four 16-byte
  // stores when the unit starts on an even word, else word by word.
  // The stores of plain units (8 words, even first word, no word shared with
  // a neighbouring segment) are held in registers for up to SB::kUnits
  // consecutive units of one layer and issued together.  In the unit-major
  // signature layout a unit that starts on a multiple of 8 words is one
  // contiguous block of E * 64 bytes, so a block's batch writes up to
  // SB::kUnits * E * 64 contiguous bytes (with expert-major rows, 64-byte
  // pieces 256 rows apart cost up to 1 ms more per 1 GiB on some buffer
  // placements; contiguous blocks 0.4 ms).  Only for E <= 256.
  // Whole-vector stores carry the non-temporal hint: the signatures are not
  // read again by this kernel.
  auto batch_flush = [&]() __attribute__((always_inline)) {
    if (sb_n == 0) return;
    const int e_lo = (wave * E) >> 3, e_hi = ((wave + 1) * E) >> 3;
#pragma unroll
    for (int i = 0; i < SB::kItems; ++i) {
      const int item = e_lo * 4 + lane + i * kWave;
      if (item < e_hi * 4) {
        u64* dst = sb_lb + sig_off(sb_w0 + (item & 3) * 2, item >> 2, E);
#pragma unroll
        for (int j = 0; j < SB::kUnits; ++j)  // unit j of the batch: 8 words further for every expert
          if (j < sb_n) __builtin_nontemporal_store(sreg[j][i], reinterpret_cast<v2u64*>(dst + (int64_t)E * 8 * j));
      }
    }
    sb_n = 0;
  };
  auto store_share = [&](const u64* pbt) __attribute__((always_inline)) {
    if (pend.lb == nullptr) return;
    const int e_lo = (wave * E) >> 3, e_hi = ((wave + 1) * E) >> 3;
    const bool plain_unit =
        AL || ((pend.w0 & 1) == 0 && pend.cnt == kFusedWaves && !pend.shared_lo && pend.shared_hi < 0);
    if (EPW <= 256 && plain_unit) {
      if (sb_n > 0 && (sb_lb != pend.lb || sb_w0 + 8 * sb_n != pend.w0)) batch_flush();
      if (sb_n == 0) {
        sb_lb = pend.lb;
        sb_w0 = pend.w0;
      }
      v2u64 v[SB::kItems];
#pragma unroll
      for (int i = 0; i < SB::kItems; ++i) {
        const int item = e_lo * 4 + lane + i * kWave;
        const int e = item >> 2, s0 = (item & 3) * 2;
        v[i] = item < e_hi * 4 ? v2u64{pbt[s0 * EPW + (e ^ bt_swz(s0))], pbt[(s0 + 1) * EPW + (e ^ bt_swz(s0 + 1))]}
                               : v2u64{0ull, 0ull};
      }
#pragma unroll
      for (int j = 0; j < SB::kUnits; ++j)
        if (j == sb_n) {
#pragma unroll
          for (int i = 0; i < SB::kItems; ++i) sreg[j][i] = v[i];
        }
      if (++sb_n == SB::kUnits) batch_flush();
      return;
    }
    batch_flush();
    auto plain = [&](int s_) { return !((s_ == 0 && pend.shared_lo) || s_ == pend.shared_hi); };
    auto put = [&](int e_, int s_, u64 word) {
      u64* dst = pend.lb + sig_off(pend.w0 + s_, e_, E);
      if (plain(s_))
        *dst = word;
      else if (word)
        atomicOr(dst, word);
    };
    // without or_partial a segment is a whole layer that starts on a unit, so
    // the words of its last unit past the segment are the layer's padding:
    // they are written as zeros (the output is then fully determined)
    const bool pad = a.or_partial == 0;
    if ((pend.w0 & 1) == 0) {
      for (int item = e_lo * 4 + lane; item < e_hi * 4; item += kWave) {
        const int e = item >> 2, s0 = (item & 3) * 2;
        if (s0 >= pend.cnt) {
          if (pad)
            __builtin_nontemporal_store(v2u64{0ull, 0ull},
                                        reinterpret_cast<v2u64*>(pend.lb + sig_off(pend.w0 + s0, e, E)));
          continue;
        }
        const u64 wa = pbt[s0 * EPW + (e ^ bt_swz(s0))];
        const u64 wb = pbt[(s0 + 1) * EPW + (e ^ bt_swz(s0 + 1))];
        if (s0 + 1 < pend.cnt && plain(s0) && plain(s0 + 1)) {
          // an even word and the next lie in one unit: 16 contiguous bytes
          __builtin_nontemporal_store(v2u64{wa, wb}, reinterpret_cast<v2u64*>(pend.lb + sig_off(pend.w0 + s0, e, E)));
        } else {
          put(e, s0, wa);
          if (s0 + 1 < pend.cnt)
            put(e, s0 + 1, wb);
          else if (pad)
            put(e, s0 + 1, 0ull);
        }
      }
    } else {
      for (int item = e_lo * kFusedWaves + lane; item < e_hi * kFusedWaves; item += kWave) {
        const int e = item >> 3, s0 = item & 7;
        if (s0 < pend.cnt) put(e, s0, pbt[s0 * EPW + (e ^ bt_swz(s0))]);
      }
    }
  };
  // Gram of slots [s0, s1) of the pending unit (empty slots are zero).
  auto gram_slots = [&](const u64* pbt, int s0, int s1) {
    if (GM == kGramMfma) mfma_slots<GS::TS>(acc, wt, pbt, EPW, s0, s1, lane);
    if (GM == kGramPopc) pg.accumulate(pbt, s0, min(s1, pend.cnt), EPW);
  };
  // 64-bit atomics need even E (8-byte aligned rows) and an 8-byte aligned matrix
  const bool pair64 = (E & 1) == 0 && (reinterpret_cast<uintptr_t>(a.cacc) & 7) == 0;
  auto flush = [&](int layer) {
    if (GM == kGramNone) return;
    uint32_t* cl = a.cacc + (int64_t)layer * a.cacc_layer_elems +
                   (a.ncopies > 1 ? (int64_t)(blockIdx.x % (uint32_t)a.ncopies) * a.cacc_copy_elems : 0);
    if (GM == kGramMfma) {
      mfma_flush_ool<GS::TS>(acc[0], acc[1], acc[2], acc[3], acc[4], wt, cl, E, (int)(blockIdx.x % kGP), pair64);
      zero_acc();
    }
    if (GM == kGramPopc) {
      pg.flush(cl, E);
      pg.init(tid, E);
    }
  };

  // fp32 waves start with positive keys (general keys cost ~3 more
  // instructions per score) and switch for the rest of the kernel after
  // meeting a non-positive threshold; bf16 general keys cost ~1 more per
  // score, less than the exact re-rank a first non-positive threshold costs
  // in a short launch, so bf16 rows start with them and move to positive
  // keys within the row (below).
  bool gen = Traits<T>::kExact;
  int cb = 0;  // stage buffer holding the current chunk
  // key byte selectors, opaque to the compiler so that they stay in VGPRs
  // instead of being rematerialised for every key
  KeySel ks;
#pragma unroll
  for (int j = 0; j < 4; ++j) ks.f32[j] = 0x07060500u | (uint32_t)j;
  ks.lo[0] = 0x05040C00u;
  ks.lo[1] = 0x05040C02u;
  ks.hi[0] = 0x07060C01u;
  ks.hi[1] = 0x07060C03u;
#pragma unroll
  for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(ks.f32[j]));
#pragma unroll
  for (int j = 0; j < 2; ++j) asm volatile("" : "+v"(ks.lo[j]), "+v"(ks.hi[j]));

  int seg = seg_of(tab, ug, 0);
  Seg sv = load_seg(tab, seg, rowB);
  uint32_t tl0 = 8 * (ug - sv.u_begin);  // local word of slot 0 of the current unit
  if (fast && tl0 + wave < sv.words) dma(sv, tl0 + wave, 0, st);

  int buf = 0;
  for (uint32_t u = ug; u < U; buf ^= 1) {
    const uint32_t wl = tl0 + wave;                      // this wave's local word
    const int cnt = AL ? kFusedWaves : (int)min((uint32_t)kFusedWaves, sv.words - tl0);  // words in this unit
    // next unit and its segment (wave-uniform)
    const uint32_t un = next_unit(u);
    int seg_n = seg;
    Seg svn = sv;
    uint32_t tl0n = tl0 + 8;
    if (un < U) {
      if (un >= (uint32_t)tab->tile_start[seg + 1]) {
        seg_n = seg_of(tab, un, seg);
        svn = load_seg(tab, seg_n, rowB);
      }
      tl0n = 8 * (un - svn.u_begin);
    }
    const uint32_t wln = tl0n + wave;
    const bool next_mine = un < U && (AL || wln < svn.words);

    u64* bt = bt_all + buf * kFusedWaves * EPW;
    const u64* pbt = bt_all + (buf ^ 1) * kFusedWaves * EPW;  // the pending unit's tile
    u64* mybt = bt + wave * EPW;
#pragma unroll
    for (int e0 = 0; e0 < EPW; e0 += 64)
      if (e0 + lane < EPW) mybt[e0 + lane] = 0;
    DOL_WAVE_FENCE();
    int gram_done = have_pend ? 0 : kFusedWaves;  // slots of the pending unit already accumulated
    bool stored = !have_pend;
    if (!AL && fast && wave >= cnt && next_mine) {
      // idle in this unit (segment end) but busy in the next one: start that
      // word's first chunk now, into the buffer the next unit reads first
      dma(svn, wln, 0, st + cb * kChunkBytes);
    }
    if (AL || wave < cnt) {
      // the lane's row holds a token of the segment (every row of an interior word does)
      const uint32_t row = (wl << 6) + (uint32_t)lane;
      const bool valid = AL || (wl >= sv.full_lo && wl < sv.full_hi) ||
                         (row >= sv.sh && (uint64_t)row < (uint64_t)sv.sh + (uint64_t)sv.n);
      bool need_slow = valid;
      if (fast) {
        int top[8];
        int rej = INT_MIN;
#pragma unroll
        for (int i = 0; i < 8; ++i) top[i] = INT_MIN;
        bool gk = gen;  // key kind of the next chunk of this row
        for (int c = 0; c < nch; ++c) {
          unsigned char* cur = st + cb * kChunkBytes;
          // Two waves share each SIMD and its arbiter prefers the older one:
          // left to it, waves 0-3 end every unit early and wait at the block
          // barrier (29 % of their time) while waves 4-7 finish alone.
          // Waves 4-7 therefore take the higher priority for even chunks (bf16:
          // after their share of the signature stores), which evens out when
          // the two waves of a SIMD reach the barrier.
          if (wave >= 4) {
            if (c & 1)
              __builtin_amdgcn_s_setprio(0);
            else if constexpr (!Traits<T>::kExact)
              __builtin_amdgcn_s_setprio(1);
          }
          if (AL || c * 8 + 8 <= rowv) {
            DOL_WAIT_VMEM();  // this chunk's direct-to-LDS loads (and earlier stores) have completed
          } else {
            fill_partial(sv, wl, c, cur);
          }
          DOL_WAVE_FENCE();
          unsigned char* other = st + (cb ^ 1) * kChunkBytes;
          if (c + 1 < nch)
            dma(sv, wl, c + 1, other);
          else if (next_mine)
            dma(svn, wln, 0, other);
          if (!stored) {
            store_share(pbt);
            stored = true;
          }
          if constexpr (Traits<T>::kExact)
            if (wave >= 4 && !(c & 1)) __builtin_amdgcn_s_setprio(1);
          if (gk)
            rank_chunk<T, true>(cur, lane, c * 8, ks, top, rej);
          else
            rank_chunk<T, false>(cur, lane, c * 8, ks, top, rej);
          // bf16: once the 8th key of every token of the wave is a positive
          // number, the rest of the row takes positive keys.  A negative score
          // then keys below zero instead of at its general key, below that 8th
          // key either way, and positive scores key the same under both kinds,
          // so the list ends exactly as with general keys throughout.
          if (Traits<T>::kExact && gk && c + 1 < nch &&
              __ballot(valid && top[7] < Traits<T>::kPosMin) == 0ull)
            gk = false;
          if (gram_done < kFusedWaves) {
            const int s_end = (((c + 1) * kFusedWaves) / nch) & ~(kGramStep - 1);
            gram_slots(pbt, gram_done, s_end);
            gram_done = s_end;
          }
          DOL_WAVE_FENCE();
          cb ^= 1;
        }
        if (wave >= 4) __builtin_amdgcn_s_setprio(0);
        // the k-th and (k+1)-th keys: a wave-uniform branch on k, so that no
        // per-position predicate on k stays live (in registers) across the loop
        int sk, sk1;
        switch (k) {
          case 1: sk = top[0]; sk1 = top[1]; break;
          case 2: sk = top[1]; sk1 = top[2]; break;
          case 3: sk = top[2]; sk1 = top[3]; break;
          case 4: sk = top[3]; sk1 = top[4]; break;
          case 5: sk = top[4]; sk1 = top[5]; break;
          case 6: sk = top[5]; sk1 = top[6]; break;
          case 7: sk = top[6]; sk1 = top[7]; break;
          default: sk = top[7]; sk1 = rej; break;
        }
        bool ok = top[0] < kCompPosInf;
        bool nonpos = false;
        if (gen) {
          ok = ok && sk > kCompNegInfMax && (sk < Traits<T>::kZeroLo || sk > Traits<T>::kZeroHi);
        } else {
          nonpos = valid && sk < Traits<T>::kPosMin;
          ok = ok && !nonpos;
        }
        // fp32 keys keep 24 value bits: when the k-th and (k+1)-th keys share a
        // bucket, the experts above the bucket are certain and the rest are
        // picked from the bucket by resolve_ties
        const bool tie = !Traits<T>::kExact && valid && ok && ((sk1 >> 8) == (sk >> 8));
        need_slow = valid && !ok;
        int need = 0;
        if (valid && ok) {
          // keys are unique, so the k selected entries are those >= sk
          const u64 bit = 1ull << lane;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            if (top[i] >= sk) {
              if (!tie || (top[i] >> 8) > (sk >> 8))
                atomicOr(&mybt[(255 - (top[i] & 255)) ^ bt_swz(wave)], bit);
              else
                ++need;
            }
          }
        }
        if (!Traits<T>::kExact) {
          const u64 tm = __ballot(tie);
          if (tm != 0ull) resolve_ties(tm, sk, need, gen, mybt, word_rows(sv, wl, rowB), rowB, bt_swz(wave));
        }
        if (__ballot(nonpos) != 0ull) gen = true;
      }
      if (__ballot(need_slow) != 0ull) {
        if (need_slow) {
          const T* rp = reinterpret_cast<const T*>(word_rows(sv, wl, rowB) + (uint32_t)lane * (uint32_t)rowB);
          exact_select_lane<T>(rp, E, k, mybt, bt_swz(wave), 1ull << lane);
        }
      }
    }
    // waves without a fast chunk loop in this unit finish the pending unit here
    if (!stored) store_share(pbt);
    if (gram_done < kFusedWaves) gram_slots(pbt, gram_done, kFusedWaves);
    __syncthreads();  // this unit's bit tile is complete; the pending unit's tile is free
    // the fp32 Gram accumulators hold exact counts below 2^24: flush at a
    // layer change and before a block has accumulated 2^24 tokens
    if (have_pend && (pend.layer != sv.layer || ++acc_units >= kMaxAccUnits)) {
      flush(pend.layer);
      acc_units = 0;
    }
    pend.lb = a.bits != nullptr ? a.bits + (int64_t)sv.layer * a.bits_layer_words : nullptr;
    pend.w0 = sv.w_first + tl0;
    pend.cnt = cnt;
    pend.layer = sv.layer;
    pend.shared_lo = !AL && a.or_partial && tl0 == 0 && sv.sh != 0;
    pend.shared_hi = (!AL && a.or_partial && tl0 + cnt == sv.words && ((sv.sh + sv.n) & 63) != 0) ? cnt - 1 : -1;
    have_pend = true;
    u = un;
    seg = seg_n;
    sv = svn;
    tl0 = tl0n;
  }
  // the last unit
  store_share(bt_all + (buf ^ 1) * kFusedWaves * EPW);
  batch_flush();
  gram_slots(bt_all + (buf ^ 1) * kFusedWaves * EPW, 0, kFusedWaves);
  flush(pend.layer);
}

// Process-wide overrides of choices that never change results (do_set_option):
// the Gram kind and the unit schedule.
std::atomic<int> g_opt_gram{0};    // 0: fp4 MFMA, 1: VALU popcount
std::atomic<int> g_opt_sched{-1};  // -1: measured per launch shape, else an index into kSchedCand

int gram_mode() { return g_opt_gram.load(std::memory_order_relaxed) == 1 ? kGramPopc : kGramMfma; }

// Unit schedule of the Top-K kernel: groups of gu consecutive units (gu = 0:
// one contiguous range per block), in one partition or one per XCD.
struct Sched {
  int64_t gu;
  bool xcd;
};

template <typename T, int EP, int GM, bool AL = false>
hipError_t launch_one(const SegTable& tab, const PathArgs& a, bool fast, Sched sc, hipStream_t s, const ProfEv& pe) {
  constexpr int EPW = EP < 32 ? 32 : EP;
  auto kern = k_topk<T, EP, GM, AL>;
  const size_t lds = (fast ? (size_t)kStageBytes : 0) + 2 * (size_t)kFusedWaves * EPW * sizeof(u64);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  int occ = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, kFusedThreads, lds) != hipSuccess || occ < 1) occ = 1;
  const DevInfo di = device_info();
  const int64_t units = tab.tile_start[tab.nseg];
  int64_t blocks = std::min<int64_t>((int64_t)di.cu_count * occ, units);
  blocks = std::max<int64_t>(blocks, 1);
  int64_t gu = sc.gu;
  const int64_t per_part = sc.xcd ? (units + 7) / 8 : units;
  const int64_t gs = sc.xcd ? std::max<int64_t>(blocks / 8, 1) : blocks;
  if (gu <= 0 || gu * gs > per_part) gu = (per_part + gs - 1) / gs;  // contiguous ranges
  const int flags = (fast ? 1 : 0) | (sc.xcd ? 2 : 0);
  if (pe.start != nullptr || pe.stop != nullptr)  // caller's timing events bound to this dispatch
    hipExtLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kFusedThreads), lds, s, pe.start, pe.stop, 0u, tab, a,
                          flags, (uint32_t)gu);
  else
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kFusedThreads), lds, s, tab, a, flags, (uint32_t)gu);
  return hipGetLastError();
}

// Segments on unit boundaries with rows of whole 128-byte chunks (the
// condition of k_topk's AL specialization).
bool aligned_segments(const SegTable& tab, int rowB) {
  if (rowB % 128 != 0) return false;
  for (int i = 0; i < tab.nseg; ++i)
    if (tab.s[i].n % 512 != 0 || tab.s[i].tok_off % 512 != 0) return false;
  return true;
}

template <typename T, int EP>
hipError_t launch_gm(const SegTable& tab, const PathArgs& a, bool fast, Sched sc, hipStream_t s, const ProfEv& pe) {
  // the aligned specialization: bf16 at 128 experts -11 %; fp32 at 256 experts
  // -8.5 % without signature output and -5 % with it where the stores are cheap
  // (halved SGPR spills)
  if constexpr (EP <= 256) {
    if (fast && aligned_segments(tab, a.E * (int)sizeof(T))) {
      if (a.cacc == nullptr) return launch_one<T, EP, kGramNone, true>(tab, a, fast, sc, s, pe);
      if (gram_mode() == kGramPopc) return launch_one<T, EP, kGramPopc, true>(tab, a, fast, sc, s, pe);
      return launch_one<T, EP, kGramMfma, true>(tab, a, fast, sc, s, pe);
    }
  }
  if (a.cacc == nullptr) return launch_one<T, EP, kGramNone>(tab, a, fast, sc, s, pe);
  if (gram_mode() == kGramPopc) return launch_one<T, EP, kGramPopc>(tab, a, fast, sc, s, pe);
  return launch_one<T, EP, kGramMfma>(tab, a, fast, sc, s, pe);
}

template <typename T>
hipError_t launch_ep(const SegTable& tab, const PathArgs& a, bool fast, Sched sc, hipStream_t s, const ProfEv& pe) {
  const int E = a.E;
  if (E <= 32) return launch_gm<T, 32>(tab, a, fast, sc, s, pe);
  if (E <= 64) return launch_gm<T, 64>(tab, a, fast, sc, s, pe);
  if (E <= 128) return launch_gm<T, 128>(tab, a, fast, sc, s, pe);
  if (E <= 256) return launch_gm<T, 256>(tab, a, fast, sc, s, pe);
  // E in (256, 1024]: exact per-lane selection, signatures only
  if (a.cacc != nullptr) return hipErrorInvalidValue;
  if (E <= 512) return launch_one<T, 512, kGramNone>(tab, a, false, sc, s, pe);
  return launch_one<T, 1024, kGramNone>(tab, a, false, sc, s, pe);
}

// Launch-time choice of the unit schedule for large launches.  The cost of
// the signature stores under a given schedule differs between otherwise
// identical boards (it follows how the concurrent store streams fall on
// the HBM channels), while it repeats within one process.  So for each
// large launch shape the first launches try the candidates in turn with
// events around them; completed measurements are collected with
// hipEventQuery, which never waits, and once every candidate has kTuneTrials
// of them, the one with the fastest launch is used for all later launches of
// that shape (it must beat the first candidate by 2 %).  Measuring starts
// kTuneDelayMs after the first launch of a shape: launches right after an idle
// period run slower for some tens of milliseconds (7.3 ms falling to 5.6 ms
// over the first six launches of workload 4), which would hide a 12 %
// difference between the schedules.  Launches under stream capture and
// launches below kTuneMinUnits use the first candidate (or the one already
// chosen for the shape); a capture never touches the measurement events.
// When every slot of the table holds a shape, a decided one is recycled.
constexpr Sched kSchedCand[2] = {Sched{4, true}, Sched{0, false}};  // XCD partitions; contiguous ranges
constexpr int kNumCand = 2;
constexpr int64_t kTuneMinUnits = 1024;  // 512 Ki tokens
constexpr int kTuneTrials = 3;           // measured launches per candidate
constexpr double kTuneDelayMs = 100.0;   // no measurement before this long after a shape's first launch
constexpr int kTuneSlots = 16;

struct Tune {
  uint64_t key;
  int device;
  int calls;
  std::chrono::steady_clock::time_point first;  // host time of the shape's first launch
  int chosen;                 // index into kSchedCand, or -1 while measuring
  float best[kNumCand];       // fastest completed launch per candidate (ms), < 0 if none yet
  int trials[kNumCand];       // completed measurements per candidate
  bool pending[kNumCand];     // a measured launch is in flight
  hipEvent_t ev[kNumCand][2];
};
std::mutex g_tune_mu;
Tune g_tune[kTuneSlots];
int g_ntune = 0;
int g_tune_next = 0;  // next slot considered for recycling

uint64_t mix(uint64_t h, uint64_t v) {
  h ^= v + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
  return h;
}

void release_events(Tune& t) {
  for (int c = 0; c < kNumCand; ++c)
    for (int i = 0; i < 2; ++i)
      if (t.ev[c][i] != nullptr) {
        (void)hipEventDestroy(t.ev[c][i]);
        t.ev[c][i] = nullptr;
      }
}

void decide(Tune& t, int c) {
  t.chosen = c;
  release_events(t);  // no trial is pending once a candidate is chosen
}

// Picks the schedule of one launch and, when it is a measured trial, sets
// *ev_out to the candidate's start/stop events.
Sched tuned_schedule(do_dtype dt, const SegTable& tab, const PathArgs& a, bool fast, hipStream_t s,
                     hipEvent_t* ev_out) {
  ev_out[0] = ev_out[1] = nullptr;
  const int64_t units = tab.tile_start[tab.nseg];
  if (units < kTuneMinUnits) return kSchedCand[0];
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  const bool capturing = hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return kSchedCand[0];
  uint64_t key = 0;
  key = mix(key, (uint64_t)dt);
  key = mix(key, (uint64_t)a.E);
  key = mix(key, (uint64_t)a.k);
  key = mix(key, (uint64_t)units);
  key = mix(key, (uint64_t)tab.nseg);
  key = mix(key, (uint64_t)tab.s[tab.nseg - 1].layer - (uint64_t)tab.s[0].layer);
  key = mix(key, (uint64_t)(a.bits != nullptr) | ((uint64_t)(a.cacc != nullptr) << 1) |
                     ((uint64_t)a.or_partial << 2) | ((uint64_t)fast << 3));
  std::lock_guard<std::mutex> lock(g_tune_mu);
  Tune* t = nullptr;
  for (int i = 0; i < g_ntune; ++i)
    if (g_tune[i].key == key && g_tune[i].device == dev) t = &g_tune[i];
  if (t != nullptr && t->chosen >= 0) return kSchedCand[t->chosen];
  if (capturing) return kSchedCand[0];
  if (t == nullptr) {
    if (g_ntune < kTuneSlots) {
      t = &g_tune[g_ntune++];
    } else {
      for (int i = 0; i < kTuneSlots && t == nullptr; ++i) {
        Tune& c = g_tune[(g_tune_next + i) % kTuneSlots];
        if (c.chosen >= 0) {
          t = &c;
          g_tune_next = (g_tune_next + i + 1) % kTuneSlots;
        }
      }
      if (t == nullptr) return kSchedCand[0];  // every slot is still measuring
    }
    *t = Tune{};
    t->key = key;
    t->device = dev;
    t->chosen = -1;
    for (int c = 0; c < kNumCand; ++c) t->best[c] = -1.f;
  }
  // collect finished trials
  bool all = true;
  for (int c = 0; c < kNumCand; ++c) {
    if (t->pending[c]) {
      const hipError_t q = hipEventQuery(t->ev[c][1]);
      if (q == hipSuccess) {
        float ms = -1.f;
        if (hipEventElapsedTime(&ms, t->ev[c][0], t->ev[c][1]) == hipSuccess && ms > 0.f) {
          t->best[c] = t->best[c] < 0.f ? ms : std::min(t->best[c], ms);
          ++t->trials[c];
        }
        t->pending[c] = false;
      } else if (q != hipErrorNotReady) {
        t->pending[c] = false;
        decide(*t, 0);  // measurement failed: keep the first candidate
        return kSchedCand[0];
      }
    }
    all = all && t->trials[c] >= kTuneTrials;
  }
  if (all) {
    int bc = 0;
    for (int c = 1; c < kNumCand; ++c)
      if (t->best[c] < 0.98f * t->best[bc]) bc = c;  // switch only for a clear gain
    if (getenv("DOLOSS_TUNE_LOG") != nullptr)
      fprintf(stderr, "[doloss] unit schedule for %lld units: candidates %.4f / %.4f ms, chose %d\n",
              (long long)units, t->best[0], t->best[1], bc);
    decide(*t, bc);
    return kSchedCand[bc];
  }
  const auto now = std::chrono::steady_clock::now();
  if (t->calls++ == 0) t->first = now;
  if (std::chrono::duration<double, std::milli>(now - t->first).count() < kTuneDelayMs) return kSchedCand[0];
  // the candidate with the fewest measurements that has none in flight
  // (ties to the one measured least recently, so the candidates alternate)
  int pick = -1;
  for (int i = 0; i < kNumCand; ++i) {
    const int c = (t->calls + i) % kNumCand;
    if (t->pending[c] || t->trials[c] >= kTuneTrials) continue;
    if (pick < 0 || t->trials[c] < t->trials[pick]) pick = c;
  }
  if (pick < 0) return kSchedCand[0];  // every candidate still has a launch in flight
  if (t->ev[pick][0] == nullptr) {
    if (hipEventCreate(&t->ev[pick][0]) != hipSuccess || hipEventCreate(&t->ev[pick][1]) != hipSuccess) {
      decide(*t, 0);
      return kSchedCand[0];
    }
  }
  t->pending[pick] = true;
  ev_out[0] = t->ev[pick][0];
  ev_out[1] = t->ev[pick][1];
  return kSchedCand[pick];
}

// ---------------------------------------------------------------------------
// Gram of stored signatures (do_pairwise_hamming, E <= 256) on the same fp4
// MFMA tiles as k_topk.  Block b takes layer b / bpl and the part b % bpl of
// that layer's 8-word chunks, kGramGroup chunks per step.  A chunk's words of
// every expert are staged in LDS in the bit-tile layout of k_topk (word s of
// expert e at s * EPW + (e ^ bt_swz(s))); the next step's words are loaded
// into registers while the current step is multiplied, so one barrier and one
// memory round trip cover kGramGroup chunks.  Each block adds its counts into
// cacc at the end; its chunk count stays below 2^24 / 512 (exact fp32 counts).
// ---------------------------------------------------------------------------
constexpr int64_t kGramMaxChunks = ((1 << 24) / 512) - 1;
constexpr int kGramGroup = 4;  // chunks per step

template <int EP>
__global__ __launch_bounds__(kFusedThreads) void k_gram_mfma(const u64* bits, int64_t W, int E, int L, int bpl,
                                                             uint32_t* cacc, bool pair64) {
  constexpr int EPW = EP < 32 ? 32 : EP;
  constexpr int kTileWords = EPW * kFusedWaves;
  constexpr int kPer = (kTileWords + kFusedThreads - 1) / kFusedThreads;  // words per thread and chunk (1..4)
  typedef GramShape<EPW> GS;
  typedef typename Mfma<GS::TS>::Acc Acc;
  __shared__ __align__(16) u64 bt[2][kGramGroup][kTileWords];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l = (int)blockIdx.x / bpl, part = (int)blockIdx.x % bpl;
  if (l >= L) return;
  const int64_t nch = (W + kFusedWaves - 1) / kFusedWaves;
  const int64_t c0 = part * nch / bpl, c1 = (part + 1) * nch / bpl;
  if (c0 >= c1) return;
  const u64* lb = bits + (int64_t)l * E * sig_words(W);
  const WaveTiles wt = wave_tiles(GS::T, wave);
  Acc acc[kGP];
#pragma unroll
  for (int p = 0; p < kGP; ++p)
#pragma unroll
    for (int r = 0; r < Mfma<GS::TS>::kRegs; ++r) acc[p][r] = 0.0f;
  // thread tid holds words (e, s) = (idx / 8, idx % 8) for idx = tid + q * 512
  // of each chunk: a chunk is one unit of the signature layout, E * 64
  // contiguous bytes; chunks at or past c1 read as zero
  u64 r[kGramGroup][kPer];
  auto load = [&](int64_t g0) {
#pragma unroll
    for (int g = 0; g < kGramGroup; ++g)
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int idx = tid + q * kFusedThreads, e = idx >> 3;
        const int64_t w = (g0 + g) * kFusedWaves + (idx & 7);
        r[g][q] = (idx < kTileWords && g0 + g < c1 && e < E && w < W)
                      ? __builtin_nontemporal_load(lb + sig_off(w, e, E))
                      : 0ull;
      }
  };
  load(c0);
  int buf = 0;
  for (int64_t g0 = c0; g0 < c1; g0 += kGramGroup) {
#pragma unroll
    for (int g = 0; g < kGramGroup; ++g)
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int idx = tid + q * kFusedThreads, e = idx >> 3, sl = idx & 7;
        if (idx < kTileWords) bt[buf][g][sl * EPW + (e ^ bt_swz(sl))] = r[g][q];
      }
    // the tiles are complete; every wave is done with the tiles written two
    // steps ago (it multiplied those before reaching this barrier)
    __syncthreads();
    if (g0 + kGramGroup < c1) load(g0 + kGramGroup);
    const int ng = (int)min((int64_t)kGramGroup, c1 - g0);
    for (int g = 0; g < ng; ++g) mfma_slots<GS::TS>(acc, wt, bt[buf][g], EPW, 0, kFusedWaves, lane);
    buf ^= 1;
  }
  mfma_flush<GS::TS>(acc, wt, cacc + (int64_t)l * E * E, E, lane, (int)(blockIdx.x % kGP), pair64);
}

}  // namespace

hipError_t launch_topk(do_dtype dt, SegTable& tab, int nseg, const PathArgs& a, bool fast_ok, hipStream_t s,
                       const ProfEv& pe) {
  tab.nseg = nseg;
  tab.tile_start[0] = 0;
  for (int i = 0; i < nseg; ++i) {
    const int64_t n = tab.s[i].n, off = tab.s[i].tok_off;
    const int64_t words = n > 0 ? ((off + n - 1) >> 6) - (off >> 6) + 1 : 0;
    tab.tile_start[i + 1] = tab.tile_start[i] + (words + kFusedWaves - 1) / kFusedWaves;  // 8-word units
  }
  if (tab.tile_start[nseg] == 0) {  // nothing to launch: the timing events still complete, back to back
    if (pe.start != nullptr) {
      const hipError_t e = hipEventRecord(pe.start, s);
      if (e != hipSuccess) return e;
    }
    return pe.stop != nullptr ? hipEventRecord(pe.stop, s) : hipSuccess;
  }
  const bool fast = fast_ok && a.k <= kFastMaxK && a.E <= kFastMaxE;
  hipEvent_t ev[2] = {nullptr, nullptr};
  const int forced = g_opt_sched.load(std::memory_order_relaxed);
  const Sched sc = forced >= 0 ? kSchedCand[forced] : tuned_schedule(dt, tab, a, fast, s, ev);
  // a tuner trial binds its events to the dispatch (the kernel alone), unless
  // the caller's timing events already are; then they go around the launch
  ProfEv use = pe;
  const bool around = ev[0] != nullptr && (pe.start != nullptr || pe.stop != nullptr);
  if (ev[0] != nullptr && !around) use = ProfEv{ev[0], ev[1]};
  if (around) {
    const hipError_t e = hipEventRecord(ev[0], s);
    if (e != hipSuccess) return e;
  }
  const hipError_t e =
      dt == DO_F32 ? launch_ep<float>(tab, a, fast, sc, s, use) : launch_ep<uint16_t>(tab, a, fast, sc, s, use);
  if (e != hipSuccess || !around) return e;
  return hipEventRecord(ev[1], s);
}

bool gram_mfma_enabled() { return gram_mode() == kGramMfma; }

bool set_option(int opt, int value) {
  if (opt == DO_OPT_SCHEDULE && value >= -1 && value < kNumCand) {
    g_opt_sched.store(value, std::memory_order_relaxed);
    return true;
  }
  if (opt == DO_OPT_GRAM && (value == 0 || value == 1)) {
    g_opt_gram.store(value, std::memory_order_relaxed);
    return true;
  }
  return false;
}

hipError_t launch_gram_mfma(const u64* bits, int64_t W, int32_t E, int32_t L, uint32_t* cacc, hipStream_t s) {
  if (E > kFastMaxE || W < 1) return hipErrorInvalidValue;
  const int64_t nch = (W + kFusedWaves - 1) / kFusedWaves;
  const DevInfo di = device_info();
  // about as many blocks as fit on the GPU at once (two per CU up to 128
  // experts, one at 256 where the kernel takes 208 VGPRs), each below the
  // exact-count limit; every block flushes its counts with atomics at its end
  const int64_t per_cu = E <= 128 ? 2 : 1;
  int64_t bpl = std::max<int64_t>(1, ((int64_t)di.cu_count * per_cu + L - 1) / L);
  bpl = std::max<int64_t>(bpl, (nch + kGramMaxChunks - 1) / kGramMaxChunks);
  bpl = std::min<int64_t>(bpl, nch);
  if ((int64_t)L * bpl > 0x7FFFFFFF) return hipErrorInvalidValue;
  const bool pair64 = (E & 1) == 0 && (reinterpret_cast<uintptr_t>(cacc) & 7) == 0;
  const dim3 grid((unsigned)(L * bpl));
  if (E <= 32)
    hipLaunchKernelGGL(k_gram_mfma<32>, grid, dim3(kFusedThreads), 0, s, bits, W, E, L, (int)bpl, cacc, pair64);
  else if (E <= 64)
    hipLaunchKernelGGL(k_gram_mfma<64>, grid, dim3(kFusedThreads), 0, s, bits, W, E, L, (int)bpl, cacc, pair64);
  else if (E <= 128)
    hipLaunchKernelGGL(k_gram_mfma<128>, grid, dim3(kFusedThreads), 0, s, bits, W, E, L, (int)bpl, cacc, pair64);
  else
    hipLaunchKernelGGL(k_gram_mfma<256>, grid, dim3(kFusedThreads), 0, s, bits, W, E, L, (int)bpl, cacc, pair64);
  return hipGetLastError();
}

}  // namespace dol
