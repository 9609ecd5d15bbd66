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
// (double-buffered) from which the block writes them out as 64-byte runs and
// feeds the Gram.
//
// Exact Top-K with composite 32-bit keys.  Each element becomes one signed
// integer whose high bits order the score and whose low byte is (255 - expert
// index), so larger keys rank first and equal scores fall to the lower index.
// "Positive" keys use the raw bit pattern (one instruction, exact whenever the
// k-th score is a positive number); "general" keys first map the pattern to
// an order-preserving integer (exact for all non-NaN values except that -0
// sorts one step below +0).  bf16 keeps all 16 value bits; fp32 keeps 24, so
// a token is re-ranked exactly when its k-th and (k+1)-th keys share a 24-bit
// bucket.  Any token whose threshold lands on +-0, +-inf, NaN or a bucket tie,
// or whose threshold is not positive under positive keys, is re-ranked by an
// exact per-lane fallback on 64-bit keys.  bf16 always uses general keys (they
// cost it little); an fp32 wave starts with positive keys and switches to
// general keys for the rest of its tiles after meeting a non-positive threshold.
//
// Gram.  mode 2 (default): int8 MFMA 32x32x32 on 0/1 bytes expanded from the
// signature words, one or more 32x32 expert tile pairs per wave, accumulators
// in registers for the whole kernel.  mode 1: VALU popcount(a & b) on 4x4
// micro-tiles per thread.  Either way each block adds its integer partial
// counts into the accumulator matrix once at the end (order-independent).
#include <cstdlib>

#include "common.h"

namespace dol {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
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

#define DOL_CAS(a, b)          \
  {                            \
    const int hi_ = max(a, b); \
    const int lo_ = min(a, b); \
    a = hi_;                   \
    b = lo_;                   \
  }

// Batcher odd-even merge sort of 8 keys, descending (19 compare-exchanges).
__device__ __forceinline__ void sort8_desc(int (&g)[8]) {
  DOL_CAS(g[0], g[1]) DOL_CAS(g[2], g[3]) DOL_CAS(g[4], g[5]) DOL_CAS(g[6], g[7])
  DOL_CAS(g[0], g[2]) DOL_CAS(g[1], g[3]) DOL_CAS(g[4], g[6]) DOL_CAS(g[5], g[7])
  DOL_CAS(g[1], g[2]) DOL_CAS(g[5], g[6])
  DOL_CAS(g[0], g[4]) DOL_CAS(g[1], g[5]) DOL_CAS(g[2], g[6]) DOL_CAS(g[3], g[7])
  DOL_CAS(g[2], g[4]) DOL_CAS(g[3], g[5])
  DOL_CAS(g[1], g[2]) DOL_CAS(g[3], g[4]) DOL_CAS(g[5], g[6])
}

// top <- the 8 largest of top and g (both sorted descending); with TRACK,
// rej <- max(rej, largest key dropped), i.e. the running 9th largest.
template <bool TRACK>
__device__ __forceinline__ void merge8(int (&top)[8], const int (&g)[8], int& rej) {
  int m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = max(top[i], g[7 - i]);
  if (TRACK) {
    const int r0 = max(min(top[0], g[7]), min(top[1], g[6]));
    const int r1 = max(min(top[2], g[5]), min(top[3], g[4]));
    const int r2 = max(min(top[4], g[3]), min(top[5], g[2]));
    const int r3 = max(min(top[6], g[1]), min(top[7], g[0]));
    rej = max(max(rej, max(r0, r1)), max(r2, r3));
  }
  DOL_CAS(m[0], m[4]) DOL_CAS(m[1], m[5]) DOL_CAS(m[2], m[6]) DOL_CAS(m[3], m[7])
  DOL_CAS(m[0], m[2]) DOL_CAS(m[1], m[3]) DOL_CAS(m[4], m[6]) DOL_CAS(m[5], m[7])
  DOL_CAS(m[0], m[1]) DOL_CAS(m[2], m[3]) DOL_CAS(m[4], m[5]) DOL_CAS(m[6], m[7])
#pragma unroll
  for (int i = 0; i < 8; ++i) top[i] = m[i];
}

// (x & mask) | (y & ~mask) in one instruction.  Written out because the
// compiler otherwise splits it into AND + OR: gfx9 VOP3 encodings take no
// literal, so the mask sits in a VGPR and the expert index in an SGPR.
__device__ __forceinline__ uint32_t bfi(uint32_t vmask, uint32_t x, uint32_t sidx) {
  uint32_t r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(vmask), "v"(x), "s"(sidx));
  return r;
}

// Composite keys.  e: expert index (< 256).  vm24 = 0xFFFFFF00, vm16 = 0xFFFF0000 (VGPRs).
template <bool GEN>
__device__ __forceinline__ int key_f32(uint32_t u, int e, uint32_t vm24) {
  if (GEN) u ^= (uint32_t)((int32_t)u >> 31) & 0x7FFFFF00u;
  return (int)bfi(vm24, u, (uint32_t)(255 - e));
}

// Two bf16 scores packed in x (element e0 in the low half, e0 + 1 in the high half).
template <bool GEN>
__device__ __forceinline__ void key_bf16x2(uint32_t x, int e0, uint32_t vm16, int& lo, int& hi) {
  if (GEN) {
    const v2s s = __builtin_bit_cast(v2s, x) >> (short)15;
    x ^= __builtin_bit_cast(uint32_t, s) & 0x7FFF7FFFu;
  }
  lo = (int)((x << 16) | (uint32_t)(255 - e0));
  hi = (int)bfi(vm16, x, (uint32_t)(254 - e0));
}

// Rank one staged 128-byte chunk (vectors cv0..cv0+7 of the lane's row) into top/rej.
template <typename T, bool GEN>
__device__ __forceinline__ void rank_chunk(const unsigned char* sbuf, int lane, int cv0, uint32_t vmask,
                                           int (&top)[8], int& rej) {
  const unsigned char* row = sbuf + lane * 128;
  const int sw = row_swizzle(lane);
  auto piece = [&](int q) { return *reinterpret_cast<const v4u*>(row + ((q ^ sw) << 4)); };
  if (Traits<T>::kVec == 4) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      int g[8];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const v4u x = piece(2 * gq + h);
        const int e0 = (cv0 + 2 * gq + h) * 4;
        g[4 * h + 0] = key_f32<GEN>(x.x, e0 + 0, vmask);
        g[4 * h + 1] = key_f32<GEN>(x.y, e0 + 1, vmask);
        g[4 * h + 2] = key_f32<GEN>(x.z, e0 + 2, vmask);
        g[4 * h + 3] = key_f32<GEN>(x.w, e0 + 3, vmask);
      }
      sort8_desc(g);
      merge8<!Traits<T>::kExact>(top, g, rej);
    }
  } else {
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      int g[8];
      const v4u x = piece(v);
      const int e0 = (cv0 + v) * 8;
      key_bf16x2<GEN>(x.x, e0 + 0, vmask, g[0], g[1]);
      key_bf16x2<GEN>(x.y, e0 + 2, vmask, g[2], g[3]);
      key_bf16x2<GEN>(x.z, e0 + 4, vmask, g[4], g[5]);
      key_bf16x2<GEN>(x.w, e0 + 6, vmask, g[6], g[7]);
      sort8_desc(g);
      merge8<false>(top, g, rej);
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

// Exact Top-k (k <= 8) of one row in a single pass: insertion of unique
// 64-bit keys (value key, then the complemented index) into a sorted list.
template <typename T>
__device__ void exact_topk8_lane(const T* row, int E, int k, u64* bt, int swz, u64 bit) {
  u64 lst[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) lst[i] = 0ull;  // every real key is > 0
  for (int e = 0; e < E; ++e) {
    const u64 key = exact_key64(elem_bits<T>(row, e), e);
    if (key <= lst[7]) continue;
#pragma unroll
    for (int i = 7; i > 0; --i) lst[i] = max(lst[i], min(lst[i - 1], key));
    lst[0] = max(lst[0], key);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
    if (i < k) atomicOr(&bt[(int)(0xFFFFFFFFu - (uint32_t)(lst[i] & 0xFFFFFFFFull)) ^ swz], bit);
}

// Exact Top-k for any k: k selection passes, each taking the largest key
// below the previous one.
template <typename T>
__device__ void exact_topk_passes_lane(const T* row, int E, int k, u64* bt, int swz, u64 bit) {
  u64 prev = ~0ull;
  for (int r = 0; r < k; ++r) {
    u64 best = 0;
    for (int e = 0; e < E; ++e) {
      const u64 key = exact_key64(elem_bits<T>(row, e), e);
      if (key < prev && key > best) best = key;
    }
    atomicOr(&bt[(int)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFull)) ^ swz], bit);
    prev = best;
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

  // bt: nslot signature words per expert, slot-major with `stride` words per slot
  __device__ __forceinline__ void accumulate(const u64* bt, int nslot, int stride) {
    for (int s = 0; s < nslot; ++s) {
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
// MFMA Gram.  Expert tiles of 32; the tile pairs (I <= J) of the upper
// triangle are split over the 8 waves so that each wave needs few distinct
// tiles (each tile costs one bits->bytes expansion per 32 tokens).
// ---------------------------------------------------------------------------
constexpr int kMaxPairs = 5;  // per wave (T = 8)


constexpr int kMaxTiles = 4;  // distinct tiles per wave

struct WavePairs {
  int nt, np;
  int tile[kMaxTiles];
  int pa[kMaxPairs], pb[kMaxPairs];  // indices into tile[]
};

// T = 8 tiles (E <= 256): 36 pairs, 4-5 pairs and 3-4 tiles per wave.
constexpr WavePairs kPairs8[8] = {
    {3, 4, {2, 6, 7, 0}, {0, 0, 1, 2}, {1, 2, 2, 2}},        // (2,6)(2,7)(6,7)(7,7)
    {4, 5, {1, 3, 5, 7}, {0, 0, 1, 1, 2}, {1, 3, 2, 3, 3}},  // (1,3)(1,7)(3,5)(3,7)(5,7)
    {3, 4, {4, 5, 6, 0}, {0, 0, 1, 1}, {1, 2, 1, 2}},        // (4,5)(4,6)(5,5)(5,6)
    {4, 4, {0, 2, 3, 4}, {0, 1, 2, 2}, {2, 2, 2, 3}},        // (0,3)(2,3)(3,3)(3,4)
    {3, 5, {1, 2, 4, 0}, {0, 0, 1, 1, 2}, {1, 2, 1, 2, 2}},  // (1,2)(1,4)(2,2)(2,4)(4,4)
    {4, 4, {1, 3, 5, 6}, {0, 0, 1, 3}, {2, 3, 3, 3}},        // (1,5)(1,6)(3,6)(6,6)
    {4, 5, {0, 1, 2, 5}, {0, 0, 0, 1, 2}, {1, 2, 3, 1, 3}},  // (0,1)(0,2)(0,5)(1,1)(2,5)
    {4, 5, {0, 4, 6, 7}, {0, 0, 0, 0, 1}, {0, 1, 2, 3, 3}},  // (0,0)(0,4)(0,6)(0,7)(4,7)
};
// T = 4 tiles (E <= 128): 10 pairs.
constexpr WavePairs kPairs4[8] = {
    {2, 2, {2, 3, 0, 0}, {0, 1}, {1, 1}},  // (2,3)(3,3)
    {2, 2, {1, 3, 0, 0}, {0, 0}, {0, 1}},  // (1,1)(1,3)
    {2, 2, {0, 1, 0, 0}, {0, 0}, {0, 1}},  // (0,0)(0,1)
    {2, 2, {0, 2, 0, 0}, {0, 1}, {1, 1}},  // (0,2)(2,2)
    {2, 1, {0, 3, 0, 0}, {0}, {1}},        // (0,3)
    {2, 1, {1, 2, 0, 0}, {0}, {1}},        // (1,2)
    {0, 0, {0, 0, 0, 0}, {0}, {0}},
    {0, 0, {0, 0, 0, 0}, {0}, {0}},
};
// T = 2 tiles (E <= 64): 3 pairs.
constexpr WavePairs kPairs2[8] = {
    {1, 1, {0, 0, 0, 0}, {0}, {0}},  // (0,0)
    {2, 1, {0, 1, 0, 0}, {0}, {1}},  // (0,1)
    {1, 1, {1, 0, 0, 0}, {0}, {0}},  // (1,1)
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
};
// T = 1 tile (E <= 32).
constexpr WavePairs kPairs1[8] = {
    {1, 1, {0, 0, 0, 0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
    {0, 0, {0}, {0}, {0}},
};

template <int T, int W>
struct PairsOf {
  static constexpr WavePairs v = T == 8 ? kPairs8[W] : T == 4 ? kPairs4[W] : T == 2 ? kPairs2[W] : kPairs1[W];
};

// 16 signature bits -> 16 bytes of 0/1 (byte b = bit b).
__device__ __forceinline__ v4i expand16(uint32_t b) {
  v4i r;
  r.x = (int)((((b >> 0) & 0xFu) * 0x00204081u) & 0x01010101u);
  r.y = (int)((((b >> 4) & 0xFu) * 0x00204081u) & 0x01010101u);
  r.z = (int)((((b >> 8) & 0xFu) * 0x00204081u) & 0x01010101u);
  r.w = (int)((((b >> 12) & 0xFu) * 0x00204081u) & 0x01010101u);
  return r;
}

// MFMA shapes for TS-expert tiles.  A and B operands of lane l hold the same
// k indices, so one expanded fragment serves as both operands of a Gram.
//   TS = 32: v_mfma_i32_32x32x32_i8, lane l = expert l%32, k-step ks covers
//            tokens 32*ks + 16*(l/32) .. +15 of the word; C row 8*(r/4)+4*(l/32)+r%4, col l%32
//   TS = 16: v_mfma_i32_16x16x64_i8, lane l = expert l%16, tokens 16*(l/16) .. +15;
//            C row 4*(l/16)+r, col l%16
template <int TS>
struct Mfma;
template <>
struct Mfma<32> {
  typedef v16i Acc;
  static constexpr int kSteps = 2, kRegs = 16;
  __device__ static __forceinline__ int expert(int tile, int lane) { return tile * 32 + (lane & 31); }
  __device__ static __forceinline__ int chunk16(int ks, int lane) { return ks * 2 + (lane >> 5); }
  __device__ static __forceinline__ Acc mac(v4i a, v4i b, Acc c) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ int row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
  __device__ static __forceinline__ int col(int lane) { return lane & 31; }
};
template <>
struct Mfma<16> {
  typedef v4i Acc;
  static constexpr int kSteps = 1, kRegs = 4;
  __device__ static __forceinline__ int expert(int tile, int lane) { return tile * 16 + (lane & 15); }
  __device__ static __forceinline__ int chunk16(int, int lane) { return lane >> 4; }
  __device__ static __forceinline__ Acc mac(v4i a, v4i b, Acc c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
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
  static constexpr int MP = T == 8 ? 5 : T == 4 ? 2 : 1;  // tile pairs per wave at most
};

// Accumulate the wave's tile pairs over `nslot` words of the bit tile.
template <int TS, int T, int W>
__device__ __forceinline__ void mfma_wave(typename Mfma<TS>::Acc (&acc)[GramShape<T * TS>::MP], const u64* bt,
                                          int stride, int nslot, int lane) {
  constexpr WavePairs P = PairsOf<T, W>::v;
  if (P.np == 0) return;
#pragma unroll 1
  for (int s = 0; s < nslot; ++s) {  // not unrolled: keeps the fragment registers to one word's worth
    const uint16_t* w16 = reinterpret_cast<const uint16_t*>(bt + s * stride);
#pragma unroll
    for (int ks = 0; ks < Mfma<TS>::kSteps; ++ks) {
      v4i f[kMaxTiles];
#pragma unroll
      for (int t = 0; t < P.nt; ++t)
        f[t] = expand16(w16[(Mfma<TS>::expert(P.tile[t], lane) ^ bt_swz(s)) * 4 + Mfma<TS>::chunk16(ks, lane)]);
#pragma unroll
      for (int p = 0; p < P.np; ++p) acc[p] = Mfma<TS>::mac(f[P.pa[p]], f[P.pb[p]], acc[p]);
    }
  }
}

// Add the wave's partial counts into c (upper triangle, integer atomics).
template <int TS, int T, int W>
__device__ __forceinline__ void mfma_flush(const typename Mfma<TS>::Acc (&acc)[GramShape<T * TS>::MP], uint32_t* c,
                                           int E, int lane) {
  constexpr WavePairs P = PairsOf<T, W>::v;
#pragma unroll
  for (int p = 0; p < P.np; ++p) {
    const int I = P.tile[P.pa[p]], J = P.tile[P.pb[p]];
#pragma unroll
    for (int r = 0; r < Mfma<TS>::kRegs; ++r) {
      const int gi = TS * I + Mfma<TS>::row(r, lane);
      const int gj = TS * J + Mfma<TS>::col(lane);
      const uint32_t v = (uint32_t)acc[p][r];
      if (gi <= gj && gj < E && v) atomicAdd(&c[(int64_t)gi * E + gj], v);
    }
  }
}

template <int TS, int T>
__device__ __forceinline__ void mfma_dispatch(int wave, typename Mfma<TS>::Acc (&acc)[GramShape<T * TS>::MP],
                                              const u64* bt, int stride, int nslot, int lane) {
  switch (wave) {
    case 0: mfma_wave<TS, T, 0>(acc, bt, stride, nslot, lane); break;
    case 1: mfma_wave<TS, T, 1>(acc, bt, stride, nslot, lane); break;
    case 2: mfma_wave<TS, T, 2>(acc, bt, stride, nslot, lane); break;
    case 3: mfma_wave<TS, T, 3>(acc, bt, stride, nslot, lane); break;
    case 4: mfma_wave<TS, T, 4>(acc, bt, stride, nslot, lane); break;
    case 5: mfma_wave<TS, T, 5>(acc, bt, stride, nslot, lane); break;
    case 6: mfma_wave<TS, T, 6>(acc, bt, stride, nslot, lane); break;
    default: mfma_wave<TS, T, 7>(acc, bt, stride, nslot, lane); break;
  }
}

template <int TS, int T>
__device__ __forceinline__ void mfma_flush_dispatch(int wave, const typename Mfma<TS>::Acc (&acc)[GramShape<T * TS>::MP],
                                                    uint32_t* c, int E, int lane) {
  switch (wave) {
    case 0: mfma_flush<TS, T, 0>(acc, c, E, lane); break;
    case 1: mfma_flush<TS, T, 1>(acc, c, E, lane); break;
    case 2: mfma_flush<TS, T, 2>(acc, c, E, lane); break;
    case 3: mfma_flush<TS, T, 3>(acc, c, E, lane); break;
    case 4: mfma_flush<TS, T, 4>(acc, c, E, lane); break;
    case 5: mfma_flush<TS, T, 5>(acc, c, E, lane); break;
    case 6: mfma_flush<TS, T, 6>(acc, c, E, lane); break;
    default: mfma_flush<TS, T, 7>(acc, c, E, lane); break;
  }
}

#define DOL_WAVE_FENCE() asm volatile("" ::: "memory")

// Per-segment view used by the kernel.
struct SegView {
  const unsigned char* base;
  int64_t n, off, w_first, words;  // words: signature words this segment covers
  int64_t u_begin, u_end;          // its range of global 8-word units
  int layer;
};

__device__ __forceinline__ SegView seg_view(const SegTable& tab, int i) {
  SegView v;
  v.base = reinterpret_cast<const unsigned char*>(tab.s[i].scores);
  v.n = tab.s[i].n;
  v.off = tab.s[i].tok_off;
  v.w_first = v.off >> 6;
  v.words = v.n > 0 ? ((v.off + v.n - 1) >> 6) - v.w_first + 1 : 0;
  v.u_begin = tab.tile_start[i];
  v.u_end = tab.tile_start[i + 1];
  v.layer = tab.s[i].layer;
  return v;
}

// Segment holding global unit u (segments with no units are skipped).
__device__ __forceinline__ int seg_of(const SegTable& tab, int64_t u, int from) {
  int i = from;
  while (i + 1 < tab.nseg && u >= tab.tile_start[i + 1]) ++i;
  return i;
}

typedef unsigned long long v2u64 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Top-K (+ Gram) kernel.  Work unit: 8 consecutive signature words (512
// output positions) of one segment, starting 8-aligned within it; one unit
// per block step, one word (64 tokens) per wave.  One persistent block per CU
// slot takes the contiguous unit range [b*U/G, (b+1)*U/G).  Gram
// accumulators are flushed whenever the next unit belongs to another layer,
// and at the end.  flags bit 0: fast path allowed (16-byte rows, k <= 8,
// E <= 256).
// ---------------------------------------------------------------------------
template <typename T, int EP, int GM>
__global__ __launch_bounds__(kFusedThreads) void k_topk(const SegTable tab, const PathArgs a, int flags) {
  constexpr int EPW = EP < 32 ? 32 : EP;  // signature words per slot of the bit tile
  typedef GramShape<EPW> GS;
  typedef typename Mfma<GS::TS>::Acc Acc;
  extern __shared__ __align__(16) unsigned char smem[];
  const bool fast = (flags & 1) != 0;
  unsigned char* stage_all = smem;
  u64* bt_all = reinterpret_cast<u64*>(smem + (fast ? kStageBytes : 0));  // [2][kFusedWaves][EPW]

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int E = a.E, k = a.k;
  const int rowB = E * (int)sizeof(T);
  const int rowv = rowB >> 4;
  const int nch = (rowv + 7) >> 3;
  unsigned char* st = stage_all + wave * 2 * kChunkBytes;  // this wave's two stage buffers

  const int64_t U = tab.tile_start[tab.nseg];
  const int64_t ug = (int64_t)blockIdx.x * U / gridDim.x;
  const int64_t ue = (int64_t)(blockIdx.x + 1) * U / gridDim.x;
  if (ug >= ue) return;

  PopcGram<EPW, kFusedThreads, GM == kGramPopc> pg;
  if (GM == kGramPopc) pg.init(tid, E);
  Acc acc[GS::MP];
  auto zero_acc = [&]() {
#pragma unroll
    for (int p = 0; p < GS::MP; ++p)
#pragma unroll
      for (int r = 0; r < Mfma<GS::TS>::kRegs; ++r) acc[p][r] = 0;
  };
  zero_acc();

  // Lane offsets inside a chunk: instruction j fills rows 8j..8j+7; lane i
  // fills slot (i & 7) of row 8j + i/8, which holds piece
  // q = (i & 7) ^ swz(8j + i/8) = (i & 7) ^ (i >> 3) ^ (j & 1).
  const int q_even = (lane & 7) ^ (lane >> 3);
  const uint32_t off_even = (uint32_t)((lane >> 3) * rowB + q_even * 16);        // bytes from the chunk's row 0
  const uint32_t off_odd = (uint32_t)((lane >> 3) * rowB + (q_even ^ 1) * 16);  // odd j: piece q_even ^ 1

  // Direct-to-LDS load of a full 64-row x 128-byte chunk of local word `tl` of
  // segment `sv` (asynchronous; the consumer waits with DOL_WAIT_VMEM).
  auto dma = [&](const SegView& sv, int64_t tl, int c_, unsigned char* sbuf) {
    if (c_ * 8 + 8 > rowv) return;
    const int64_t t0_ = (sv.w_first + tl) * 64 - sv.off;
    const unsigned char* cbase = sv.base + t0_ * rowB + c_ * 128;  // row 0 of the chunk (uniform)
    if (t0_ >= 0 && t0_ + 64 <= sv.n) {  // every row inside the segment
#pragma unroll
      for (int j = 0; j < 8; ++j)
        __builtin_amdgcn_global_load_lds(cbase + (uint32_t)(j * 8 * rowB) + ((j & 1) ? off_odd : off_even),
                                         (__attribute__((address_space(3))) void*)(sbuf + j * 1024), 16, 0, kStreamPolicy);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int64_t tr = t0_ + 8 * j + (lane >> 3);
        if (tr >= 0 && tr < sv.n)
          __builtin_amdgcn_global_load_lds(cbase + (uint32_t)(j * 8 * rowB) + ((j & 1) ? off_odd : off_even),
                                           (__attribute__((address_space(3))) void*)(sbuf + j * 1024), 16, 0, kStreamPolicy);
      }
    }
  };
  // Synchronous fill of a partial chunk (the row ends inside it): missing
  // vectors read as all-ones (a NaN), ranked last and never selected on the fast path.
  auto fill_partial = [&](const SegView& sv, int64_t t0_, int c_, unsigned char* sbuf) {
    const int cvn = rowv - c_ * 8;
    const unsigned char* cbase = sv.base + t0_ * rowB + c_ * 128;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t tr = t0_ + 8 * j + (lane >> 3);
      const int q = q_even ^ (j & 1);
      v4u val = v4u{~0u, ~0u, ~0u, ~0u};
      if (q < cvn && tr >= 0 && tr < sv.n)
        val = *reinterpret_cast<const v4u*>(cbase + (uint32_t)(j * 8 * rowB) + ((j & 1) ? off_odd : off_even));
      *reinterpret_cast<v4u*>(sbuf + j * 1024 + lane * 16) = val;
    }
  };

  // General keys cost bf16 ~0.75 extra instructions per score and fp32 ~3, so
  // bf16 starts with them; an fp32 wave switches after meeting a non-positive threshold.
  bool gen = Traits<T>::kExact;
  int cb = 0;  // stage buffer holding the current chunk
  const uint32_t vmask = Traits<T>::kExact ? 0xFFFF0000u : 0xFFFFFF00u;  // value bits of a key (VGPR operand of bfi)

  int seg = seg_of(tab, ug, 0);
  SegView sv = seg_view(tab, seg);
  {
    const int64_t tl = 8 * (ug - sv.u_begin) + wave;
    if (fast && tl < sv.words) dma(sv, tl, 0, st);
  }

  int buf = 0;
  int64_t u = ug;
  while (u < ue) {  // one run of units within one layer, then a flush
    const int run_layer = sv.layer;
    for (; u < ue && sv.layer == run_layer; buf ^= 1) {
      const int64_t tl0 = 8 * (u - sv.u_begin);                  // local word of slot 0
      const int64_t cnt = min((int64_t)kFusedWaves, sv.words - tl0);  // words in this unit
      // next unit and its segment (block-uniform)
      const int64_t un = u + 1;
      const int seg_n = (un < ue) ? seg_of(tab, un, seg) : seg;
      const SegView svn = seg_view(tab, seg_n);
      const int64_t tln = 8 * (un - svn.u_begin) + wave;  // this wave's word in the next unit
      const bool next_mine = un < ue && tln < svn.words;

      u64* bt = bt_all + buf * kFusedWaves * EPW;
      u64* mybt = bt + wave * EPW;
#pragma unroll
      for (int e0 = 0; e0 < EPW; e0 += 64)
        if (e0 + lane < EPW) mybt[e0 + lane] = 0;
      DOL_WAVE_FENCE();
      if (fast && wave >= cnt && next_mine) {
        // idle in this unit (segment end) but busy in the next one: start that
        // word's first chunk now, into the buffer the next unit reads first
        dma(svn, tln, 0, st + cb * kChunkBytes);
      }
      if (wave < cnt) {
        const int64_t tl = tl0 + wave;
        const int64_t t0 = (sv.w_first + tl) * 64 - sv.off;  // token of lane 0 (negative in a history's first partial word)
        const int64_t t = t0 + lane;
        const bool valid = (t >= 0) && (t < sv.n);
        bool need_slow = valid;
        if (fast) {
          int top[8];
          int rej = INT_MIN;
#pragma unroll
          for (int i = 0; i < 8; ++i) top[i] = INT_MIN;
          for (int c = 0; c < nch; ++c) {
            unsigned char* cur = st + cb * kChunkBytes;
            if (c * 8 + 8 <= rowv) {
              DOL_WAIT_VMEM();  // this chunk's direct-to-LDS loads have landed
            } else {
              fill_partial(sv, t0, c, cur);
            }
            DOL_WAVE_FENCE();
            unsigned char* other = st + (cb ^ 1) * kChunkBytes;
            if (c + 1 < nch)
              dma(sv, tl, c + 1, other);
            else if (next_mine)
              dma(svn, tln, 0, other);
            if (gen)
              rank_chunk<T, true>(cur, lane, c * 8, vmask, top, rej);
            else
              rank_chunk<T, false>(cur, lane, c * 8, vmask, top, rej);
            DOL_WAVE_FENCE();
            cb ^= 1;
          }
          int sk = INT_MIN, sk1 = rej;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            sk = (i == k - 1) ? top[i] : sk;
            sk1 = (i == k) ? top[i] : sk1;
          }
          bool ok = top[0] < kCompPosInf;
          bool nonpos = false;
          if (gen) {
            ok = ok && sk > kCompNegInfMax && (sk < Traits<T>::kZeroLo || sk > Traits<T>::kZeroHi);
          } else {
            nonpos = valid && sk < Traits<T>::kPosMin;
            ok = ok && !nonpos;
          }
          if (!Traits<T>::kExact) ok = ok && ((sk1 >> 8) < (sk >> 8));
          need_slow = valid && !ok;
          if (valid && ok) {
            const u64 bit = 1ull << lane;
#pragma unroll
            for (int i = 0; i < 8; ++i)
              if (i < k) atomicOr(&mybt[(255 - (top[i] & 255)) ^ bt_swz(wave)], bit);
          }
          if (__ballot(nonpos) != 0ull) gen = true;
        }
        if (__ballot(need_slow) != 0ull) {
          if (need_slow) {
            const T* row = reinterpret_cast<const T*>(sv.base) + t * (int64_t)E;
            if (k <= 8)
              exact_topk8_lane<T>(row, E, k, mybt, bt_swz(wave), 1ull << lane);
            else
              exact_topk_passes_lane<T>(row, E, k, mybt, bt_swz(wave), 1ull << lane);
          }
        }
      }
      __syncthreads();
      // signatures of the unit's words: pairs of words as 16-byte stores
      // (8-aligned units make them 16-byte aligned unless the history starts
      // mid-word), partial history words OR-ed in
      // One wave per unit (rotating) issues all of the unit's stores, so only
      // it later waits for their completion in its next vmcnt(0).
      if (a.bits != nullptr && wave == (int)(u & 7)) {
        u64* lb = a.bits + (int64_t)sv.layer * a.bits_layer_words;
        const int64_t w0 = sv.w_first + tl0;
        auto plain = [&](int s_) {
          const int64_t t0s = (w0 + s_) * 64 - sv.off;
          return !a.or_partial || (t0s >= 0 && t0s + 64 <= sv.n);
        };
        auto put = [&](int e_, int s_, u64 word) {
          u64* dst = lb + (int64_t)e_ * a.W + w0 + s_;
          if (plain(s_))
            *dst = word;
          else if (word)
            atomicOr(dst, word);
        };
        if ((w0 & 1) == 0) {
          for (int item = lane; item < E * 4; item += kWave) {
            const int e = item >> 2, s0 = (item & 3) * 2;
            if (s0 >= cnt) continue;
            const u64 wa = bt[s0 * EPW + (e ^ bt_swz(s0))];
            const u64 wb = bt[(s0 + 1) * EPW + (e ^ bt_swz(s0 + 1))];
            if (s0 + 1 < cnt && plain(s0) && plain(s0 + 1)) {
              *reinterpret_cast<v2u64*>(lb + (int64_t)e * a.W + w0 + s0) = v2u64{wa, wb};
            } else {
              put(e, s0, wa);
              if (s0 + 1 < cnt) put(e, s0 + 1, wb);
            }
          }
        } else {
          for (int item = lane; item < E * kFusedWaves; item += kWave) {
            const int e = item >> 3, s0 = item & 7;
            if (s0 < cnt) put(e, s0, bt[s0 * EPW + (e ^ bt_swz(s0))]);
          }
        }
      }
      if (GM == kGramMfma) mfma_dispatch<GS::TS, GS::T>(wave, acc, bt, EPW, kFusedWaves, lane);  // empty slots are zero
      if (GM == kGramPopc) pg.accumulate(bt, (int)cnt, EPW);
      u = un;
      seg = seg_n;
      sv = svn;
    }
    if (GM != kGramNone) {
      uint32_t* cl = a.cacc + (int64_t)run_layer * a.cacc_layer_elems;
      if (GM == kGramMfma) {
        mfma_flush_dispatch<GS::TS, GS::T>(wave, acc, cl, E, lane);
        zero_acc();
      }
      if (GM == kGramPopc) {
        pg.flush(cl, E);
        pg.init(tid, E);
      }
    }
  }
}

int g_gram_mode = -1;  // kGramPopc or kGramMfma; read once from DOLOSS_GRAM ("popc" selects popcount)

int gram_mode() {
  if (g_gram_mode < 0) {
    const char* v = getenv("DOLOSS_GRAM");
    g_gram_mode = (v != nullptr && v[0] == 'p') ? kGramPopc : kGramMfma;
  }
  return g_gram_mode;
}

template <typename T, int EP, int GM>
hipError_t launch_one(const SegTable& tab, const PathArgs& a, bool fast, hipStream_t s) {
  constexpr int EPW = EP < 32 ? 32 : EP;
  auto kern = k_topk<T, EP, GM>;
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
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kFusedThreads), lds, s, tab, a, fast ? 1 : 0);
  return hipGetLastError();
}

template <typename T, int EP>
hipError_t launch_gm(const SegTable& tab, const PathArgs& a, bool fast, hipStream_t s) {
  if (a.cacc == nullptr) return launch_one<T, EP, kGramNone>(tab, a, fast, s);
  if (gram_mode() == kGramPopc) return launch_one<T, EP, kGramPopc>(tab, a, fast, s);
  return launch_one<T, EP, kGramMfma>(tab, a, fast, s);
}

template <typename T>
hipError_t launch_ep(const SegTable& tab, const PathArgs& a, bool fast, hipStream_t s) {
  const int E = a.E;
  if (E <= 32) return launch_gm<T, 32>(tab, a, fast, s);
  if (E <= 64) return launch_gm<T, 64>(tab, a, fast, s);
  if (E <= 128) return launch_gm<T, 128>(tab, a, fast, s);
  if (E <= 256) return launch_gm<T, 256>(tab, a, fast, s);
  // E in (256, 1024]: exact per-lane selection, signatures only
  if (a.cacc != nullptr) return hipErrorInvalidValue;
  if (E <= 512) return launch_one<T, 512, kGramNone>(tab, a, false, s);
  return launch_one<T, 1024, kGramNone>(tab, a, false, s);
}

}  // namespace

hipError_t launch_topk(do_dtype dt, SegTable& tab, int nseg, const PathArgs& a, bool fast_ok, hipStream_t s) {
  tab.nseg = nseg;
  tab.tile_start[0] = 0;
  for (int i = 0; i < nseg; ++i) {
    const int64_t n = tab.s[i].n, off = tab.s[i].tok_off;
    const int64_t words = n > 0 ? ((off + n - 1) >> 6) - (off >> 6) + 1 : 0;
    tab.tile_start[i + 1] = tab.tile_start[i] + (words + kFusedWaves - 1) / kFusedWaves;  // 8-word units
  }
  if (tab.tile_start[nseg] == 0) return hipSuccess;
  const bool fast = fast_ok && a.k <= kFastMaxK && a.E <= kFastMaxE;
  return dt == DO_F32 ? launch_ep<float>(tab, a, fast, s) : launch_ep<uint16_t>(tab, a, fast, s);
}

}  // namespace dol
