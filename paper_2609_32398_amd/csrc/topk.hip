// Router Top-K, signature packing and (optionally) the co-occurrence Gram of
// the DO-loss path, in one pass over the scores.
//
// Paper: Sec. 3.1.1, Eq. (1) -- f_it = 1 iff expert i is in the Top-K of
// token t; the binary load signature F_i collects f_it over the batch.
// Sec. 3.1.3, Eq. (6) and App. C.3 -- ||F_i - F_j||_1 = c_ii + c_jj - 2 c_ij
// with c_ij = sum_t f_it f_jt, which is what the Gram part accumulates.
//
// Layout of the work: one wavefront owns 64 consecutive output bit positions
// (one signature word per expert); lane l ranks token (64*w + l - tok_off).
// Score rows are streamed through LDS in 128-byte column chunks so that the
// global loads are fully coalesced, then every lane reads its own row back.
//
// Exact Top-K with a composite 32-bit key per element: the score's bits are
// mapped to an order-preserving signed integer, the low byte (fp32) or the
// low half (bf16) is replaced by (255 - expert index), so larger keys rank
// first and equal values fall to the lower index.  bf16 keeps its full 16-bit
// value, so the key order is exact; fp32 keeps the top 24 bits, so a token is
// re-ranked exactly when the k-th and (k+1)-th keys share a 24-bit bucket.
// Signed zeros, infinities and NaN near the threshold also send the token to
// the exact per-lane fallback (64-bit keys, k selection passes).
#include "common.h"

namespace dol {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kStageStride = 144;  // bytes per staged row: 8 x 16-byte vectors + 16 bytes of padding

template <typename T>
struct Traits;
template <>
struct Traits<float> {
  static constexpr int kVec = 4;                    // elements per 16-byte vector
  static constexpr uint32_t kHiMask = 0xFFFFFF00u;  // kept value bits of a composite key
  static constexpr bool kExact = false;
  static constexpr int kZeroLo = -256, kZeroHi = 255;  // composite keys of the -0 / +0 buckets
};
template <>
struct Traits<uint16_t> {
  static constexpr int kVec = 8;
  static constexpr uint32_t kHiMask = 0xFFFF0000u;
  static constexpr bool kExact = true;
  static constexpr int kZeroLo = -65536, kZeroHi = 65535;
};

constexpr int kCompPosInf = 0x7F800000;        // composite >= this: +inf or NaN
constexpr int kCompNegInfMax = (int)0x807FFFFF; // composite <= this: -inf or NaN

// u: fp32 bit pattern (bf16 widened by << 16).  Order-preserving for all
// non-NaN values except that -0 sorts one step below +0.
__device__ __forceinline__ int composite(uint32_t u, uint32_t himask, int e) {
  const uint32_t m = (uint32_t)((int32_t)u >> 31) & 0x7FFFFFFFu;
  return (int)(((u ^ m) & himask) | (uint32_t)(255 - e));
}

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

// top <- the 8 largest of top (sorted desc) and g (sorted desc); with
// TRACK, rej <- max(rej, largest key dropped).
template <bool TRACK>
__device__ __forceinline__ void merge8(int (&top)[8], const int (&g)[8], int& rej) {
  int m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    m[i] = max(top[i], g[7 - i]);
    if (TRACK) rej = max(rej, min(top[i], g[7 - i]));
  }
  DOL_CAS(m[0], m[4]) DOL_CAS(m[1], m[5]) DOL_CAS(m[2], m[6]) DOL_CAS(m[3], m[7])
  DOL_CAS(m[0], m[2]) DOL_CAS(m[1], m[3]) DOL_CAS(m[4], m[6]) DOL_CAS(m[5], m[7])
  DOL_CAS(m[0], m[1]) DOL_CAS(m[2], m[3]) DOL_CAS(m[4], m[5]) DOL_CAS(m[6], m[7])
#pragma unroll
  for (int i = 0; i < 8; ++i) top[i] = m[i];
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

// Exact Top-k of one row by k selection passes over unique 64-bit keys
// (value key, then the complemented index); sets the lane's bit of each
// chosen expert's word in `bt`.
template <typename T>
__device__ void slow_topk_lane(const T* row, int E, int k, u64* bt, u64 bit) {
  u64 prev = ~0ull;
  for (int r = 0; r < k; ++r) {
    u64 best = 0;
    for (int e = 0; e < E; ++e) {
      const u64 key = ((u64)exact_key(elem_bits<T>(row, e)) << 32) | (u64)(0xFFFFFFFFu - (uint32_t)e);
      if (key < prev && key > best) best = key;
    }
    const int idx = (int)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFull));
    atomicOr(&bt[idx], bit);
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
      if (mt < NMT) {
        a = 0;
        while (mt >= NB - a) {
          mt -= NB - a;
          ++a;
        }
        b = a + mt;
        if (4 * b >= E) a = b = -1;  // b >= a, so this also drops a >= E/4 blocks
      }
      ra[q] = a;
      rb[q] = b;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[q][i] = 0;
    }
  }

  // bt: nslot signature words per expert, slot-major [nslot][EP]
  __device__ __forceinline__ void accumulate(const u64* bt, int nslot) {
    for (int s = 0; s < nslot; ++s) {
      const u64* w = bt + s * EP;
#pragma unroll
      for (int q = 0; q < MTQ; ++q) {
        if (ra[q] < 0) continue;
        const ulonglong2 a01 = *reinterpret_cast<const ulonglong2*>(w + 4 * ra[q]);
        const ulonglong2 a23 = *reinterpret_cast<const ulonglong2*>(w + 4 * ra[q] + 2);
        const ulonglong2 b01 = *reinterpret_cast<const ulonglong2*>(w + 4 * rb[q]);
        const ulonglong2 b23 = *reinterpret_cast<const ulonglong2*>(w + 4 * rb[q] + 2);
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

#define DOL_WAVE_FENCE() asm volatile("" ::: "memory")

// ---------------------------------------------------------------------------
// Top-K (+ Gram) kernel.  grid = (blocks per segment, segments).
// ---------------------------------------------------------------------------
template <typename T, int EP, bool GRAM>
__global__ __launch_bounds__(kFusedThreads) void k_topk(const SegTable tab, const PathArgs a, int fast) {
  constexpr int VEC = Traits<T>::kVec;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage_all = smem;                                                  // [waves][64][stride]
  u64* bt_all = reinterpret_cast<u64*>(smem + (fast ? kFusedWaves * 64 * kStageStride : 0));  // [waves][EP]

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const Segment sg = tab.s[blockIdx.y];
  const int E = a.E, k = a.k;
  const int64_t n = sg.n, off = sg.tok_off;
  if (n <= 0) return;
  const int64_t w_first = off >> 6;
  const int64_t ntile = ((off + n - 1) >> 6) - w_first + 1;
  const int rowB = E * (int)sizeof(T);
  const int rowv = rowB >> 4;
  const int nch = (rowv + 7) >> 3;
  const unsigned char* base = reinterpret_cast<const unsigned char*>(sg.scores);
  unsigned char* st = stage_all + wave * 64 * kStageStride;
  u64* mybt = bt_all + wave * EP;

  PopcGram<EP, kFusedThreads, GRAM> gram;
  if (GRAM) gram.init(tid, E);

  for (int64_t tb = (int64_t)blockIdx.x * kFusedWaves; tb < ntile; tb += (int64_t)gridDim.x * kFusedWaves) {
    const int64_t tile = tb + wave;
#pragma unroll
    for (int e0 = 0; e0 < EP; e0 += 64)
      if (e0 + lane < EP) mybt[e0 + lane] = 0;
    DOL_WAVE_FENCE();
    if (tile < ntile) {
      const int64_t w = w_first + tile;
      const int64_t t0 = w * 64 - off;  // token of lane 0 (negative in a history's first partial word)
      const int64_t t = t0 + lane;
      const bool valid = (t >= 0) && (t < n);
      bool need_slow = valid;
      if (fast) {
        int top[8];
        int rej = INT_MIN;
#pragma unroll
        for (int i = 0; i < 8; ++i) top[i] = INT_MIN;
        for (int c = 0; c < nch; ++c) {
          const int cv0 = c * 8;
          const int cvn = min(8, rowv - cv0);
          // cooperative, coalesced load of a 64-row x 128-byte chunk into LDS
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int flat = j * 64 + lane;
            const int r = flat >> 3, v = flat & 7;
            const int64_t tr = t0 + r;
            if (v < cvn && tr >= 0 && tr < n) {
              const v4u val = __builtin_nontemporal_load(
                  reinterpret_cast<const v4u*>(base + tr * rowB + (int64_t)(cv0 + v) * 16));
              *reinterpret_cast<v4u*>(st + r * kStageStride + v * 16) = val;
            }
          }
          DOL_WAVE_FENCE();
          v4u vv[8];
#pragma unroll
          for (int v = 0; v < 8; ++v) vv[v] = *reinterpret_cast<const v4u*>(st + lane * kStageStride + v * 16);
          DOL_WAVE_FENCE();
          if (VEC == 4) {
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
              int g[8];
#pragma unroll
              for (int h = 0; h < 2; ++h) {
                const int v = 2 * gq + h;
                const v4u x = vv[v];
                const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
                const int e0 = (cv0 + v) * 4;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                  g[h * 4 + i] = (v < cvn) ? composite(xs[i], Traits<T>::kHiMask, e0 + i) : INT_MIN;
              }
              sort8_desc(g);
              merge8<!Traits<T>::kExact>(top, g, rej);
            }
          } else {
#pragma unroll
            for (int v = 0; v < 8; ++v) {
              int g[8];
              const v4u x = vv[v];
              const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
              const int e0 = (cv0 + v) * 8;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                g[2 * i] = (v < cvn) ? composite(xs[i] << 16, Traits<T>::kHiMask, e0 + 2 * i) : INT_MIN;
                g[2 * i + 1] = (v < cvn) ? composite(xs[i] & 0xFFFF0000u, Traits<T>::kHiMask, e0 + 2 * i + 1) : INT_MIN;
              }
              sort8_desc(g);
              merge8<!Traits<T>::kExact>(top, g, rej);
            }
          }
        }
        // threshold checks (k <= 8 on this path)
        int sk = INT_MIN, sk1 = rej;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          sk = (i == k - 1) ? top[i] : sk;
          sk1 = (i == k) ? top[i] : sk1;
        }
        bool ok = (top[0] < kCompPosInf) && (sk > kCompNegInfMax) && (sk < Traits<T>::kZeroLo || sk > Traits<T>::kZeroHi);
        if (!Traits<T>::kExact) ok = ok && ((sk1 >> 8) < (sk >> 8));
        need_slow = valid && !ok;
        if (valid && ok) {
          const u64 bit = 1ull << lane;
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (i < k) atomicOr(&mybt[255 - (top[i] & 255)], bit);
        }
      }
      if (__ballot(need_slow) != 0ull) {
        if (need_slow)
          slow_topk_lane<T>(reinterpret_cast<const T*>(base) + t * (int64_t)E, E, k, mybt, 1ull << lane);
      }
      DOL_WAVE_FENCE();
      if (a.bits != nullptr) {
        u64* dst = a.bits + (int64_t)sg.layer * a.bits_layer_words + w;
        const bool full = (t0 >= 0) && (t0 + 64 <= n);
        for (int e = lane; e < E; e += 64) {
          const u64 word = mybt[e];
          if (full || !a.or_partial)
            dst[(int64_t)e * a.W] = word;
          else if (word)
            atomicOr(dst + (int64_t)e * a.W, word);
        }
      }
    }
    if (GRAM) {
      __syncthreads();
      gram.accumulate(bt_all, kFusedWaves);
      __syncthreads();
    }
  }
  if (GRAM) gram.flush(a.cacc + (int64_t)sg.layer * a.cacc_layer_elems, E);
}

template <typename T, int EP, bool GRAM>
hipError_t launch_one(const SegTable& tab, int nseg, int64_t max_seg_tokens, const PathArgs& a, bool fast,
                      hipStream_t s) {
  auto kern = k_topk<T, EP, GRAM>;
  const size_t lds = (fast ? (size_t)kFusedWaves * 64 * kStageStride : 0) + (size_t)kFusedWaves * EP * sizeof(u64);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  int occ = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, kFusedThreads, lds) != hipSuccess || occ < 1) occ = 1;
  const DevInfo di = device_info();
  const int64_t tiles = (max_seg_tokens + 63) / 64 + 1;
  int64_t bx = ((int64_t)di.cu_count * occ + nseg - 1) / nseg;
  bx = std::min<int64_t>(bx, (tiles + kFusedWaves - 1) / kFusedWaves);
  bx = std::max<int64_t>(bx, 1);
  hipLaunchKernelGGL(kern, dim3((unsigned)bx, (unsigned)nseg), dim3(kFusedThreads), lds, s, tab, a, fast ? 1 : 0);
  return hipGetLastError();
}

template <typename T, bool GRAM>
hipError_t launch_ep(const SegTable& tab, int nseg, int64_t max_seg_tokens, const PathArgs& a, bool fast,
                     hipStream_t s) {
  const int E = a.E;
  if (E <= 8) return launch_one<T, 8, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  if (E <= 16) return launch_one<T, 16, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  if (E <= 32) return launch_one<T, 32, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  if (E <= 64) return launch_one<T, 64, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  if (E <= 128) return launch_one<T, 128, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  if (E <= 256) return launch_one<T, 256, GRAM>(tab, nseg, max_seg_tokens, a, fast, s);
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_slow_wide(const SegTable& tab, int nseg, int64_t max_seg_tokens, const PathArgs& a, hipStream_t s) {
  // E in (256, 1024]: exact per-lane selection, signatures only.
  if (a.E <= 512) return launch_one<T, 512, false>(tab, nseg, max_seg_tokens, a, false, s);
  return launch_one<T, 1024, false>(tab, nseg, max_seg_tokens, a, false, s);
}

}  // namespace

hipError_t launch_topk(do_dtype dt, const SegTable& tab, int nseg, int64_t max_seg_tokens, const PathArgs& a,
                       bool fast_ok, hipStream_t s) {
  const bool gram = a.cacc != nullptr;
  const bool fast = fast_ok && a.k <= kFastMaxK && a.E <= kFastMaxE;
  if (a.E > kFastMaxE) {
    if (gram) return hipErrorInvalidValue;
    return dt == DO_F32 ? launch_slow_wide<float>(tab, nseg, max_seg_tokens, a, s)
                        : launch_slow_wide<uint16_t>(tab, nseg, max_seg_tokens, a, s);
  }
  if (dt == DO_F32)
    return gram ? launch_ep<float, true>(tab, nseg, max_seg_tokens, a, fast, s)
                : launch_ep<float, false>(tab, nseg, max_seg_tokens, a, fast, s);
  return gram ? launch_ep<uint16_t, true>(tab, nseg, max_seg_tokens, a, fast, s)
              : launch_ep<uint16_t, false>(tab, nseg, max_seg_tokens, a, fast, s);
}

}  // namespace dol
