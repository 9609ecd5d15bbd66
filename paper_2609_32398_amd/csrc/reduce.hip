// Gram of stored signatures, distance finalisation and the loss reduction.
//
// Paper: Sec. 3.1.3, Eq. (6) -- G_ij = ||F_i - F_j||_1, evaluated through the
// identity of App. C.3, ||F_i - F_j||_1 = ||F_i||_1 + ||F_j||_1 - 2 c_ij with
// c_ij = sum_t f_it f_jt = popcount(F_i AND F_j) and ||F_i||_1 = c_ii.
// Sec. 3.1.1, Eq. (3) -- L_origin_DO = sum_{i != j} G_ij^2, reported with the
// mean and the population variance of the off-diagonal G_ij (App. C.1: under
// the fixed total of Eq. (2), minimising the sum of squares minimises the
// variance).  All counts and sums are exact integers; only mean, variance and
// the fp64 copy of the loss are rounded.
#include <algorithm>

#include "common.h"

namespace dol {
namespace {

constexpr int kGramThreads = 256;
constexpr int kGramSlots = 8;   // signature words per expert staged per step
constexpr int kGramMtq = 4;     // 4x4 micro-tiles per thread

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// NaN scan of the check-finite mode: *flag = 1 when any of the n elements
// (fp32 or bf16 bit patterns of elem_bytes 4 or 2) is a NaN.  The magnitude
// bits of a NaN exceed those of infinity, and one add per 32-bit word moves
// that comparison into each element's sign position: (w & 0x7FFFFFFF) +
// 0x007FFFFF carries into bit 31 exactly when w & 0x7FFFFFFF > 0x7F800000, and
// two bf16 halves do the same with 0x7FFF7FFF and 0x007F007F (a half's sum
// stays below 0x10000, so nothing carries into the other half).
__global__ void k_nan_scan(const unsigned char* x, int eb, int64_t n, uint32_t* flag) {
  typedef uint32_t v4w __attribute__((ext_vector_type(4)));
  const uint32_t mag = eb == 4 ? 0x7FFFFFFFu : 0x7FFF7FFFu;
  const uint32_t add = eb == 4 ? 0x007FFFFFu : 0x007F007Fu;
  const uint32_t top = eb == 4 ? 0x80000000u : 0x80008000u;
  auto nan_in = [&](uint32_t w) { return ((w & mag) + add) & top; };
  auto elem = [&](int64_t e) {
    return eb == 4 ? reinterpret_cast<const uint32_t*>(x)[e] : (uint32_t)reinterpret_cast<const uint16_t*>(x)[e];
  };
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t bytes = n * eb;
  // x is aligned to its element size, so the bytes before the first 16-byte
  // boundary and after the last one are whole elements
  int64_t head = (int64_t)((16 - (reinterpret_cast<uintptr_t>(x) & 15)) & 15);
  if (head > bytes) head = bytes;
  const int64_t nv = (bytes - head) / 16;
  const v4w* v = reinterpret_cast<const v4w*>(x + head);
  uint32_t any = 0;
  for (int64_t i = i0; i < nv; i += stride) {
    const v4w q = __builtin_nontemporal_load(v + i);
    any |= nan_in(q.x) | nan_in(q.y) | nan_in(q.z) | nan_in(q.w);
  }
  for (int64_t e = i0; e < head / eb; e += stride) any |= nan_in(elem(e));
  for (int64_t e = (head + nv * 16) / eb + i0; e < n; e += stride) any |= nan_in(elem(e));
  if (any != 0u) *flag = 1u;
}

// Zeroes n words; 16-byte stores when p is 16-byte aligned.
__global__ void k_fill_u64(u64* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
    // four 16-byte stores per thread and pass, written past the caches
    typedef unsigned long long v2u __attribute__((ext_vector_type(2)));
    v2u* q = reinterpret_cast<v2u*>(p);
    const int64_t nq = n >> 1;
    const v2u z = {0ull, 0ull};
    int64_t i = i0;
    for (; i + 3 * stride < nq; i += 4 * stride) {
#pragma unroll
      for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(z, q + i + u * stride);
    }
    for (; i < nq; i += stride) __builtin_nontemporal_store(z, q + i);
    if (i0 == 0 && (n & 1)) p[n - 1] = 0ull;
  } else {
    for (int64_t i = i0; i < n; i += stride) p[i] = 0ull;
  }
}

// Zeroes signature words [w0, w0 + nw) of all E experts of one layer
// (unit-major layout, sig_off).
__global__ void k_fill_sig_words(u64* p, int E, int64_t w0, int64_t nw) {
  const int64_t total = (int64_t)E * nw;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x)
    p[sig_off(w0 + i / E, i % E, E)] = 0ull;
}

// grid = (word-chunk blocks, micro-tile slices, layers).  Each thread owns up
// to kGramMtq 4x4 micro-tiles of the upper triangle and accumulates
// popcount(F_i & F_j) over the word chunks of its block in registers.  A
// chunk is one unit of the signature layout (8 words of every expert, E * 64
// contiguous bytes); layers are E * ld words apart.
__global__ __launch_bounds__(kGramThreads) void k_gram_bits(const u64* __restrict__ bits, int64_t W, int64_t ld,
                                                            int E, uint32_t* __restrict__ cacc) {
  extern __shared__ __align__(16) u64 tile[];  // [kGramSlots][E4]
  const int E4 = (E + 3) & ~3;
  const int NB = E4 / 4;
  const int NMT = NB * (NB + 1) / 2;
  const int tid = threadIdx.x;
  const int layer = blockIdx.z;
  const u64* lb = bits + (int64_t)layer * E * ld;

  int ra[kGramMtq], rb[kGramMtq];
  uint32_t acc[kGramMtq][16];
#pragma unroll
  for (int q = 0; q < kGramMtq; ++q) {
    int mt = (int)blockIdx.y * kGramThreads * kGramMtq + q * kGramThreads + tid;
    int a = -1, b = -1;
    if (mt < NMT) {
      a = 0;
      while (mt >= NB - a) {
        mt -= NB - a;
        ++a;
      }
      b = a + mt;
    }
    ra[q] = a;
    rb[q] = b;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[q][i] = 0;
  }

  const int64_t nchunks = (W + kGramSlots - 1) / kGramSlots;
  for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
    const int64_t w0 = ch * kGramSlots;
    __syncthreads();
    // eight loads per thread in flight before their stores (a load followed
    // by its store per iteration would be one memory round trip each);
    // out-of-range positions read word 0 and store zero
    constexpr int kB = 8;
    const int total = E4 * kGramSlots;
    for (int f0 = tid; f0 < total; f0 += kB * kGramThreads) {
      u64 v[kB];
#pragma unroll
      for (int b = 0; b < kB; ++b) {
        const int f = f0 + b * kGramThreads, e = f / kGramSlots, s = f % kGramSlots;
        const bool in = f < total && e < E && w0 + s < W;
        v[b] = lb[in ? sig_off(w0 + s, e, E) : 0];
        v[b] = in ? v[b] : 0ull;
      }
#pragma unroll
      for (int b = 0; b < kB; ++b) {
        const int f = f0 + b * kGramThreads;
        if (f < total) tile[(f % kGramSlots) * E4 + f / kGramSlots] = v[b];
      }
    }
    __syncthreads();
    for (int s = 0; s < kGramSlots; ++s) {
      const u64* w = tile + s * E4;
#pragma unroll
      for (int q = 0; q < kGramMtq; ++q) {
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
  uint32_t* c = cacc + (int64_t)layer * E * E;
#pragma unroll
  for (int q = 0; q < kGramMtq; ++q) {
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

// 64 x 64 -> 128-bit product as (hi, lo).
__device__ __forceinline__ void mul128(u64 a, u64 b, u64& hi, u64& lo) {
  lo = a * b;
  hi = __umul64hi(a, b);
}

// Fill one loss record from exact sums over the E(E-1) off-diagonal entries;
// the sum of squares is the 128-bit (s2h, s2l).  Entries are below 2^32 and
// E <= 1024, so S1 < 2^52, S2 < 2^84 and P*S2, S1^2 < 2^104.  sumsq saturates
// at 2^64 - 1 when S2 does not fit 64 bits; loss is always S2 rounded to fp64.
__device__ void write_result(do_loss_result* o, u64 s1, u64 s2h, u64 s2l, int E) {
  if (E < 2) {
    (void)s2h;
    o->sum = 0;
    o->sumsq = 0;
    o->loss = 0.0;
    o->mean = 0.0;
    o->var = 0.0;
    return;
  }
  const u64 P = (u64)E * (u64)(E - 1);
  o->sum = s1;
  o->sumsq = s2h != 0ull ? ~0ull : s2l;
  o->loss = s2h != 0ull ? (double)s2h * 18446744073709551616.0 + (double)s2l : (double)s2l;
  o->mean = (double)s1 / (double)P;
  // population variance = (P*S2 - S1^2) / P^2 with an exact 128-bit numerator
  u64 ah, al, bh, bl;
  mul128(P, s2l, ah, al);
  ah += P * s2h;
  mul128(s1, s1, bh, bl);
  const u64 nl = al - bl;
  const u64 nh = ah - bh - (al < bl ? 1ull : 0ull);
  const double num = (double)nh * 18446744073709551616.0 + (double)nl;
  o->var = num / ((double)P * (double)P);
}

__device__ __forceinline__ u64 wave_sum(u64 v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum (s1, s2) across the block; valid in thread 0.
__device__ void block_sum2(u64& s1, u64& s2) {
  __shared__ u64 part[2][16];
  s1 = wave_sum(s1);
  s2 = wave_sum(s2);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nw = (blockDim.x + 63) >> 6;
  if (lane == 0) {
    part[0][wave] = s1;
    part[1][wave] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    u64 a = 0, b = 0;
    for (int i = 0; i < nw; ++i) {
      a += part[0][i];
      b += part[1][i];
    }
    s1 = a;
    s2 = b;
  }
}

constexpr int kFinRows = 8;  // rows a wave reads before it writes (loads in flight per lane)
constexpr int kFinCols = 2;  // 64-column blocks k_finalize reads together

// One block per layer.  cacc may alias D: the diagonal is read before any
// write, and every other element is read and written only by the thread that
// owns its (i < j) pair.  Wave w takes rows [8w, 8w + 8), then 8 rows 8 nw
// further, ...; its lanes walk the columns right of the diagonal.  A lane
// loads its entries of all 8 rows in up to 2 column blocks (16 loads) before
// it computes and writes them, so the reads of a wave overlap instead of
// forming a chain of memory round trips (the stores may alias the loads, so
// the compiler cannot move later loads above them).  A position outside the
// upper triangle loads entry 0 and discards it.  The mirrored (column) writes
// are strided.
__global__ __launch_bounds__(1024) void k_finalize(const uint32_t* cacc, uint32_t* D, do_loss_result* out, int E) {
  __shared__ uint32_t diag[kMaxE];
  const int64_t EE = (int64_t)E * E;
  const uint32_t* c = cacc + blockIdx.x * EE;
  uint32_t* d = D + blockIdx.x * EE;
  for (int i = threadIdx.x; i < E; i += blockDim.x) diag[i] = c[(int64_t)i * E + i];
  __syncthreads();
  const int nw = (int)(blockDim.x >> 6), w = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63);
  u64 s1 = 0, s2 = 0;
  for (int i0 = w * kFinRows; i0 < E; i0 += nw * kFinRows) {
    if (lane < kFinRows && i0 + lane < E) d[(int64_t)(i0 + lane) * E + i0 + lane] = 0u;
    for (int jb = ((i0 + 1) & ~63) + lane; jb - lane < E; jb += 64 * kFinCols) {
      uint32_t cv[kFinCols][kFinRows];
#pragma unroll
      for (int q = 0; q < kFinCols; ++q) {
#pragma unroll
        for (int r = 0; r < kFinRows; ++r) {
          const int i = i0 + r, j = jb + 64 * q;
          const bool in = j > i && j < E;
          cv[q][r] = c[in ? (uint32_t)(i * E + j) : 0u];  // E <= 1024: offsets fit 32 bits
        }
      }
#pragma unroll
      for (int q = 0; q < kFinCols; ++q) {
#pragma unroll
        for (int r = 0; r < kFinRows; ++r) {
          const int i = i0 + r, j = jb + 64 * q;
          if (j > i && j < E) {
            const uint32_t v = diag[i] + diag[j] - 2u * cv[q][r];
            d[(uint32_t)(i * E + j)] = v;
            d[(uint32_t)(j * E + i)] = v;
            s1 += 2ull * v;
            s2 += 2ull * (u64)v * (u64)v;
          }
        }
      }
    }
  }
  if (out == nullptr) return;
  block_sum2(s1, s2);
  if (threadIdx.x == 0) write_result(out + blockIdx.x, s1, 0ull, s2, E);
}

constexpr int kSplitRows = 8;  // rows per block of the split finalize, one per wave

// Before a block's ticket: wait until this thread's atomics on the sums are
// performed.  The block that takes the last ticket reads the sums with
// atomics, so it needs no cache writeback from the others; an agent-scope
// fence (__threadfence) would write back the whole L2 in every block.
__device__ __forceinline__ void fin_wait() { __builtin_amdgcn_s_waitcnt(0); }

// The finalize of one layer over ceil(E/8) blocks of 512 threads (E <= 256),
// for a single layer where one block would leave the GPU idle: wave w of
// block b owns row 8b + w.  Every block adds its exact (S1, S2) into fin[0],
// fin[1] and takes a ticket from fin[2]; the block with the last ticket
// writes the loss record and clears fin for the next call.  All accesses to
// fin are atomics (the ticket needs no fence, see fin_wait).  c must not alias D.
__global__ __launch_bounds__(512) void k_finalize_split(const uint32_t* __restrict__ c, uint32_t* __restrict__ d,
                                                        do_loss_result* out, int E, u64* fin) {
  __shared__ uint32_t diag[kFastMaxE];
  for (int i = threadIdx.x; i < E; i += blockDim.x) diag[i] = c[(int64_t)i * E + i];
  __syncthreads();
  const int w = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63);
  const int i = (int)blockIdx.x * kSplitRows + w;
  u64 s1 = 0, s2 = 0;
  if (i < E) {
    const int64_t row = (int64_t)i * E;
    if (lane == 0) d[row + i] = 0u;
    const uint32_t di = diag[i];
    uint32_t cv[kFastMaxE / 64];
#pragma unroll
    for (int q = 0; q < kFastMaxE / 64; ++q) {
      const int j = lane + 64 * q;
      cv[q] = (j > i && j < E) ? c[row + j] : 0u;
    }
#pragma unroll
    for (int q = 0; q < kFastMaxE / 64; ++q) {
      const int j = lane + 64 * q;
      if (j > i && j < E) {
        const uint32_t v = di + diag[j] - 2u * cv[q];
        d[row + j] = v;
        d[(int64_t)j * E + i] = v;
        s1 += 2ull * v;
        s2 += 2ull * (u64)v * (u64)v;
      }
    }
  }
  block_sum2(s1, s2);
  if (threadIdx.x == 0) {
    atomicAdd(&fin[0], s1);
    atomicAdd(&fin[1], s2);
    fin_wait();
    if (atomicAdd(&fin[2], 1ull) == (u64)gridDim.x - 1) {
      const u64 S1 = atomicAdd(&fin[0], 0ull), S2 = atomicAdd(&fin[1], 0ull);
      write_result(out, S1, 0ull, S2, E);
      atomicExch(&fin[0], 0ull);
      atomicExch(&fin[1], 0ull);
      atomicExch(&fin[2], 0ull);
    }
  }
}

// (hi, lo) += (bh, bl) in 128 bits.
__device__ __forceinline__ void add128(u64& hi, u64& lo, u64 bh, u64 bl) {
  lo += bl;
  hi += bh + (lo < bl ? 1ull : 0ull);
}

// Sum of (s1, s2h:s2l) across the block; valid in thread 0.
__device__ void block_sum3(u64& s1, u64& s2h, u64& s2l) {
  __shared__ u64 part[3][16];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    s1 += __shfl_xor(s1, off, 64);
    add128(s2h, s2l, __shfl_xor(s2h, off, 64), __shfl_xor(s2l, off, 64));
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nw = (blockDim.x + 63) >> 6;
  if (lane == 0) {
    part[0][wave] = s1;
    part[1][wave] = s2h;
    part[2][wave] = s2l;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    u64 a = 0, h = 0, l = 0;
    for (int i = 0; i < nw; ++i) {
      a += part[0][i];
      add128(h, l, part[1][i], part[2][i]);
    }
    s1 = a;
    s2h = h;
    s2l = l;
  }
}

// The stream's finalize (one layer, E <= 256), over ceil(E/8) blocks of 512
// threads with wave w of block b on row 8b + w, as k_finalize_split.  The
// co-occurrence count c_ij is snap_ij (when snap_valid) plus the sum of the
// ncopies counter copies.  Each row's owner stores the totals of its
// off-diagonal entries in snap and zeroes them in the copies right after
// reading them; the diagonal, which every block reads, is moved into snap by
// the block that takes the last ticket.  A repeated finalize therefore reads
// the same totals (snap plus zero copies).
__global__ __launch_bounds__(512) void k_finalize_stream(uint32_t* copies, int ncopies, int64_t copy_elems,
                                                         uint32_t* snap, int snap_valid, uint32_t* __restrict__ d,
                                                         do_loss_result* out, int E, u64* fin) {
  __shared__ uint32_t diag[kFastMaxE];
  __shared__ int last;
  for (int i = threadIdx.x; i < E; i += blockDim.x) {
    const int64_t o = (int64_t)i * E + i;
    uint32_t v = snap_valid ? snap[o] : 0u;
    for (int c = 0; c < ncopies; ++c) v += copies[c * copy_elems + o];
    diag[i] = v;
  }
  __syncthreads();
  const int w = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63);
  const int i = (int)blockIdx.x * kSplitRows + w;
  u64 s1 = 0, s2 = 0;
  if (i < E) {
    const int64_t row = (int64_t)i * E;
    if (lane == 0) d[row + i] = 0u;
    const uint32_t di = diag[i];
    uint32_t tot[kFastMaxE / 64];
    // every load of the row (snapshot and copies) is issued before any store
#pragma unroll
    for (int q = 0; q < kFastMaxE / 64; ++q) {
      const int j = lane + 64 * q;
      const bool in = j > i && j < E;
      const int64_t o = row + (in ? j : i);
      uint32_t v = (snap_valid && in) ? snap[o] : 0u;
      for (int c = 0; c < ncopies; ++c) v += in ? copies[c * copy_elems + o] : 0u;
      tot[q] = v;
    }
#pragma unroll
    for (int q = 0; q < kFastMaxE / 64; ++q) {
      const int j = lane + 64 * q;
      if (j > i && j < E) {
        const uint32_t v = di + diag[j] - 2u * tot[q];
        d[row + j] = v;
        d[(int64_t)j * E + i] = v;
        s1 += 2ull * v;
        s2 += 2ull * (u64)v * (u64)v;
        snap[row + j] = tot[q];
        for (int c = 0; c < ncopies; ++c) copies[c * copy_elems + row + j] = 0u;
      }
    }
  }
  block_sum2(s1, s2);
  if (threadIdx.x == 0) {
    atomicAdd(&fin[0], s1);
    atomicAdd(&fin[1], s2);
    fin_wait();
    last = atomicAdd(&fin[2], 1ull) == (u64)gridDim.x - 1;
  }
  __syncthreads();
  if (!last) return;
  // every block has read the diagonal (its loads returned before its ticket):
  // move it into the snapshot
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    const int64_t o = (int64_t)j * E + j;
    snap[o] = diag[j];
    for (int c = 0; c < ncopies; ++c) copies[c * copy_elems + o] = 0u;
  }
  if (threadIdx.x == 0) {
    const u64 S1 = atomicAdd(&fin[0], 0ull), S2 = atomicAdd(&fin[1], 0ull);
    write_result(out, S1, 0ull, S2, E);
    atomicExch(&fin[0], 0ull);
    atomicExch(&fin[1], 0ull);
    atomicExch(&fin[2], 0ull);
  }
}

// Sums of a stored D (every off-diagonal entry), 8 rows per wave per pass.
// Entries are arbitrary u32 values, so the sum of squares is kept in 128
// bits per lane (one entry's square alone may reach 2^64 - 2^33 + 1).
__global__ __launch_bounds__(1024) void k_loss(const uint32_t* D, do_loss_result* out, int E) {
  const int64_t EE = (int64_t)E * E;
  const uint32_t* d = D + blockIdx.x * EE;
  const int nw = (int)(blockDim.x >> 6), w = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63);
  u64 s1 = 0, s2h = 0, s2l = 0;
  // as in k_finalize: 16 loads per lane (8 rows x 2 column blocks) per round
  // trip, 32-bit offsets, positions off the matrix or on the diagonal read
  // entry 0 and count as zero
  for (int i0 = w * kFinRows; i0 < E; i0 += nw * kFinRows) {
    for (int jb = lane; jb - lane < E; jb += 64 * kFinCols) {
      uint32_t dv[kFinCols][kFinRows];
#pragma unroll
      for (int q = 0; q < kFinCols; ++q) {
#pragma unroll
        for (int r = 0; r < kFinRows; ++r) {
          const int i = i0 + r, j = jb + 64 * q;
          const bool in = i < E && j < E && j != i;
          const uint32_t v = d[in ? (uint32_t)(i * E + j) : 0u];
          dv[q][r] = in ? v : 0u;
        }
      }
#pragma unroll
      for (int q = 0; q < kFinCols; ++q) {
#pragma unroll
        for (int r = 0; r < kFinRows; ++r) {
          s1 += dv[q][r];
          add128(s2h, s2l, 0ull, (u64)dv[q][r] * (u64)dv[q][r]);
        }
      }
    }
  }
  block_sum3(s1, s2h, s2l);
  if (threadIdx.x == 0) write_result(out + blockIdx.x, s1, s2h, s2l, E);
}

}  // namespace

DevInfo device_info() {
  static thread_local int cached_dev = -1;
  static thread_local int cached_cu = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (dev != cached_dev) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu < 1) cu = 1;
    cached_dev = dev;
    cached_cu = cu;
  }
  return DevInfo{cached_dev, cached_cu};
}

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_nan_scan(const void* x, int32_t elem_bytes, int64_t n, uint32_t* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nv = n * elem_bytes / 16 + 1;
  const int64_t blocks = std::min<int64_t>((nv + 255) / 256, 2048);
  hipLaunchKernelGGL(k_nan_scan, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<const unsigned char*>(x),
                     (int)elem_bytes, n, flag);
  return hipGetLastError();
}

hipError_t launch_fill_u64(u64* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n / 2 + 1023) / 1024 + 1, 2048);
  hipLaunchKernelGGL(k_fill_u64, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_gram_bits(const u64* bits, int64_t W, int64_t ld, int32_t E, int32_t L, uint32_t* cacc,
                            hipStream_t s) {
  const int E4 = (E + 3) & ~3;
  const int NB = E4 / 4;
  const int NMT = NB * (NB + 1) / 2;
  const int per_slice = kGramThreads * kGramMtq;
  const int slices = (NMT + per_slice - 1) / per_slice;
  const size_t lds = (size_t)kGramSlots * E4 * sizeof(u64);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_gram_bits),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t nchunks = (W + kGramSlots - 1) / kGramSlots;
  const DevInfo di = device_info();
  int64_t bx = ((int64_t)di.cu_count * 4 + (int64_t)slices * L - 1) / ((int64_t)slices * L);
  bx = std::max<int64_t>(1, std::min<int64_t>(bx, nchunks));
  hipLaunchKernelGGL(k_gram_bits, dim3((unsigned)bx, (unsigned)slices, (unsigned)L), dim3(kGramThreads), lds, s,
                     bits, W, ld, E, cacc);
  return hipGetLastError();
}

hipError_t launch_finalize(const uint32_t* cacc, uint32_t* D, do_loss_result* out, int32_t E, int32_t L,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_finalize, dim3((unsigned)L), dim3(1024), 0, s, cacc, D, out, E);
  return hipGetLastError();
}

hipError_t launch_finalize_split(const uint32_t* cacc, uint32_t* D, do_loss_result* out, int32_t E, u64* fin,
                                 hipStream_t s) {
  if (E > kFastMaxE) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_finalize_split, dim3((unsigned)((E + kSplitRows - 1) / kSplitRows)), dim3(kSplitRows * kWave), 0,
                     s, cacc, D, out, E, fin);
  return hipGetLastError();
}

hipError_t launch_finalize_stream(uint32_t* copies, int32_t ncopies, int64_t copy_elems, uint32_t* snap,
                                  int32_t snap_valid, uint32_t* D, do_loss_result* out, int32_t E, u64* fin,
                                  hipStream_t s) {
  if (E > kFastMaxE) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_finalize_stream, dim3((unsigned)((E + kSplitRows - 1) / kSplitRows)), dim3(kSplitRows * kWave),
                     0, s, copies, ncopies, copy_elems, snap, snap_valid, D, out, E, fin);
  return hipGetLastError();
}

hipError_t launch_fill_sig_words(u64* p, int32_t E, int64_t w0, int64_t nw, hipStream_t s) {
  if (E <= 0 || nw <= 0) return hipSuccess;
  const int64_t total = (int64_t)E * nw;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(k_fill_sig_words, dim3((unsigned)blocks), dim3(256), 0, s, p, E, w0, nw);
  return hipGetLastError();
}

hipError_t launch_loss(const uint32_t* D, int32_t E, int32_t L, do_loss_result* out, hipStream_t s) {
  hipLaunchKernelGGL(k_loss, dim3((unsigned)L), dim3(1024), 0, s, D, out, E);
  return hipGetLastError();
}

}  // namespace dol
