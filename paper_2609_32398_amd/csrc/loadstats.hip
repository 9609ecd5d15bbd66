// Load statistics of signatures: per-expert loads (App. C.3), the Local-LBL
// balance loss (Sec. 4.2) and the MaxVio imbalance (App. E).
//
//   n_i     = popcount of the signature of expert i (the tokens routed to it)
//   lbl     = sum_i f_i P_i,  f_i = n_i / (N k),  P_i = (1/N) sum_t p_it
//           = (1 / (N^2 k)) sum_i n_i sum_t p_it
//   maxvio  = max_r |L_r / tau - 1|,  L_r = sum of n_i over the experts on
//             rank r,  tau = mean of the L_r
//
// Four launches: a fill of the loads, k_unit_loads (a streaming popcount of
// the signatures, unit by unit), k_lbl_sums (column sums of p weighted by the
// loads, read once; only when p is given) and k_load_finalize (one block per
// layer).
#include <algorithm>

#include "common.h"

namespace dol {
namespace {

constexpr int kLsThreads = 256;
typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int kLsUnroll = 8;
constexpr int kLsVecFlight = 8;  // 16-byte loads in flight per thread in k_lbl_sums_vec

template <typename V>
__device__ __forceinline__ V block_sum(V v, V* red) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) v += __shfl_xor(v, d);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[w] = v;
  __syncthreads();
  V t = 0;
  if (threadIdx.x == 0)
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  __syncthreads();
  return t;  // valid in thread 0
}

// grid = (blocks per layer, layers).  Block b takes a contiguous range of the
// layer's units (signature layout: a unit is the 8 words of every expert,
// E * 8 contiguous words; words at or past W are not counted).  Thread t
// reads the word pairs f = t + 256 i of every unit with 16-byte loads (words
// 2f, 2f + 1 of expert f / 4), so its experts are fixed: t / 4 + 64 i, i < NE;
// two units are loaded before they are counted.  The four lanes of an expert
// then sum their counts, and one of them adds the sum into loads (zeroed by
// the caller).
template <int NE>
__global__ __launch_bounds__(kLsThreads) void k_unit_loads(const u64* bits, int64_t W, int64_t ld, int32_t E,
                                                           uint32_t* loads) {
  static_assert(kLsThreads == 256, "experts t / 4 + 64 i");
  const int l = blockIdx.y, t = threadIdx.x, s2 = 2 * (t & 3);  // the pair's first word in the unit
  const int64_t U = (W + 7) >> 3;
  const int64_t u0 = (int64_t)blockIdx.x * U / gridDim.x, u1 = (int64_t)(blockIdx.x + 1) * U / gridDim.x;
  const u64* lb = bits + (int64_t)l * E * ld;
  uint32_t c[NE];
#pragma unroll
  for (int i = 0; i < NE; ++i) c[i] = 0u;
  auto count = [&](const v2u64& v, int64_t u, int i) {
    const int64_t w = 8 * u + s2;
    c[i] += (w < W ? (uint32_t)__popcll(v[0]) : 0u) + (w + 1 < W ? (uint32_t)__popcll(v[1]) : 0u);
  };
  int64_t u = u0;
  for (; u + 1 < u1; u += 2) {
    v2u64 va[NE], vb[NE];
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int f = t + kLsThreads * i;
      const bool in = f < 4 * E;
      va[i] = in ? __builtin_nontemporal_load(reinterpret_cast<const v2u64*>(lb + u * E * 8) + f) : v2u64{0, 0};
      vb[i] = in ? __builtin_nontemporal_load(reinterpret_cast<const v2u64*>(lb + (u + 1) * E * 8) + f) : v2u64{0, 0};
    }
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      count(va[i], u, i);
      count(vb[i], u + 1, i);
    }
  }
  if (u < u1) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int f = t + kLsThreads * i;
      if (f < 4 * E) count(__builtin_nontemporal_load(reinterpret_cast<const v2u64*>(lb + u * E * 8) + f), u, i);
    }
  }
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    c[i] += (uint32_t)__shfl_xor((int)c[i], 1);
    c[i] += (uint32_t)__shfl_xor((int)c[i], 2);
    const int e = (t >> 2) + 64 * i;
    if ((t & 3) == 0 && e < E && c[i] != 0u) atomicAdd(&loads[(int64_t)l * E + e], c[i]);
  }
}

template <typename T>
__device__ __forceinline__ double prob(const T* p, int64_t idx);
// read once: non-temporal loads
template <>
__device__ __forceinline__ double prob<float>(const float* p, int64_t idx) {
  return (double)__builtin_nontemporal_load(p + idx);
}
template <>
__device__ __forceinline__ double prob<uint16_t>(const uint16_t* p, int64_t idx) {
  return (double)__uint_as_float((uint32_t)__builtin_nontemporal_load(p + idx) << 16);
}

// blockIdx.x = token slice, blockIdx.y = layer.  Each thread sums the
// probabilities of fixed columns over the slice's rows, then the block adds
// sum_i n_i * (its column sums) into out[layer].lbl.  E <= 256: thread tid
// takes column tid % E and rows tid / E, tid / E + E', ... with E' = 256 / E
// rows per step (threads past E' * E idle); E > 256: columns tid, tid + 256, ...
template <typename T>
__global__ __launch_bounds__(kLsThreads) void k_lbl_sums(const T* p, int64_t N, int32_t E, int64_t rows_per_block,
                                                         const uint32_t* loads, do_load_stats_result* out) {
  __shared__ double red[kLsThreads / kWave];
  const int l = blockIdx.y;
  const int64_t t0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t t1 = min(N, t0 + rows_per_block);
  const T* pl = p + (int64_t)l * N * E;
  const uint32_t* nl = loads + (int64_t)l * E;
  double acc = 0.0;
  if (E <= kLsThreads) {
    const int rs = kLsThreads / E;  // rows per step
    const int col = threadIdx.x % E, r0 = threadIdx.x / E;
    if (r0 < rs) {
      double s[kLsUnroll];  // independent sums: kLsUnroll loads in flight per thread
#pragma unroll
      for (int u = 0; u < kLsUnroll; ++u) s[u] = 0.0;
      int64_t t = t0 + r0;
      for (; t + (kLsUnroll - 1) * rs < t1; t += kLsUnroll * rs) {
#pragma unroll
        for (int u = 0; u < kLsUnroll; ++u) s[u] += prob<T>(pl, (t + u * rs) * E + col);
      }
      for (; t < t1; t += rs) s[0] += prob<T>(pl, t * E + col);
      double tsum = 0.0;
#pragma unroll
      for (int u = 0; u < kLsUnroll; ++u) tsum += s[u];
      acc = (double)nl[col] * tsum;
    }
  } else {
    for (int col = threadIdx.x; col < E; col += kLsThreads) {
      double s = 0.0;
      for (int64_t t = t0; t < t1; ++t) s += prob<T>(pl, t * E + col);
      acc += (double)nl[col] * s;
    }
  }
  const double b = block_sum<double>(acc, red);
  if (threadIdx.x == 0 && b != 0.0) atomicAdd(&out[l].lbl, b);
}

// k_lbl_sums for fp32 rows of whole 16-byte vectors (p 16-byte aligned, E a
// multiple of 4, at most 256 vectors per row): thread tid keeps vector column
// tid % VR of every row tid / VR + i * (256 / VR), with eight vectors in
// flight, and one fp64 sum per element of its vector.
__global__ __launch_bounds__(kLsThreads) void k_lbl_sums_vec(const float* p, int64_t N, int32_t E,
                                                             int64_t rows_per_block, const uint32_t* loads,
                                                             do_load_stats_result* out) {
  __shared__ double red[kLsThreads / kWave];
  const int l = blockIdx.y;
  const int64_t t0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t t1 = min(N, t0 + rows_per_block);
  const int vr = E / 4;            // vectors per row
  const int rs = kLsThreads / vr;  // rows per step
  const int vc = threadIdx.x % vr, r0 = threadIdx.x / vr;
  const v4f* pl = reinterpret_cast<const v4f*>(p + (int64_t)l * N * E);
  const uint32_t* nl = loads + (int64_t)l * E;
  double acc = 0.0;
  if (r0 < rs) {
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    auto add = [&](const v4f q) {
#pragma unroll
      for (int c = 0; c < 4; ++c) s[c] += (double)q[c];
    };
    int64_t t = t0 + r0;
    for (; t + (kLsVecFlight - 1) * rs < t1; t += kLsVecFlight * rs) {
      v4f q[kLsVecFlight];
#pragma unroll
      for (int i = 0; i < kLsVecFlight; ++i) q[i] = __builtin_nontemporal_load(pl + (t + i * rs) * vr + vc);
#pragma unroll
      for (int i = 0; i < kLsVecFlight; ++i) add(q[i]);
    }
    for (; t < t1; t += rs) add(__builtin_nontemporal_load(pl + t * vr + vc));
#pragma unroll
    for (int c = 0; c < 4; ++c) acc += (double)nl[vc * 4 + c] * s[c];
  }
  const double b = block_sum<double>(acc, red);
  if (threadIdx.x == 0 && b != 0.0) atomicAdd(&out[l].lbl, b);
}

// One block per layer: total / max / min of the loads, MaxVio over the rank
// placement, and the Local-LBL scaling.  out[l].lbl holds the raw sum (or 0).
__global__ __launch_bounds__(kLsThreads) void k_load_finalize(const uint32_t* loads, int64_t N, int32_t E, int32_t k,
                                                              const RankMap rm, do_load_stats_result* out) {
  __shared__ uint64_t rank_load[kMaxE];
  __shared__ uint64_t red64[kLsThreads / kWave];
  __shared__ uint32_t redmx[kLsThreads / kWave], redmn[kLsThreads / kWave];
  __shared__ double redv[kLsThreads / kWave];
  const int l = blockIdx.x;
  const uint32_t* nl = loads + (int64_t)l * E;
  const int R = rm.given ? rm.R : E;
  for (int r = threadIdx.x; r < R; r += kLsThreads) rank_load[r] = 0;
  __syncthreads();
  uint64_t tot = 0;
  uint32_t mx = 0, mn = 0xFFFFFFFFu;
  for (int i = threadIdx.x; i < E; i += kLsThreads) {
    const uint32_t n = nl[i];
    tot += n;
    mx = max(mx, n);
    mn = min(mn, n);
    atomicAdd(reinterpret_cast<unsigned long long*>(&rank_load[rm.given ? rm.rank[i] : i]), (unsigned long long)n);
  }
  const uint64_t T = block_sum<uint64_t>(tot, red64);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    mx = max(mx, (uint32_t)__shfl_xor((int)mx, d));
    mn = min(mn, (uint32_t)__shfl_xor((int)mn, d));
  }
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) {
    redmx[w] = mx;
    redmn[w] = mn;
  }
  __syncthreads();  // also orders the rank-load atomics before the reads below
  __shared__ uint64_t total_s;
  if (threadIdx.x == 0) total_s = T;
  __syncthreads();
  // tau = total / R; |L_r / tau - 1| = |R L_r - total| / total, exact in integers up to the division
  const uint64_t tot_all = total_s;
  double v = 0.0;
  if (tot_all > 0)
    for (int r = threadIdx.x; r < R; r += kLsThreads) {
      const uint64_t a = (uint64_t)R * rank_load[r];
      const uint64_t dev = a > tot_all ? a - tot_all : tot_all - a;
      v = max(v, (double)dev / (double)tot_all);
    }
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) v = max(v, __shfl_xor(v, d));
  if (lane == 0) redv[w] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t M = 0, m = 0xFFFFFFFFu;
    double V = 0.0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
      M = max(M, redmx[i]);
      m = min(m, redmn[i]);
      V = max(V, redv[i]);
    }
    do_load_stats_result& o = out[l];
    o.total = tot_all;
    o.max_load = M;
    o.min_load = m;
    o.maxvio = V;
    o.lbl = o.lbl / ((double)N * (double)N * (double)k);
  }
}

}  // namespace

hipError_t launch_load_stats(const u64* bits, int64_t N, int64_t ld, int32_t E, int32_t k, int32_t L, const void* p,
                             do_dtype dt, const RankMap& rm, uint32_t* loads, do_load_stats_result* out,
                             hipStream_t s) {
  const int64_t W = (N + 63) / 64;
  hipError_t e = launch_fill_u64(reinterpret_cast<u64*>(out), (int64_t)L * (sizeof(do_load_stats_result) / 8), s);
  if (e != hipSuccess) return e;
  if ((e = launch_fill_u32(loads, (int64_t)L * E, 0u, s)) != hipSuccess) return e;
  {
    // about four blocks per CU in total, each over a contiguous range of units
    const DevInfo di = device_info();
    const int64_t U = (W + 7) / 8;
    const int64_t per_layer = std::max<int64_t>(1, std::min<int64_t>(U, ((int64_t)di.cu_count * 4 + L - 1) / L));
    const dim3 grid((unsigned)per_layer, (unsigned)L);
    const int ne = (E + 63) / 64;  // counters per thread
    if (ne <= 1)
      hipLaunchKernelGGL(k_unit_loads<1>, grid, dim3(kLsThreads), 0, s, bits, W, ld, E, loads);
    else if (ne <= 2)
      hipLaunchKernelGGL(k_unit_loads<2>, grid, dim3(kLsThreads), 0, s, bits, W, ld, E, loads);
    else if (ne <= 4)
      hipLaunchKernelGGL(k_unit_loads<4>, grid, dim3(kLsThreads), 0, s, bits, W, ld, E, loads);
    else if (ne <= 8)
      hipLaunchKernelGGL(k_unit_loads<8>, grid, dim3(kLsThreads), 0, s, bits, W, ld, E, loads);
    else
      hipLaunchKernelGGL(k_unit_loads<16>, grid, dim3(kLsThreads), 0, s, bits, W, ld, E, loads);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (p != nullptr) {
    // about 8 blocks per CU in total, each over a contiguous slice of rows
    const DevInfo di = device_info();
    const int64_t want = std::max<int64_t>(1, (int64_t)di.cu_count * 8 / L);
    const int64_t rows = std::max<int64_t>(1, (N + want - 1) / want);
    const int64_t slices = (N + rows - 1) / rows;
    // fp32 rows of whole 16-byte vectors take the vector form (workload 4:
    // 2.69 -> 2.60 ms for four layers); for bf16 its eight fp64 sums per
    // vector made workload 2 slower (0.528 -> 0.550 ms), so bf16 keeps
    // element loads
    const bool vec = dt == DO_F32 && (reinterpret_cast<uintptr_t>(p) & 15) == 0 && E % 4 == 0 && E / 4 <= kLsThreads;
    const dim3 grid((unsigned)slices, (unsigned)L);
    if (vec)
      hipLaunchKernelGGL(k_lbl_sums_vec, grid, dim3(kLsThreads), 0, s, static_cast<const float*>(p), N, E,
                         rows, loads, out);
    else if (dt == DO_F32)
      hipLaunchKernelGGL(k_lbl_sums<float>, grid, dim3(kLsThreads), 0, s, static_cast<const float*>(p), N, E, rows,
                         loads, out);
    else
      hipLaunchKernelGGL(k_lbl_sums<uint16_t>, grid, dim3(kLsThreads), 0, s, static_cast<const uint16_t*>(p), N, E,
                         rows, loads, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_load_finalize, dim3((unsigned)L), dim3(kLsThreads), 0, s, loads, N, E, k, rm, out);
  return hipGetLastError();
}

}  // namespace dol
