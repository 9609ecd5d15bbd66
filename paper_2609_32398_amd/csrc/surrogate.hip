// Surrogate DO-loss (Sec. 3.1.3, Eq. 6-7) and its gradient with respect to
// the routing probabilities, with the magnitude G detached:
//
//   L        = s * sum_{i,j} G_ij C_ij,   C_ij = sum_t p_it (f_it - f_jt)
//   dL/dp_it = s * (f_it R_i - sum_{j in S_t} G_ij),   R_i = sum_j G_ij
//
// s = scale / (N^2 k), S_t the experts token t selected.  The gradient is the
// definition with the sum over j split into its f_it and f_jt parts (exact
// 32-bit integers until the final scaling).  L is linear in p, so it is
// accumulated as sum_t sum_i p_it dL/dp_it in fp64.
//
// Work item: one signature word (64 tokens) of one layer and one range of up
// to 128 experts i.  A block keeps the rows of G for its range in LDS,
// transposed (gt[j][i], E x 128 u32, 128 KiB at 256 experts), with R for the
// range and the signature words of the current tokens; lane l of a wave owns
// experts 2l, 2l+1 of the range, so the loads of p and stores of the gradient
// are coalesced rows and the reads of G for one selected expert j are a
// contiguous LDS row.  The selected experts of a token come from its bit in
// every expert's word (one ballot per 64 experts).
#include <algorithm>

#include "common.h"

namespace dol {
namespace {

constexpr int kSurThreads = 512;
constexpr int kSurWaves = kSurThreads / kWave;
constexpr int kTokPerWave = kWave / kSurWaves;  // tokens of a 64-token word per wave
constexpr int kRange = 128;  // experts per range (2 per lane)

// Two consecutive probabilities as fp32 (one vector load when idx is even).
template <typename T>
struct Prob;
template <>
struct Prob<float> {
  __device__ static __forceinline__ void pair(const void* base, int64_t idx, float& a, float& b) {
    const float2 v = *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(base) + idx);
    a = v.x;
    b = v.y;
  }
  __device__ static __forceinline__ float one(const void* base, int64_t idx) {
    return reinterpret_cast<const float*>(base)[idx];
  }
};
template <>
struct Prob<uint16_t> {
  __device__ static __forceinline__ void pair(const void* base, int64_t idx, float& a, float& b) {
    const uint32_t v = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint16_t*>(base) + idx);
    a = __uint_as_float(v << 16);
    b = __uint_as_float(v & 0xFFFF0000u);
  }
  __device__ static __forceinline__ float one(const void* base, int64_t idx) {
    return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(base)[idx] << 16);
  }
};

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) v += __shfl_xor(v, d);
  return v;
}

template <typename T>
__global__ __launch_bounds__(kSurThreads) void k_surrogate(const SurrogateArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int E = a.E;
  const int nr = (E + kRange - 1) / kRange;
  uint32_t* gt = reinterpret_cast<uint32_t*>(smem);          // [E][kRange]: gt[j][il] = G[range + il][j]
  int32_t* rr = reinterpret_cast<int32_t*>(gt + (size_t)E * kRange);  // [kRange] R_i for the range
  u64* wd = reinterpret_cast<u64*>(rr + kRange);             // [E] signature words of the current tokens

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool even = (E & 1) == 0;  // rows start on an even element: pairs are one vector access
  const int64_t W = a.W;
  const int64_t items = (int64_t)a.L * nr * W;
  const int64_t ib = (int64_t)blockIdx.x * items / gridDim.x;
  const int64_t ie = (int64_t)(blockIdx.x + 1) * items / gridDim.x;
  if (ib >= ie) return;

  int cur_lr = -1;  // layer * nr + range held in LDS
  double lacc = 0.0;
  int cur_layer = -1;
  auto flush_loss = [&]() {
    const double v = wave_sum(lacc);
    if (lane == 0 && cur_layer >= 0) atomicAdd(&a.loss[cur_layer], v * a.s64);
    lacc = 0.0;
  };

  for (int64_t it = ib; it < ie; ++it) {
    const int lr = (int)(it / W);
    const int64_t w = it - (int64_t)lr * W;
    const int layer = lr / nr, r = lr - layer * nr;
    const int iw = min(kRange, E - r * kRange);  // experts in this range
    __syncthreads();  // previous item's readers of wd (and of the tile) are done
    if (lr != cur_lr) {
      if (layer != cur_layer) {
        flush_loss();
        cur_layer = layer;
      }
      const uint32_t* Dl = a.D + (int64_t)layer * E * E;
      for (int idx = tid; idx < E * iw; idx += kSurThreads) {  // rows i of the range, read along j
        const int il = idx / E, j = idx - il * E;
        gt[j * kRange + il] = Dl[(int64_t)(r * kRange + il) * E + j];
      }
      __syncthreads();
      for (int il = tid; il < iw; il += kSurThreads) {
        int32_t acc = 0;
        for (int j = 0; j < E; ++j) acc += (int32_t)gt[j * kRange + il];  // R_i = sum_j G_ij
        rr[il] = acc;
      }
      cur_lr = lr;
    }
    const u64* bl = a.bits + (int64_t)layer * E * W;
    for (int e = tid; e < E; e += kSurThreads) wd[e] = bl[(int64_t)e * W + w];
    __syncthreads();

    // this lane's experts of the range and their words
    const int il0 = 2 * lane, il1 = il0 + 1;
    const bool v0 = il0 < iw, v1 = il1 < iw;
    const int i0 = r * kRange + il0;
    const u64 w0 = v0 ? wd[i0] : 0ull, w1 = v1 ? wd[i0 + 1] : 0ull;
    const int32_t R0 = v0 ? rr[il0] : 0, R1 = v1 ? rr[il1] : 0;
    // the words of experts lane, lane+64, ... (for the selection ballots)
    u64 wg[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) wg[g] = (g * 64 + lane < E) ? wd[g * 64 + lane] : 0ull;

    const int64_t tok0 = w * 64;
    const int64_t prow = (int64_t)layer * a.N;  // token row offset of this layer
    // this wave's tokens of the word: prefetch their p values first
    float pa[kTokPerWave], pb[kTokPerWave];
#pragma unroll
    for (int q = 0; q < kTokPerWave; ++q) {
      const int64_t t = tok0 + wave * kTokPerWave + q;
      pa[q] = pb[q] = 0.f;
      if (t < a.N && v0) {
        const int64_t base = (prow + t) * E + i0;
        if (v1 && even)
          Prob<T>::pair(a.p, base, pa[q], pb[q]);
        else {
          pa[q] = Prob<T>::one(a.p, base);
          if (v1) pb[q] = Prob<T>::one(a.p, base + 1);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kTokPerWave; ++q) {
      const int tb = wave * kTokPerWave + q;  // bit of the token in the words
      const int64_t t = tok0 + tb;
      if (t >= a.N) break;  // wave-uniform
      int32_t acc0 = 0, acc1 = 0;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (g * 64 >= E) break;
        u64 m = __ballot(((wg[g] >> tb) & 1ull) != 0ull);
        while (m != 0ull) {
          const int j = g * 64 + __builtin_ctzll(m);
          m &= m - 1;
          const uint2 gv = *reinterpret_cast<const uint2*>(gt + j * kRange + il0);
          acc0 += (int32_t)gv.x;
          acc1 += (int32_t)gv.y;
        }
      }
      const int32_t c0 = (((w0 >> tb) & 1ull) ? R0 : 0) - acc0;
      const int32_t c1 = (((w1 >> tb) & 1ull) ? R1 : 0) - acc1;
      if (v0) {
        lacc += (double)pa[q] * (double)c0 + (double)pb[q] * (double)c1;
        if (a.grad != nullptr) {
          float* g = a.grad + (prow + t) * E + i0;
          if (v1 && even) {
            *reinterpret_cast<float2*>(g) = float2{(float)c0 * a.s32, (float)c1 * a.s32};
          } else {
            g[0] = (float)c0 * a.s32;
            if (v1) g[1] = (float)c1 * a.s32;
          }
        }
      }
    }
  }
  flush_loss();
}

}  // namespace

hipError_t launch_surrogate(do_dtype dt, const SurrogateArgs& a, hipStream_t s) {
  const int nr = (a.E + kRange - 1) / kRange;
  const size_t lds = (size_t)a.E * kRange * 4 + kRange * 4 + (size_t)a.E * 8;
  const void* kern = dt == DO_F32 ? reinterpret_cast<const void*>(k_surrogate<float>)
                                  : reinterpret_cast<const void*>(k_surrogate<uint16_t>);
  hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  int occ = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, kSurThreads, lds) != hipSuccess || occ < 1) occ = 1;
  const DevInfo di = device_info();
  const int64_t items = (int64_t)a.L * nr * a.W;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((int64_t)di.cu_count * occ, items));
  if (dt == DO_F32)
    hipLaunchKernelGGL(k_surrogate<float>, dim3((unsigned)blocks), dim3(kSurThreads), lds, s, a);
  else
    hipLaunchKernelGGL(k_surrogate<uint16_t>, dim3((unsigned)blocks), dim3(kSurThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace dol
