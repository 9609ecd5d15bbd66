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
// to 128 experts i, handled by one wave.  A block keeps the rows of G for its
// range in LDS, transposed (gt[j][i], E x 128 u32, 128 KiB at 256 experts),
// with R for the range; lane l owns experts 2l, 2l+1 of the range, so the
// loads of p and the stores of the gradient are coalesced rows and the reads
// of G for one selected expert j are a contiguous LDS row.  The selected
// experts of a token are collected per item into a small LDS list of row
// offsets (each expert appends itself to the tokens set in its word), so a
// token's G rows are read with eight independent LDS loads.
#include <algorithm>

#include "common.h"

namespace dol {
namespace {

constexpr int kSurThreads = 1024;
constexpr int kSurWaves = kSurThreads / kWave;
constexpr int kRange = 128;  // experts per range (2 per lane)



// Two consecutive probabilities as fp32 (one vector load when idx is even).
// The probabilities are read once and the gradient is written once, so both
// carry the non-temporal hint (10 % faster at workload 4 than plain accesses).
template <typename T>
struct Prob;
template <>
struct Prob<float> {
  __device__ static __forceinline__ void pair(const void* base, int64_t idx, float& a, float& b) {
    const u64 v = __builtin_nontemporal_load(reinterpret_cast<const u64*>(reinterpret_cast<const float*>(base) + idx));
    a = __uint_as_float((uint32_t)v);
    b = __uint_as_float((uint32_t)(v >> 32));
  }
  __device__ static __forceinline__ float one(const void* base, int64_t idx) {
    return __builtin_nontemporal_load(reinterpret_cast<const float*>(base) + idx);
  }
};
template <>
struct Prob<uint16_t> {
  __device__ static __forceinline__ void pair(const void* base, int64_t idx, float& a, float& b) {
    const uint32_t v =
        __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint16_t*>(base) + idx));
    a = __uint_as_float(v << 16);
    b = __uint_as_float(v & 0xFFFF0000u);
  }
  __device__ static __forceinline__ float one(const void* base, int64_t idx) {
    return __uint_as_float((uint32_t)__builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(base) + idx) << 16);
  }
};

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) v += __shfl_xor(v, d);
  return v;
}

// Per-wave LDS scratch of one item: for each of its 64 tokens the number of
// selected experts and the offsets (in 8-byte units of the G tile) of the rows
// of the first kSurMaxK of them; unused entries point at the all-zero row E.
// A token with more selected experts than that is summed from the signature
// words instead.
constexpr int kSurMaxK = 8;
constexpr uint32_t kRowUnits = kRange * 4 / 8;  // one G tile row in 8-byte units
struct WaveLists {
  uint32_t cnt[64];
  uint16_t off[64][kSurMaxK];
};

// FULL: the range has 128 experts and E is even (every lane owns two valid,
// pair-aligned experts), the common case; otherwise lanes and pairs are guarded.
// GRAD: the gradient is written (else only the loss is accumulated).
template <typename T, bool FULL, bool GRAD>
__device__ __forceinline__ void surrogate_item(const SurrogateArgs& a, const uint32_t* gt, WaveLists& wl, int E,
                                               int ng, int iw, int r, int layer, int64_t w, int32_t R0, int32_t R1,
                                               double& lacc, int lane) {
  const u64* bl = a.bits + (int64_t)layer * E * sig_words(a.W);
  const int il0 = 2 * lane;
  const bool v0 = FULL || il0 < iw, v1 = FULL || il0 + 1 < iw;
  const bool even = FULL || (E & 1) == 0;
  const int i0 = r * kRange + il0;
  // words of experts g*64 + lane
  u64 wg[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) wg[g] = (g < ng && g * 64 + lane < E) ? bl[sig_off(w, g * 64 + lane, E)] : 0ull;
  // token lists: expert g*64 + lane appends its row offset to the list of
  // every token whose bit is set in its word (order within a list is
  // irrelevant: summed)
  wl.cnt[lane] = 0u;
  {
    const uint32_t z = (uint32_t)E * kRowUnits * 0x10001u;  // the zero row E, twice
    *reinterpret_cast<uint4*>(&wl.off[lane][0]) = uint4{z, z, z, z};
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    u64 bits = wg[g];
    while (bits != 0ull) {
      const int q = __builtin_ctzll(bits);
      bits &= bits - 1;
      const uint32_t slot = atomicAdd(&wl.cnt[q], 1u);
      if (slot < (uint32_t)kSurMaxK) wl.off[q][slot] = (uint16_t)((uint32_t)(g * 64 + lane) * kRowUnits);
    }
  }
  __builtin_amdgcn_wave_barrier();
  // this lane's two experts: expert i0 (+1) sits in group 2r + lane/32 at lane i0 & 63
  u64 w0, w1;
  {
    const u64 xa = r == 0 ? wg[0] : wg[2];
    const u64 xb = r == 0 ? wg[1] : wg[3];
    const u64 a0 = __shfl(xa, il0 & 63), b0 = __shfl(xb, il0 & 63);
    const u64 a1 = __shfl(xa, (il0 + 1) & 63), b1 = __shfl(xb, (il0 + 1) & 63);
    w0 = v0 ? (lane < 32 ? a0 : b0) : 0ull;
    w1 = v1 ? (lane < 32 ? a1 : b1) : 0ull;
  }
  const int64_t tok0 = w * 64;
  const int nt = (int)min((int64_t)64, a.N - tok0);
  const int64_t row0 = (int64_t)layer * a.N + tok0;  // global row of token 0 of the word
  const T* prow = reinterpret_cast<const T*>(a.p) + row0 * E;
  float* grow = GRAD ? a.grad + row0 * E : nullptr;
  const unsigned char* glb = reinterpret_cast<const unsigned char*>(gt + il0);  // this lane's pair in row 0

  // token tb: c = f R - sum_{j selected} G_ij for this lane's two experts
  // (fsel0 / fsel1: all ones when the expert selected the token, else 0)
  auto emit = [&](int tb, float pa, float pb, int32_t fsel0, int32_t fsel1, int32_t acc0, int32_t acc1) {
    const int32_t c0 = (fsel0 & R0) - acc0;
    const int32_t c1 = (fsel1 & R1) - acc1;
    if (v0) {
      lacc += (double)pa * (double)c0 + (double)pb * (double)c1;
      if (GRAD) {
        float* g = grow + (int64_t)tb * E + i0;
        if (FULL || (v1 && even)) {
          const u64 gv = ((u64)__float_as_uint((float)c1 * a.s32) << 32) | __float_as_uint((float)c0 * a.s32);
          __builtin_nontemporal_store(gv, reinterpret_cast<u64*>(g));
        } else {
          __builtin_nontemporal_store((float)c0 * a.s32, g);
          if (v1) __builtin_nontemporal_store((float)c1 * a.s32, g + 1);
        }
      }
    }
  };
  // Every batch position loads: a token past the word's last one reads the
  // last token's row instead, and its values are never used.  A branch on
  // tb < nt would make each load wait for its data before the next one.
  auto load_p = [&](int tb, float& pa, float& pb) {
    pa = pb = 0.f;
    if (v0) {
      const int64_t off = (int64_t)min(tb, nt - 1) * E + i0;
      if (FULL || (v1 && even)) {
        Prob<T>::pair(prow, off, pa, pb);
      } else {
        pa = Prob<T>::one(prow, off);
        if (v1) pb = Prob<T>::one(prow, off + 1);
      }
    }
  };

  // token tb of the word: its G rows summed for this lane's two experts
  auto token = [&](int tb, float pa, float pb, uint32_t b0, uint32_t b1, int q) __attribute__((always_inline)) {
    const uint4 la = *reinterpret_cast<const uint4*>(&wl.off[tb][0]);  // same address (and value) in every lane
    const uint32_t lw[4] = {la.x, la.y, la.z, la.w};
    uint2 gv[kSurMaxK];
#pragma unroll
    for (int rr = 0; rr < kSurMaxK; ++rr) {
      const uint32_t u = (rr & 1) ? (lw[rr >> 1] >> 16) : (lw[rr >> 1] & 0xFFFFu);
      gv[rr] = *reinterpret_cast<const uint2*>(glb + 8u * u);
    }
    int32_t acc0 = 0, acc1 = 0;
#pragma unroll
    for (int rr = 0; rr < kSurMaxK; ++rr) {
      acc0 += (int32_t)gv[rr].x;
      acc1 += (int32_t)gv[rr].y;
    }
    const int32_t f0 = -(int32_t)((b0 >> q) & 1u), f1 = -(int32_t)((b1 >> q) & 1u);
    emit(tb, pa, pb, f0, f1, acc0, acc1);
  };
  if (__ballot(wl.cnt[lane] > (uint32_t)kSurMaxK) == 0ull) {
    for (int q0 = 0; q0 < nt; q0 += 16) {
      // probabilities of 16 tokens, loaded together before this batch's stores
      float xa[16], xb[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) load_p(q0 + q, xa[q], xb[q]);
      const uint32_t b0 = (uint32_t)(w0 >> q0), b1 = (uint32_t)(w1 >> q0);  // this batch's selection bits
      if (q0 + 16 <= nt) {
        // a whole batch: straight-line code, so the LDS reads of one token
        // can be issued while earlier tokens are summed and stored
#pragma unroll
        for (int q = 0; q < 16; ++q) token(q0 + q, xa[q], xb[q], b0, b1, q);
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q)
          if (q0 + q < nt) token(q0 + q, xa[q], xb[q], b0, b1, q);  // wave-uniform
      }
    }
  } else {
    // some token selected more experts than a list holds (signatures not made
    // by a top-k with k <= kSurMaxK): sum over the set bits of every token
    const uint32_t* gl = gt + il0;
    for (int tb = 0; tb < nt; ++tb) {
      float pa, pb;
      load_p(tb, pa, pb);
      int32_t acc0 = 0, acc1 = 0;
#pragma unroll
      for (int g = 0; g < 4; ++g) {  // wg[g] is zero past the last group
        u64 sel = __ballot((wg[g] >> tb) & 1ull);
        while (sel != 0ull) {
          const int j = g * 64 + __builtin_ctzll(sel);
          sel &= sel - 1;
          const uint2 v = *reinterpret_cast<const uint2*>(gl + j * kRange);
          acc0 += (int32_t)v.x;
          acc1 += (int32_t)v.y;
        }
      }
      emit(tb, pa, pb, -(int32_t)((w0 >> tb) & 1ull), -(int32_t)((w1 >> tb) & 1ull), acc0, acc1);
    }
  }
  __builtin_amdgcn_wave_barrier();  // the lists are rebuilt by the next item
}

template <typename T>
__global__ __launch_bounds__(kSurThreads) void k_surrogate(const SurrogateArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int E = a.E;
  const int nr = (E + kRange - 1) / kRange;
  uint32_t* gt = reinterpret_cast<uint32_t*>(smem);  // [E + 1][kRange]: gt[j][il] = G[range + il][j]; row E zero
  int32_t* rr = reinterpret_cast<int32_t*>(gt + (size_t)(E + 1) * kRange);  // [kRange] R_i for the range
  WaveLists* lists = reinterpret_cast<WaveLists*>(rr + kRange);              // [kSurWaves]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ng = (E + 63) >> 6;  // 64-expert groups
  const int64_t W = a.W;
  const int64_t items = (int64_t)a.L * nr * W;
  const int64_t ib = (int64_t)blockIdx.x * items / gridDim.x;
  const int64_t ie = (int64_t)(blockIdx.x + 1) * items / gridDim.x;
  if (ib >= ie) return;
  for (int il = tid; il < kRange; il += kSurThreads) gt[(size_t)E * kRange + il] = 0u;

  double lacc = 0.0;
  int cur_layer = -1;
  auto flush_loss = [&]() {
    const double v = wave_sum(lacc);
    if (lane == 0 && cur_layer >= 0) atomicAdd(&a.loss[cur_layer], v * a.s64);
    lacc = 0.0;
  };

  // runs of items with one (layer, range): the tile is loaded once per run,
  // then each wave takes every kSurWaves-th item of the run without barriers
  for (int64_t sb = ib; sb < ie;) {
    const int lr = (int)(sb / W);
    const int64_t se = min(ie, (int64_t)(lr + 1) * W);
    const int layer = lr / nr, r = lr - layer * nr;
    const int iw = min(kRange, E - r * kRange);  // experts in this range
    if (layer != cur_layer) {
      flush_loss();
      cur_layer = layer;
    }
    __syncthreads();  // every wave is done with the previous tile
    const uint32_t* Dl = a.D + (int64_t)layer * E * E;
    // rows i of the range, read along j, eight loads in flight per thread
    // before their stores; positions outside read entry 0 and store zero
    for (int idx0 = tid; idx0 < E * kRange; idx0 += 8 * kSurThreads) {
      uint32_t v[8];
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const int idx = idx0 + b * kSurThreads, il = idx / E, j = idx - il * E;
        const bool in = idx < E * kRange && il < iw;
        v[b] = Dl[in ? (int64_t)(r * kRange + il) * E + j : 0];
        v[b] = in ? v[b] : 0u;
      }
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const int idx = idx0 + b * kSurThreads, il = idx / E, j = idx - il * E;
        if (idx < E * kRange) gt[j * kRange + il] = v[b];
      }
    }
    __syncthreads();
    for (int il = tid; il < iw; il += kSurThreads) {
      int32_t acc = 0;
      for (int j = 0; j < E; ++j) acc += (int32_t)gt[j * kRange + il];  // R_i = sum_j G_ij
      rr[il] = acc;
    }
    __syncthreads();
    const int32_t R0 = 2 * lane < iw ? rr[2 * lane] : 0, R1 = 2 * lane + 1 < iw ? rr[2 * lane + 1] : 0;
    const bool full = iw == kRange && (E & 1) == 0;
    for (int64_t it = sb + wave; it < se; it += kSurWaves) {
      const int64_t w = it - (int64_t)lr * W;
      if (a.grad != nullptr) {
        if (full)
          surrogate_item<T, true, true>(a, gt, lists[wave], E, ng, iw, r, layer, w, R0, R1, lacc, lane);
        else
          surrogate_item<T, false, true>(a, gt, lists[wave], E, ng, iw, r, layer, w, R0, R1, lacc, lane);
      } else {
        if (full)
          surrogate_item<T, true, false>(a, gt, lists[wave], E, ng, iw, r, layer, w, R0, R1, lacc, lane);
        else
          surrogate_item<T, false, false>(a, gt, lists[wave], E, ng, iw, r, layer, w, R0, R1, lacc, lane);
      }
    }
    sb = se;
  }
  flush_loss();
}

}  // namespace

hipError_t launch_surrogate(do_dtype dt, const SurrogateArgs& a, hipStream_t s) {
  const int nr = (a.E + kRange - 1) / kRange;
  const size_t lds = (size_t)(a.E + 1) * kRange * 4 + kRange * 4 + kSurWaves * sizeof(WaveLists);
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
