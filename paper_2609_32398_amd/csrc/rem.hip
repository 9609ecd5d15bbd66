// REM scheduler: global-batch replica allocation and micro-batch token
// dispatching on the device, one wavefront per independent problem (layer).
//
// Paper: Sec. 3.2.1 -- the Benefit Score S(e, r_s, r_r, tau), the number of
// tokens a replica of expert e on the receiving rank r_r takes over from the
// sending rank r_s, with tau the mean rank load:
//   min(tau - L_r, T_e, L_s - tau)        if L_r < tau < L_s
//   min(floor((L_s - L_r) / 2), T_e)      if L_r >= tau and L_s > L_r
//   -1                                    otherwise.
// App. B, Alg. 1 -- while a rank has a free replica slot, the least-loaded
// such rank receives a replica of the expert with the largest score; the
// loads and the expert's volume move by that score; a score <= 0 stops it.
// App. B, Alg. 2 -- D passes; each orders the ranks by queue depth (lightest
// first, without re-sorting inside the pass) and lets every rank pull tokens
// through the best of the replicas it holds.
//
// All arithmetic is exact in 64-bit integers: tau = total / R is compared as
// R * L against the total, and the two differences with tau are rounded down
// to whole tokens.  An expert's tokens come from its home rank.  Ties: the
// lowest rank index among equally loaded receivers, the lowest expert index
// among equal scores (Alg. 1), the earliest replica (Alg. 2), ranks of equal
// depth by index.  Alg. 2 applies a move only when its score is positive.
//
// Each search is a wave-wide reduction of one 64-bit key that orders the
// candidates and carries the winner's index in its low bits: loads and
// volumes are below 2^40, so R * L < 2^50 and every key fits.
#include <algorithm>

#include "common.h"

namespace dol {
namespace {

constexpr int64_t kRemMaxVal = int64_t(1) << 40;  // loads and volumes must be below this

__device__ __forceinline__ int64_t benefit(int64_t T, int64_t Ls, int64_t Lr, int64_t total, int64_t R) {
  if (R * Lr < total && R * Ls > total) return min(min((total - R * Lr) / R, T), (R * Ls - total) / R);
  if (R * Lr >= total && Ls > Lr) return min((Ls - Lr) >> 1, T);
  return -1;
}

__device__ __forceinline__ u64 wave_min_u64(u64 v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = min(v, (u64)__shfl_xor((unsigned long long)v, off, 64));
  return v;
}

__device__ __forceinline__ u64 wave_max_u64(u64 v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, (u64)__shfl_xor((unsigned long long)v, off, 64));
  return v;
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor((long long)v, off, 64);
  return v;
}

// Loads the layer's volumes into LDS and checks that every value is in
// [0, 2^40); returns false (wave-uniform) otherwise.
__device__ bool load_tokens(const int64_t* src, int64_t* T, int E, int lane) {
  bool bad = false;
  for (int e = lane; e < E; e += kWave) {
    const int64_t v = src[e];
    bad = bad || v < 0 || v >= kRemMaxVal;
    T[e] = v;
  }
  return __ballot(bad) == 0ull;
}

// Alg. 1 for layer blockIdx.x (one wavefront).
__global__ __launch_bounds__(kWave) void k_rem_allocate(const int64_t* rank_load, const int64_t* tokens, RankMap rm,
                                                        int E, int D, do_rem_move* moves, int32_t* n_moves,
                                                        int64_t* load_out, int64_t* tokens_out) {
  __shared__ int64_t T[kMaxE];
  __shared__ int64_t Ld[kMaxE];
  __shared__ int32_t used[kMaxE];
  const int lane = threadIdx.x, l = blockIdx.x, R = rm.R;
  const int cap = R * D;
  bool ok = load_tokens(tokens + (int64_t)l * E, T, E, lane);
  for (int r = lane; r < R; r += kWave) {
    used[r] = 0;
    Ld[r] = 0;
  }
  __syncthreads();
  if (rank_load != nullptr) {
    ok = load_tokens(rank_load + (int64_t)l * R, Ld, R, lane) && ok;
  } else if (lane == 0) {
    for (int e = 0; e < E; ++e) Ld[rm.rank[e]] += T[e];  // below 2^50: no overflow
  }
  __syncthreads();
  if (!ok) {
    if (lane == 0) n_moves[l] = -1;
    return;
  }
  int64_t part = 0;
  for (int r = lane; r < R; r += kWave) part += Ld[r];
  const int64_t total = wave_sum_i64(part);
  int n = 0;
  while (true) {
    // the receiver: least-loaded rank with a free slot, lowest index on ties
    u64 kr = ~0ull;
    for (int r = lane; r < R; r += kWave)
      if (used[r] < D) kr = min(kr, ((u64)Ld[r] << 10) | (u64)r);
    kr = wave_min_u64(kr);
    if (kr == ~0ull) break;  // every rank is full
    const int rr = (int)(kr & 1023u);
    const int64_t Lr = Ld[rr];
    // the expert with the largest score, lowest index on ties
    u64 ke = 0;
    for (int e = lane; e < E; e += kWave) {
      const int rs = rm.rank[e];
      if (rs == rr) continue;
      const int64_t s = benefit(T[e], Ld[rs], Lr, total, R);
      ke = max(ke, ((u64)(s + 1) << 10) | (u64)(1023 - e));
    }
    ke = wave_max_u64(ke);
    const int64_t delta = (int64_t)(ke >> 10) - 1;
    if (delta <= 0 || n >= cap) break;
    if (lane == 0) {
      const int e = 1023 - (int)(ke & 1023u);
      const int rs = rm.rank[e];
      do_rem_move m;
      m.expert = e;
      m.src_rank = rs;
      m.dst_rank = rr;
      m.reserved = 0;
      m.tokens = delta;
      moves[(int64_t)l * cap + n] = m;
      used[rr] += 1;
      Ld[rr] += delta;
      Ld[rs] -= delta;
      T[e] -= delta;
    }
    ++n;
    __syncthreads();
  }
  __syncthreads();
  if (lane == 0) n_moves[l] = n;
  if (load_out != nullptr)
    for (int r = lane; r < R; r += kWave) load_out[(int64_t)l * R + r] = Ld[r];
  if (tokens_out != nullptr)
    for (int e = lane; e < E; e += kWave) tokens_out[(int64_t)l * E + e] = T[e];
}

// Alg. 2 for layer blockIdx.x (one wavefront).  replicas [L][rep_stride]
// with n_rep[l] valid entries (dst_rank = the rank holding the replica).
__global__ __launch_bounds__(kWave) void k_rem_dispatch(const do_rem_move* replicas, const int32_t* n_rep,
                                                        int rep_stride, const int64_t* tokens, RankMap rm, int E,
                                                        int D, do_rem_move* routes, int32_t* n_routes,
                                                        int64_t* queue_out, int64_t* tokens_out) {
  __shared__ int64_t T[kMaxE];
  __shared__ int64_t Q[kMaxE];
  __shared__ int16_t order[kMaxE];
  const int lane = threadIdx.x, l = blockIdx.x, R = rm.R;
  const int cap = R * D;
  bool ok = load_tokens(tokens + (int64_t)l * E, T, E, lane);
  const int nr = n_rep[l];
  ok = ok && nr >= 0 && nr <= rep_stride;
  const do_rem_move* rep = replicas + (int64_t)l * rep_stride;
  if (ok) {
    bool bad = false;
    for (int i = lane; i < nr; i += kWave) {
      const do_rem_move m = rep[i];
      bad = bad || m.expert < 0 || m.expert >= E || m.dst_rank < 0 || m.dst_rank >= R ||
            m.src_rank != (int)rm.rank[m.expert];
    }
    ok = __ballot(bad) == 0ull;
  }
  for (int r = lane; r < R; r += kWave) Q[r] = 0;
  __syncthreads();
  if (!ok) {
    if (lane == 0) n_routes[l] = -1;
    return;
  }
  if (lane == 0)
    for (int e = 0; e < E; ++e) Q[rm.rank[e]] += T[e];
  __syncthreads();
  int64_t part = 0;
  for (int r = lane; r < R; r += kWave) part += Q[r];
  const int64_t total = wave_sum_i64(part);
  int n = 0;
  for (int d = 0; d < D; ++d) {
    // ranks by queue depth, ties by index: position = number of smaller keys
    for (int r = lane; r < R; r += kWave) {
      const u64 key = ((u64)Q[r] << 10) | (u64)r;
      int pos = 0;
      for (int q = 0; q < R; ++q) pos += (((u64)Q[q] << 10) | (u64)q) < key ? 1 : 0;
      order[pos] = (int16_t)r;
    }
    __syncthreads();
    for (int j = 0; j < R; ++j) {
      const int r = order[j];
      const int64_t Qr = Q[r];
      u64 kb = 0;  // 0: no replica on r
      for (int i = lane; i < nr; i += kWave) {
        const do_rem_move m = rep[i];
        if (m.dst_rank != r) continue;
        const int64_t s = benefit(T[m.expert], Q[m.src_rank], Qr, total, R);
        kb = max(kb, ((u64)(s + 2) << 12) | (u64)(4095 - i));  // s + 2 >= 1 marks a replica
      }
      kb = wave_max_u64(kb);
      const int64_t delta = (int64_t)(kb >> 12) - 2;
      if (kb == 0ull || delta <= 0) continue;
      if (lane == 0) {
        const do_rem_move m = rep[4095 - (int)(kb & 4095u)];
        do_rem_move o;
        o.expert = m.expert;
        o.src_rank = m.src_rank;
        o.dst_rank = r;
        o.reserved = 0;
        o.tokens = delta;
        routes[(int64_t)l * cap + n] = o;
        Q[r] += delta;
        Q[m.src_rank] -= delta;
        T[m.expert] -= delta;
      }
      ++n;
      __syncthreads();
    }
    __syncthreads();
  }
  if (lane == 0) n_routes[l] = n;
  if (queue_out != nullptr)
    for (int r = lane; r < R; r += kWave) queue_out[(int64_t)l * R + r] = Q[r];
  if (tokens_out != nullptr)
    for (int e = lane; e < E; e += kWave) tokens_out[(int64_t)l * E + e] = T[e];
}

}  // namespace

hipError_t launch_rem_allocate(const int64_t* rank_load, const int64_t* tokens, const RankMap& rm, int32_t E,
                               int32_t D, int32_t L, do_rem_move* moves, int32_t* n_moves, int64_t* load_out,
                               int64_t* tokens_out, hipStream_t s) {
  hipLaunchKernelGGL(k_rem_allocate, dim3((unsigned)L), dim3(kWave), 0, s, rank_load, tokens, rm, E, D, moves, n_moves,
                     load_out, tokens_out);
  return hipGetLastError();
}

hipError_t launch_rem_dispatch(const do_rem_move* replicas, const int32_t* n_rep, int32_t rep_stride,
                               const int64_t* tokens, const RankMap& rm, int32_t E, int32_t D, int32_t L,
                               do_rem_move* routes, int32_t* n_routes, int64_t* queue_out, int64_t* tokens_out,
                               hipStream_t s) {
  hipLaunchKernelGGL(k_rem_dispatch, dim3((unsigned)L), dim3(kWave), 0, s, replicas, n_rep, rep_stride, tokens, rm, E,
                     D, routes, n_routes, queue_out, tokens_out);
  return hipGetLastError();
}

}  // namespace dol
