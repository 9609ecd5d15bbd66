// Host side of the C ABI declared in include/doloss.h: argument validation,
// dispatch to the kernels, and the streaming-history handles.
#include <algorithm>
#include <atomic>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "common.h"

#define DOLOSS_API extern "C" __attribute__((visibility("default")))

using dol::u64;

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_prof_start = nullptr;
thread_local hipEvent_t g_prof_stop = nullptr;

// Hands the one-shot profiling events to the Top-K launch `f(pe)`, which binds
// them to its kernel dispatch.
template <typename F>
hipError_t profiled_topk(F&& f) {
  dol::ProfEv pe;
  pe.start = g_prof_start;
  pe.stop = g_prof_stop;
  g_prof_start = g_prof_stop = nullptr;
  return f(pe);
}

// Records the one-shot profiling events around the main kernel launch `f`.
template <typename F>
hipError_t profiled(hipStream_t s, F&& f) {
  hipEvent_t a = g_prof_start, b = g_prof_stop;
  g_prof_start = g_prof_stop = nullptr;
  if (a) {
    const hipError_t e = hipEventRecord(a, s);
    if (e != hipSuccess) return e;
  }
  const hipError_t e = f();
  if (e != hipSuccess) return e;
  if (b) return hipEventRecord(b, s);
  return hipSuccess;
}

do_status fail(do_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

do_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return DO_OK;
  g_last_error = std::string(where) + ": " + hipGetErrorString(e);
  return DO_ERR_HIP;
}

size_t dtype_size(do_dtype dt) { return dt == DO_F32 ? 4 : 2; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

do_status check_dtype(int dt) {
  if (dt != DO_F32 && dt != DO_BF16) return fail(DO_ERR_UNSUPPORTED_DTYPE, "dtype must be DO_F32 or DO_BF16");
  return DO_OK;
}

// Shape checks shared by every entry point.
do_status check_shape(int64_t N, int32_t E, int32_t L) {
  if (E < 1 || E > dol::kMaxE) return fail(DO_ERR_INVALID_ARG, "E must be in [1, 1024]");
  if (L < 1 || L > 65535) return fail(DO_ERR_INVALID_ARG, "L must be in [1, 65535]");
  if (N < 1) return fail(DO_ERR_INVALID_ARG, "N must be >= 1");
  if (N >= (int64_t(1) << 32)) return fail(DO_ERR_OVERFLOW, "N must be < 2^32 (distances are uint32)");
  const unsigned __int128 s2max = (unsigned __int128)(uint64_t)E * (uint64_t)(E - 1) * (uint64_t)N * (uint64_t)N;
  if (s2max >> 64) return fail(DO_ERR_OVERFLOW, "E*(E-1)*N^2 must be < 2^64 (exact sum of squares)");
  return DO_OK;
}

do_status check_k(int32_t k, int32_t E) {
  if (k < 1 || k > E) return fail(DO_ERR_INVALID_ARG, "k must be in [1, E]");
  return DO_OK;
}

do_status check_scores(const void* scores, do_dtype dt) {
  if (scores == nullptr) return fail(DO_ERR_INVALID_ARG, "scores is NULL");
  if (!aligned(scores, dtype_size(dt))) return fail(DO_ERR_INVALID_ARG, "scores is not aligned to its element size");
  return DO_OK;
}

bool fast_layout(const void* scores, do_dtype dt, int32_t E) {
  return aligned(scores, 16) && ((int64_t)E * (int64_t)dtype_size(dt)) % 16 == 0;
}

#define DO_TRY(expr)                 \
  do {                               \
    const do_status st_ = (expr);    \
    if (st_ != DO_OK) return st_;    \
  } while (0)

// Top-K over L layers of [N][E] scores, batched up to kMaxSeg layers per launch.
do_status run_layers(const void* scores, do_dtype dt, int64_t N, int32_t E, int32_t k, int32_t L, u64* bits,
                     uint32_t* cacc, hipStream_t s) {
  const int64_t W = (N + 63) / 64;
  const bool fast = fast_layout(scores, dt, E);
  dol::PathArgs a{};
  a.E = E;
  a.k = k;
  a.bits = bits;
  a.bits_layer_words = (int64_t)E * dol::sig_words(W);
  a.or_partial = 0;
  a.cacc = cacc;
  a.cacc_layer_elems = (int64_t)E * E;
  const size_t layer_bytes = (size_t)N * (size_t)E * dtype_size(dt);
  for (int32_t l0 = 0; l0 < L; l0 += dol::kMaxSeg) {
    const int nseg = (L - l0) < dol::kMaxSeg ? (L - l0) : dol::kMaxSeg;
    dol::SegTable tab{};
    for (int i = 0; i < nseg; ++i) {
      tab.s[i].scores = static_cast<const unsigned char*>(scores) + (size_t)(l0 + i) * layer_bytes;
      tab.s[i].n = N;
      tab.s[i].tok_off = 0;
      tab.s[i].layer = l0 + i;
    }
    DO_TRY(hip_status(
        profiled_topk([&](const dol::ProfEv& pe) { return dol::launch_topk(dt, tab, nseg, a, fast, s, pe); }),
        "top-k launch"));
  }
  return DO_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Check-finite mode (do_set_option DO_OPT_CHECK_FINITE): the calls that rank
// scores first scan them for NaN into a one-word flag, read it back and fail
// before any other launch.  The flag is a file-scope device variable whose
// address is looked up once per device; the scan, the copy and the wait run
// under one host lock, so check-mode calls of a process never share the flag.
// ---------------------------------------------------------------------------
static __device__ uint32_t nan_flag;

namespace {

constexpr int kFlagDevices = 64;
std::atomic<int> g_check_finite{0};
std::mutex g_flag_mu;
uint32_t* g_flag_ptr[kFlagDevices] = {};

do_status check_finite(const void* const* xs, int32_t count, int64_t elems_each, do_dtype dt, hipStream_t s) {
  if (g_check_finite.load(std::memory_order_relaxed) == 0) return DO_OK;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  DO_TRY(hip_status(hipStreamIsCapturing(s, &cs), "hipStreamIsCapturing"));
  if (cs != hipStreamCaptureStatusNone)
    return fail(DO_ERR_INVALID_ARG, "the check-finite mode waits for its scan and cannot run under stream capture");
  int dev = -1;
  DO_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
  if (dev < 0 || dev >= kFlagDevices) return fail(DO_ERR_INVALID_ARG, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_flag_mu);
  if (g_flag_ptr[dev] == nullptr) {
    void* p = nullptr;
    DO_TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(nan_flag)), "hipGetSymbolAddress(nan_flag)"));
    if (p == nullptr) return fail(DO_ERR_HIP, "hipGetSymbolAddress(nan_flag) returned NULL");
    g_flag_ptr[dev] = static_cast<uint32_t*>(p);
  }
  uint32_t* flag = g_flag_ptr[dev];
  DO_TRY(hip_status(dol::launch_fill_u32(flag, 1, 0u, s), "flag clear"));
  for (int32_t i = 0; i < count; ++i)
    DO_TRY(hip_status(dol::launch_nan_scan(xs[i], (int32_t)dtype_size(dt), elems_each, flag, s), "NaN scan"));
  uint32_t seen = 0;
  DO_TRY(hip_status(hipMemcpyAsync(&seen, flag, sizeof(seen), hipMemcpyDeviceToHost, s), "flag copy"));
  DO_TRY(hip_status(hipStreamSynchronize(s), "hipStreamSynchronize"));
  if (seen != 0u) return fail(DO_ERR_NONFINITE, "the scores hold a NaN (check-finite mode); nothing was written");
  return DO_OK;
}

}  // namespace

// Copies of a stream's co-occurrence counters (block b of an append adds its
// counts into copy b % kStreamCopies).  Eight copies, one per XCD, were
// measured: the append kernel took the same time at workload 3 and the
// finalize, which reads every copy, took longer, so one copy is kept.
constexpr int32_t kStreamCopies = 1;

struct do_stream_s {
  int32_t E;
  int32_t k;
  int64_t capacity;
  int64_t W;        // signature words per expert: whole units (a multiple of 8)
  int64_t tokens;
  u64* hist;        // E * W words in the signature layout (sig_off), at the start of one allocation
  uint32_t* cacc;   // kStreamCopies x [E][E] counters, after the history
  uint32_t* snap;   // [E][E]: the totals of the last finalize
  u64* fin;         // 3 words: the finalize's two sums and its ticket
  int64_t words;    // u64 words of the allocation
  int device;
  // Host-side state (the device work it describes is ordered on the caller's
  // stream): the counter copies hold nothing since the last finalize or
  // clear; snap holds totals of this epoch (since the last reset); history
  // words [0, hist_dirty) may hold bits, of this epoch or of earlier ones.
  bool copies_clean;
  bool snap_valid;
  int64_t hist_dirty;
};

DOLOSS_API const char* do_status_string(do_status s) {
  switch (s) {
    case DO_OK: return "DO_OK";
    case DO_ERR_INVALID_ARG: return "DO_ERR_INVALID_ARG";
    case DO_ERR_UNSUPPORTED_DTYPE: return "DO_ERR_UNSUPPORTED_DTYPE";
    case DO_ERR_CAPACITY: return "DO_ERR_CAPACITY";
    case DO_ERR_OVERFLOW: return "DO_ERR_OVERFLOW";
    case DO_ERR_HIP: return "DO_ERR_HIP";
    case DO_ERR_NONFINITE: return "DO_ERR_NONFINITE";
  }
  return "DO_ERR_UNKNOWN";
}

DOLOSS_API const char* do_last_error(void) { return g_last_error.c_str(); }

DOLOSS_API int32_t do_version(void) { return 100; }

DOLOSS_API do_status do_set_option(do_option opt, int32_t value) {
  if (opt == DO_OPT_CHECK_FINITE) {
    if (value != 0 && value != 1) return fail(DO_ERR_INVALID_ARG, "DO_OPT_CHECK_FINITE takes 0 or 1");
    g_check_finite.store(value, std::memory_order_relaxed);
    return DO_OK;
  }
  if (!dol::set_option((int)opt, value)) return fail(DO_ERR_INVALID_ARG, "unknown option or value out of range");
  return DO_OK;
}

DOLOSS_API do_status do_profile_next(hipEvent_t start, hipEvent_t stop) {
  g_prof_start = start;
  g_prof_stop = stop;
  return DO_OK;
}

DOLOSS_API do_status do_topk_signature(const void* scores, do_dtype dtype, int64_t N, int32_t E, int32_t k,
                                       int32_t L, uint64_t* bits, hipStream_t stream) {
  DO_TRY(check_dtype(dtype));
  DO_TRY(check_shape(N, E, L));
  DO_TRY(check_k(k, E));
  DO_TRY(check_scores(scores, dtype));
  if (bits == nullptr || !aligned(bits, 8)) return fail(DO_ERR_INVALID_ARG, "bits is NULL or not 8-byte aligned");
  DO_TRY(check_finite(&scores, 1, N * E * L, dtype, stream));
  return run_layers(scores, dtype, N, E, k, L, reinterpret_cast<u64*>(bits), nullptr, stream);
}

DOLOSS_API do_status do_pairwise_hamming(const uint64_t* bits, int64_t N, int32_t E, int32_t L, uint32_t* D,
                                         hipStream_t stream) {
  DO_TRY(check_shape(N, E, L));
  if (bits == nullptr || !aligned(bits, 8)) return fail(DO_ERR_INVALID_ARG, "bits is NULL or not 8-byte aligned");
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  const int64_t W = (N + 63) / 64;
  DO_TRY(hip_status(dol::launch_fill_u32(D, (int64_t)L * E * E, 0u, stream), "fill"));
  if (E <= dol::kFastMaxE && dol::gram_mfma_enabled())
    DO_TRY(hip_status(dol::launch_gram_mfma(reinterpret_cast<const u64*>(bits), W, E, L, D, stream), "gram"));
  else
    DO_TRY(hip_status(
        dol::launch_gram_bits(reinterpret_cast<const u64*>(bits), W, dol::sig_words(W), E, L, D, stream), "gram"));
  return hip_status(dol::launch_finalize(D, D, nullptr, E, L, stream), "finalize");
}

DOLOSS_API do_status do_loss(const uint32_t* D, int32_t E, int32_t L, do_loss_result* out, hipStream_t stream) {
  DO_TRY(check_shape(1, E, L));
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  if (out == nullptr || !aligned(out, 8)) return fail(DO_ERR_INVALID_ARG, "out is NULL or not 8-byte aligned");
  return hip_status(dol::launch_loss(D, E, L, out, stream), "loss");
}

DOLOSS_API do_status do_fused(const void* scores, do_dtype dtype, int64_t N, int32_t E, int32_t k, int32_t L,
                              uint64_t* bits, uint32_t* D, do_loss_result* out, hipStream_t stream) {
  DO_TRY(check_dtype(dtype));
  DO_TRY(check_shape(N, E, L));
  DO_TRY(check_k(k, E));
  DO_TRY(check_scores(scores, dtype));
  if (bits != nullptr && !aligned(bits, 8)) return fail(DO_ERR_INVALID_ARG, "bits is not 8-byte aligned");
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  if (out == nullptr || !aligned(out, 8)) return fail(DO_ERR_INVALID_ARG, "out is NULL or not 8-byte aligned");
  if (E > dol::kFastMaxE && bits == nullptr)
    return fail(DO_ERR_INVALID_ARG, "do_fused needs a bits buffer when E > 256");
  DO_TRY(check_finite(&scores, 1, N * E * L, dtype, stream));
  DO_TRY(hip_status(dol::launch_fill_u32(D, (int64_t)L * E * E, 0u, stream), "fill"));
  if (E <= dol::kFastMaxE) {
    DO_TRY(run_layers(scores, dtype, N, E, k, L, reinterpret_cast<u64*>(bits), D, stream));
  } else {
    DO_TRY(run_layers(scores, dtype, N, E, k, L, reinterpret_cast<u64*>(bits), nullptr, stream));
    const int64_t W = (N + 63) / 64;
    DO_TRY(hip_status(
        dol::launch_gram_bits(reinterpret_cast<const u64*>(bits), W, dol::sig_words(W), E, L, D, stream), "gram"));
  }
  return hip_status(dol::launch_finalize(D, D, out, E, L, stream), "finalize");
}

DOLOSS_API do_status do_surrogate(const void* p, do_dtype dtype, int64_t N, int32_t E, int32_t k, int32_t L,
                                  const uint64_t* bits, const uint32_t* D, double scale, double* loss, float* grad,
                                  hipStream_t stream) {
  DO_TRY(check_dtype(dtype));
  DO_TRY(check_shape(N, E, L));
  DO_TRY(check_k(k, E));
  if (E > dol::kFastMaxE) return fail(DO_ERR_INVALID_ARG, "do_surrogate supports E <= 256");
  if ((int64_t)(E - 1) * N >= (int64_t(1) << 31))
    return fail(DO_ERR_OVERFLOW, "(E-1)*N must be < 2^31 (row sums of G are int32)");
  if (p == nullptr || !aligned(p, 2 * dtype_size(dtype)))
    return fail(DO_ERR_INVALID_ARG, "p is NULL or not aligned to two elements");
  if (bits == nullptr || !aligned(bits, 8)) return fail(DO_ERR_INVALID_ARG, "bits is NULL or not 8-byte aligned");
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  if (loss == nullptr || !aligned(loss, 8)) return fail(DO_ERR_INVALID_ARG, "loss is NULL or not 8-byte aligned");
  if (grad != nullptr && !aligned(grad, 8)) return fail(DO_ERR_INVALID_ARG, "grad is not 8-byte aligned");
  if (!(scale == scale) || scale - scale != 0.0) return fail(DO_ERR_INVALID_ARG, "scale must be finite");
  dol::SurrogateArgs a{};
  a.p = p;
  a.bits = reinterpret_cast<const u64*>(bits);
  a.D = D;
  a.loss = loss;
  a.grad = grad;
  a.N = N;
  a.W = (N + 63) / 64;
  a.E = E;
  a.L = L;
  a.s64 = scale / ((double)N * (double)N * (double)k);
  a.s32 = (float)a.s64;
  DO_TRY(hip_status(dol::launch_fill_u64(reinterpret_cast<u64*>(loss), L, stream), "fill"));
  return hip_status(profiled(stream, [&] { return dol::launch_surrogate(dtype, a, stream); }), "surrogate");
}

DOLOSS_API do_status do_load_stats(const uint64_t* bits, int64_t N, int64_t ld, int32_t E, int32_t k, int32_t L,
                                   const void* p, do_dtype dtype, const int32_t* expert_rank, int32_t R,
                                   uint32_t* loads, do_load_stats_result* out, hipStream_t stream) {
  DO_TRY(check_shape(N, E, L));
  DO_TRY(check_k(k, E));
  const int64_t W = (N + 63) / 64;
  if (ld == 0) ld = dol::sig_words(W);
  if (ld < dol::sig_words(W) || ld % 8 != 0)
    return fail(DO_ERR_INVALID_ARG, "ld must be 0, or a multiple of 8 of at least 8 * ceil(N/512)");
  if (bits == nullptr || !aligned(bits, 8)) return fail(DO_ERR_INVALID_ARG, "bits is NULL or not 8-byte aligned");
  if (loads == nullptr || !aligned(loads, 4)) return fail(DO_ERR_INVALID_ARG, "loads is NULL or not 4-byte aligned");
  if (out == nullptr || !aligned(out, 8)) return fail(DO_ERR_INVALID_ARG, "out is NULL or not 8-byte aligned");
  if (p != nullptr) {
    DO_TRY(check_dtype(dtype));
    DO_TRY(check_scores(p, dtype));
  }
  dol::RankMap rm{};
  rm.R = E;
  rm.given = 0;
  if (expert_rank != nullptr) {
    if (R < 1 || R > dol::kMaxE) return fail(DO_ERR_INVALID_ARG, "R must be in [1, 1024]");
    for (int32_t i = 0; i < E; ++i) {
      if (expert_rank[i] < 0 || expert_rank[i] >= R)
        return fail(DO_ERR_INVALID_ARG, "expert_rank[" + std::to_string(i) + "] is not in [0, R)");
      rm.rank[i] = (uint16_t)expert_rank[i];
    }
    rm.R = R;
    rm.given = 1;
  }
  return hip_status(dol::launch_load_stats(reinterpret_cast<const u64*>(bits), N, ld, E, k, L, p, dtype, rm, loads,
                                           out, stream),
                    "load stats");
}

namespace {

// Shared checks of the REM entry points; fills the home-rank map.
do_status check_rem(const int32_t* expert_rank, int32_t E, int32_t R, int32_t D, int32_t L, dol::RankMap& rm) {
  if (E < 1 || E > dol::kMaxE) return fail(DO_ERR_INVALID_ARG, "E must be in [1, 1024]");
  if (R < 1 || R > dol::kMaxE) return fail(DO_ERR_INVALID_ARG, "R must be in [1, 1024]");
  if (D < 1 || (int64_t)R * D > 4096) return fail(DO_ERR_INVALID_ARG, "D must be >= 1 with R*D <= 4096");
  if (L < 1 || L > 65535) return fail(DO_ERR_INVALID_ARG, "L must be in [1, 65535]");
  if (expert_rank == nullptr) return fail(DO_ERR_INVALID_ARG, "expert_rank is NULL");
  for (int32_t i = 0; i < E; ++i) {
    if (expert_rank[i] < 0 || expert_rank[i] >= R)
      return fail(DO_ERR_INVALID_ARG, "expert_rank[" + std::to_string(i) + "] is not in [0, R)");
    rm.rank[i] = (uint16_t)expert_rank[i];
  }
  rm.R = R;
  rm.given = 1;
  return DO_OK;
}

}  // namespace

DOLOSS_API do_status do_rem_allocate(const int64_t* rank_load, const int64_t* expert_tokens,
                                     const int32_t* expert_rank, int32_t E, int32_t R, int32_t D, int32_t L,
                                     do_rem_move* moves, int32_t* n_moves, int64_t* load_out, int64_t* tokens_out,
                                     hipStream_t stream) {
  dol::RankMap rm{};
  DO_TRY(check_rem(expert_rank, E, R, D, L, rm));
  if (rank_load != nullptr && !aligned(rank_load, 8)) return fail(DO_ERR_INVALID_ARG, "rank_load is not 8-byte aligned");
  if (expert_tokens == nullptr || !aligned(expert_tokens, 8))
    return fail(DO_ERR_INVALID_ARG, "expert_tokens is NULL or not 8-byte aligned");
  if (moves == nullptr || !aligned(moves, 8)) return fail(DO_ERR_INVALID_ARG, "moves is NULL or not 8-byte aligned");
  if (n_moves == nullptr || !aligned(n_moves, 4)) return fail(DO_ERR_INVALID_ARG, "n_moves is NULL or not 4-byte aligned");
  if ((load_out != nullptr && !aligned(load_out, 8)) || (tokens_out != nullptr && !aligned(tokens_out, 8)))
    return fail(DO_ERR_INVALID_ARG, "load_out / tokens_out is not 8-byte aligned");
  return hip_status(dol::launch_rem_allocate(rank_load, expert_tokens, rm, E, D, L, moves, n_moves, load_out,
                                             tokens_out, stream),
                    "rem allocate");
}

DOLOSS_API do_status do_rem_dispatch(const do_rem_move* replicas, const int32_t* n_replicas, int32_t replica_stride,
                                     const int64_t* expert_tokens, const int32_t* expert_rank, int32_t E, int32_t R,
                                     int32_t D, int32_t L, do_rem_move* routes, int32_t* n_routes, int64_t* queue_out,
                                     int64_t* tokens_out, hipStream_t stream) {
  dol::RankMap rm{};
  DO_TRY(check_rem(expert_rank, E, R, D, L, rm));
  if (replica_stride < 1 || replica_stride > 4096)
    return fail(DO_ERR_INVALID_ARG, "replica_stride must be in [1, 4096]");
  if (replicas == nullptr || !aligned(replicas, 8))
    return fail(DO_ERR_INVALID_ARG, "replicas is NULL or not 8-byte aligned");
  if (n_replicas == nullptr || !aligned(n_replicas, 4))
    return fail(DO_ERR_INVALID_ARG, "n_replicas is NULL or not 4-byte aligned");
  if (expert_tokens == nullptr || !aligned(expert_tokens, 8))
    return fail(DO_ERR_INVALID_ARG, "expert_tokens is NULL or not 8-byte aligned");
  if (routes == nullptr || !aligned(routes, 8)) return fail(DO_ERR_INVALID_ARG, "routes is NULL or not 8-byte aligned");
  if (n_routes == nullptr || !aligned(n_routes, 4))
    return fail(DO_ERR_INVALID_ARG, "n_routes is NULL or not 4-byte aligned");
  if ((queue_out != nullptr && !aligned(queue_out, 8)) || (tokens_out != nullptr && !aligned(tokens_out, 8)))
    return fail(DO_ERR_INVALID_ARG, "queue_out / tokens_out is not 8-byte aligned");
  return hip_status(dol::launch_rem_dispatch(replicas, n_replicas, replica_stride, expert_tokens, rm, E, D, L, routes,
                                             n_routes, queue_out, tokens_out, stream),
                    "rem dispatch");
}

DOLOSS_API do_status do_stream_create(int32_t E, int32_t k, int64_t capacity_tokens, do_stream** out) {
  if (out == nullptr) return fail(DO_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  DO_TRY(check_shape(capacity_tokens, E, 1));
  DO_TRY(check_k(k, E));
  do_stream* h = new (std::nothrow) do_stream_s{};  // no exception may cross the C ABI
  if (h == nullptr) return fail(DO_ERR_HIP, "do_stream_create: host allocation failed");
  h->E = E;
  h->k = k;
  h->capacity = capacity_tokens;
  h->W = dol::sig_words((capacity_tokens + 63) / 64);  // whole units
  h->tokens = 0;
  // one allocation: the history, the counter copies, the snapshot, the finalize words
  const int64_t mat_words = ((int64_t)E * E + 1) / 2;  // one E x E uint32 matrix, in u64 words
  h->words = (int64_t)E * h->W + (kStreamCopies + 1) * mat_words + 4;
  h->copies_clean = true;
  h->snap_valid = false;
  h->hist_dirty = 0;
  hipError_t e = hipGetDevice(&h->device);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->hist), (size_t)h->words * sizeof(u64));
  if (e == hipSuccess) {
    u64* c = h->hist + (int64_t)E * h->W;
    h->cacc = reinterpret_cast<uint32_t*>(c);
    h->snap = reinterpret_cast<uint32_t*>(c + kStreamCopies * mat_words);
    h->fin = c + (kStreamCopies + 1) * mat_words;
    e = hipMemset(h->hist, 0, (size_t)h->words * sizeof(u64));
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    if (h->hist) (void)hipFree(h->hist);
    delete h;
    return hip_status(e, "do_stream_create");
  }
  *out = h;
  return DO_OK;
}

namespace {

do_status check_handle(const do_stream* h) {
  if (h == nullptr) return fail(DO_ERR_INVALID_ARG, "stream handle is NULL");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device)
    return fail(DO_ERR_INVALID_ARG, "the handle's device is not the current device");
  return DO_OK;
}

// Zeroes words [w0, w1) of every expert row of the history.
hipError_t clear_history_words(do_stream* h, int64_t w0, int64_t w1, hipStream_t s) {
  if (w1 <= w0) return hipSuccess;
  if (w0 == 0 && w1 == h->W) return dol::launch_fill_u64(h->hist, (int64_t)h->E * h->W, s);
  return dol::launch_fill_sig_words(h->hist, h->E, w0, w1 - w0, s);
}

do_status stream_append(do_stream* h, const void* const* scores, do_dtype dtype, int64_t n, int32_t count,
                        hipStream_t stream) {
  DO_TRY(check_handle(h));
  DO_TRY(check_dtype(dtype));
  if (n < 0) return fail(DO_ERR_INVALID_ARG, "n_tokens must be >= 0");
  if (count < 1 || count > dol::kMaxSeg) return fail(DO_ERR_INVALID_ARG, "count must be in [1, 64]");
  if (n == 0) return DO_OK;  // nothing is read: the score pointers may be NULL
  bool fast = true;
  for (int i = 0; i < count; ++i) {
    DO_TRY(check_scores(scores[i], dtype));
    fast = fast && fast_layout(scores[i], dtype, h->E);
  }
  if ((h->capacity - h->tokens) / count < n)
    return fail(DO_ERR_CAPACITY, "append would exceed the history capacity");
  DO_TRY(check_finite(scores, count, n * h->E, dtype, stream));
  // Words that this append writes.  When the micro-batches start and end on
  // word boundaries every word is written whole by exactly one of them, with
  // plain stores.  Otherwise words shared between micro-batches are OR-ed, so
  // words not yet written in this epoch that may still hold bits from before
  // the last reset are cleared first.
  const int64_t w_fresh = (h->tokens + 63) / 64;  // first word with no bits of this epoch
  const int64_t w_end = (h->tokens + (int64_t)count * n + 63) / 64;
  const bool aligned_words = (h->tokens % 64) == 0 && (n % 64) == 0;
  if (!aligned_words && w_fresh < h->hist_dirty) {
    DO_TRY(hip_status(clear_history_words(h, w_fresh, h->hist_dirty, stream), "history clear"));
    h->hist_dirty = w_fresh;
  }
  dol::PathArgs a{};
  a.E = h->E;
  a.k = h->k;
  a.bits = h->hist;
  a.bits_layer_words = (int64_t)h->E * h->W;
  a.or_partial = 1;
  const bool gram = h->E <= dol::kFastMaxE;  // wider E: Gram of the whole history at finalize
  a.cacc = gram ? h->cacc : nullptr;
  a.cacc_layer_elems = (int64_t)h->E * h->E;
  a.ncopies = kStreamCopies;
  a.cacc_copy_elems = 2 * (((int64_t)h->E * h->E + 1) / 2);
  dol::SegTable tab{};
  for (int i = 0; i < count; ++i) {
    tab.s[i].scores = scores[i];
    tab.s[i].n = n;
    tab.s[i].tok_off = h->tokens + (int64_t)i * n;
    tab.s[i].layer = 0;
  }
  DO_TRY(hip_status(profiled_topk([&](const dol::ProfEv& pe) {
                      return dol::launch_topk(dtype, tab, count, a, fast, stream, pe);
                    }),
                    "stream append"));
  h->tokens += (int64_t)count * n;
  h->hist_dirty = std::max(h->hist_dirty, w_end);
  if (gram) h->copies_clean = false;
  return DO_OK;
}

}  // namespace

DOLOSS_API do_status do_stream_append(do_stream* h, const void* scores, do_dtype dtype, int64_t n_tokens,
                                      hipStream_t stream) {
  const void* one[1] = {scores};
  return stream_append(h, one, dtype, n_tokens, 1, stream);
}

DOLOSS_API do_status do_stream_append_many(do_stream* h, const void* const* scores, do_dtype dtype,
                                           int64_t n_tokens_each, int32_t count, hipStream_t stream) {
  if (scores == nullptr) return fail(DO_ERR_INVALID_ARG, "scores pointer array is NULL");
  if (count < 1 || count > dol::kMaxSeg) return fail(DO_ERR_INVALID_ARG, "count must be in [1, 64]");
  return stream_append(h, scores, dtype, n_tokens_each, count, stream);
}

DOLOSS_API do_status do_stream_finalize(do_stream* h, uint32_t* D, do_loss_result* out, hipStream_t stream) {
  DO_TRY(check_handle(h));
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  if (out == nullptr || !aligned(out, 8)) return fail(DO_ERR_INVALID_ARG, "out is NULL or not 8-byte aligned");
  if (h->E <= dol::kFastMaxE) {
    const int64_t copy_elems = 2 * (((int64_t)h->E * h->E + 1) / 2);
    DO_TRY(hip_status(dol::launch_finalize_stream(h->cacc, kStreamCopies, copy_elems, h->snap, h->snap_valid ? 1 : 0,
                                                  D, out, h->E, h->fin, stream),
                      "finalize"));
    h->copies_clean = true;  // the totals now live in the snapshot
    h->snap_valid = true;
    return DO_OK;
  }
  // wider E: the Gram of the words holding this epoch's tokens
  DO_TRY(hip_status(dol::launch_fill_u32(D, (int64_t)h->E * h->E, 0u, stream), "fill"));
  DO_TRY(hip_status(dol::launch_gram_bits(h->hist, (h->tokens + 63) / 64, h->W, h->E, 1, D, stream), "gram"));
  return hip_status(dol::launch_finalize(D, D, out, h->E, 1, stream), "finalize");
}

DOLOSS_API do_status do_stream_reset(do_stream* h, hipStream_t stream) {
  DO_TRY(check_handle(h));
  // The history is cleared lazily (see stream_append); the counter copies
  // need a clear only if an append added to them since the last finalize.
  if (!h->copies_clean) {
    const int64_t mat_words = ((int64_t)h->E * h->E + 1) / 2;
    DO_TRY(hip_status(dol::launch_fill_u64(reinterpret_cast<u64*>(h->cacc), kStreamCopies * mat_words, stream),
                      "reset"));
    h->copies_clean = true;
  }
  h->snap_valid = false;
  h->tokens = 0;
  return DO_OK;
}

DOLOSS_API do_status do_stream_destroy(do_stream* h) {
  if (h == nullptr) return DO_OK;
  // wait for the handle's own device (the current one may differ), then free
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  const bool other = e == hipSuccess && cur != h->device;
  if (other) e = hipSetDevice(h->device);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  const hipError_t e1 = hipFree(h->hist);  // the counters share this allocation
  if (other) (void)hipSetDevice(cur);
  delete h;
  if (e == hipSuccess) e = e1;
  return hip_status(e, "do_stream_destroy");
}

DOLOSS_API const uint64_t* do_stream_bits(const do_stream* h) {
  return h ? reinterpret_cast<const uint64_t*>(h->hist) : nullptr;
}

DOLOSS_API int64_t do_stream_tokens(const do_stream* h) { return h ? h->tokens : -1; }

DOLOSS_API int64_t do_stream_words_per_expert(const do_stream* h) { return h ? h->W : -1; }

// ---------------------------------------------------------------------------
// Global batch without any allocation (do_global_batch_noalloc).  The running
// co-occurrence counts and the split finalize's two sums and ticket live in a
// file-scope device array instead of a handle's allocation.  Its address is
// looked up once per device with hipGetSymbolAddress (in host code the
// array's name is not a device address) and only that pointer is used.
// ---------------------------------------------------------------------------
namespace {

constexpr int32_t kNoAllocMaxE = dol::kFastMaxE;                                  // 256 experts
constexpr int64_t kNoAllocCountWords = (int64_t)kNoAllocMaxE * kNoAllocMaxE / 2;  // E*E uint32 counters
constexpr int64_t kNoAllocWords = kNoAllocCountWords + 4;                         // + sums, ticket, pad
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) u64 scratch[kNoAllocWords];  // 256 KiB + 32 B on every device

namespace {

std::mutex g_scratch_mu;
u64* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (looked up on the
// first call on that device).
do_status scratch_on_device(u64** out) {
  int dev = -1;
  DO_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
  if (dev < 0 || dev >= kMaxDevices) return fail(DO_ERR_INVALID_ARG, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    DO_TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
    if (p == nullptr) return fail(DO_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = static_cast<u64*>(p);
  }
  *out = g_scratch_ptr[dev];
  return DO_OK;
}

}  // namespace

DOLOSS_API do_status do_global_batch_noalloc(const void* const* scores, do_dtype dtype, int64_t n_tokens_each,
                                             int32_t count, int32_t E, int32_t k, uint64_t* hist, uint32_t* D,
                                             do_loss_result* out, hipStream_t stream) {
  DO_TRY(check_dtype(dtype));
  if (E > kNoAllocMaxE)
    return fail(DO_ERR_INVALID_ARG, "do_global_batch_noalloc supports E <= 256 (its static counters hold 256 x 256)");
  if (count < 1 || count > dol::kMaxSeg) return fail(DO_ERR_INVALID_ARG, "count must be in [1, 64]");
  if (n_tokens_each < 1) return fail(DO_ERR_INVALID_ARG, "n_tokens_each must be >= 1");
  if (n_tokens_each > ((int64_t(1) << 32) - 1) / count)
    return fail(DO_ERR_OVERFLOW, "count * n_tokens_each must be < 2^32 (distances are uint32)");
  const int64_t N = (int64_t)count * n_tokens_each;
  DO_TRY(check_shape(N, E, 1));
  DO_TRY(check_k(k, E));
  if (scores == nullptr) return fail(DO_ERR_INVALID_ARG, "scores pointer array is NULL");
  bool fast = true;
  for (int i = 0; i < count; ++i) {
    DO_TRY(check_scores(scores[i], dtype));
    fast = fast && fast_layout(scores[i], dtype, E);
  }
  if (hist == nullptr || !aligned(hist, 8)) return fail(DO_ERR_INVALID_ARG, "hist is NULL or not 8-byte aligned");
  if (D == nullptr || !aligned(D, 4)) return fail(DO_ERR_INVALID_ARG, "D is NULL or not 4-byte aligned");
  if (out == nullptr || !aligned(out, 8)) return fail(DO_ERR_INVALID_ARG, "out is NULL or not 8-byte aligned");
  u64* sp = nullptr;
  DO_TRY(scratch_on_device(&sp));
  uint32_t* cacc = reinterpret_cast<uint32_t*>(sp);
  u64* fin = sp + kNoAllocCountWords;
  const int64_t Wp = dol::sig_words((N + 63) / 64);
  // every word the appends OR into starts at zero, and so do the counts and
  // the finalize's sums (fill kernels: no memset nodes under graph capture)
  DO_TRY(hip_status(dol::launch_fill_u64(reinterpret_cast<u64*>(hist), (int64_t)E * Wp, stream), "fill history"));
  DO_TRY(hip_status(dol::launch_fill_u64(sp, ((int64_t)E * E + 1) / 2, stream), "fill counters"));
  DO_TRY(hip_status(dol::launch_fill_u64(fin, 3, stream), "fill finalize words"));
  dol::PathArgs a{};
  a.E = E;
  a.k = k;
  a.bits = reinterpret_cast<u64*>(hist);
  a.bits_layer_words = (int64_t)E * Wp;
  a.or_partial = 1;
  a.cacc = cacc;
  a.cacc_layer_elems = (int64_t)E * E;
  dol::SegTable tab{};
  for (int i = 0; i < count; ++i) {
    tab.s[i].scores = scores[i];
    tab.s[i].n = n_tokens_each;
    tab.s[i].tok_off = (int64_t)i * n_tokens_each;
    tab.s[i].layer = 0;
  }
  DO_TRY(hip_status(profiled_topk([&](const dol::ProfEv& pe) {
                      return dol::launch_topk(dtype, tab, count, a, fast, stream, pe);
                    }),
                    "global batch"));
  return hip_status(dol::launch_finalize_split(cacc, D, out, E, fin, stream), "finalize");
}
