// Internal declarations shared by the kernels and the host dispatch of the
// DO-loss library.  Not part of the public ABI (see include/doloss.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/doloss.h"

namespace dol {

using u64 = unsigned long long;
typedef unsigned long long v2u64 __attribute__((ext_vector_type(2)));  // 16-byte vector of two words

constexpr int kWave = 64;
constexpr int kFusedWaves = 8;                       // waves per block of the Top-K (+Gram) kernel
constexpr int kFusedThreads = kFusedWaves * kWave;   // 512
constexpr int kMaxSeg = 64;                          // score segments per launch
constexpr int kMaxE = 1024;
constexpr int kFastMaxE = 256;                       // expert index fits the 8 low bits of a composite key
constexpr int kFastMaxK = 8;                         // width of the in-register Top-K network

// One contiguous block of token rows [n][E] and where its signatures go.
struct Segment {
  const void* scores;  // device, [n][E]
  int64_t n;           // tokens in this segment
  int64_t tok_off;     // bit position of token 0 in the output signature rows
  int32_t layer;       // output layer (bits / accumulator / D index)
  int32_t pad_;
};

// Segments of one launch.  tile_start[i] is the number of 8-word units
// (512 output positions, 8-aligned within their segment) of segments
// 0..i-1, filled by launch_topk: the blocks of a launch split the
// concatenated unit range [0, tile_start[nseg]) evenly.
struct SegTable {
  Segment s[kMaxSeg];
  int64_t tile_start[kMaxSeg + 1];
  int32_t nseg;
  int32_t pad_;
};

// Where one launch writes its results.
// Signature layout.  A layer of N tokens is U = ceil(N/512) units of 512
// tokens, and unit u holds the 8 words of every expert, expert after expert
// (word s of the unit: tokens 512u + 64s .. 512u + 64s + 63, bit b = token
// 512u + 64s + b).  Word w of expert e sits at sig_off(w, e, E) words from
// the layer's start, and a layer takes E * sig_words(W) words, W = ceil(N/64).
// The Top-K kernel writes a unit's signatures as one contiguous block.
__host__ __device__ __forceinline__ int64_t sig_words(int64_t W) { return (W + 7) & ~int64_t(7); }
__host__ __device__ __forceinline__ int64_t sig_off(int64_t w, int64_t e, int64_t E) {
  return ((w >> 3) * E + e) * 8 + (w & 7);
}

struct PathArgs {
  int32_t E;
  int32_t k;
  u64* bits;                // nullable: signatures, the layers E * sig_words(W) words apart (sig_off)
  int64_t bits_layer_words; // words per layer of `bits`
  int32_t or_partial;       // words shared with other segments are OR-ed (history), else stored
  int32_t ncopies;          // copies of the accumulators (0 or 1: one); block b adds into copy b % ncopies
  uint32_t* cacc;           // nullable: co-occurrence accumulators [layer][E][E], upper triangle
  int64_t cacc_layer_elems;
  int64_t cacc_copy_elems;  // distance between copies
};

// Arguments of the surrogate-loss kernel.
struct SurrogateArgs {
  const void* p;       // [L][N][E] routing probabilities (fp32 or bf16)
  const u64* bits;     // signatures (layout: sig_off), W = ceil(N/64) words per expert
  const uint32_t* D;   // [L][E][E] distances G
  double* loss;        // [L], accumulated into (zeroed by the caller)
  float* grad;         // nullable [L][N][E]
  int64_t N, W;
  int32_t E, L;
  double s64;          // scale / (N^2 k)
  float s32;
  int32_t pad_;
};

struct DevInfo {
  int device;
  int cu_count;
};
DevInfo device_info();

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);
hipError_t launch_fill_u64(u64* p, int64_t n, hipStream_t s);
// Sets *flag to 1 when any of the n elements at x (fp32 or bf16 bit patterns,
// elem_bytes 4 or 2, x aligned to its element size) is a NaN; else leaves it.
hipError_t launch_nan_scan(const void* x, int32_t elem_bytes, int64_t n, uint32_t* flag, hipStream_t s);
// Zeroes signature words [w0, w0 + nw) of all E experts of one layer at p.
hipError_t launch_fill_sig_words(u64* p, int32_t E, int64_t w0, int64_t nw, hipStream_t s);

// A caller's timing events for one kernel dispatch (either may be null):
// bound to the dispatch itself, so their interval is that kernel's run.
struct ProfEv {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// Top-K signatures of `nseg` segments; with a.cacc also the co-occurrence
// counts of each segment's tokens added into a.cacc.  `pe` times the launch.
hipError_t launch_topk(do_dtype dt, SegTable& tab, int nseg, const PathArgs& a, bool fast_ok, hipStream_t s,
                       const ProfEv& pe = ProfEv{});

// Co-occurrence counts of existing signatures: cacc[l][i][j] += popcount(F_i & F_j), i <= j,
// over words [0, W) of each expert; ld = words per expert of a layer (a
// multiple of 8), layers E * ld words apart (signature layout: sig_off).
hipError_t launch_gram_bits(const u64* bits, int64_t W, int64_t ld, int32_t E, int32_t L, uint32_t* cacc,
                            hipStream_t s);
// The same Gram on fp4 MFMA tiles (E <= 256): counts added into cacc [L][E][E]
// (upper triangle, zeroed by the caller); layers E * sig_words(W) words apart.
hipError_t launch_gram_mfma(const u64* bits, int64_t W, int32_t E, int32_t L, uint32_t* cacc, hipStream_t s);
// False when do_set_option selects the popcount Gram (a comparison switch).
bool gram_mfma_enabled();
// do_set_option: false for an unknown option or a value out of range.
bool set_option(int opt, int value);

// D = c_ii + c_jj - 2 c_ij (symmetric, zero diagonal); out (nullable) = loss.
// cacc may alias D.
hipError_t launch_finalize(const uint32_t* cacc, uint32_t* D, do_loss_result* out, int32_t E, int32_t L,
                           hipStream_t s);

// Surrogate loss (Eq. 7) and its gradient; a.loss must be zero.
hipError_t launch_surrogate(do_dtype dt, const SurrogateArgs& a, hipStream_t s);

// Expert-to-rank placement passed by value to the load-statistics finalize.
struct RankMap {
  uint16_t rank[kMaxE];
  int32_t R;      // ranks; the placement is the identity (R = E) when `given` is 0
  int32_t given;
};

// Load statistics: loads[l][e] = popcount of the signature of expert e of
// layer l (words [0, ceil(N/64)); ld = words per expert of a layer, a
// multiple of 8, layers E * ld words apart); with p, the Local-LBL sum
// accumulated into out[l].lbl (zeroed by the caller) and scaled in the
// finalize, which also writes total / max / min / MaxVio.
hipError_t launch_load_stats(const u64* bits, int64_t N, int64_t ld, int32_t E, int32_t k, int32_t L, const void* p,
                             do_dtype dt, const RankMap& rm, uint32_t* loads, do_load_stats_result* out,
                             hipStream_t s);

// REM scheduling (one wavefront per layer); the rank map gives the home
// ranks (rm.R ranks, rm.given set).
hipError_t launch_rem_allocate(const int64_t* rank_load, const int64_t* tokens, const RankMap& rm, int32_t E,
                               int32_t D, int32_t L, do_rem_move* moves, int32_t* n_moves, int64_t* load_out,
                               int64_t* tokens_out, hipStream_t s);
hipError_t launch_rem_dispatch(const do_rem_move* replicas, const int32_t* n_rep, int32_t rep_stride,
                               const int64_t* tokens, const RankMap& rm, int32_t E, int32_t D, int32_t L,
                               do_rem_move* routes, int32_t* n_routes, int64_t* queue_out, int64_t* tokens_out,
                               hipStream_t s);

// Loss of arbitrary distance matrices.
// One layer (E <= 256) over ceil(E/8) blocks; fin: three u64 that are zero
// before the call and zero again after it (cacc must not alias D).
hipError_t launch_finalize_split(const uint32_t* cacc, uint32_t* D, do_loss_result* out, int32_t E, u64* fin,
                                 hipStream_t s);
hipError_t launch_loss(const uint32_t* D, int32_t E, int32_t L, do_loss_result* out, hipStream_t s);

// The stream's finalize (one layer, E <= 256): the co-occurrence counts are
// snap (if snap_valid) plus the sum of the ncopies copies (copy_elems apart);
// writes D and out, then stores the totals in snap and zeroes the copies, so
// that a repeated finalize gives the same result.  fin: three u64, zero before
// and after.
hipError_t launch_finalize_stream(uint32_t* copies, int32_t ncopies, int64_t copy_elems, uint32_t* snap,
                                  int32_t snap_valid, uint32_t* D, do_loss_result* out, int32_t E, u64* fin,
                                  hipStream_t s);

}  // namespace dol
