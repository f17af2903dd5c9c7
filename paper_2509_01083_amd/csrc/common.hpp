// Internal definitions shared by the HIP translation units of libdsde.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dsde.h"

namespace dsde {

constexpr int kThreads = 256;              // threads per workgroup of the row kernels (4 wavefronts)
constexpr int kWaves = kThreads / 64;
constexpr int kEltsPerThread = 32;         // logits per row per thread in one chunk
constexpr int kChunk = kThreads * kEltsPerThread;  // logits per row chunk (8192)
constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLn2 = 0.6931471805599453;
// Temperatures outside [2^-16, 2^16] are rejected so that every scaled logit
// z * log2(e) / T of a finite logit with |z| <= 2^64 stays far inside fp32.
constexpr float kMinTemp = 1.52587890625e-05f, kMaxTemp = 65536.0f;

// One row pair of the statistics pass, in processing order: the drafted
// position (pair index = draft row), its target row (-1 when the layout is
// invalid), the log2-domain scale c = log2(e) / T_b as raw float bits, and
// its slot b * k_max + j, under which its chunk partials and gathered logits
// are stored (so that their address depends on the sequence alone).
// Sign bit of WorkItem::scale_bits: a greedy pair (T_b = 0), whose chunk
// argmax of the target row is also wanted.
constexpr uint32_t kGreedyBit = 0x80000000u;

struct WorkItem {
  int32_t pair;
  int32_t target_row;
  uint32_t scale_bits;
  int32_t slot;
};

// Row statistics of one chunk of one drafted row pair, relative to the
// chunk's reference shifts mt, md (log2 domain):
//   sp = sum 2^(z_t c - mt),  sq = sum 2^(z_d c - md),
//   a  = sum 2^(z_t c - mt) * ((z_t c - mt) - (z_d c - md)),
//   h  = sum 2^(z_d c - md) * (z_d c - md).
struct alignas(16) PairChunk {
  float mt, md;
  double sp, sq, a, h;
};

// Greedy pairs: the target row's largest logit in a chunk (raw, unscaled) and
// the smallest token id holding it.
struct ChunkArg {
  float zmax;
  int32_t idx;
};

// The target and draft logits at the drafted token, captured by the chunk
// that holds it.
struct Gathered {
  float zt, zd;
};

// Largest vocabulary: the per-sequence kernel keeps the draw-weight totals of
// every chunk of a row in LDS.
constexpr int kMaxChunks = 512;
static_assert(int64_t(kMaxChunks) * kChunk == DSDE_MAX_VOCAB, "vocabulary limit of the ABI");

inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

struct WorkspaceLayout {
  size_t work, pair_chunk, gathered, chunk_arg, total;
};

inline int64_t num_chunks(int64_t V) { return (V + kChunk - 1) / kChunk; }

inline WorkspaceLayout workspace_layout(int32_t B, int64_t N, int64_t V, int32_t k_max) {
  const int64_t nc = num_chunks(V);
  const size_t n = size_t(N > 0 ? N : 1);
  const size_t slots = size_t(int64_t(B) * k_max > 0 ? int64_t(B) * k_max : 1);
  WorkspaceLayout L;
  size_t off = 0;
  L.work = off;
  off += align_up(sizeof(WorkItem) * n);
  L.pair_chunk = off;
  off += align_up(sizeof(PairChunk) * slots * size_t(nc));
  L.gathered = off;
  off += align_up(sizeof(Gathered) * slots);
  L.chunk_arg = off;
  off += align_up(sizeof(ChunkArg) * slots * size_t(nc));
  L.total = off;
  return L;
}

// Arguments of the signal update and the SL rule when they run fused behind
// the verification (dsde_step).
struct SignalArgs {
  float *hist;
  int32_t *head, *count;
  int32_t W, n_short, n_long;
  float delta, eps;
  float *mu_last, *var_short, *var_long, *wvir, *sf;
  const float *sl_max;
  float sl_min;
  int32_t sl_hi;
  const int32_t *budget;  // may be null
  float *sl_hat, *sl_cap;
  int32_t *sl_next;
};

struct VerifyArgs {
  const void *target, *draft;
  int32_t dtype;
  int64_t V;
  int32_t B;
  int64_t N;
  int32_t k_max;
  const int32_t *sl, *cu_sl, *draft_tokens;
  const float *temperature, *u_acc, *u_res;
  int32_t pad_id;
  int32_t *accepted, *tokens;
  float *kld;
  uint32_t *seq_err;
  double *row_lse;
  float *draft_entropy;
  void *workspace;
  hipStream_t stream;
  hipEvent_t prof_start, prof_stop;
  const SignalArgs *signal;  // non-null: fused signal update and SL rule
  // subtracted from each drafted token before its logits are gathered: the
  // first id of a vocabulary slice whose logits the rows hold, else 0
  int64_t token_base = 0;
};

int launch_verify(const VerifyArgs &a);
// The set-up and statistics kernels of one verification step (stats.hip).
// With `entropy` false the bf16 statistics kernel leaves the draft entropy
// accumulator (PairChunk::h) at zero.
void launch_stats_pass(const VerifyArgs &a, WorkItem *work, PairChunk *part, Gathered *gath, ChunkArg *chunk_arg,
                       bool entropy);
// Rows are 16-byte aligned and V a multiple of the vector width.
bool rows_vectorizable(const VerifyArgs &a);
int launch_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const float *kld,
                      float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                      float delta, float eps, float *mu_last, float *var_short, float *var_long, float *wvir,
                      float *sf, uint32_t *seq_err, hipStream_t stream);
int launch_calibration_update(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const int32_t *accepted,
                              const float *kld, const uint32_t *seq_err, int32_t *a_max, double *kld_sum,
                              int64_t *kld_count, float *kld_max, hipStream_t stream);
int launch_calibrate_sl_max(int32_t B, const int32_t *a_max, const double *kld_sum, const int64_t *kld_count,
                            const float *kld_max, float eps, bool pooled, float *sl_max, hipStream_t stream);
int launch_stream_read(const void *buf, int64_t bytes, uint32_t *out, hipStream_t stream);
int launch_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max, float sl_min,
                   int32_t sl_hi, const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next,
                   uint32_t *seq_err, bool or_err, hipStream_t stream);

}  // namespace dsde
