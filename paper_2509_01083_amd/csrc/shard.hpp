// Host side of the vocabulary-shard calls: workspace layout and launchers
// (shard.hip).
#pragma once

#include "common.hpp"

namespace dsde {

// One shard's workspace: the statistics pass's buffers for the slice width,
// then the draw's chunk totals of every sequence (call 3 writes them, call 4
// reads them).
struct ShardLayout {
  WorkspaceLayout stats;
  size_t ch_w, ch_ref, ch_bad, sub, total;
};

inline ShardLayout shard_layout(int32_t B, int64_t N, int64_t V_shard, int32_t k_max) {
  ShardLayout L;
  L.stats = workspace_layout(B, N, V_shard, k_max);
  const size_t cells = size_t(B) * size_t(num_chunks(V_shard));
  size_t off = L.stats.total;
  L.ch_w = off;
  off += align_up(sizeof(double) * cells);
  L.ch_ref = off;
  off += align_up(sizeof(float) * cells);
  L.ch_bad = off;
  off += align_up(sizeof(int32_t) * cells);
  L.sub = off;
  off += align_up(sizeof(float) * 64 * cells);
  L.total = off;
  return L;
}

struct ShardRows {
  const void *target, *draft;
  int32_t dtype;
  int64_t V_shard, v_begin;
  int32_t B;
  int64_t N;
  int32_t k_max;
  void *workspace;
  hipStream_t stream;
};

int launch_shard_stats(const ShardRows &r, int64_t V, const int32_t *sl, const int32_t *cu_sl,
                       const int32_t *draft_tokens, const float *temperature, dsde_shard_partial *part,
                       uint32_t *seq_err);
int launch_shard_accept(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N, int32_t k_max,
                        const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                        const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                        int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                        dsde_draw_job *jobs, uint32_t *seq_err, const SignalArgs *signal, hipStream_t stream);
int launch_shard_draw_mass(const ShardRows &r, const dsde_shard_partial *part, const dsde_draw_job *jobs,
                           dsde_shard_mass *mass);
int launch_shard_draw_pick(const ShardRows &r, int32_t G, int32_t g, const dsde_shard_mass *masses,
                           const dsde_draw_job *jobs, int32_t pad_id, int32_t *accepted, int32_t *tokens,
                           int32_t *drawn, uint32_t *seq_err);

}  // namespace dsde
