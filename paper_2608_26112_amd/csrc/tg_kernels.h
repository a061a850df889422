// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/treegraft.h"


namespace tg {

// ------------------------------------------------------------ launching
// Takes a start/stop event pair when tracing is on (trace.hip).
bool trace_slot(const char *name, hipEvent_t *start, hipEvent_t *stop);

// Callers check hipGetLastError() afterwards.
template <typename F, typename... Args>
void launch(const char *name, F kernel, dim3 grid, dim3 block, size_t shmem,
            hipStream_t stream, Args... args) {
  hipEvent_t a, b;
  const bool traced = trace_slot(name, &a, &b);
  if (traced) (void)hipEventRecord(a, stream);
  hipLaunchKernelGGL(kernel, grid, block, shmem, stream, args...);
  if (traced) (void)hipEventRecord(b, stream);
}

// ------------------------------------------------------------ logits rows
// A logits row is cut into grains of kGrain elements; every grain yields one
// (max, sum-exp) partial per wave of the row pass over a fixed element set,
// so a row's log-sum-exp does not depend on the call's chunking.  A
// workgroup handles `grains_per_chunk` consecutive grains (one chunk) and
// emits the chunk's top-K; `chunks` chunks cover a row.
constexpr int kGrain = 8192;
struct RowPlan {
  int chunks;
  int grains_per_chunk;
  int ms_per_row;  // (max, sum-exp) partials per row (one per grain)
};
RowPlan plan_rows(long long rows, int V);

// Row partials of every live row slot s = b * rows_per_batch + r of a
// [*, rows_per_batch, V] logits array: live iff r < n_live[b] (n_live may be
// NULL = all) when `needed` is NULL, else iff needed[s] != 0.  Writes per
// grain (max, sum-exp) and per chunk top-K keys; the tree kernels finish rows.
hipError_t launch_row_partials(const float *logits, int B, int rows_per_batch,
                               int V, int K, RowPlan plan,
                               const int32_t *n_live, const uint8_t *needed,
                               float2 *part_ms, uint64_t *part_keys,
                               uint32_t *d_err, hipStream_t stream);

// Finishes the same live rows: lse[s] (a fixed fold of the grain partials) and the row's top-K keys
// out_keys[s * K + j], best first (one wave per row over the whole chip).
hipError_t launch_row_finish(int B, int rows_per_batch, int K, RowPlan plan,
                             const int32_t *n_live, const uint8_t *needed,
                             const float2 *part_ms, const uint64_t *part_keys, float *lse,
                             uint64_t *out_keys, hipStream_t stream);

// The tree kernels read finished rows: row_lse [B, rows] and row_keys
// [B, rows, K] as written by launch_row_finish.
hipError_t launch_expand_tree(const tg_tree &tree, const int32_t *frontier,
                              const int32_t *n_frontier, int B, int F, int K,
                              int N, const float *row_lse, const uint64_t *row_keys,
                              int32_t *next_frontier, int32_t *n_next,
                              uint32_t *d_err, hipStream_t stream);

hipError_t launch_tree_reset(const tg_tree &tree, int B, hipStream_t stream);

hipError_t launch_rescore_pool(const tg_tree &tree, int B, int R, uint8_t *needed,
                               uint32_t flags, const int32_t *new_from,
                               hipStream_t stream);
// dynamic LDS of rescore_tree_kernel (and the offset of its variant region)
size_t rescore_tree_lds(int cap, uint32_t flags, int *var_off);

hipError_t launch_rescore_tree(const tg_tree &tree, const float *strong, int B,
                               int R, int V, int W, int M, const float *row_lse,
                               const uint64_t *row_keys,
                               int32_t *graft_frontier, int32_t *n_graft,
                               int32_t *next_frontier, int32_t *n_next, int N,
                               uint32_t flags, const int32_t *new_from,
                               uint32_t *d_err, hipStream_t stream);

// ----------------------------------------------------------------- accept
// n-gram small drafter
hipError_t launch_ngram_cache(long long rows, int m, RowPlan plan, const float2 *part_ms,
                              const uint64_t *part_keys, int32_t *cand_tok, float *cand_logp,
                              hipStream_t stream);
hipError_t launch_ngram_fallback(const int32_t *context, const int32_t *ctx_len, int B, int L,
                                 int V, int32_t *counts, int32_t *fallback_pos, uint32_t *d_err,
                                 hipStream_t stream);
hipError_t launch_ngram_expand(const tg_tree &tree, const int32_t *frontier,
                               const int32_t *n_frontier, int B, int F,
                               const int32_t *context, const int32_t *ctx_len, int L,
                               const int32_t *cand_tok, const float *cand_logp,
                               const int32_t *fallback_pos, int m, int K, int N, int n_max,
                               int32_t *match_pos, int32_t *next_frontier, int32_t *n_next,
                               uint32_t *d_err, hipStream_t stream);
hipError_t launch_argmax_rows(const float *logits, const int32_t *n_nodes, int B, int cap,
                              int R, int V, int32_t *greedy, uint32_t *d_err,
                              hipStream_t stream);
hipError_t launch_accept(const int32_t *parent, const int32_t *token,
                         const int32_t *n_nodes, const int32_t *greedy, int B,
                         int cap, int max_depth, int32_t *accept_len,
                         int32_t *accept_path, int32_t *bonus, uint32_t *d_err,
                         hipStream_t stream);

// ------------------------------------------------------- prune / cache
hipError_t launch_global_prune(const tg_tree &tree, int B, int B_ver, int max_path,
                               int32_t *kept, int32_t *vparent, int32_t *vtoken,
                               int32_t *position_ids, uint32_t *mask, int32_t *retrieval,
                               int32_t *n_keep, int32_t *n_leaves, uint32_t *d_err,
                               hipStream_t stream);
hipError_t launch_kv_compact(void *k_cache, void *v_cache, const int32_t *prefix_len,
                             const int32_t *path, const int32_t *n_path, int B, int Hkv,
                             int S_max, int D, int max_path, tg_dtype dtype,
                             int32_t *new_prefix_len, uint32_t *d_err, hipStream_t stream);

// ------------------------------------------------------------- scheduler
hipError_t launch_signals(const tg_tree &tree, const int32_t *frontier, const int32_t *n_frontier,
                          int B, int F, int W, int lookback, const float *context,
                          const float *params, float *signals, float *margin, int32_t *action,
                          uint32_t *d_err, hipStream_t stream);

// -------------------------------------------------------------- attention
struct AttnShape {
  int B, N, Hq, Hkv, D, S_max;
  float sm_scale;
};
// Number of prefix splits the bf16 kernel uses for this shape (1 = none).
int attn_splits(const AttnShape &s);
size_t attn_workspace_bytes(const AttnShape &s, tg_dtype dtype);

hipError_t launch_attn_f32(const AttnShape &s, const float *q, const float *k,
                           const float *v, const int32_t *parent,
                           const int32_t *prefix_len, float *out,
                           uint32_t *d_err, hipStream_t stream);

hipError_t launch_attn_bf16(const AttnShape &s, const void *q, const void *k,
                            const void *v, const int32_t *parent,
                            const int32_t *prefix_len, void *out,
                            void *workspace, uint32_t *d_err,
                            hipStream_t stream);

}  // namespace tg
