// libtreegraft C ABI: argument checks, workspace layout and kernel launches.
// Every call is asynchronous on the caller's stream and allocates nothing.
#include <hip/hip_runtime.h>

#include <initializer_list>
#include <mutex>

#include "../../include/treegraft.h"
#include "tg_kernels.h"

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace of the row-statistics pass: per (row, grain) (max, sum-exp)
// partials, per (row, chunk) top-K keys, then `extra` bytes for the caller.
// Workspace of a row pass: per grain (max, sum-exp) partials | per chunk
// top-K keys | finished top-K keys per row | the caller's extra bytes.
struct RowWs {
  size_t ms_off, keys_off, fin_off, extra_off, bytes;
};
RowWs row_ws(long long slots, int V, int K, size_t extra) {
  tg::RowPlan plan = tg::plan_rows(slots, V);
  size_t ms = (size_t)slots * plan.ms_per_row;
  size_t parts = (size_t)slots * plan.chunks;
  RowWs w;
  w.ms_off = 0;
  w.keys_off = align_up(ms * sizeof(float2), 256);
  w.fin_off = align_up(w.keys_off + parts * (size_t)K * sizeof(uint64_t), 256);
  w.extra_off = align_up(w.fin_off + (size_t)slots * K * sizeof(uint64_t), 256);
  w.bytes = align_up(w.extra_off + extra, 256);
  return w;
}

tg_status from_hip(hipError_t e) { return e == hipSuccess ? TG_OK : TG_ERR_HIP; }

bool tree_ok(const tg_tree *t) {
  return t && t->parent && t->token && t->depth && t->logp && t->cum &&
         t->visited && t->root_visited && t->n_nodes && t->cap > 0;
}

}  // namespace

extern "C" {

const char *tg_status_str(tg_status s) {
  switch (s) {
    case TG_OK: return "ok";
    case TG_ERR_INVALID_ARG: return "invalid argument";
    case TG_ERR_UNSUPPORTED: return "unsupported shape or option";
    case TG_ERR_WORKSPACE: return "workspace missing or too small";
    case TG_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

tg_status tg_tree_reset(const tg_tree *tree, int B, void *stream) {
  if (!tree_ok(tree) || B <= 0) return TG_ERR_INVALID_ARG;
  return from_hip(tg::launch_tree_reset(*tree, B, reinterpret_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------------ verify attention
size_t tg_verify_attention_workspace(int B, int N, int Hq, int Hkv, int D,
                                     int S_max, tg_dtype dtype) {
  if (B <= 0 || N <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || S_max < N) return 0;
  tg::AttnShape s{B, N, Hq, Hkv, D, S_max, 1.0f};
  return tg::attn_workspace_bytes(s, dtype);
}

}  // extern "C"

// Scratch memory of tg_tree_verify_attention_noalloc, held by every device
// the library runs on until the process ends.  In host code this name is
// only a stand-in for the symbol: the device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static __device__ __align__(256) unsigned char scratch[TG_NOALLOC_SCRATCH_BYTES];

namespace {

tg_status verify_attention_args(const void *q, const void *k_cache, const void *v_cache,
                                const int32_t *parent, const int32_t *prefix_len, void *out,
                                int B, int N, int Hq, int Hkv, int D, int S_max, float sm_scale,
                                tg_dtype dtype) {
  if (!q || !k_cache || !v_cache || !parent || !prefix_len || !out)
    return TG_ERR_INVALID_ARG;
  // the kernels move q, the caches and out in 16-byte vectors
  for (const void *p : {q, k_cache, v_cache, static_cast<const void *>(out)})
    if (reinterpret_cast<uintptr_t>(p) & 15) return TG_ERR_INVALID_ARG;
  if (B <= 0 || N <= 0 || Hq <= 0 || Hkv <= 0 || S_max < N) return TG_ERR_INVALID_ARG;
  if (Hq % Hkv) return TG_ERR_INVALID_ARG;
  // a finite, non-negative softmax scale (the kernels take each row's
  // maximum of the unscaled scores as the maximum of the scaled ones)
  if (!(sm_scale >= 0.0f) || sm_scale == __builtin_inff()) return TG_ERR_INVALID_ARG;
  if (D != 64 && D != 128) return TG_ERR_UNSUPPORTED;
  if (N > TG_MAX_VERIFY_NODES) return TG_ERR_UNSUPPORTED;
  if (dtype != TG_F32 && dtype != TG_BF16) return TG_ERR_INVALID_ARG;
  return TG_OK;
}

// Launches after the argument checks; `workspace` holds at least the bytes
// attn_workspace_bytes() asks for.
tg_status verify_attention_launch(const void *q, const void *k_cache, const void *v_cache,
                                  const int32_t *parent, const int32_t *prefix_len, void *out,
                                  const tg::AttnShape &s, tg_dtype dtype, void *workspace,
                                  uint32_t *d_err, hipStream_t st) {
  if (dtype == TG_F32)
    return from_hip(tg::launch_attn_f32(
        s, static_cast<const float *>(q), static_cast<const float *>(k_cache),
        static_cast<const float *>(v_cache), parent, prefix_len,
        static_cast<float *>(out), d_err, st));
  return from_hip(tg::launch_attn_bf16(s, q, k_cache, v_cache, parent, prefix_len,
                                       out, workspace, d_err, st));
}

constexpr int kMaxDevices = 64;
void *g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

// The current device's address of `scratch` (looked up on its first call on
// that device, with that device current).
tg_status scratch_addr(void **addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return TG_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return TG_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TG_ERR_HIP;
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return TG_OK;
}

}  // namespace

extern "C" {

tg_status tg_tree_verify_attention(const void *q, const void *k_cache,
                                   const void *v_cache, const int32_t *parent,
                                   const int32_t *prefix_len, void *out, int B,
                                   int N, int Hq, int Hkv, int D, int S_max,
                                   float sm_scale, tg_dtype dtype,
                                   void *workspace, size_t ws_bytes,
                                   uint32_t *d_err, void *stream) {
  const tg_status a = verify_attention_args(q, k_cache, v_cache, parent, prefix_len, out, B, N,
                                            Hq, Hkv, D, S_max, sm_scale, dtype);
  if (a != TG_OK) return a;
  tg::AttnShape s{B, N, Hq, Hkv, D, S_max, sm_scale};
  const size_t need = tg::attn_workspace_bytes(s, dtype);
  if (need && (!workspace || ws_bytes < need)) return TG_ERR_WORKSPACE;
  return verify_attention_launch(q, k_cache, v_cache, parent, prefix_len, out, s, dtype,
                                 workspace, d_err, reinterpret_cast<hipStream_t>(stream));
}

tg_status tg_tree_verify_attention_noalloc(const void *q, const void *k_cache,
                                           const void *v_cache, const int32_t *parent,
                                           const int32_t *prefix_len, void *out, int B, int N,
                                           int Hq, int Hkv, int D, int S_max, float sm_scale,
                                           tg_dtype dtype, uint32_t *d_err, void *stream) {
  const tg_status a = verify_attention_args(q, k_cache, v_cache, parent, prefix_len, out, B, N,
                                            Hq, Hkv, D, S_max, sm_scale, dtype);
  if (a != TG_OK) return a;
  tg::AttnShape s{B, N, Hq, Hkv, D, S_max, sm_scale};
  const size_t need = tg::attn_workspace_bytes(s, dtype);
  if (need > TG_NOALLOC_SCRATCH_BYTES) return TG_ERR_WORKSPACE;
  void *ws = nullptr;
  if (need) {
    const tg_status r = scratch_addr(&ws);
    if (r != TG_OK) return r;
  }
  return verify_attention_launch(q, k_cache, v_cache, parent, prefix_len, out, s, dtype, ws,
                                 d_err, reinterpret_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------------- expand
size_t tg_expand_topk_workspace(int B, int F, int V, int K, int N) {
  if (B <= 0 || F <= 0 || V <= 0 || K <= 0 || N <= 0) return 0;
  return row_ws((long long)B * F, V, K, 0).bytes;
}

tg_status tg_tree_expand_topk(const tg_tree *tree, const float *logits,
                              const int32_t *frontier,
                              const int32_t *n_frontier, int B, int F, int V,
                              int K, int N, float *row_lse,
                              int32_t *next_frontier, int32_t *n_next,
                              void *workspace, size_t ws_bytes,
                              uint32_t *d_err, void *stream) {
  if (!tree_ok(tree) || !logits || !frontier || !row_lse || !next_frontier || !n_next)
    return TG_ERR_INVALID_ARG;
  if (B <= 0 || F <= 0 || V <= 0 || K <= 0 || N <= 0) return TG_ERR_INVALID_ARG;
  if (K > V) return TG_ERR_INVALID_ARG;
  if (K > TG_MAX_TOPK || (long long)F * K > TG_MAX_EXPAND_CHILDREN ||
      tree->cap > TG_MAX_CAP)
    return TG_ERR_UNSUPPORTED;
  RowWs w = row_ws((long long)B * F, V, K, 0);
  if (!workspace || ws_bytes < w.bytes) return TG_ERR_WORKSPACE;
  tg::RowPlan plan = tg::plan_rows((long long)B * F, V);
  char *ws = static_cast<char *>(workspace);
  float2 *ms = reinterpret_cast<float2 *>(ws + w.ms_off);
  uint64_t *keys = reinterpret_cast<uint64_t *>(ws + w.keys_off);
  uint64_t *fin = reinterpret_cast<uint64_t *>(ws + w.fin_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = tg::launch_row_partials(logits, B, F, V, K, plan, n_frontier, nullptr, ms,
                                         keys, d_err, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  e = tg::launch_row_finish(B, F, K, plan, n_frontier, nullptr, ms, keys, row_lse, fin, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  return from_hip(tg::launch_expand_tree(*tree, frontier, n_frontier, B, F, K, N, row_lse,
                                         fin, next_frontier, n_next, d_err, st));
}

// ------------------------------------------------------------ rescore + graft
size_t tg_rescore_graft_workspace(int B, int R, int V, int W, int M, int cap) {
  (void)W;
  (void)cap;
  if (B <= 0 || R <= 0 || V <= 0 || M <= 0) return 0;
  return row_ws((long long)B * R, V, M, (size_t)B * R).bytes;
}

tg_status tg_tree_rescore_graft(const tg_tree *tree, const float *strong_logits,
                                int B, int R, int V, int W, int M,
                                uint32_t flags, const int32_t *new_from, float *row_lse,
                                int32_t *graft_frontier, int32_t *n_graft,
                                int32_t *next_frontier, int32_t *n_next, int N,
                                void *workspace, size_t ws_bytes,
                                uint32_t *d_err, void *stream) {
  if (!tree_ok(tree) || !strong_logits || !row_lse || !graft_frontier || !n_graft)
    return TG_ERR_INVALID_ARG;
  if ((next_frontier == nullptr) != (n_next == nullptr)) return TG_ERR_INVALID_ARG;
  if (next_frontier && N <= 0) return TG_ERR_INVALID_ARG;
  if (B <= 0 || R <= 0 || V <= 0 || W <= 0 || M <= 0) return TG_ERR_INVALID_ARG;
  if (M > V) return TG_ERR_INVALID_ARG;
  if (flags & ~(TG_POOL_NEWONLY | TG_GRAFT_OVERWRITE | TG_GRAFT_DEDUP))
    return TG_ERR_UNSUPPORTED;
  if ((flags & TG_POOL_NEWONLY) && !new_from) return TG_ERR_INVALID_ARG;
  if (M > TG_MAX_TOPK || tree->cap > TG_MAX_CAP)
    return TG_ERR_UNSUPPORTED;
  RowWs w = row_ws((long long)B * R, V, M, (size_t)B * R);
  if (!workspace || ws_bytes < w.bytes) return TG_ERR_WORKSPACE;
  tg::RowPlan plan = tg::plan_rows((long long)B * R, V);
  {
    int vo = 0;
    if (tg::rescore_tree_lds(tree->cap, flags, &vo) > 160 * 1024) return TG_ERR_UNSUPPORTED;
  }
  char *ws = static_cast<char *>(workspace);
  float2 *ms = reinterpret_cast<float2 *>(ws + w.ms_off);
  uint64_t *keys = reinterpret_cast<uint64_t *>(ws + w.keys_off);
  uint64_t *fin = reinterpret_cast<uint64_t *>(ws + w.fin_off);
  uint8_t *needed = reinterpret_cast<uint8_t *>(ws + w.extra_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = tg::launch_rescore_pool(*tree, B, R, needed, flags, new_from, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  e = tg::launch_row_partials(strong_logits, B, R, V, M, plan, nullptr, needed, ms, keys,
                              d_err, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  e = tg::launch_row_finish(B, R, M, plan, nullptr, needed, ms, keys, row_lse, fin, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  return from_hip(tg::launch_rescore_tree(*tree, strong_logits, B, R, V, W, M, row_lse, fin,
                                          graft_frontier, n_graft,
                                          next_frontier, n_next, next_frontier ? N : 0,
                                          flags, new_from, d_err, st));
}

// ------------------------------------------------------------ n-gram drafter
size_t tg_ngram_cache_workspace(int B, int L, int V, int m) {
  if (B <= 0 || L <= 0 || V <= 0 || m <= 0) return 0;
  return row_ws((long long)B * L, V, m, (size_t)B * V * sizeof(int32_t)).bytes;
}

tg_status tg_ngram_cache(const float *logits, const int32_t *context, const int32_t *ctx_len,
                         int B, int L, int V, int m, int32_t *cand_tok, float *cand_logp,
                         int32_t *fallback_pos, void *workspace, size_t ws_bytes,
                         uint32_t *d_err, void *stream) {
  if (!logits || !context || !ctx_len || !cand_tok || !cand_logp || !fallback_pos)
    return TG_ERR_INVALID_ARG;
  if (B <= 0 || L <= 0 || V <= 0 || m <= 0 || m > V) return TG_ERR_INVALID_ARG;
  if (m > TG_MAX_TOPK) return TG_ERR_UNSUPPORTED;
  RowWs w = row_ws((long long)B * L, V, m, (size_t)B * V * sizeof(int32_t));
  if (!workspace || ws_bytes < w.bytes) return TG_ERR_WORKSPACE;
  tg::RowPlan plan = tg::plan_rows((long long)B * L, V);
  char *ws = static_cast<char *>(workspace);
  float2 *ms = reinterpret_cast<float2 *>(ws + w.ms_off);
  uint64_t *keys = reinterpret_cast<uint64_t *>(ws + w.keys_off);
  int32_t *counts = reinterpret_cast<int32_t *>(ws + w.extra_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = tg::launch_row_partials(logits, B, L, V, m, plan, nullptr, nullptr, ms, keys,
                                         d_err, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  e = tg::launch_ngram_cache((long long)B * L, m, plan, ms, keys, cand_tok, cand_logp, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  return from_hip(
      tg::launch_ngram_fallback(context, ctx_len, B, L, V, counts, fallback_pos, d_err, st));
}

tg_status tg_tree_expand_ngram(const tg_tree *tree, const int32_t *frontier,
                               const int32_t *n_frontier, const int32_t *context,
                               const int32_t *ctx_len, const int32_t *cand_tok,
                               const float *cand_logp, const int32_t *fallback_pos, int B,
                               int F, int L, int m, int K, int N, int n_max,
                               int32_t *match_pos, int32_t *next_frontier, int32_t *n_next,
                               uint32_t *d_err, void *stream) {
  if (!tree_ok(tree) || !frontier || !context || !ctx_len || !cand_tok || !cand_logp ||
      !fallback_pos || !next_frontier || !n_next)
    return TG_ERR_INVALID_ARG;
  if (B <= 0 || F <= 0 || L <= 0 || m <= 0 || K <= 0 || K > m || N <= 0 || n_max <= 0)
    return TG_ERR_INVALID_ARG;
  if (n_max > TG_MAX_NGRAM || F > TG_MAX_NGRAM_FRONTIER ||
      (long long)F * K > TG_MAX_EXPAND_CHILDREN || tree->cap > TG_MAX_CAP)
    return TG_ERR_UNSUPPORTED;
  return from_hip(tg::launch_ngram_expand(*tree, frontier, n_frontier, B, F, context, ctx_len,
                                          L, cand_tok, cand_logp, fallback_pos, m, K, N, n_max,
                                          match_pos, next_frontier, n_next, d_err,
                                          reinterpret_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------------------- accept
tg_status tg_tree_accept(const int32_t *parent, const int32_t *token,
                         const int32_t *n_nodes, const int32_t *greedy, int B,
                         int cap, int max_depth, int32_t *accept_len,
                         int32_t *accept_path, int32_t *bonus, uint32_t *d_err,
                         void *stream) {
  if (!parent || !token || !n_nodes || !greedy || !accept_len || !bonus)
    return TG_ERR_INVALID_ARG;
  if (B <= 0 || cap <= 0 || max_depth < 0) return TG_ERR_INVALID_ARG;
  if (max_depth > 0 && !accept_path) return TG_ERR_INVALID_ARG;
  if (cap > TG_MAX_CAP) return TG_ERR_UNSUPPORTED;
  return from_hip(tg::launch_accept(parent, token, n_nodes, greedy, B, cap, max_depth,
                                    accept_len, accept_path, bonus, d_err,
                                    reinterpret_cast<hipStream_t>(stream)));
}

tg_status tg_tree_accept_logits(const int32_t *parent, const int32_t *token,
                                const int32_t *n_nodes, const float *logits, int B, int cap,
                                int R, int V, int max_depth, int32_t *greedy,
                                int32_t *accept_len, int32_t *accept_path, int32_t *bonus,
                                uint32_t *d_err, void *stream) {
  if (!logits || !greedy) return TG_ERR_INVALID_ARG;
  if (R <= 0 || V <= 0) return TG_ERR_INVALID_ARG;
  if (!parent || !token || !n_nodes || !accept_len || !bonus) return TG_ERR_INVALID_ARG;
  if (B <= 0 || cap <= 0 || max_depth < 0) return TG_ERR_INVALID_ARG;
  if (max_depth > 0 && !accept_path) return TG_ERR_INVALID_ARG;
  if (cap > TG_MAX_CAP) return TG_ERR_UNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = tg::launch_argmax_rows(logits, n_nodes, B, cap, R, V, greedy, d_err, st);
  if (e != hipSuccess) return TG_ERR_HIP;
  return from_hip(tg::launch_accept(parent, token, n_nodes, greedy, B, cap, max_depth,
                                    accept_len, accept_path, bonus, d_err, st));
}

tg_status tg_tree_global_prune(const tg_tree *tree, int B, int B_ver, int max_path,
                               int32_t *kept, int32_t *vparent, int32_t *vtoken,
                               int32_t *position_ids, uint32_t *mask, int32_t *retrieval,
                               int32_t *n_keep, int32_t *n_leaves, uint32_t *d_err,
                               void *stream) {
  if (!tree_ok(tree) || !kept || !vparent || !vtoken || !position_ids || !mask ||
      !retrieval || !n_keep || !n_leaves)
    return TG_ERR_INVALID_ARG;
  if (B <= 0 || B_ver < 1 || max_path < 1) return TG_ERR_INVALID_ARG;
  if (B_ver > TG_MAX_CAP || tree->cap > TG_MAX_CAP) return TG_ERR_UNSUPPORTED;
  return from_hip(tg::launch_global_prune(*tree, B, B_ver, max_path, kept, vparent, vtoken,
                                          position_ids, mask, retrieval, n_keep, n_leaves,
                                          d_err, reinterpret_cast<hipStream_t>(stream)));
}

tg_status tg_kv_compact(void *k_cache, void *v_cache, const int32_t *prefix_len,
                        const int32_t *path, const int32_t *n_path, int B, int Hkv, int S_max,
                        int D, int max_path, tg_dtype dtype, int32_t *new_prefix_len,
                        uint32_t *d_err, void *stream) {
  if (!k_cache || !v_cache || !prefix_len || !n_path || !new_prefix_len)
    return TG_ERR_INVALID_ARG;
  if ((const void *)new_prefix_len == (const void *)prefix_len) return TG_ERR_INVALID_ARG;
  if (B <= 0 || Hkv <= 0 || S_max <= 0 || max_path < 0) return TG_ERR_INVALID_ARG;
  if (max_path > 0 && !path) return TG_ERR_INVALID_ARG;
  if (dtype != TG_F32 && dtype != TG_BF16) return TG_ERR_INVALID_ARG;
  if (D != 64 && D != 128) return TG_ERR_UNSUPPORTED;
  return from_hip(tg::launch_kv_compact(k_cache, v_cache, prefix_len, path, n_path, B, Hkv,
                                        S_max, D, max_path, dtype, new_prefix_len, d_err,
                                        reinterpret_cast<hipStream_t>(stream)));
}

tg_status tg_tree_signals(const tg_tree *tree, const int32_t *frontier, const int32_t *n_frontier,
                          int B, int F, int W, int lookback, const float *context,
                          const float *params, float *signals, float *margin, int32_t *action,
                          uint32_t *d_err, void *stream) {
  if (!tree_ok(tree) || !frontier || !signals) return TG_ERR_INVALID_ARG;
  if (B <= 0 || F < 1 || W < 1 || lookback < 0) return TG_ERR_INVALID_ARG;
  if (params && (!context || !margin || !action)) return TG_ERR_INVALID_ARG;
  if (tree->cap > TG_MAX_CAP) return TG_ERR_UNSUPPORTED;
  return from_hip(tg::launch_signals(*tree, frontier, n_frontier, B, F, W, lookback, context,
                                     params, signals, margin, action, d_err,
                                     reinterpret_cast<hipStream_t>(stream)));
}

}  // extern "C"
