// Per-tree phases of the expansion step (Sec. 3.1; Alg. 1) and of the
// middle-drafter step (Sec. 3.2; Alg. 2, middle branch).
//
// One workgroup owns one tree.  The vocabulary-wide work already happened in
// row_partial_kernel; here the chunk partials of each needed row are merged
// into its log-sum-exp and top-K list, then the tree is edited in place:
// children appended (expand), pool rescored, graft positions reselected and
// new children grafted without touching existing nodes (rescore_graft).
// Node selection (Top_W) ranks 64-bit keys in LDS ordered by (cum desc,
// depth asc, id asc): by counting the larger keys, or a bitonic sort past
// 1024 keys.
#include <algorithm>

#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

// ------------------------------------------------------- finishing rows
// log-sum-exp of one row from its per-grain (max, sum-exp) partials, folded
// in grain order (the same bits whatever the call's chunking).
__device__ float finish_lse(const float2 *__restrict__ ms, int n) {
  float m = -__builtin_inff(), s = 0.0f;
#pragma unroll 8
  for (int i = 0; i < n; ++i) {
    const float2 p = ms[i];
    merge_ms(m, s, p.x, p.y);
  }
  return m == -__builtin_inff() ? -__builtin_inff() : m + logf(s);
}

// K-round merge of one row's `chunks` sorted lists (each K keys, best
// first) staged in LDS at `lists`: lane c holds list c's head, the wave takes
// the largest head, that list advances.  Lane j < K returns the j-th best key.
__device__ uint64_t wave_merge_lists(const uint64_t *lists, int chunks, int K) {
  const int lane = threadIdx.x & (kWave - 1);
  int idx = 0;
  uint64_t head = lane < chunks ? lists[lane * K] : 0;
  uint64_t mine = 0;
  for (int j = 0; j < K; ++j) {
    const uint64_t best = wave_max_u64(head);
    if (head == best && best != 0) {
      ++idx;
      head = idx < K ? lists[lane * K + idx] : 0;
    }
    if (lane == j) mine = best;
  }
  return mine;
}

// Top-K of nr consecutive rows (row r's `chunks` lists of K keys at
// lists + r * chunks * K) into out[r * K + j], best first.  The lists are
// staged in LDS (`stage`, room for stage_cap >= chunks * K keys) with one
// global round trip per batch, then a wave merges each row.  chunks <= 64.
// Called by the whole block; ends synchronised.
__device__ void block_finish_topk(const uint64_t *__restrict__ lists, int chunks, int K,
                                  int nr, uint64_t *out, uint64_t *stage, int stage_cap) {
  const int nk = chunks * K;
  if (chunks == 1) {
    for (int i = threadIdx.x; i < nr * K; i += blockDim.x) out[i] = lists[i];
    __syncthreads();
    return;
  }
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int per = stage_cap / nk;
  for (int r0 = 0; r0 < nr; r0 += per) {
    const int rb = min(per, nr - r0);
    for (int i = threadIdx.x; i < rb * nk; i += blockDim.x) stage[i] = lists[(size_t)r0 * nk + i];
    __syncthreads();
    for (int r = w; r < rb; r += kWaves) {
      const uint64_t key = wave_merge_lists(stage + r * nk, chunks, K);
      if (lane < K) out[(r0 + r) * K + lane] = key;
    }
    __syncthreads();
  }
}

// One wave finishes one row's top-K: lane j < K returns the j-th best key.
// `ws` is this wave's LDS scratch (chunks * K keys).  chunks <= 64.
__device__ uint64_t wave_finish_topk(const uint64_t *__restrict__ lists, int chunks, int K,
                                     uint64_t *ws) {
  const int lane = threadIdx.x & (kWave - 1);
  if (chunks == 1) return lane < K ? lists[lane] : 0;
  const int nk = chunks * K;
  for (int i = lane; i < nk; i += kWave) ws[i] = lists[i];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint64_t r = wave_merge_lists(ws, chunks, K);
  __builtin_amdgcn_wave_barrier();   // ws is reused by the wave's next row
  return r;
}

__device__ __forceinline__ int sane_parent(int p, int v, bool &bad) {
  bool b = p < -1 || p >= v;
  bad |= b;
  return b ? -1 : p;
}

// --------------------------------------------------------------- expand
__global__ __launch_bounds__(kThreads) void expand_tree_kernel(
    tg_tree tree, const int32_t *__restrict__ frontier,
    const int32_t *__restrict__ n_frontier, int F, int K, int N, int chunks,
    int n_ms, const float2 *__restrict__ part_ms, const uint64_t *__restrict__ part_keys,
    float *__restrict__ row_lse, int32_t *__restrict__ next_frontier,
    int32_t *__restrict__ n_next, uint32_t *d_err, int skey_cap) {
  extern __shared__ uint64_t smem[];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int cap = tree.cap;
  int Fb = n_frontier ? n_frontier[b] : F;
  Fb = Fb < 0 ? 0 : (Fb > F ? F : Fb);
  const int nb = tree.n_nodes[b];
  const int total = Fb * K;
  const int P2 = pow2_at_least(total > 0 ? total : 1);
  uint64_t *topk = smem;                       // [F*K]
  uint64_t *skey = smem + (size_t)F * K;       // [skey_cap >= max(P2, chunks*K)]
  float *lse_s = reinterpret_cast<float *>(skey + skey_cap);  // [F]

  bool bad = nb < 0 || nb > cap;
  for (int f = tid; f < Fb; f += kThreads) {
    int v = frontier[(size_t)b * F + f];
    bad |= v < -1 || v >= nb;
  }
  bad = __syncthreads_or(bad);

  // finish the live rows: lse (a thread per row) and top-K (skey as stage)
  for (int f = tid; f < Fb; f += kThreads) {
    const size_t slot = (size_t)b * F + f;
    const float lse = finish_lse(part_ms + slot * n_ms, n_ms);
    lse_s[f] = lse;
    row_lse[slot] = lse;
  }
  block_finish_topk(part_keys + (size_t)b * F * chunks * K, chunks, K, Fb, topk, skey,
                    skey_cap);

  const bool full = !bad && (nb + total > cap);
  if (bad || full) {
    if (tid == 0) {
      report(d_err, bad ? TG_DERR_BAD_NODE : TG_DERR_CAPACITY);
      n_next[b] = 0;
    }
    for (int j = tid; j < N; j += kThreads) next_frontier[(size_t)b * N + j] = TG_NO_NODE;
    return;
  }

  const size_t base = (size_t)b * cap;
  for (int c = tid; c < P2; c += kThreads) {
    if (c >= total) {
      skey[c] = 0;
      continue;
    }
    const int f = c / K;
    const uint64_t key = topk[c];
    const int v = frontier[(size_t)b * F + f];
    const float cv = v < 0 ? 0.0f : tree.cum[base + v];
    const int dv = v < 0 ? 0 : tree.depth[base + v];
    const float lp = edge_logp(key_logit(key), lse_s[f]);
    const float cum = __fadd_rn(cv, lp);
    const int id = nb + c;
    tree.parent[base + id] = v;
    tree.token[base + id] = (int)key_token(key);
    tree.depth[base + id] = dv + 1;
    tree.logp[base + id] = lp;
    tree.cum[base + id] = cum;
    tree.visited[base + id] = 0;
    skey[c] = node_key(cum, dv + 1, id);
  }
  __syncthreads();
  const int nn = min(N, total);
  block_top_keys<kThreads>(skey, total, P2, nn);
  for (int j = tid; j < N; j += kThreads)
    next_frontier[(size_t)b * N + j] = j < nn ? node_key_id(skey[j]) : TG_NO_NODE;
  if (tid == 0) {
    n_next[b] = nn;
    tree.n_nodes[b] = nb + total;
  }
}

// ------------------------------------------------------- middle-step pool
// needed[b, r] = 1 iff logits row r is read by this middle step: the row of
// each pool node (its children) and the row of each pool node's parent (its
// edge score).  Rows of trees that cannot be processed are all 0.
__global__ __launch_bounds__(kThreads) void rescore_pool_kernel(
    tg_tree tree, int R, uint8_t *__restrict__ needed) {
  __shared__ uint8_t flag[TG_MAX_CAP + 1];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int nb = tree.n_nodes[b];
  const bool ok = nb >= 0 && nb <= tree.cap && nb + 1 <= R;
  const int rows = ok ? nb + 1 : 0;
  for (int r = tid; r < rows; r += kThreads) flag[r] = 0;
  __syncthreads();
  const size_t base = (size_t)b * tree.cap;
  if (ok) {
    if (tid == 0 && !tree.root_visited[b]) flag[0] = 1;
    bool dummy = false;
    for (int v = tid; v < nb; v += kThreads) {
      if (!tree.visited[base + v]) {
        flag[v + 1] = 1;
        flag[sane_parent(tree.parent[base + v], v, dummy) + 1] = 1;
      }
    }
  }
  __syncthreads();
  for (int r = tid; r < R; r += kThreads)
    needed[(size_t)b * R + r] = r < rows ? flag[r] : 0;
}

// ------------------------------------------------ rescore + reselect + graft
__global__ __launch_bounds__(kThreads) void rescore_tree_kernel(
    tg_tree tree, const float *__restrict__ strong, int R, int V, int W, int M,
    int chunks, int n_ms, const uint8_t *__restrict__ needed,
    const float2 *__restrict__ part_ms, const uint64_t *__restrict__ part_keys,
    float *__restrict__ row_lse, int32_t *__restrict__ graft_frontier,
    int32_t *__restrict__ n_graft, int32_t *__restrict__ next_frontier,
    int32_t *__restrict__ n_next, int N, uint32_t *d_err, int stage_off) {
  extern __shared__ uint64_t smem[];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & (kWave - 1), w = tid / kWave;
  const int cap = tree.cap;
  const int nb = tree.n_nodes[b];
  const size_t base = (size_t)b * cap;

  auto fail = [&](uint32_t bit) {
    if (tid == 0) {
      report(d_err, bit);
      n_graft[b] = 0;
      if (N > 0) n_next[b] = 0;
    }
    for (int f = tid; f < W; f += kThreads) graft_frontier[(size_t)b * W + f] = TG_NO_NODE;
    for (int j = tid; j < N; j += kThreads) next_frontier[(size_t)b * N + j] = TG_NO_NODE;
  };
  if (nb < 0 || nb > cap || nb + 1 > R) {
    fail(TG_DERR_BAD_NODE);
    return;
  }
  // LDS layout sized by cap (as allocated by the launcher), used up to nb
  const int P2cap = pow2_at_least(cap + 1);
  const int P2 = pow2_at_least(nb + 1);
  uint64_t *skey = smem;                                   // [P2cap]
  float *lse_s = reinterpret_cast<float *>(skey + P2cap);  // [cap + 1]
  float *cum_s = lse_s + (cap + 1);                        // [cap]
  float *lp_s = cum_s + cap;                               // [cap]
  int *par_s = reinterpret_cast<int *>(lp_s + cap);        // [cap]
  uint8_t *inC = reinterpret_cast<uint8_t *>(par_s + cap); // [cap]
  uint8_t *done = inC + cap;                               // [cap]

  // ---- pool C and parents
  bool badp = false;
  int cnt = 0;
  for (int v = tid; v < nb; v += kThreads) {
    uint8_t in = tree.visited[base + v] ? 0 : 1;
    inC[v] = in;
    done[v] = in ? 0 : 1;
    cum_s[v] = tree.cum[base + v];
    par_s[v] = sane_parent(tree.parent[base + v], v, badp);
    cnt += in;
  }
  const int root_in = tree.root_visited[b] ? 0 : 1;
  if (badp) report(d_err, TG_DERR_BAD_PARENT);
  __shared__ int red[kWaves];
  int wsum = wave_sum_i32(cnt);
  if (lane == 0) red[w] = wsum;
  __syncthreads();
  int poolC = root_in;
  for (int i = 0; i < kWaves; ++i) poolC += red[i];

  // ---- log-sum-exp of every needed row (a thread per row), exported
  const uint8_t *need = needed + (size_t)b * R;
  for (int r = tid; r <= nb; r += kThreads) {
    if (!need[r]) continue;
    const size_t slot = (size_t)b * R + r;
    const float lse = finish_lse(part_ms + slot * n_ms, n_ms);
    lse_s[r] = lse;
    row_lse[slot] = lse;
  }
  __syncthreads();

  const int nF = min(W, poolC);
  if (nb + nF * M > cap) {
    fail(TG_DERR_CAPACITY);
    return;
  }

  // ---- rescoring: logp[v] = fl(x[pa(v)+1][tok v] - lse[pa(v)+1])
  bool badtok = false, nonfin = false;
  for (int v = tid; v < nb; v += kThreads) {
    if (!inC[v]) continue;
    const int p = par_s[v];
    const int tok = tree.token[base + v];
    float x = -__builtin_inff();
    if (tok >= 0 && tok < V)
      x = clean_logit(strong[((size_t)b * R + (p + 1)) * V + tok], nonfin);
    else
      badtok = true;
    const float lp = edge_logp(x, lse_s[p + 1]);
    lp_s[v] = lp;
    tree.logp[base + v] = lp;
  }
  if (badtok) report(d_err, TG_DERR_BAD_NODE);
  if (nonfin) report(d_err, TG_DERR_NONFINITE);
  __syncthreads();

  // ---- cum recompute, parents before children: rounds of "every pool node
  // whose parent is final takes cum[parent] + logp" (one round per level)
  for (;;) {
    // phase 1: decide who is ready from the previous round's state
    uint32_t ready = 0;  // bit i <-> node tid + i * kThreads
    int pending = 0;
    for (int i = 0, v = tid; v < nb; ++i, v += kThreads) {
      if (!inC[v] || done[v]) continue;
      const int p = par_s[v];
      if (p < 0 || done[p]) ready |= 1u << i;
      else pending = 1;
    }
    __syncthreads();
    for (int i = 0, v = tid; v < nb; ++i, v += kThreads) {
      if (!(ready >> i & 1u)) continue;
      const int p = par_s[v];
      cum_s[v] = __fadd_rn(p < 0 ? 0.0f : cum_s[p], lp_s[v]);
      done[v] = 1;
    }
    if (!__syncthreads_or(pending)) break;
  }

  // ---- reselection: Top_W(C) by (cum desc, depth asc, id asc)
  for (int i = tid; i < P2; i += kThreads) {
    uint64_t k = 0;
    if (i < nb) {
      if (inC[i]) k = node_key(cum_s[i], tree.depth[base + i], i);
    } else if (i == nb && root_in) {
      k = node_key(0.0f, 0, -1);
    }
    skey[i] = k;
  }
  __syncthreads();
  block_top_keys<kThreads>(skey, nb + 1, P2, nF);

  // ---- P <- P u C; write back rescored path scores (before the graft,
  // whose staging reuses the per-node scratch)
  for (int v = tid; v < nb; v += kThreads) {
    if (inC[v]) tree.cum[base + v] = cum_s[v];
    tree.visited[base + v] = 1;
  }
  __syncthreads();

  // ---- non-destructive graft: new children only, ids nb + f*M + j
  // (wave-private LDS for finishing each graft point's top-M; the region of
  // the per-node scratch, free by now, or extra room past it)
  uint64_t *wstage = reinterpret_cast<uint64_t *>(reinterpret_cast<char *>(smem) + stage_off) +
                     (size_t)w * (chunks * M);
  for (int f = w; f < nF; f += kWaves) {
    const int v = node_key_id(skey[f]);
    const int row = v + 1;
    const size_t slot = (size_t)b * R + row;
    const uint64_t key = wave_finish_topk(part_keys + slot * chunks * M, chunks, M, wstage);
    const float cv = v < 0 ? 0.0f : cum_s[v];
    const int dv = v < 0 ? 0 : tree.depth[base + v];
    const float lse = lse_s[row];
    if (lane < M) {
      const int j = lane;
      const float lp = edge_logp(key_logit(key), lse);
      const int id = nb + f * M + j;
      tree.parent[base + id] = v;
      tree.token[base + id] = (int)key_token(key);
      tree.depth[base + id] = dv + 1;
      tree.logp[base + id] = lp;
      tree.cum[base + id] = __fadd_rn(cv, lp);
      tree.visited[base + id] = 0;
    }
  }
  for (int f = tid; f < W; f += kThreads)
    graft_frontier[(size_t)b * W + f] = f < nF ? node_key_id(skey[f]) : TG_NO_NODE;
  if (tid == 0) {
    tree.root_visited[b] = 1;
    tree.n_nodes[b] = nb + nF * M;
    n_graft[b] = nF;
  }
  // ---- Top_N of the grafted children (the next small step's frontier)
  if (N > 0) {
    __syncthreads();  // children written above are visible to the block
    const int total = nF * M;
    const int P2c = pow2_at_least(total > 0 ? total : 1);
    for (int c = tid; c < P2c; c += kThreads) {
      uint64_t k = 0;
      if (c < total) {
        const int id = nb + c;
        k = node_key(tree.cum[base + id], tree.depth[base + id], id);
      }
      skey[c] = k;
    }
    __syncthreads();
    const int nn = min(N, total);
    block_top_keys<kThreads>(skey, total, P2c, nn);
    for (int j = tid; j < N; j += kThreads)
      next_frontier[(size_t)b * N + j] = j < nn ? node_key_id(skey[j]) : TG_NO_NODE;
    if (tid == 0) n_next[b] = nn;
  }
}

__global__ __launch_bounds__(kThreads) void tree_reset_kernel(tg_tree tree, int B) {
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b < B) {
    tree.n_nodes[b] = 0;
    tree.root_visited[b] = 0;
  }
}

}  // namespace

hipError_t launch_tree_reset(const tg_tree &tree, int B, hipStream_t stream) {
  launch("tree_reset", tree_reset_kernel, dim3((B + kThreads - 1) / kThreads),
         dim3(kThreads), 0, stream, tree, B);
  return hipGetLastError();
}

static int expand_skey_cap(int F, int K, int chunks) {
  // the sort needs pow2(F*K) keys; finishing rows wants every row's chunk
  // lists staged at once (one global round trip), up to 64 KiB of them
  const int total = F * K;
  const int stage_all = std::min(F * chunks * K, 8192);
  return std::max({pow2_at_least(total > 0 ? total : 1), chunks * K, stage_all});
}

hipError_t launch_expand_tree(const tg_tree &tree, const int32_t *frontier,
                              const int32_t *n_frontier, int B, int F, int K,
                              int N, RowPlan plan, const float2 *part_ms,
                              const uint64_t *part_keys, float *row_lse,
                              int32_t *next_frontier, int32_t *n_next,
                              uint32_t *d_err, hipStream_t stream) {
  const int skey_cap = expand_skey_cap(F, K, plan.chunks);
  const size_t lds = (size_t)F * K * 8 + (size_t)skey_cap * 8 + (size_t)F * 4;
  hipError_t e = hipFuncSetAttribute((const void *)expand_tree_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  launch("expand_tree", expand_tree_kernel, dim3(B), dim3(kThreads), lds, stream, tree,
         frontier, n_frontier, F, K, N, plan.chunks, plan.ms_per_row, part_ms, part_keys,
         row_lse, next_frontier, n_next, d_err, skey_cap);
  return hipGetLastError();
}

hipError_t launch_rescore_pool(const tg_tree &tree, int B, int R,
                               uint8_t *needed, hipStream_t stream) {
  launch("rescore_pool", rescore_pool_kernel, dim3(B), dim3(kThreads), 0, stream,
                     tree, R, needed);
  return hipGetLastError();
}

hipError_t launch_rescore_tree(const tg_tree &tree, const float *strong, int B,
                               int R, int V, int W, int M, RowPlan plan,
                               const uint8_t *needed, const float2 *part_ms,
                               const uint64_t *part_keys, float *row_lse,
                               int32_t *graft_frontier, int32_t *n_graft,
                               int32_t *next_frontier, int32_t *n_next, int N,
                               uint32_t *d_err, hipStream_t stream) {
  // layout sized by cap (the kernel uses it up to the live node count):
  // keys [pow2(cap+1)] | lse [cap+1] | cum, logp, parent [cap] | inC, done [cap]
  const int n = tree.cap;
  const size_t keys_b = (size_t)pow2_at_least(n + 1) * 8;
  const size_t head_b = keys_b + (size_t)(n + 1) * 4 + (size_t)n * 4;  // up to logp
  const size_t scratch_b = (size_t)n * (4 + 4 + 1 + 1);                // logp..done
  size_t lds = head_b + scratch_b;
  // per-wave top-M staging reuses logp..done when they are large enough
  const size_t stage_b = (size_t)(kThreads / kWave) * plan.chunks * M * 8;
  size_t stage_off = (head_b + 7) / 8 * 8;
  if (plan.chunks > 1 && stage_off + stage_b > head_b + scratch_b) {
    stage_off = (lds + 7) / 8 * 8;
    lds = stage_off + stage_b;
  }
  hipError_t e = hipFuncSetAttribute((const void *)rescore_tree_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  launch("rescore_tree", rescore_tree_kernel, dim3(B), dim3(kThreads), lds, stream, tree,
         strong, R, V, W, M, plan.chunks, plan.ms_per_row, needed, part_ms, part_keys,
         row_lse, graft_frontier, n_graft, next_frontier, n_next, N, d_err, (int)stage_off);
  return hipGetLastError();
}

}  // namespace tg
