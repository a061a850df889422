// Per-tree phases of the expansion step (Sec. 3.1; Alg. 1) and of the
// middle-drafter step (Sec. 3.2; Alg. 2, middle branch).
//
// One workgroup owns one tree.  The vocabulary-wide work already happened in
// the row pass and its finish (a wave per row across the chip): each needed
// row's log-sum-exp and top-K list are read from there, then the tree is
// edited in place:
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

__device__ __forceinline__ int sane_parent(int p, int v, bool &bad) {
  bool b = p < -1 || p >= v;
  bad |= b;
  return b ? -1 : p;
}

// --------------------------------------------------------------- expand
__global__ __launch_bounds__(kThreads) void expand_tree_kernel(
    tg_tree tree, const int32_t *__restrict__ frontier,
    const int32_t *__restrict__ n_frontier, int F, int K, int N,
    const float *__restrict__ row_lse, const uint64_t *__restrict__ row_keys,
    int32_t *__restrict__ next_frontier, int32_t *__restrict__ n_next, uint32_t *d_err) {
  extern __shared__ uint64_t skey[];  // [pow2(F * K)]
  const int b = blockIdx.x, tid = threadIdx.x;
  const int cap = tree.cap;
  int Fb = n_frontier ? n_frontier[b] : F;
  Fb = Fb < 0 ? 0 : (Fb > F ? F : Fb);
  const int nb = tree.n_nodes[b];
  const int total = Fb * K;
  const int P2 = pow2_at_least(total > 0 ? total : 1);

  bool bad = nb < 0 || nb > cap;
  for (int f = tid; f < Fb; f += kThreads) {
    int v = frontier[(size_t)b * F + f];
    bad |= v < -1 || v >= nb;
  }
  bad = __syncthreads_or(bad);

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
    const uint64_t key = row_keys[(size_t)b * F * K + c];
    const int v = frontier[(size_t)b * F + f];
    const float cv = v < 0 ? 0.0f : tree.cum[base + v];
    const int dv = v < 0 ? 0 : tree.depth[base + v];
    const float lp = edge_logp(key_logit(key), row_lse[(size_t)b * F + f]);
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
// The candidate pool C of a middle step (Sec. 3.2): the unvisited nodes and
// the root while unvisited; with TG_POOL_NEWONLY (the w/o EG ablation, Sec.
// 4.4) the previous step's new nodes, ids new_from[b] .. n_b - 1, the root
// when new_from[b] == -1 (read clamped to [-1, n_b]).
struct PoolRule {
  bool newonly;
  int lo;
  __device__ bool in(const tg_tree &t, size_t base, int v) const {
    return newonly ? v >= lo : !t.visited[base + v];
  }
  __device__ bool root_in(const tg_tree &t, int b) const {
    return newonly ? lo <= -1 : !t.root_visited[b];
  }
};
__device__ inline PoolRule pool_rule(const tg_tree &t, int b, int nb, uint32_t flags,
                                     const int32_t *new_from) {
  PoolRule r{(flags & TG_POOL_NEWONLY) != 0, 0};
  if (r.newonly) r.lo = min(max(new_from[b], -1), max(nb, 0));
  return r;
}


// needed[b, r] = 1 iff logits row r is read by this middle step: the row of
// each pool node (its children) and the row of each pool node's parent (its
// edge score).  Rows of trees that cannot be processed are all 0.
__global__ __launch_bounds__(kThreads) void rescore_pool_kernel(
    tg_tree tree, int R, uint8_t *__restrict__ needed, uint32_t flags,
    const int32_t *__restrict__ new_from) {
  __shared__ uint8_t flag[TG_MAX_CAP + 1];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int nb = tree.n_nodes[b];
  const bool ok = nb >= 0 && nb <= tree.cap && nb + 1 <= R;
  const int rows = ok ? nb + 1 : 0;
  for (int r = tid; r < rows; r += kThreads) flag[r] = 0;
  __syncthreads();
  const size_t base = (size_t)b * tree.cap;
  const PoolRule pool = pool_rule(tree, b, nb, flags, new_from);
  if (ok) {
    if (tid == 0 && pool.root_in(tree, b)) flag[0] = 1;
    bool dummy = false;
    for (int v = tid; v < nb; v += kThreads) {
      const int p = tree.parent[base + v];  // read with the pool flag, not after it
      if (pool.in(tree, base, v)) {
        flag[v + 1] = 1;
        flag[sane_parent(p, v, dummy) + 1] = 1;
      }
    }
  }
  __syncthreads();
  for (int r = tid; r < R; r += kThreads)
    needed[(size_t)b * R + r] = r < rows ? flag[r] : 0;
}

// ------------------------------------------------------- graft variants
// The middle step's graft under TG_GRAFT_OVERWRITE (w/o ND, Sec. 5.3: the
// frontier nodes' existing subtrees are removed and the tree compacted
// before the new children are attached) and TG_GRAFT_DEDUP (a child whose
// token an existing child of the same parent carries is skipped; kept
// children take dense ids in (slot, rank) order).  Entered after the
// reselection (F = skey[0, nF)) and the P <- P u C write-back.  LDS:
//   vmap, rrow, rpid, rdep, rcum  [cap] each (the variant region);
//   stage = the logp scratch, flags = inC / done, candidates = skey.
__device__ void graft_variant(const tg_tree &tree, int b, int nb, int nF, int M, int W,
                              int N, int R, uint32_t flags,
                              const uint64_t *__restrict__ row_keys, const float *lse_s,
                              const float *cum_s, const int *par_s, int *stage,
                              uint8_t *flag_a, uint8_t *flag_b, uint64_t *skey, int *var,
                              int *red, int32_t *graft_frontier,
                              int32_t *n_graft, int32_t *next_frontier, int32_t *n_next) {
  __shared__ int rootF_s, nF2_s, rootslot_s;
  const int tid = threadIdx.x;
  const int cap = tree.cap;
  const size_t base = (size_t)b * cap;
  int *vmap = var, *rrow = var + cap, *rpid = var + 2 * cap, *rdep = var + 3 * cap;
  float *rcum = reinterpret_cast<float *>(var + 4 * cap);

  // frontier records (logits row, id, depth, cum) from the old ids
  for (int f = tid; f < nF; f += kThreads) {
    const int v = node_key_id(skey[f]);
    rrow[f] = v + 1;
    rpid[f] = v;
    rdep[f] = v < 0 ? 0 : tree.depth[base + v];
    rcum[f] = v < 0 ? 0.0f : cum_s[v];
  }
  if (tid == 0) {
    rootF_s = 0;
    nF2_s = nF;
    rootslot_s = -1;
  }
  __syncthreads();
  int nb2 = nb;

  if (flags & TG_GRAFT_OVERWRITE) {
    uint8_t *inF = flag_a, *dead = flag_b;
    for (int v = tid; v < nb; v += kThreads) {
      inF[v] = 0;
      dead[v] = 0;
    }
    __syncthreads();
    for (int f = tid; f < nF; f += kThreads) {
      if (rpid[f] < 0) rootF_s = 1;
      else inF[rpid[f]] = 1;
    }
    __syncthreads();
    const bool rootF = rootF_s != 0;
    // dead = a strict ancestor is in F; one more level settles per round
    for (;;) {
      int changed = 0;
      for (int v = tid; v < nb; v += kThreads) {
        if (dead[v]) continue;
        const int p = par_s[v];
        if (rootF || (p >= 0 && (inF[p] || dead[p]))) {
          dead[v] = 1;
          changed = 1;
        }
      }
      if (!__syncthreads_or(changed)) break;
    }
    // survivors get dense ids in id order
    const int per = (nb + kThreads - 1) / kThreads;
    const int lo = min(nb, tid * per), hi = min(nb, lo + per);
    int mine = 0;
    for (int v = lo; v < hi; ++v) mine += dead[v] ? 0 : 1;
    int total = 0;
    int pos = block_exclusive_scan<kThreads>(mine, red, total);
    for (int v = lo; v < hi; ++v) vmap[v] = dead[v] ? -1 : pos++;
    nb2 = total;
    __syncthreads();
    // move the survivors down (every read lands in LDS before any write)
    auto move = [&](int32_t *field, int which) {
      for (int v = tid; v < nb; v += kThreads) {
        if (dead[v]) continue;
        int x;
        if (which == 0) x = par_s[v] < 0 ? -1 : vmap[par_s[v]];
        else if (which == 1) x = tree.visited[base + v];
        else x = field[base + v];
        stage[v] = x;
      }
      __syncthreads();
      for (int v = tid; v < nb; v += kThreads) {
        if (dead[v]) continue;
        if (which == 1) tree.visited[base + vmap[v]] = (uint8_t)stage[v];
        else field[base + vmap[v]] = stage[v];
      }
      __syncthreads();
    };
    move(tree.parent, 0);
    move(nullptr, 1);
    move(tree.token, 2);
    move(tree.depth, 2);
    move(reinterpret_cast<int32_t *>(tree.logp), 2);
    for (int v = tid; v < nb; v += kThreads)
      if (!dead[v]) tree.cum[base + vmap[v]] = cum_s[v];
    // surviving frontier slots, in order, with their new ids
    if (tid == 0) {
      int k = 0;
      for (int f = 0; f < nF; ++f) {
        const int v = rpid[f];
        if (v >= 0 && dead[v]) continue;
        rrow[k] = rrow[f];
        rdep[k] = rdep[f];
        rcum[k] = rcum[f];
        rpid[k] = v < 0 ? -1 : vmap[v];
        ++k;
      }
      nF2_s = k;
    }
    __syncthreads();
  }
  const int nF2 = nF2_s;

  // candidates of every (slot, rank) in skey
  for (int c = tid; c < nF2 * M; c += kThreads) {
    const int f = c / M;
    skey[c] = row_keys[((size_t)b * R + rrow[f]) * M + (c - f * M)];
  }
  __syncthreads();
  const int total_c = nF2 * M;
  uint8_t *dup = flag_a;
  for (int i = tid; i < total_c; i += kThreads) dup[i] = 0;
  if ((flags & TG_GRAFT_DEDUP) && !(flags & TG_GRAFT_OVERWRITE)) {
    for (int v = tid; v < nb; v += kThreads) vmap[v] = -1;
    __syncthreads();
    for (int f = tid; f < nF2; f += kThreads) {
      if (rpid[f] < 0) rootslot_s = f;
      else vmap[rpid[f]] = f;
    }
    __syncthreads();
    for (int u = tid; u < nb; u += kThreads) {
      const int p = par_s[u];
      const int f = p < 0 ? rootslot_s : vmap[p];
      if (f < 0) continue;
      const uint32_t tok = (uint32_t)tree.token[base + u];
      for (int j = 0; j < M; ++j)
        if (key_token(skey[f * M + j]) == tok) dup[f * M + j] = 1;
    }
  }
  __syncthreads();

  // kept candidates get dense ids nb2 + rank in (slot, rank) order
  const int per2 = (total_c + kThreads - 1) / kThreads;
  const int lo2 = min(total_c, tid * per2), hi2 = min(total_c, lo2 + per2);
  int mine2 = 0;
  for (int i = lo2; i < hi2; ++i) mine2 += dup[i] ? 0 : 1;
  int total_k = 0;
  const int first = block_exclusive_scan<kThreads>(mine2, red, total_k);
  int pos2 = first;
  for (int i = lo2; i < hi2; ++i) {
    if (dup[i]) continue;
    const int f = i / M;
    const uint64_t key = skey[i];
    const int id = nb2 + pos2++;
    const float lp = edge_logp(key_logit(key), lse_s[rrow[f]]);
    tree.parent[base + id] = rpid[f];
    tree.token[base + id] = (int)key_token(key);
    tree.depth[base + id] = rdep[f] + 1;
    tree.logp[base + id] = lp;
    tree.cum[base + id] = __fadd_rn(rcum[f], lp);
    tree.visited[base + id] = 0;
  }
  for (int f = tid; f < W; f += kThreads)
    graft_frontier[(size_t)b * W + f] = f < nF2 ? rpid[f] : TG_NO_NODE;
  if (tid == 0) {
    tree.n_nodes[b] = nb2 + total_k;
    n_graft[b] = nF2;
  }
  if (N <= 0) return;
  __syncthreads();  // every candidate key has been read
  // Top_N of the new children
  pos2 = first;
  for (int i = lo2; i < hi2; ++i) {
    if (dup[i]) continue;
    const int id = nb2 + pos2++;
    skey[id - nb2] = node_key(tree.cum[base + id], tree.depth[base + id], id);
  }
  const int P2c = pow2_at_least(total_k > 0 ? total_k : 1);
  for (int c = total_k + tid; c < P2c; c += kThreads) skey[c] = 0;
  __syncthreads();
  const int nn = min(N, total_k);
  block_top_keys<kThreads>(skey, total_k, P2c, nn);
  for (int j = tid; j < N; j += kThreads)
    next_frontier[(size_t)b * N + j] = j < nn ? node_key_id(skey[j]) : TG_NO_NODE;
  if (tid == 0) n_next[b] = nn;
}

// ------------------------------------------------ rescore + reselect + graft
__global__ __launch_bounds__(kThreads) void rescore_tree_kernel(
    tg_tree tree, const float *__restrict__ strong, int R, int V, int W, int M,
    const float *__restrict__ row_lse,
    const uint64_t *__restrict__ row_keys, int32_t *__restrict__ graft_frontier,
    int32_t *__restrict__ n_graft, int32_t *__restrict__ next_frontier,
    int32_t *__restrict__ n_next, int N, uint32_t *d_err, uint32_t flags,
    const int32_t *__restrict__ new_from, int var_off) {
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
  int *dep_s = par_s + cap;                                // [cap]
  uint8_t *inC = reinterpret_cast<uint8_t *>(dep_s + cap); // [cap]
  uint8_t *done = inC + cap;                               // [cap]

  // ---- pool C, node fields and the rescored edges
  // logp[v] = fl(x[pa(v)+1][tok v] - lse[pa(v)+1]) for v in C.  Per batch of
  // nodes: the fields and the row lse in one round of reads, then for the
  // pool nodes the strong logit and the parent row's lse in a second.  Rows
  // that are not needed hold whatever the buffer held and are never read.
  const PoolRule pool = pool_rule(tree, b, nb, flags, new_from);
  if (tid == 0 && pool.newonly && (new_from[b] < -1 || new_from[b] > nb))
    report(d_err, TG_DERR_BAD_NODE);
  bool badp = false, badtok = false, nonfin = false;
  int cnt = 0;
  constexpr int kBatch = 4;
  for (int v0 = 0; v0 <= nb; v0 += kBatch * kThreads) {
    int pv[kBatch], tv[kBatch], dv[kBatch];
    float cv[kBatch], rl[kBatch];
    bool in[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int v = v0 + tid + k * kThreads;
      const bool ok = v < nb;
      pv[k] = ok ? tree.parent[base + v] : -1;
      tv[k] = ok ? tree.token[base + v] : 0;
      dv[k] = ok ? tree.depth[base + v] : 0;
      cv[k] = ok ? tree.cum[base + v] : 0.0f;
      in[k] = ok && pool.in(tree, base, v);
      rl[k] = v <= nb ? row_lse[(size_t)b * R + v] : 0.0f;
    }
    float xv[kBatch], lv[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int v = v0 + tid + k * kThreads;
      xv[k] = -__builtin_inff();
      lv[k] = 0.0f;
      if (v < nb) {
        pv[k] = sane_parent(pv[k], v, badp);
        if (in[k]) {
          const size_t prow = (size_t)b * R + (pv[k] + 1);
          lv[k] = row_lse[prow];
          if (tv[k] >= 0 && tv[k] < V) xv[k] = strong[prow * V + tv[k]];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int v = v0 + tid + k * kThreads;
      if (v <= nb) lse_s[v] = rl[k];
      if (v >= nb) continue;
      inC[v] = in[k] ? 1 : 0;
      done[v] = in[k] ? 0 : 1;
      cum_s[v] = cv[k];
      par_s[v] = pv[k];
      dep_s[v] = dv[k];
      cnt += in[k] ? 1 : 0;
      if (in[k]) {
        float x = -__builtin_inff();
        if (tv[k] >= 0 && tv[k] < V)
          x = clean_logit(xv[k], nonfin);
        else
          badtok = true;
        lp_s[v] = edge_logp(x, lv[k]);
      }
    }
  }
  const int root_in = pool.root_in(tree, b) ? 1 : 0;
  if (badp) report(d_err, TG_DERR_BAD_PARENT);
  __shared__ int red[kWaves];
  int wsum = wave_sum_i32(cnt);
  if (lane == 0) red[w] = wsum;
  __syncthreads();
  int poolC = root_in;
  for (int i = 0; i < kWaves; ++i) poolC += red[i];

  const int nF = min(W, poolC);
  if (nb + nF * M > cap) {
    fail(TG_DERR_CAPACITY);
    return;
  }
  if (badtok) report(d_err, TG_DERR_BAD_NODE);
  if (nonfin) report(d_err, TG_DERR_NONFINITE);

  // ---- cum recompute, parents before children.  Each pool node walks up to
  // its nearest ancestor outside the pool (or the root), up to kChain steps,
  // and folds the logps of the path down from there: the same additions in
  // the same order as level by level, with no barrier.  Nodes further below
  // the pool's edge are finished by rounds of "every pool node whose parent
  // is final takes cum[parent] + logp" (one round per level).
  constexpr int kChain = 16;
  bool deep = false;
  for (int v = tid; v < nb; v += kThreads) {
    if (!inC[v]) continue;
    int ch[kChain];
    int len = 0, u = v;
    bool up = true;
#pragma unroll
    for (int t = 0; t < kChain; ++t) {
      if (up) {
        ch[t] = u;
        len = t + 1;
        u = par_s[u];
        up = u >= 0 && inC[u];
      }
    }
    if (up) {  // the pool continues above kChain levels
      deep = true;
      continue;
    }
    float c = u < 0 ? 0.0f : cum_s[u];
#pragma unroll
    for (int t = kChain - 1; t >= 0; --t)
      if (t < len) c = __fadd_rn(c, lp_s[ch[t]]);
    cum_s[v] = c;
    done[v] = 1;
  }
  if (__syncthreads_or(deep)) {
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
  }

  // ---- reselection: Top_W(C) by (cum desc, depth asc, id asc)
  for (int i = tid; i < P2; i += kThreads) {
    uint64_t k = 0;
    if (i < nb) {
      if (inC[i]) k = node_key(cum_s[i], dep_s[i], i);
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
    if (inC[v]) {
      tree.logp[base + v] = lp_s[v];
      tree.cum[base + v] = cum_s[v];
      tree.visited[base + v] = 1;
    }
  }
  if (tid == 0 && root_in) tree.root_visited[b] = 1;
  __syncthreads();

  if (flags & (TG_GRAFT_OVERWRITE | TG_GRAFT_DEDUP)) {
    graft_variant(tree, b, nb, nF, M, W, N, R, flags, row_keys, lse_s, cum_s, par_s,
                  reinterpret_cast<int *>(lp_s), inC, done, skey,
                  reinterpret_cast<int *>(reinterpret_cast<char *>(smem) + var_off), red,
                  graft_frontier, n_graft, next_frontier, n_next);
    return;
  }

  // ---- non-destructive graft: new children only, ids nb + f*M + j (a
  // thread per child; the keys of a thread's first children stay in
  // registers for the Top_N below)
  const int total = nF * M;
  auto graft_child = [&](int c) {
    const int f = c / M;
    const int v = node_key_id(skey[f]);
    const int row = v + 1;
    const uint64_t key = row_keys[((size_t)b * R + row) * M + (c - f * M)];
    const float cv = v < 0 ? 0.0f : cum_s[v];
    const int dv = v < 0 ? 0 : dep_s[v];
    const float lp = edge_logp(key_logit(key), lse_s[row]);
    const float cum = __fadd_rn(cv, lp);
    const int id = nb + c;
    tree.parent[base + id] = v;
    tree.token[base + id] = (int)key_token(key);
    tree.depth[base + id] = dv + 1;
    tree.logp[base + id] = lp;
    tree.cum[base + id] = cum;
    tree.visited[base + id] = 0;
    return node_key(cum, dv + 1, id);
  };
  constexpr int kRegChildren = 4;
  uint64_t ck[kRegChildren];
#pragma unroll
  for (int k = 0; k < kRegChildren; ++k) {
    const int c = tid + k * kThreads;
    ck[k] = c < total ? graft_child(c) : 0;
  }
  for (int c = tid + kRegChildren * kThreads; c < total; c += kThreads) graft_child(c);
  for (int f = tid; f < W; f += kThreads)
    graft_frontier[(size_t)b * W + f] = f < nF ? node_key_id(skey[f]) : TG_NO_NODE;
  if (tid == 0) {
    tree.n_nodes[b] = nb + total;
    n_graft[b] = nF;
  }
  // ---- Top_N of the grafted children (the next small step's frontier)
  if (N > 0) {
    __syncthreads();  // the graft frontier is read; children past the
                      // registers are visible to the block
    const int P2c = pow2_at_least(total > 0 ? total : 1);
#pragma unroll
    for (int k = 0; k < kRegChildren; ++k) {
      const int c = tid + k * kThreads;
      if (c < P2c) skey[c] = ck[k];
    }
    for (int c = tid + kRegChildren * kThreads; c < P2c; c += kThreads) {
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

hipError_t launch_expand_tree(const tg_tree &tree, const int32_t *frontier,
                              const int32_t *n_frontier, int B, int F, int K,
                              int N, const float *row_lse, const uint64_t *row_keys,
                              int32_t *next_frontier, int32_t *n_next,
                              uint32_t *d_err, hipStream_t stream) {
  const size_t lds = (size_t)pow2_at_least(F * K) * 8;
  hipError_t e = hipFuncSetAttribute((const void *)expand_tree_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  launch("expand_tree", expand_tree_kernel, dim3(B), dim3(kThreads), lds, stream, tree,
         frontier, n_frontier, F, K, N, row_lse, row_keys, next_frontier, n_next, d_err);
  return hipGetLastError();
}

hipError_t launch_rescore_pool(const tg_tree &tree, int B, int R, uint8_t *needed,
                               uint32_t flags, const int32_t *new_from,
                               hipStream_t stream) {
  launch("rescore_pool", rescore_pool_kernel, dim3(B), dim3(kThreads), 0, stream,
                     tree, R, needed, flags, new_from);
  return hipGetLastError();
}

size_t rescore_tree_lds(int cap, uint32_t flags, int *var_off) {
  // layout sized by cap (the kernel uses it up to the live node count):
  // keys [pow2(cap+1)] | lse [cap+1] | cum, logp, parent, depth [cap] |
  // inC, done [cap] (| variant records [5 cap] ints when a graft variant is on)
  const int n = cap;
  size_t lds = (size_t)pow2_at_least(n + 1) * 8 + (size_t)(n + 1) * 4 +
               (size_t)n * (4 + 4 + 4 + 4 + 1 + 1);
  size_t vo = 0;
  if (flags & (TG_GRAFT_OVERWRITE | TG_GRAFT_DEDUP)) {
    vo = (lds + 15) / 16 * 16;
    lds = vo + (size_t)5 * n * 4;
  }
  *var_off = (int)vo;
  return lds;
}

hipError_t launch_rescore_tree(const tg_tree &tree, const float *strong, int B,
                               int R, int V, int W, int M, const float *row_lse, const uint64_t *row_keys,
                               int32_t *graft_frontier, int32_t *n_graft,
                               int32_t *next_frontier, int32_t *n_next, int N,
                               uint32_t flags, const int32_t *new_from,
                               uint32_t *d_err, hipStream_t stream) {
  int var_off = 0;
  const size_t lds = rescore_tree_lds(tree.cap, flags, &var_off);
  hipError_t e = hipFuncSetAttribute((const void *)rescore_tree_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  launch("rescore_tree", rescore_tree_kernel, dim3(B), dim3(kThreads), lds, stream, tree,
         strong, R, V, W, M, row_lse, row_keys, graft_frontier, n_graft,
         next_frontier, n_next, N, d_err, flags, new_from, var_off);
  return hipGetLastError();
}

}  // namespace tg
