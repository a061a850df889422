// Final pruning to the verification budget with ancestor closure and the
// verification buffers (Alg. 3), and the cache update after acceptance.
//
// prune_kernel: one workgroup per tree, everything in LDS (n <= 4096); the
// parents, path scores and tokens are read in one batch up front:
//   depths by pointer jumping over the parent links (until every chain has
//         reached the root);
//   keep: node keys (cum desc, depth asc, id asc) are distinct and order the
//         nodes as their ranks do, so one parallel pass checks that every
//         parent's key is larger than its children's; then the kept set is
//         the B_ver largest keys (selected, not ranked); otherwise the nodes
//         are ranked exactly (counting the larger keys, a bitonic sort past
//         1024 nodes) and one thread runs the literal loop (chains added
//         while they fit);
//   re-index: the kept nodes, compacted by a block scan, ranked the same way
//         by (depth, id);
//   buffers: parents, tokens, depths, ancestor bitsets, root-to-leaf paths.
// kv_compact_kernel: one workgroup per (sequence, KV head); every thread
// copies its 16-byte column of the accepted rows in path order, which is
// safe in place because a row is only overwritten after it has been read
// (path[j] >= j, strictly increasing).
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;

constexpr int kRankCountMax = kRankPerThread * kThreads;  // rank by counting up to here
constexpr int kPre = 4;  // node slots per thread read in the first batch

__global__ __launch_bounds__(kThreads) void prune_kernel(
    tg_tree tree, int B_ver, int max_path, int32_t *__restrict__ kept,
    int32_t *__restrict__ vparent, int32_t *__restrict__ vtoken,
    int32_t *__restrict__ position_ids, uint32_t *__restrict__ mask,
    int32_t *__restrict__ retrieval, int32_t *__restrict__ n_keep,
    int32_t *__restrict__ n_leaves, uint32_t *d_err) {
  __shared__ __align__(16) uint64_t key[TG_MAX_CAP];
  __shared__ int16_t par[TG_MAX_CAP];
  __shared__ int16_t anc[2][TG_MAX_CAP];
  __shared__ int16_t dep[2][TG_MAX_CAP];
  __shared__ int16_t newid[TG_MAX_CAP];    // original id -> verify index (0 = dropped)
  __shared__ int16_t order[TG_MAX_CAP];    // kept index -> original id
  __shared__ uint8_t flag[TG_MAX_CAP + 1];
  __shared__ int32_t tok_s[TG_MAX_CAP];
  __shared__ int cnt[kThreads];
  __shared__ int nk_s, nl_s, viol_s, deep_s;

  const int b = blockIdx.x, tid = threadIdx.x;
  const int cap = tree.cap;
  const int M = B_ver + 1;
  const int W = (M + 31) / 32;
  const size_t base = (size_t)b * cap;
  // ---- one batch of reads: the parents, path scores and tokens of the
  // first kPre * kThreads slots, bounded by the capacity so that they need
  // not wait for the node count (the count masks them once it arrives)
  const int n_ld = load_vmem(tree.n_nodes + b);
  int pr[kPre], tk[kPre];
  float cm[kPre];
#pragma unroll
  for (int j = 0; j < kPre; ++j) {
    const int v = tid + j * kThreads;
    pr[j] = v < cap ? tree.parent[base + v] : -1;
    cm[j] = v < cap ? tree.cum[base + v] : 0.0f;
    tk[j] = v < cap ? tree.token[base + v] : 0;
  }
  int n = uniform_int(n_ld);
  if (n < 0 || n > cap) {
    if (tid == 0) report(d_err, TG_DERR_BAD_NODE);
    n = -1;  // nothing kept, outputs padded below
  }
  const int nn = n < 0 ? 0 : n;

  // ---- parents (sanitised) and depths by pointer jumping
  bool badp = false;
  auto put_node = [&](int v, int p, int tok) {
    if (p < -1 || p >= v) {
      badp = true;
      p = -1;
    }
    par[v] = (int16_t)p;
    anc[0][v] = (int16_t)p;
    dep[0][v] = 1;
    tok_s[v] = tok;
  };
#pragma unroll
  for (int j = 0; j < kPre; ++j) {
    const int v = tid + j * kThreads;
    if (v < nn) put_node(v, pr[j], tk[j]);
  }
  for (int v = tid + kPre * kThreads; v < nn; v += kThreads)
    put_node(v, tree.parent[base + v], tree.token[base + v]);
  if (badp) report(d_err, TG_DERR_BAD_PARENT);
  if (tid == 0) {
    viol_s = 0;
    deep_s = 0;
  }
  __syncthreads();
  // (until every chain has reached the root: depth+1 rounds at most)
  int cur = 0;
  for (int span = 1; span < nn; span <<= 1) {
    const int nxt = cur ^ 1;
    bool more = false;
    for (int v = tid; v < nn; v += kThreads) {
      const int a = anc[cur][v];
      const int16_t na = a >= 0 ? anc[cur][a] : (int16_t)-1;
      anc[nxt][v] = na;
      dep[nxt][v] = a >= 0 ? (int16_t)(dep[cur][v] + dep[cur][a]) : dep[cur][v];
      more |= na >= 0;
    }
    cur = nxt;
    if (!__syncthreads_or(more)) break;
  }
  const int16_t *depth = dep[cur];

  // ---- keys by (cum desc, depth asc, id asc); keys are distinct, and a
  // node ranks before another exactly when its key is larger
  const int P2 = pow2_at_least(nn > 0 ? nn : 1);
#pragma unroll
  for (int j = 0; j < kPre; ++j) {
    const int i = tid + j * kThreads;
    if (i < P2) key[i] = i < nn ? node_key(cm[j], depth[i], i) : 0;
  }
  for (int i = tid + kPre * kThreads; i < P2; i += kThreads)
    key[i] = i < nn ? node_key(tree.cum[base + i], depth[i], i) : 0;
  for (int v = tid; v < nn; v += kThreads) flag[v] = 0;
  __syncthreads();

  // ---- keep (`sel`: the kept set is key[0, B_ver), selected below)
  bool sel = false;
  if (nn <= B_ver) {
    for (int v = tid; v < nn; v += kThreads) flag[v] = 1;
  } else {
    // does some node rank before its parent?  (one direct pass: parent key
    // against child key)
    bool viol = false;
    for (int v = tid; v < nn; v += kThreads) viol |= par[v] >= 0 && key[par[v]] < key[v];
    if (viol) viol_s = 1;
    __syncthreads();
    if (!viol_s) {
      // every ancestor outranks its descendants, so the B_ver best nodes are
      // closed under parents and are the kept set: select them
      if (nn > kThreads && nn <= kRankCountMax && B_ver <= kWave)
        block_select_top<kThreads>(key, nn, B_ver);
      else
        block_top_keys<kThreads>(key, nn, P2, B_ver);
      sel = B_ver <= kWave;
      if (!sel)
        for (int i = tid; i < B_ver; i += kThreads) flag[node_key_id(key[i])] = 1;
    } else {
      // exact ranks (counting for up to kRankCountMax nodes, else a bitonic
      // sort), then the literal loop: add each ranked node's missing
      // ancestor chain if it fits
      if (nn <= kRankCountMax) {
        rank_each<kThreads>(key, nn, [&](int v, uint64_t, int r) { order[r] = (int16_t)v; });
      } else {
        block_bitonic_desc(key, P2);
        for (int i = tid; i < nn; i += kThreads) order[i] = (int16_t)node_key_id(key[i]);
      }
      __syncthreads();
      if (tid == 0) {
        int size = 1;
        for (int i = 0; i < nn && size < M; ++i) {
          int len = 0;
          for (int u = order[i]; u >= 0 && !flag[u]; u = par[u]) ++len;
          if (size + len <= M) {
            for (int u = order[i]; u >= 0 && !flag[u]; u = par[u]) flag[u] = 1;
            size += len;
          }
        }
      }
    }
  }
  __syncthreads();

  // ---- re-index the kept nodes by (depth, id)
  for (int v = tid; v < nn; v += kThreads) newid[v] = 0;
  int nk;
  if (sel) {
    // the selected set (at most a wave's width): wave 0 ranks (depth, id)
    // packed in 32 bits (both below 2^16) against the set
    nk = B_ver;
    __syncthreads();  // newid cleared before the kept nodes' entries land
    if (tid < kWave) {
      const int v = tid < nk ? node_key_id(key[tid]) : 0;
      const uint32_t dk = tid < nk ? ((uint32_t)depth[v] << 16) | (uint32_t)v : ~0u;
      cnt[tid] = (int)dk;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      int r = 0;
      for (int j = 0; j < nk; ++j) r += (uint32_t)cnt[j] < dk ? 1 : 0;
      if (tid < nk) {
        order[r] = (int16_t)v;
        newid[v] = (int16_t)(r + 1);
      }
    }
  } else {
    // compact them (id order), then rank the compacted keys
    const int per_c = (nn + kThreads - 1) / kThreads;
    const int c_lo = min(nn, tid * per_c), c_hi = min(nn, c_lo + per_c);
    int mine_k = 0;
    for (int v = c_lo; v < c_hi; ++v) mine_k += flag[v];
    int nk_total = 0;
    int pos = block_exclusive_scan<kThreads>(mine_k, cnt, nk_total);
    for (int v = c_lo; v < c_hi; ++v)
      if (flag[v]) key[pos++] = ~(((uint64_t)depth[v] << 32) | (uint64_t)v);
    if (tid == 0) nk_s = nk_total;
    __syncthreads();
    nk = nk_s;
    if (nk <= kRankCountMax) {
      rank_each<kThreads>(key, nk, [&](int, uint64_t k, int r) {
        const int v = (int)(uint32_t)~k;
        order[r] = (int16_t)v;
        newid[v] = (int16_t)(r + 1);
      });
    } else {
      const int P2k = pow2_at_least(nk);
      for (int i = nk + tid; i < P2k; i += kThreads) key[i] = 0;
      __syncthreads();
      block_bitonic_desc(key, P2k);
      for (int j = tid; j < nk; j += kThreads) {
        const int v = (int)(uint32_t)~key[j];
        order[j] = (int16_t)v;
        newid[v] = (int16_t)(j + 1);
      }
    }
  }
  __syncthreads();

  // ---- per-node buffers
  const size_t ob = (size_t)b * B_ver;
  for (int j = tid; j < B_ver; j += kThreads) {
    if (j < nk) {
      const int v = order[j];
      const int p = par[v];
      kept[ob + j] = v;
      vparent[ob + j] = p < 0 ? -1 : newid[p] - 1;
      vtoken[ob + j] = tok_s[v];
    } else {
      kept[ob + j] = -1;
      vparent[ob + j] = -1;
      vtoken[ob + j] = -1;
    }
  }
  const size_t pb = (size_t)b * M;
  for (int u = tid; u < M; u += kThreads)
    position_ids[pb + u] = u == 0 ? 0 : (u <= nk ? depth[order[u - 1]] : -1);
  // verify parent of row u (root row 0 has none)
  auto vpar = [&](int u) { return u == 0 ? -1 : (par[order[u - 1]] < 0 ? 0 : newid[par[order[u - 1]]]); };
  // ancestor-or-self bitsets, one row per thread: verify indices decrease
  // up the chain, so each word is complete when the walk leaves it and is
  // written once (highest word first)
  for (int u = tid; u < M; u += kThreads) {
    uint32_t *row = mask + (pb + u) * W;
    uint32_t acc = 0;
    int cw = W - 1;
    if (u <= nk && n >= 0) {
      for (int a = u; a >= 0; a = vpar(a)) {
        for (; cw > (a >> 5); --cw) {
          row[cw] = acc;
          acc = 0;
        }
        acc |= 1u << (a & 31);
      }
    }
    for (; cw >= 0; --cw) {
      row[cw] = acc;
      acc = 0;
    }
  }

  // ---- leaves in verify order and their root-to-leaf paths
  for (int u = tid; u <= nk; u += kThreads) flag[u] = 1;
  __syncthreads();
  for (int u = 1 + tid; u <= nk; u += kThreads) flag[vpar(u)] = 0;
  __syncthreads();
  const int live = n < 0 ? 0 : nk + 1;  // verify rows (no root row for a bad tree)
  const int per = (live + kThreads - 1) / kThreads;
  const int lo = min(live, tid * per), hi = min(live, lo + per);
  int mine = 0;
  bool deep = false;
  for (int u = lo; u < hi; ++u) {
    if (!flag[u]) continue;
    ++mine;
    deep |= (u == 0 ? 0 : depth[order[u - 1]]) + 1 > max_path;
  }
  if (deep) deep_s = 1;
  int total = 0;
  const int first_rank = block_exclusive_scan<kThreads>(mine, cnt, total);
  if (tid == 0) {
    nl_s = total;
    if (deep_s) report(d_err, TG_DERR_CAPACITY);
  }
  __syncthreads();
  const bool write_paths = !deep_s;
  const size_t rb = (size_t)b * M * max_path;
  for (size_t i = tid; i < (size_t)M * max_path; i += kThreads) retrieval[rb + i] = -1;
  __syncthreads();
  if (write_paths) {
    int r = first_rank;
    for (int u = lo; u < hi; ++u) {
      if (!flag[u]) continue;
      int32_t *row = retrieval + rb + (size_t)r * max_path;
      for (int a = u; a >= 0; a = vpar(a)) row[a == 0 ? 0 : depth[order[a - 1]]] = a;
      ++r;
    }
  }
  if (tid == 0) {
    n_keep[b] = nk;
    n_leaves[b] = n < 0 ? 0 : nl_s;
  }
}

template <typename T>
__global__ __launch_bounds__(64) void kv_compact_kernel(
    T *__restrict__ k_cache, T *__restrict__ v_cache, const int32_t *__restrict__ prefix_len,
    const int32_t *__restrict__ path, const int32_t *__restrict__ n_path, int Hkv, int S_max,
    int D, int max_path, int32_t *__restrict__ new_prefix_len, uint32_t *d_err) {
  const int b = blockIdx.x / Hkv, h = blockIdx.x - b * Hkv;
  const int L = prefix_len[b];
  const int n = n_path[b];
  const int32_t *pp = path + (size_t)b * max_path;
  bool ok = n >= 0 && n <= max_path && L >= 0;
  for (int j = 0; ok && j < n; ++j) {
    const int x = pp[j];
    ok = x >= j && (j == 0 || x > pp[j - 1]) && L + x < S_max;
  }
  if (h == 0 && threadIdx.x == 0) {
    if (!ok) report(d_err, TG_DERR_BAD_NODE);
    new_prefix_len[b] = ok ? L + n : L;
  }
  if (!ok) return;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int cols = D * (int)sizeof(T) / 16;  // 16-byte columns per row
  const size_t hb = ((size_t)b * Hkv + h) * (size_t)S_max * D;
  for (int c = threadIdx.x; c < 2 * cols; c += blockDim.x) {
    T *base = (c < cols ? k_cache : v_cache) + hb;
    const int col = c < cols ? c : c - cols;
    for (int j = 0; j < n; ++j) {
      const int x = pp[j];
      if (x == j) continue;
      const u32x4 val = reinterpret_cast<const u32x4 *>(base + (size_t)(L + x) * D)[col];
      reinterpret_cast<u32x4 *>(base + (size_t)(L + j) * D)[col] = val;
    }
  }
}

}  // namespace

hipError_t launch_global_prune(const tg_tree &tree, int B, int B_ver, int max_path,
                               int32_t *kept, int32_t *vparent, int32_t *vtoken,
                               int32_t *position_ids, uint32_t *mask, int32_t *retrieval,
                               int32_t *n_keep, int32_t *n_leaves, uint32_t *d_err,
                               hipStream_t stream) {
  launch("global_prune", prune_kernel, dim3(B), dim3(kThreads), 0, stream, tree, B_ver,
         max_path, kept, vparent, vtoken, position_ids, mask, retrieval, n_keep, n_leaves,
         d_err);
  return hipGetLastError();
}

hipError_t launch_kv_compact(void *k_cache, void *v_cache, const int32_t *prefix_len,
                             const int32_t *path, const int32_t *n_path, int B, int Hkv,
                             int S_max, int D, int max_path, tg_dtype dtype,
                             int32_t *new_prefix_len, uint32_t *d_err, hipStream_t stream) {
  const dim3 grid((unsigned)((long long)B * Hkv)), blk(64);
  if (dtype == TG_BF16)
    launch("kv_compact", kv_compact_kernel<__bf16>, grid, blk, 0, stream,
           reinterpret_cast<__bf16 *>(k_cache), reinterpret_cast<__bf16 *>(v_cache),
           prefix_len, path, n_path, Hkv, S_max, D, max_path, new_prefix_len, d_err);
  else
    launch("kv_compact", kv_compact_kernel<float>, grid, blk, 0, stream,
           reinterpret_cast<float *>(k_cache), reinterpret_cast<float *>(v_cache), prefix_len,
           path, n_path, Hkv, S_max, D, max_path, new_prefix_len, d_err);
  return hipGetLastError();
}

}  // namespace tg
