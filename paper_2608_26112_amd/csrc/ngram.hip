// The n-gram small drafter (App. C.1, the small drafter's implementation):
// a prefill cache of the target's top-m next tokens per context
// position, and the small-step expansion that matches each frontier node's
// prefix suffix against the context (longest n-gram first, shorter on a miss,
// the most frequent context token's position as the last resort) and grows
// the node's children from the matched position's cache row.
//
// ngram_cache_kernel: one wave per context position; the position's logits
//   row was already reduced by row_partial_kernel (lse partials and top-m
//   chunk lists), the wave merges them: cand_logp = fl(x - lse).
// ngram_fallback_kernel: one workgroup per sequence; token counts by global
//   atomics into a zeroed [V] slice, then the (count desc, token asc) best
//   token and its last position, both as block maxima of packed keys.
// ngram_expand_kernel: one workgroup per tree.  The prompt is staged in LDS
//   (up to 4096 tokens) and every frontier node's suffix built at once; then
//   for each node the block scans the prompt: end position j scores the
//   length l(j) of the longest common suffix of x[..j] and the node's prefix
//   (capped at n_max), and the maximum of (l, j) with l >= 1 is the latest
//   longest match: the longest n-gram that occurs, shorter ones only when no
//   longer one does, at its latest occurrence.  Children take ids n_b + f*K + k, then
//   Top_N of them by (cum desc, depth asc, id asc).
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

__global__ __launch_bounds__(kThreads) void ngram_cache_kernel(
    long long rows, int m, int chunks, int n_ms, const float2 *__restrict__ part_ms,
    const uint64_t *__restrict__ part_keys, int32_t *__restrict__ cand_tok,
    float *__restrict__ cand_logp) {
  extern __shared__ uint64_t wsmem[];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const long long r = (long long)blockIdx.x * kWaves + w;
  if (r >= rows) return;  // wave-uniform
  const float2 *ms = part_ms + r * n_ms;
  const float lse = wave_fold_lse(
      ms, n_ms, lane < n_ms ? ms[lane] : make_float2(-__builtin_inff(), 0.0f));
  const uint64_t key =
      wave_finish_topk(part_keys + r * chunks * m, chunks, m, wsmem + (size_t)w * chunks * m);
  if (lane < m) {
    cand_tok[r * m + lane] = (int32_t)key_token(key);
    cand_logp[r * m + lane] = edge_logp(key_logit(key), lse);
  }
}

__device__ uint64_t block_max_u64(uint64_t v, uint64_t *red) {
  v = wave_max_u64(v);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  uint64_t r = red[0];
  for (int i = 1; i < kWaves; ++i) r = red[i] > r ? red[i] : r;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void ngram_fallback_kernel(
    const int32_t *__restrict__ context, const int32_t *__restrict__ ctx_len, int L, int V,
    int32_t *__restrict__ counts, int32_t *__restrict__ fallback_pos, uint32_t *d_err) {
  __shared__ uint64_t red[kWaves];
  const int b = blockIdx.x, tid = threadIdx.x;
  int n = ctx_len[b];
  n = n < 0 ? 0 : (n > L ? L : n);
  int32_t *cnt = counts + (size_t)b * V;
  const int32_t *ctx = context + (size_t)b * L;
  for (int t = tid; t < V; t += kThreads) cnt[t] = 0;
  __syncthreads();
  bool bad = false;
  for (int i = tid; i < n; i += kThreads) {
    const int t = ctx[i];
    if (t < 0 || t >= V) bad = true;
    else atomicAdd(cnt + t, 1);
  }
  if (bad) report(d_err, TG_DERR_BAD_NODE);
  __syncthreads();
  // best token: count desc, token asc
  uint64_t best = 0;
  for (int t = tid; t < V; t += kThreads) {
    const uint32_t c = (uint32_t)cnt[t];
    if (c == 0) continue;
    const uint64_t k = ((uint64_t)c << 32) | (uint64_t)(0xffffffffu - (uint32_t)t);
    best = k > best ? k : best;
  }
  best = block_max_u64(best, red);
  const int tok = best ? (int)(0xffffffffu - (uint32_t)best) : -1;
  // its last position
  uint64_t last = 0;
  for (int i = tid; i < n; i += kThreads)
    if (ctx[i] == tok) last = (uint64_t)(i + 1) > last ? (uint64_t)(i + 1) : last;
  last = block_max_u64(last, red);
  if (tid == 0) fallback_pos[b] = (int32_t)last - 1;
}

constexpr int kCtxLds = 4096;             // prompts up to this many tokens are scanned from LDS
constexpr int kCtxPer = kCtxLds / kThreads;  // prompt tokens a thread holds in registers
constexpr int kTreeLds = 1024;            // nodes whose fields are staged in LDS
constexpr int kTreePer = kTreeLds / kThreads;

// 64-bit words of the region the suffixes and then the child keys share.
__host__ __device__ inline int ngram_region_words(int F, int K, int n_max) {
  const int keys = pow2_at_least(F * K > 0 ? F * K : 1);
  const int sufw = (F * n_max + 1) / 2;
  return keys > sufw ? keys : sufw;
}

// One workgroup per tree.  Every global read the step can issue up front is
// issued in one batch (bounded by the array sizes; the live sizes mask the
// values afterwards): the prompt's first kCtxLds tokens (kept in registers
// for the scan and copied to LDS for the match extension), the fields of the
// first kTreeLds nodes, the frontier (kept in LDS).
__global__ __launch_bounds__(kThreads) void ngram_expand_kernel(
    tg_tree tree, const int32_t *__restrict__ frontier, const int32_t *__restrict__ n_frontier,
    int F, const int32_t *__restrict__ context, const int32_t *__restrict__ ctx_len, int L,
    const int32_t *__restrict__ cand_tok, const float *__restrict__ cand_logp,
    const int32_t *__restrict__ fallback_pos, int m, int K, int N, int n_max,
    int32_t *__restrict__ match_pos, int32_t *__restrict__ next_frontier,
    int32_t *__restrict__ n_next, uint32_t *d_err) {
  // dynamic LDS: one region holding first the suffixes [F * n_max] int32,
  // then (once the matching is done) the child keys [pow2(F*K)] u64 | best
  // [F] u64 | plen [F] | frontier [F]
  extern __shared__ uint64_t skey[];
  __shared__ int32_t ctx_s[kCtxLds];
  __shared__ int32_t par_s[kTreeLds], tok_s[kTreeLds], dep_s[kTreeLds];
  __shared__ float cum_s[kTreeLds];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1);
  const int cap = tree.cap;
  const size_t base = (size_t)b * cap;
  int Fb = n_frontier ? n_frontier[b] : F;
  Fb = Fb < 0 ? 0 : (Fb > F ? F : Fb);
  const int nb = tree.n_nodes[b];
  const int Lb = ctx_len[b];
  const int total = Fb * K;
  const int P2 = pow2_at_least(F * K > 0 ? F * K : 1);
  int32_t *suf = reinterpret_cast<int32_t *>(skey);
  uint64_t *best = skey + ngram_region_words(F, K, n_max);
  int32_t *plen = reinterpret_cast<int32_t *>(best + F);
  int32_t *fr_s = plen + F;
  const int32_t *ctx_g = context + (size_t)b * L;
  const int32_t *fr = frontier + (size_t)b * F;

  // ---- one batch of reads
  const int Lr = min(L, kCtxLds), nt = min(cap, kTreeLds);
  int32_t cr[kCtxPer];
#pragma unroll
  for (int i = 0; i < kCtxPer; ++i) {
    const int j = tid + i * kThreads;
    cr[i] = j < Lr ? ctx_g[j] : 0;
  }
  int32_t tp[kTreePer], tt[kTreePer], td[kTreePer];
  float tc[kTreePer];
#pragma unroll
  for (int i = 0; i < kTreePer; ++i) {
    const int v = tid + i * kThreads;
    tp[i] = v < nt ? tree.parent[base + v] : -1;
    tt[i] = v < nt ? tree.token[base + v] : 0;
    td[i] = v < nt ? tree.depth[base + v] : 0;
    tc[i] = v < nt ? tree.cum[base + v] : 0.0f;
  }
  const int fv = tid < F ? fr[tid] : 0;  // before the frontier's live size arrives
  bool bad = nb < 0 || nb > cap;
  for (int f = tid; f < Fb; f += kThreads) {
    const int v = f == tid ? fv : fr[f];
    fr_s[f] = v;
    bad |= v < -1 || v >= nb;
  }
#pragma unroll
  for (int i = 0; i < kCtxPer; ++i) {
    const int j = tid + i * kThreads;
    if (j < Lr) ctx_s[j] = cr[i];
  }
#pragma unroll
  for (int i = 0; i < kTreePer; ++i) {
    const int v = tid + i * kThreads;
    if (v < nt) {
      par_s[v] = tp[i];
      tok_s[v] = tt[i];
      dep_s[v] = td[i];
      cum_s[v] = tc[i];
    }
  }
  bad = __syncthreads_or(bad);
  const bool no_ctx = !bad && (Lb <= 0 || Lb > L);
  const bool full = !bad && !no_ctx && nb + total > cap;
  if (match_pos)
    for (int f = tid; f < F; f += kThreads) match_pos[(size_t)b * F + f] = -1;
  if (bad || no_ctx || full) {
    if (tid == 0) {
      report(d_err, bad ? TG_DERR_BAD_NODE : (no_ctx ? TG_DERR_BAD_PREFIX : TG_DERR_CAPACITY));
      n_next[b] = 0;
    }
    for (int j = tid; j < N; j += kThreads) next_frontier[(size_t)b * N + j] = TG_NO_NODE;
    return;
  }
  int fb = fallback_pos[b];
  if (fb < 0 || fb >= Lb) {
    if (tid == 0) report(d_err, TG_DERR_BAD_NODE);
    fb = Lb - 1;
  }
  const bool in_lds = Lb <= kCtxLds;
  auto tok_of = [&](int u) { return u < nt ? tok_s[u] : tree.token[base + u]; };
  auto par_of = [&](int u) { return u < nt ? par_s[u] : tree.parent[base + u]; };
  auto ctx_at = [&](int i) { return in_lds ? ctx_s[i] : ctx_g[i]; };

  // ---- every frontier node's suffix: the prefix's last n_max tokens, newest
  // first (the node's path, then the prompt's tail)
  for (int f = tid; f < Fb; f += kThreads) {
    int32_t *sf = suf + f * n_max;
    int k = 0;
    for (int u = fr_s[f]; u >= 0 && k < n_max; ++k) {
      sf[k] = tok_of(u);
      const int p = par_of(u);
      u = (p < -1 || p >= u) ? -1 : p;
    }
    for (int i = Lb - 1; i >= 0 && k < n_max; --i, ++k) sf[k] = ctx_at(i);
    plen[f] = k;
    best[f] = 0;
  }
  __syncthreads();

  // ---- latest longest match of every node.  The first token decides almost
  // every position: a thread compares its prompt tokens (registers) for every
  // node, then extends all of its hits together, one suffix token per round
  // (one LDS round trip for every hit of the thread), until no hit of the
  // wave extends.  Key (length, position), larger is better.
  if (in_lds) {
    for (int f = 0; f < Fb; ++f) {
      const int32_t *sf = suf + f * n_max;
      const int pl = plen[f];
      const int32_t s0 = sf[0];
      int len[kCtxPer];  // matched length at position tid + i * kThreads, 0 = no hit
      bool hit = false;
#pragma unroll
      for (int i = 0; i < kCtxPer; ++i) {
        const int j = tid + i * kThreads;
        len[i] = j < Lb && cr[i] == s0 ? 1 : 0;
        hit |= len[i] != 0;
      }
      if (!__any(hit)) continue;
      for (int l = 1; l < pl; ++l) {
        const int32_t want = sf[l];
        bool ext = false;
#pragma unroll
        for (int i = 0; i < kCtxPer; ++i) {
          const int j = tid + i * kThreads;
          if (len[i] == l && j >= l && ctx_s[j - l] == want) {
            len[i] = l + 1;
            ext = true;
          }
        }
        if (!__any(ext)) break;
      }
      uint32_t mine = 0;  // length << 27 | position (positions < kCtxLds)
#pragma unroll
      for (int i = 0; i < kCtxPer; ++i) {
        const uint32_t key = ((uint32_t)len[i] << 27) | (uint32_t)(tid + i * kThreads);
        mine = len[i] != 0 && key > mine ? key : mine;
      }
      mine = wave_max_u32(mine);
      if (lane == 0 && mine)
        atomicMax(reinterpret_cast<unsigned long long *>(best + f),
                  ((unsigned long long)(mine >> 27) << 32) | (mine & 0x7ffffffu));
    }
  } else {
    for (int f = 0; f < Fb; ++f) {
      const int32_t *sf = suf + f * n_max;
      const int pl = plen[f];
      const int s0 = sf[0];
      uint64_t mine = 0;
      for (int j = tid; j < Lb; j += kThreads) {
        if (ctx_g[j] != s0) continue;
        int l = 1;
        const int lim = min(pl, j + 1);
        while (l < lim && ctx_g[j - l] == sf[l]) ++l;
        const uint64_t key = ((uint64_t)l << 32) | (uint64_t)j;
        mine = key > mine ? key : mine;
      }
      mine = wave_max_u64(mine);
      if (lane == 0 && mine)
        atomicMax(reinterpret_cast<unsigned long long *>(best + f), (unsigned long long)mine);
    }
  }
  __syncthreads();
  for (int f = tid; f < Fb; f += kThreads) {
    const int pos = best[f] ? (int)(uint32_t)best[f] : fb;
    plen[f] = pos;  // reused: the matched position
    if (match_pos) match_pos[(size_t)b * F + f] = pos;
  }
  __syncthreads();

  // ---- children from the cache rows, then Top_N
  for (int c = tid; c < P2; c += kThreads) {
    if (c >= total) {
      skey[c] = 0;
      continue;
    }
    const int f = c / K, k = c - f * K;
    const int v = fr_s[f];
    const size_t row = ((size_t)b * L + plen[f]) * m + k;
    const float cv = v < 0 ? 0.0f : (v < nt ? cum_s[v] : tree.cum[base + v]);
    const int dv = v < 0 ? 0 : (v < nt ? dep_s[v] : tree.depth[base + v]);
    const float lp = cand_logp[row];
    const float cum = __fadd_rn(cv, lp);
    const int id = nb + c;
    tree.parent[base + id] = v;
    tree.token[base + id] = cand_tok[row];
    tree.depth[base + id] = dv + 1;
    tree.logp[base + id] = lp;
    tree.cum[base + id] = cum;
    tree.visited[base + id] = 0;
    skey[c] = node_key(cum, dv + 1, id);
  }
  __syncthreads();
  const int nn = min(N, total);
  block_top_keys<kThreads>(skey, total, pow2_at_least(total > 0 ? total : 1), nn);
  for (int j = tid; j < N; j += kThreads)
    next_frontier[(size_t)b * N + j] = j < nn ? node_key_id(skey[j]) : TG_NO_NODE;
  if (tid == 0) {
    n_next[b] = nn;
    tree.n_nodes[b] = nb + total;
  }
}

}  // namespace

hipError_t launch_ngram_cache(long long rows, int m, RowPlan plan, const float2 *part_ms,
                              const uint64_t *part_keys, int32_t *cand_tok, float *cand_logp,
                              hipStream_t stream) {
  const size_t lds = (size_t)kWaves * plan.chunks * m * sizeof(uint64_t);
  hipError_t e = hipFuncSetAttribute((const void *)ngram_cache_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const long long grid = (rows + kWaves - 1) / kWaves;
  launch("ngram_cache", ngram_cache_kernel, dim3((unsigned)grid), dim3(kThreads), lds, stream,
         rows, m, plan.chunks, plan.ms_per_row, part_ms, part_keys, cand_tok, cand_logp);
  return hipGetLastError();
}

hipError_t launch_ngram_fallback(const int32_t *context, const int32_t *ctx_len, int B, int L,
                                 int V, int32_t *counts, int32_t *fallback_pos, uint32_t *d_err,
                                 hipStream_t stream) {
  launch("ngram_fallback", ngram_fallback_kernel, dim3(B), dim3(kThreads), 0, stream, context,
         ctx_len, L, V, counts, fallback_pos, d_err);
  return hipGetLastError();
}

hipError_t launch_ngram_expand(const tg_tree &tree, const int32_t *frontier,
                               const int32_t *n_frontier, int B, int F,
                               const int32_t *context, const int32_t *ctx_len, int L,
                               const int32_t *cand_tok, const float *cand_logp,
                               const int32_t *fallback_pos, int m, int K, int N, int n_max,
                               int32_t *match_pos, int32_t *next_frontier, int32_t *n_next,
                               uint32_t *d_err, hipStream_t stream) {
  const size_t lds = ((size_t)ngram_region_words(F, K, n_max) + F) * sizeof(uint64_t) +
                    (size_t)F * 2 * sizeof(int32_t);
  hipError_t e = hipFuncSetAttribute((const void *)ngram_expand_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  launch("ngram_expand", ngram_expand_kernel, dim3(B), dim3(kThreads), lds, stream, tree,
         frontier, n_frontier, F, context, ctx_len, L, cand_tok, cand_logp, fallback_pos, m, K,
         N, n_max, match_pos, next_frontier, n_next, d_err);
  return hipGetLastError();
}

}  // namespace tg
