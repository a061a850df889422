// Greedy acceptance (temperature 0): the deepest draft node whose whole
// root path agrees with the target's arg-max tokens (Sec. 3.2,
// "Distribution preservation"; App. E sets temperature 0).
//
// One workgroup per tree.  match[i] = (token[i] == greedy[parent[i] + 1]);
// a node is acceptable iff match holds on its whole path.  Both "all of the
// path matches" and the depth are computed by pointer jumping over the parent
// links in LDS (log2(n) rounds), so adversarial chains cost O(n log n), not
// O(n * depth).  The winner is the block-wide maximum of (depth, -id).
//
// argmax_rows_kernel: the target's greedy tokens straight from its logits,
// for the accept-from-logits entry point.
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void accept_kernel(
    const int32_t *__restrict__ parent, const int32_t *__restrict__ token,
    const int32_t *__restrict__ n_nodes, const int32_t *__restrict__ greedy,
    int cap, int max_depth, int32_t *__restrict__ accept_len,
    int32_t *__restrict__ accept_path, int32_t *__restrict__ bonus,
    uint32_t *d_err) {
  __shared__ int16_t anc[2][TG_MAX_CAP];
  __shared__ int16_t dep[2][TG_MAX_CAP];
  __shared__ uint8_t ok[2][TG_MAX_CAP];
  __shared__ int16_t par[TG_MAX_CAP];
  __shared__ unsigned long long best_s;

  const int b = blockIdx.x, tid = threadIdx.x;
  int n = n_nodes[b];
  if (n < 0 || n > cap) {
    if (tid == 0) report(d_err, TG_DERR_BAD_NODE);
    n = 0;
  }
  const size_t base = (size_t)b * cap;
  const int32_t *g = greedy + (size_t)b * (cap + 1);

  bool badp = false;
  for (int i = tid; i < n; i += kThreads) {
    int p = parent[base + i];
    if (p < -1 || p >= i) {
      badp = true;
      p = -1;
    }
    par[i] = (int16_t)p;
    anc[0][i] = (int16_t)p;
    dep[0][i] = 1;
    ok[0][i] = token[base + i] == g[p + 1];
  }
  if (tid == 0) best_s = 0;
  if (badp) report(d_err, TG_DERR_BAD_PARENT);
  __syncthreads();

  // pointer jumping: after round t, anc[i] is the 2^t-th ancestor (or -1),
  // dep[i] counts the nodes on the segment [i, anc[i]), ok[i] ANDs match there
  int cur = 0;
  for (int span = 1; span < n; span <<= 1) {
    const int nxt = cur ^ 1;
    for (int i = tid; i < n; i += kThreads) {
      int a = anc[cur][i];
      if (a >= 0) {
        anc[nxt][i] = anc[cur][a];
        dep[nxt][i] = dep[cur][i] + dep[cur][a];
        ok[nxt][i] = ok[cur][i] & ok[cur][a];
      } else {
        anc[nxt][i] = -1;
        dep[nxt][i] = dep[cur][i];
        ok[nxt][i] = ok[cur][i];
      }
    }
    cur = nxt;
    __syncthreads();
  }

  // deepest acceptable node within max_depth, ties to the smallest id
  unsigned long long mine = 0;
  bool too_deep = false;
  for (int i = tid; i < n; i += kThreads) {
    if (!ok[cur][i]) continue;
    int d = dep[cur][i];
    if (d > max_depth) {
      too_deep = true;
      continue;
    }
    unsigned long long k = ((unsigned long long)d << 32) | (unsigned)(0xffffu - i);
    mine = k > mine ? k : mine;
  }
  if (too_deep) report(d_err, TG_DERR_CAPACITY);
  mine = wave_max_u64(mine);
  if ((tid & (kWave - 1)) == 0 && mine) atomicMax(&best_s, mine);
  __syncthreads();

  const unsigned long long best = best_s;
  const int A = (int)(best >> 32);
  const int vbest = best ? (int)(0xffffu - (unsigned)(best & 0xffffu)) : -1;
  int32_t *path = accept_path + (size_t)b * max_depth;
  for (int d = A + tid; d < max_depth; d += kThreads) path[d] = -1;
  if (tid == 0) {
    int u = vbest;
    for (int d = A - 1; d >= 0; --d) {
      path[d] = u;
      u = par[u];
    }
    accept_len[b] = A;
    bonus[b] = g[vbest + 1];
  }
}

// The target's greedy token of every row a tree uses (temperature 0):
// greedy[b, r] = arg-max of logits[b, r] for r <= n_nodes[b] (ties to the
// smallest token: the max of (logit, -token) keys; NaN and +inf read as
// -inf), -1 for the other rows.  One workgroup per (tree, row) of the
// greedy array; rows past the logits (r >= R) are -1 and raise BAD_NODE
// when the tree needs them.
__global__ __launch_bounds__(kThreads) void argmax_rows_kernel(
    const float *__restrict__ logits, const int32_t *__restrict__ n_nodes, int cap, int R,
    int V, int32_t *__restrict__ greedy, uint32_t *d_err) {
  __shared__ uint64_t red[kThreads / kWave];
  const int rows = cap + 1;
  const int b = blockIdx.x / rows, r = blockIdx.x - b * rows;
  const int tid = threadIdx.x;
  int nb = n_nodes[b];
  nb = nb < 0 ? 0 : (nb > cap ? cap : nb);
  int32_t *out = greedy + (size_t)b * rows + r;
  if (r > nb || r >= R) {
    if (tid == 0) {
      *out = -1;
      if (r <= nb) report(d_err, TG_DERR_BAD_NODE);
    }
    return;
  }
  const float *x = logits + ((size_t)b * R + r) * V;
  uint64_t best = 0;
  bool bad = false;
  if ((V & 3) == 0) {
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    for (int i = tid; i < V / 4; i += kThreads) {
      const float4 q = x4[i];
      const uint32_t t0 = 4u * (uint32_t)i;
      uint64_t k = token_key(clean_logit(q.x, bad), t0);
      k = max(k, token_key(clean_logit(q.y, bad), t0 + 1));
      k = max(k, token_key(clean_logit(q.z, bad), t0 + 2));
      k = max(k, token_key(clean_logit(q.w, bad), t0 + 3));
      best = max(best, k);
    }
  } else {
    for (int i = tid; i < V; i += kThreads)
      best = max(best, token_key(clean_logit(x[i], bad), (uint32_t)i));
  }
  if (bad) report(d_err, TG_DERR_NONFINITE);
  best = wave_max_u64(best);
  if ((tid & (kWave - 1)) == 0) red[tid / kWave] = best;
  __syncthreads();
  if (tid == 0) {
    for (int i = 1; i < kThreads / kWave; ++i) best = max(best, red[i]);
    best = max(best, red[0]);
    *out = (int32_t)key_token(best);
  }
}

}  // namespace

hipError_t launch_argmax_rows(const float *logits, const int32_t *n_nodes, int B, int cap,
                              int R, int V, int32_t *greedy, uint32_t *d_err,
                              hipStream_t stream) {
  launch("argmax_rows", argmax_rows_kernel, dim3((unsigned)((long long)B * (cap + 1))),
         dim3(kThreads), 0, stream, logits, n_nodes, cap, R, V, greedy, d_err);
  return hipGetLastError();
}

hipError_t launch_accept(const int32_t *parent, const int32_t *token,
                         const int32_t *n_nodes, const int32_t *greedy, int B,
                         int cap, int max_depth, int32_t *accept_len,
                         int32_t *accept_path, int32_t *bonus, uint32_t *d_err,
                         hipStream_t stream) {
  launch("accept", accept_kernel, dim3(B), dim3(kThreads), 0, stream, parent,
                     token, n_nodes, greedy, cap, max_depth, accept_len,
                     accept_path, bonus, d_err);
  return hipGetLastError();
}

}  // namespace tg
