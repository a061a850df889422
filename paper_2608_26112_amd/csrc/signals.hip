// The scheduler's pre-action tree signals and its margin predictor (App.
// B.2: the candidate tree signals and the reselection preview frontier;
// App. B.4: the margin predictor Linear(17,64)-ReLU-Linear(64,32)-ReLU-
// Linear(32,1)).
//
// One workgroup per tree, all in LDS: child counts, the frontier's depth set
// D_F and its lookback closure D_C as bitsets over depth, the candidate set R
// (root included) as node keys, ranked by counting (a sort past 1024 keys)
// for the preview Top_W(R, s), block reductions for the ten signals, then the
// 3,265-parameter MLP (weights prefetched into LDS at the start) with four
// lanes per hidden unit (fp32, fixed summation order).
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kSigs = 10;
constexpr int kCtx = 11;
constexpr int kIn = 17;
constexpr int kParams = 64 * kIn + 64 + 32 * 64 + 32 + 32 + 1;  // 3265
constexpr int kMaxKeys = 2 * TG_MAX_CAP;  // pow2 >= cap + 1 (root)

// block sums of up to four floats (fixed order: waves by shuffle tree, then
// the waves in order)
__device__ void block_sum4(float (&v)[4], float (*red)[kThreads / kWave]) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float s = wave_sum_f32(v[i]);
    if (lane == 0) red[i][w] = s;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = 0.0f;
    for (int j = 0; j < kThreads / kWave; ++j) t += red[i][j];
    v[i] = t;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void signals_kernel(
    tg_tree tree, const int32_t *__restrict__ frontier, const int32_t *__restrict__ n_frontier,
    int F, int W, int lookback, const float *__restrict__ context,
    const float *__restrict__ params, float *__restrict__ signals, float *__restrict__ margin,
    int32_t *__restrict__ action, uint32_t *d_err) {
  __shared__ uint64_t key[kMaxKeys];
  __shared__ int childcnt[TG_MAX_CAP + 1];  // [v + 1], v = -1 is the root
  __shared__ uint8_t inF[TG_MAX_CAP + 1];
  __shared__ uint32_t dF[(TG_MAX_CAP + 1 + 31) / 32], dC[(TG_MAX_CAP + 1 + 31) / 32];
  __shared__ float red[4][kThreads / kWave];
  __shared__ float x_s[kIn], h1_s[64], h2_s[32];
  __shared__ float par_s[kParams];   // the predictor's weights, prefetched
  __shared__ int dep_s[TG_MAX_CAP];
  __shared__ float cum_s[TG_MAX_CAP];
  __shared__ int bad_s;

  const int b = blockIdx.x, tid = threadIdx.x;
  const int cap = tree.cap;
  const size_t base = (size_t)b * cap;
  const int DW = (TG_MAX_CAP + 1 + 31) / 32;
  int n = tree.n_nodes[b];
  int Fb = n_frontier ? n_frontier[b] : F;
  Fb = Fb < 0 ? 0 : (Fb > F ? F : Fb);
  const bool bad_n = n < 0 || n > cap;
  if (bad_n) n = 0;
  if (tid == 0) bad_s = bad_n ? 1 : 0;
  // the weights stream into LDS while the tree is read
  if (params)
    for (int i = tid; i < kParams; i += kThreads) par_s[i] = params[i];
  for (int i = tid; i <= n; i += kThreads) {
    childcnt[i] = 0;
    inF[i] = 0;
  }
  for (int i = tid; i < DW; i += kThreads) dF[i] = dC[i] = 0;
  // node depths and scores, read once
  for (int v = tid; v < n; v += kThreads) {
    dep_s[v] = tree.depth[base + v];
    cum_s[v] = tree.cum[base + v];
  }
  __syncthreads();
  const int32_t *fr = frontier + (size_t)b * F;
  auto depth_of = [&](int v) { return v < 0 ? 0 : dep_s[v]; };
  auto cum_of = [&](int v) { return v < 0 ? 0.0f : cum_s[v]; };

  // ---- children, frontier membership, D_F, D_C
  for (int v = tid; v < n; v += kThreads) {
    int p = tree.parent[base + v];
    p = (p < -1 || p >= v) ? -1 : p;
    atomicAdd(&childcnt[p + 1], 1);
  }
  bool badf = false;
  for (int f = tid; f < Fb; f += kThreads) {
    const int v = fr[f];
    if (v < -1 || v >= n) {
      badf = true;
      continue;
    }
    inF[v + 1] = 1;
    const int d = min(max(depth_of(v), 0), TG_MAX_CAP);
    atomicOr(&dF[d >> 5], 1u << (d & 31));
    for (int x = max(0, d - lookback); x <= d; ++x) atomicOr(&dC[x >> 5], 1u << (x & 31));
  }
  if (badf) bad_s = 1;
  __syncthreads();
  const bool bad = bad_s != 0;
  auto in_set = [&](const uint32_t *bits, int d) {
    return d >= 0 && d <= TG_MAX_CAP && ((bits[d >> 5] >> (d & 31)) & 1u);
  };

  // ---- candidate set R (root included) ranked by (cum desc, depth asc, id asc)
  const int P2 = pow2_at_least(n + 1);
  float cnt_r = 0.0f;
  for (int i = tid; i < P2; i += kThreads) {
    uint64_t k = 0;
    if (i <= n) {
      const int v = i - 1;
      const int d = depth_of(v);
      if (in_set(dC, d)) {
        k = node_key(cum_of(v), d, v);
        cnt_r += 1.0f;
      }
    }
    key[i] = k;
  }
  __syncthreads();
  block_top_keys<kThreads>(key, n + 1, P2, W);

  // ---- frontier sums: depth, leaves, max depth, finite scores
  float fs[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  float mx = -__builtin_inff();
  for (int f = tid; f < Fb; f += kThreads) {
    const int v = fr[f];
    if (v < -1 || v >= n) continue;
    const float d = (float)depth_of(v);
    fs[0] += d;
    fs[1] += childcnt[v + 1] == 0 ? 1.0f : 0.0f;
    fs[2] += cum_of(v) > -__builtin_inff() ? 1.0f : 0.0f;
    mx = fmaxf(mx, d);
  }
  fs[3] = cnt_r;
  block_sum4(fs, red);
  const float nR = fs[3];
  // max depth of the frontier (block max through the same scratch)
  {
    const float m = wave_max_f32(mx);
    if ((tid & (kWave - 1)) == 0) red[0][tid / kWave] = m;
    __syncthreads();
    mx = red[0][0];
    for (int j = 1; j < kThreads / kWave; ++j) mx = fmaxf(mx, red[0][j]);
    __syncthreads();
  }
  // ---- preview frontier sums: depth, past depths, overlap, finite scores
  const int nh = min(W, (int)nR);
  float hs[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  float hscore = 0.0f, hfin = 0.0f;
  for (int i = tid; i < nh; i += kThreads) {
    const int v = node_key_id(key[i]);
    const int d = depth_of(v);
    hs[0] += (float)d;
    hs[1] += in_set(dF, d) ? 0.0f : 1.0f;
    hs[2] += inF[v + 1] ? 1.0f : 0.0f;
    const float c = cum_of(v);
    if (c > -__builtin_inff()) {
      hscore += c;
      hfin += 1.0f;
    }
  }
  hs[3] = hfin;
  block_sum4(hs, red);
  float sc[4] = {hscore, 0.0f, 0.0f, 0.0f};
  block_sum4(sc, red);

  if (tid == 0) {
    const float nan = __builtin_nanf("");
    const float nf = (float)Fb;
    const float mean_f = Fb > 0 ? fs[0] / nf : nan;
    const float mean_h = nh > 0 ? hs[0] / (float)nh : nan;
    const float delta = mean_h - mean_f;
    float s[kSigs];
    s[0] = mean_f;                                  // depth_before
    s[1] = Fb > 0 ? fs[1] / nf : nan;               // leaf_ratio_before
    s[2] = delta;                                   // pre_reselect_depth_delta
    s[3] = nR;                                      // pre_reselect_cands
    s[4] = Fb > 0 ? mx : nan;                       // max_depth_before
    s[5] = delta == delta ? fmaxf(0.0f, -delta) : nan;  // collapse_debt
    s[6] = nh > 0 ? hs[1] / (float)nh : nan;        // pre_reselect_past_ratio
    s[7] = nh > 0 ? hs[2] / (float)nh : nan;        // pre_reselect_overlap
    s[8] = hs[3] > 0.0f ? sc[0] / hs[3] : nan;      // pre_reselect_score
    s[9] = Fb > 0 ? fs[2] / nf : nan;               // finite_score_ratio_before
    if (bad) {
      for (int i = 0; i < kSigs; ++i) s[i] = nan;
      report(d_err, TG_DERR_BAD_NODE);
    }
    for (int i = 0; i < kSigs; ++i) signals[(size_t)b * kSigs + i] = s[i];
    if (params) {
      for (int i = 0; i < kCtx; ++i) x_s[i] = context[(size_t)b * kCtx + i];
      x_s[11] = s[0];  // depth_before
      x_s[12] = s[1];  // leaf_ratio_before
      x_s[13] = s[5];  // collapse_debt
      x_s[14] = s[6];  // pre_reselect_past_ratio
      x_s[15] = s[7];  // pre_reselect_overlap
      x_s[16] = s[8];  // pre_reselect_score
    }
  }
  if (!params) return;
  __syncthreads();
  // ---- margin predictor: W1[64,17] b1[64] W2[32,64] b2[32] W3[1,32] b3[1]
  // (weights from LDS; four lanes per hidden unit, partial sums in fixed
  // order, combined by lane shuffles)
  const float *W1 = par_s, *b1 = W1 + 64 * kIn, *W2 = b1 + 64, *b2 = W2 + 32 * 64;
  const float *W3 = b2 + 32, *b3 = W3 + 32;
  {
    const int u = tid >> 2, q = tid & 3;   // 64 units x 4 lanes
    float a = 0.0f;
    for (int i = q; i < kIn; i += 4) a = fmaf(W1[u * kIn + i], x_s[i], a);
    a += __shfl_xor(a, 1, kWave);
    a += __shfl_xor(a, 2, kWave);
    if (q == 0) h1_s[u] = fmaxf(a + b1[u], 0.0f);
  }
  __syncthreads();
  if (tid < 128) {
    const int u = tid >> 2, q = tid & 3;   // 32 units x 4 lanes
    float a = 0.0f;
    for (int i = q; i < 64; i += 4) a = fmaf(W2[u * 64 + i], h1_s[i], a);
    a += __shfl_xor(a, 1, kWave);
    a += __shfl_xor(a, 2, kWave);
    if (q == 0) h2_s[u] = fmaxf(a + b2[u], 0.0f);
  }
  __syncthreads();
  if (tid < kWave) {
    float y = tid < 32 ? W3[tid] * h2_s[tid] : 0.0f;
    y = wave_sum_f32(y);
    if (tid == 0) {
      y += b3[0];
      margin[b] = y;
      action[b] = y > 0.0f ? 1 : 0;
    }
  }
}

}  // namespace

hipError_t launch_signals(const tg_tree &tree, const int32_t *frontier, const int32_t *n_frontier,
                          int B, int F, int W, int lookback, const float *context,
                          const float *params, float *signals, float *margin, int32_t *action,
                          uint32_t *d_err, hipStream_t stream) {
  launch("tree_signals", signals_kernel, dim3(B), dim3(kThreads), 0, stream, tree, frontier,
         n_frontier, F, W, lookback, context, params, signals, margin, action, d_err);
  return hipGetLastError();
}

}  // namespace tg
