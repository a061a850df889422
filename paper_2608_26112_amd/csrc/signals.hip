// The scheduler's pre-action tree signals and its margin predictor (App.
// B.2: the candidate tree signals and the reselection preview frontier;
// App. B.4: the margin predictor Linear(17,64)-ReLU-Linear(64,32)-ReLU-
// Linear(32,1)).
//
// One workgroup per tree, all in LDS: every global read (tree fields, the
// frontier, the predictor's weights and context) is issued in one batch up
// front; then child counts, the frontier's depth set D_F and its lookback
// closure D_C as bitsets over depth, the candidate set R (root included) as
// node keys ranked by counting (a sort past 1024 keys) for the preview
// Top_W(R, s), and the sums: by wave 0 alone when the frontier and the
// preview fit in a wave (the other waves hand over their candidate counts),
// else one block reduction.  Wave 0 then evaluates the 3,265-parameter MLP
// alone (no block barriers), with its weights in registers (loaded with the
// first batch): a lane per hidden unit, fp32, fixed summation order.
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kSigs = 10;
constexpr int kCtx = 11;
constexpr int kIn = 17;
constexpr int kH1 = 64, kH2 = 32;
constexpr int kOffB1 = kH1 * kIn, kOffW2 = kOffB1 + kH1, kOffB2 = kOffW2 + kH2 * kH1;
constexpr int kOffW3 = kOffB2 + kH2, kOffB3 = kOffW3 + kH2;
constexpr int kParams = kOffB3 + 1;  // 3265
constexpr int kNodePer = 4;          // node fields a thread loads per batch
constexpr int kMaxKeys = 2 * TG_MAX_CAP;  // pow2 >= cap + 1 (root)
constexpr int kSums = 9;             // block sums


__global__ __launch_bounds__(kThreads) void signals_kernel(
    tg_tree tree, const int32_t *__restrict__ frontier, const int32_t *__restrict__ n_frontier,
    int F, int W, int lookback, const float *__restrict__ context,
    const float *__restrict__ params, float *__restrict__ signals, float *__restrict__ margin,
    int32_t *__restrict__ action, uint32_t *d_err) {
  __shared__ uint64_t key[kMaxKeys];
  __shared__ int childcnt[TG_MAX_CAP + 1];  // [v + 1], v = -1 is the root
  __shared__ uint8_t inF[TG_MAX_CAP + 1];
  __shared__ uint32_t dF[(TG_MAX_CAP + 1 + 31) / 32], dC[(TG_MAX_CAP + 1 + 31) / 32];
  __shared__ float red[kSums + 2][kWaves];  // sums | frontier max | preview count
  __shared__ __attribute__((aligned(16))) float x_s[kCtx + 1];
  __shared__ __attribute__((aligned(16))) float h1_s[kH1];
  __shared__ int dep_s[TG_MAX_CAP];
  __shared__ float cum_s[TG_MAX_CAP];
  __shared__ int bad_s;

  const int b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & (kWave - 1), w = tid / kWave;
  const int cap = tree.cap;
  const size_t base = (size_t)b * cap;
  const int DW = (TG_MAX_CAP + 1 + 31) / 32;
  const float ninf = -__builtin_inff();
  int n = tree.n_nodes[b];
  int Fb = n_frontier ? n_frontier[b] : F;
  Fb = Fb < 0 ? 0 : (Fb > F ? F : Fb);
  const bool bad_n = n < 0 || n > cap;
  if (bad_n) n = 0;
  const int32_t *fr = frontier + (size_t)b * F;

  // ---- one batch of global reads.  Wave 0's lanes hold the predictor's
  // weights: lane u the 17 layer-1 weights and the bias of hidden unit u;
  // lane u (half h = u / 32) the layer-2 weights of unit u % 32 on inputs
  // 32 h .. 32 h + 31, that unit's bias and its layer-3 weight.
  float w1[kIn], w2[kH1 / 2];
  float b1 = 0.0f, b2 = 0.0f, w3 = 0.0f, b3 = 0.0f;
  if (params && w == 0) {
#pragma unroll
    for (int i = 0; i < kIn; ++i) w1[i] = params[lane * kIn + i];
    b1 = params[kOffB1 + lane];
    const int u = lane & (kH2 - 1), half = lane >> 5;
#pragma unroll
    for (int i = 0; i < kH1 / 2; ++i) w2[i] = params[kOffW2 + u * kH1 + half * (kH1 / 2) + i];
    b2 = params[kOffB2 + u];
    w3 = params[kOffW3 + u];
    b3 = params[kOffB3];
  }
  float ctx = 0.0f;
  if (params && tid < kCtx) ctx = context[(size_t)b * kCtx + tid];
  int pr[kNodePer], dp[kNodePer];
  float cm[kNodePer];
#pragma unroll
  for (int j = 0; j < kNodePer; ++j) {
    const int v = tid + j * kThreads;
    pr[j] = v < n ? tree.parent[base + v] : -1;
    dp[j] = v < n ? tree.depth[base + v] : 0;
    cm[j] = v < n ? tree.cum[base + v] : 0.0f;
  }
  const int fv = tid < Fb ? fr[tid] : 0;
  // ---- LDS set-up (no dependence on the reads)
  if (tid == 0) bad_s = bad_n ? 1 : 0;
  for (int i = tid; i <= n; i += kThreads) {
    childcnt[i] = 0;
    inF[i] = 0;
  }
  for (int i = tid; i < DW; i += kThreads) dF[i] = dC[i] = 0;
  if (params && tid < kCtx) x_s[tid] = ctx;
#pragma unroll
  for (int j = 0; j < kNodePer; ++j) {
    const int v = tid + j * kThreads;
    if (v < n) {
      dep_s[v] = dp[j];
      cum_s[v] = cm[j];
    }
  }
  for (int v = tid + kNodePer * kThreads; v < n; v += kThreads) {  // trees past 1024 nodes
    dep_s[v] = tree.depth[base + v];
    cum_s[v] = tree.cum[base + v];
  }
  __syncthreads();
  auto depth_of = [&](int v) { return v < 0 ? 0 : dep_s[v]; };
  auto cum_of = [&](int v) { return v < 0 ? 0.0f : cum_s[v]; };

  // ---- children, frontier membership, D_F, D_C
  auto count_child = [&](int p, int v) {
    p = (p < -1 || p >= v) ? -1 : p;
    atomicAdd(&childcnt[p + 1], 1);
  };
#pragma unroll
  for (int j = 0; j < kNodePer; ++j) {
    const int v = tid + j * kThreads;
    if (v < n) count_child(pr[j], v);
  }
  for (int v = tid + kNodePer * kThreads; v < n; v += kThreads)
    count_child(tree.parent[base + v], v);
  bool badf = false;
  for (int f = tid; f < Fb; f += kThreads) {
    const int v = f == tid ? fv : fr[f];
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
  float sums[kSums] = {};   // |R|, frontier: depth, leaves, finite; preview:
                            // depth, past depths, overlap, finite, score
  for (int i = tid; i < P2; i += kThreads) {
    uint64_t k = 0;
    if (i <= n) {
      const int v = i - 1;
      const int d = depth_of(v);
      if (in_set(dC, d)) {
        k = node_key(cum_of(v), d, v);
        sums[0] += 1.0f;
      }
    }
    key[i] = k;
  }
  // frontier sums (before the ranking's barriers: they need no keys)
  float mx = ninf;
  for (int f = tid; f < Fb; f += kThreads) {
    const int v = f == tid ? fv : fr[f];
    if (v < -1 || v >= n) continue;
    const float d = (float)depth_of(v);
    sums[1] += d;
    sums[2] += childcnt[v + 1] == 0 ? 1.0f : 0.0f;
    sums[3] += cum_of(v) > ninf ? 1.0f : 0.0f;
    mx = fmaxf(mx, d);
  }
  // With at most a wave's width of frontier and preview slots (the usual
  // case) every sum but the candidate count comes from wave 0 alone, which
  // then finishes the call: the other waves hand over their counts and leave
  // after the ranking.
  const bool one_wave = F <= kWave && W <= kWave;
  if (one_wave) {
    const float c0 = wave_sum_f32(sums[0]);
    if (lane == 0) red[0][w] = c0;
  }
  __syncthreads();
  block_top_keys<kThreads>(key, n + 1, P2, W);
  if (one_wave && w != 0) return;

  // ---- preview frontier: the present keys among the first W
  float nh_f = 0.0f;
  for (int i = tid; i < W && i <= n; i += kThreads) {
    const uint64_t k = key[i];
    if (k == 0) continue;
    const int v = node_key_id(k);
    const int d = depth_of(v);
    nh_f += 1.0f;
    sums[4] += (float)d;
    sums[5] += in_set(dF, d) ? 0.0f : 1.0f;
    sums[6] += inF[v + 1] ? 1.0f : 0.0f;
    const float c = cum_of(v);
    if (c > ninf) {
      sums[7] += 1.0f;
      sums[8] += c;
    }
  }
  // ---- totals, the same in every lane of wave 0: waves by a DPP tree, then
  // the waves in order
  float t[kSums], fmx;
  int nh;
  if (one_wave) {
    t[0] = red[0][0];
    for (int j = 1; j < kWaves; ++j) t[0] += red[0][j];
    // a lane holds at most one frontier and one preview slot, so the six
    // counts are 0 or 1 per lane and at most 64 in total: a byte each in two
    // integer sums (the same totals as float sums of the counts)
    const int ca = (int)sums[2] | ((int)sums[3] << 8) | ((int)sums[5] << 16) | ((int)sums[6] << 24);
    const int cb = (int)sums[7] | ((int)nh_f << 8);
    const int ta = wave_sum_i32(ca), tb = wave_sum_i32(cb);
    t[1] = wave_sum_f32(sums[1]);
    t[4] = wave_sum_f32(sums[4]);
    t[8] = wave_sum_f32(sums[8]);
    t[2] = (float)(ta & 255);
    t[3] = (float)((ta >> 8) & 255);
    t[5] = (float)((ta >> 16) & 255);
    t[6] = (float)((ta >> 24) & 255);
    t[7] = (float)(tb & 255);
    nh = (tb >> 8) & 255;
    fmx = wave_max_f32(mx);
  } else {
#pragma unroll
    for (int i = 0; i < kSums; ++i) {
      const float r = wave_sum_f32(sums[i]);
      if (lane == 0) red[i][w] = r;
    }
    {
      const float r = wave_max_f32(mx);
      if (lane == 0) red[kSums][w] = r;
    }
    {
      const float r = wave_sum_f32(nh_f);
      if (lane == 0) red[kSums + 1][w] = r;
    }
    __syncthreads();
    if (w != 0) return;
    for (int i = 0; i < kSums; ++i) {
      t[i] = red[i][0];
      for (int j = 1; j < kWaves; ++j) t[i] += red[i][j];
    }
    fmx = red[kSums][0];
    for (int j = 1; j < kWaves; ++j) fmx = fmaxf(fmx, red[kSums][j]);
    nh = 0;
    for (int j = 0; j < kWaves; ++j) nh += (int)red[kSums + 1][j];
  }
  const float nan = __builtin_nanf("");
  const float nf = (float)Fb;
  const float mean_f = Fb > 0 ? t[1] / nf : nan;
  const float mean_h = nh > 0 ? t[4] / (float)nh : nan;
  const float delta = mean_h - mean_f;
  float sg[kSigs];
  sg[0] = mean_f;                                  // depth_before
  sg[1] = Fb > 0 ? t[2] / nf : nan;                // leaf_ratio_before
  sg[2] = delta;                                   // pre_reselect_depth_delta
  sg[3] = t[0];                                    // pre_reselect_cands
  sg[4] = Fb > 0 ? fmx : nan;                      // max_depth_before
  sg[5] = delta == delta ? fmaxf(0.0f, -delta) : nan;  // collapse_debt
  sg[6] = nh > 0 ? t[5] / (float)nh : nan;         // pre_reselect_past_ratio
  sg[7] = nh > 0 ? t[6] / (float)nh : nan;         // pre_reselect_overlap
  sg[8] = t[7] > 0.0f ? t[8] / t[7] : nan;         // pre_reselect_score
  sg[9] = Fb > 0 ? t[3] / nf : nan;                // finite_score_ratio_before
  if (bad) {
#pragma unroll
    for (int i = 0; i < kSigs; ++i) sg[i] = nan;
    if (lane == 0) report(d_err, TG_DERR_BAD_NODE);
  }
  {
    float mine = sg[0];
#pragma unroll
    for (int i = 1; i < kSigs; ++i) mine = lane == i ? sg[i] : mine;
    if (lane < kSigs) signals[(size_t)b * kSigs + lane] = mine;
  }
  if (!params) return;
  // ---- margin predictor: W1[64,17] b1[64] W2[32,64] b2[32] W3[1,32] b3[1];
  // inputs: the context, then depth_before, leaf_ratio_before, collapse_debt,
  // pre_reselect_past_ratio, pre_reselect_overlap, pre_reselect_score
  float xin[kIn];
#pragma unroll
  for (int i = 0; i < kCtx; ++i) xin[i] = x_s[i];
  xin[11] = sg[0];
  xin[12] = sg[1];
  xin[13] = sg[5];
  xin[14] = sg[6];
  xin[15] = sg[7];
  xin[16] = sg[8];
  // layer 1: lane u is unit u
  {
    float a = 0.0f;
#pragma unroll
    for (int i = 0; i < kIn; ++i) a = fmaf(w1[i], xin[i], a);
    h1_s[lane] = fmaxf(a + b1, 0.0f);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // layer 2: lane u < 32 and lane u + 32 take unit u's inputs 0..31 and
  // 32..63, added in that order
  const int u = lane & (kH2 - 1), half = lane >> 5;
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < kH1 / 2; ++i) a = fmaf(w2[i], h1_s[half * (kH1 / 2) + i], a);
  const float hi_half = __shfl_down(a, 32, kWave);
  const float h2 = fmaxf((a + hi_half) + b2, 0.0f);
  // layer 3
  const float y = wave_sum_f32(lane < kH2 ? w3 * h2 : 0.0f) + b3;
  if (lane == 0) {
    margin[b] = y;
    action[b] = y > 0.0f ? 1 : 0;
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
