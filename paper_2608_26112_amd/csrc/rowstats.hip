// Per-row log-sum-exp and top-K over a logits vocabulary, in chunks.
//
// Each workgroup streams one chunk of one fp32 logits row once from HBM
// (float4 loads, 16 elements in flight per thread) and produces the chunk's
// partial statistics: m = max, s = sum exp(x - m), and its top-K tokens by
// (logit desc, token asc) as 64-bit keys.  The tree-phase kernels merge the
// chunks of a row.  This is the "run the drafter, take Top_m of the
// next-token logits" step of Alg. 1 / Alg. 2 and the normaliser of the edge
// score p(u) (Sec. 3.1).
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kUnroll = 8;  // float4 loads in flight per thread (one grain)
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int KC>
struct TopList {
  uint64_t a[KC];  // descending; 0 = empty

  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int j = 0; j < KC; ++j) a[j] = 0;
  }
  __device__ __forceinline__ void insert(uint64_t k) {
    if (k <= a[KC - 1]) return;
    a[KC - 1] = k;
#pragma unroll
    for (int j = KC - 1; j > 0; --j) {
      uint64_t hi = a[j - 1], lo = a[j];
      bool sw = lo > hi;
      a[j - 1] = sw ? lo : hi;
      a[j] = sw ? hi : lo;
    }
  }
  __device__ __forceinline__ uint64_t kth(int k) const {  // a[k-1], k in [1, KC]
    uint64_t r = 0;
#pragma unroll
    for (int j = 0; j < KC; ++j) r = (j == k - 1) ? a[j] : r;
    return r;
  }
  __device__ __forceinline__ void pop() {
#pragma unroll
    for (int j = 0; j < KC - 1; ++j) a[j] = a[j + 1];
    a[KC - 1] = 0;
  }
};

__device__ __forceinline__ float key_threshold(uint64_t k) {
  uint32_t hi = (uint32_t)(k >> 32);
  return hi == 0 ? -__builtin_inff() : order_float(hi);
}

template <int KC>
__global__ __launch_bounds__(kThreads) void row_partial_kernel(
    const float *__restrict__ logits, int rows_per_batch, int V, int K,
    int chunks, int grains_per_chunk, const int32_t *__restrict__ n_live,
    const uint8_t *__restrict__ needed, float2 *__restrict__ part_ms,
    uint64_t *__restrict__ part_keys, uint32_t *d_err) {
  const int slot = blockIdx.x / chunks;
  const int c = blockIdx.x - slot * chunks;
  const int b = slot / rows_per_batch;
  const int r = slot - b * rows_per_batch;
  if (needed) {
    if (!needed[slot]) return;
  } else {
    int live = n_live ? n_live[b] : rows_per_batch;
    if (r >= live) return;
  }

  const float *row = logits + (size_t)slot * (size_t)V;
  const int n_grains = (V + kGrain - 1) / kGrain;
  const int g_beg = c * grains_per_chunk;
  const int g_end = min(n_grains, g_beg + grains_per_chunk);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), w = tid / kWave;
  // Rows are 16-byte aligned iff V % 4 == 0 (the base is); the choice depends
  // on V only, so a row's partials never depend on where it sits.
  const bool vec = (V & 3) == 0;

  float m = -__builtin_inff();
  float s = 0.0f;
  bool bad = false;
  TopList<KC> top;
  top.clear();
  uint64_t thr_key = 0;  // keys <= thr_key can never reach the row's top-K
  float thr = -__builtin_inff();

  auto consume1 = [&](float x, int idx) {
    x = clean_logit(x, bad);
    if (x > m) {
      s *= __builtin_amdgcn_exp2f((m - x) * kLog2e);
      m = x;
    }
    if (m != -__builtin_inff()) s += __builtin_amdgcn_exp2f(fmaf(x, kLog2e, -m * kLog2e));
    if (x >= thr) {
      uint64_t k = token_key(x, idx);
      if (k > thr_key) top.insert(k);
    }
  };
  auto consume4 = [&](float x0, float x1, float x2, float x3, int idx) {
    x0 = clean_logit(x0, bad);
    x1 = clean_logit(x1, bad);
    x2 = clean_logit(x2, bad);
    x3 = clean_logit(x3, bad);
    float bm = fmaxf(fmaxf(x0, x1), fmaxf(x2, x3));
    if (bm > m) {
      s *= __builtin_amdgcn_exp2f((m - bm) * kLog2e);
      m = bm;
    }
    if (m != -__builtin_inff()) {
      float ml = m * kLog2e;
      s += __builtin_amdgcn_exp2f(fmaf(x0, kLog2e, -ml)) +
           __builtin_amdgcn_exp2f(fmaf(x1, kLog2e, -ml)) +
           __builtin_amdgcn_exp2f(fmaf(x2, kLog2e, -ml)) +
           __builtin_amdgcn_exp2f(fmaf(x3, kLog2e, -ml));
    }
    if (x0 >= thr) {
      uint64_t k = token_key(x0, idx);
      if (k > thr_key) top.insert(k);
    }
    if (x1 >= thr) {
      uint64_t k = token_key(x1, idx + 1);
      if (k > thr_key) top.insert(k);
    }
    if (x2 >= thr) {
      uint64_t k = token_key(x2, idx + 2);
      if (k > thr_key) top.insert(k);
    }
    if (x3 >= thr) {
      uint64_t k = token_key(x3, idx + 3);
      if (k > thr_key) top.insert(k);
    }
  };
  auto refresh = [&]() {
    uint64_t wk = wave_max_u64(top.kth(K));
    uint64_t t = top.a[KC - 1];
    thr_key = wk > t ? wk : t;
    thr = key_threshold(thr_key);
  };

  // Each grain of kGrain elements yields one (max, sum-exp) partial over a
  // fixed set of elements in a fixed reduction order, so the merged
  // log-sum-exp of a row is the same bits whatever the chunking.  Trip counts are uniform per workgroup
  // (the threshold refresh shuffles across lanes).
  for (int gr = g_beg; gr < g_end; ++gr) {
    m = -__builtin_inff();
    s = 0.0f;
    const int e0 = gr * kGrain;
    const int e1 = min(V, e0 + kGrain);
    if (vec) {
      for (int base0 = e0; base0 < e1; base0 += 4 * kThreads * kUnroll) {
        const int base = base0 + 4 * tid;
        f32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          int idx = base + u * 4 * kThreads;
          if (idx < e1)
            v[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(row + idx));
          else
            v[u] = f32x4{-__builtin_inff(), -__builtin_inff(), -__builtin_inff(),
                         -__builtin_inff()};
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          int idx = base + u * 4 * kThreads;
          if (idx < e1) consume4(v[u].x, v[u].y, v[u].z, v[u].w, idx);
        }
        refresh();
      }
    } else {
      for (int base0 = e0; base0 < e1; base0 += kThreads * 16) {
        float xs[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          int i = base0 + tid + j * kThreads;
          xs[j] = i < e1 ? row[i] : -__builtin_inff();
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          int i = base0 + tid + j * kThreads;
          if (i < e1) consume1(xs[j], i);
        }
        refresh();
      }
    }
    // one (max, sum-exp) partial per grain: waves by a fixed shuffle tree,
    // then the four waves in order (LDS double-buffered by grain parity)
    __shared__ float gm[2][kWavesPerBlock], gs[2][kWavesPerBlock];
    const float mw = wave_max_f32(m);
    const float sc = (m == -__builtin_inff()) ? 0.0f
                                              : s * __builtin_amdgcn_exp2f((m - mw) * kLog2e);
    const float sw = wave_sum_f32(sc);
    const int par = gr & 1;
    if (lane == 0) {
      gm[par][w] = mw;
      gs[par][w] = sw;
    }
    __syncthreads();
    if (tid == 0) {
      float M = gm[par][0], S = gs[par][0];
      for (int i = 1; i < kWavesPerBlock; ++i) merge_ms(M, S, gm[par][i], gs[par][i]);
      part_ms[(size_t)slot * n_grains + gr] = make_float2(M, S);
    }
  }
  if (bad) report(d_err, TG_DERR_NONFINITE);

  // ---- wave top-K: K rounds of "largest head wins, winner pops"
  __shared__ uint64_t cand[kWavesPerBlock * TG_MAX_TOPK];
  for (int j = 0; j < K; ++j) {
    uint64_t head = top.a[0];
    uint64_t best = wave_max_u64(head);
    if (head == best && best != 0) top.pop();
    if (lane == 0) cand[w * K + j] = best;
  }
  __syncthreads();
  const size_t part = (size_t)slot * chunks + c;
  // ---- workgroup top-K by rank counting over the waves' candidates
  const int nc = kWavesPerBlock * K;
  for (int t = tid; t < nc; t += kThreads) {
    uint64_t key = cand[t];
    if (key == 0) continue;
    int rank = 0;
    for (int u = 0; u < nc; ++u) rank += cand[u] > key;
    if (rank < K) part_keys[part * K + rank] = key;
  }
  // slots past the number of real keys (chunks shorter than K) stay empty
  for (int t = tid; t < K; t += kThreads) {
    int real = 0;
    for (int u = 0; u < nc; ++u) real += cand[u] != 0;
    if (t >= real) part_keys[part * K + t] = 0;
  }

}

}  // namespace

RowPlan plan_rows(long long rows, int V) {
  // One grain per workgroup (all of it loaded in one batch), so every row is
  // spread over the chip whatever the row count; rows wider than 64 grains
  // give each workgroup several grains (the per-row merge holds one chunk
  // list per lane).
  (void)rows;
  const int n_grains = (V + kGrain - 1) / kGrain;
  const int per = (n_grains + 63) / 64;
  const int chunks = (n_grains + per - 1) / per;
  return RowPlan{chunks, per, n_grains};
}

hipError_t launch_row_partials(const float *logits, int B, int rows_per_batch,
                               int V, int K, RowPlan plan,
                               const int32_t *n_live, const uint8_t *needed,
                               float2 *part_ms, uint64_t *part_keys,
                               uint32_t *d_err, hipStream_t stream) {
  long long slots = (long long)B * rows_per_batch;
  long long grid = slots * plan.chunks;
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  dim3 g((unsigned)grid), blk(kThreads);
#define TG_ROWS(KC)                                                          \
  launch("row_partial", (row_partial_kernel<KC>), g, blk, 0, stream, logits,     \
                     rows_per_batch, V, K, plan.chunks, plan.grains_per_chunk,      \
                     n_live, needed, part_ms, part_keys, d_err)
  if (K <= 4)
    TG_ROWS(4);
  else if (K <= 8)
    TG_ROWS(8);
  else if (K <= 16)
    TG_ROWS(16);
  else if (K <= 32)
    TG_ROWS(32);
  else
    TG_ROWS(64);
#undef TG_ROWS
  return hipGetLastError();
}

}  // namespace tg
