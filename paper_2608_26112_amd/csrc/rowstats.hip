// Per-row log-sum-exp and top-K over a logits vocabulary, in chunks.
//
// Each workgroup streams one chunk of one fp32 logits row once from HBM
// (a grain of 8192 values at a time, 32 per thread in one batch of float4
// loads) and produces the chunk's partial statistics: m = max,
// s = sum exp(x - m), and its top-K tokens by (logit desc, token asc) as
// 64-bit keys.  The tree-phase kernels merge the chunks of a row.  Top-m
// selection over a drafter's next-token distribution is the expansion step
// of Alg. 1 / Alg. 2; the log-sum-exp normalises the edge score p(u)
// (Sec. 3.1).
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kPer = kGrain / kThreads;  // elements per thread per grain (32)
constexpr int kCandCap = 256;            // candidates per grain on the fast path
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Logit of a running-list key; -inf for an empty slot.
__device__ __forceinline__ float key_threshold(uint64_t k) {
  uint32_t hi = (uint32_t)(k >> 32);
  return hi == 0 ? -__builtin_inff() : order_float(hi);
}

// Token of a thread's j-th element in the grain starting at e0.  16-byte rows
// use float4 columns (four consecutive tokens per thread, 1024 tokens per
// load step); other rows use one token per thread per step.
__device__ __forceinline__ int elem_token(bool vec, int e0, int tid, int j) {
  return vec ? e0 + (j >> 2) * (4 * kThreads) + 4 * tid + (j & 3) : e0 + j * kThreads + tid;
}

__device__ __forceinline__ float lane_max(const float (&x)[kPer]) {
  float a = fmaxf(x[0], x[1]), b = fmaxf(x[2], x[3]);
#pragma unroll
  for (int j = 4; j < kPer; j += 4) {
    a = fmaxf(a, fmaxf(x[j], x[j + 1]));
    b = fmaxf(b, fmaxf(x[j + 2], x[j + 3]));
  }
  return fmaxf(a, b);
}

// sum_j exp(x_j - m) in the exp2 domain, four interleaved partial sums.
// A NaN element, or +inf (then m = +inf), makes the result NaN.
__device__ __forceinline__ float lane_sumexp(const float (&x)[kPer], float m) {
  const float ml = m == -__builtin_inff() ? 0.0f : m * kLog2e;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int j = 0; j < kPer; ++j) s[j & 3] += __builtin_amdgcn_exp2f(fmaf(x[j], kLog2e, -ml));
  return (s[0] + s[1]) + (s[2] + s[3]);
}

// Descending bitonic sort of one value per lane across the wave.
__device__ __forceinline__ float wave_sort_desc(float v, int lane) {
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const float p = __shfl_xor(v, j, kWave);
      const bool take_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = take_max ? fmaxf(v, p) : fminf(v, p);
    }
  }
  return v;
}

// The K-th and the kq-th largest (kq <= K <= 64) of the wave's values, ties
// counted: at least K (kq) lanes hold a value >= tK (tq); -inf when fewer
// lanes hold finite values.  Larger K: a bitonic sort of the wave gives
// both.  Small K: only tq, by kq rounds of "take the wave maximum, retire
// the lanes holding it" (tK stays -inf): the K rounds for tK took longer
// than the few extra candidates the looser bound lets through.
__device__ __forceinline__ void wave_order_stats(float v, int K, int kq, int lane, float &tK,
                                                 float &tq) {
  const float ninf = -__builtin_inff();
  tK = ninf;
  tq = ninf;
  if (K > 16) {
    const float srt = wave_sort_desc(v, lane);
    tK = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(srt), K - 1));
    tq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(srt), kq - 1));
    return;
  }
  int taken = 0;
  for (int j = 0; j < kq && taken < kq; ++j) {
    const float mx = wave_max_f32(v);
    if (mx == ninf) return;
    const bool hit = v == mx;
    taken += __popcll(__ballot(hit));
    if (taken >= kq) tq = mx;
    v = hit ? ninf : v;
  }
}

// Workgroup-wide sum of one int per thread (one barrier; slots alternate).
__device__ __forceinline__ int block_sum(int c, int *slots, int &par) {
  c = wave_sum_i32(c);
  if ((threadIdx.x & (kWave - 1)) == 0) slots[par * kWavesPerBlock + threadIdx.x / kWave] = c;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) t += slots[par * kWavesPerBlock + i];
  par ^= 1;
  return t;
}

// Heavy ties (more than kCandCap elements reach the bound): the grain's
// exact K-th key by bisection, first over the order image o (the largest o
// with at least K elements >= o), then over the token bound among the
// elements equal to o that completes K; the elements with a larger key go to
// cand[K ..] (cntf_s counts them).  The grain is re-read from global memory
// (values cleaned as in the row pass) in batches of eight, so the row pass
// keeps no per-element state for this rare path.  Called by the whole block.
__device__ __noinline__ void grain_bisect_topk(const float *__restrict__ row, int e0, int e1,
                                               bool vec, int K, uint64_t *cand, int *cntf_s,
                                               int *red) {
  const int tid = threadIdx.x;
  constexpr int kB = 8;
  // f(j, order image) over the thread's valid elements
  auto each = [&](auto f) {
#pragma unroll 1
    for (int j0 = 0; j0 < kPer; j0 += kB) {
      float v[kB];
#pragma unroll
      for (int u = 0; u < kB; ++u) {
        const int t = elem_token(vec, e0, tid, j0 + u);
        v[u] = t < e1 ? row[t] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < kB; ++u) {
        const int t = elem_token(vec, e0, tid, j0 + u);
        bool b = false;
        if (t < e1) f(t, float_order(clean_logit(v[u], b)));
      }
    }
  };
  int par = 0;
  __syncthreads();  // the caller's block sums are done with red
  uint32_t o = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cb = o | (1u << bit);
    int q = 0;
    each([&](int, uint32_t oj) { q += oj >= cb; });
    if (block_sum(q, red, par) >= K) o = cb;
  }
  int q = 0;
  each([&](int, uint32_t oj) { q += oj > o; });
  const int need = K - block_sum(q, red, par);
  int lo = e0, hi = e1 - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    int qq = 0;
    each([&](int t, uint32_t oj) { qq += oj == o && t <= mid; });
    if (block_sum(qq, red, par) >= need)
      hi = mid;
    else
      lo = mid + 1;
  }
  each([&](int t, uint32_t oj) {
    if (oj > o || (oj == o && t <= lo)) {
      const int p = atomicAdd(cntf_s, 1);
      cand[K + p] = ((uint64_t)oj << 32) | (uint64_t)(0xffffffffu - (uint32_t)t);
    }
  });
}

// One workgroup per chunk of a row; see the file comment.  Per grain:
//  1. the grain sits in registers (32 elements per thread, one batch of
//     loads); per thread max, then sum of exp (a NaN result flags NaN/+inf
//     input, and only then are the values cleaned);
//  2. one (max, sum-exp) partial per grain, waves by a fixed DPP tree,
//     then the four waves in order: the same bits whatever the chunking;
//  3. a lower bound T on the grain's K-th largest logit from the thread
//     maxima, each wave on its own: the smallest over waves of a wave's
//     ceil(K/4)-th largest (every wave then holds ceil(K/4) elements >= it),
//     for K > 16 raised to the largest over waves of a wave's K-th largest
//     maximum (K threads hold an element >= it), and to the running chunk
//     list's K-th entry;
//  4. elements >= T are compacted into LDS (a few times K of them for
//     continuous logits); with more than kCandCap (heavy ties) the grain's
//     exact K-th key is found by bisection over the key bits instead (out of
//     line);
//  5. the running list and the candidates are ranked by (logit desc, token
//     asc) and the best K kept.
__global__ __launch_bounds__(kThreads) void row_partial_kernel(
    const float *__restrict__ logits, int rows_per_batch, int V, int K,
    int chunks, int grains_per_chunk, const int32_t *__restrict__ n_live,
    const uint8_t *__restrict__ needed, float2 *__restrict__ part_ms,
    uint64_t *__restrict__ part_keys, uint32_t *d_err) {
  __shared__ uint64_t cand[TG_MAX_TOPK + kCandCap];  // [0, K): running list
  __shared__ uint64_t run[TG_MAX_TOPK];
  __shared__ float lmax[kWavesPerBlock], lmaxq[kWavesPerBlock];
  __shared__ float gm[kWavesPerBlock], gs[kWavesPerBlock];
  __shared__ int cnt_s, cntf_s;
  __shared__ int red[2 * kWavesPerBlock];

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
  // Rows are 16-byte aligned iff V % 4 == 0 (the base is); the layout
  // depends on V only, so a row's partials never depend on where it sits.
  const bool vec = (V & 3) == 0;
  const float ninf = -__builtin_inff();

  if (tid < K) run[tid] = 0;
  bool bad = false;

  for (int gr = g_beg; gr < g_end; ++gr) {
    const int e0 = gr * kGrain;
    const int e1 = min(V, e0 + kGrain);
    const bool full = e1 - e0 == kGrain;
    float x[kPer];
    if (vec) {
      // e1 is a multiple of 4 here, so a float4 is wholly in or out
      const f32x4 *p = reinterpret_cast<const f32x4 *>(row + e0) + tid;
      if (full) {
#pragma unroll
        for (int u = 0; u < kPer / 4; ++u) {
          f32x4 v = __builtin_nontemporal_load(p + u * kThreads);
          x[4 * u] = v.x, x[4 * u + 1] = v.y, x[4 * u + 2] = v.z, x[4 * u + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int u = 0; u < kPer / 4; ++u) {
          f32x4 v = {ninf, ninf, ninf, ninf};
          if (elem_token(true, e0, tid, 4 * u) < e1) v = __builtin_nontemporal_load(p + u * kThreads);
          x[4 * u] = v.x, x[4 * u + 1] = v.y, x[4 * u + 2] = v.z, x[4 * u + 3] = v.w;
        }
      }
    } else {
      if (full) {
#pragma unroll
        for (int j = 0; j < kPer; ++j) x[j] = row[e0 + j * kThreads + tid];
      } else {
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
          const int i = e0 + j * kThreads + tid;
          x[j] = i < e1 ? row[i] : ninf;
        }
      }
    }

    // ---- 1. thread statistics
    float m = lane_max(x);
    float s = lane_sumexp(x, m);
    if (__any(!(s == s) || m == __builtin_inff())) {
#pragma unroll
      for (int j = 0; j < kPer; ++j) x[j] = clean_logit(x[j], bad);
      m = lane_max(x);
      s = lane_sumexp(x, m);
    }

    // ---- 2. wave partials; 3. the wave's bound on the K-th largest
    const float mw = wave_max_f32(m);
    const float sc = (m == ninf) ? 0.0f : s * __builtin_amdgcn_exp2f((m - mw) * kLog2e);
    const float sw = wave_sum_f32(sc);
    float tk, tq;
    wave_order_stats(m, K, (K + kWavesPerBlock - 1) / kWavesPerBlock, lane, tk, tq);
    if (lane == 0) {
      gm[w] = mw;
      gs[w] = sw;
      lmax[w] = tk;
      lmaxq[w] = tq;
    }
    if (tid < K) cand[tid] = run[tid];
    if (tid == 0) {
      cnt_s = 0;
      cntf_s = 0;
    }
    __syncthreads();
    if (tid < K) run[tid] = 0;
    float T = key_threshold(cand[K - 1]), Tq = lmaxq[0];
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) {
      T = fmaxf(T, lmax[i]);
      Tq = fminf(Tq, lmaxq[i]);
    }
    T = fmaxf(T, Tq);

    // ---- 4. candidates
    if (T > ninf) {
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        if (x[j] >= T) {
          const int p = atomicAdd(&cnt_s, 1);
          if (p < kCandCap) cand[K + p] = token_key(x[j], elem_token(vec, e0, tid, j));
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const int t = elem_token(vec, e0, tid, j);
        if (t < e1) {
          const int p = atomicAdd(&cnt_s, 1);
          if (p < kCandCap) cand[K + p] = token_key(x[j], t);
        }
      }
    }
    __syncthreads();
    int n = cnt_s;
    if (n > kCandCap) {
      grain_bisect_topk(row, e0, e1, vec, K, cand, &cntf_s, red);
      __syncthreads();
      n = cntf_s;
    }

    // ---- 5. rank the running list (empty on a chunk's first grain) and
    // the candidates; keys are distinct (distinct tokens)
    // the grain's (max, sum-exp) from the wave partials, by the last thread
    // (its wave has no candidate to rank unless the candidates nearly fill
    // the block)
    if (tid == kThreads - 1) {
      float M = gm[0], S = gs[0];
      for (int i = 1; i < kWavesPerBlock; ++i) merge_ms(M, S, gm[i], gs[i]);
      part_ms[(size_t)slot * n_grains + gr] = make_float2(M, S);
    }
    const int r0 = gr == g_beg ? K : 0;
    const int total = K + n;
    for (int t = r0 + tid; t < total; t += kThreads) {
      const uint64_t key = cand[t];
      if (key == 0) continue;
      int rank = 0, u = r0;
      for (; u + 4 <= total; u += 4) {  // four reads in flight
        const uint64_t a0 = cand[u], a1 = cand[u + 1], a2 = cand[u + 2], a3 = cand[u + 3];
        rank += (int)(a0 > key) + (int)(a1 > key) + (int)(a2 > key) + (int)(a3 > key);
      }
      for (; u < total; ++u) rank += cand[u] > key;
      if (rank < K) run[rank] = key;
    }
    __syncthreads();
  }
  if (bad) report(d_err, TG_DERR_NONFINITE);
  if (tid < K) part_keys[((size_t)slot * chunks + c) * K + tid] = run[tid];
}

// One wave per row slot, live by the row pass's rule: the row's
// log-sum-exp from its grain partials (wave_fold_lse: a fixed pairwise tree
// over the grains, the same bits whatever the chunking), and its top-K from
// the chunk lists (staged in LDS, K-round merge).  The
// partials and up to 256 list keys are loaded before the row's liveness is
// known (the workspace holds every row), so one round trip covers both.
// Writes lse[s] and out_keys[s * K + j], best first.
__global__ __launch_bounds__(kThreads) void row_finish_kernel(
    long long slots, int rows_per_batch, int K, int chunks, int n_ms,
    const int32_t *__restrict__ n_live, const uint8_t *__restrict__ needed,
    const float2 *__restrict__ part_ms, const uint64_t *__restrict__ part_keys,
    float *__restrict__ lse, uint64_t *__restrict__ out_keys) {
  extern __shared__ uint64_t stage[];  // [kWavesPerBlock][chunks * K]
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const long long s = (long long)blockIdx.x * kWavesPerBlock + w;
  if (s >= slots) return;  // wave-uniform from here on
  const int b = (int)(s / rows_per_batch);
  const int r = (int)(s - (long long)b * rows_per_batch);
  const float2 *ms = part_ms + s * n_ms;
  const uint64_t *lists = part_keys + s * chunks * K;
  const int nk = chunks * K;
  const float2 p = lane < n_ms ? ms[lane] : make_float2(-__builtin_inff(), 0.0f);
  uint64_t t[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = u * kWave + lane;
    t[u] = (chunks > 1 && i < nk) ? lists[i] : 0;
  }
  const bool live = needed ? needed[s] != 0 : r < (n_live ? n_live[b] : rows_per_batch);
  if (!live) return;
  uint64_t key;
  uint64_t *ws = stage + (size_t)w * nk;
  if (chunks == 1) {
    key = lane < K ? lists[lane] : 0;
  } else if (nk <= 4 * kWave) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = u * kWave + lane;
      if (i < nk) ws[i] = t[u];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    key = wave_merge_lists(ws, chunks, K);
  } else {
    key = wave_finish_topk(lists, chunks, K, ws);
  }
  const float l = wave_fold_lse(ms, n_ms, p);
  if (lane < K) out_keys[s * K + lane] = key;
  if (lane == 0) lse[s] = l;
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
launch("row_partial", row_partial_kernel, g, blk, 0, stream, logits, rows_per_batch, V, K,
         plan.chunks, plan.grains_per_chunk, n_live, needed, part_ms, part_keys, d_err);
  return hipGetLastError();
}

hipError_t launch_row_finish(int B, int rows_per_batch, int K, RowPlan plan,
                             const int32_t *n_live, const uint8_t *needed,
                             const float2 *part_ms, const uint64_t *part_keys, float *lse,
                             uint64_t *out_keys, hipStream_t stream) {
  const long long slots = (long long)B * rows_per_batch;
  const long long grid = (slots + kWavesPerBlock - 1) / kWavesPerBlock;
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const size_t lds = (size_t)kWavesPerBlock * plan.chunks * K * sizeof(uint64_t);
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute((const void *)row_finish_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  launch("row_finish", row_finish_kernel, dim3((unsigned)grid), dim3(kThreads), lds, stream,
         slots, rows_per_batch, K, plan.chunks, plan.ms_per_row, n_live, needed, part_ms,
         part_keys, lse, out_keys);
  return hipGetLastError();
}

}  // namespace tg
