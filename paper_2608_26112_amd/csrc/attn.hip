// Tree-verify attention on gfx950.
//
// Semantics (Alg. 3 tree-attention mask; Sec. 3.1 root = verified prefix):
// tree node i of sequence b attends to the prefix cache rows [0, L_b) and to
// the tree rows L_b + a for every a on its root path (ancestors and itself).
//
// attn_mfma_kernel (bf16): rows are (node, q-head-in-group) pairs of one
// (batch, KV head), so one staged K/V tile serves G*N query rows.  A
// workgroup owns 128 rows (4 waves x 32).  Per 64-key tile:
//   S^T[key][row] = K Q^T   with v_mfma_f32_32x32x16_bf16 (K from LDS, Q in
//                           registers), so every lane owns one query row and
//                           16 of its scores per 32-key block;
//   online softmax in fp32 (exp2 domain, one cross-lane max per tile);
//   O^T[d][row] += V^T P^T  with the same MFMA (V staged transposed in LDS,
//                           P straight from the score registers as bf16).
// The tree mask is built in-kernel from `parent`: each workgroup walks the
// ancestor chains of its own nodes into LDS bitsets.  Long prefixes can be
// split over workgroups (partial O and log-sum-exp, merged by
// attn_combine_kernel) when (batch x KV head x row tiles) cannot fill the chip.
//
// attn_f32_kernel (fp32): one wave per (batch, node, head) row, VALU dot
// products, online softmax, fp32 throughout.
#include "tg_device.h"
#include "tg_kernels.h"

namespace tg {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int BM = 128;  // query rows per workgroup
constexpr int BN = 64;   // keys per tile
constexpr int kMaxNodeWords = TG_MAX_VERIFY_NODES / 32;

__device__ __forceinline__ bool bad_prefix(int L, int N, int S_max) {
  return L < 0 || L + N > S_max;
}

// ------------------------------------------------------------ bf16 / MFMA
template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_mfma_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ kc,
    const __bf16 *__restrict__ vc, const int32_t *__restrict__ parent,
    const int32_t *__restrict__ prefix_len, __bf16 *__restrict__ out,
    float *__restrict__ part_o, float *__restrict__ part_lse, int B, int N,
    int Hq, int Hkv, int S_max, float scale2, int n_tiles, int n_splits,
    uint32_t *d_err) {
  constexpr int KS = D / 16;  // k-steps of the QK^T product
  constexpr int DB = D / 32;  // 32-wide d blocks of the output
  constexpr int KPAD = D + 8;
  constexpr int VPAD = BN + 8;
  __shared__ __attribute__((aligned(16))) __bf16 Ks[BN * KPAD];
  __shared__ __attribute__((aligned(16))) __bf16 Vt[D * VPAD];
  __shared__ int par_s[TG_MAX_VERIFY_NODES];
  __shared__ uint32_t anc_s[BM * kMaxNodeWords];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int G = Hq / Hkv;

  // ---- block -> (b, g, split, tile); tiles of one K/V stream share an XCD
  const int total = gridDim.x;
  int li = blockIdx.x;
  if ((total & 7) == 0) li = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const int tile = li % n_tiles;
  int rest = li / n_tiles;
  const int split = rest % n_splits;
  rest /= n_splits;
  const int g = rest % Hkv;
  const int b = rest / Hkv;

  const int L = prefix_len[b];
  const int rows_total = N * G;
  const int row0 = tile * BM;
  if (bad_prefix(L, N, S_max)) {
    if (tid == 0 && split == 0 && tile == 0 && g == 0) report(d_err, TG_DERR_BAD_PREFIX);
    if (n_splits == 1) {
      for (int rr = w; rr < BM; rr += 4) {
        int row = row0 + rr;
        if (row >= rows_total) break;
        int node = row / G, hq = g * G + row % G;
        __bf16 *o = out + (((size_t)b * N + node) * Hq + hq) * D;
        for (int d = lane; d < D; d += 64) o[d] = (__bf16)0.0f;
      }
    }
    // split mode: attn_combine_kernel writes the zeros
    return;
  }

  // ---- parents and ancestor-or-self bitsets of this tile's nodes
  const int node_lo = row0 / G;
  const int node_hi = min(N, (row0 + BM - 1) / G + 1);
  const int nloc = node_hi - node_lo;
  const int NW = (N + 31) >> 5;
  bool badp = false;
  for (int i = tid; i < N; i += kThreads) {
    int p = parent[(size_t)b * N + i];
    if (p < -1 || p >= i) {
      badp = true;
      p = -1;
    }
    par_s[i] = p;
  }
  if (badp && split == 0 && g == 0 && tile == 0) report(d_err, TG_DERR_BAD_PARENT);
  for (int i = tid; i < nloc * NW; i += kThreads) anc_s[i] = 0;
  __syncthreads();
  if (tid < nloc) {
    uint32_t *row = anc_s + tid * NW;
    for (int u = node_lo + tid; u >= 0; u = par_s[u]) row[u >> 5] |= 1u << (u & 31);
  }
  __syncthreads();

  // ---- this lane's query row, Q fragment in registers
  const int qrow = row0 + w * 32 + r32;
  const bool qvalid = qrow < rows_total;
  const int qnode = qvalid ? qrow / G : node_lo;
  const int qhead = g * G + (qvalid ? qrow % G : 0);
  const uint32_t *my_anc = anc_s + (qnode - node_lo) * NW;
  bf16x8 qf[KS];
  {
    const __bf16 *qp = q + (((size_t)b * N + qnode) * Hq + qhead) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (qvalid)
        qf[s] = *reinterpret_cast<const bf16x8 *>(qp + 16 * s);
      else
        qf[s] = bf16x8{};
    }
  }

  // ---- key ranges: this split's share of the prefix, then (last split) tree
  int chunk = (L + n_splits - 1) / n_splits;
  chunk = ((chunk + BN - 1) / BN) * BN;
  const int p_beg = min(L, split * chunk);
  const int p_end = min(L, p_beg + chunk);
  const bool do_tree = split == n_splits - 1;
  const int n_ptiles = (p_end - p_beg + BN - 1) / BN;
  const int n_ttiles = do_tree ? (N + BN - 1) / BN : 0;

  const size_t kv_base = ((size_t)b * Hkv + g) * (size_t)S_max * D;
  const __bf16 *kb = kc + kv_base;
  const __bf16 *vb = vc + kv_base;

  f32x16 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x16{};
  float m = -__builtin_inff();  // running max, log2 domain
  float l = 0.0f;               // this lane's share of the running sum

  constexpr int CPR = D / 8;                 // 16-byte chunks per row
  constexpr int LOADS = BN * CPR / kThreads; // per thread per matrix

  for (int t = 0; t < n_ptiles + n_ttiles; ++t) {
    const bool tree_tile = t >= n_ptiles;
    const int k0 = tree_tile ? L + (t - n_ptiles) * BN : p_beg + t * BN;
    const int k_lim = tree_tile ? L + N : p_end;

    // ---- stage K (row-major) and V (transposed) tiles in LDS
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int c = tid + i * kThreads;
      const int kr = c / CPR, cc = c % CPR;
      const int row = k0 + kr;
      bf16x8 kv8 = bf16x8{}, vv8 = bf16x8{};
      if (row < k_lim) {
        kv8 = *reinterpret_cast<const bf16x8 *>(kb + (size_t)row * D + cc * 8);
        vv8 = *reinterpret_cast<const bf16x8 *>(vb + (size_t)row * D + cc * 8);
      }
      *reinterpret_cast<bf16x8 *>(Ks + kr * KPAD + cc * 8) = kv8;
#pragma unroll
      for (int e = 0; e < 8; ++e) Vt[(cc * 8 + e) * VPAD + kr] = vv8[e];
    }
    __syncthreads();

    // ---- S^T = K Q^T for two 32-key blocks
    f32x16 acc[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      acc[blk] = f32x16{};
      const __bf16 *kp = Ks + (blk * 32 + r32) * KPAD + 8 * h;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 a = *reinterpret_cast<const bf16x8 *>(kp + 16 * s);
        acc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], acc[blk], 0, 0, 0);
      }
    }

    // ---- mask + online softmax (lane owns query r32, keys below)
    uint32_t tw[2] = {0xffffffffu, 0xffffffffu};
    if (tree_tile) {
      const int j0 = k0 - L;  // multiple of 64
      tw[0] = my_anc[(j0 >> 5)];
      tw[1] = ((j0 >> 5) + 1) < NW ? my_anc[(j0 >> 5) + 1] : 0u;
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kk = blk * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        bool valid = (k0 + kk) < k_lim;
        if (tree_tile) valid = valid && ((tw[blk] >> (kk & 31)) & 1u);
        float sv = valid ? acc[blk][r] * scale2 : -__builtin_inff();
        acc[blk][r] = sv;
        mx = fmaxf(mx, sv);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m, mx);
    // Rows whose keys are all masked so far keep m = -inf; they use 0 as the
    // reference so every p is exactly 0.  No branch: the MFMAs below run with
    // the whole wave active.
    const float m_use = m_new == -__builtin_inff() ? 0.0f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m - m_use);
    float ps = 0.0f;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(acc[blk][r] - m_use);
        acc[blk][r] = p;
        ps += p;
      }
    }
    l = l * alpha + ps;
#pragma unroll
    for (int i = 0; i < DB; ++i) o[i] *= alpha;
    m = m_new;

    // ---- O^T += V^T P^T, four 16-key steps
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        bf16x8 pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)acc[blk][8 * u + e];
        const int kb0 = blk * 32 + 16 * u + 4 * h;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const __bf16 *vp = Vt + (db * 32 + r32) * VPAD + kb0;
          bf16x4 lo = *reinterpret_cast<const bf16x4 *>(vp);
          bf16x4 hi = *reinterpret_cast<const bf16x4 *>(vp + 8);
          bf16x8 a = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[db], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // ---- finalize
  const float lt = l + __shfl_xor(l, 32, 64);
  if (!qvalid) return;
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  if (n_splits == 1) {
    __bf16 *op = out + (((size_t)b * N + qnode) * Hq + qhead) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = db * 32 + 8 * j + 4 * h;
        bf16x4 v4 = bf16x4{(__bf16)(o[db][4 * j] * inv), (__bf16)(o[db][4 * j + 1] * inv),
                           (__bf16)(o[db][4 * j + 2] * inv), (__bf16)(o[db][4 * j + 3] * inv)};
        *reinterpret_cast<bf16x4 *>(op + d) = v4;
      }
    }
  } else {
    const size_t prow = (((size_t)split * B + b) * N + qnode) * Hq + qhead;
    float *op = part_o + prow * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = db * 32 + 8 * j + 4 * h;
        *reinterpret_cast<f32x4 *>(op + d) =
            f32x4{o[db][4 * j] * inv, o[db][4 * j + 1] * inv, o[db][4 * j + 2] * inv,
                  o[db][4 * j + 3] * inv};
      }
    }
    if (h == 0) part_lse[prow] = lt > 0.0f ? m + __log2f(lt) : -__builtin_inff();
  }
}

// Merge split partials: out = sum_s 2^(lse_s - M) O_s / sum_s 2^(lse_s - M).
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(
    const float *__restrict__ part_o, const float *__restrict__ part_lse,
    const int32_t *__restrict__ prefix_len, __bf16 *__restrict__ out, int B,
    int N, int Hq, int S_max, int n_splits) {
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int rows = B * N * Hq;
  if (gw >= rows) return;
  const int b = gw / (N * Hq);
  __bf16 *op = out + (size_t)gw * D;
  if (bad_prefix(prefix_len[b], N, S_max)) {
    for (int d = lane; d < D; d += 64) op[d] = (__bf16)0.0f;
    return;
  }
  float M = -__builtin_inff();
  for (int s = 0; s < n_splits; ++s) M = fmaxf(M, part_lse[(size_t)s * rows + gw]);
  float acc[D / 64] = {};
  float den = 0.0f;
  for (int s = 0; s < n_splits; ++s) {
    float ls = part_lse[(size_t)s * rows + gw];
    if (ls == -__builtin_inff()) continue;
    float wgt = exp2f(ls - M);
    den += wgt;
    const float *po = part_o + ((size_t)s * rows + gw) * D;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) acc[e] += wgt * po[lane + 64 * e];
  }
  const float inv = den > 0.0f ? 1.0f / den : 0.0f;
#pragma unroll
  for (int e = 0; e < D / 64; ++e) op[lane + 64 * e] = (__bf16)(acc[e] * inv);
}

// ------------------------------------------------------------------- fp32
template <int D>
__global__ __launch_bounds__(kThreads) void attn_f32_kernel(
    const float *__restrict__ q, const float *__restrict__ kc,
    const float *__restrict__ vc, const int32_t *__restrict__ parent,
    const int32_t *__restrict__ prefix_len, float *__restrict__ out, int B,
    int N, int Hq, int Hkv, int S_max, float sm_scale, uint32_t *d_err) {
  constexpr int E = D / 64;
  __shared__ int path_s[4][TG_MAX_VERIFY_NODES];
  __shared__ float q_s[4][D];
  __shared__ float p_s[4][64];
  __shared__ int row_s[4][64];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + w;
  if (gw >= B * N * Hq) return;  // wave-uniform
  const int hq = gw % Hq;
  const int i = (gw / Hq) % N;
  const int b = gw / (Hq * N);
  const int g = hq / (Hq / Hkv);
  float *op = out + (size_t)gw * D;
  const int L = prefix_len[b];
  if (bad_prefix(L, N, S_max)) {
    if (lane == 0) report(d_err, TG_DERR_BAD_PREFIX);
    for (int d = lane; d < D; d += 64) op[d] = 0.0f;
    return;
  }
  // root path of node i (ancestors first), built by lane 0
  int t = 0;
  if (lane == 0) {
    bool badp = false;
    int u = i;
    while (u >= 0) {
      path_s[w][t++] = u;
      int p = parent[(size_t)b * N + u];
      if (p < -1 || p >= u) {
        badp = true;
        p = -1;
      }
      u = p;
    }
    for (int a = 0; a < t / 2; ++a) {
      int x = path_s[w][a];
      path_s[w][a] = path_s[w][t - 1 - a];
      path_s[w][t - 1 - a] = x;
    }
    if (badp) report(d_err, TG_DERR_BAD_PARENT);
  }
  t = __shfl(t, 0, 64);
  const float *qp = q + (size_t)gw * D;
  for (int d = lane; d < D; d += 64) q_s[w][d] = qp[d];
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();

  const size_t kv_base = ((size_t)b * Hkv + g) * (size_t)S_max * D;
  const int nkeys = L + t;
  float m = -__builtin_inff(), l = 0.0f;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  for (int k0 = 0; k0 < nkeys; k0 += 64) {
    const int kk = k0 + lane;
    float s = -__builtin_inff();
    int row = 0;
    if (kk < nkeys) {
      row = kk < L ? kk : L + path_s[w][kk - L];
      const float *kp = kc + kv_base + (size_t)row * D;
      float dot = 0.0f;
      for (int d = 0; d < D; d += 4) {
        f32x4 k4 = *reinterpret_cast<const f32x4 *>(kp + d);
        dot = fmaf(q_s[w][d], k4[0], dot);
        dot = fmaf(q_s[w][d + 1], k4[1], dot);
        dot = fmaf(q_s[w][d + 2], k4[2], dot);
        dot = fmaf(q_s[w][d + 3], k4[3], dot);
      }
      s = dot * sm_scale;
    }
    const float mt = wave_max_f32(s);
    const float mn = fmaxf(m, mt);
    const float alpha = m == -__builtin_inff() ? 0.0f : expf(m - mn);
    const float p = s == -__builtin_inff() ? 0.0f : expf(s - mn);
    l = l * alpha + wave_sum_f32(p);
    p_s[w][lane] = p;
    row_s[w][lane] = row;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const int nk = min(64, nkeys - k0);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= alpha;
    for (int j = 0; j < nk; ++j) {
      const float pj = p_s[w][j];
      const float *vp = vc + kv_base + (size_t)row_s[w][j] * D;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(pj, vp[lane + 64 * e], acc[e]);
    }
    m = mn;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
  const float inv = 1.0f / l;
#pragma unroll
  for (int e = 0; e < E; ++e) op[lane + 64 * e] = acc[e] * inv;
}

}  // namespace

int attn_splits(const AttnShape &s) {
  const int G = s.Hq / s.Hkv;
  const int tiles = (s.N * G + BM - 1) / BM;
  const long long base = (long long)s.B * s.Hkv * tiles;
  const long long want_wgs = 512;  // two workgroups per CU
  if (base >= want_wgs) return 1;
  const int max_prefix = s.S_max - s.N;
  int by_len = max_prefix / 512;  // keep >= 512 keys per split
  if (by_len < 1) by_len = 1;
  long long sp = (want_wgs + base - 1) / base;
  if (sp > by_len) sp = by_len;
  if (sp > 64) sp = 64;
  return (int)(sp < 1 ? 1 : sp);
}

size_t attn_workspace_bytes(const AttnShape &s, tg_dtype dtype) {
  if (dtype != TG_BF16) return 0;
  const int sp = attn_splits(s);
  if (sp <= 1) return 0;
  const size_t rows = (size_t)s.B * s.N * s.Hq;
  return (size_t)sp * rows * (s.D + 1) * sizeof(float) + 256;
}

hipError_t launch_attn_f32(const AttnShape &s, const float *q, const float *k,
                           const float *v, const int32_t *parent,
                           const int32_t *prefix_len, float *out,
                           uint32_t *d_err, hipStream_t stream) {
  const long long rows = (long long)s.B * s.N * s.Hq;
  dim3 grid((unsigned)((rows + 3) / 4)), blk(kThreads);
  if (s.D == 64)
    launch("attn_f32", attn_f32_kernel<64>, grid, blk, 0, stream, q, k, v, parent,
                       prefix_len, out, s.B, s.N, s.Hq, s.Hkv, s.S_max, s.sm_scale, d_err);
  else
    launch("attn_f32", attn_f32_kernel<128>, grid, blk, 0, stream, q, k, v, parent,
                       prefix_len, out, s.B, s.N, s.Hq, s.Hkv, s.S_max, s.sm_scale, d_err);
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const AttnShape &s, const void *q, const void *k,
                            const void *v, const int32_t *parent,
                            const int32_t *prefix_len, void *out,
                            void *workspace, uint32_t *d_err,
                            hipStream_t stream) {
  const int G = s.Hq / s.Hkv;
  const int tiles = (s.N * G + BM - 1) / BM;
  const int sp = attn_splits(s);
  const size_t rows = (size_t)s.B * s.N * s.Hq;
  float *part_o = sp > 1 ? reinterpret_cast<float *>(workspace) : nullptr;
  float *part_lse = sp > 1 ? part_o + (size_t)sp * rows * s.D : nullptr;
  const long long grid = (long long)s.B * s.Hkv * sp * tiles;
  const float scale2 = s.sm_scale * kLog2e;
  auto qb = reinterpret_cast<const __bf16 *>(q);
  auto kb = reinterpret_cast<const __bf16 *>(k);
  auto vb = reinterpret_cast<const __bf16 *>(v);
  auto ob = reinterpret_cast<__bf16 *>(out);
  if (s.D == 64)
    launch("attn_mfma", attn_mfma_kernel<64>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, qb, kb, vb, parent, prefix_len, ob, part_o, part_lse,
                       s.B, s.N, s.Hq, s.Hkv, s.S_max, scale2, tiles, sp, d_err);
  else
    launch("attn_mfma", attn_mfma_kernel<128>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, qb, kb, vb, parent, prefix_len, ob, part_o, part_lse,
                       s.B, s.N, s.Hq, s.Hkv, s.S_max, scale2, tiles, sp, d_err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || sp <= 1) return e;
  const unsigned cgrid = (unsigned)((rows + 3) / 4);
  if (s.D == 64)
    launch("attn_combine", attn_combine_kernel<64>, dim3(cgrid), dim3(kThreads), 0, stream,
                       part_o, part_lse, prefix_len, ob, s.B, s.N, s.Hq, s.S_max, sp);
  else
    launch("attn_combine", attn_combine_kernel<128>, dim3(cgrid), dim3(kThreads), 0, stream,
                       part_o, part_lse, prefix_len, ob, s.B, s.N, s.Hq, s.S_max, sp);
  return hipGetLastError();
}

}  // namespace tg
