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
#include <algorithm>

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
constexpr int kMaxSplits = 64;  // key-tile splits of one sequence at most

__device__ __forceinline__ bool bad_prefix(int L, int N, int S_max) {
  return L < 0 || L + N > S_max;
}

// ------------------------------------------------------------ bf16 / MFMA
// LDS tiles: K and V rows of D bf16, unpadded, written straight from global
// memory by global_load_lds (lane l of an instruction lands at base + 16 l).
// 16-byte chunks are XOR-swizzled with a function of the row,
// chunk' = chunk ^ swz(row), chosen for 64 banks of 4 bytes so that both
// read patterns are conflict-free:
//   K fragment (ds_read_b128, 16 lanes per pass): 16 consecutive rows, one
//     logical chunk -> swz must be a bijection on any 16 aligned rows
//     (D = 128: 16 rows per bank cycle; D = 64: two rows share a cycle, so on
//     each parity class);
//   transposed V (ds_read_b64_tr_b16, 32 lanes per pass): 4 consecutive rows
//     x 4 consecutive chunks -> the 4 rows must move the chunk's upper bits.
template <int D> struct AttnLds {
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int CM = CPR - 1;          // swizzle mask
  static constexpr int TILE = BN * D;         // bf16 elements per K (or V) tile
  static constexpr int STAGE = 2 * TILE;      // K then V
  static constexpr size_t bytes(int anc_words) { return (size_t)anc_words * 4; }
  static __device__ __forceinline__ int swz(int row) {
    if constexpr (D == 128)
      return ((row & 3) << 2) | ((row >> 2) & 3);
    else
      return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
  }
  // element offset of (row, d) inside a tile
  static __device__ __forceinline__ int at(int row, int d) {
    return row * D + ((((d >> 3) ^ swz(row)) & CM) << 3) + (d & 7);
  }
};

// max / sum with the lane 32 apart (the other half of a query row's keys),
// by v_permlane32_swap: no LDS round trip
__device__ __forceinline__ float half_swap(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  // lanes < 32: r[0] = own, r[1] = lane + 32; lanes >= 32: r[0] = lane - 32, r[1] = own
  return __uint_as_float(threadIdx.x & 32 ? r[0] : r[1]);
}

__device__ __forceinline__ bf16x4 lds_read_tr4(const __bf16 *p) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4 *)(p));
  return __builtin_bit_cast(bf16x4, v);
}

// byte address of a pointer into LDS (the low 32 bits of the generic address)
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// One global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's bytes land at LDS byte address lds_base + 16 l, lds_base wave-
// uniform.  Written as assembly so the compiler does not track it: a kernel
// that uses it orders its LDS reads after these copies with explicit waits
// (vmcnt) and barriers.  M0 is saved and restored around the copy.
__device__ __forceinline__ void dma16(const void *gaddr, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gaddr), "s"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory");
}

// Workgroup barrier for LDS data: waits for this wave's LDS accesses
// (lgkmcnt 0; vmcnt and expcnt at their maxima, i.e. no wait), not for its
// global loads in flight, which __syncthreads() would also wait for through
// its release fence.  The "memory" clobber keeps the compiler from moving
// memory operations across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Write-out of one wave's 32 query rows (lane (h, r) holds O^T of row r in
// the 32x32 MFMA output layout: d = 32 db + 8 j + 4 h + i in o[db][4 j + i]).
// The rows, scaled by `inv` and rounded to bf16, pass through `stage` (32 x D
// bf16 of LDS that only this wave uses) so that every global store writes
// whole 16-byte chunks, D / 8 lanes per row, instead of 8-byte pieces of 32
// different rows.  8-byte slots are XOR-swizzled by row so that both the
// writes (32 rows, one slot) and the reads (whole rows) are conflict-free.
// Row r of the wave is query row row_first + r, i.e. node (row_first + r) / G
// and head g G + (row_first + r) % G; it goes to
// dst + ((row_off + node) Hq + head) D, and only if row_first + r < rows_total.
template <int D>
__device__ __forceinline__ void store_rows(const f32x16 (&o)[D / 32], float inv, __bf16 *stage,
                                           __bf16 *__restrict__ dst, size_t row_off,
                                           int row_first, int rows_total, int G, int g, int Hq) {
  constexpr int DB = D / 32;
  constexpr int CPR = D / 8;       // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;    // rows per read instruction
  const int lane = threadIdx.x & (kWave - 1);
  const int h = lane >> 5, r32 = lane & 31;
  auto swz = [](int r) { return D == 128 ? (r & 31) : ((r >> 1) & 15); };
  const int f = swz(r32);
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int slot = (db * 8 + 2 * j + h) ^ f;  // 8-byte slot (4 bf16)
      *reinterpret_cast<bf16x4 *>(stage + r32 * D + 4 * slot) =
          bf16x4{(__bf16)(o[db][4 * j] * inv), (__bf16)(o[db][4 * j + 1] * inv),
                 (__bf16)(o[db][4 * j + 2] * inv), (__bf16)(o[db][4 * j + 3] * inv)};
    }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int c = lane % CPR;
#pragma unroll
  for (int it = 0; it < 32 / RPI; ++it) {
    const int r = it * RPI + lane / CPR;
    const int fr = swz(r);
    // logical slots 2c, 2c+1 sit in physical chunk c ^ (fr >> 1), swapped
    // when fr is odd
    bf16x8 v = *reinterpret_cast<const bf16x8 *>(stage + r * D + 8 * (c ^ (fr >> 1)));
    if (fr & 1) v = __builtin_shufflevector(v, v, 4, 5, 6, 7, 0, 1, 2, 3);
    const int qrow = row_first + r;
    if (qrow < rows_total) {
      const int node = qrow / G, head = g * G + (qrow - node * G);
      *reinterpret_cast<bf16x8 *>(dst + ((row_off + node) * Hq + head) * D + 8 * c) = v;
    }
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_mfma_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ kc,
    const __bf16 *__restrict__ vc, const int32_t *__restrict__ parent,
    const int32_t *__restrict__ prefix_len, __bf16 *__restrict__ out,
    __bf16 *__restrict__ part_o, float *__restrict__ part_lse, int B, int N,
    int Hq, int Hkv, int S_max, float scale2, int n_tiles, int n_splits,
    uint32_t *d_err) {
  using Lds = AttnLds<D>;
  constexpr int KS = D / 16;  // k-steps of the QK^T product
  constexpr int DB = D / 32;  // 32-wide d blocks of the output
  constexpr int LOADS = BN * D * 2 / 16 / kThreads;  // 16-byte loads per thread per tile
  // two stages as distinct objects, so the compiler can tell that loads in
  // flight into one stage do not alias reads of the other
  __shared__ __attribute__((aligned(16))) __bf16 stage0[Lds::STAGE];
  __shared__ __attribute__((aligned(16))) __bf16 stage1[Lds::STAGE];
  // dynamic: the bitsets of the tile's nodes, then the parent array
  extern __shared__ __attribute__((aligned(16))) uint32_t anc_s[];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int G = Hq / Hkv;
  const int NW = (N + 31) >> 5;
  int *par_s = reinterpret_cast<int *>(anc_s + min(N, (BM + G - 1) / G + 1) * NW);

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

  // Every global read of the prologue is issued before the first one is
  // waited for: this thread's parents (at most TG_MAX_VERIFY_NODES / kThreads
  // of them), its Q fragment and the prefix length.  All of them are consumed
  // before the first tile is requested, so no later wait for a register
  // operand can cover the tile loads.
  const int rows_total = N * G;
  const int row0 = tile * BM;
  constexpr int kParPerThread = (TG_MAX_VERIFY_NODES + kThreads - 1) / kThreads;
  int pv[kParPerThread];
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = tid + k * kThreads;
    pv[k] = i < N ? parent[(size_t)b * N + i] : -1;
  }
  const int node_lo = row0 / G;
  const int qrow = row0 + w * 32 + r32;
  const bool qvalid = qrow < rows_total;
  const int qnode = qvalid ? qrow / G : node_lo;
  const int qhead = g * G + (qvalid ? qrow % G : 0);
  bf16x8 qf[KS];
  {
    const __bf16 *qp = q + (((size_t)b * N + qnode) * Hq + qhead) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qf[s] = *reinterpret_cast<const bf16x8 *>(qp + 16 * s);
  }
  const int L_in = prefix_len[b];
  // A prefix length out of range (BAD_PREFIX) runs no key tile: its rows
  // leave as zeros (o = 0, l = 0), or in split mode as empty partials, which
  // the combine turns into zeros.  No early return: the compiler would move
  // the Q loads behind the prefix length's arrival.
  const bool bad_len = bad_prefix(L_in, N, S_max);
  if (bad_len && tid == 0 && split == 0 && tile == 0 && g == 0) report(d_err, TG_DERR_BAD_PREFIX);
  const int L = bad_len ? 0 : L_in;

  // ---- key tiles: the prefix's 64-key tiles, then the tree's, dealt out to
  // the splits as equal runs (the tree's tiles weigh like any other)
  const int n_pt = (L + BN - 1) / BN;
  const int n_vt = n_pt + (N + BN - 1) / BN;
  const int per_split = (n_vt + n_splits - 1) / n_splits;
  const int vt0 = min(n_vt, split * per_split);
  const int n_tiles_all = bad_len ? 0 : min(n_vt, vt0 + per_split) - vt0;

  const size_t kv_base = ((size_t)b * Hkv + g) * (size_t)S_max * D;
  const __bf16 *kb = kc + kv_base;
  const __bf16 *vb = vc + kv_base;

  f32x16 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x16{};
  float m = -__builtin_inff();  // running max, scaled log2 units
  float l = 0.0f;               // this lane's share of the running sum

  auto tree_tile_at = [&](int t) { return vt0 + t >= n_pt; };
  auto tile_k0 = [&](int t) { return tree_tile_at(t) ? L + (vt0 + t - n_pt) * BN : (vt0 + t) * BN; };
  auto tile_lim = [&](int t) { return tree_tile_at(t) ? L + N : L; };
  // Direct global -> LDS loads.  Instruction i of wave w fills the 1 KB
  // block j = w * LOADS + i of a tile: rows j * RPI .. + RPI - 1, and lane l
  // writes physical chunk l % CPR of its row, i.e. loads logical chunk
  // (l % CPR) ^ swz(row).  Offsets are per-thread constants.
  constexpr int RPI = 64 / Lds::CPR;  // rows per 1 KB instruction
  int goff[LOADS];
  int grow[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int row = (w * LOADS + i) * RPI + lane / Lds::CPR;
    const int chunk = ((lane % Lds::CPR) ^ Lds::swz(row)) & Lds::CM;
    grow[i] = row;
    goff[i] = row * D + chunk * 8;
  }
  // The copies are assembly (dma16), invisible to the compiler's waits: the
  // compiler, tracking them, made tile t's fragment reads wait for tile
  // t + 1's copies.  Every read of a stage follows an explicit wait for its
  // copies and a barrier.
  auto issue = [&](int t, __bf16 *dst) {
    const int k0 = tile_k0(t), lim = tile_lim(t);
    const __bf16 *kt = kb + (size_t)k0 * D;  // wave-uniform tile base
    const __bf16 *vt = vb + (size_t)k0 * D;
    const uint32_t dk = lds_addr(dst), dv = lds_addr(dst + Lds::TILE);
    auto one = [&](int i, int off) {
      const uint32_t blk = (w * LOADS + i) * 1024;   // 1 KB block
      dma16(kt + off, dk + blk);
      dma16(vt + off, dv + blk);
    };
    if (k0 + BN <= lim) {
#pragma unroll
      for (int i = 0; i < LOADS; ++i) one(i, goff[i]);
    } else {
      // rows past the range re-read the last valid row (finite, masked later)
#pragma unroll
      for (int i = 0; i < LOADS; ++i)
        one(i, goff[i] - max(0, k0 + grow[i] - (lim - 1)) * D);
    }
  };

  // ---- parents into LDS; then nothing read into registers is in flight
  bool badp = false;
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = tid + k * kThreads;
    int p = pv[k];
    if (i < N) {
      if (p < -1 || p >= i) {
        badp = true;
        p = -1;
      }
      par_s[i] = p;
    }
  }
  if (badp && split == 0 && g == 0 && tile == 0) report(d_err, TG_DERR_BAD_PARENT);
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): Q, parents (expcnt, lgkmcnt: no wait)

  // tiles 0 and 1 stream in while the bitsets are built
  if (n_tiles_all > 0) issue(0, stage0);
  if (n_tiles_all > 1) issue(1, stage1);

  // ---- ancestor-or-self bitsets of this tile's nodes (a1)
  const int node_hi = min(N, (row0 + BM - 1) / G + 1);
  const int nloc = node_hi - node_lo;
  lds_barrier();  // the parents are in LDS
  // word j of node i's ancestor-or-self bitset, by one thread: it walks the
  // chain (ids fall along it) down to the word's first id
  for (int it = tid; it < nloc * NW; it += kThreads) {
    const int i = it / NW, j = it - i * NW;
    uint32_t word = 0;
    for (int u = node_lo + i; u >= 32 * j; u = par_s[u])
      if (u < 32 * (j + 1)) word |= 1u << (u & 31);
    anc_s[it] = word;
  }

  // ---- this lane's query row: its ancestor-or-self bitset
  const uint32_t *my_anc = anc_s + (qnode - node_lo) * NW;

  // the bitsets are complete and tile 0 has landed (this wave's part of it:
  // tile 1's 2 LOADS younger loads may stay in flight), in every wave
  if (n_tiles_all > 1)
    __builtin_amdgcn_s_waitcnt((2 * LOADS) | (7 << 4));
  else
    __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);

  auto step = [&](int t, const __bf16 *cur, __bf16 *nxt) {
    const __bf16 *Kt = cur;
    const __bf16 *Vt = cur + Lds::TILE;
    // tile t + 1 lands in LDS while tile t computes (tile 1 was requested
    // by the prologue)
    if (t >= 1 && t + 1 < n_tiles_all) issue(t + 1, nxt);
    const bool tree_tile = tree_tile_at(t);
    const int k0 = tile_k0(t);
    const int k_lim = tile_lim(t);

    // ---- S^T = K Q^T for two 32-key blocks
    f32x16 acc[2] = {f32x16{}, f32x16{}};
    {
      // K fragments one step ahead of the MFMAs that consume them
      const int kr0 = r32, kr1 = 32 + r32;
      auto kfrag = [&](int kr, int s) {
        return *reinterpret_cast<const bf16x8 *>(Kt + Lds::at(kr, 16 * s + 8 * h));
      };
      bf16x8 a0 = kfrag(kr0, 0);
      bf16x8 a1 = kfrag(kr1, 0);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 n0 = a0, n1 = a1;
        if (s + 1 < KS) {
          n0 = kfrag(kr0, s + 1);
          n1 = kfrag(kr1, s + 1);
        }
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[s], acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[s], acc[1], 0, 0, 0);
        a0 = n0;
        a1 = n1;
      }
    }

    // ---- mask (partial prefix tile or tree tile only)
    if (tree_tile || k0 + BN > k_lim) {
      uint32_t tw0 = 0xffffffffu, tw1 = 0xffffffffu;
      if (tree_tile) {
        const int wj = (k0 - L) >> 5;  // k0 - L is a multiple of 64
        tw0 = my_anc[wj];
        tw1 = wj + 1 < NW ? my_anc[wj + 1] : 0u;
      }
      // key kk = blk*32 + 8(r/4) + 4h + r%4: shifts by 4h once, then by constants
      const int lim_h = k_lim - k0 - 4 * h;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const uint32_t tw = (blk ? tw1 : tw0) >> (4 * h);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kc = blk * 32 + 8 * (r >> 2) + (r & 3);
          const bool valid = kc < lim_h && ((tw >> (kc & 31)) & 1u);
          acc[blk][r] = valid ? acc[blk][r] : -__builtin_inff();
        }
      }
    }

    // ---- online softmax: one cross-lane max per tile, lazy O rescale
    float mx;
    {
      // 32 values -> 11 three-input maxima -> 4 -> 2 -> 1
      float t3[11];
#pragma unroll
      for (int i = 0; i < 10; ++i) {
        const int a = 3 * i, b = a + 1, c = a + 2;
        t3[i] = __builtin_fmaxf(acc[a >> 4][a & 15],
                                __builtin_fmaxf(acc[b >> 4][b & 15], acc[c >> 4][c & 15]));
      }
      t3[10] = __builtin_fmaxf(acc[1][14], acc[1][15]);
      const float u0 = __builtin_fmaxf(t3[0], __builtin_fmaxf(t3[1], t3[2]));
      const float u1 = __builtin_fmaxf(t3[3], __builtin_fmaxf(t3[4], t3[5]));
      const float u2 = __builtin_fmaxf(t3[6], __builtin_fmaxf(t3[7], t3[8]));
      const float u3 = __builtin_fmaxf(t3[9], t3[10]);
      mx = __builtin_fmaxf(__builtin_fmaxf(u0, u1), __builtin_fmaxf(u2, u3));
    }
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m, mx * scale2);
    if (__any(m_new > m)) {
      // some row's max grew: rescale that row's running sum and output
      const float alpha = __builtin_amdgcn_exp2f(m - (m_new == -__builtin_inff() ? 0.0f : m_new));
      l *= alpha;
#pragma unroll
      for (int i = 0; i < DB; ++i) o[i] *= alpha;
      m = m_new;
    }
    // rows whose keys are all masked so far keep m = -inf and use 0 as the
    // reference, so every p is exactly 0
    const float m_use = m == -__builtin_inff() ? 0.0f : m;
    bf16x8 pb[2][2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        pb[blk][r >> 3][r & 7] =
            (__bf16)__builtin_amdgcn_exp2f(fmaf(acc[blk][r], scale2, -m_use));
    // the normaliser sums exactly the bf16 probabilities the PV product uses
    {
      typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
      const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 8; e += 2)
            l = __builtin_amdgcn_fdot2_f32_bf16(
                bf16x2{pb[blk][u][e], pb[blk][u][e + 1]}, one2, l, false);
    }

    // ---- O^T += V^T P^T, four 16-key steps; V^T fragments by transposed
    // reads of the row-major V tile (lane group: 4 keys x 16 d)
    const int grp = lane >> 4, gl = lane & 15;
    const int vrow = 4 * (grp >> 1) + (gl >> 2);           // key within the 8-key half
    const int vcol = 16 * (grp & 1) + 4 * (gl & 3);        // d within the 32-wide block
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int vr = blk * 32 + 16 * u + vrow;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x4 lo = lds_read_tr4(Vt + Lds::at(vr, db * 32 + vcol));
          const bf16x4 hi = lds_read_tr4(Vt + Lds::at(vr + 8, db * 32 + vcol));
          const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[blk][u], o[db], 0, 0, 0);
        }
      }
    }
    // this thread's loads into the next stage have landed; then every wave's
    // loads have landed and nobody reads the current stage any more
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  // Tile 0 peeled (tile 1's loads, from the prologue, are in flight while it
  // computes); then unrolled by two so each half reads and fills fixed stages.
  if (n_tiles_all > 0) step(0, stage0, stage1);
  for (int t = 1; t < n_tiles_all; t += 2) {
    step(t, stage1, stage0);
    if (t + 1 < n_tiles_all) step(t + 1, stage0, stage1);
  }

  // ---- finalize: every wave is past its last read of the stages (the
  // last step ends with a barrier), so wave w stages its rows in stage 0
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  const bool split_mode = n_splits > 1;
  store_rows<D>(o, inv, stage0 + w * 32 * D, split_mode ? part_o : out,
                split_mode ? ((size_t)split * B + b) * N : (size_t)b * N, row0 + w * 32,
                rows_total, G, g, Hq);
  if (split_mode && qvalid && h == 0)
    part_lse[(((size_t)split * B + b) * N + qnode) * Hq + qhead] =
        lt > 0.0f ? m + __log2f(lt) : -__builtin_inff();
}

// --------------------------------------------- bf16, ping-pong schedule
// For long prefixes: 8 waves (two per SIMD) share each K/V tile; a
// workgroup owns 256 query rows (32 per wave, the same MFMA layout as
// attn_mfma_kernel).  Each wave alternates an MFMA phase M(t) = {PV of tile
// t-1, QK^T of tile t} and a vector phase S(t) = {mask, reference, rescale,
// exponentials of tile t}.  On every SIMD one wave (group A) runs one phase
// ahead of the other (group B), so one wave feeds the matrix core while the
// other runs its softmax; a workgroup barrier ends every phase.
//   phase 2j  : K(j+2) and V(j+1) are requested; group A runs M(j),
//               group B runs S(j-1)
//   phase 2j+1: group A runs S(j), group B runs M(j)
// K and V have three LDS stages each, so the requests of phase pair j land
// during pair j+1 and are waited for only at the barrier that ends it.
// At D = 128 the MFMA phase is inline assembly (mfma_phase_d128.inc) that
// keeps its fragment reads four MFMAs ahead; the compiler, at 256 VGPRs for
// two waves per SIMD, would wait for every read.
#include "mfma_phase_d128.inc"

template <int D>
__global__ __launch_bounds__(512, 1) void attn_pingpong_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ kc,
    const __bf16 *__restrict__ vc, const int32_t *__restrict__ parent,
    const int32_t *__restrict__ prefix_len, __bf16 *__restrict__ out,
    __bf16 *__restrict__ part_o, float *__restrict__ part_lse, int B, int N,
    int Hq, int Hkv, int S_max, float scale2, int n_tiles, int n_splits,
    uint32_t *d_err) {
  using Lds = AttnLds<D>;
  constexpr int NT = 512;
  constexpr int BMP = 256;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int LOADS = BN * D * 2 / 16 / NT;  // 16-byte loads per thread per tile
  // three stages each of K and V (distinct objects, so the compiler knows a
  // read of one stage does not alias loads in flight into another): tiles
  // are requested two tiles ahead of their use
  __shared__ __attribute__((aligned(16))) __bf16 kst0[Lds::TILE];
  __shared__ __attribute__((aligned(16))) __bf16 kst1[Lds::TILE];
  __shared__ __attribute__((aligned(16))) __bf16 kst2[Lds::TILE];
  __shared__ __attribute__((aligned(16))) __bf16 vst0[Lds::TILE];
  __shared__ __attribute__((aligned(16))) __bf16 vst1[Lds::TILE];
  __shared__ __attribute__((aligned(16))) __bf16 vst2[Lds::TILE];
  extern __shared__ __attribute__((aligned(16))) uint32_t anc_s[];
  // prologue only (N ints fit a tile); no tile is loaded into it before the loop
  int *par_s = reinterpret_cast<int *>(vst2);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int G = Hq / Hkv;
  // Group A / B by SIMD: the first wave (in wave order) placed on each SIMD
  // leads.  HW_ID bits [5:4] hold the wave's SIMD (s_getreg, size 2, offset 4).
  // Only the overlap depends on this; every wave runs the same barriers.
  __shared__ int simd_s[NT / 64];
  const int my_simd = __builtin_amdgcn_s_getreg((1 << 11) | (4 << 6) | 4);
  if (lane == 0) simd_s[w] = my_simd;

  const int total = gridDim.x;
  int li = blockIdx.x;
  if ((total & 7) == 0) li = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const int tile = li % n_tiles;
  int rest = li / n_tiles;
  const int split = rest % n_splits;
  rest /= n_splits;
  const int g = rest % Hkv;
  const int b = rest / Hkv;

  // Every global read of the prologue is issued before the first one is
  // waited for: this thread's parents, its Q fragment and the prefix length.
  const int rows_total = N * G;
  const int row0 = tile * BMP;
  constexpr int kParPerThread = (TG_MAX_VERIFY_NODES + NT - 1) / NT;
  int pv[kParPerThread];
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = tid + k * NT;
    pv[k] = i < N ? parent[(size_t)b * N + i] : -1;
  }
  const int node_lo = row0 / G;
  const int qrow = row0 + w * 32 + r32;
  const bool qvalid = qrow < rows_total;
  const int qnode = qvalid ? qrow / G : node_lo;
  const int qhead = g * G + (qvalid ? qrow % G : 0);
  // Q as given; scores leave the MFMA in raw units and are scaled to log2
  // units (sm_scale * log2 e) by the fused multiply-add that also subtracts
  // the reference
  bf16x8 qf[KS];
  {
    const __bf16 *qp = q + (((size_t)b * N + qnode) * Hq + qhead) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qf[s] = *reinterpret_cast<const bf16x8 *>(qp + 16 * s);
  }
  const int L_in = prefix_len[b];
  // A prefix length out of range (BAD_PREFIX) runs no key tile: its rows
  // leave as zeros, or in split mode as empty partials (no early return, as
  // in attn_mfma_kernel)
  const bool bad_len = bad_prefix(L_in, N, S_max);
  if (bad_len && tid == 0 && split == 0 && tile == 0 && g == 0) report(d_err, TG_DERR_BAD_PREFIX);
  const int L = bad_len ? 0 : L_in;

  // key tiles: the prefix's, then the tree's, dealt out as equal runs
  const int n_pt = (L + BN - 1) / BN;
  const int n_vt = n_pt + (N + BN - 1) / BN;
  const int per_split = (n_vt + n_splits - 1) / n_splits;
  const int vt0 = min(n_vt, split * per_split);
  const int n = bad_len ? 0 : min(n_vt, vt0 + per_split) - vt0;

  const size_t kv_base = ((size_t)b * Hkv + g) * (size_t)S_max * D;
  const __bf16 *kb = kc + kv_base;
  const __bf16 *vb = vc + kv_base;

  auto tree_tile_at = [&](int t) { return vt0 + t >= n_pt; };
  auto tile_k0 = [&](int t) { return tree_tile_at(t) ? L + (vt0 + t - n_pt) * BN : (vt0 + t) * BN; };
  auto tile_lim = [&](int t) { return tree_tile_at(t) ? L + N : L; };
  constexpr int RPI = 64 / Lds::CPR;
  // offsets recomputed per issue (a few VALU ops) rather than held in registers
  auto issue = [&](const __bf16 *src, int t, __bf16 *dst) __attribute__((always_inline)) {
    const int k0 = tile_k0(t), lim = tile_lim(t);
    const __bf16 *st = src + (size_t)k0 * D;
    int goff[LOADS], grow[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int row = (w * LOADS + i) * RPI + lane / Lds::CPR;
      grow[i] = row;
      goff[i] = row * D + (((lane % Lds::CPR) ^ Lds::swz(row)) & Lds::CM) * 8;
    }
    auto one = [&](int i, int off) {
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void *)(st + off),
          (__attribute__((address_space(3))) void *)(dst + (w * LOADS + i) * 512), 16, 0, 0);
    };
    if (k0 + BN <= lim) {
#pragma unroll
      for (int i = 0; i < LOADS; ++i) one(i, goff[i]);
    } else {
      // rows past the range re-read the last valid row (finite, masked later)
#pragma unroll
      for (int i = 0; i < LOADS; ++i) one(i, goff[i] - max(0, k0 + grow[i] - (lim - 1)) * D);
    }
  };

  // ---- parents into LDS; then nothing read into registers is in flight,
  // so no later wait for a register operand can cover the tile loads
  bool badp = false;
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = tid + k * NT;
    int p = pv[k];
    if (i < N) {
      if (p < -1 || p >= i) {
        badp = true;
        p = -1;
      }
      par_s[i] = p;
    }
  }
  if (badp && split == 0 && g == 0 && tile == 0) report(d_err, TG_DERR_BAD_PARENT);
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): Q, parents (expcnt, lgkmcnt: no wait)

  // the first tiles stream in while the bitsets are built
  if (n > 0) issue(kb, 0, kst0);
  if (n > 1) issue(kb, 1, kst1);
  if (n > 0) issue(vb, 0, vst0);

  // ---- ancestor-or-self bitsets of this tile's nodes (a1)
  const int node_hi = min(N, (row0 + BMP - 1) / G + 1);
  const int nloc = node_hi - node_lo;
  const int NW = (N + 31) >> 5;
  lds_barrier();  // the parents are in LDS; the prologue's tile loads stay in flight
  // word j of node i's ancestor-or-self bitset, by one thread (as in
  // attn_mfma_kernel)
  for (int it = tid; it < nloc * NW; it += NT) {
    const int i = it / NW, j = it - i * NW;
    uint32_t word = 0;
    for (int u = node_lo + i; u >= 32 * j; u = par_s[u])
      if (u < 32 * (j + 1)) word |= 1u << (u & 31);
    anc_s[it] = word;
  }
  bool lead = true;
  for (int i = 0; i < w; ++i) lead = lead && simd_s[i] != my_simd;

  // ---- this lane's query row: its ancestor-or-self bitset
  const uint32_t *my_anc = anc_s + (qnode - node_lo) * NW;

  // Running row reference m (log2 units): the max of the row's first tile
  // with a visible key, then moved up only when a tile's scores exceed it by
  // more than kSlack, so the exponentials stay below 2^kSlack and the O / l
  // rescale is rare.
  constexpr float kSlack = 8.0f;
  f32x16 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x16{};
  float m = 0.0f;
  bool m_set = false;
  float l = 0.0f;
  f32x16 acc[2];
  bf16x8 pb[2][2];

  // Per-lane LDS element offsets of the fragment reads.  The swizzle only
  // looks at the low four row bits, so the row offset of a 16- or 32-key
  // block is a constant added to these.
  const int grp = lane >> 4, gl = lane & 15;
  const int vrow = 4 * (grp >> 1) + (gl >> 2);
  const int vcol = 16 * (grp & 1) + 4 * (gl & 3);
  int voff[DB][2];  // V^T fragment (transposed reads): [d block][key half]
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    voff[db][0] = Lds::at(vrow, db * 32 + vcol);
    voff[db][1] = Lds::at(vrow + 8, db * 32 + vcol);
  }
  int koff[KS];  // K fragment: [k-step], key r32 (the second block is +32 rows)
#pragma unroll
  for (int s = 0; s < KS; ++s) koff[s] = Lds::at(r32, 16 * s + 8 * h);

  // MFMA phase: PV of the previous tile (pb, V in Vp) then QK^T of this one
  // With `bar` (D = 128 only) the phase takes the workgroup barrier that
  // precedes it inside its statement, after issuing its first fragment reads.
  auto mphase = [&](bool do_pv, const __bf16 *Vp, bool do_qk, const __bf16 *Kt, bool bar)
                    __attribute__((always_inline)) {
    // the MFMA wave issues first whenever the matrix core is free; the
    // softmax wave on the same SIMD fills the remaining issue slots
    __builtin_amdgcn_s_setprio(1);
    if constexpr (D == 128) {
      // the generated statements assume this tile geometry: 64-key tiles of
      // 256-byte rows, the second 32-key block 8 KB into a K stage, 16-key
      // halves 4 KB apart in a V stage
      static_assert(BN == 64 && Lds::TILE == BN * 128 && KS == 8 && DB == 4,
                    "mfma_phase_d128.inc is generated for 64-key tiles at D = 128");
      // operands in registers the statements name: LDS byte addresses
      // (stage base in an SGPR, per-lane offsets in VGPRs), fragments as
      // 4-dword vectors
      using i32x4 = int __attribute__((ext_vector_type(4)));
      const uint32_t vbase = lds_addr(Vp), kbase = lds_addr(Kt);
      const i32x4 p00 = __builtin_bit_cast(i32x4, pb[0][0]);
      const i32x4 p01 = __builtin_bit_cast(i32x4, pb[0][1]);
      const i32x4 p10 = __builtin_bit_cast(i32x4, pb[1][0]);
      const i32x4 p11 = __builtin_bit_cast(i32x4, pb[1][1]);
      i32x4 qq[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) qq[s] = __builtin_bit_cast(i32x4, qf[s]);
      int va[8], ka[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        va[i] = 2 * voff[i >> 1][i & 1];
        ka[i] = 2 * koff[i];
      }
#define TG_O_OUT [o0] "+v"(o[0]), [o1] "+v"(o[1]), [o2] "+v"(o[2]), [o3] "+v"(o[3])
#define TG_ACC_OUT [a0] "=&v"(acc[0]), [a1] "=&v"(acc[1])
#define TG_PV_IN                                                                           \
  [p00] "v"(p00), [p01] "v"(p01), [p10] "v"(p10), [p11] "v"(p11), [va0] "v"(va[0]),        \
      [va1] "v"(va[1]), [va2] "v"(va[2]), [va3] "v"(va[3]), [va4] "v"(va[4]),               \
      [va5] "v"(va[5]), [va6] "v"(va[6]), [va7] "v"(va[7]), [vb] "s"(vbase)
#define TG_QK_IN                                                                           \
  [q0] "v"(qq[0]), [q1] "v"(qq[1]), [q2] "v"(qq[2]), [q3] "v"(qq[3]), [q4] "v"(qq[4]),     \
      [q5] "v"(qq[5]), [q6] "v"(qq[6]), [q7] "v"(qq[7]), [ka0] "v"(ka[0]), [ka1] "v"(ka[1]), \
      [ka2] "v"(ka[2]), [ka3] "v"(ka[3]), [ka4] "v"(ka[4]), [ka5] "v"(ka[5]),               \
      [ka6] "v"(ka[6]), [ka7] "v"(ka[7]), [kb] "s"(kbase)
#define TG_RING_CLOBBERS                                                                   \
  "v220", "v221", "v222", "v223", "v224", "v225", "v226", "v227", "v228", "v229", "v230", \
      "v231", "v232", "v233", "v234", "v235", "v236", "v237", "v238", "v239", "v240",     \
      "v241", "v242", "v243", "v244", "v245", "v246", "v247", "v248", "v249", "v250",     \
      "v251", "v252", "v253", "v254", "v255"
      // the barrier statements also order memory ("memory" clobber), as the
      // barriers outside them do
      if (do_pv && do_qk) {
        if (bar)
          asm volatile(TG_ASM_PVQK_BAR : TG_O_OUT, TG_ACC_OUT : TG_PV_IN, TG_QK_IN
                       : "memory", TG_RING_CLOBBERS);
        else
          asm volatile(TG_ASM_PVQK : TG_O_OUT, TG_ACC_OUT : TG_PV_IN, TG_QK_IN
                       : TG_RING_CLOBBERS);
      } else if (do_pv) {
        if (bar)
          asm volatile(TG_ASM_PV_BAR : TG_O_OUT : TG_PV_IN : "memory", TG_RING_CLOBBERS);
        else
          asm volatile(TG_ASM_PV : TG_O_OUT : TG_PV_IN : TG_RING_CLOBBERS);
      } else if (do_qk) {
        if (bar)
          asm volatile(TG_ASM_QK_BAR : TG_ACC_OUT : TG_QK_IN : "memory", TG_RING_CLOBBERS);
        else
          asm volatile(TG_ASM_QK : TG_ACC_OUT : TG_QK_IN : TG_RING_CLOBBERS);
      }
#undef TG_O_OUT
#undef TG_ACC_OUT
#undef TG_PV_IN
#undef TG_QK_IN
#undef TG_RING_CLOBBERS
      __builtin_amdgcn_s_setprio(0);
      return;
    }
    // D = 64: fragment reads one MFMA group ahead
    if (do_pv) {
      auto vfrag = [&](int blk, int u, int db) {
        const __bf16 *vb0 = Vp + (blk * 32 + 16 * u) * D;
        const bf16x4 lo = lds_read_tr4(vb0 + voff[db][0]);
        const bf16x4 hi = lds_read_tr4(vb0 + voff[db][1]);
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      };
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          bf16x8 cur = vfrag(blk, u, 0);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            bf16x8 nxt = cur;
            if (db + 1 < DB) nxt = vfrag(blk, u, db + 1);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur, pb[blk][u], o[db], 0, 0, 0);
            cur = nxt;
          }
        }
    }
    if (do_qk) {
      auto kfrag = [&](int kblk, int s) {
        return *reinterpret_cast<const bf16x8 *>(Kt + kblk * 32 * D + koff[s]);
      };
      bf16x8 a0 = kfrag(0, 0), a1 = kfrag(1, 0);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 n0 = a0, n1 = a1;
        if (s + 1 < KS) {
          n0 = kfrag(0, s + 1);
          n1 = kfrag(1, s + 1);
        }
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[s], s == 0 ? f32x16{} : acc[0],
                                                         0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[s], s == 0 ? f32x16{} : acc[1],
                                                         0, 0, 0);
        a0 = n0;
        a1 = n1;
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };
  // vector phase: softmax of tile t's scores (acc) into pb, m, l, o scale
  auto sphase = [&](int t) __attribute__((always_inline)) {
    const bool tree_tile = tree_tile_at(t);
    const int k0 = tile_k0(t);
    const int k_lim = tile_lim(t);
    if (tree_tile || k0 + BN > k_lim) {
      uint32_t tw0 = 0xffffffffu, tw1 = 0xffffffffu;
      if (tree_tile) {
        const int wj = (k0 - L) >> 5;
        tw0 = my_anc[wj];
        tw1 = wj + 1 < NW ? my_anc[wj + 1] : 0u;
      }
      // key kk = blk*32 + 8(r/4) + 4h + r%4: shifts by 4h once, then by constants
      const int lim_h = k_lim - k0 - 4 * h;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const uint32_t tw = (blk ? tw1 : tw0) >> (4 * h);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kc = blk * 32 + 8 * (r >> 2) + (r & 3);
          const bool valid = kc < lim_h && ((tw >> (kc & 31)) & 1u);
          acc[blk][r] = valid ? acc[blk][r] : -__builtin_inff();
        }
      }
    }
    // Fast path, no row maximum: every row keeps its reference m and the
    // probabilities are taken against it.  It stands when, in every lane of
    // the wave, the sum of the lane's 32 probabilities is at most
    // 32 * 2^kSlack (so each is bounded; 32 of them at most 2^kSlack always
    // pass) and no row without a reference has a visible key.  Otherwise
    // the row maxima are taken and the rows whose maximum exceeds the
    // reference by more than kSlack move it (the same decision for both
    // lanes of a row).
    auto probs = [&](float *ls) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(acc[0][r], scale2, -m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(acc[0][r + 4], scale2, -m));
        pb[0][0][r] = (__bf16)p0;
        pb[0][0][r + 4] = (__bf16)p1;
        ls[r] = p0 + p1;
      }
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int r = blk ? 0 : 8; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(acc[blk][r], scale2, -m));
          ls[r & 3] += p;
          pb[blk][r >> 3][r & 7] = (__bf16)p;
        }
    };
    float ls[4];
    probs(ls);
    float lsum = (ls[0] + ls[1]) + (ls[2] + ls[3]);
    constexpr float kFastMax = 32.0f * (1 << (int)kSlack);
    const bool fast = m_set ? lsum <= kFastMax : lsum == 0.0f;
    if (!__all(fast)) {
      float mx;
      {
        float t3[11];
#pragma unroll
        for (int i = 0; i < 10; ++i) {
          const int a = 3 * i, bb = a + 1, c = a + 2;
          t3[i] = __builtin_fmaxf(acc[a >> 4][a & 15],
                                  __builtin_fmaxf(acc[bb >> 4][bb & 15], acc[c >> 4][c & 15]));
        }
        t3[10] = __builtin_fmaxf(acc[1][14], acc[1][15]);
        const float u0 = __builtin_fmaxf(t3[0], __builtin_fmaxf(t3[1], t3[2]));
        const float u1 = __builtin_fmaxf(t3[3], __builtin_fmaxf(t3[4], t3[5]));
        const float u2 = __builtin_fmaxf(t3[6], __builtin_fmaxf(t3[7], t3[8]));
        const float u3 = __builtin_fmaxf(t3[9], t3[10]);
        mx = __builtin_fmaxf(__builtin_fmaxf(u0, u1), __builtin_fmaxf(u2, u3));
      }
      // max over the row's 64 keys, relative to the reference
      mx = fmaf(__builtin_fmaxf(mx, half_swap(mx)), scale2, -m);
      const bool need = m_set ? mx > kSlack : mx != -__builtin_inff();
      if (__any(need)) {
        // set or move the reference of the rows that need it; every other
        // row keeps its own, so a row's arithmetic never depends on its
        // neighbours (its probabilities are recomputed to the same bits)
        float shift = 0.0f, alpha = 1.0f;
        if (need) {
          shift = mx;
          if (m_set) alpha = __builtin_amdgcn_exp2f(-mx);  // else o and l are still 0
          m_set = true;
        }
        l *= alpha;
#pragma unroll
        for (int i = 0; i < DB; ++i) o[i] *= alpha;
        m += shift;
        probs(ls);
        lsum = (ls[0] + ls[1]) + (ls[2] + ls[3]);
      }
    }
    // the normaliser sums the fp32 probabilities (plain adds: the bf16 dot
    // instruction would wait for the other wave's MFMAs)
    l += lsum;
  };

  // phase barriers: the even ones leave loads in flight
  auto bar_even = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // the odd ones wait for this wave's loads of the next phase pair's tiles
  // and for its LDS reads; `younger` loads (issued after those) may stay in
  // flight.  s_waitcnt immediate: vmcnt in bits [3:0], expcnt [6:4] left at
  // its maximum (no wait), lgkmcnt [11:8] = 0.  The barrier is not
  // __syncthreads: its workgroup release fence would wait for every load
  // in flight (vmcnt(0)), the younger ones included.  The "memory" clobber
  // keeps the compiler from moving memory operations across it.
  auto bar_odd = [&](int younger) __attribute__((always_inline)) {
    if (younger >= 2 * LOADS)
      __builtin_amdgcn_s_waitcnt((2 * LOADS) | (7 << 4));
    else if (younger >= LOADS)
      __builtin_amdgcn_s_waitcnt(LOADS | (7 << 4));
    else
      __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
  };

  // The bitsets are complete (this barrier also waits for the LDS accesses
  // that built them); of the prologue's loads (K(0), K(1), V(0) in that
  // order) only K(0) is needed by pair 0, the rest land behind it.
  bar_odd(n > 1 ? 2 * LOADS : LOADS);
  // One pair of phases per j (tile j's QK^T, tile j-1's PV).  Tile j's K sits
  // in stage j % 3 and its V in stage j % 3; phase 2j requests K(j+2) and
  // V(j+1), whose stages held K(j-1) and V(j-2), last read in phase 2j-1.
  // The odd barrier of pair j needs K(j+1) and V(j) (requested in pair j-1):
  // the two requests of pair j are younger and may stay in flight.
  auto requests = [&](int j, __bf16 *kis, __bf16 *vis) __attribute__((always_inline)) {
    const bool ld_k = j + 2 < n, ld_v = j + 1 < n;
    if (ld_k) issue(kb, j + 2, kis);
    if (ld_v) issue(vb, j + 1, vis);
    return LOADS * ((int)ld_k + (int)ld_v);
  };
  // Group B's MFMA phase follows its own softmax phase and reads tiles every
  // wave could see since the last odd barrier, so at D = 128 it issues its
  // first fragment reads before the even barrier, inside its statement.
  // pairs 1 .. n-1 run both products
  auto pair = [&](int j, __bf16 *kq, __bf16 *kis, __bf16 *vis, __bf16 *vp)
                  __attribute__((always_inline)) {
    const int younger = requests(j, kis, vis);
    if (lead)
      mphase(true, vp, true, kq, false);
    else
      sphase(j - 1);
    if (lead || D != 128) bar_even();
    if (lead)
      sphase(j);
    else
      mphase(true, vp, true, kq, D == 128);
    bar_odd(younger);
  };
  if (n > 0) {
    // pair 0: QK^T of tile 0 only
    {
      const int younger = requests(0, kst2, vst1);
      if (lead) mphase(false, vst2, true, kst0, false);
      if (lead || D != 128) bar_even();
      if (lead)
        sphase(0);
      else
        mphase(false, vst2, true, kst0, D == 128);
      bar_odd(younger);
    }
    int j = 1;
    for (; j + 2 < n; j += 3) {
      pair(j, kst1, kst0, vst2, vst0);
      pair(j + 1, kst2, kst1, vst0, vst1);
      pair(j + 2, kst0, kst2, vst1, vst2);
    }
    if (j < n) pair(j, kst1, kst0, vst2, vst0);
    if (j + 1 < n) pair(j + 1, kst2, kst1, vst0, vst1);
    // pair n: PV of tile n-1 only
    const int r = (n - 1) % 3;
    __bf16 *vlast = r == 0 ? vst0 : (r == 1 ? vst1 : vst2);
    if (lead)
      mphase(true, vlast, false, kst0, false);
    else
      sphase(n - 1);
    if (lead || D != 128) bar_even();
    if (!lead) mphase(true, vlast, false, kst0, D == 128);
    bar_odd(0);
  }

  // ---- finalize: every wave is past its last read of the stages (the last
  // pair ends with a barrier); waves 2i and 2i+1 stage their rows in the
  // i-th of K stages 0-2 and V stage 0
  const float lt = l + half_swap(l);
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  const bool split_mode = n_splits > 1;
  __bf16 *ost = (w >> 1) == 0 ? kst0 : (w >> 1) == 1 ? kst1 : (w >> 1) == 2 ? kst2 : vst0;
  store_rows<D>(o, inv, ost + (w & 1) * 32 * D, split_mode ? part_o : out,
                split_mode ? ((size_t)split * B + b) * N : (size_t)b * N, row0 + w * 32,
                rows_total, G, g, Hq);
  if (split_mode && qvalid && h == 0)
    part_lse[(((size_t)split * B + b) * N + qnode) * Hq + qhead] =
        lt > 0.0f ? m + __log2f(lt) : -__builtin_inff();
}

// Merge split partials: out = sum_s 2^(lse_s - M) O_s / sum_s 2^(lse_s - M).
// One wave per query row: lane s holds split s's log-sum-exp (n_splits <=
// 64), read back wave-uniform; the bf16 partial rows are loaded eight splits
// at a time with no branch in between (an empty split has weight 0 and a
// zero row), so a round's loads are in flight together.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(
    const __bf16 *__restrict__ part_o, const float *__restrict__ part_lse,
    const int32_t *__restrict__ prefix_len, __bf16 *__restrict__ out, int B,
    int N, int Hq, int S_max, int n_splits) {
  // kLpr = D / 8 lanes per row, eight outputs each (one 16-byte load per
  // split); a wave combines kWave / kLpr rows.  Lane `sub` of a row holds
  // the log2-sum-exp of splits sub, sub + kLpr, ...  Every read is issued
  // before the prefix check (rows past the end read the last row), and the
  // splits are added in split order.
  constexpr int kLpr = D / 8, kRpw = kWave / kLpr, kSlots = kMaxSplits / kLpr;
  typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
  const int lane = threadIdx.x & (kWave - 1), sub = lane & (kLpr - 1);
  const int base = lane & ~(kLpr - 1);
  const int rows = B * N * Hq;
  const int waves = (int)(blockDim.x / kWave);
  const int gw = ((int)blockIdx.x * waves + (int)(threadIdx.x / kWave)) * kRpw + lane / kLpr;
  const int row = gw < rows ? gw : rows - 1;
  const size_t sstride = (size_t)rows * D;
  const __bf16 *po = part_o + (size_t)row * D + 8 * sub;
  const int L = prefix_len[row / (N * Hq)];
  const float ninf = -__builtin_inff();
  float ls[kSlots];
#pragma unroll
  for (int k = 0; k < kSlots; ++k) {
    const int sp = k * kLpr + sub;
    ls[k] = sp < n_splits ? part_lse[(size_t)sp * rows + row] : ninf;
  }
  bf16x8 v0[8];  // the first eight splits' values (clamped indices)
#pragma unroll
  for (int i = 0; i < 8; ++i)
    v0[i] = *reinterpret_cast<const bf16x8 *>(po + (size_t)min(i, n_splits - 1) * sstride);
  float M = ls[0];
#pragma unroll
  for (int k = 1; k < kSlots; ++k) M = fmaxf(M, ls[k]);
#pragma unroll
  for (int m = 1; m < kLpr; m <<= 1) M = fmaxf(M, __shfl_xor(M, m, kWave));
  float wl[kSlots];
#pragma unroll
  for (int k = 0; k < kSlots; ++k) wl[k] = ls[k] != ninf ? exp2f(ls[k] - M) : 0.0f;
  float acc[8] = {};
  float den = 0.0f;
#pragma unroll
  for (int k = 0; k < kSlots; ++k) {
#pragma unroll
    for (int h = 0; h < kLpr / 8; ++h) {
      const int s0 = k * kLpr + h * 8;
      if (s0 >= n_splits) break;
      bf16x8 v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v[i] = s0 == 0 ? v0[i]
                       : *reinterpret_cast<const bf16x8 *>(
                             po + (size_t)min(s0 + i, n_splits - 1) * sstride);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float w = s0 + i < n_splits ? __shfl(wl[k], base + h * 8 + i, kWave) : 0.0f;
        den += w;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(w, (float)v[i][e], acc[e]);
      }
    }
  }
  if (gw >= rows) return;
  // a sequence with a bad prefix length has no partials (its output is 0)
  const bool bad = bad_prefix(L, N, S_max);
  const float inv = den > 0.0f ? 1.0f / den : 0.0f;
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = bad ? (__bf16)0.0f : (__bf16)(acc[e] * inv);
  *reinterpret_cast<bf16x8 *>(out + (size_t)gw * D + 8 * sub) = o;
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

// Kernel choice and prefix splits of a bf16 shape.  Long prefixes over at
// least 256 query rows per KV head take the ping-pong kernel (one 8-wave
// workgroup per CU); the rest the 4-wave kernel (two per CU).  Splits bring
// the grid to about one (ping-pong) or two (4-wave) workgroups per CU; each
// split takes a run of at least 16 (ping-pong) or 2 (4-wave) key tiles.
struct AttnPlan {
  bool pingpong;
  int tiles;
  int splits;
};
static AttnPlan attn_plan(const AttnShape &s) {
  const int G = s.Hq / s.Hkv;
  const int rows = s.N * G;
  const int max_prefix = s.S_max - s.N;
  const bool pp = rows >= 256 && max_prefix >= 4096;
  const int bm = pp ? 256 : BM;
  const int tiles = (rows + bm - 1) / bm;
  const long long base = (long long)s.B * s.Hkv * tiles;
  const long long want_wgs = pp ? 256 : 512;
  // key tiles of the longest sequence, dealt out in runs of `per` tiles
  const int n_vt = (max_prefix + BN - 1) / BN + (s.N + BN - 1) / BN;
  int sp = 1;
  if (base < want_wgs) {
    // at least 3 tiles per run for the 4-wave kernel: its prologue and
    // write-out cost about as much as a tile each (Llama-3-8B shape: 11
    // splits of 3 tiles, 14.9 us per call, against 17 of 2, 15.5 us)
    const long long min_per = pp ? 16 : 3;
    const long long per = std::max(min_per, (n_vt * base + want_wgs - 1) / want_wgs);
    sp = (int)std::min<long long>(kMaxSplits, (n_vt + per - 1) / per);
  }
  return AttnPlan{pp, tiles, std::max(sp, 1)};
}

int attn_splits(const AttnShape &s) { return attn_plan(s).splits; }

size_t attn_workspace_bytes(const AttnShape &s, tg_dtype dtype) {
  if (dtype != TG_BF16) return 0;
  const int sp = attn_splits(s);
  if (sp <= 1) return 0;
  const size_t rows = (size_t)s.B * s.N * s.Hq;
  // bf16 partial rows, then fp32 log-sum-exps
  return (size_t)sp * rows * s.D * sizeof(__bf16) + (size_t)sp * rows * sizeof(float) + 256;
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
  const AttnPlan plan = attn_plan(s);
  const int tiles = plan.tiles;
  const int sp = plan.splits;
  const size_t rows = (size_t)s.B * s.N * s.Hq;
  __bf16 *part_o = sp > 1 ? reinterpret_cast<__bf16 *>(workspace) : nullptr;
  float *part_lse =
      sp > 1 ? reinterpret_cast<float *>(part_o + (size_t)sp * rows * s.D) : nullptr;
  const long long grid = (long long)s.B * s.Hkv * sp * tiles;
  const float scale2 = s.sm_scale * kLog2e;
  auto qb = reinterpret_cast<const __bf16 *>(q);
  auto kb = reinterpret_cast<const __bf16 *>(k);
  auto vb = reinterpret_cast<const __bf16 *>(v);
  auto ob = reinterpret_cast<__bf16 *>(out);
  // bitset words of the nodes one row tile can hold
  const int bm = plan.pingpong ? 256 : BM;
  const int nodes_per_tile = std::min(s.N, (bm + G - 1) / G + 1);
  // (the 4-wave kernel keeps the parent array after them)
  const size_t lds = (size_t)nodes_per_tile * ((s.N + 31) / 32) * 4 +
                     (plan.pingpong ? 0 : (size_t)s.N * 4);
  auto go = [&](auto kernel, const char *name, int threads) {
    hipError_t r = hipFuncSetAttribute((const void *)kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (r != hipSuccess) return r;
    launch(name, kernel, dim3((unsigned)grid), dim3(threads), lds, stream, qb, kb, vb, parent,
           prefix_len, ob, part_o, part_lse, s.B, s.N, s.Hq, s.Hkv, s.S_max, scale2, tiles, sp,
           d_err);
    return hipSuccess;
  };
  hipError_t e;
  if (plan.pingpong)
    e = s.D == 64 ? go(attn_pingpong_kernel<64>, "attn_pingpong", 512)
                  : go(attn_pingpong_kernel<128>, "attn_pingpong", 512);
  else
    e = s.D == 64 ? go(attn_mfma_kernel<64>, "attn_mfma", kThreads)
                  : go(attn_mfma_kernel<128>, "attn_mfma", kThreads);
  if (e != hipSuccess) return e;
  e = hipGetLastError();
  if (e != hipSuccess || sp <= 1) return e;
  // four waves per workgroup when that still makes 1024 workgroups or more,
  // else one: a small combine spread over every compute unit leaves none idle
  // for the next launch (measured: one-wave groups took the llama8b-shaped
  // call's following attention kernel back from 15.9 to 14.3 us)
  const int rows_per_wave = kWave / (s.D / 8);
  const long long waves_needed = ((long long)rows + rows_per_wave - 1) / rows_per_wave;
  const int wpb = waves_needed >= 4 * 1024 ? kThreads / kWave : 1;
  const unsigned cgrid = (unsigned)((waves_needed + wpb - 1) / wpb);
  if (s.D == 64)
    launch("attn_combine", attn_combine_kernel<64>, dim3(cgrid), dim3(wpb * kWave), 0, stream,
                       part_o, part_lse, prefix_len, ob, s.B, s.N, s.Hq, s.S_max, sp);
  else
    launch("attn_combine", attn_combine_kernel<128>, dim3(cgrid), dim3(wpb * kWave), 0, stream,
                       part_o, part_lse, prefix_len, ob, s.B, s.N, s.Hq, s.S_max, sp);
  return hipGetLastError();
}

}  // namespace tg
