// Internal device helpers shared by the HIP kernels of libtreegraft (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/treegraft.h"

namespace tg {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kWave = 64;

__device__ __forceinline__ void report(uint32_t *d_err, uint32_t bits) {
  if (d_err && bits) atomicOr(d_err, bits);
}

// ---------------------------------------------------------------- key order
// A 32-bit unsigned image of an fp32 value that orders like the float
// (-inf smallest); -0.0 is folded onto +0.0 first.
__device__ __forceinline__ uint32_t float_order(float x) {
  uint32_t b = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float order_float(uint32_t o) {
  uint32_t b = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  return __uint_as_float(b);
}

// Logits-row key: larger is better; (logit desc, token asc).  0 = empty slot
// (every real key is larger: the order image of -inf is 0x007fffff).
__device__ __forceinline__ uint64_t token_key(float x, uint32_t tok) {
  return ((uint64_t)float_order(x) << 32) | (uint64_t)(0xffffffffu - tok);
}
__device__ __forceinline__ uint32_t key_token(uint64_t k) {
  return 0xffffffffu - (uint32_t)k;
}
__device__ __forceinline__ float key_logit(uint64_t k) {
  return order_float((uint32_t)(k >> 32));
}

// Node key: larger is better; (cum desc, depth asc, id asc).  The root is
// id -1 (stored as id + 1 = 0).  Requires depth < 65536 and id < 65535.
__device__ __forceinline__ uint64_t node_key(float cum, int depth, int id) {
  uint32_t lo = 0xffffffffu - (((uint32_t)depth << 16) | (uint32_t)(id + 1));
  return ((uint64_t)float_order(cum) << 32) | lo;
}
__device__ __forceinline__ int node_key_id(uint64_t k) {
  return (int)((0xffffffffu - (uint32_t)k) & 0xffffu) - 1;
}

// NaN and +inf are read as -inf (flagged by the caller).
__device__ __forceinline__ float clean_logit(float x, bool &bad) {
  bool b = !(x < __builtin_inff());
  bad |= b;
  return b ? -__builtin_inff() : x;
}

// logp = fl(x - lse), -inf when the row has no finite logit.
__device__ __forceinline__ float edge_logp(float x, float lse) {
  return lse == -__builtin_inff() ? -__builtin_inff() : __fsub_rn(x, lse);
}

// One value that every lane needs (a live count, a flag), read through the
// vector memory path: a scalar load shares its wait counter with the
// kernel-argument loads and with LDS accesses, so the first wait for any of
// those would also wait for this global read.  load_vmem issues the read (the
// value lands in a vector register); uniform_int, called once the loads that
// need not wait for it are issued, waits for it and makes it wave-uniform.
template <typename T>
__device__ __forceinline__ T load_vmem(const T *p) {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return p[z];
}
__device__ __forceinline__ int uniform_int(int v) {
  asm volatile("" : "+v"(v));
  return __builtin_amdgcn_readfirstlane(v);
}

// ------------------------------------------------------------ wave helpers
// Wave reductions by DPP lane moves (all VALU, no LDS round trips): two quad
// swaps, row shifts by 4 and 8 (lane 15 of each row of 16 then holds the
// row's result), row broadcasts of lanes 15 and 31 into the next rows; lane
// 63 ends with the wave's result, returned to every lane.  Lanes a move
// cannot source contribute the identity.  The combination order is fixed.
// Every lane of the wave must be active.
template <int kCtrl, int kRowMask, typename T>
__device__ __forceinline__ T dpp_move(T v, T fill) {
  static_assert(sizeof(T) == 4, "32-bit lanes");
  return __builtin_bit_cast(
      T, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill), __builtin_bit_cast(int, v),
                                     kCtrl, kRowMask, 0xf, false));
}
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, T id, Op op) {
  v = op(v, dpp_move<0xb1, 0xf>(v, id));   // quad_perm [1,0,3,2]
  v = op(v, dpp_move<0x4e, 0xf>(v, id));   // quad_perm [2,3,0,1]
  v = op(v, dpp_move<0x114, 0xf>(v, id));  // row_shr:4
  v = op(v, dpp_move<0x118, 0xf>(v, id));  // row_shr:8
  v = op(v, dpp_move<0x142, 0xa>(v, id));  // row_bcast:15 into rows 1 and 3
  v = op(v, dpp_move<0x143, 0xc>(v, id));  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), kWave - 1));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  return wave_reduce(v, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}
// 64-bit keys: the high words first, then (unless one lane holds the high
// maximum) the low words of the lanes that hold it.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  const uint32_t hi = (uint32_t)(v >> 32);
  const uint32_t mh = wave_max_u32(hi);
  const uint64_t at = __ballot(hi == mh);
  if (__builtin_popcountll(at) == 1)  // one lane holds the high maximum: its key
    return ((uint64_t)mh << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, __builtin_ctzll(at));
  const uint32_t ml = wave_max_u32(hi == mh ? (uint32_t)v : 0u);
  return ((uint64_t)mh << 32) | ml;
}
// fp32 maximum through the order-preserving unsigned image (one integer DPP
// max per step; fmaxf would quiet its operands first).  -0.0 comes back as
// +0.0; a NaN with the sign bit clear orders above +inf.
__device__ __forceinline__ float wave_max_f32(float v) {
  return order_float(wave_max_u32(float_order(v)));
}
__device__ __forceinline__ float wave_sum_f32(float v) {
  return wave_reduce(v, 0.0f, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ int wave_sum_i32(int v) {
  return wave_reduce(v, 0, [](int a, int b) { return a + b; });
}

// Merge two (max, sum-of-exp relative to max) pairs in the log2 domain.
__device__ __forceinline__ void merge_ms(float &m, float &s, float m2, float s2) {
  float mn = fmaxf(m, m2);
  if (mn == -__builtin_inff()) return;  // both empty
  s = s * exp2f((m - mn) * kLog2e) + s2 * exp2f((m2 - mn) * kLog2e);
  m = mn;
}

// Descending bitonic sort of n (power of two) 64-bit keys in LDS by the whole
// block.  Callers synchronise before and the function synchronises after.
__device__ inline void block_bitonic_desc(uint64_t *a, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += blockDim.x) {
        int p = i ^ j;
        if (p > i) {
          uint64_t x = a[i], y = a[p];
          bool desc = (i & k) == 0;
          if (desc ? (x < y) : (x > y)) {
            a[i] = y;
            a[p] = x;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Exclusive prefix sum of one int per thread in thread order (waves by
// shuffles, then the wave totals); `slots` holds kBlock / kWave ints of LDS.
// Called by the whole block; ends synchronised.
template <int kBlock>
__device__ int block_exclusive_scan(int v, int *slots, int &total) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  int incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  if (lane == kWave - 1) slots[wv] = incl;
  __syncthreads();
  int before = 0;
  total = 0;
  for (int i = 0; i < kBlock / kWave; ++i) {
    before += i < wv ? slots[i] : 0;
    total += slots[i];
  }
  __syncthreads();
  return before + incl - v;
}

// ---------------------------------------------------- ranks by counting
// A key's exact rank among a small set is the number of larger keys: one pass
// over LDS broadcasts with no barrier, where a bitonic sort of the same set
// pays a barrier per stage.  Distinct keys get distinct ranks.
constexpr int kRankPerThread = 4;  // keys a thread ranks (sets up to 4 * block)

// r[j] = how many of key[0..n) are larger than mk[j] = key[threadIdx.x +
// j * kBlock] (~0, ranking nothing, past n).  n <= R * kBlock.
template <int kBlock, int R, typename P>
__device__ __forceinline__ void count_larger(P key, int n, uint64_t (&mk)[R],
                                             int (&r)[R]) {
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int i = threadIdx.x + j * kBlock;
    mk[j] = i < n ? key[i] : ~0ull;
    r[j] = 0;
  }
  int u = 0;
#pragma unroll 4
  for (; u + 1 < n; u += 2) {
    const uint64_t a = key[u], c = key[u + 1];
#pragma unroll
    for (int j = 0; j < R; ++j) r[j] += (int)(a > mk[j]) + (int)(c > mk[j]);
  }
  if (u < n) {
    const uint64_t a = key[u];
#pragma unroll
    for (int j = 0; j < R; ++j) r[j] += (int)(a > mk[j]);
  }
}

// f(i, key[i], rank of key[i]) for every i < n (n <= kRankPerThread * kBlock),
// each thread comparing as many keys as the set needs.  No synchronisation.
template <int kBlock, int R, typename Fn>
__device__ __forceinline__ void rank_each_r(const uint64_t *key, int n, Fn f) {
  uint64_t mk[R];
  int r[R];
  count_larger<kBlock, R>(key, n, mk, r);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int i = threadIdx.x + j * kBlock;
    if (i < n) f(i, mk[j], r[j]);
  }
}
template <int kBlock, typename Fn>
__device__ __forceinline__ void rank_each(const uint64_t *key, int n, Fn f) {
  if (n > 2 * kBlock)
    rank_each_r<kBlock, 4>(key, n, f);
  else if (n > kBlock)
    rank_each_r<kBlock, 2>(key, n, f);
  else
    rank_each_r<kBlock, 1>(key, n, f);
}

// Moves the k largest of key[0..n) (distinct; 0 = no key) to key[0..k), best
// first, 0 in the places past the last present key; what lies past
// min(k, n) is undefined afterwards.  Sets up to kRankPerThread * kBlock are
// ranked by counting (each thread compares as many keys as the set needs),
// larger ones sorted whole: then key[n..P2) must hold 0, P2 a power of two
// >= n.  Callers synchronise before; ends synchronised.
template <int kBlock, int R, typename P>
__device__ void block_top_keys_r(P key, int n, int k) {
  uint64_t mk[R];
  int r[R];
  count_larger<kBlock, R, P>(key, n, mk, r);
  __syncthreads();
  for (int j = threadIdx.x; j < k && j < n; j += kBlock) key[j] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < R; ++j)
    if (threadIdx.x + j * kBlock < n && mk[j] != 0 && r[j] < k) key[r[j]] = mk[j];
  __syncthreads();
}

// Descending bitonic sort of one 64-bit key per lane across the wave.
__device__ __forceinline__ uint64_t wave_sort_desc_u64(uint64_t v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint64_t p = __shfl_xor(v, j, kWave);
      const bool take_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = take_max ? (p > v ? p : v) : (p < v ? p : v);
    }
  }
  return v;
}

// The k-th and kq-th largest (kq <= k <= 64) of the wave's keys, 0 when
// fewer lanes hold a present (non-zero) key; keys are distinct.  Small k:
// rounds of "take the wave maximum, retire its lane"; larger k: a wave sort.
__device__ __forceinline__ void wave_key_order_stats(uint64_t v, int k, int kq, uint64_t &tk,
                                                     uint64_t &tq) {
  tk = 0;
  tq = 0;
  if (k > 16) {
    const uint64_t srt = wave_sort_desc_u64(v);
    const uint32_t lo = (uint32_t)srt, hi = (uint32_t)(srt >> 32);
    tk = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, k - 1) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)lo, k - 1);
    tq = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, kq - 1) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)lo, kq - 1);
    return;
  }
  for (int j = 0; j < k; ++j) {
    const uint64_t mx = wave_max_u64(v);
    if (mx == 0) return;
    if (j == kq - 1) tq = mx;
    if (j == k - 1) tk = mx;
    v = v == mx ? 0 : v;
  }
}

// block_top_keys for a small k against a larger set (n <= kRankPerThread *
// kBlock): the keys are dealt round-robin over the waves, so each wave holds
// about n / waves of them, and each wave's ceil(k / waves)-th largest thread
// maximum is found (that many rounds of wave maxima); the smallest of those,
// T, has at least k present keys at or above it (every wave holds that many
// distinct thread maxima >= T), so only the keys >= T are compacted to the
// front and ranked by counting, by wave 0 alone when at most a wave's width
// of them remain.  A wave with too few keys gives T = 0 (every key ranked).
// Same contract as block_top_keys.  Kept out of line: the common small sets
// take the inlined counting paths.
template <int kBlock>
__device__ __noinline__ void block_select_top(uint64_t *key_generic, int n, int k) {
  // out of line, so a generic pointer would cost an address conversion (with
  // a null check) per access; the keys live in LDS
  using lds_u64 = __attribute__((address_space(3))) uint64_t;
  lds_u64 *key = (lds_u64 *)key_generic;
  constexpr int kW = kBlock / kWave;
  __shared__ uint64_t bnd_s[kW];
  __shared__ int cnt_s;
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  uint64_t mk[kRankPerThread];
  uint64_t tmax = 0;
#pragma unroll
  for (int j = 0; j < kRankPerThread; ++j) {
    const int i = j * kBlock + lane * kW + w;
    mk[j] = i < n ? key[i] : 0;
    tmax = mk[j] > tmax ? mk[j] : tmax;
  }
  const int kq = (k + kW - 1) / kW;
  uint64_t tq = 0;
  if (kq <= 4) {
    uint64_t unused;
    wave_key_order_stats(tmax, kq, kq, tq, unused);
  } else {
    // the kq-th largest thread maximum of the wave by counting the larger
    // ones among the wave's 64 (LDS broadcasts within the wave)
    __shared__ uint64_t tm_s[kW][kWave];
    tm_s[w][lane] = tmax;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int r = 0;
#pragma unroll 8
    for (int j = 0; j < kWave; ++j) r += (int)(tm_s[w][j] > tmax);
    const uint64_t hit = __ballot(tmax != 0 && r == kq - 1);
    if (hit) {
      const int src = __builtin_ctzll(hit);
      tq = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(tmax >> 32), src) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)tmax, src);
    }
  }
  if (lane == 0) bnd_s[w] = tq;
  if (threadIdx.x == 0) cnt_s = 0;
  __syncthreads();
  uint64_t T = ~0ull;
#pragma unroll
  for (int i = 0; i < kW; ++i) T = bnd_s[i] < T ? bnd_s[i] : T;
#pragma unroll
  for (int j = 0; j < kRankPerThread; ++j)
    if (mk[j] != 0 && mk[j] >= T) key[atomicAdd(&cnt_s, 1)] = mk[j];
  __syncthreads();
  const int c = cnt_s;
  for (int j = c + threadIdx.x; j < k && j < n; j += kBlock) key[j] = 0;
  if (c <= kWave) {
    // wave 0: lane l ranks candidate l against the others (LDS broadcasts;
    // the wave's reads are done before its writes, in issue order)
    if (w == 0) {
      const uint64_t mine = lane < c ? key[lane] : 0;
      int r = 0;
      int u = 0;
#pragma unroll 4
      for (; u + 1 < c; u += 2) r += (int)(key[u] > mine) + (int)(key[u + 1] > mine);
      if (u < c) r += (int)(key[u] > mine);
      if (lane < c && r < k) key[r] = mine;
    }
    __syncthreads();
  } else if (c > 2 * kBlock) {
    block_top_keys_r<kBlock, 4, lds_u64 *>(key, c, k);
  } else if (c > kBlock) {
    block_top_keys_r<kBlock, 2, lds_u64 *>(key, c, k);
  } else {
    block_top_keys_r<kBlock, 1, lds_u64 *>(key, c, k);
  }
}

// block_top_keys for 1 <= k <= 16 and at most one key per thread: the keys
// are dealt round-robin over the waves; each wave ranks its own keys against
// its own (LDS broadcasts of a quarter of the set, no barrier) and keeps
// those of local rank < k (a key of the k largest has fewer than k larger
// keys in its wave), then wave 0 ranks the at most waves * k survivors the
// same way and writes the result.  Two barriers.  Same contract as
// block_top_keys.
template <int kBlock>
__device__ void block_small_top(uint64_t *key, int n, int k) {
  constexpr int kW = kBlock / kWave;
  static_assert(kW * 16 <= kWave, "survivors fit one wave");
  __shared__ uint64_t cand_s[kW * 16];
  __shared__ int ncand_s[kW];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int i = lane * kW + w;
  const uint64_t mine = i < n ? key[i] : 0;
  const int nw = n > w ? (n - w + kW - 1) / kW : 0;  // keys of this wave: key[j * kW + w]
  int r = 0;
  int j = 0;
#pragma unroll 4
  for (; j + 1 < nw; j += 2) {
    const uint64_t a = key[j * kW + w], c = key[(j + 1) * kW + w];
    r += (int)(a > mine) + (int)(c > mine);
  }
  if (j < nw) r += (int)(key[j * kW + w] > mine);
  const int present = __builtin_popcountll(__ballot(mine != 0));
  const int nc = present < k ? present : k;
  if (mine != 0 && r < k) cand_s[w * k + r] = mine;
  if (lane >= nc && lane < k) cand_s[w * k + lane] = 0;
  if (lane == 0) ncand_s[w] = nc;
  __syncthreads();
  if (w == 0) {
    const int m = kW * k;
    const uint64_t c = lane < m ? cand_s[lane] : 0;
    int tot = 0;
#pragma unroll
    for (int u = 0; u < kW; ++u) tot += ncand_s[u];
    int rr = 0;
    int u = 0;
#pragma unroll 4
    for (; u + 1 < m; u += 2) rr += (int)(cand_s[u] > c) + (int)(cand_s[u + 1] > c);
    if (u < m) rr += (int)(cand_s[u] > c);
    if (c != 0 && rr < k) key[rr] = c;
    if (lane >= tot && lane < k && lane < n) key[lane] = 0;
  }
  __syncthreads();
}

// sets of more keys than this, up to one per thread, take block_small_top
// for k <= 16 (larger ones block_select_top)
constexpr int kSmallFrom = 32;
template <int kBlock>
__device__ void block_top_keys(uint64_t *key, int n, int P2, int k) {
  if (n > kRankPerThread * kBlock) {
    block_bitonic_desc(key, P2);
  } else if (k >= 1 && k <= 16 && n > kSmallFrom && n <= kBlock) {
    block_small_top<kBlock>(key, n, k);
  } else if ((k <= 16 && n > kBlock) || (k <= kWave && n > 2 * kBlock)) {
    block_select_top<kBlock>(key, n, k);
  } else if (n > 2 * kBlock) {
    block_top_keys_r<kBlock, 4>(key, n, k);
  } else if (n > kBlock) {
    block_top_keys_r<kBlock, 2>(key, n, k);
  } else {
    block_top_keys_r<kBlock, 1>(key, n, k);
  }
}

// ------------------------------------------------------- finishing rows
// log-sum-exp of one row from its per-grain (max, sum-exp) partials, by one
// wave (every lane calls it; the result is the same in all): the grains 64
// at a time, each batch folded as a fixed pairwise tree over the lanes (lane
// l takes lane l + d for d = 1, 2, 4, ... while l is a multiple of 2d), the
// batches in order.  The partials are per grain, so this is the same bits
// whatever the call's chunking.  `first` is the lane's partial of the first
// batch (ms[lane] for lane < n, already loaded by the caller).
__device__ inline float wave_fold_lse(const float2 *__restrict__ ms, int n, float2 first) {
  const int lane = threadIdx.x & (kWave - 1);
  float m = -__builtin_inff(), s = 0.0f;
  for (int i0 = 0; i0 < n; i0 += kWave) {
    const int cnt = n - i0 < kWave ? n - i0 : kWave;
    float2 p = first;
    if (i0 > 0) p = lane < cnt ? ms[i0 + lane] : make_float2(-__builtin_inff(), 0.0f);
    float bm = p.x, bs = p.y;
    for (int d = 1; d < cnt; d <<= 1) {
      const float om = __shfl_down(bm, d, kWave), os = __shfl_down(bs, d, kWave);
      if ((lane & (2 * d - 1)) == 0 && lane + d < cnt) merge_ms(bm, bs, om, os);
    }
    merge_ms(m, s, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bm), 0)),
             __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bs), 0)));
  }
  return m == -__builtin_inff() ? -__builtin_inff() : m + logf(s);
}

// K-round merge of one row's `chunks` sorted lists (each K keys, best
// first) staged in LDS at `lists`: lane c holds list c's head, the wave takes
// the largest head, that list advances.  Lane j < K returns the j-th best key.
__device__ inline uint64_t wave_merge_lists(const uint64_t *lists, int chunks, int K) {
  const int lane = threadIdx.x & (kWave - 1);
  const bool own = lane < chunks;
  // the head and the entry after it sit in registers, so the LDS read that
  // refills them overlaps the next round's reduction
  uint64_t head = own ? lists[lane * K] : 0;
  uint64_t next = own && K > 1 ? lists[lane * K + 1] : 0;
  int idx = 1;
  uint64_t mine = 0;
  for (int j = 0; j < K; ++j) {
    const uint64_t best = wave_max_u64(head);
    if (head == best && best != 0) {
      head = next;
      ++idx;
      next = own && idx < K ? lists[lane * K + idx] : 0;
    }
    if (lane == j) mine = best;
  }
  return mine;
}

// One wave finishes one row's top-K: lane j < K returns the j-th best key.
// `ws` is this wave's LDS scratch (chunks * K keys).  chunks <= 64.  The
// lists are staged four loads per lane at a time, one wait per batch.
__device__ inline uint64_t wave_finish_topk(const uint64_t *__restrict__ lists, int chunks, int K,
                                     uint64_t *ws) {
  const int lane = threadIdx.x & (kWave - 1);
  if (chunks == 1) return lane < K ? lists[lane] : 0;
  const int nk = chunks * K;
  for (int i0 = 0; i0 < nk; i0 += 4 * kWave) {
    uint64_t t[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kWave + lane;
      t[u] = i < nk ? lists[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kWave + lane;
      if (i < nk) ws[i] = t[u];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint64_t r = wave_merge_lists(ws, chunks, K);
  __builtin_amdgcn_wave_barrier();   // ws is reused by the wave's next row
  return r;
}

__host__ __device__ constexpr int pow2_at_least(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

}  // namespace tg
