// Register-resident top-K lists and log-sum-exp pairs for the projection
// epilogue and the row merge.
//
// A candidate (logit value v, token id i) is packed into one 64-bit key that
// orders exactly like the search's ranking key: larger value first, equal
// values by smaller token id. High word: the float's bits mapped to an
// order-preserving unsigned integer; low word: ~i. Key 0 is "empty" and
// ranks below every real candidate (even a -inf logit).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace sb {

typedef unsigned long long cand_key;

__device__ __forceinline__ cand_key make_key(float v, int idx) {
  // Negative values: all bits flipped; others: the sign bit set.
  const uint32_t u = __float_as_uint(v);
  const uint32_t o = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
  return ((cand_key)o << 32) | (uint32_t)(~idx);
}
__device__ __forceinline__ float key_val(cand_key k) {
  uint32_t u = (uint32_t)(k >> 32);
  u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(u);
}
__device__ __forceinline__ int key_idx(cand_key k) { return (int)(~(uint32_t)k); }

template <int K>
struct TopK {
  cand_key k[K];   // sorted, best first
};

template <int K>
__device__ __forceinline__ void topk_init(TopK<K> &t) {
#pragma unroll
  for (int j = 0; j < K; ++j) t.k[j] = 0ull;
}

// Compare-exchange: after it, a holds the larger key when `desc`.
__device__ __forceinline__ void cex(cand_key &a, cand_key &b, bool desc) {
  const bool sw = desc ? (b > a) : (a > b);
  const cand_key x = sw ? b : a, y = sw ? a : b;
  a = x;
  b = y;
}

// out <- the 2N keys of a and b (each sorted best first) sorted best first:
// a followed by b reversed is bitonic, and half-cleaners sort it.
template <int N>
__device__ __forceinline__ void merge_sorted(const cand_key *a, const cand_key *b, cand_key *out) {
#pragma unroll
  for (int j = 0; j < N; ++j) {
    out[j] = a[j];
    out[N + j] = b[N - 1 - j];
  }
#pragma unroll
  for (int st = N; st > 0; st >>= 1)
#pragma unroll
    for (int j = 0; j < 2 * N; ++j)
      if ((j & st) == 0) cex(out[j], out[j + st], true);
}

// Sort N keys (N a power of two) best first with a bitonic network.
template <int N>
__device__ __forceinline__ void bitonic_sort_desc(cand_key *a) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) cex(a[i], a[l], (i & k) == 0);
      }
}

// a <- best K of (a union b); both sorted best first. Pairing a[j] with
// b[K-1-j] keeps the K best as a bitonic sequence; half-cleaners sort it.
template <int K>
__device__ __forceinline__ void topk_merge(TopK<K> &a, const TopK<K> &b) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const cand_key o = b.k[K - 1 - j];
    a.k[j] = a.k[j] > o ? a.k[j] : o;
  }
#pragma unroll
  for (int s = K / 2; s > 0; s >>= 1)
#pragma unroll
    for (int j = 0; j < K; ++j)
      if ((j & s) == 0) cex(a.k[j], a.k[j + s], true);
}

template <int K>
__device__ __forceinline__ void topk_shfl_xor(TopK<K> &out, const TopK<K> &in, int mask) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const uint32_t lo = __shfl_xor((uint32_t)in.k[j], mask, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(in.k[j] >> 32), mask, 64);
    out.k[j] = ((cand_key)hi << 32) | lo;
  }
}

// Stored as two 32-bit words (low, high) in a float array.
template <int K>
__device__ __forceinline__ void topk_store(float *p, const TopK<K> &t) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    p[2 * j] = __uint_as_float((uint32_t)t.k[j]);
    p[2 * j + 1] = __uint_as_float((uint32_t)(t.k[j] >> 32));
  }
}
template <int K>
__device__ __forceinline__ void topk_load(TopK<K> &t, const float *p) {
#pragma unroll
  for (int j = 0; j < K; ++j)
    t.k[j] = ((cand_key)__float_as_uint(p[2 * j + 1]) << 32) | __float_as_uint(p[2 * j]);
}

// Floats per partial record (max, sum exp, kb keys as two words each),
// padded to a multiple of 4 so that records are 16-byte aligned.
__host__ __device__ constexpr int part_width(int kb) { return (2 + 2 * kb + 3) & ~3; }

// Short per-(row, vocabulary tile) key list of the projection, used when the
// vocabulary has many tiles: a tile holding more of a row's best k than
// this is found by the row merge (its last kept key still ranks among the
// best k) and recomputed there; with few tiles that is common, and the list
// holds the full k-bucket instead.
constexpr int TILE_KEYS_SHORT = 4;

// The best 4 of 16 keys, sorted: four groups of 4 sorted by the 5-exchange
// network, merged pairwise keeping the best 4.
__device__ __forceinline__ void top4_of_16(cand_key *a, TopK<4> &out) {
  TopK<4> g[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    cand_key *k = g[x].k;
#pragma unroll
    for (int j = 0; j < 4; ++j) k[j] = a[4 * x + j];
    cex(k[0], k[1], true);
    cex(k[2], k[3], true);
    cex(k[0], k[2], true);
    cex(k[1], k[3], true);
    cex(k[1], k[2], true);
  }
  topk_merge(g[0], g[1]);
  topk_merge(g[2], g[3]);
  topk_merge(g[0], g[2]);
  out = g[0];
}

// Insert one key into a sorted list (the smallest key falls off).
template <int K>
__device__ __forceinline__ void topk_insert(TopK<K> &t, cand_key x) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const cand_key hi = t.k[j] > x ? t.k[j] : x;
    x = t.k[j] > x ? x : t.k[j];
    t.k[j] = hi;
  }
}

// (m, s) represents log(s) + m: a running max and a sum of exp(z - m).
__device__ __forceinline__ void lse_merge(float &m, float &s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;
  s = s * __expf(m - M) + s2 * __expf(m2 - M);
  m = M;
}

}  // namespace sb
