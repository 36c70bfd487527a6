// Register-resident top-K lists and log-sum-exp pairs for the projection
// epilogue and the row merge. Order: larger value first; equal values are
// ordered by smaller token id (the ranking key of the search).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace sb {

constexpr int TOPK_NONE = 0x7fffffff;

template <int K>
struct TopK {
  float v[K];
  int i[K];
};

__device__ __forceinline__ bool key_beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

template <int K>
__device__ __forceinline__ void topk_init(TopK<K> &t) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    t.v[j] = -INFINITY;
    t.i[j] = TOPK_NONE;
  }
}

// Insert a value whose id is larger than every id already inserted (ids are
// pushed in increasing order), so strict '>' keeps equal values in id order.
template <int K>
__device__ __forceinline__ void topk_push_ordered(TopK<K> &t, float v, int id) {
  if (v > t.v[K - 1]) {
#pragma unroll
    for (int j = K - 1; j > 0; --j) {
      const bool up = v > t.v[j - 1];
      const bool here = v > t.v[j];
      const float nv = up ? t.v[j - 1] : (here ? v : t.v[j]);
      const int ni = up ? t.i[j - 1] : (here ? id : t.i[j]);
      t.v[j] = nv;
      t.i[j] = ni;
    }
    if (v > t.v[0]) {
      t.v[0] = v;
      t.i[0] = id;
    }
  }
}

// a <- best K of (a union b); both sorted. Bitonic: pairing a[j] with
// b[K-1-j] keeps the K best in a bitonic sequence, half-cleaners sort it.
template <int K>
__device__ __forceinline__ void topk_merge(TopK<K> &a, const TopK<K> &b) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const float bv = b.v[K - 1 - j];
    const int bi = b.i[K - 1 - j];
    if (!key_beats(a.v[j], a.i[j], bv, bi)) {
      a.v[j] = bv;
      a.i[j] = bi;
    }
  }
#pragma unroll
  for (int s = K / 2; s > 0; s >>= 1) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      if ((j & s) == 0) {
        const float v0 = a.v[j], v1 = a.v[j + s];
        const int i0 = a.i[j], i1 = a.i[j + s];
        const bool sw = key_beats(v1, i1, v0, i0);
        a.v[j] = sw ? v1 : v0;
        a.i[j] = sw ? i1 : i0;
        a.v[j + s] = sw ? v0 : v1;
        a.i[j + s] = sw ? i0 : i1;
      }
    }
  }
}

template <int K>
__device__ __forceinline__ void topk_shfl_xor(TopK<K> &out, const TopK<K> &in, int mask) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    out.v[j] = __shfl_xor(in.v[j], mask, 64);
    out.i[j] = __shfl_xor(in.i[j], mask, 64);
  }
}

// (m, s) represents log(s) + m: a running max and a sum of exp(z - m).
__device__ __forceinline__ void lse_merge(float &m, float &s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;
  s = s * expf(m - M) + s2 * expf(m2 - M);
  m = M;
}

}  // namespace sb
