// Length-dependent decoder step: the projection input of a row is
// x = bf16(h + (1/L) sum_l a_l), a_l = sum_s softmax_s(K_l[s] . h / sqrt(d)) V_l[s]
// over the candidate's own KV rows s = 0 .. t-1 (row s is stored at
// (beam, s, rank of its ancestor at level s); the current step's row at the
// candidate's own rank). This is the self-attention whose cost grows with
// the output position (App. A.2, Fig. 2).
//
// All arithmetic after the bf16 loads is fp64: products of bf16 values are
// exact there and the sums lose nothing in practice, so the rounded x does
// not depend on summation order (the same reasoning as the bf16 recurrence).
//
// Two kernels: k_attn computes a_l of one (row, layer) per workgroup visit
// into an fp64 scratch [R][L][d] (so the layers of a row run side by side),
// k_attn_combine adds the layers in order and rounds x.
#include <math.h>

#include "sb_internal.h"
#include "bf16_round.h"

namespace sb {
namespace {

constexpr int AT_THREADS = 256;   // 4 waves

__device__ __forceinline__ double bf_to_d(uint32_t bits16) { return (double)__uint_as_float(bits16 << 16); }

template <int E>
struct Vec;
template <>
struct Vec<1> { typedef uint16_t t; };
template <>
struct Vec<2> { typedef uint32_t t; };
template <>
struct Vec<4> { typedef unsigned int t __attribute__((ext_vector_type(2))); };
template <>
struct Vec<8> { typedef unsigned int t __attribute__((ext_vector_type(4))); };

// E bf16 values (2E bytes) as 16-bit codes.
template <int E>
__device__ __forceinline__ void load_bf(const uint16_t *p, uint32_t (&out)[E]) {
  const typename Vec<E>::t v = *reinterpret_cast<const typename Vec<E>::t *>(p);
  if constexpr (E == 1) {
    out[0] = v;
  } else if constexpr (E == 2) {
    out[0] = v & 0xFFFFu;
    out[1] = v >> 16;
  } else {
#pragma unroll
    for (int i = 0; i < E / 2; ++i) {
      out[2 * i] = v[i] & 0xFFFFu;
      out[2 * i + 1] = v[i] >> 16;
    }
  }
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// d = 256 E. Lane l of wave w owns columns w d/4 + l E .. + E - 1 (the V
// pass), and for the K pass the four pieces p d/4 + l E .. + E - 1.
// Persistent over the R*L (row, layer) pairs.
template <int E>
__global__ __launch_bounds__(AT_THREADS) void k_attn(DevState st) {
  extern __shared__ double sc[];   // [max_len_cap] scores, then weights; then the ranks
  __shared__ double red[4];
  const int R = st.ctrl->R;
  const int d = st.d, L = st.kv_layers, planes = 2 * L, k = st.k;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int q4 = d / 4;
  const double scale = 1.0 / sqrt((double)d);
  uint8_t *arank = reinterpret_cast<uint8_t *>(sc + st.max_len_cap);   // [max_len_cap]
  const uint16_t *hb = static_cast<const uint16_t *>(st.hbuf);

  // Pairs in layer-major order (rows come in beam order, so the siblings
  // that share ancestor rows are adjacent); XCD x walks the x-th eighth of
  // the list, so siblings read those rows through one L2.
  const int T = R * L;
  const int xcd = blockIdx.x & 7, gx = gridDim.x >> 3;
  const int lo = (int)((long long)T * xcd / 8), hi = (int)((long long)T * (xcd + 1) / 8);
  for (int pr = lo + (int)(blockIdx.x >> 3); pr < hi; pr += gx) {
    const int l = pr / R, r = pr - l * R;
    const int slot = st.r_slot[r];
    const int t = st.r_t[r];                         // positions, the new one included
    const int b = slot / k;
    // Rank of the candidate whose expansion wrote position s: its ancestors'
    // (current ancestry buffer of the beam), then its own.
    const uint8_t *an = st.anc + ((size_t)st.b_par[b] * st.n * k + slot) * st.anc_stride;
    for (int s = threadIdx.x; s < t - 1; s += AT_THREADS) arank[s] = (uint8_t)min((int)an[s], k - 1);
    if (threadIdx.x == 0) arank[t - 1] = (uint8_t)(slot - b * k);
    __syncthreads();
    const uint16_t *kvb = st.kvs + (size_t)b * st.max_len_cap * k * planes * d;
    // Query (this row's new state), the lane's four K-pass pieces.
    double q[4][E];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t c[E];
      load_bf<E>(hb + (size_t)r * d + p * q4 + lane * E, c);
#pragma unroll
      for (int e = 0; e < E; ++e) q[p][e] = bf_to_d(c[e]);
    }
    {
      // Row of position s in plane j of this layer.
      auto row_of = [&](int s, int j) {
        return kvb + (((size_t)s * k + arank[s]) * planes + 2 * l + j) * d;
      };
      // Scores: wave w takes positions s = w, w + 4, ..., four at a time
      // (their loads issued together; positions past t re-read the last row
      // and are dropped).
      double mx = -INFINITY;
      for (int s0 = w; s0 < t; s0 += 16) {
        uint32_t c[4][4][E];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint16_t *row = row_of(min(s0 + 4 * u, t - 1), 0);
#pragma unroll
          for (int p = 0; p < 4; ++p) load_bf<E>(row + p * q4 + lane * E, c[u][p]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          double part = 0.0;
#pragma unroll
          for (int p = 0; p < 4; ++p)
#pragma unroll
            for (int e = 0; e < E; ++e) part = fma(q[p][e], bf_to_d(c[u][p][e]), part);
          const int s = s0 + 4 * u;
          const double sv = wave_sum_d(part) * scale;
          if (s < t) {
            if (lane == 0) sc[s] = sv;
            mx = fmax(mx, sv);
          }
        }
      }
      if (lane == 0) red[w] = mx;
      __syncthreads();
      const double m = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
      __syncthreads();
      // Weights exp(s - max) and their sum (fixed order: lanes, then waves).
      double ls = 0.0;
      for (int s = threadIdx.x; s < t; s += AT_THREADS) {
        const double ev = exp(sc[s] - m);
        sc[s] = ev;
        ls += ev;
      }
      ls = wave_sum_d(ls);
      if (lane == 0) red[w] = ls;
      __syncthreads();
      const double den = (red[0] + red[1]) + (red[2] + red[3]);
      // Read-out over the lane's columns, positions in order.
      double a[E];
#pragma unroll
      for (int e = 0; e < E; ++e) a[e] = 0.0;
      const int col = w * q4 + lane * E;
#pragma unroll 4
      for (int s = 0; s < t; ++s) {
        const uint16_t *row = row_of(s, 1);
        uint32_t c[E];
        load_bf<E>(row + col, c);
        const double ws = sc[s];
#pragma unroll
        for (int e = 0; e < E; ++e) a[e] = fma(ws, bf_to_d(c[e]), a[e]);
      }
      double *out = st.attn_part + ((size_t)r * L + l) * d + col;
#pragma unroll
      for (int e = 0; e < E; ++e) out[e] = a[e] / den;
      __syncthreads();   // sc, red and arank are rewritten by the next pair
    }
  }
}

// x[r][j] = bf16(h[r][j] + (a_0 + a_1 + ... + a_{L-1})[j] / L), layers added
// in order. One thread per 4 columns.
__global__ __launch_bounds__(AT_THREADS) void k_attn_combine(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d, L = st.kv_layers, nq = d / 4;
  const uint16_t *hb = static_cast<const uint16_t *>(st.hbuf);
  uint16_t *xb = static_cast<uint16_t *>(st.xbuf);
  for (int i = blockIdx.x * AT_THREADS + threadIdx.x; i < R * nq; i += gridDim.x * AT_THREADS) {
    const int r = i / nq, j = (i - r * nq) * 4;
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    for (int l = 0; l < L; ++l) {
      const double *p = st.attn_part + ((size_t)r * L + l) * d + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] += p[e];
    }
    uint32_t c[4];
    load_bf<4>(hb + (size_t)r * d + j, c);
    unsigned int o[2];
#pragma unroll
    for (int e = 0; e < 2; ++e)
      o[e] = (uint32_t)bf16_rne_from_double(bf_to_d(c[2 * e]) + s[2 * e] / (double)L) |
             ((uint32_t)bf16_rne_from_double(bf_to_d(c[2 * e + 1]) + s[2 * e + 1] / (double)L) << 16);
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    *reinterpret_cast<u2 *>(xb + (size_t)r * d + j) = u2{o[0], o[1]};
  }
}

}  // namespace

hipError_t launch_attn(const DevState &st, hipStream_t s) {
  const int G = (std::min(st.R_max * st.kv_layers, st.n_cu * 8) + 7) / 8 * 8;   // a multiple of the 8 XCDs
  const size_t lds = (size_t)st.max_len_cap * (sizeof(double) + 1);
  switch (st.d) {
    case 256: hipLaunchKernelGGL(k_attn<1>, dim3(G), dim3(AT_THREADS), lds, s, st); break;
    case 512: hipLaunchKernelGGL(k_attn<2>, dim3(G), dim3(AT_THREADS), lds, s, st); break;
    case 1024: hipLaunchKernelGGL(k_attn<4>, dim3(G), dim3(AT_THREADS), lds, s, st); break;
    case 2048: hipLaunchKernelGGL(k_attn<8>, dim3(G), dim3(AT_THREADS), lds, s, st); break;
    default: return hipErrorInvalidValue;
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int G2 = std::min((st.R_max * (st.d / 4) + AT_THREADS - 1) / AT_THREADS, st.n_cu * 4);
  hipLaunchKernelGGL(k_attn_combine, dim3(G2), dim3(AT_THREADS), 0, s, st);
  return hipGetLastError();
}

}  // namespace sb
