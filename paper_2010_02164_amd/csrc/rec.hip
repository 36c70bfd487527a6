// Recurrence of the synthetic decoder D (Sec. 2) on gfx950 MFMA:
//   h = tanh(W_h h_prev + E[y])      [R,d] x [d,d]^T, fused epilogue
// W_h (out-feature rows) is the MFMA A operand and the previous states the B
// operand, both K-contiguous. bf16 workloads accumulate in fp64 (see k_rec_bf16).
#include <algorithm>
#include <type_traits>

#include "bf16_round.h"
#include "mfma_common.h"

namespace sb {
namespace {

// ---------------------------------------------------------------- K_rec
// The recurrence GEMM is small ([R,d] x [d,d]) next to the projection, so it
// is cut into 32 (out features) x 32 (rows) tiles to reach hundreds of
// workgroups, and the K loop of each tile is split over the RSPLIT = 8 waves
// of the workgroup (a 128-wide K slice each at d = 1024); the 8 partial sums
// are added in a fixed order (wave 0 + 1 + ... + 7), so the result does not
// depend on which rows share the step. Operands
// are read straight from global memory (W_h and the states are L2/MALL
// resident); each lane loads the 16 bytes it feeds to the MFMA.
constexpr int RT = 32;          // tile edge
constexpr int RSPLIT = 8;       // K split over the waves of a workgroup
constexpr int RTHREADS = 64 * RSPLIT;
// Row stride of the reduction buffer: one value more than a tile row, so
// that the lanes of a store (consecutive rows, same feature) fall in
// different LDS banks (a 32-value stride puts them all in one).
constexpr int RS = RT + 1;

__device__ __forceinline__ const unsigned char *rec_state_row(const DevState &st, int r, int R, int rowbytes) {
  return state_row(st, min(r, R - 1), rowbytes);
}

__device__ __forceinline__ void rec_tile_f32(const DevState &st, float (*red)[RT * RS], int vt, int rt, int R) {
  const int d = st.d;
  const int v0 = vt * RT, r0 = rt * RT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rowbytes = d * 4;
  const int kq = d / RSPLIT;                       // K range of this wave (multiple of 8)
  // Epilogue mapping: thread -> row j = tid/16, features 2*(tid%16)..+1. Its
  // embedding values are fetched before the K loop so that their latency
  // overlaps the GEMM.
  const int j = threadIdx.x >> 4, i0 = (threadIdx.x & 15) * 2;
  const int row = r0 + j;
  float ev[2] = {0.0f, 0.0f};
  if (row < R) {
    const float *E = static_cast<const float *>(st.E) + (size_t)st.r_y[row] * d + v0 + i0;
    ev[0] = E[0];
    ev[1] = E[1];
  }
  // A: this wave's K slice of the fragment-ordered W_h copy, one coalesced
  // 1 KB block per 8 K values (lane (h, l): row v0 + l, K + 4h .. +3).
  const f4 *afr = reinterpret_cast<const f4 *>(st.wh_t) + ((size_t)vt * (d / 8) + (w * kq) / 8) * 64 + lane;
  const float *brow = reinterpret_cast<const float *>(rec_state_row(st, r0 + (lane & 31), R, rowbytes)) + w * kq;
  const int h = (lane >> 5) * 4;
  f16v acc = {};
  // K permutation: lanes 0-31 feed k = kk + e, lanes 32-63 k = kk + 4 + e.
  // Blocks of 128 K values have all their loads issued before their MFMAs
  // (the MFMA order is unchanged); the rest goes 8 at a time.
  int kk = 0;
  for (; kk + 128 <= kq; kk += 128) {
    f4 a[16], b[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      a[i] = afr[(size_t)(kk / 8 + i) * 64];
      b[i] = *reinterpret_cast<const f4 *>(brow + kk + 8 * i + h);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[i][e], acc, 0, 0, 0);
  }
#pragma unroll 8
  for (; kk < kq; kk += 8) {
    const f4 a = afr[(size_t)(kk / 8) * 64];
    const f4 b = *reinterpret_cast<const f4 *>(brow + kk + h);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
  }
  // acc: out feature i = 8*(reg/4) + 4*(lane/32) + reg%4, row j = lane%32.
#pragma unroll
  for (int reg = 0; reg < 16; ++reg) {
    const int i = 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
    red[w][(lane & 31) * RS + i] = acc[reg];
  }
  __syncthreads();
  if (row < R) {
    float hv[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int o = j * RS + i0 + q;
      float pre = red[0][o];
#pragma unroll
      for (int x = 1; x < RSPLIT; ++x) pre += red[x][o];   // fixed order
      hv[q] = tanhf(pre + ev[q]);
    }
    float *out = static_cast<float *>(st.hbuf) + (size_t)row * d + v0 + i0;
    out[0] = hv[0];
    out[1] = hv[1];
  }
}

// bf16 states are rounded after tanh, a discontinuous map: any difference
// in the pre-activation can flip a rounding and then grows step after step.
// Products of two bf16 values are exact in fp64 and so is their sum over
// the state size in practice, so the pre-activation is accumulated with the
// fp64 MFMA (16x16x4), tanh taken in fp64 and the result rounded once.
__device__ __forceinline__ void rec_tile_bf16(const DevState &st, double (*red)[RT * RS], int vt, int rt, int R) {
  const int d = st.d;
  const int v0 = vt * RT, r0 = rt * RT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rowbytes = d * 2;
  const int kq = d / RSPLIT;                       // multiple of 16
  const int r16 = lane & 15, g = lane >> 4;
  const int j = threadIdx.x >> 4, i0 = (threadIdx.x & 15) * 2;
  const int row = r0 + j;
  uint32_t ev = 0u;   // embedding pair, fetched before the K loop
  if (row < R)
    ev = *reinterpret_cast<const uint32_t *>(static_cast<const uint16_t *>(st.E) + (size_t)st.r_y[row] * d + v0 + i0);
  // A: 2 blocks of 16 out features, B: 2 blocks of 16 rows; the lane feeds
  // 4 consecutive bf16 at k = kk + 4g to 4 MFMAs (same permutation for A, B).
  // A from the fragment-ordered bf16 W_h copy: one coalesced 512-byte block
  // per row half and 16 K values.
  const u2 *afr = reinterpret_cast<const u2 *>(st.wh16_t) + ((size_t)vt * (d / 16) + (w * kq) / 16) * 128 + lane;
  const uint16_t *b0 = reinterpret_cast<const uint16_t *>(rec_state_row(st, r0 + r16, R, rowbytes)) + w * kq + 4 * g;
  const uint16_t *b1 = reinterpret_cast<const uint16_t *>(rec_state_row(st, r0 + 16 + r16, R, rowbytes)) + w * kq + 4 * g;
  d4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = d4{0.0, 0.0, 0.0, 0.0};
  auto cvt = [](u2 raw, double *o) {
    o[0] = (double)__uint_as_float(raw[0] << 16);
    o[1] = (double)__uint_as_float(raw[0] & 0xFFFF0000u);
    o[2] = (double)__uint_as_float(raw[1] << 16);
    o[3] = (double)__uint_as_float(raw[1] & 0xFFFF0000u);
  };
#pragma unroll 4
  for (int kk = 0; kk < kq; kk += 16) {
    double a[2][4], b[2][4];
    cvt(afr[(size_t)(kk / 16) * 128], a[0]);
    cvt(afr[(size_t)(kk / 16) * 128 + 64], a[1]);
    cvt(*reinterpret_cast<const u2 *>(b0 + kk), b[0]);
    cvt(*reinterpret_cast<const u2 *>(b1 + kk), b[1]);
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[x][e], b[y][e], acc[x][y], 0, 0, 0);
  }
  // f64 16x16x4 result: lane l, register q hold out feature (l/16) + 4q of
  // the block and row l%16.
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = x * 16 + g + 4 * q, j = y * 16 + r16;
        red[w][j * RS + i] = acc[x][y][q];
      }
  __syncthreads();
  if (row < R) {
    uint16_t hb[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int o = j * RS + i0 + q;
      double pre = red[0][o];
#pragma unroll
      for (int x = 1; x < RSPLIT; ++x) pre += red[x][o];   // fixed order
      hb[q] = bf16_rne_from_double(tanh(pre + (double)bf16f((uint16_t)(q ? ev >> 16 : ev & 0xFFFFu))));
    }
    *reinterpret_cast<uint32_t *>(static_cast<uint16_t *>(st.hbuf) + (size_t)row * d + v0 + i0) =
        (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
  }
}

// Persistent launch over the active tiles (rows of this step only): the
// workgroups of XCD x walk the x-th eighth of the tile list. No workgroup is
// launched just to exit.
template <bool BF16>
__global__ __launch_bounds__(RTHREADS) void k_rec(DevState st) {
  const int R = st.ctrl->R;
  if (R <= 0) return;
  const int nra = (R + RT - 1) / RT;
  const int T = (st.d / RT) * nra;
  const int x = blockIdx.x & 7, gx = gridDim.x >> 3;
  const int lo = (int)((long long)T * x / 8), hi = (int)((long long)T * (x + 1) / 8);
  __shared__ typename std::conditional<BF16, double, float>::type red[RSPLIT][RT * RS];
  for (int tile = lo + (int)(blockIdx.x >> 3); tile < hi; tile += gx) {
    const int vt = tile / nra, rt = tile - vt * nra;
    if constexpr (BF16)
      rec_tile_bf16(st, red, vt, rt, R);
    else
      rec_tile_f32(st, red, vt, rt, R);
    __syncthreads();   // red is reused by the next tile
  }
}

// fp32 W_h [d][d] -> the A-fragment order of rec_tile_f32 (above).
__global__ void k_relayout_wh(const float *__restrict__ W, f4 *__restrict__ dst, int d) {
  const size_t n = (size_t)(d / 32) * (d / 8) * 64;
  for (size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += (size_t)gridDim.x * blockDim.x) {
    const int ln = (int)(p & 63);
    const size_t vs = p >> 6;
    const int s = (int)(vs % (d / 8)), vt = (int)(vs / (d / 8));
    dst[p] = *reinterpret_cast<const f4 *>(W + (size_t)(vt * 32 + (ln & 31)) * d + 8 * s + 4 * (ln >> 5));
  }
}

// bf16 W_h [d][d] -> the A-fragment order of rec_tile_bf16 (above).
__global__ void k_relayout_wh16(const uint16_t *__restrict__ W, u2 *__restrict__ dst, int d) {
  const size_t n = (size_t)(d / 32) * (d / 16) * 128;
  for (size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += (size_t)gridDim.x * blockDim.x) {
    const int ln = (int)(p & 63), x = (int)((p >> 6) & 1);
    const size_t vs = p >> 7;
    const int s = (int)(vs % (d / 16)), vt = (int)(vs / (d / 16));
    dst[p] = *reinterpret_cast<const u2 *>(W + (size_t)(vt * 32 + 16 * x + (ln & 15)) * d + 16 * s + 4 * (ln >> 4));
  }
}

}  // namespace

hipError_t launch_relayout_wh(const DevState &st, hipStream_t s) {
  if (st.dtype == 1)
    hipLaunchKernelGGL(k_relayout_wh16, dim3(1024), dim3(256), 0, s, static_cast<const uint16_t *>(st.W_h),
                       reinterpret_cast<u2 *>(const_cast<uint2 *>(st.wh16_t)), st.d);
  else
    hipLaunchKernelGGL(k_relayout_wh, dim3(1024), dim3(256), 0, s, static_cast<const float *>(st.W_h),
                       reinterpret_cast<f4 *>(const_cast<float4 *>(st.wh_t)), st.d);
  return hipGetLastError();
}

hipError_t launch_rec(const DevState &st, hipStream_t s) {
  // Multiple of 8, no more than the tiles of a full step, and at most the
  // workgroups that fit on the device at once: two per compute unit for
  // bf16 (66 KB of LDS each), four for fp32 (33 KB).
  const int tiles = xcd_grid((st.d / RT) * ((st.R_max + RT - 1) / RT));
  const int G = std::max(8, std::min(st.n_cu / (st.dtype == 1 ? 4 : 2) * 8, tiles));
  if (st.dtype == 1)
    hipLaunchKernelGGL(k_rec<true>, dim3(G), dim3(RTHREADS), 0, s, st);
  else
    hipLaunchKernelGGL(k_rec<false>, dim3(G), dim3(RTHREADS), 0, s, st);
  return hipGetLastError();
}

}  // namespace sb
