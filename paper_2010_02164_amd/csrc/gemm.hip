// Decoder-step GEMMs of the synthetic decoder D (Sec. 2) on gfx950 MFMA:
//   K_rec : h = tanh(W_h h_prev + E[y])          [R,d] x [d,d]^T, fused epilogue
//   K_proj: z = W_out h, z[0] += beta (t - L_x),  [R,d] x [V,d]^T, fused online
//           log-sum-exp and per-row partial top-k (the logits never reach HBM)
//
// Both are "TN" products: the weight matrix (out-feature rows) is the MFMA A
// operand and the batch of candidate states is the B operand, both
// K-contiguous. A workgroup (4 waves) owns a 128 (out features) x 64 (rows)
// tile; K is staged through LDS in 128-byte row chunks, double-buffered.
// Every output element accumulates over K in the same fixed order whatever
// rows share the step, so a row's results do not depend on the batch.
#include "sb_internal.h"
#include "topk.h"

namespace sb {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef double d4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));

constexpr int THREADS = 256;
constexpr int BV = GEMM_BV;
constexpr int BR = GEMM_BR;
constexpr int ROWB = 128;              // bytes of one row's K chunk per stage
constexpr int LSTRIDE = ROWB + 16;     // padded LDS row stride (bytes)

struct Smem {
  unsigned char A[2][BV][LSTRIDE];
  unsigned char B[2][BR][LSTRIDE];
};

// Global -> register -> LDS staging of one K chunk: A 128 rows, B 64 rows,
// 8 lanes per 128-byte row chunk (fully coalesced 16-byte loads).
struct Stager {
  const unsigned char *a[4];
  const unsigned char *b[2];
  u4 ra[4], rb[2];
  int row0, col;

  __device__ void load(int kt) {
    const int off = kt * ROWB;
#pragma unroll
    for (int u = 0; u < 4; ++u) ra[u] = *reinterpret_cast<const u4 *>(a[u] + off);
#pragma unroll
    for (int u = 0; u < 2; ++u) rb[u] = *reinterpret_cast<const u4 *>(b[u] + off);
  }
  __device__ void store(Smem &sm, int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
      *reinterpret_cast<u4 *>(&sm.A[buf][row0 + 32 * u][col * 16]) = ra[u];
#pragma unroll
    for (int u = 0; u < 2; ++u)
      *reinterpret_cast<u4 *>(&sm.B[buf][row0 + 32 * u][col * 16]) = rb[u];
  }
};

// Address of the K-contiguous state row feeding batch row r.
__device__ __forceinline__ const unsigned char *state_row(const DevState &st, int r, int rowbytes) {
  const int src = st.r_hsrc[r];
  if (src >= 0) return static_cast<const unsigned char *>(st.s_h) + (size_t)src * rowbytes;
  return static_cast<const unsigned char *>(st.q_h0) + (size_t)(-1 - src) * rowbytes;
}

// XCD-aware tile order: consecutive workgroup ids land on different XCDs
// (round robin over 8); remap so that each XCD walks a contiguous range of
// tiles in which the row-tile index varies fastest, so the workgroups that
// share one weight tile share that XCD's L2.
__device__ __forceinline__ void tile_of(int nvt, int nrt, int &vt, int &rt) {
  const int G = nvt * nrt;
  const int g = blockIdx.x;
  int lin = g;
  if ((G & 7) == 0) lin = (g & 7) * (G >> 3) + (g >> 3);
  vt = lin / nrt;
  rt = lin - vt * nrt;
}

// MFMA inner product over one staged 128-byte K chunk for a wave's
// 64 (out) x 32 (rows) sub-tile: acc0 covers out rows [0,32), acc1 [32,64).
template <bool BF16>
__device__ __forceinline__ void mma_chunk(const Smem &sm, int buf, int wv, int wb, int lane,
                                          f16v &acc0, f16v &acc1) {
  const int r = lane & 31;
  const int h = (lane >> 5) * 16;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int off = ks * 32 + h;
    if constexpr (BF16) {
      // 32x32x16 bf16: lane supplies A[r][8*(lane/32) .. +7] of a 16-wide K step.
      const bf8 a0 = *reinterpret_cast<const bf8 *>(&sm.A[buf][wv * 64 + r][off]);
      const bf8 a1 = *reinterpret_cast<const bf8 *>(&sm.A[buf][wv * 64 + 32 + r][off]);
      const bf8 b0 = *reinterpret_cast<const bf8 *>(&sm.B[buf][wb * 32 + r][off]);
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc1, 0, 0, 0);
    } else {
      // 32x32x2 f32 with a K permutation: the lane's 4 consecutive floats feed
      // 4 MFMAs; lanes 0-31 supply k = 8ks+e, lanes 32-63 k = 8ks+4+e, the
      // same for A and B, so each MFMA pairs matching k.
      const f4 a0 = *reinterpret_cast<const f4 *>(&sm.A[buf][wv * 64 + r][off]);
      const f4 a1 = *reinterpret_cast<const f4 *>(&sm.A[buf][wv * 64 + 32 + r][off]);
      const f4 b0 = *reinterpret_cast<const f4 *>(&sm.B[buf][wb * 32 + r][off]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[e], b0[e], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[e], b0[e], acc1, 0, 0, 0);
      }
    }
  }
}

// Shared mainloop: stages A rows (weights, clamped to nA) and the B rows
// (prepared by the caller) and accumulates the wave's sub-tile.
template <bool BF16>
__device__ __forceinline__ void gemm_mainloop(Smem &sm, Stager &sg, int nk, int wv, int wb,
                                              int lane, f16v &acc0, f16v &acc1) {
  sg.load(0);
  sg.store(sm, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) sg.load(kt + 1);
    mma_chunk<BF16>(sm, cur, wv, wb, lane, acc0, acc1);
    if (kt + 1 < nk) sg.store(sm, cur ^ 1);
    __syncthreads();
  }
}

// B rows come from `dense` ([R][d], row r at r*rowbytes) when it is given,
// else from each row's recorded state source (slot state or queued h0).
__device__ __forceinline__ void setup_stager(Stager &sg, const DevState &st, const void *W, int nA,
                                             int v0, int r0, int R, int rowbytes, const void *dense) {
  const int tid = threadIdx.x;
  sg.row0 = tid >> 3;
  sg.col = tid & 7;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int v = min(v0 + sg.row0 + 32 * u, nA - 1);
    sg.a[u] = static_cast<const unsigned char *>(W) + (size_t)v * rowbytes + sg.col * 16;
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int r = min(r0 + sg.row0 + 32 * u, R - 1);
    const unsigned char *row = dense ? static_cast<const unsigned char *>(dense) + (size_t)r * rowbytes
                                     : state_row(st, r, rowbytes);
    sg.b[u] = row + sg.col * 16;
  }
}

// Zero-extend bf16 bits to float.
__device__ __forceinline__ float bf16f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round a binary64 value to bfloat16 (nearest, ties to even) directly, with
// no float intermediate: keep 8 significant bits; below bf16's smallest
// normal (2^-126) the step is the subnormal quantum 2^-133.
__device__ __forceinline__ uint16_t bf16_rne_from_double(double x) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const unsigned long long sign = u & 0x8000000000000000ull;
  unsigned long long a = u & 0x7FFFFFFFFFFFFFFFull;
  const int e = (int)(a >> 52);
  float f;
  if (e >= 1023 - 126) {
    const unsigned long long lsb = (a >> 45) & 1ull;
    a += 0x0FFFFFFFFFFFull + lsb;   // half of the dropped 45 bits, minus one
    a &= ~0x1FFFFFFFFFFFull;
    f = (float)__longlong_as_double((long long)(a | sign));
  } else {
    const double q = 0x1p-133;
    f = (float)(rint(x / q) * q);
  }
  return (uint16_t)(__float_as_uint(f) >> 16);
}

// ---------------------------------------------------------------- K_rec
// The recurrence GEMM is small ([R,d] x [d,d]) next to the projection, so it
// is cut into 32 (out features) x 32 (rows) tiles to reach hundreds of
// workgroups, and the K loop of each tile is split over the 4 waves of the
// workgroup; the 4 partial sums are added in a fixed order (wave 0 + 1 + 2
// + 3), so the result does not depend on which rows share the step. Operands
// are read straight from global memory (W_h and the states are L2/MALL
// resident); each lane loads the 16 bytes it feeds to the MFMA.
constexpr int RT = 32;        // tile edge
constexpr int RSPLIT = 4;     // K split over the waves

__device__ __forceinline__ const unsigned char *rec_state_row(const DevState &st, int r, int R, int rowbytes) {
  return state_row(st, min(r, R - 1), rowbytes);
}

__global__ __launch_bounds__(THREADS) void k_rec_f32(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d;
  const int nvt = d / RT, nrt = (st.R_max + RT - 1) / RT;
  int vt, rt;
  tile_of(nvt, nrt, vt, rt);
  const int v0 = vt * RT, r0 = rt * RT;
  if (r0 >= R) return;
  __shared__ float red[RSPLIT][RT * RT];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rowbytes = d * 4;
  const int kq = d / RSPLIT;                       // K range of this wave
  const float *arow = static_cast<const float *>(st.W_h) + (size_t)(v0 + (lane & 31)) * d + w * kq;
  const float *brow = reinterpret_cast<const float *>(rec_state_row(st, r0 + (lane & 31), R, rowbytes)) + w * kq;
  const int h = (lane >> 5) * 4;
  f16v acc = {};
#pragma unroll 4
  for (int kk = 0; kk < kq; kk += 8) {
    const f4 a = *reinterpret_cast<const f4 *>(arow + kk + h);
    const f4 b = *reinterpret_cast<const f4 *>(brow + kk + h);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
  }
  // acc: out feature i = 8*(reg/4) + 4*(lane/32) + reg%4, row j = lane%32.
#pragma unroll
  for (int reg = 0; reg < 16; ++reg) {
    const int i = 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
    red[w][(lane & 31) * RT + i] = acc[reg];
  }
  __syncthreads();
  // 256 threads x 4 outputs: thread -> row j = tid/8, features 4*(tid%8)..+3.
  const int j = threadIdx.x >> 3, i0 = (threadIdx.x & 7) * 4;
  const int row = r0 + j;
  if (row >= R) return;
  const float *E = static_cast<const float *>(st.E) + (size_t)st.r_y[row] * d + v0 + i0;
  const f4 e = *reinterpret_cast<const f4 *>(E);
  f4 hv;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int o = j * RT + i0 + q;
    const float pre = ((red[0][o] + red[1][o]) + red[2][o]) + red[3][o];
    hv[q] = tanhf(pre + e[q]);
  }
  *reinterpret_cast<f4 *>(static_cast<float *>(st.hbuf) + (size_t)row * d + v0 + i0) = hv;
}

// bf16 states are rounded after tanh, a discontinuous map: any difference
// in the pre-activation can flip a rounding and then grows step after step.
// Products of two bf16 values are exact in fp64 and so is their sum over
// the state size in practice, so the pre-activation is accumulated with the
// fp64 MFMA (16x16x4), tanh taken in fp64 and the result rounded once.
__global__ __launch_bounds__(THREADS) void k_rec_bf16(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d;
  const int nvt = d / RT, nrt = (st.R_max + RT - 1) / RT;
  int vt, rt;
  tile_of(nvt, nrt, vt, rt);
  const int v0 = vt * RT, r0 = rt * RT;
  if (r0 >= R) return;
  __shared__ double red[RSPLIT][RT * RT];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rowbytes = d * 2;
  const int kq = d / RSPLIT;
  const int r16 = lane & 15, g = lane >> 4;
  // A: 2 blocks of 16 out features, B: 2 blocks of 16 rows; the lane feeds
  // 4 consecutive bf16 at k = kk + 4g to 4 MFMAs (same permutation for A, B).
  const uint16_t *a0 = static_cast<const uint16_t *>(st.W_h) + (size_t)(v0 + r16) * d + w * kq + 4 * g;
  const uint16_t *a1 = a0 + (size_t)16 * d;
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
#pragma unroll 2
  for (int kk = 0; kk < kq; kk += 16) {
    double a[2][4], b[2][4];
    cvt(*reinterpret_cast<const u2 *>(a0 + kk), a[0]);
    cvt(*reinterpret_cast<const u2 *>(a1 + kk), a[1]);
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
        red[w][j * RT + i] = acc[x][y][q];
      }
  __syncthreads();
  const int j = threadIdx.x >> 3, i0 = (threadIdx.x & 7) * 4;
  const int row = r0 + j;
  if (row >= R) return;
  const uint16_t *E = static_cast<const uint16_t *>(st.E) + (size_t)st.r_y[row] * d + v0 + i0;
  const u2 eraw = *reinterpret_cast<const u2 *>(E);
  double e[4];
  cvt(eraw, e);
  uint16_t hb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int o = j * RT + i0 + q;
    const double pre = ((red[0][o] + red[1][o]) + red[2][o]) + red[3][o];
    hb[q] = bf16_rne_from_double(tanh(pre + e[q]));
  }
  u2 packed;
  packed[0] = (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
  packed[1] = (uint32_t)hb[2] | ((uint32_t)hb[3] << 16);
  *reinterpret_cast<u2 *>(static_cast<uint16_t *>(st.hbuf) + (size_t)row * d + v0 + i0) = packed;
}

// ------------------------------------------------------------------- K_proj
// After the mainloop each lane holds, for one batch row, 32 logits of the
// wave's 64-wide vocab slice (two 32x32 blocks). The epilogue adds the EOS
// bias, folds the 32 values into (max, sum exp) and a sorted top-KB list,
// merges with the partner lane holding the other 32, then with the other
// vocab wave through LDS, and writes one partial per (row, 128-wide tile).
template <bool BF16, int KB>
__global__ __launch_bounds__(THREADS, 2) void k_proj(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d, V = st.V;
  const int nvt = st.S, nrt = (st.R_max + BR - 1) / BR;
  int vt, rt;
  tile_of(nvt, nrt, vt, rt);
  const int v0 = vt * BV, r0 = rt * BR;
  if (r0 >= R) return;
  __shared__ Smem sm;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wv = w & 1, wb = w >> 1;
  const int rowbytes = d * (BF16 ? 2 : 4);
  Stager sg;
  setup_stager(sg, st, st.W_out, V, v0, r0, R, rowbytes, st.hbuf);
  f16v acc0 = {}, acc1 = {};
  gemm_mainloop<BF16>(sm, sg, rowbytes / ROWB, wv, wb, lane, acc0, acc1);

  const int jl = wb * 32 + (lane & 31);   // row within the tile
  const int j = r0 + jl;
  const bool row_ok = j < R;
  float bias = 0.0f;
  if (v0 == 0 && row_ok) bias = st.beta * (float)(st.r_t[j] - st.r_Lx[j]);

  float vals[32];
#pragma unroll
  for (int vb = 0; vb < 2; ++vb) {
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int v = v0 + wv * 64 + vb * 32 + 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
      float z = vb ? acc1[reg] : acc0[reg];
      if (v == 0) z += bias;
      vals[vb * 16 + reg] = v < V ? z : -INFINITY;
    }
  }
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < 32; ++q) m = fmaxf(m, vals[q]);
  float s = 0.0f;
  if (m > -INFINITY) {
#pragma unroll
    for (int q = 0; q < 32; ++q) s += expf(vals[q] - m);
  }
  TopK<KB> tk;
  topk_init(tk);
#pragma unroll
  for (int vb = 0; vb < 2; ++vb)
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int v = v0 + wv * 64 + vb * 32 + 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
      topk_push_ordered(tk, vals[vb * 16 + reg], v);
    }
  {
    TopK<KB> o;
    topk_shfl_xor(o, tk, 32);
    const float m2 = __shfl_xor(m, 32, 64), s2 = __shfl_xor(s, 32, 64);
    lse_merge(m, s, m2, s2);
    topk_merge(tk, o);
  }

  // Cross-wave merge through LDS (reusing the staging buffers).
  constexpr int PW = 2 + 2 * KB;
  float *xch = reinterpret_cast<float *>(&sm.A[0][0][0]);
  __syncthreads();
  if (wv == 1 && lane < 32) {
    float *p = xch + jl * PW;
    p[0] = m;
    p[1] = s;
#pragma unroll
    for (int q = 0; q < KB; ++q) {
      p[2 + q] = tk.v[q];
      p[2 + KB + q] = __int_as_float(tk.i[q]);
    }
  }
  __syncthreads();
  if (wv == 0 && lane < 32 && row_ok) {
    const float *p = xch + jl * PW;
    TopK<KB> o;
#pragma unroll
    for (int q = 0; q < KB; ++q) {
      o.v[q] = p[2 + q];
      o.i[q] = __float_as_int(p[2 + KB + q]);
    }
    lse_merge(m, s, p[0], p[1]);
    topk_merge(tk, o);
    float *out = st.part + ((size_t)j * st.S + vt) * PW;
    out[0] = m;
    out[1] = s;
#pragma unroll
    for (int q = 0; q < KB; ++q) {
      out[2 + q] = tk.v[q];
      out[2 + KB + q] = __int_as_float(tk.i[q]);
    }
  }
}

template <bool BF16>
hipError_t launch_proj_t(const DevState &st, hipStream_t s) {
  const int G = st.S * ((st.R_max + BR - 1) / BR);
  switch (st.kbucket) {
    case 4: hipLaunchKernelGGL((k_proj<BF16, 4>), dim3(G), dim3(THREADS), 0, s, st); break;
    case 8: hipLaunchKernelGGL((k_proj<BF16, 8>), dim3(G), dim3(THREADS), 0, s, st); break;
    default: hipLaunchKernelGGL((k_proj<BF16, 16>), dim3(G), dim3(THREADS), 0, s, st); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rec(const DevState &st, hipStream_t s) {
  const int G = (st.d / RT) * ((st.R_max + RT - 1) / RT);
  if (st.dtype == 1)
    hipLaunchKernelGGL(k_rec_bf16, dim3(G), dim3(THREADS), 0, s, st);
  else
    hipLaunchKernelGGL(k_rec_f32, dim3(G), dim3(THREADS), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_proj(const DevState &st, hipStream_t s) {
  return st.dtype == 1 ? launch_proj_t<true>(st, s) : launch_proj_t<false>(st, s);
}

}  // namespace sb
