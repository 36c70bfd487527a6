// Per-candidate KV-like state: every expansion appends the rows
// bf16(h . W_kv[l][j]) (l < L layers, j in {K, V}) at position l_t - 1, and
// every beam update hands each surviving active candidate its parent's rows
// (the reorder of incremental decoder state that the paper's transformer
// decoder performs, App. A.2). The rows are not copied: the row of an
// expansion is stored once, at (beam, level, rank) of the expanded
// candidate, and a candidate reaches its rows through the ranks of its
// ancestors per level, which the beam update passes on (a few bytes per
// child instead of 2 L d t bytes).
#include "mfma_common.h"

namespace sb {
namespace {


constexpr int THREADS = 256;
constexpr int BV = GEMM_BV, BR = GEMM_BR;
constexpr int ROWB = 128, LSTRIDE = ROWB + 16;

struct Smem {
  unsigned char A[2][BV][LSTRIDE];
  unsigned char B[2][BR][LSTRIDE];
};

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// kvs[beam][t-1][rank][o] = bf16(sum_i h[r][i] * W_kvT[o][i]) for row r
// (the candidate at rank `rank` of the beam, emitting position t), o over
// the L*2*d outputs.
__global__ __launch_bounds__(THREADS, 2) void k_kv_append(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d, NO = st.kv_layers * 2 * d;
  // XCD-aware order: the row tiles of one W_kv column tile run on one XCD
  // and share its L2 copy of the tile.
  int vt, rt;
  if (!tile_of(NO / BV, (st.R_max + BR - 1) / BR, vt, rt)) return;
  const int v0 = vt * BV, r0 = rt * BR;
  if (r0 >= R) return;
  __shared__ Smem sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wv = w & 1, wb = w >> 1;
  const int rowbytes = d * 2;
  const int row0 = tid >> 3, col = tid & 7;
  const unsigned char *ap[4], *bp[2];
#pragma unroll
  for (int u = 0; u < 4; ++u)
    ap[u] = reinterpret_cast<const unsigned char *>(st.wkvT) + (size_t)(v0 + row0 + 32 * u) * rowbytes + col * 16;
#pragma unroll
  for (int u = 0; u < 2; ++u)
    bp[u] = static_cast<const unsigned char *>(st.hbuf) + (size_t)min(r0 + row0 + 32 * u, R - 1) * rowbytes + col * 16;
  u4 ra[4], rb[2];
  auto load = [&](int kt) {
#pragma unroll
    for (int u = 0; u < 4; ++u) ra[u] = *reinterpret_cast<const u4 *>(ap[u] + kt * ROWB);
#pragma unroll
    for (int u = 0; u < 2; ++u) rb[u] = *reinterpret_cast<const u4 *>(bp[u] + kt * ROWB);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<u4 *>(&sm.A[buf][row0 + 32 * u][col * 16]) = ra[u];
#pragma unroll
    for (int u = 0; u < 2; ++u) *reinterpret_cast<u4 *>(&sm.B[buf][row0 + 32 * u][col * 16]) = rb[u];
  };
  f16v acc0 = {}, acc1 = {};
  const int nk = rowbytes / ROWB;
  load(0);
  store(0);
  __syncthreads();
  const int r = lane & 31, h = (lane >> 5) * 16;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load(kt + 1);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int off = ks * 32 + h;
      const bf8 a0 = *reinterpret_cast<const bf8 *>(&sm.A[cur][wv * 64 + r][off]);
      const bf8 a1 = *reinterpret_cast<const bf8 *>(&sm.A[cur][wv * 64 + 32 + r][off]);
      const bf8 b0 = *reinterpret_cast<const bf8 *>(&sm.B[cur][wb * 32 + r][off]);
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc1, 0, 0, 0);
    }
    if (kt + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }
  const int j = r0 + wb * 32 + (lane & 31);
  if (j >= R) return;
  const int slot = st.r_slot[j], beam = slot / st.k, rank = slot - beam * st.k;
  uint16_t *out = st.kvs + (((size_t)beam * st.max_len_cap + (st.r_t[j] - 1)) * st.k + rank) * NO;
#pragma unroll
  for (int vb = 0; vb < 2; ++vb) {
    const f16v &acc = vb ? acc1 : acc0;
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int o = v0 + wv * 64 + vb * 32 + 8 * gq + 4 * (lane >> 5);
      u2 pk;
      pk[0] = (uint32_t)bf16_rne(acc[4 * gq + 0]) | ((uint32_t)bf16_rne(acc[4 * gq + 1]) << 16);
      pk[1] = (uint32_t)bf16_rne(acc[4 * gq + 2]) | ((uint32_t)bf16_rne(acc[4 * gq + 3]) << 16);
      *reinterpret_cast<u2 *>(out + o) = pk;
    }
  }
}

__global__ void k_transpose(const uint16_t *W, uint16_t *WT, int L2, int d) {
  // W [L2][d_in][d_out] -> WT [L2][d_out][d_in]
  const size_t total = (size_t)L2 * d * d;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    const size_t p = e / ((size_t)d * d);
    const size_t rem = e - p * d * d;
    const size_t i = rem / d, o = rem - i * d;
    WT[p * d * d + o * d + i] = W[e];
  }
}

}  // namespace

hipError_t launch_kv_append(const DevState &st, hipStream_t s) {
  const int NO = st.kv_layers * 2 * st.d;
  const int G = xcd_grid((NO / BV) * ((st.R_max + BR - 1) / BR));
  hipLaunchKernelGGL(k_kv_append, dim3(G), dim3(THREADS), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_transpose_wkv(const DevState &st, const uint16_t *W_kv, hipStream_t s) {
  hipLaunchKernelGGL(k_transpose, dim3(1024), dim3(256), 0, s, W_kv, st.wkvT, st.kv_layers * 2, st.d);
  return hipGetLastError();
}

}  // namespace sb
