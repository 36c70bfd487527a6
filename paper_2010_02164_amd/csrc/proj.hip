// Vocabulary projection of the synthetic decoder D (Sec. 2) on gfx950 MFMA,
// fused with the EOS bias, an online log-sum-exp and a per-row partial top-k:
//   z = W_out h,  z[0] += beta (t - L_x)      [R,d] x [V,d]^T
// The R x |V| logits never reach memory: each workgroup writes, per row and
// 128-wide vocabulary tile, (max, sum exp) and its best kb (value, token).
//
// Workgroup: 4 waves, tile 128 vocabulary rows (32 per wave) x 128 batch rows
// (4 blocks of 32). W_out, the large streamed operand, is kept 3 K-chunks
// ahead in registers (48 KB in flight per workgroup) to cover HBM/MALL
// latency, and both operands pass through a double-buffered LDS tile so
// that global loads stay fully coalesced. Blocks of 32 rows past R are
// skipped, so small steps cost proportionally less. The K loop runs in 128-byte
// chunks per row; every output accumulates over K in the same fixed order
// whatever rows share the step, so a row's results do not depend on the batch.
#include "mfma_common.h"
#include "topk.h"

namespace sb {
namespace {

constexpr int THREADS = 256;
constexpr int NB = 4;            // 32-row batch blocks per workgroup
constexpr int TR = 32 * NB;      // batch rows per workgroup
constexpr int TV = GEMM_BV;      // vocabulary rows per workgroup (4 waves x 32)
constexpr int CH = 128;          // bytes of a row's K chunk
constexpr int LS = CH + 16;      // padded LDS row stride (bytes)
constexpr int AD = 3;            // W_out prefetch depth (chunks)

template <int KB>
union ProjSmem {
  struct {
    unsigned char A[2][TV][LS];
    unsigned char B[2][TR][LS];
  } t;
  float xch[4][TR][2 + 2 * KB];
};

// K loop of one workgroup: acc[b] (b < NBV) += W_out tile x batch block b.
// Both operands are staged through a double-buffered LDS tile with fully
// coalesced loads (8 lanes per 128-byte row segment): W_out through a
// 3-chunk register prefetch ring, the states one chunk ahead. Loads return in
// issue order, so each iteration issues them in the order they are consumed
// (states chunk kt+2, then W_out chunk kt+4); prefetch indices are clamped
// instead of guarded, so no load sits inside a branch.
template <bool BF16, int NBV>
__device__ __forceinline__ void proj_mainloop(unsigned char (*A)[TV][LS], unsigned char (*B)[TR][LS],
                                              const unsigned char *abase, const uint32_t *aoff,
                                              const unsigned char *bbase, const uint32_t *boff,
                                              int srow, int scol, int nk, int w, int l32, int h, f16v *acc) {
  u4 as[AD][4];
  u4 bs[4];
  // Uniform base + 32-bit per-lane offset (SGPR-based addressing); chunk
  // stride `cs` bytes (tiled W_out: one 16 KB block per chunk).
  auto load = [&](const unsigned char *base, const uint32_t *off, uint32_t cs, int kt, u4 *dst) {
#pragma unroll
    for (int u = 0; u < 4; ++u) dst[u] = *reinterpret_cast<const u4 *>(base + (off[u] + (uint32_t)kt * cs));
  };
  auto store = [&](unsigned char (*T)[LS], const u4 *src) {
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<u4 *>(&T[srow + 32 * u][scol]) = src[u];
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // K permutation: lane half h at piece q feeds k = chunk + 16h + 4q + e
      // (fp32) or chunk + 32h + 8q + e (bf16), identically for both operands.
      const u4 araw = *reinterpret_cast<const u4 *>(&A[buf][32 * w + l32][64 * h + 16 * q]);
      u4 braw[NBV];
#pragma unroll
      for (int b = 0; b < NBV; ++b) braw[b] = *reinterpret_cast<const u4 *>(&B[buf][32 * b + l32][64 * h + 16 * q]);
#pragma unroll
      for (int b = 0; b < NBV; ++b) {
        if constexpr (BF16) {
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf8, araw),
                                                           __builtin_bit_cast(bf8, braw[b]), acc[b], 0, 0, 0);
        } else {
          const f4 av = __builtin_bit_cast(f4, araw);
          const f4 bv = __builtin_bit_cast(f4, braw[b]);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], bv[e], acc[b], 0, 0, 0);
        }
      }
    }
  };

  // Prologue: chunk 0 in LDS; states 1 and W_out 1, 2, 3 in flight.
  load(bbase, boff, CH, 0, bs);
#pragma unroll
  for (int c = 0; c < AD; ++c) load(abase, aoff, TV * CH, min(c, nk - 1), as[c]);
  store(A[0], as[0]);
  store(B[0], bs);
  load(bbase, boff, CH, min(1, nk - 1), bs);
  load(abase, aoff, TV * CH, min(AD, nk - 1), as[0]);
  __syncthreads();

  for (int kt0 = 0; kt0 < nk; kt0 += AD) {
#pragma unroll
    for (int j = 0; j < AD; ++j) {
      const int kt = kt0 + j;   // kt % AD == j
      if (kt < nk) compute(kt & 1);
      // W_out chunk kt+1 sits in as[(kt+1)%AD], states chunk kt+1 in bs.
      if (kt + 1 < nk) {
        store(A[(kt + 1) & 1], as[(j + 1) % AD]);
        store(B[(kt + 1) & 1], bs);
      }
      load(bbase, boff, CH, min(kt + 2, nk - 1), bs);
      load(abase, aoff, TV * CH, min(kt + 1 + AD, nk - 1), as[(j + 1) % AD]);
      __syncthreads();
    }
  }
}

template <bool BF16, int KB>
__global__ __launch_bounds__(THREADS, 2) void k_proj(DevState st) {
  const int R = st.ctrl->R;
  const int d = st.d, V = st.V;
  const int nvt = st.S, nrt = (st.R_max + TR - 1) / TR;
  int vt, rt;
  if (!tile_of(nvt, nrt, vt, rt)) return;
  const int v0 = vt * TV, r0 = rt * TR;
  if (r0 >= R) return;
  const int nbv = min(NB, (R - r0 + 31) >> 5);    // blocks holding valid rows
  __shared__ ProjSmem<KB> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int rowbytes = d * (BF16 ? 2 : 4);
  const int nk = rowbytes / CH;

  // Staging: thread -> rows (tid/8) + 32u, 16-byte column tid%8, of the
  // W_out tile (a contiguous 16 KB block per K chunk in the tiled copy) and
  // of the state tile (batch rows, clamped to R-1). Chunk kt of W_out sits
  // kt * 16 KB further; of the states, kt * 128 bytes further.
  const int srow = tid >> 3, scol = (tid & 7) * 16;
  // Byte offsets fit 32 bits (the tiled W_out is checked at create time).
  uint32_t aoff[4], boff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    aoff[u] = ((uint32_t)vt * (uint32_t)nk * TV + srow + 32 * u) * CH + scol;
    boff[u] = (uint32_t)min(r0 + srow + 32 * u, R - 1) * (uint32_t)rowbytes + scol;
  }
  const unsigned char *abase = st.wout_t;
  const unsigned char *bbase = static_cast<const unsigned char *>(st.hbuf);
  f16v acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f16v{};
  // One mainloop instantiation per count of valid 32-row blocks, so the
  // K loop has no per-block branches.
  switch (nbv) {
    case 1: proj_mainloop<BF16, 1>(sm.t.A, sm.t.B, abase, aoff, bbase, boff, srow, scol, nk, w, l32, h, acc); break;
    case 2: proj_mainloop<BF16, 2>(sm.t.A, sm.t.B, abase, aoff, bbase, boff, srow, scol, nk, w, l32, h, acc); break;
    case 3: proj_mainloop<BF16, 3>(sm.t.A, sm.t.B, abase, aoff, bbase, boff, srow, scol, nk, w, l32, h, acc); break;
    default: proj_mainloop<BF16, 4>(sm.t.A, sm.t.B, abase, aoff, bbase, boff, srow, scol, nk, w, l32, h, acc); break;
  }

  // Epilogue. Block b: lane holds batch row r0 + 32b + l32 and the wave's
  // vocabulary rows v0 + 32w + 8*(reg/4) + 4h + reg%4, increasing with reg.
  constexpr int PW = 2 + 2 * KB;
  float bias_row[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int j = r0 + 32 * b + l32;
    bias_row[b] = (v0 == 0 && j < R) ? st.beta * (float)(st.r_t[j] - st.r_Lx[j]) : 0.0f;
  }
  TopK<KB> tks[NB];
  float ms[NB], ss[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (b < nbv) {
      float vals[16];
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int v = v0 + 32 * w + 8 * (reg >> 2) + 4 * h + (reg & 3);
        float z = acc[b][reg];
        if (v == 0) z += bias_row[b];
        vals[reg] = v < V ? z : -INFINITY;
      }
      float m = -INFINITY;
#pragma unroll
      for (int q = 0; q < 16; ++q) m = fmaxf(m, vals[q]);
      float s = 0.0f;
      if (m > -INFINITY) {
#pragma unroll
        for (int q = 0; q < 16; ++q) s += __expf(vals[q] - m);
      }
      // The lane's 16 candidates as ranking keys, sorted by a network.
      cand_key keys[16];
#pragma unroll
      for (int reg = 0; reg < 16; ++reg)
        keys[reg] = make_key(vals[reg], v0 + 32 * w + 8 * (reg >> 2) + 4 * h + (reg & 3));
      bitonic_sort_desc<16>(keys);
#pragma unroll
      for (int q = 0; q < KB; ++q) tks[b].k[q] = keys[q];
      TopK<KB> o;
      topk_shfl_xor(o, tks[b], 32);
      const float m2 = __shfl_xor(m, 32, 64), s2 = __shfl_xor(s, 32, 64);
      lse_merge(m, s, m2, s2);
      topk_merge(tks[b], o);
      ms[b] = m;
      ss[b] = s;
    }
  }
  // The staging tile is dead after the last barrier of the K loop.
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (b < nbv && lane < 32) {
      float *p = sm.xch[w][32 * b + l32];
      p[0] = ms[b];
      p[1] = ss[b];
      topk_store(p + 2, tks[b]);
    }
  }
  __syncthreads();
  // Wave w merges the four vocabulary quarters of batch block w.
  if (w < nbv && lane < 32) {
    const int row = 32 * w + l32;
    const int j = r0 + row;
    if (j < R) {
      float m = -INFINITY, s = 0.0f;
      TopK<KB> tk;
      topk_init(tk);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const float *p = sm.xch[x][row];
        TopK<KB> o;
        topk_load(o, p + 2);
        lse_merge(m, s, p[0], p[1]);
        topk_merge(tk, o);
      }
      float *out = st.part + ((size_t)j * st.S + vt) * PW;
      out[0] = m;
      out[1] = s;
      topk_store(out + 2, tk);
    }
  }
}

// W_out [V][d] -> tiled [S][nk][128][128 bytes], zero rows past V.
__global__ void k_relayout_wout(const unsigned char *__restrict__ src, unsigned char *__restrict__ dst, int V,
                                int rowbytes, int S) {
  const int nk = rowbytes / CH;
  const size_t pieces = (size_t)S * nk * TV * (CH / 16);
  for (size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x; p < pieces; p += (size_t)gridDim.x * blockDim.x) {
    const int piece = (int)(p % (CH / 16));
    const size_t rowblk = p / (CH / 16);          // ((vt * nk + kt) * TV + row)
    const int row = (int)(rowblk % TV);
    const size_t vk = rowblk / TV;
    const int kt = (int)(vk % nk);
    const int vt = (int)(vk / nk);
    const int v = vt * TV + row;
    u4 val = {0u, 0u, 0u, 0u};
    if (v < V) val = *reinterpret_cast<const u4 *>(src + (size_t)v * rowbytes + (size_t)kt * CH + piece * 16);
    *reinterpret_cast<u4 *>(dst + p * 16) = val;
  }
}

template <bool BF16>
hipError_t launch_proj_t(const DevState &st, hipStream_t s) {
  const int G = xcd_grid(st.S * ((st.R_max + TR - 1) / TR));
  switch (st.kbucket) {
    case 4: hipLaunchKernelGGL((k_proj<BF16, 4>), dim3(G), dim3(THREADS), 0, s, st); break;
    case 8: hipLaunchKernelGGL((k_proj<BF16, 8>), dim3(G), dim3(THREADS), 0, s, st); break;
    default: hipLaunchKernelGGL((k_proj<BF16, 16>), dim3(G), dim3(THREADS), 0, s, st); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_relayout_wout(const DevState &st, hipStream_t s) {
  const int rowbytes = st.d * (st.dtype == 1 ? 2 : 4);
  hipLaunchKernelGGL(k_relayout_wout, dim3(2048), dim3(256), 0, s, static_cast<const unsigned char *>(st.W_out),
                     st.wout_t, st.V, rowbytes, st.S);
  return hipGetLastError();
}

hipError_t launch_proj(const DevState &st, hipStream_t s) {
  return st.dtype == 1 ? launch_proj_t<true>(st, s) : launch_proj_t<false>(st, s);
}

}  // namespace sb
