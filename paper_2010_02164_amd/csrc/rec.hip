// Recurrence of the synthetic decoder D (Sec. 2) on gfx950 MFMA:
//   h = tanh(W_h h_prev + E[y])      [R,d] x [d,d]^T, fused epilogue
// W_h (out-feature rows) is the MFMA A operand and the previous states the B
// operand, both K-contiguous. bf16 workloads form the pre-activation
// exactly from int8 digit products (k_rec_i8, below), or, where that does
// not apply, accumulate it with the fp64 MFMA (rec_tile_bf16).
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

// The tiles of XCD x: a block of output tiles (rows of W_h) times a block
// of row tiles, walked row tile by row tile with the output tiles inner, so
// that the XCD's L2 keeps its share of W_h and each row tile's states are
// fetched once and used by consecutive workgroups. Small steps give each
// XCD fewer output tiles and more of the rows.
struct RecWalk {
  int vlo, nv, rlo, n;
  __device__ RecWalk(int nvt, int nra, int x) {
    const int nrg = nra >= 16 ? 4 : (nra >= 4 ? 2 : 1), nvg = 8 / nrg;
    const int vg = x % nvg, rg = x / nvg;
    vlo = nvt * vg / nvg;
    nv = nvt * (vg + 1) / nvg - vlo;
    rlo = nra * rg / nrg;
    n = nv * (nra * (rg + 1) / nrg - rlo);
  }
  __device__ void at(int t, int &vt, int &rt) const {
    const int q = t / nv;
    rt = rlo + q;
    vt = vlo + t - q * nv;
  }
};

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

// ---------------------------------------------------- exact bf16 recurrence
// The bf16 pre-activation without fp64 MFMA. A bf16 value is M * 2^(eu-134)
// with an integer M < 256 (eu = the exponent field, 1 for subnormals).
// Scaled by 2^(21 - Ew) for a W_h row (|W| < 2^Ew) or 2^(21 - F) for a state
// row (|h| < 2^F), every value of the row down to 2^(E-13) becomes an
// integer below 2^21, held as three signed 7-bit digits:
//   omega = sum_a w_a 128^a,   eta = sum_b h_b 128^b,   |w_a|, |h_b| <= 127,
// and sum_i W h = 2^(Ew + F - 42) Z with Z = sum_s 128^s T_s and
//   T_s = sum_{a+b=s} sum_i w_a[i] h_b[i],
// each T_s an exact int32 sum of int8 products (v_mfma_i32_32x32x32_i8;
// below 3 d 127^2 < 2^31), in any order. Z itself is an integer below
// d 2^42, exact in fp64 for d <= 2048. The values below a row's window
// (rare: a W_h entry below 2^(Ew-13), a state entry below 2^(F-13)) are
// added as fp64 products from per-row lists. The digits of a state are
// written once, by the step that produces it (F = 1 for tanh outputs), or
// when an encoding is submitted.
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// Digits of bf16 bits b under the row exponent E (|x| < 2^E for the row);
// false (digits 0) for a value below the window.
__device__ __forceinline__ bool bf16_digits3(uint32_t b, int E, int &d0, int &d1, int &d2) {
  const uint32_t e8 = (b >> 7) & 0xFFu, man = b & 0x7Fu;
  const uint32_t M = (e8 ? 0x80u : 0u) | man;
  d0 = d1 = d2 = 0;
  if (M == 0u) return true;
  const int shift = (int)max(e8, 1u) - 113 - E;
  if (shift < 0) return false;
  const uint32_t mag = M << shift;   // < 2^21
  const int sg = (b & 0x8000u) ? -1 : 1;
  d0 = sg * (int)(mag & 0x7Fu);
  d1 = sg * (int)((mag >> 7) & 0x7Fu);
  d2 = sg * (int)((mag >> 14) & 0x7Fu);
  return true;
}

// Smallest E with every |x| < 2^E over n bf16 values (strided by `step`
// from `first`), as this thread's partial maximum of eu - 126.
__device__ __forceinline__ int bf16_max_eu(const uint16_t *x, int first, int n, int step) {
  uint32_t mx = 1u;
  for (int i = first; i < n; i += step) mx = max(mx, ((uint32_t)x[i] >> 7) & 0xFFu);
  return (int)mx;
}

// Digits of the four new state values (outputs o .. o + 3) of row r, F = 1.
__device__ __forceinline__ void emit_state_digits4(const DevState &st, int r, int o, const uint16_t *h) {
  const int d = st.d;
  int dg[4][3];
  bool in[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) in[q] = bf16_digits3(h[q], 1, dg[q][0], dg[q][1], dg[q][2]);
  int8_t *dst = st.hd + (size_t)r * rec_dig_row_bytes(d);
#pragma unroll
  for (int p = 0; p < 3; ++p)
    *reinterpret_cast<uint32_t *>(dst + rec_dig_off(o, p)) =
        (uint32_t)(uint8_t)dg[0][p] | ((uint32_t)(uint8_t)dg[1][p] << 8) | ((uint32_t)(uint8_t)dg[2][p] << 16) |
        ((uint32_t)(uint8_t)dg[3][p] << 24);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (in[q]) continue;
    RowAux &ax = st.haux[r];
    const int i = atomicAdd(&ax.n, 1);
    if (i < REC_HL) {
      ax.col[i] = o + q;
      ax.val[i] = bf16f(h[q]);
    }
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
      hb[q] = bf16_tanh(pre + (double)bf16f((uint16_t)(q ? ev >> 16 : ev & 0xFFFFu)));
    }
    *reinterpret_cast<uint32_t *>(static_cast<uint16_t *>(st.hbuf) + (size_t)row * d + v0 + i0) =
        (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
  }
}

// A row's list record in registers (32 dwords: F, n, columns, values),
// fetched with eight 16-byte loads at once.
struct AuxRegs {
  uint32_t w[32];
};
__device__ __forceinline__ AuxRegs load_aux(const RowAux *ax) {
  AuxRegs r;
  const u4 *p = reinterpret_cast<const u4 *>(ax);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const u4 v = p[i];
    r.w[4 * i] = v.x;
    r.w[4 * i + 1] = v.y;
    r.w[4 * i + 2] = v.z;
    r.w[4 * i + 3] = v.w;
  }
  return r;
}

// Digit planes (rec_dig_off layout) and list of the state feeding row r.
__device__ __forceinline__ const int8_t *row_digits(const DevState &st, int r) {
  const int src = st.r_hsrc[r];
  return (src >= 0 ? st.s_hd : st.q_hd) + (size_t)(src >= 0 ? src : -1 - src) * rec_dig_row_bytes(st.d);
}
__device__ __forceinline__ const RowAux *row_aux(const DevState &st, int r) {
  const int src = st.r_hsrc[r];
  return src >= 0 ? st.s_haux + src : st.q_haux + (-1 - src);
}

__device__ __forceinline__ bool w_in_window(uint32_t b, int Ew) {
  const uint32_t e8 = (b >> 7) & 0xFFu;
  return (b & 0x7FFFu) == 0u || (int)max(e8, 1u) - 113 - Ew >= 0;
}

// The exact tile: 32 out features x 32 rows, the K range split over the
// RSPLIT_I8 = 4 waves of a 256-thread workgroup (two fit on a compute
// unit); the waves' T_s are added into LDS (integer sums, any order).
// The out-of-window corrections are staged through LDS so that no chain of
// dependent loads is left for the epilogue: the tile's W_h lists (built
// when the decoder is made) and its state rows' lists (sorted by column
// here) are read at the start, and the state values at the W_h lists'
// columns and the W_h values at the state lists' columns are gathered by
// all threads while the K loop runs. A row whose list overflowed, or does
// not fit the tile's staging, is scanned instead (same terms, same order).
constexpr int RSPLIT_I8 = 4;
constexpr int RTHREADS_I8 = 64 * RSPLIT_I8;
constexpr int REC_HTILE = 64;    // staged state-list values per tile
constexpr int REC_GATHER = 2;    // gathered values per thread held through the K loop

struct RecI8Lds {
  int redi[5][RT * RS];
  int src[RT];                   // state source of each row (r_hsrc)
  int F[RT];                     // row exponents
  int hoff[RT], hcnt[RT];        // a row's staged list: start, length (0: scanned or empty)
  int scan[RT];                  // 1: the row is scanned
  int htot;                      // staged state-list values
  int hcol[REC_HTILE];
  float hval[REC_HTILE];
  int woff[RT + 1];
  int wcol[REC_WTILE];
  float wval[REC_WTILE];
  float hg[REC_WTILE][RT];       // state value of row r at W list entry e
  uint16_t wg[REC_HTILE][RT];    // W_h bits of output o at state list entry e
};

__device__ __forceinline__ const uint16_t *src_row16(const DevState &st, int src) {
  return static_cast<const uint16_t *>(src >= 0 ? st.s_h : st.q_h0) + (size_t)(src >= 0 ? src : -1 - src) * st.d;
}

__device__ __forceinline__ void rec_tile_i8(const DevState &st, RecI8Lds &L, int vt, int rt, int R) {
  const int d = st.d, nkb = d / 32;
  const int v0 = vt * RT, r0 = rt * RT;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int kbw = d / RSPLIT_I8 / 32;         // K-blocks of 32 per wave (even)
  const int kb0 = w * kbw;
  // Epilogue mapping: thread -> row j = tid/8, outputs v0 + 4*(tid%8) .. +3.
  const int j = tid >> 3, i0 = (tid & 7) * 4;
  const int row = r0 + j;
  const uint16_t *Wh = static_cast<const uint16_t *>(st.W_h);
  // Tile set-up: wave 0 stages the rows' lists, wave 1 the W_h lists'
  // starts, wave 2 their entries; every thread fetches its embedding pair
  // (its outputs' exponents follow the K loop).
  const uint2 ev = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(st.E) +
                                                    (size_t)st.r_y[min(row, R - 1)] * d + v0 + i0);
  if (tid < RT) {
    const int src = st.r_hsrc[min(r0 + tid, R - 1)];
    const AuxRegs ar = load_aux(src >= 0 ? st.s_haux + src : st.q_haux + (-1 - src));
    const int n = r0 + tid < R ? (int)ar.w[1] : 0;
    L.src[tid] = src;
    L.F[tid] = (int)ar.w[0];
    int cnt = n > REC_HL ? 0 : n;
    int inc = cnt;   // inclusive scan over the 32 rows
#pragma unroll
    for (int o = 1; o < RT; o <<= 1) {
      const int t = __shfl_up(inc, o, RT);
      if (tid >= o) inc += t;
    }
    const int off = inc - cnt;
    const bool scan = n > REC_HL || inc > REC_HTILE;
    if (scan) cnt = 0;
    L.hoff[tid] = off;
    L.hcnt[tid] = cnt;
    L.scan[tid] = scan ? 1 : 0;
    if (tid == RT - 1) L.htot = min(inc, REC_HTILE);
#pragma unroll
    for (int x = 0; x < REC_HL; ++x) {   // insertion into column order
      if (x < cnt) {
        const int c = (int)ar.w[2 + x];
        const float v = __uint_as_float(ar.w[2 + REC_HL + x]);
        int y = off + x;
        for (; y > off && L.hcol[y - 1] > c; --y) {
          L.hcol[y] = L.hcol[y - 1];
          L.hval[y] = L.hval[y - 1];
        }
        L.hcol[y] = c;
        L.hval[y] = v;
      }
    }
  } else if (tid >= 64 && tid < 64 + RT + 1) {
    L.woff[tid - 64] = st.wt_off[vt * (RT + 1) + tid - 64];
  } else if (tid >= 128 && tid < 128 + REC_WTILE) {
    L.wcol[tid - 128] = st.wt_col[vt * REC_WTILE + tid - 128] & 0xFFFF;
    L.wval[tid - 128] = st.wt_val[vt * REC_WTILE + tid - 128];
  }
  // A: lane (h, l) holds the digits of W_h[v0 + l][32 kb + 16 h .. +15];
  // B likewise for state row r0 + l (K values in the same lane order).
  const int8_t *bdig = row_digits(st, min(r0 + l32, R - 1)) + 48 * hh;
  const u4 *ap = reinterpret_cast<const u4 *>(st.wd3) + ((size_t)vt * nkb + kb0) * 3 * 64 + lane;
  __syncthreads();
  // Gathers held in registers through the K loop (the rest after it).
  const int nwe = L.woff[RT] * RT, nhe = L.htot * RT;
  uint16_t gw[REC_GATHER], gh[REC_GATHER];
#pragma unroll
  for (int g = 0; g < REC_GATHER; ++g) {
    const int idx = tid + g * RTHREADS_I8;
    gw[g] = idx < nwe ? src_row16(st, L.src[idx % RT])[L.wcol[idx / RT]] : 0;
    gh[g] = idx < nhe ? Wh[(size_t)(v0 + idx % RT) * d + L.hcol[idx / RT]] : 0;
  }
  v16i T[5];
#pragma unroll
  for (int q = 0; q < 5; ++q) T[q] = v16i{};
  // Two K-blocks of operands in flight. Loads complete in issue order and
  // every step issues the same loads (past the end, the last block again),
  // so the wait before a block's MFMAs leaves the other block's loads
  // outstanding; within a block the order follows first use.
  u4 A[2][3], B[2][3];
  auto load = [&](u4 *Ar, u4 *Br, int kb) {
    Ar[0] = ap[(size_t)(kb * 3) * 64];
#pragma unroll
    for (int b = 0; b < 3; ++b) Br[b] = *reinterpret_cast<const u4 *>(bdig + (kb0 + kb) * 128 + b * 16);
    Ar[1] = ap[(size_t)(kb * 3 + 1) * 64];
    Ar[2] = ap[(size_t)(kb * 3 + 2) * 64];
  };
  load(A[0], B[0], 0);
  __builtin_amdgcn_sched_barrier(0);
  load(A[1], B[1], 1);
  __builtin_amdgcn_sched_barrier(0);
  for (int kb = 0; kb < kbw; kb += 2) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b)
          T[a + b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(v4i, A[s][a]),
                                                           __builtin_bit_cast(v4i, B[s][b]), T[a + b], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      load(A[s], B[s], min(kb + s + 2, kbw - 1));
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int g = 0; g < REC_GATHER; ++g) {
    const int idx = tid + g * RTHREADS_I8;
    if (idx < nwe) L.hg[idx / RT][idx % RT] = bf16f(gw[g]);
    if (idx < nhe) L.wg[idx / RT][idx % RT] = gh[g];
  }
  for (int idx = tid + REC_GATHER * RTHREADS_I8; idx < nwe; idx += RTHREADS_I8)
    L.hg[idx / RT][idx % RT] = bf16f(src_row16(st, L.src[idx % RT])[L.wcol[idx / RT]]);
  for (int idx = tid + REC_GATHER * RTHREADS_I8; idx < nhe; idx += RTHREADS_I8)
    L.wg[idx / RT][idx % RT] = Wh[(size_t)(v0 + idx % RT) * d + L.hcol[idx / RT]];
  const int4 Ew = *reinterpret_cast<const int4 *>(st.w_exp + v0 + i0);
  // T_s: output v0 + 8*(reg/4) + 4*hh + reg%4, row l32.
#pragma unroll
  for (int q = 0; q < 5; ++q)
#pragma unroll
    for (int reg = 0; reg < 16; ++reg)
      atomicAdd(&L.redi[q][l32 * RS + 8 * (reg >> 2) + 4 * hh + (reg & 3)], T[q][reg]);
  __syncthreads();
  // Z = sum_s 128^s T_s (Horner, exact); each sum is cleared for the next
  // tile by the thread that read it.
  double pre[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = j * RS + i0 + q;
    double Z = (double)L.redi[4][idx];
    L.redi[4][idx] = 0;
#pragma unroll
    for (int s2 = 3; s2 >= 0; --s2) {
      Z = fma(Z, 128.0, (double)L.redi[s2][idx]);
      L.redi[s2][idx] = 0;
    }
    pre[q] = Z;
  }
  if (row >= R) return;
  const int F = L.F[j];
  const int ew[4] = {Ew.x, Ew.y, Ew.z, Ew.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    pre[q] = ldexp(pre[q], ew[q] + F - 42);
    // W_h values below their row's window, times the full state value.
    for (int e = L.woff[i0 + q]; e < L.woff[i0 + q + 1]; ++e) pre[q] += (double)L.wval[e] * (double)L.hg[e][j];
  }
  // State values below the window, times the W_h values inside theirs (the
  // others are in the W_h lists).
  auto add_h = [&](double hv, const uint16_t *wb) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (w_in_window(wb[q], ew[q])) pre[q] += (double)bf16f(wb[q]) * hv;
  };
  if (!L.scan[j]) {
    for (int e = L.hoff[j]; e < L.hoff[j] + L.hcnt[j]; ++e) {
      const uint16_t wb[4] = {L.wg[e][i0], L.wg[e][i0 + 1], L.wg[e][i0 + 2], L.wg[e][i0 + 3]};
      add_h((double)L.hval[e], wb);
    }
  } else {
    const uint16_t *hrow = src_row16(st, L.src[j]);
    for (int col = 0; col < d; ++col) {
      const uint32_t hb = hrow[col];
      if (w_in_window(hb, F)) continue;
      const uint16_t wb[4] = {Wh[(size_t)(v0 + i0) * d + col], Wh[(size_t)(v0 + i0 + 1) * d + col],
                              Wh[(size_t)(v0 + i0 + 2) * d + col], Wh[(size_t)(v0 + i0 + 3) * d + col]};
      add_h((double)bf16f((uint16_t)hb), wb);
    }
  }
  uint16_t hb[4];
  const uint32_t e2[2] = {ev.x, ev.y};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    hb[q] = bf16_tanh(pre[q] + (double)bf16f((uint16_t)((q & 1) ? e2[q >> 1] >> 16 : e2[q >> 1] & 0xFFFFu)));
  *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(st.hbuf) + (size_t)row * d + v0 + i0) =
      uint2{(uint32_t)hb[0] | ((uint32_t)hb[1] << 16), (uint32_t)hb[2] | ((uint32_t)hb[3] << 16)};
  emit_state_digits4(st, row, v0 + i0, hb);
}

// Epilogue of a wave's 32 x 32 quadrant (lane (h, l): row `row`, outputs
// v0 + 8g + 4h + i at register 4g + i). Values below the windows: the
// output tile's W_h list (sorted by output, then column) is held one entry
// per lane and walked by the wave, each entry's state value gathered by the
// lanes holding its output; a row's own list is walked by its lanes in
// column order, or the row is scanned if the list overflowed. The fp64
// corrections are thus added in a fixed order.
__device__ __forceinline__ void rec_quadrant_epilogue(const DevState &st, const v16i *T, int v0, int row, int R,
                                                      int src, const RowAux *ax, const int4 *ew4, const uint2 *ev,
                                                      int ne, int wcol, float wval) {
  const int d = st.d;
  const int lane = threadIdx.x & 63, hh = lane >> 5;
  const AuxRegs ar = load_aux(ax);   // in flight with the gathers below
  int ew[16];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    ew[4 * g] = ew4[g].x;
    ew[4 * g + 1] = ew4[g].y;
    ew[4 * g + 2] = ew4[g].z;
    ew[4 * g + 3] = ew4[g].w;
  }
  const uint16_t *hrow = src_row16(st, src);
  // Z = sum_s 128^s T_s (Horner, exact), scaled by 2^(E_w + F - 42).
  double pre[16];
#pragma unroll
  for (int reg = 0; reg < 16; ++reg) {
    double Z = (double)T[4][reg];
#pragma unroll
    for (int s2 = 3; s2 >= 0; --s2) Z = fma(Z, 128.0, (double)T[s2][reg]);
    pre[reg] = Z;
  }
  const int F = (int)ar.w[0], hn = (int)ar.w[1];
#pragma unroll
  for (int reg = 0; reg < 16; ++reg) pre[reg] = ldexp(pre[reg], ew[reg] + F - 42);
  // Entry e (held by lane e) of output f belongs to the lanes with
  // h = (f / 4) % 2, at register 4 (f / 8) + f % 4.
  for (int e0 = 0; e0 < ne; e0 += 16) {
    uint16_t gv[16];
#pragma unroll
    for (int x = 0; x < 16; ++x) {
      const int ce = __shfl(wcol, (e0 + x) & 63);
      gv[x] = (e0 + x < ne && ((ce >> 18) & 1) == hh) ? hrow[ce & 0xFFFF] : (uint16_t)0;
    }
#pragma unroll
    for (int x = 0; x < 16; ++x) {
      if (e0 + x >= ne) break;
      const int ce = __builtin_amdgcn_readfirstlane(__shfl(wcol, e0 + x));
      const float ve = __shfl(wval, e0 + x);
      const int fe = ce >> 16, rege = 4 * (fe >> 3) + (fe & 3);
      if (((fe >> 2) & 1) == hh) {
#pragma unroll
        for (int reg = 0; reg < 16; ++reg)
          if (reg == rege) pre[reg] += (double)ve * (double)bf16f(gv[x]);
      }
    }
  }
  const uint16_t *Wh = static_cast<const uint16_t *>(st.W_h) + (size_t)(v0 + 4 * hh) * d;
  auto add_h = [&](int col, double hv) {
    uint16_t wb[16];
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) wb[reg] = Wh[(size_t)(8 * (reg >> 2) + (reg & 3)) * d + col];
#pragma unroll
    for (int reg = 0; reg < 16; ++reg)
      if (w_in_window(wb[reg], ew[reg])) pre[reg] += (double)bf16f(wb[reg]) * hv;
  };
  if (row >= R) return;
  if (hn <= REC_HL) {
    int last = -1;
    for (int x = 0; x < hn; ++x) {   // next column after `last`
      int c = d;
      uint32_t vb = 0u;
#pragma unroll
      for (int z = 0; z < REC_HL; ++z) {
        const int cz = (int)ar.w[2 + z];
        if (z < hn && cz > last && cz < c) {
          c = cz;
          vb = ar.w[2 + REC_HL + z];
        }
      }
      add_h(c, (double)__uint_as_float(vb));
      last = c;
    }
  } else {
    for (int col = 0; col < d; ++col) {
      const uint32_t hb = hrow[col];
      if (!w_in_window(hb, F)) add_h(col, (double)bf16f((uint16_t)hb));
    }
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint16_t hb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t e = (i & 2) ? ev[g].y : ev[g].x;
      hb[i] = bf16_tanh(pre[4 * g + i] + (double)bf16f((uint16_t)((i & 1) ? e >> 16 : e & 0xFFFFu)));
    }
    const int o = v0 + 8 * g + 4 * hh;
    *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(st.hbuf) + (size_t)row * d + o) =
        uint2{(uint32_t)hb[0] | ((uint32_t)hb[1] << 16), (uint32_t)hb[2] | ((uint32_t)hb[3] << 16)};
    emit_state_digits4(st, row, o, hb);
  }
}

// Large steps: 64 out features x 64 rows per workgroup, each wave one
// 32 x 32 quadrant over the whole K range, so a K-block's operands (64 W_h
// rows and 64 state rows, 12 KB of digits) are fetched once for four
// quadrants: half the bytes per output of the 32 x 32 tiles. The block
// passes through a three-stage LDS ring (one barrier per block) and
// R64_INFLIGHT more blocks are in flight in registers. Lane (h, l) of wave w ends with T_s for
// row r0 + 32 (w / 2) + l and outputs v0 + 32 (w % 2) + 8g + 4h + i.
constexpr int R64_STAGES = 3;
constexpr int R64_INFLIGHT = 2;   // K-blocks in flight in registers (d / 32 a multiple of it)
constexpr int R64_PIECES = 768;   // 16-byte pieces per K-block: 384 of W_h digits, 384 of state digits

struct Rec64Lds {
  u4 stage[R64_STAGES][R64_PIECES];
};

__device__ __forceinline__ void rec_tile64_i8(const DevState &st, Rec64Lds &L, int vq, int rq, int R) {
  const int d = st.d, nkb = d / 32;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int fq = w & 1, rq4 = w >> 1;
  const int vt = 2 * vq + fq, v0 = vt * RT;
  const int r0 = 2 * rq * RT + rq4 * RT;
  // The thread's three pieces of every K-block: piece p < 384 is W_h digit
  // fragment p of output tiles 2vq, 2vq + 1 (the layout of wd3); piece
  // 384 + q is the state fragment q: half q / 192 of the rows, plane
  // (q / 64) % 3, lane q % 64 (row l, bytes 48h + 16 plane of the block).
  const u4 *gp[3];
  int gs[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const int p = tid + RTHREADS_I8 * i;
    if (p < 384) {
      const int f = p / 192, rem = p - 192 * f;
      gp[i] = reinterpret_cast<const u4 *>(st.wd3) + (size_t)(2 * vq + f) * nkb * 192 + rem;
      gs[i] = 192;
    } else {
      const int q = p - 384, hq = q / 192, rem = q - 192 * hq, a = rem / 64, ln = rem & 63;
      const int src = st.r_hsrc[min(2 * rq * RT + hq * RT + (ln & 31), R - 1)];
      gp[i] = reinterpret_cast<const u4 *>((src >= 0 ? st.s_hd : st.q_hd) +
                                           (size_t)(src >= 0 ? src : -1 - src) * rec_dig_row_bytes(d) +
                                           48 * (ln >> 5) + 16 * a);
      gs[i] = 8;
    }
  }
  // Epilogue inputs, fetched before the K loop.
  const int row = r0 + l32, rowc = min(row, R - 1);
  const int src = st.r_hsrc[rowc];
  const int y = st.r_y[rowc];
  const RowAux *ax = src >= 0 ? st.s_haux + src : st.q_haux + (-1 - src);
  const int ne = st.wt_off[vt * (RT + 1) + RT];
  const int wcol = lane < ne ? st.wt_col[vt * REC_WTILE + lane] : 0;
  const float wval = lane < ne ? st.wt_val[vt * REC_WTILE + lane] : 0.0f;
  int4 ew4[4];
  uint2 ev[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int o = v0 + 8 * g + 4 * hh;
    ew4[g] = *reinterpret_cast<const int4 *>(st.w_exp + o);
    ev[g] = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(st.E) + (size_t)y * d + o);
  }

  u4 G[R64_INFLIGHT][3];
  auto gload = [&](u4 *g, int kb) {
#pragma unroll
    for (int i = 0; i < 3; ++i) g[i] = gp[i][(size_t)kb * gs[i]];
  };
  auto lstore = [&](int sg, const u4 *g) {
#pragma unroll
    for (int i = 0; i < 3; ++i) L.stage[sg][tid + RTHREADS_I8 * i] = g[i];
  };
  v16i T[5];
#pragma unroll
  for (int q = 0; q < 5; ++q) T[q] = v16i{};
  auto compute = [&](int sg) {
    const u4 *stg = L.stage[sg];
    u4 A[3], B[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      A[a] = stg[fq * 192 + a * 64 + lane];
      B[a] = stg[384 + rq4 * 192 + a * 64 + lane];
    }
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 3; ++b)
        T[a + b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(v4i, A[a]), __builtin_bit_cast(v4i, B[b]),
                                                         T[a + b], 0, 0, 0);
  };
  // Blocks 0 and 1 in stages 0 and 1, blocks 2 .. R64_INFLIGHT + 1 in
  // flight. Step j reads stage j % 3, then stores block j + 2 into stage
  // (j + 2) % 3 (last read at step j - 1, before the barrier that ended it)
  // and fetches block j + 2 + R64_INFLIGHT; past the end the last block is
  // fetched and stored again into a stage no later step reads, so every
  // step issues the same loads.
  gload(G[0], 0);
  gload(G[1], 1);
  lstore(0, G[0]);
  lstore(1, G[1]);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int j = 0; j < R64_INFLIGHT; ++j) gload(G[j], min(2 + j, nkb - 1));
  __syncthreads();
  for (int kb = 0; kb < nkb; kb += R64_INFLIGHT) {
#pragma unroll
    for (int j = 0; j < R64_INFLIGHT; ++j) {
      compute((kb + j) % R64_STAGES);
      lstore((kb + j + 2) % R64_STAGES, G[j]);
      __builtin_amdgcn_sched_barrier(0);
      gload(G[j], min(kb + j + 2 + R64_INFLIGHT, nkb - 1));
      __syncthreads();
    }
  }
  rec_quadrant_epilogue(st, T, v0, row, R, src, ax, ew4, ev, ne, wcol, wval);
}

// Persistent exact bf16 recurrence over the active tiles (RecWalk): 64 x 64
// tiles for steps with enough rows to fill half the grid with them, else
// 32 x 32 tiles with the K range split over the waves.
__global__ __launch_bounds__(RTHREADS_I8, 2) void k_rec_i8(DevState st) {
  const int R = st.ctrl->R;
  if (R <= 0) return;
  __shared__ union {
    RecI8Lds ks;
    Rec64Lds t64;
  } L;
  const int nq = (R + 2 * RT - 1) / (2 * RT), nvq = st.d / (2 * RT);
  if (nq * nvq * 2 >= (int)gridDim.x) {
    // 64 x 64 tiles once they fill half the grid
    const RecWalk walk(nvq, nq, blockIdx.x & 7);
    for (int t = (int)(blockIdx.x >> 3); t < walk.n; t += (int)(gridDim.x >> 3)) {
      int vq, rq;
      walk.at(t, vq, rq);
      rec_tile64_i8(st, L.t64, vq, rq, R);
      __syncthreads();   // the ring is reused by the next tile
    }
    return;
  }
  const RecWalk walk(st.d / RT, (R + RT - 1) / RT, blockIdx.x & 7);
  for (int i = threadIdx.x; i < 5 * RT * RS; i += RTHREADS_I8) (&L.ks.redi[0][0])[i] = 0;
  __syncthreads();
  for (int t = (int)(blockIdx.x >> 3); t < walk.n; t += (int)(gridDim.x >> 3)) {
    int vt, rt;
    walk.at(t, vt, rt);
    rec_tile_i8(st, L.ks, vt, rt, R);
    __syncthreads();   // L is reused by the next tile
  }
}

// Digits of `count` bf16 rows [count][d] (one workgroup per row): the row
// exponent, the three planes and the list of values below the window.
__global__ __launch_bounds__(256) void k_row_digits(const uint16_t *__restrict__ rows, int count, int d,
                                                    int8_t *__restrict__ dig, RowAux *__restrict__ aux) {
  const int r = blockIdx.x;
  if (r >= count) return;
  const uint16_t *x = rows + (size_t)r * d;
  __shared__ int smx, sn;
  if (threadIdx.x == 0) {
    smx = 1;
    sn = 0;
  }
  __syncthreads();
  atomicMax(&smx, bf16_max_eu(x, threadIdx.x, d, blockDim.x));
  __syncthreads();
  const int E = smx - 126;
  int8_t *dr = dig + (size_t)r * rec_dig_row_bytes(d);
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    int a0, a1, a2;
    if (!bf16_digits3(x[i], E, a0, a1, a2)) {
      const int k = atomicAdd(&sn, 1);
      if (k < REC_HL) {
        aux[r].col[k] = i;
        aux[r].val[k] = bf16f(x[i]);
      }
    }
    dr[rec_dig_off(i, 0)] = (int8_t)a0;
    dr[rec_dig_off(i, 1)] = (int8_t)a1;
    dr[rec_dig_off(i, 2)] = (int8_t)a2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    aux[r].F = E;
    aux[r].n = sn;
  }
}

// Lists of the new states emptied (F = 1: tanh outputs are below 2).
__global__ void k_aux_reset(RowAux *aux, int count) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < count) {
    aux[r].F = 1;
    aux[r].n = 0;
  }
}

// W_h, once per decoder: row exponents and empty lists (one wave per row) ...
__global__ void k_w_exp(DevState st) {
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (o >= st.d) return;
  int mx = bf16_max_eu(static_cast<const uint16_t *>(st.W_h) + (size_t)o * st.d, lane, st.d, 64);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, __shfl_xor(mx, off, 64));
  if (lane == 0) {
    st.w_exp[o] = mx - 126;
    st.w_ln[o] = 0;
    if (o == 0) st.w_ln[st.d] = 0;
  }
}

// ... the digit planes in fragment order (a thread per 16 values of a row;
// lane (h, l) of output tile o/32 at K-block kb: row 32*(o/32) + l, K values
// kb*32 + 16h .. +15, the K mapping of the state fragments) and the lists ...
__global__ void k_w_digits(DevState st) {
  const int d = st.d, nkb = d / 32;
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (long long)d * (d / 16)) return;
  const int o = (int)(t / (d / 16)), k0 = (int)(t % (d / 16)) * 16;
  const int Ew = st.w_exp[o];
  const uint16_t *row = static_cast<const uint16_t *>(st.W_h) + (size_t)o * d;
  uint32_t word[3][4] = {};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint32_t b = row[k0 + e];
    int dg[3];
    if (!bf16_digits3(b, Ew, dg[0], dg[1], dg[2])) {
      const int idx = atomicAdd(&st.w_ln[o], 1);
      if (idx < REC_WLIST) {
        st.w_li[o * REC_WLIST + idx] = k0 + e;
        st.w_lv[o * REC_WLIST + idx] = bf16f((uint16_t)b);
      }
    }
#pragma unroll
    for (int a = 0; a < 3; ++a) word[a][e >> 2] |= (uint32_t)(uint8_t)dg[a] << (8 * (e & 3));
  }
  const int kb = k0 / 32, ln = ((k0 % 32) / 16) * 32 + (o & 31);
  u4 *dst = reinterpret_cast<u4 *>(st.wd3) + ((size_t)(o / 32) * nkb + kb) * 3 * 64 + ln;
#pragma unroll
  for (int a = 0; a < 3; ++a) dst[a * 64] = u4{word[a][0], word[a][1], word[a][2], word[a][3]};
}

// ... and, per output tile, the rows' lists sorted by column and
// concatenated (one thread per row), each entry's column with its row in
// the tile above bit 16; w_ln[d] = 1 if a list overflowed.
__global__ void k_w_tiles(DevState st) {
  const int vt = blockIdx.x, o = threadIdx.x;   // 32 threads
  const int n = st.w_ln[vt * RT + o];
  __shared__ int off[RT + 1];
  if (o == 0) {
    off[0] = 0;
    for (int x = 0; x < RT; ++x) off[x + 1] = off[x] + min(st.w_ln[vt * RT + x], REC_WLIST);
  }
  __syncthreads();
  const bool bad = n > REC_WLIST || off[RT] > REC_WTILE;
  if (bad) st.w_ln[st.d] = 1;   // every writer stores the same value
  st.wt_off[vt * (RT + 1) + o] = off[o];
  if (o == 0) st.wt_off[vt * (RT + 1) + RT] = off[RT];
  if (bad) return;
  int col[REC_WLIST];
  float val[REC_WLIST];
  const int m = min(n, REC_WLIST);
  const int g = (vt * RT + o) * REC_WLIST;
  for (int x = 0; x < m; ++x) {
    col[x] = st.w_li[g + x];
    val[x] = st.w_lv[g + x];
  }
  // insertion sort by column (the order of the fp64 corrections)
  for (int x = 1; x < m; ++x)
    for (int y = x; y > 0 && col[y - 1] > col[y]; --y) {
      const int c = col[y];
      col[y] = col[y - 1];
      col[y - 1] = c;
      const float v = val[y];
      val[y] = val[y - 1];
      val[y - 1] = v;
    }
  for (int x = 0; x < m; ++x) {
    st.wt_col[vt * REC_WTILE + off[o] + x] = col[x] | (o << 16);
    st.wt_val[vt * REC_WTILE + off[o] + x] = val[x];
  }
}

// Persistent launch over the active tiles (rows of this step only): the
// workgroups of XCD x walk that XCD's block of tiles (RecWalk).
template <bool BF16>
__global__ __launch_bounds__(RTHREADS) void k_rec(DevState st) {
  const int R = st.ctrl->R;
  if (R <= 0) return;
  const RecWalk walk(st.d / RT, (R + RT - 1) / RT, blockIdx.x & 7);
  __shared__ typename std::conditional<BF16, double, float>::type red[RSPLIT][RT * RS];
  for (int t = (int)(blockIdx.x >> 3); t < walk.n; t += (int)(gridDim.x >> 3)) {
    int vt, rt;
    walk.at(t, vt, rt);
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

hipError_t launch_rec_prepare(const DevState &st, hipStream_t s) {
  const int d = st.d;
  hipLaunchKernelGGL(k_w_exp, dim3((d + 3) / 4), dim3(256), 0, s, st);
  const long long nt = (long long)d * (d / 16);
  hipLaunchKernelGGL(k_w_digits, dim3((unsigned)((nt + 255) / 256)), dim3(256), 0, s, st);
  hipLaunchKernelGGL(k_w_tiles, dim3(d / RT), dim3(RT), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_row_digits(const DevState &st, const void *rows, int count, int8_t *dig, RowAux *aux,
                             hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_row_digits, dim3(count), dim3(256), 0, s, static_cast<const uint16_t *>(rows), count, st.d,
                     dig, aux);
  return hipGetLastError();
}

hipError_t launch_aux_reset(RowAux *aux, int count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_aux_reset, dim3((count + 255) / 256), dim3(256), 0, s, aux, count);
  return hipGetLastError();
}

hipError_t launch_rec(const DevState &st, hipStream_t s) {
  // Multiple of 8, no more than the tiles of a full step, and at most the
  // workgroups that fit on the device at once: two per compute unit for
  // bf16 (66 KB of LDS each), four for fp32 (33 KB).
  const int tiles = xcd_grid((st.d / RT) * ((st.R_max + RT - 1) / RT));
  if (st.rec_i8) {
    const int G = std::max(8, std::min(st.n_cu * 2 / 8 * 8, tiles));
    hipLaunchKernelGGL(k_rec_i8, dim3(G), dim3(RTHREADS_I8), 0, s, st);
    return hipGetLastError();
  }
  const int G = std::max(8, std::min(st.n_cu / (st.dtype == 1 ? 4 : 2) * 8, tiles));
  if (st.dtype == 1)
    hipLaunchKernelGGL(k_rec<true>, dim3(G), dim3(RTHREADS), 0, s, st);
  else
    hipLaunchKernelGGL(k_rec<false>, dim3(G), dim3(RTHREADS), 0, s, st);
  return hipGetLastError();
}

}  // namespace sb
