// Small device helpers shared by the decoder-step GEMM kernels.
#pragma once

#include "sb_internal.h"

namespace sb {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef double d4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));

// Address of the K-contiguous previous state feeding batch row r: the slot's
// state, or the queued encoding h0 of a beam that has not stepped yet.
__device__ __forceinline__ const unsigned char *state_row(const DevState &st, int r, int rowbytes) {
  const int src = st.r_hsrc[r];
  if (src >= 0) return static_cast<const unsigned char *>(st.s_h) + (size_t)src * rowbytes;
  return static_cast<const unsigned char *>(st.q_h0) + (size_t)(-1 - src) * rowbytes;
}

// Number of workgroups to launch for G tiles: a multiple of the 8 XCDs.
__host__ __device__ inline int xcd_grid(int G) { return (G + 7) / 8 * 8; }

// XCD-aware tile order. Workgroup ids are dealt round robin to the 8 XCDs;
// remap so that each XCD walks a contiguous range of tiles in which the
// row-tile index varies fastest: workgroups sharing one weight tile then
// share that XCD's L2. Returns false for the padding workgroups.
__device__ __forceinline__ bool tile_of(int nvt, int nrt, int &vt, int &rt) {
  const int G = nvt * nrt;
  const int Gp = xcd_grid(G);
  const int g = blockIdx.x;
  const int lin = (g & 7) * (Gp >> 3) + (g >> 3);
  if (lin >= G) return false;
  vt = lin / nrt;
  rt = lin - vt * nrt;
  return true;
}

__device__ __forceinline__ float bf16f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

}  // namespace sb
