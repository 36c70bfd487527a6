// Vocabulary projection of the synthetic decoder D (Sec. 2) on gfx950 MFMA,
// fused with the EOS bias, an online log-sum-exp and a per-row partial top-k:
//   z = W_out h,  z[0] += beta (t - L_x)      [R,d] x [V,d]^T
// The R x |V| logits never reach memory: each workgroup writes, per row and
// 128-wide vocabulary tile, (max, sum exp) and its best keys (value, token).
//
// Workgroups of 8 waves walk the step's tiles on a persistent grid. Tile
// kinds (chosen per step on the device from the row count):
//   - 128 vocabulary rows x 1..4 blocks of 32 batch rows: the K range is
//     split in two fixed halves, waves 0-3 summing the first, waves 4-7 the
//     second, each wave over its own 32 vocabulary rows; the two partial
//     sums are added once at the end;
//   - 128 vocabulary rows x 5..8 blocks: each wave group takes half of the
//     blocks and sums the two K halves one after the other into two
//     accumulator sets, added once at the end;
//   - bf16 only, 256 vocabulary rows x 4 blocks: K halves as in the first
//     kind, each wave over 64 vocabulary rows.
// In all of them an output accumulates its K halves through the same MFMA
// sequence and adds them once, so a row's result does not depend on the
// batch or on the tiling.
//
// The same tile walk, with W_kv in place of W_out and a bf16 store in place
// of the log-sum-exp / top-k epilogue, appends each expansion's KV rows
// (k_kv_append, below).
//
// W_out is streamed straight into registers from a copy laid out in MFMA
// fragment order (one coalesced 1 KB load per wave and fragment), kept D
// chunks ahead; the states of each half pass through a double-buffered LDS
// tile shared by the waves of that half, loaded D chunks ahead as well.
// Blocks of 32 rows past R are neither loaded nor computed.
#include <algorithm>

#include "mfma_common.h"
#include "topk.h"
#include "wave.h"

namespace sb {
namespace {

constexpr int THREADS = 512;
constexpr int NB = 4;            // 32-row batch blocks per workgroup
constexpr int TR = 32 * NB;      // batch rows per workgroup
constexpr int TV = GEMM_BV;      // vocabulary rows per workgroup (4 waves x 32)
constexpr int CH = 128;          // bytes of a row's K chunk
constexpr int LS = CH + 16;      // padded LDS row stride (bytes)
constexpr int FRAG = 1024;       // bytes of one wave-wide 16-byte-per-lane fragment
constexpr int WCH = 4 * FRAG;    // bytes of one wave's W_out fragments per chunk

template <int KB>
union ProjSmem {
  unsigned char B[2][2][TR][LS];          // [buffer][wave group][row][byte]
  float red[2][4][2][16][64];             // [sending half][slice][block][reg][lane]
  float xch[4][TR][part_width(KB)];       // [slice][row][max, sumexp, keys]
  // [buffer][group][slice][row][...]: with 4-key lists one buffer per owned
  // block, else two used in turn
  float xr[KB == 4 ? NB : 2][2][4][32][part_width(KB)];
  float xw[KB == 4 ? 2 : 1][4][TR][part_width(KB)];   // wide tile: [128-row vocabulary tile][slice][row][...]
};

// K loop of one wave over its half: acc[b] (b < NBV) += W_out fragment x
// batch block b. Chunk c of the half: W_out fragments at abase + c * 16 KB
// (+ lane * 16 + q * 1 KB), the half's state tile at bbase + c * 128 bytes
// (+ boff[u]). Loads of a chunk are issued together, D chunks ahead of use,
// at indices clamped to the last chunk so that no load sits in a branch.
// With NA = 2 the wave covers two adjacent 32-row vocabulary slices
// (fragments at abase and abase + WCH) and acc[x * NBV + bb] is slice x,
// block bb; each state fragment read from LDS then feeds two MFMAs.
template <bool BF16, int NBV, int D, int NA = 1>
__device__ __forceinline__ void proj_mainloop(unsigned char (*Bt)[LS], unsigned char (*Bt1)[LS],
                                              const unsigned char *abase, uint32_t alane,
                                              const unsigned char *bbase, const uint32_t *boff, int srow,
                                              int scol, int nh, int l32, int h, f16v *acc) {
  u4 a[D][NA * 4];
  u4 b[D][NBV];
  auto loadA = [&](int c, u4 *dst) {
    const unsigned char *p = abase + (uint32_t)c * (uint32_t)(4 * WCH);
#pragma unroll
    for (int x = 0; x < NA; ++x)
#pragma unroll
      for (int q = 0; q < 4; ++q) dst[4 * x + q] = *reinterpret_cast<const u4 *>(p + x * WCH + alane + q * FRAG);
  };
  auto loadB = [&](int c, u4 *dst) {
    const unsigned char *p = bbase + (uint32_t)c * CH;
#pragma unroll
    for (int u = 0; u < NBV; ++u) dst[u] = *reinterpret_cast<const u4 *>(p + boff[u]);
  };
  auto storeB = [&](unsigned char (*T)[LS], const u4 *src) {
#pragma unroll
    for (int u = 0; u < NBV; ++u) *reinterpret_cast<u4 *>(&T[srow + 32 * u][scol]) = src[u];
  };
  auto compute = [&](unsigned char (*T)[LS], const u4 *af) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // K permutation: lane half h at piece q feeds k = chunk + 16h + 4q + e
      // (fp32) or chunk + 32h + 8q + e (bf16), identically for both operands.
      u4 braw[NBV];
#pragma unroll
      for (int bb = 0; bb < NBV; ++bb) braw[bb] = *reinterpret_cast<const u4 *>(&T[32 * bb + l32][64 * h + 16 * q]);
      // Raised wave priority while this piece's MFMAs issue, so that of the
      // two waves sharing a SIMD the one whose operands are in keeps the
      // matrix unit fed (fp32 steps of 128-640 rows: 1-2 % faster).
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int bb = 0; bb < NBV; ++bb) {
#pragma unroll
        for (int x = 0; x < NA; ++x) {
          f16v &c = acc[x * NBV + bb];
          if constexpr (BF16) {
            c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf8, af[4 * x + q]),
                                                        __builtin_bit_cast(bf8, braw[bb]), c, 0, 0, 0);
          } else {
            const f4 av = __builtin_bit_cast(f4, af[4 * x + q]);
            const f4 bv = __builtin_bit_cast(f4, braw[bb]);
#pragma unroll
            for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], bv[e], c, 0, 0, 0);
          }
        }
      }
      __builtin_amdgcn_s_setprio(0);
    }
  };

  // Loads complete in issue order, so a wait for one chunk's states also
  // waits for every load issued before them: the scheduling fences keep the
  // issue order chunk by chunk (W_out, then states), which leaves D-1 chunks
  // in flight at every wait.
  // Prologue: chunks 0 .. D-1 in flight, chunk 0's states in LDS.
#pragma unroll
  for (int c = 0; c < D; ++c) {
    loadA(min(c, nh - 1), a[c]);
    __builtin_amdgcn_sched_barrier(0);
    loadB(min(c, nh - 1), b[c]);
    __builtin_amdgcn_sched_barrier(0);
  }
  storeB(Bt, b[0]);
  __syncthreads();

  for (int i0 = 0; i0 < nh; i0 += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      const int i = i0 + j;   // i % D == j
      if (i < nh) compute((i & 1) ? Bt1 : Bt, a[j]);
      __builtin_amdgcn_sched_barrier(0);
      // States of chunk i+1 sit in b[(j+1) % D]; buffer (i+1)&1 was last
      // read before the previous barrier.
      if (i + 1 < nh) storeB(((i + 1) & 1) ? Bt1 : Bt, b[(j + 1) % D]);
      __builtin_amdgcn_sched_barrier(0);
      loadA(min(i + D, nh - 1), a[j]);
      __builtin_amdgcn_sched_barrier(0);
      loadB(min(i + D, nh - 1), b[j]);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
    }
  }
}

// Lane-level epilogue of one 32-row block: lane holds batch row l32 of the
// block and the wave's vocabulary rows v0 + 32wv + 8*(reg/4) + 4h + reg%4
// (increasing with reg). Adds the EOS bias, folds the 16 logits into
// (max, sum exp) and a sorted best-KB key list, then combines lanes l and
// l+32 (same row), which end with identical results. KB = 4 takes a
// cheaper network than a full sort.
template <int KB>
__device__ __forceinline__ void block_lists(const f16v &z, int v0, int wv, int h, int V, float bias, float &m_out,
                                            float &s_out, TopK<KB> &tk) {
  float vals[16];
  if (v0 != 0 && v0 + TV <= V) {   // interior tile: no EOS bias, no rows past V
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) vals[reg] = z[reg];
  } else {
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int v = v0 + 32 * wv + 8 * (reg >> 2) + 4 * h + (reg & 3);
      const float zz = v == 0 ? z[reg] + bias : z[reg];
      vals[reg] = v < V ? zz : -INFINITY;
    }
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
  for (int reg = 0; reg < 16; ++reg) keys[reg] = make_key(vals[reg], v0 + 32 * wv + 8 * (reg >> 2) + 4 * h + (reg & 3));
  TopK<KB> mine;
  if constexpr (KB == 4) {
    top4_of_16(keys, mine);
  } else {
    bitonic_sort_desc<16>(keys);
#pragma unroll
    for (int q = 0; q < KB; ++q) mine.k[q] = keys[q];
  }
  TopK<KB> lo, hi;
#pragma unroll
  for (int q = 0; q < KB; ++q) stage64<5>(mine.k[q], lo.k[q], hi.k[q]);
  topk_merge(lo, hi);
  tk = lo;
  uint32_t ma, mb, sa, sb;
  stage32<5>(__float_as_uint(m), ma, mb);
  stage32<5>(__float_as_uint(s), sa, sb);
  m = __uint_as_float(ma);
  s = __uint_as_float(sa);
  lse_merge(m, s, __uint_as_float(mb), __uint_as_float(sb));
  m_out = m;
  s_out = s;
}

// Partial record of (row j, vocabulary tile vt): the merge of the four
// vocabulary slices' (max, sum exp, key list), read from LDS.
template <int KB>
__device__ __forceinline__ void write_record(const DevState &st, int j, int vt, const float *const *slices) {
  constexpr int PW = part_width(KB);
  float m = -INFINITY, s = 0.0f;
  TopK<KB> tk;
  topk_init(tk);
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const float *p = slices[x];
    TopK<KB> o;
    topk_load(o, p + 2);
    lse_merge(m, s, p[0], p[1]);
    topk_merge(tk, o);
  }
  float rec[PW];
  rec[0] = m;
  rec[1] = s;
  topk_store(rec + 2, tk);
#pragma unroll
  for (int x = 2 + 2 * KB; x < PW; ++x) rec[x] = 0.0f;
  u4 *out = reinterpret_cast<u4 *>(st.part + ((size_t)j * st.S + vt) * PW);
#pragma unroll
  for (int x = 0; x < PW / 4; ++x)
    out[x] = u4{__float_as_uint(rec[4 * x]), __float_as_uint(rec[4 * x + 1]), __float_as_uint(rec[4 * x + 2]),
                __float_as_uint(rec[4 * x + 3])};
}

// KV append epilogue of one 32-row block of a wave's 32 outputs (the layout
// of block_lists): row j's bf16(sum) values go to the KV rows of the
// expanded candidate, at (beam, level t-1, rank), outputs o0 + 8*(reg/4) +
// 4h + reg%4.
__device__ __forceinline__ uint16_t bf16_rne_f(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ void kv_store_block(const DevState &st, const f16v &z, int o0, int h, int j, int R) {
  if (j >= R) return;
  const int NO = st.kv_layers * 2 * st.d;
  const int slot = st.r_slot[j], beam = slot / st.k, rank = slot - beam * st.k;
  uint16_t *out = st.kvs + (((size_t)beam * st.max_len_cap + (st.r_t[j] - 1)) * st.k + rank) * NO + o0 + 4 * h;
#pragma unroll
  for (int gq = 0; gq < 4; ++gq) {
    u2 pk;
    pk[0] = (uint32_t)bf16_rne_f(z[4 * gq + 0]) | ((uint32_t)bf16_rne_f(z[4 * gq + 1]) << 16);
    pk[1] = (uint32_t)bf16_rne_f(z[4 * gq + 2]) | ((uint32_t)bf16_rne_f(z[4 * gq + 3]) << 16);
    *reinterpret_cast<u2 *>(out + 8 * gq) = pk;
  }
}

// Weights and rows a tile walk reads: W_out and the projection input for
// the vocabulary projection; W_kv and the new states for the KV append.
struct GemmOperands {
  const unsigned char *w;   // fragment-ordered weights, 128 outputs per tile
  const void *in;           // [R][d] rows
};

// Tile of at most 4 blocks (128 rows from r0): the K range is split in two
// fixed halves, waves 0-3 summing the first, waves 4-7 the second; the two
// partial sums are added once.
template <bool BF16, int KB, bool KV>
__device__ __forceinline__ void proj_tile_ksplit(const DevState &st, const GemmOperands &op, ProjSmem<KB> &sm, int vt,
                                                 int r0, int R, int nbv) {
  const int d = st.d, V = st.V;
  const int v0 = vt * TV;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = w >> 2, wv = w & 3;               // K half, vocabulary slice
  const int l32 = lane & 31, h = lane >> 5;
  const int rowbytes = d * (BF16 ? 2 : 4);
  const int nk = rowbytes / CH;                   // even: d is a multiple of 64 (fp32) / 128 (bf16)
  const int nh = nk >> 1;
  const int kbeg = g * nh;

  // W_out fragments of this wave: chunk kt at ((vt*nk + kt)*4 + wv) * 4 KB.
  const unsigned char *abase = op.w + ((size_t)(vt * nk + kbeg) * 4 + wv) * WCH;
  // State staging: thread -> rows (tg/8) + 32u of the tile (clamped to R-1),
  // 16-byte column tg%8 of the half's chunk.
  const int tg = tid & 255;
  const int srow = tg >> 3, scol = (tg & 7) * 16;
  uint32_t boff[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) boff[u] = (uint32_t)min(r0 + srow + 32 * u, R - 1) * (uint32_t)rowbytes + scol;
  const unsigned char *bbase = static_cast<const unsigned char *>(op.in) + (size_t)kbeg * CH;
  f16v acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f16v{};
  // One mainloop instantiation per count of valid 32-row blocks, so the
  // K loop has no per-block branches.
  unsigned char (*Bt)[LS] = sm.B[0][g];
  unsigned char (*Bt1)[LS] = sm.B[1][g];
  const uint32_t alane = (uint32_t)lane * 16u;
  switch (nbv) {
    case 1: proj_mainloop<BF16, 1, 3>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc); break;
    case 2: proj_mainloop<BF16, 2, 3>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc); break;
    case 3: proj_mainloop<BF16, 3, 3>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc); break;
    default: proj_mainloop<BF16, 4, 3>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc); break;
  }

  // Combine the halves. Half g owns blocks 2g and 2g+1: it sends its sums of
  // the other half's blocks through LDS and adds the received ones to its own
  // (one addition per output, commutative, so the order is fixed).
  f16v own[2], snd[2];
#pragma unroll
  for (int bl = 0; bl < 2; ++bl) {
    own[bl] = g ? acc[2 + bl] : acc[bl];
    snd[bl] = g ? acc[bl] : acc[2 + bl];
  }
#pragma unroll
  for (int bl = 0; bl < 2; ++bl) {
    if (2 * (1 - g) + bl < nbv) {
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) sm.red[g][wv][bl][reg][lane] = snd[bl][reg];
    }
  }
  __syncthreads();
#pragma unroll
  for (int bl = 0; bl < 2; ++bl) {
    if (2 * g + bl < nbv) {
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) own[bl][reg] += sm.red[1 - g][wv][bl][reg][lane];
    }
  }

  if constexpr (KV) {
#pragma unroll
    for (int bl = 0; bl < 2; ++bl)
      if (2 * g + bl < nbv) kv_store_block(st, own[bl], v0 + 32 * wv, h, r0 + 32 * (2 * g + bl) + l32, R);
    return;
  }

  // Epilogue on the owned blocks 2g + bl.
  TopK<KB> tks[2];
  float ms[2], ss[2];
#pragma unroll
  for (int bl = 0; bl < 2; ++bl) {
    const int blk = 2 * g + bl;
    if (blk < nbv) {
      const int j = r0 + 32 * blk + l32;
      const float bias = (v0 == 0 && j < R) ? st.beta * (float)(st.r_t[j] - st.r_Lx[j]) : 0.0f;
      block_lists<KB>(own[bl], v0, wv, h, V, bias, ms[bl], ss[bl], tks[bl]);
    }
  }
  __syncthreads();   // the exchange area is reused below
#pragma unroll
  for (int bl = 0; bl < 2; ++bl) {
    const int blk = 2 * g + bl;
    if (blk < nbv && lane < 32) {
      float *p = sm.xch[wv][32 * blk + l32];
      p[0] = ms[bl];
      p[1] = ss[bl];
      topk_store(p + 2, tks[bl]);
    }
  }
  __syncthreads();
  // Wave w < 4 merges the four vocabulary slices of batch block w.
  if (w < nbv && lane < 32) {
    const int row = 32 * w + l32;
    const int j = r0 + row;
    if (j < R) {
      const float *sl[4] = {sm.xch[0][row], sm.xch[1][row], sm.xch[2][row], sm.xch[3][row]};
      write_record<KB>(st, j, vt, sl);
    }
  }
}

// Tile of 5 to 8 blocks (rows r0 .. r0+255): the blocks are split between
// the two wave groups (group 0 takes nbh = ceil(nbt/2), group 1 the other
// nbt - nbh, so an odd count leaves group 1 one block short rather than
// computing a padding block: the two waves that share a SIMD then issue
// nbt blocks' MFMAs, not 2 nbh), and every wave sums its blocks over the
// first K half and then over the second, in two accumulators added once at
// the end: the same order of additions as a K-split tile, so a row's
// logits do not depend on how the step was tiled.
template <bool BF16, int KB, bool KV>
__device__ __forceinline__ void proj_tile_big(const DevState &st, const GemmOperands &op, ProjSmem<KB> &sm, int vt,
                                              int r0, int R, int nbt) {
  const int d = st.d, V = st.V;
  const int v0 = vt * TV;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = w >> 2, wv = w & 3;               // row group, vocabulary slice
  const int l32 = lane & 31, h = lane >> 5;
  const int rowbytes = d * (BF16 ? 2 : 4);
  const int nk = rowbytes / CH;
  const int nh = nk >> 1;
  const int nbh = (nbt + 1) >> 1;                 // blocks of group 0 (3 or 4)
  const int nbg = g ? nbt - nbh : nbh;            // blocks of this group (2 to 4)
  const int gb0 = g * nbh;                        // first block of this group

  const int tg = tid & 255;
  const int srow = tg >> 3, scol = (tg & 7) * 16;
  uint32_t boff[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u)
    boff[u] = (uint32_t)min(r0 + 32 * (gb0 + u) + srow, R - 1) * (uint32_t)rowbytes + scol;
  unsigned char (*Bt)[LS] = sm.B[0][g];
  unsigned char (*Bt1)[LS] = sm.B[1][g];
  const uint32_t alane = (uint32_t)lane * 16u;
  const unsigned char *hb = static_cast<const unsigned char *>(op.in);
  f16v acc0[NB], acc1[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    acc0[b] = f16v{};
    acc1[b] = f16v{};
  }
  // The two K halves in turn, each into its own accumulators.
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int kbeg = half * nh;
    const unsigned char *abase = op.w + ((size_t)(vt * nk + kbeg) * 4 + wv) * WCH;
    const unsigned char *bbase = hb + (size_t)kbeg * CH;
    f16v *acc = half ? acc1 : acc0;
    if (half) __syncthreads();   // the staging tile of the first half is done
    // Both instantiations pass the same barriers (one per chunk).
    if (nbg == 2)
      proj_mainloop<BF16, 2, 2>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc);
    else if (nbg == 3)
      proj_mainloop<BF16, 3, 2>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc);
    else
      proj_mainloop<BF16, 4, 2>(Bt, Bt1, abase, alane, bbase, boff, srow, scol, nh, l32, h, acc);
  }

  if constexpr (KV) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int blk = gb0 + i;
      if (i < nbh && blk < nbt) {
        f16v z;
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) z[reg] = acc0[i][reg] + acc1[i][reg];
        kv_store_block(st, z, v0 + 32 * wv, h, r0 + 32 * blk + l32, R);
      }
    }
  } else if constexpr (KB == 4) {
    // Epilogue: the lane lists of every owned block, then wave i of each
    // group merges block i's four vocabulary slices, all blocks at once.
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int blk = gb0 + i;
      if (i < nbh && blk < nbt) {
        f16v z;
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) z[reg] = acc0[i][reg] + acc1[i][reg];
        const int j = r0 + 32 * blk + l32;
        const float bias = (v0 == 0 && j < R) ? st.beta * (float)(st.r_t[j] - st.r_Lx[j]) : 0.0f;
        float m, s;
        TopK<KB> tk;
        block_lists<KB>(z, v0, wv, h, V, bias, m, s, tk);
        if (lane < 32) {
          float *p = sm.xr[i][g][wv][l32];
          p[0] = m;
          p[1] = s;
          topk_store(p + 2, tk);
        }
      }
    }
    __syncthreads();
    const int blk = gb0 + wv;
    if (wv < nbh && blk < nbt && lane < 32) {
      const int j = r0 + 32 * blk + l32;
      if (j < R) {
        const float *sl[4] = {sm.xr[wv][g][0][l32], sm.xr[wv][g][1][l32], sm.xr[wv][g][2][l32], sm.xr[wv][g][3][l32]};
        write_record<KB>(st, j, vt, sl);
      }
    }
  } else {
    // Epilogue, one owned block at a time: lane lists, then wave i of the
    // group merges block i's four vocabulary slices (double-buffered LDS).
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i < nbh) {
        const int blk = gb0 + i;
        const int buf = i & 1;
        if (blk < nbt) {
          f16v z;
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) z[reg] = acc0[i][reg] + acc1[i][reg];
          const int j = r0 + 32 * blk + l32;
          const float bias = (v0 == 0 && j < R) ? st.beta * (float)(st.r_t[j] - st.r_Lx[j]) : 0.0f;
          float m, s;
          TopK<KB> tk;
          block_lists<KB>(z, v0, wv, h, V, bias, m, s, tk);
          if (lane < 32) {
            float *p = sm.xr[buf][g][wv][l32];
            p[0] = m;
            p[1] = s;
            topk_store(p + 2, tk);
          }
        }
        __syncthreads();
        if (blk < nbt && wv == i && lane < 32) {
          const int j = r0 + 32 * blk + l32;
          if (j < R) {
            const float *sl[4] = {sm.xr[buf][g][0][l32], sm.xr[buf][g][1][l32], sm.xr[buf][g][2][l32],
                                  sm.xr[buf][g][3][l32]};
            write_record<KB>(st, j, vt, sl);
          }
        }
      }
    }
  }
}

// Wide tile (bf16, 4-key lists): 256 vocabulary rows x 128 batch rows. Wave
// w sums K half w/4 over vocabulary rows 64*(w%4) .. +63 (two 32-row slices)
// of the 256 and all four blocks, so each state fragment read from LDS
// feeds two MFMAs (the LDS reads per MFMA halve next to a 32-row wave). The
// K halves and each half's MFMA sequence are those of the other tiles, so
// the sums are the same. vw: 256-row vocabulary tile; its second 128-row
// half may lie past the vocabulary (odd tile count): those waves compute a
// copy of the last tile and write nothing.
template <int KB, bool KV>
__device__ __forceinline__ void proj_tile_wide(const DevState &st, const GemmOperands &op, ProjSmem<KB> &sm, int vw,
                                               int r0, int R, int nvt) {
  const int d = st.d, V = st.V;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = w >> 2, vq = w & 3;               // K half, vocabulary quarter
  const int l32 = lane & 31, h = lane >> 5;
  const int rowbytes = d * 2;
  const int nk = rowbytes / CH, nh = nk >> 1, kbeg = g * nh;
  const int t2 = vq >> 1;                          // which 128-row half of the 256
  const int vt = min(2 * vw + t2, nvt - 1);        // 128-row tile of this wave's rows
  const int s0 = 2 * (vq & 1);                     // its first slice in that tile
  const int v0 = vt * TV;
  const unsigned char *abase = op.w + ((size_t)(vt * nk + kbeg) * 4 + s0) * WCH;
  const int tg = tid & 255;
  const int srow = tg >> 3, scol = (tg & 7) * 16;
  uint32_t boff[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) boff[u] = (uint32_t)min(r0 + srow + 32 * u, R - 1) * (uint32_t)rowbytes + scol;
  const unsigned char *bbase = static_cast<const unsigned char *>(op.in) + (size_t)kbeg * CH;
  f16v acc[2 * NB];
#pragma unroll
  for (int b = 0; b < 2 * NB; ++b) acc[b] = f16v{};
  proj_mainloop<true, NB, 2, 2>(sm.B[0][g], sm.B[1][g], abase, (uint32_t)lane * 16u, bbase, boff, srow, scol, nh,
                                l32, h, acc);

  // Combine the halves, one slice at a time: half g owns blocks 2g, 2g+1,
  // sends its sums of the other two and adds the received ones once.
  f16v own[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x) {
#pragma unroll
    for (int bl = 0; bl < 2; ++bl) {
      const f16v snd = acc[x * NB + (g ? bl : 2 + bl)];
      own[x][bl] = acc[x * NB + (g ? 2 + bl : bl)];
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) sm.red[g][vq][bl][reg][lane] = snd[reg];
    }
    __syncthreads();
#pragma unroll
    for (int bl = 0; bl < 2; ++bl)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) own[x][bl][reg] += sm.red[1 - g][vq][bl][reg][lane];
    __syncthreads();
  }

  if constexpr (KV) {
    if (2 * vw + t2 < nvt) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int bl = 0; bl < 2; ++bl)
          kv_store_block(st, own[x][bl], v0 + 32 * (s0 + x), h, r0 + 32 * (2 * g + bl) + l32, R);
    }
    return;
  }

  // Lane lists of the four owned (slice, block) tiles, then wave w merges
  // the four slices of 128-row tile w/4, block w%4.
#pragma unroll
  for (int x = 0; x < 2; ++x) {
#pragma unroll
    for (int bl = 0; bl < 2; ++bl) {
      const int blk = 2 * g + bl;
      const int j = r0 + 32 * blk + l32;
      const float bias = (v0 == 0 && j < R) ? st.beta * (float)(st.r_t[j] - st.r_Lx[j]) : 0.0f;
      float m, s;
      TopK<KB> tk;
      block_lists<KB>(own[x][bl], v0, s0 + x, h, V, bias, m, s, tk);
      if (lane < 32) {
        float *p = sm.xw[t2][s0 + x][32 * blk + l32];
        p[0] = m;
        p[1] = s;
        topk_store(p + 2, tk);
      }
    }
  }
  __syncthreads();
  {
    const int mt = w >> 2, row = 32 * (w & 3) + l32;
    const int j = r0 + row;
    if (lane < 32 && j < R && 2 * vw + mt < st.S) {
      const float *sl[4] = {sm.xw[mt][0][row], sm.xw[mt][1][row], sm.xw[mt][2][row], sm.xw[mt][3][row]};
      write_record<KB>(st, j, 2 * vw + mt, sl);
    }
  }
}

// Row tile rt covers blocks bt*rt .. bt*rt + bt - 1 (32 rows each) of
// vocabulary tile vt.
template <bool BF16, int KB, bool KV>
__device__ __forceinline__ void proj_tile(const DevState &st, const GemmOperands &op, ProjSmem<KB> &sm, int vt, int rt,
                                          int R, int bt) {
  const int r0 = rt * bt * 32;
  const int nbt = min(bt, (R - r0 + 31) >> 5);   // blocks holding valid rows
  if (nbt <= NB)
    proj_tile_ksplit<BF16, KB, KV>(st, op, sm, vt, r0, R, nbt);
  else
    proj_tile_big<BF16, KB, KV>(st, op, sm, vt, r0, R, nbt);
}

// Blocks per row tile for a step of R rows: the count (1..8) that minimizes
// rounds x tile cost, where a round is one tile per workgroup and a tile
// costs its MFMA blocks plus a fixed part worth 0.7 block (prologue,
// epilogue). Ties go to the larger tile.
__device__ __forceinline__ int row_tile_blocks(int R, int S, int G) {
  const int B = (R + 31) >> 5;
  int best_bt = NB;
  float best = 3.0e38f;
  for (int bt = 1; bt <= 2 * NB; ++bt) {
    const int nra = (B + bt - 1) / bt;
    const int be = min(bt, B);
    const int rounds = (S * nra + G - 1) / G;
    const float cost = (float)rounds * ((float)be + 0.7f);
    if (cost <= best) {
      best = cost;
      best_bt = bt;
    }
  }
  return best_bt;
}

// Persistent launch: at most one workgroup per compute unit, each walking
// its share of the active tiles (vocabulary tile major, batch tile minor).
// Workgroup ids are dealt round robin to the 8 XCDs; XCD x takes the x-th
// eighth of the tile list, so the batch tiles of one vocabulary tile run
// side by side on one XCD and share its L2 copy of the W_out tile. Rounds
// alternate direction over the XCD's workgroups, so that a workgroup which
// drew a full batch tile in one round draws a partial one in the next. Only
// tiles holding rows of this step are visited, and no workgroup is launched
// just to exit (idle ones would occupy compute units that the dispatcher
// then withholds from working ones).
template <bool BF16, int KB, bool KV>
__device__ __forceinline__ void tile_walk(const DevState &st, const GemmOperands &op, int nvt) {
  const int R = st.ctrl->R;
  if (R <= 0) return;
  // bf16 steps whose 256-wide tiles fill at least one round use them.
  const int S2 = (nvt + 1) >> 1, nrw = (R + TR - 1) / TR;
  const bool wide = BF16 && KB == 4 && S2 * nrw >= (int)gridDim.x;
  const int bt = wide ? NB : row_tile_blocks(R, nvt, (int)gridDim.x);
  const int nra = wide ? nrw : (R + 32 * bt - 1) / (32 * bt);
  const int T = (wide ? S2 : nvt) * nra;
  const int x = blockIdx.x & 7, gx = gridDim.x >> 3, j = blockIdx.x >> 3;
  const int lo = (int)((long long)T * x / 8), nt = (int)((long long)T * (x + 1) / 8) - lo;
  __shared__ ProjSmem<KB> sm;
  for (int r = 0; r * gx < nt; ++r) {
    const int idx = (r & 1) ? (r + 1) * gx - 1 - j : r * gx + j;
    if (idx >= nt) continue;
    const int tile = lo + idx;
    const int vt = tile / nra, rt = tile - vt * nra;
    if constexpr (BF16 && KB == 4) {
      if (wide) {
        proj_tile_wide<KB, KV>(st, op, sm, vt, rt * TR, R, nvt);
        __syncthreads();   // LDS is reused by the next tile
        continue;
      }
    }
    proj_tile<BF16, KB, KV>(st, op, sm, vt, rt, R, bt);
    __syncthreads();   // LDS is reused by the next tile
  }
}

template <bool BF16, int KB>
__global__ __launch_bounds__(THREADS, 1) void k_proj(DevState st) {
  tile_walk<BF16, KB, false>(st, GemmOperands{st.wout_t, st.proj_in}, st.S);
}

// KV rows of every expansion of the step: bf16(h . W_kv[l][j]) for the
// L*2*d outputs, the [R,d] x [d, L*2*d] product on the projection's tiles
// and K order (K halves summed apart and added once, so a row's KV values do
// not depend on the rows sharing the step), stored at the candidate's
// (beam, level, rank) place (App. A.2's incremental decoder state).
__global__ __launch_bounds__(THREADS, 1) void k_kv_append(DevState st) {
  tile_walk<true, 4, true>(st, GemmOperands{st.wkv_t, st.hbuf}, st.kv_layers * 2 * st.d / TV);
}

// W_out [V][d] -> MFMA fragment order [S][nk][4 slices][4 pieces][64 lanes][16 B]:
// lane (h, l) of slice s at piece q holds bytes kt*128 + 64h + 16q .. +15 of
// vocabulary row 128*vt + 32s + l (zero past V).
__global__ void k_relayout_wout(const unsigned char *__restrict__ src, unsigned char *__restrict__ dst, int V,
                                int rowbytes, int S) {
  const int nk = rowbytes / CH;
  const size_t pieces = (size_t)S * nk * 4 * 4 * 64;
  for (size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x; p < pieces; p += (size_t)gridDim.x * blockDim.x) {
    const int ln = (int)(p & 63);
    const int q = (int)((p >> 6) & 3);
    const int s = (int)((p >> 8) & 3);
    const size_t vk = p >> 10;                  // vt * nk + kt
    const int kt = (int)(vk % nk);
    const int vt = (int)(vk / nk);
    const int v = vt * TV + 32 * s + (ln & 31);
    u4 val = {0u, 0u, 0u, 0u};
    if (v < V)
      val = *reinterpret_cast<const u4 *>(src + (size_t)v * rowbytes + (size_t)kt * CH + 64 * (ln >> 5) + 16 * q);
    *reinterpret_cast<u4 *>(dst + p * 16) = val;
  }
}

// W_kv [L][2][d_in][d_out] -> the same fragment order, output feature
// v = plane * d + o (plane = 2l + j) in place of the vocabulary row: lane
// (h, l) of slice s at piece q holds the 8 bf16 values W_kv[plane][k0 + e][o],
// k0 = kt*64 + 32h + 8q, e < 8, of output v = 128*vt + 32s + l.
__global__ void k_relayout_wkv(const uint16_t *__restrict__ W, unsigned char *__restrict__ dst, int d, int NO) {
  const int nk = d * 2 / CH;
  const size_t pieces = (size_t)(NO / TV) * nk * 4 * 4 * 64;
  for (size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x; p < pieces; p += (size_t)gridDim.x * blockDim.x) {
    const int ln = (int)(p & 63);
    const int q = (int)((p >> 6) & 3);
    const int s = (int)((p >> 8) & 3);
    const size_t vk = p >> 10;
    const int kt = (int)(vk % nk);
    const int vt = (int)(vk / nk);
    const int v = vt * TV + 32 * s + (ln & 31);
    const int plane = v / d, o = v - plane * d;
    const int k0 = kt * (CH / 2) + 32 * (ln >> 5) + 8 * q;
    const uint16_t *src = W + ((size_t)plane * d + k0) * d + o;
    uint16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = src[(size_t)i * d];
    u4 val = {(uint32_t)e[0] | ((uint32_t)e[1] << 16), (uint32_t)e[2] | ((uint32_t)e[3] << 16),
              (uint32_t)e[4] | ((uint32_t)e[5] << 16), (uint32_t)e[6] | ((uint32_t)e[7] << 16)};
    *reinterpret_cast<u4 *>(dst + p * 16) = val;
  }
}

template <bool BF16>
hipError_t launch_proj_t(const DevState &st, hipStream_t s) {
  // Multiple of 8, at most one per compute unit, no more than the 32-row
  // tiles of a full step (a small vocabulary then still spreads a large step
  // over the device).
  const int G = std::max(8, std::min(st.n_cu / 8 * 8, xcd_grid(st.S * ((st.R_max + 31) / 32))));
  switch (st.tile_keys) {
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

hipError_t launch_kv_append(const DevState &st, hipStream_t s) {
  // Sized like the projection's grid, over the L*2*d/128 output tiles.
  const int nvt = st.kv_layers * 2 * st.d / TV;
  const int G = std::max(8, std::min(st.n_cu / 8 * 8, xcd_grid(nvt * ((st.R_max + 31) / 32))));
  hipLaunchKernelGGL(k_kv_append, dim3(G), dim3(THREADS), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_relayout_wkv(const DevState &st, const uint16_t *W_kv, hipStream_t s) {
  hipLaunchKernelGGL(k_relayout_wkv, dim3(2048), dim3(256), 0, s, W_kv, st.wkv_t, st.d, st.kv_layers * 2 * st.d);
  return hipGetLastError();
}

}  // namespace sb
