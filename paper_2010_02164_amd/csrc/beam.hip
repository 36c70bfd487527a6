// Row merge, per-beam top-k with pruning and finalization, and the
// backtrack of finished hypotheses.
//
//   K_beam     : per selected beam, merge the projection's per-tile partials
//                of each active parent's row into its log-sum-exp and best k
//                tokens, with log-probabilities lp = z - lse (Sec. 2
//                log-likelihoods); rank the k|V| expansions (only each
//                parent's best k can reach the top k) plus one no-op per
//                terminated candidate, keep the top k (Sec. 2), apply the
//                heuristics H (Sec. 4: relative threshold delta against the
//                best candidate, possibly terminated (App. A.3); at most M
//                kept expansions per parent), mark EOS / max-length
//                terminations, and finish the beam when nothing active
//                survives (App. A.1: terminated candidates stay on the beam
//                and are output once nothing active ranks above them).
//                Continuing beams get their new candidates' states.
//   K_backtrack: rebuild each finished hypothesis's tokens from the
//                backpointer history, one thread per hypothesis.
#include "mfma_common.h"
#include "sb_internal.h"
#include "topk.h"
#include "wave.h"

namespace sb {
namespace {

// Wave-wide maximum of a 64-bit key, in every lane.
template <int S>
__device__ __forceinline__ cand_key max_stage(cand_key x) {
  cand_key a, b;
  stage64<S>(x, a, b);
  return a > b ? a : b;
}
__device__ __forceinline__ cand_key wave_max_key(cand_key x) {
  x = max_stage<0>(x);
  x = max_stage<1>(x);
  x = max_stage<2>(x);
  x = max_stage<3>(x);
  x = max_stage<4>(x);
  return max_stage<5>(x);
}

// Wave-wide log-sum-exp combine of (max, sum exp) pairs; every lane ends
// with the same result. The merge is not symmetric in its operands once
// the compiler fuses a product into the sum, so both lanes of a pair take
// them in the same order: the lower lane's first (the swap stages 4 and 5
// already hand both lanes the pair in that order).
template <int S>
__device__ __forceinline__ void lse_stage(float &m, float &s) {
  uint32_t ma, mb, sa, sb;
  stage32<S>(__float_as_uint(m), ma, mb);
  stage32<S>(__float_as_uint(s), sa, sb);
  if constexpr (S <= 3) {
    const int lane = (int)(threadIdx.x & 63);
    const bool lower = S == 0 ? !(lane & 1) : S == 1 ? !(lane & 2) : S == 2 ? (lane & 7) < 4 : (lane & 15) < 8;
    if (!lower) {
      const uint32_t tm = ma, ts = sa;
      ma = mb;
      sa = sb;
      mb = tm;
      sb = ts;
    }
  }
  float M = __uint_as_float(ma), Sm = __uint_as_float(sa);
  lse_merge(M, Sm, __uint_as_float(mb), __uint_as_float(sb));
  m = M;
  s = Sm;
}
__device__ __forceinline__ void wave_lse(float &m, float &s) {
  lse_stage<0>(m, s);
  lse_stage<1>(m, s);
  lse_stage<2>(m, s);
  lse_stage<3>(m, s);
  lse_stage<4>(m, s);
  lse_stage<5>(m, s);
}

// Logit z[v] of one fp32 row recomputed from W_out and the row's
// projection input, with the EOS bias of token 0. It follows the
// projection's arithmetic exactly: each K half in chunks of 32 values, and
// per chunk, piece q and element e the two fused products of k and k + 16
// (an fp32 32x32x2 MFMA adds its two products to the sum one after the
// other, lane half 0's first), then the halves added once, so a recomputed
// logit equals the projection's bit for bit.
__device__ __forceinline__ float recompute_logit_f32(const DevState &st, int row, int v) {
  const int d = st.d;
  const float *w = static_cast<const float *>(st.W_out) + (size_t)v * d;
  const float *x = static_cast<const float *>(st.proj_in) + (size_t)row * d;
  float half[2];
  for (int g = 0; g < 2; ++g) {
    float acc = 0.0f;
    for (int c = g * (d / 2); c < (g + 1) * (d / 2); c += 32)
      for (int q = 0; q < 4; ++q)
        for (int e = 0; e < 4; ++e) {
          const int k0 = c + 4 * q + e;
          acc = fmaf(w[k0], x[k0], acc);
          acc = fmaf(w[k0 + 16], x[k0 + 16], acc);
        }
    half[g] = acc;
  }
  float z = half[0] + half[1];
  if (v == 0) z += st.beta * (float)(st.r_t[row] - st.r_Lx[row]);
  return z;
}

// bf16: the 128 logits of vocabulary tile vt for one row, recomputed by the
// projection's own MFMA sequence so that they equal its logits bit for bit
// (the bf16 MFMA's internal rounding is not modelled, it is replayed): per
// 32-row slice, each K half accumulated chunk by chunk and piece by piece
// from the same W_out fragments and state bytes, then the halves added
// once. Every column of the MFMA gets the row's state, so all 32 columns
// hold the same logits; lane (h, l) with l < 16 inserts the logit of
// register l, vocabulary row 32s + 8(l/4) + 4h + l%4 of the tile, into its
// list (each of the 128 logits once).
template <int KB>
__device__ __forceinline__ void recompute_tile_bf16(const DevState &st, int row, int vt, int lane, TopK<KB> &tk) {
  constexpr int CH = 128, FRAG = 1024;
  const int nk = st.d * 2 / CH, nh = nk >> 1;
  const int h = lane >> 5, l32 = lane & 31;
  const unsigned char *x = static_cast<const unsigned char *>(st.proj_in) + (size_t)row * st.d * 2 + 64 * h;
  const float bias = st.beta * (float)(st.r_t[row] - st.r_Lx[row]);
#pragma unroll 1
  for (int s = 0; s < 4; ++s) {
    f16v half[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      f16v acc = {};
#pragma unroll 1
      for (int c = g * nh; c < (g + 1) * nh; ++c) {
        const unsigned char *a = st.wout_t + ((size_t)(vt * nk + c) * 4 + s) * 4 * FRAG + lane * 16;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const u4 av = *reinterpret_cast<const u4 *>(a + q * FRAG);
          const u4 bv = *reinterpret_cast<const u4 *>(x + c * CH + 16 * q);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf8, av), __builtin_bit_cast(bf8, bv), acc,
                                                        0, 0, 0);
        }
      }
      half[g] = acc;
    }
    if (l32 < 16) {
      float z = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (r == l32) z = half[0][r] + half[1][r];
      const int v = vt * 128 + 32 * s + 8 * (l32 >> 2) + 4 * h + (l32 & 3);
      if (v == 0) z += bias;
      if (v < st.V) topk_insert(tk, make_key(z, v));
    }
  }
}

// Merge the per-tile partials of one row (one wave). Each lane folds the
// tiles lane, lane+64, ... into (max, sum exp) and a sorted best-KB list
// (loads issued a batch at a time before they are folded). The row's
// log-sum-exp is combined over the lanes and taken from lane 0; the row's k
// best keys are drawn in k rounds of a wave maximum over the lists' heads,
// the lane holding the winner dropping it (keys are distinct: they carry
// the token). Lane r < k receives the key of rank r.
//
// A tile record keeps its TK best keys (TK <= KB). If a tile's last kept
// key ranks above the k-th key drawn, the tile may hold further keys of the
// best k: such tiles (rare: TK of the row's best k - 1 in one
// 128-token tile) are recomputed from W_out, all their logits enter the
// lists in place of the record's keys, and the k keys are drawn again. Any
// other tile's unkept keys rank below its last kept key, so at most at the
// k-th key drawn, and adding candidates can only raise the k-th key.
template <int KB, int TK>
__device__ __forceinline__ double merge_row(const DevState &st, int row, int lane, int k, cand_key &mine) {
  constexpr int PW = part_width(TK);
  // Partials in flight per lane (full-length lists come with fewer than 64
  // tiles, one per lane).
  constexpr int NBT = TK == TILE_KEYS_SHORT ? 4 : 1;
  const float *base = st.part + (size_t)row * st.S * PW;
  float m = -INFINITY, s = 0.0f;
  TopK<KB> tk;
  topk_init(tk);
  cand_key last_max = 0ull;   // largest last kept key over the lane's tiles
#pragma unroll 1
  for (int t0 = lane; t0 < st.S; t0 += 64 * NBT) {
    float rec[NBT][PW];
#pragma unroll
    for (int u = 0; u < NBT; ++u) {
      const int t = min(t0 + 64 * u, st.S - 1);
      const uint4 *p = reinterpret_cast<const uint4 *>(base + (size_t)t * PW);
#pragma unroll
      for (int x = 0; x < PW / 4; ++x) {
        const uint4 v = p[x];
        rec[u][4 * x] = __uint_as_float(v.x);
        rec[u][4 * x + 1] = __uint_as_float(v.y);
        rec[u][4 * x + 2] = __uint_as_float(v.z);
        rec[u][4 * x + 3] = __uint_as_float(v.w);
      }
    }
    if constexpr (TK == TILE_KEYS_SHORT && NBT == 4) {
      // Four sorted 4-key runs (empty past the last tile) merged by
      // bitonic networks into the batch's best KB, then into the list.
      TopK<4> run[4];
#pragma unroll
      for (int u = 0; u < NBT; ++u) {
        const bool ok = t0 + 64 * u < st.S;
        topk_load(run[u], rec[u] + 2);
#pragma unroll
        for (int j = 0; j < 4; ++j) run[u].k[j] = ok ? run[u].k[j] : 0ull;
        if (ok) lse_merge(m, s, rec[u][0], rec[u][1]);
        last_max = run[u].k[3] > last_max ? run[u].k[3] : last_max;
      }
      TopK<KB> batch;
      if constexpr (KB == 4) {
        topk_merge(run[0], run[1]);
        topk_merge(run[2], run[3]);
        topk_merge(run[0], run[2]);
        batch = run[0];
      } else {
        cand_key a8[8], b8[8];
        merge_sorted<4>(run[0].k, run[1].k, a8);
        merge_sorted<4>(run[2].k, run[3].k, b8);
        if constexpr (KB == 8) {
          TopK<8> x, y;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            x.k[j] = a8[j];
            y.k[j] = b8[j];
          }
          topk_merge(x, y);
          batch = x;
        } else {
          merge_sorted<8>(a8, b8, batch.k);
        }
      }
      if (t0 == lane) tk = batch;
      else topk_merge(tk, batch);
    } else {
#pragma unroll
      for (int u = 0; u < NBT; ++u) {
        if (t0 + 64 * u < st.S) {
          TopK<TK> t4;
          topk_load(t4, rec[u] + 2);
          TopK<KB> o;
          topk_init(o);
#pragma unroll
          for (int j = 0; j < TK; ++j) o.k[j] = t4.k[j];
          lse_merge(m, s, rec[u][0], rec[u][1]);
          last_max = t4.k[TK - 1] > last_max ? t4.k[TK - 1] : last_max;
          topk_merge(tk, o);
        }
      }
    }
  }
  wave_lse(m, s);
  cand_key kth = 0ull;
  mine = 0ull;
#pragma unroll 1
  for (int r = 0; r < k; ++r) {
    const cand_key best = wave_max_key(tk.k[0]);
    if (lane == r) mine = best;
    kth = best;
    if (tk.k[0] == best) {
#pragma unroll
      for (int j = 0; j + 1 < KB; ++j) tk.k[j] = tk.k[j + 1];
      tk.k[KB - 1] = 0ull;
    }
  }
  // The row's log-sum-exp as lane 0 has it, for every lane.
  const double lse = __shfl((double)m + log((double)s), 0, 64);
  if (__ballot(last_max > kth) == 0ull) return lse;

  // Rare path: rebuild the lists with the saturated tiles recomputed.
  topk_init(tk);
  for (int t0 = 0; t0 < st.S; t0 += 64) {
    const int t = t0 + lane;
    bool sat = false;
    if (t < st.S) {
      const float *p = base + (size_t)t * PW;
      TopK<TK> o;
      topk_load(o, p + 2);
      sat = o.k[TK - 1] > kth;
      if (!sat) {
        TopK<KB> oo;
        topk_init(oo);
#pragma unroll
        for (int j = 0; j < TK; ++j) oo.k[j] = o.k[j];
        topk_merge(tk, oo);
      }
    }
    unsigned long long mask = __ballot(sat);
    if (lane == 0 && mask)
      atomicAdd(reinterpret_cast<unsigned long long *>(&st.ctrl->tile_recomputes),
                (unsigned long long)__popcll(mask));
    while (mask) {
      const int src = __ffsll((long long)mask) - 1;
      mask &= mask - 1;
      const int vt = t0 + src;
      if (st.dtype == 1) {
        recompute_tile_bf16<KB>(st, row, vt, lane, tk);
      } else {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int v = vt * 128 + 64 * half + lane;
          if (v < st.V) topk_insert(tk, make_key(recompute_logit_f32(st, row, v), v));
        }
      }
    }
  }
  mine = 0ull;
#pragma unroll 1
  for (int r = 0; r < k; ++r) {
    const cand_key best = wave_max_key(tk.k[0]);
    if (lane == r) mine = best;
    if (tk.k[0] == best) {
#pragma unroll
      for (int j = 0; j + 1 < KB; ++j) tk.k[j] = tk.k[j + 1];
      tk.k[KB - 1] = 0ull;
    }
  }
  return lse;
}

// Row merge as its own kernel (wave per row), for the single-expansion
// debug entry point: writes lse and the k best log-probabilities/tokens.
template <int KB, int TK>
__global__ __launch_bounds__(256) void k_rowmerge(DevState st) {
  const int R = st.ctrl->R;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= R) return;
  cand_key mine;
  const int k = st.k;
  const double lse = merge_row<KB, TK>(st, row, lane, k, mine);
  if (lane == 0) st.r_lse[row] = lse;
  if (lane < k) {
    st.top_lp[(size_t)row * k + lane] = (double)key_val(mine) - lse;
    st.top_tok[(size_t)row * k + lane] = key_idx(mine);
  }
}

// Ranking of an expansion: higher score first, then the smaller secondary
// key (parent rank << 24 | token + 1; a no-op has token -1).
__device__ __forceinline__ bool ranks_above(double sa, int ka, double sb, int kb) {
  return sa > sb || (sa == sb && ka < kb);
}

// Threads of a beam workgroup: 8 waves (a wave per parent row), or 4 waves
// when the vocabulary has at most 8 tiles and a row's merge is short (four
// workgroups then share a compute unit). Both hold a thread per candidate
// of the ranking up to k = 15.
constexpr int BEAM_THREADS = 512;
constexpr int BEAM_THREADS_SMALL = 256;
constexpr int NO_KEY = 0x7FFFFFFF;

// A candidate expansion of the per-beam ranking (16 bytes, one LDS read).
struct Cand {
  double score;
  int key, pad;
};

template <int KB, int TK, int NT>
__global__ __launch_bounds__(NT) void k_beam(DevState st) {
  constexpr int BEAM_WAVES = NT / 64;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int k = st.k;
  const int base = b * k;
  const bool fairseq = st.rule == 1;
  const int KC = k + (fairseq ? 1 : 0);   // children drawn per parent
  // Everything the beam needs from its records is loaded in one round,
  // before the selection flag is tested.
  int my_status = SLOT_EMPTY, my_row = -1;
  double my_score = 0.0;
  if (tid < k) {
    my_status = st.s_status[base + tid];
    my_row = st.s_row[base + tid];
    my_score = st.s_score[base + tid];
  }
  int my_q = 0, my_t = 0, my_ml = 0, my_nout = 0;
  if (tid == 64) {
    my_q = st.b_input[b];
    my_t = st.b_steps[b] + 1;     // 1-based index of the emitted token
    my_ml = st.b_ml[b];
    my_nout = st.b_nout[b];
  }
  // The KV ancestry buffer holding this beam's current ranks (read before
  // thread 0 flips the parity at the end of the step).
  const int apar = st.kv_layers > 0 ? st.b_par[b] : 0;
  // b_sel is cleared for every beam when nothing is live (R == 0).
  if (!st.b_sel[b]) return;
  __shared__ int sl_status[KMAX_SUPPORTED], sl_row[KMAX_SUPPORTED];
  __shared__ double sl_score[KMAX_SUPPORTED];
  __shared__ int q_in_sh, t_sh, max_len_sh, nout_sh;
  // Best KC log-probabilities and tokens of each active parent's row.
  __shared__ double ch_lp[KMAX_SUPPORTED * KMAX_SUPPORTED];
  __shared__ int ch_tok[KMAX_SUPPORTED * KMAX_SUPPORTED];
  // The new beam, in rank order, and (Fairseq rule) this step's outputs.
  __shared__ double nscore[KMAX_SUPPORTED], oscore[KMAX_SUPPORTED];
  __shared__ int npar[KMAX_SUPPORTED], ntok[KMAX_SUPPORTED], nstat[KMAX_SUPPORTED];
  __shared__ int opar[KMAX_SUPPORTED], otok[KMAX_SUPPORTED], ostat[KMAX_SUPPORTED];
  __shared__ int nw_sh, nact_sh, no_sh;
  // Candidates (at most k KC list entries + k no-ops) and the ranks kept.
  __shared__ Cand cand[KMAX_SUPPORTED * (KMAX_SUPPORTED + 1)];
  __shared__ double r_score[2 * KMAX_SUPPORTED];
  __shared__ int r_key[2 * KMAX_SUPPORTED];
  if (tid < k) {
    sl_status[tid] = my_status;
    sl_row[tid] = my_row;
    sl_score[tid] = my_score;
  }
  if (tid == 64) {
    q_in_sh = my_q;
    t_sh = my_t;
    max_len_sh = my_ml;
    nout_sh = my_nout;
  }
  __syncthreads();
  const int q_in = q_in_sh, t = t_sh, max_len = max_len_sh, nout0 = nout_sh;

  // Row merge of every active parent: wave w takes parents w, w+8.
  for (int par = wave; par < k; par += BEAM_WAVES) {
    if (sl_status[par] != SLOT_ACTIVE) continue;
    cand_key mine;
    const double lse = merge_row<KB, TK>(st, sl_row[par], lane, KC, mine);
    if (lane < KC) {
      ch_lp[par * KC + lane] = (double)key_val(mine) - lse;
      ch_tok[par * KC + lane] = key_idx(mine);
    }
  }
  __syncthreads();

  // Ranking of all expansions (key: score, parent rank, token; Sec. 2):
  // thread c < C holds candidate c (parent c / KC's child c % KC, or, paper
  // rule, the no-op of terminated parent c - k KC) and counts the valid
  // candidates that rank above it; that count is its rank, all keys being
  // distinct. Ranks below RM (k, or 2k under the Fairseq rule) are kept.
  const int NCL = k * KC;
  const int C = NCL + (fairseq ? 0 : k);
  const int RM = fairseq ? 2 * k : k;
  double cs = -INFINITY;
  int ck = NO_KEY;
  bool cv = false;
  if (tid < NCL) {
    const int p = tid / KC, j = tid - p * KC;
    if (sl_status[p] == SLOT_ACTIVE) {
      const int tok = ch_tok[p * KC + j];
      if (tok >= 0 && tok < st.V) {
        cs = sl_score[p] + ch_lp[p * KC + j];
        ck = (p << 24) | (tok + 1);
        cv = true;
      }
    }
  } else if (tid < C) {
    const int p = tid - NCL;
    if (sl_status[p] == SLOT_EOS || sl_status[p] == SLOT_MAXLEN) {
      cs = sl_score[p];
      ck = p << 24;
      cv = true;
    }
  }
  // Records up to a multiple of 8; invalid ones (score -inf) rank below
  // every valid candidate.
  const int C8 = (C + 7) & ~7;
  if (tid < C8) cand[tid] = Cand{cs, ck, 0};
  const int nvalid = __syncthreads_count(cv);
  if (cv) {
    int rank = 0;
    for (int c0 = 0; c0 < C8; c0 += 8) {
      Cand o[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) o[u] = cand[c0 + u];
#pragma unroll
      for (int u = 0; u < 8; ++u) rank += ranks_above(o[u].score, o[u].key, cs, ck) ? 1 : 0;
    }
    if (rank < RM) {
      r_score[rank] = cs;
      r_key[rank] = ck;
    }
  }
  __syncthreads();

  if (wave == 0) {
    // Lane r < nfull holds the expansion of rank r.
    const int nfull = min(RM, nvalid);
    double rs = -INFINITY;
    int rk = NO_KEY;
    if (lane < nfull) {
      rs = r_score[lane];
      rk = r_key[lane];
    }
    if (!fairseq) {
      // Heuristics H (Sec. 4) on B' in rank order: drop x if
      // score(x) < best - delta, best = B'[0] (possibly terminated,
      // App. A.3); drop an expansion whose parent already has M kept
      // expansions (no-ops exempt). A parent's kept expansions before rank r
      // are its first M delta-survivors, so the M test needs only their count.
      const double ref = __longlong_as_double(((long long)__builtin_amdgcn_readlane((int)(__double_as_longlong(rs) >> 32), 0) << 32) |
                                              (uint32_t)__builtin_amdgcn_readlane((int)__double_as_longlong(rs), 0));
      const int rpar = rk >> 24, rtok = (rk & 0xFFFFFF) - 1;
      const bool keepd = lane < nfull && !(rs < ref - st.delta);
      int before = 0;
#pragma unroll 1
      for (int o = 0; o < nfull; ++o) {
        const int okk = __builtin_amdgcn_readlane(rk, o);
        const int okeep = __builtin_amdgcn_readlane((int)keepd, o);
        before += (o < lane && okeep && (okk >> 24) == rpar && (okk & 0xFFFFFF) != 0);
      }
      const bool kept = keepd && (rtok < 0 || before < st.M);
      int status = SLOT_EMPTY;
      if (kept) {
        if (rtok < 0) status = sl_status[rpar];                   // no-op keeps EOS / MAXLEN
        else status = rtok == 0 ? SLOT_EOS : (t == max_len ? SLOT_MAXLEN : SLOT_ACTIVE);
      }
      const unsigned long long km = __ballot(kept);
      const unsigned long long am = __ballot(kept && status == SLOT_ACTIVE);
      if (kept) {
        const int nr = __popcll(km & ((1ull << lane) - 1ull));
        nscore[nr] = rs;
        npar[nr] = rpar;
        ntok[nr] = rtok;
        nstat[nr] = status;
      }
      if (lane == 0) {
        nw_sh = __popcll(km);
        nact_sh = __popcll(am);
        no_sh = 0;
      }
    } else {
      // Fairseq rule (App. A.1): a terminated expansion among the best k is
      // output at once (until k outputs); the new beam is the first k
      // active expansions in rank order. Both lie within the first 2k ranks.
      const int rpar = rk >> 24, rtok = (rk & 0xFFFFFF) - 1;
      const bool valid = lane < nfull;
      const bool term = valid && (rtok == 0 || t == max_len);
      const unsigned long long below = (1ull << lane) - 1ull;
      const unsigned long long tm = __ballot(term && lane < k);
      const int f = __popcll(tm & below);
      const bool out = term && lane < k && nout0 + f < k;
      const unsigned long long act = __ballot(valid && !term);
      const int nr = __popcll(act & below);
      const bool inbeam = valid && !term && nr < k;
      if (out) {
        oscore[f] = rs;
        opar[f] = rpar;
        otok[f] = rtok;
        ostat[f] = rtok == 0 ? SLOT_EOS : SLOT_MAXLEN;
      }
      if (inbeam) {
        nscore[nr] = rs;
        npar[nr] = rpar;
        ntok[nr] = rtok;
        nstat[nr] = SLOT_ACTIVE;
      }
      if (lane == 0) {
        const int nw = min(k, __popcll(act));
        const int no = min(__popcll(tm), k - nout0);
        nw_sh = nw;
        no_sh = no;
        // The input finishes with k outputs, or when nothing active is left.
        nact_sh = (nout0 + no >= k) ? 0 : nw;
      }
    }
  }
  __syncthreads();
  const int w = nw_sh, no = no_sh;
  const bool ends = nact_sh == 0;
  const int fin = ends ? (int)st.ctrl->timesteps : 0;

  // History: backpointers of level t, indexed by the input's queue position:
  // the new beam at positions 0..w-1, this step's outputs at k + f.
  uint32_t *bprow = st.bp + ((size_t)q_in * st.max_len_cap + (t - 1)) * st.bpw;
  if (tid < w && !(fairseq && ends)) {
    const uint32_t tokbits = ntok[tid] < 0 ? BP_NOOP : (uint32_t)ntok[tid];
    bprow[tid] = ((uint32_t)npar[tid] << 24) | tokbits;
  }
  if (fairseq && tid >= 64 && tid < 64 + no) {
    const int f = tid - 64;
    bprow[k + f] = ((uint32_t)opar[f] << 24) | (uint32_t)otok[f];
    OutHyp h;
    h.score = oscore[f];
    h.length = 0;
    h.status = ostat[f];
    h.finalize_step = fin;
    h.level = t;
    h.pos = k + f;
    h.pad = 0;
    st.o_hyp[(size_t)q_in * k + nout0 + f] = h;
  }

  if (ends) {
    int total;
    if (!fairseq) {
      // Y[i] = the survivors in rank order; tokens are rebuilt later.
      total = w;
      if (tid < w) {
        OutHyp h;
        h.score = nscore[tid];
        h.length = 0;
        h.status = nstat[tid];
        h.finalize_step = fin;
        h.level = t;
        h.pos = tid;
        h.pad = 0;
        st.o_hyp[(size_t)q_in * k + tid] = h;
      }
    } else {
      // Y[i] = the outputs in the order they were finalized; those of
      // earlier steps get the finishing timestep too.
      total = nout0 + no;
      if (tid >= 128 && tid < 128 + nout0) st.o_hyp[(size_t)q_in * k + (tid - 128)].finalize_step = fin;
    }
    if (tid < k) {
      st.s_status[base + tid] = SLOT_EMPTY;
    }
    if (tid == 0) {
      st.o_count[q_in] = total;
      st.b_input[b] = -1;
      atomicAdd(reinterpret_cast<unsigned long long *>(&st.ctrl->hyps), (unsigned long long)total);
      atomicAdd(reinterpret_cast<unsigned long long *>(&st.ctrl->finished), 1ull);
    }
    return;
  }

  // Continue: write the new beam into ranks 0..w-1 (no-ops keep their
  // state; active children take their parent's new state h).
  if (tid < k) {
    if (tid < w) {
      st.s_status[base + tid] = nstat[tid];
      st.s_score[base + tid] = nscore[tid];
      if (ntok[tid] >= 0) st.s_tok[base + tid] = ntok[tid];
    } else {
      st.s_status[base + tid] = SLOT_EMPTY;
    }
  }
  if (tid == 0) {
    st.b_steps[b] = t;
    st.b_par[b] ^= 1;
    st.b_nout[b] = nout0 + no;
  }
  // State copy: s_h[rank] <- hbuf[row(parent)] for every active survivor,
  // flattened over (survivor, 16-byte chunk) so all threads stream.
  const int rowbytes = st.d * (st.dtype == 1 ? 2 : 4);
  const int chunks = rowbytes / 16;
  const uint4 *__restrict__ hb = static_cast<const uint4 *>(st.hbuf);
  uint4 *__restrict__ sh = static_cast<uint4 *>(st.s_h);
  const int total = w * chunks;
  for (int x = tid; x < total; x += NT) {
    const int r = x / chunks, c = x - r * chunks;
    if (nstat[r] == SLOT_ACTIVE) sh[(size_t)(base + r) * chunks + c] = hb[(size_t)sl_row[npar[r]] * chunks + c];
  }
  // The state's digit planes and list, for the exact bf16 recurrence.
  if (st.rec_i8) {
    const int dch = (int)(rec_dig_row_bytes(st.d) / 16), ach = (int)(sizeof(RowAux) / 16), tch = dch + ach;
    const uint4 *__restrict__ hd = reinterpret_cast<const uint4 *>(st.hd);
    uint4 *__restrict__ shd = reinterpret_cast<uint4 *>(st.s_hd);
    const uint4 *__restrict__ ha = reinterpret_cast<const uint4 *>(st.haux);
    uint4 *__restrict__ sha = reinterpret_cast<uint4 *>(st.s_haux);
    for (int x = tid; x < w * tch; x += NT) {
      const int r = x / tch, c = x - r * tch;
      if (nstat[r] != SLOT_ACTIVE) continue;
      const size_t src = sl_row[npar[r]];
      if (c < dch) shd[(size_t)(base + r) * dch + c] = hd[src * dch + c];
      else sha[(size_t)(base + r) * ach + (c - dch)] = ha[src * ach + (c - dch)];
    }
  }
  // KV state: an active child's ancestors are its parent's (levels 0 .. t-2)
  // and the parent itself (level t-1), copied into the other buffer as
  // 4-byte words; the word holding level t-1 is built by one thread.
  if (st.kv_layers > 0) {
    const int A4 = st.anc_stride / 4;
    const uint32_t *src = reinterpret_cast<const uint32_t *>(st.anc) + ((size_t)apar * st.n * k + base) * A4;
    uint32_t *dst = reinterpret_cast<uint32_t *>(st.anc) + ((size_t)(apar ^ 1) * st.n * k + base) * A4;
    const int nw = (t - 1) / 4 + 1, last = (t - 1) / 4, sh8 = ((t - 1) & 3) * 8;
    for (int x = tid; x < w * nw; x += NT) {
      const int r = x / nw, wi = x - r * nw;
      if (nstat[r] != SLOT_ACTIVE) continue;
      uint32_t v = src[(size_t)npar[r] * A4 + wi];
      if (wi == last) v = (v & ~(0xFFu << sh8)) | ((uint32_t)npar[r] << sh8);
      dst[(size_t)r * A4 + wi] = v;
    }
  }
}

// One thread per (input, rank): walk the backpointers from the final level
// down to 1, skipping no-op levels, and write the tokens in order.
__global__ __launch_bounds__(256) void k_backtrack(DevState st, int q0, int q1) {
  const int k = st.k;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long q = q0 + gid / k;
  const int rank = (int)(gid % k);
  if (q >= q1) return;
  if (rank >= st.o_count[q]) return;
  OutHyp *h = st.o_hyp + (size_t)q * k + rank;
  const int bpw = st.bpw;
  const uint32_t *bp = st.bp + (size_t)q * st.max_len_cap * bpw;
  const int top = min(h->level, st.max_len_cap);
  const int pos0 = min(max(h->pos, 0), bpw - 1);
  int pos = pos0, len = 0;
  for (int lev = top; lev >= 1; --lev) {
    const uint32_t e = bp[(size_t)(lev - 1) * bpw + pos];
    len += (e & 0xFFFFFFu) != BP_NOOP;
    pos = min((int)(e >> 24), k - 1);
  }
  int32_t *out = st.o_tok + ((size_t)q * k + rank) * st.max_len_cap;
  pos = pos0;
  int idx = len;
  for (int lev = top; lev >= 1; --lev) {
    const uint32_t e = bp[(size_t)(lev - 1) * bpw + pos];
    const uint32_t tok = e & 0xFFFFFFu;
    if (tok != BP_NOOP) out[--idx] = (int32_t)tok;
    pos = min((int)(e >> 24), k - 1);
  }
  h->length = len;
}

// Collect: copy the tokens of the hypotheses of inputs [q0, q1) from their
// padded rows to their places in the packed buffer (offsets set by the
// host; -1 marks a rank the input does not have). Four hypotheses per
// workgroup, one wave each, lanes striding over the tokens.
__global__ __launch_bounds__(256) void k_pack(DevState st, int q0, int q1) {
  const long long hyp = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (hyp >= (long long)(q1 - q0) * st.k) return;
  const long long off = st.o_off[hyp];
  if (off < 0) return;
  const size_t slot = (size_t)q0 * st.k + hyp;
  const int len = min(st.o_hyp[slot].length, st.max_len_cap);
  const int32_t *src = st.o_tok + slot * st.max_len_cap;
  for (int j = lane; j < len; j += 64) st.o_pack[off + j] = src[j];
}

}  // namespace

hipError_t launch_rowmerge(const DevState &st, hipStream_t s) {
  const int G = (st.R_max + 3) / 4;
  const bool sh = st.tile_keys == TILE_KEYS_SHORT;
  switch (st.kbucket) {
    case 4: hipLaunchKernelGGL((k_rowmerge<4, 4>), dim3(G), dim3(256), 0, s, st); break;
    case 8:
      if (sh) hipLaunchKernelGGL((k_rowmerge<8, 4>), dim3(G), dim3(256), 0, s, st);
      else hipLaunchKernelGGL((k_rowmerge<8, 8>), dim3(G), dim3(256), 0, s, st);
      break;
    default:
      if (sh) hipLaunchKernelGGL((k_rowmerge<16, 4>), dim3(G), dim3(256), 0, s, st);
      else hipLaunchKernelGGL((k_rowmerge<16, 16>), dim3(G), dim3(256), 0, s, st);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_beam(const DevState &st, hipStream_t s) {
  const bool sh = st.tile_keys == TILE_KEYS_SHORT;
  const bool small = st.S <= 8 && st.k <= 15;   // short row merges: 4-wave workgroups
#define SB_BEAM(KB, TK)                                                                               \
  do {                                                                                                \
    if (small) hipLaunchKernelGGL((k_beam<KB, TK, BEAM_THREADS_SMALL>), dim3(st.n), dim3(BEAM_THREADS_SMALL), 0, s, st); \
    else hipLaunchKernelGGL((k_beam<KB, TK, BEAM_THREADS>), dim3(st.n), dim3(BEAM_THREADS), 0, s, st); \
  } while (0)
  switch (st.kbucket) {
    case 4: SB_BEAM(4, 4); break;
    case 8:
      if (sh) SB_BEAM(8, 4);
      else SB_BEAM(8, 8);
      break;
    default:
      if (sh) SB_BEAM(16, 4);
      else SB_BEAM(16, 16);
      break;
  }
#undef SB_BEAM
  return hipGetLastError();
}

hipError_t launch_pack(const DevState &st, int q0, int q1, hipStream_t s) {
  if (q1 <= q0) return hipSuccess;
  const long long hyps = (long long)(q1 - q0) * st.k;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((hyps + 3) / 4)), dim3(256), 0, s, st, q0, q1);
  return hipGetLastError();
}

hipError_t launch_backtrack(const DevState &st, int q0, int q1, hipStream_t s) {
  if (q1 <= q0) return hipSuccess;
  const long long total = (long long)(q1 - q0) * st.k;
  hipLaunchKernelGGL(k_backtrack, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, st, q0, q1);
  return hipGetLastError();
}

}  // namespace sb
