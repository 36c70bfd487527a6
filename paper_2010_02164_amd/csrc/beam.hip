// Row merge, per-beam top-k with pruning and finalization, and the
// backtrack of finished hypotheses.
//
//   K_rowmerge : per expanded row, merge the projection's per-tile partials
//                into log-sum-exp and the row's best k tokens; their
//                log-probabilities lp = z - lse (Sec. 2 log-likelihoods).
//   K_beam     : per selected beam, rank the k|V| expansions (only each
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
#include "sb_internal.h"
#include "topk.h"

namespace sb {
namespace {

template <int KB>
__global__ __launch_bounds__(256) void k_rowmerge(DevState st) {
  const int R = st.ctrl->R;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= R) return;
  constexpr int PW = 2 + 2 * KB;
  const float *base = st.part + (size_t)row * st.S * PW;
  float m = -INFINITY, s = 0.0f;
  TopK<KB> tk;
  topk_init(tk);
#pragma unroll 1
  for (int t = lane; t < st.S; t += 64) {
    const float *p = base + (size_t)t * PW;
    TopK<KB> o;
    topk_load(o, p + 2);
    lse_merge(m, s, p[0], p[1]);
    topk_merge(tk, o);
  }
#pragma unroll 1
  for (int mask = 1; mask < 64; mask <<= 1) {
    TopK<KB> o;
    topk_shfl_xor(o, tk, mask);
    const float m2 = __shfl_xor(m, mask, 64), s2 = __shfl_xor(s, mask, 64);
    lse_merge(m, s, m2, s2);
    topk_merge(tk, o);
  }
  const double lse = (double)m + log((double)s);
  if (lane == 0) st.r_lse[row] = lse;
  const int k = st.k;
#pragma unroll
  for (int q = 0; q < KB; ++q) {
    if (lane == q && q < k) {
      st.top_lp[(size_t)row * k + q] = (double)key_val(tk.k[q]) - lse;
      st.top_tok[(size_t)row * k + q] = key_idx(tk.k[q]);
    }
  }
}

constexpr int MAXC = KMAX_SUPPORTED * KMAX_SUPPORTED + KMAX_SUPPORTED;

// Ranking key of an expansion: higher score first, then lower parent rank,
// then lower token (a no-op has token -1).
__device__ __forceinline__ bool cand_beats(double sa, int pa, int ta, double sb, int pb, int tb) {
  if (sa != sb) return sa > sb;
  if (pa != pb) return pa < pb;
  return ta < tb;
}

constexpr int BEAM_THREADS = 256;

__global__ __launch_bounds__(BEAM_THREADS) void k_beam(DevState st) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;   // 0..255
  // b_sel is cleared for every beam when nothing is live (R == 0).
  if (!st.b_sel[b]) return;
  const int k = st.k;
  const int base = b * k;
  __shared__ double cs[MAXC];
  __shared__ int cp[MAXC], ct[MAXC], cv[MAXC];
  __shared__ int at_rank[KMAX_SUPPORTED];
  __shared__ double nscore[KMAX_SUPPORTED];
  __shared__ int npar[KMAX_SUPPORTED], ntok[KMAX_SUPPORTED], nstat[KMAX_SUPPORTED];
  __shared__ int kept_per[KMAX_SUPPORTED];
  __shared__ int nw_sh, nact_sh, nvalid_sh;
  // The beam's slots, read once (one parallel round of loads).
  __shared__ int sl_status[KMAX_SUPPORTED], sl_row[KMAX_SUPPORTED];
  __shared__ double sl_score[KMAX_SUPPORTED];
  __shared__ int q_in_sh, t_sh, max_len_sh;

  if (lane < k) {
    sl_status[lane] = st.s_status[base + lane];
    sl_row[lane] = st.s_row[base + lane];
    sl_score[lane] = st.s_score[base + lane];
  }
  if (lane == 64) {
    const int q = st.b_input[b];
    q_in_sh = q;
    t_sh = st.b_steps[b] + 1;     // 1-based index of the emitted token
    max_len_sh = st.q_ml[q];
  }
  if (lane == 128) nvalid_sh = 0;
  if (lane >= 192 && lane < 192 + KMAX_SUPPORTED) at_rank[lane - 192] = -1;
  __syncthreads();
  const int q_in = q_in_sh, t = t_sh, max_len = max_len_sh;

  // Candidate set: child c of parent j at index j*k + c; no-op of parent j
  // at index k*k + j.
  const int C = k * k + k;
  for (int q = lane; q < C; q += BEAM_THREADS) {
    int valid = 0, par, tok = -1;
    double sc = 0.0;
    if (q < k * k) {
      par = q / k;
      const int c = q - par * k;
      if (sl_status[par] == SLOT_ACTIVE) {
        const int r = sl_row[par];
        sc = sl_score[par] + st.top_lp[(size_t)r * k + c];
        tok = st.top_tok[(size_t)r * k + c];
        valid = tok >= 0 && tok < st.V;
      }
    } else {
      par = q - k * k;
      const int status = sl_status[par];
      if (status == SLOT_EOS || status == SLOT_MAXLEN) {
        sc = sl_score[par];
        valid = 1;
      }
    }
    cs[q] = sc;
    cp[q] = par;
    ct[q] = tok;
    cv[q] = valid;
    if (valid) atomicAdd(&nvalid_sh, 1);
  }
  __syncthreads();

  // Full beam B': rank of every valid candidate among the valid ones.
  for (int q = lane; q < C; q += BEAM_THREADS) {
    if (!cv[q]) continue;
    int rank = 0;
    for (int o = 0; o < C; ++o)
      rank += (cv[o] && cand_beats(cs[o], cp[o], ct[o], cs[q], cp[q], ct[q]));
    if (rank < k) at_rank[rank] = q;
  }
  __syncthreads();

  // Heuristics H and termination, in rank order (at most k entries).
  if (lane == 0) {
    const int full = min(k, nvalid_sh);
    const double ref = at_rank[0] >= 0 ? cs[at_rank[0]] : 0.0;
    for (int j = 0; j < k; ++j) kept_per[j] = 0;
    int w = 0, nact = 0;
    for (int r = 0; r < full; ++r) {
      const int q = at_rank[r];
      if (q < 0) break;
      const double sc = cs[q];
      const int par = cp[q], tok = ct[q];
      if (sc < ref - st.delta) continue;            // relative threshold
      int status;
      if (tok < 0) {
        status = sl_status[par];                   // no-op keeps EOS / MAXLEN
      } else {
        if (kept_per[par] >= st.M) continue;       // max candidates per parent
        kept_per[par] += 1;
        status = tok == 0 ? SLOT_EOS : (t == max_len ? SLOT_MAXLEN : SLOT_ACTIVE);
      }
      nscore[w] = sc;
      npar[w] = par;
      ntok[w] = tok;
      nstat[w] = status;
      nact += status == SLOT_ACTIVE;
      ++w;
    }
    nw_sh = w;
    nact_sh = nact;
  }
  __syncthreads();
  const int w = nw_sh;
  const bool ends = nact_sh == 0;

  // History: backpointers of level t, indexed by the input's queue position.
  if (lane < w) {
    const uint32_t tokbits = ntok[lane] < 0 ? BP_NOOP : (uint32_t)ntok[lane];
    st.bp[((size_t)q_in * st.max_len_cap + (t - 1)) * k + lane] = ((uint32_t)npar[lane] << 24) | tokbits;
  }

  if (ends) {
    // Y[i] = the survivors in rank order; tokens are rebuilt later.
    const int fin = (int)st.ctrl->timesteps;
    if (lane < w) {
      OutHyp h;
      h.score = nscore[lane];
      h.length = 0;
      h.status = nstat[lane];
      h.finalize_step = fin;
      h.level = t;
      st.o_hyp[(size_t)q_in * k + lane] = h;
    }
    if (lane < k) {
      st.s_status[base + lane] = SLOT_EMPTY;
      st.s_prow[base + lane] = -1;
    }
    if (lane == 0) {
      st.o_count[q_in] = w;
      st.b_input[b] = -1;
      atomicAdd(reinterpret_cast<unsigned long long *>(&st.ctrl->hyps), (unsigned long long)w);
      atomicAdd(reinterpret_cast<unsigned long long *>(&st.ctrl->finished), 1ull);
    }
    return;
  }

  // Continue: write the new beam into ranks 0..w-1 (no-ops keep their
  // state; active children take their parent's new state h).
  if (lane < k) {
    if (lane < w) {
      const int par = npar[lane];
      st.s_status[base + lane] = nstat[lane];
      st.s_score[base + lane] = nscore[lane];
      if (ntok[lane] >= 0) st.s_tok[base + lane] = ntok[lane];
      st.s_prow[base + lane] = nstat[lane] == SLOT_ACTIVE ? sl_row[par] : -1;
    } else {
      st.s_status[base + lane] = SLOT_EMPTY;
      st.s_prow[base + lane] = -1;
    }
  }
  if (lane == 0) {
    st.b_steps[b] = t;
    st.b_par[b] ^= 1;
  }
  // State copy: s_h[rank] <- hbuf[row(parent)] for every active survivor,
  // flattened over (survivor, 16-byte chunk) so all threads stream.
  const int rowbytes = st.d * (st.dtype == 1 ? 2 : 4);
  const int chunks = rowbytes / 16;
  __shared__ int cp_src[KMAX_SUPPORTED], cp_dst[KMAX_SUPPORTED];
  __shared__ int ncopy;
  if (lane == 0) {
    int c = 0;
    for (int r = 0; r < w; ++r)
      if (nstat[r] == SLOT_ACTIVE) {
        cp_src[c] = sl_row[npar[r]];
        cp_dst[c] = base + r;
        ++c;
      }
    ncopy = c;
  }
  __syncthreads();
  const uint4 *__restrict__ hb = static_cast<const uint4 *>(st.hbuf);
  uint4 *__restrict__ sh = static_cast<uint4 *>(st.s_h);
  const int total = ncopy * chunks;
  for (int x = lane; x < total; x += BEAM_THREADS) {
    const int r = x / chunks, c = x - r * chunks;
    sh[(size_t)cp_dst[r] * chunks + c] = hb[(size_t)cp_src[r] * chunks + c];
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
  const uint32_t *bp = st.bp + (size_t)q * st.max_len_cap * k;
  const int top = min(h->level, st.max_len_cap);
  int pos = rank, len = 0;
  for (int lev = top; lev >= 1; --lev) {
    const uint32_t e = bp[(size_t)(lev - 1) * k + pos];
    len += (e & 0xFFFFFFu) != BP_NOOP;
    pos = min((int)(e >> 24), k - 1);
  }
  int32_t *out = st.o_tok + ((size_t)q * k + rank) * st.max_len_cap;
  pos = rank;
  int idx = len;
  for (int lev = top; lev >= 1; --lev) {
    const uint32_t e = bp[(size_t)(lev - 1) * k + pos];
    const uint32_t tok = e & 0xFFFFFFu;
    if (tok != BP_NOOP) out[--idx] = (int32_t)tok;
    pos = min((int)(e >> 24), k - 1);
  }
  h->length = len;
}

}  // namespace

hipError_t launch_rowmerge(const DevState &st, hipStream_t s) {
  const int G = (st.R_max + 3) / 4;
  switch (st.kbucket) {
    case 4: hipLaunchKernelGGL((k_rowmerge<4>), dim3(G), dim3(256), 0, s, st); break;
    case 8: hipLaunchKernelGGL((k_rowmerge<8>), dim3(G), dim3(256), 0, s, st); break;
    default: hipLaunchKernelGGL((k_rowmerge<16>), dim3(G), dim3(256), 0, s, st); break;
  }
  return hipGetLastError();
}

hipError_t launch_beam(const DevState &st, hipStream_t s) {
  hipLaunchKernelGGL(k_beam, dim3(st.n), dim3(BEAM_THREADS), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_backtrack(const DevState &st, int q0, int q1, hipStream_t s) {
  if (q1 <= q0) return hipSuccess;
  const long long total = (long long)(q1 - q0) * st.k;
  hipLaunchKernelGGL(k_backtrack, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, st, q0, q1);
  return hipGetLastError();
}

}  // namespace sb
