// Scheduler kernel: refill/admission, beam selection by minimal l_t (or
// every live beam, or the capacity-constrained prefix) and compaction of the
// active candidates of the selected beams into a dense row list (Alg. 1: the
// refill branch, "select E_s, B_s with min l_t", and the candidate loop's
// iteration space; Sec. 3's selection up to a limit on total beam width).
// One workgroup; the step's decisions are taken on the device so no host
// round trip is needed.
#include <algorithm>

#include "sb_internal.h"

namespace sb {

namespace {

constexpr int SCHED_THREADS = 1024;   // at most; a launch takes one wave per 64 x PER beams

// Exclusive prefix sum across the workgroup; *total receives the sum.
__device__ int block_excl_scan(int v, int *sm, int *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sm[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < nw; ++i) {
      int t = sm[i];
      sm[i] = acc;
      acc += t;
    }
    sm[nw] = acc;
  }
  __syncthreads();
  int res = sm[w] + x - v;
  *total = sm[nw];
  __syncthreads();
  return res;
}

// Each thread owns a contiguous range of at most SCHED_MAXB beams (so rows
// come out in beam order) and keeps their records in registers.
constexpr int SCHED_MAXB = 4;
constexpr int SCHED_MAXP = SCHED_THREADS * SCHED_MAXB;   // beam records
constexpr int SCHED_MAXL = 4096;                         // l_t bins (max_len_cap)

// Capacity-constrained selection works on the live beams in admission
// order: b_order lists their records (the previous step's live beams, then
// the ones admitted by that step). Its LDS scratch: per record (l_t << 8 |
// active width), the new order list, the active width per l_t, the
// selection flags, and the cut (l*, rows left at l*).
struct CapSmem {
  int info[SCHED_MAXP];
  int ord[SCHED_MAXP];
  int hist[SCHED_MAXL];
  unsigned char sel[SCHED_MAXP];
  int cut[2];
};

// Capacity-constrained selection (Sec. 3, last paragraph): the live beams
// in order of (l_t, admission) are taken while their active candidates total
// at most row_budget rows. Called by the whole workgroup after admission
// with the thread's records (inp, stp, active-slot masks) and its kept
// positions of the old order list (orec); nlive = live beams after admission. Leaves cs.sel[b]
// set for the selected records and writes the new order list to b_order.
template <int PER>
__device__ void cap_select(const DevState &st, CapSmem &cs, int *sm, const int *inp, const int *stp,
                           const uint32_t *amask, const int *orec, int b0, int nb, int nlive) {
  // Kept positions are compacted in order ahead of the admitted beams.
  int kept_l = 0;
#pragma unroll
  for (int u = 0; u < PER; ++u) kept_l += u < nb && orec[u] >= 0;
  int kept_tot;
  int pos = block_excl_scan(kept_l, sm, &kept_tot);
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if (u < nb && orec[u] >= 0) cs.ord[pos++] = orec[u];
  // Per record: l_t and active width (a fresh beam has one candidate).
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (u < nb) {
      const int b = b0 + u;
      cs.sel[b] = 0;
      if (inp[u] >= 0) {
        cs.info[b] = (stp[u] << 8) | __popc(amask[u]);   // a fresh beam: one candidate
      }
    }
  }
  __syncthreads();
  // New order list to memory; active width per l_t.
  int oinfo[PER], orid[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    orid[u] = -1;
    oinfo[u] = 0;
    if (u < nb && b0 + u < nlive) {
      orid[u] = cs.ord[b0 + u];
      oinfo[u] = cs.info[orid[u]];
      st.b_order[b0 + u] = orid[u];
      atomicAdd(&cs.hist[min(oinfo[u] >> 8, st.max_len_cap - 1)], oinfo[u] & 0xff);   // live l_t < max_len
    }
  }
  __syncthreads();
  // The cut: l* = the first l_t whose cumulative width exceeds the budget;
  // every beam below l* fits, none above it is taken.
  const int L = st.max_len_cap, budget = st.row_budget;
  const int bins = (L + (int)blockDim.x - 1) / (int)blockDim.x;
  const int j0 = min(L, (int)threadIdx.x * bins), j1 = min(L, j0 + bins);
  int hsum = 0;
  for (int j = j0; j < j1; ++j) hsum += cs.hist[j];
  int htot;
  int cum = block_excl_scan(hsum, sm, &htot);
  for (int j = j0; j < j1; ++j) {
    const int h = cs.hist[j];
    if (cum <= budget && cum + h > budget) {
      cs.cut[0] = j;
      cs.cut[1] = budget - cum;
    }
    cum += h;
  }
  __syncthreads();
  const int lstar = cs.cut[0], rem = cs.cut[1];
  // At l*, beams are taken in admission order while they fit.
  int lv = 0;
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if (orid[u] >= 0 && (oinfo[u] >> 8) == lstar) lv += oinfo[u] & 0xff;
  int ltot;
  int e = block_excl_scan(lv, sm, &ltot);
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (orid[u] >= 0) {
      const int s = oinfo[u] >> 8, w = oinfo[u] & 0xff;
      bool take = s < lstar;
      if (s == lstar) {
        take = e + w <= rem;
        e += w;
      }
      cs.sel[orid[u]] = take;
    }
  }
  __syncthreads();
}

// The scheduler proper. PER = beams per thread (a contiguous range, so rows
// come out in beam order). Every beam and slot field it needs is loaded at
// the start in one batch; the step then takes two barrier phases (plus the
// capacity selection's): live/free counts with the minimal l_t, then the
// row offsets with the step's totals.
template <int PER>
__global__ __launch_bounds__(SCHED_THREADS) void k_sched(DevState st) {
  constexpr int NWMAX = SCHED_THREADS / 64;
  const int NW = (int)blockDim.x >> 6;
  __shared__ long long ph1[NWMAX + 1];
  __shared__ int ph1_min[NWMAX + 1];
  __shared__ int ph2[4][NWMAX + 1];
  __shared__ int sm[NWMAX + 1];
  __shared__ CapSmem cs;
  DevCtrl *c = st.ctrl;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = st.n, k = st.k;
  const int nq = c->n_queued, cursor = c->cursor;
  const int b0 = min(n, tid * PER), nb = min(n, b0 + PER) - b0;
  const bool cap = st.cap != 0;

  // Capacity mode: this thread's positions b0 .. b0+nb-1 of the order list
  // (which holds the live + admitted count of the previous step), read
  // before any record changes below; a beam that finished since is dropped.
  int orec[PER];
  if (cap) {
    const int nord = c->live;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      orec[u] = -1;
      if (u < nb && b0 + u < nord) {
        const int r = st.b_order[b0 + u];
        if (st.b_input[r] >= 0) orec[u] = r;
      }
    }
    for (int j = tid; j < st.max_len_cap; j += (int)blockDim.x) cs.hist[j] = 0;
    if (tid == 0) {
      cs.cut[0] = INT_MAX;
      cs.cut[1] = 0;
    }
  }

  // Beam records, slot states (active / terminated masks), the inputs'
  // source lengths and, with at most two beams per thread, the slots' last
  // tokens. The slot loops run to the compile-time bound so that all loads
  // are in flight together.
  constexpr int PT = PER <= 2 ? PER : 1;
  int inp[PER], stp[PER], lxv[PER];
  uint32_t amask[PER], tmask[PER];
  int tok[PT][KMAX_SUPPORTED];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    inp[u] = -1;
    stp[u] = 0;
    amask[u] = 0u;
    tmask[u] = 0u;
    if (u < nb) {
      inp[u] = st.b_input[b0 + u];
      stp[u] = st.b_steps[b0 + u];
#pragma unroll
      for (int j = 0; j < KMAX_SUPPORTED; ++j) {
        if (j < k) {
          const int status = st.s_status[(b0 + u) * k + j];
          amask[u] |= (uint32_t)(status == SLOT_ACTIVE) << j;
          tmask[u] |= (uint32_t)(status == SLOT_EOS || status == SLOT_MAXLEN) << j;
          if (u < PT) tok[u < PT ? u : 0][j] = st.s_tok[(b0 + u) * k + j];
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) lxv[u] = inp[u] >= 0 ? st.q_Lx[inp[u]] : 0;

  // Phase 1: live (low word) and free (high word) records, exclusive over
  // threads, and the minimal l_t of the live beams.
  int live_l = 0, mn_l = INT_MAX;
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if (u < nb && inp[u] >= 0) {
      ++live_l;
      mn_l = min(mn_l, stp[u]);
    }
  long long pre, tot;
  int mn0;
  {
    const long long v = ((long long)(nb - live_l) << 32) | live_l;
    long long x = v;
    int mm = mn_l;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const long long y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
      mm = min(mm, __shfl_xor(mm, o, 64));
    }
    if (lane == 63) ph1[w] = x;
    if (lane == 0) ph1_min[w] = mm;
    __syncthreads();
    if (tid == 0) {
      long long acc = 0;
      int m = INT_MAX;
      for (int i = 0; i < NW; ++i) {
        const long long t = ph1[i];
        ph1[i] = acc;
        acc += t;
        m = min(m, ph1_min[i]);
      }
      ph1[NW] = acc;
      ph1_min[NW] = m;
    }
    __syncthreads();
    pre = ph1[w] + x - v;
    tot = ph1[NW];
    mn0 = ph1_min[NW];
  }
  const int live = (int)(tot & 0xffffffff);

  // Refill (Alg. 1): if inputs remain and |B| <= eps*n, admit
  // m = min(n - |B|, left) new inputs, in index order, into the free beam
  // records in index order.
  int admit = 0;
  if (cursor < nq && live <= st.refill_thr) admit = min(n - live, nq - cursor);
  if (admit > 0) {
    int rank = (int)(pre >> 32);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      if (u < nb && inp[u] < 0) {
        if (rank < admit) {
          const int b = b0 + u;
          inp[u] = cursor + rank;
          stp[u] = 0;
          amask[u] = 1u;
          tmask[u] = 0u;
          lxv[u] = st.q_Lx[inp[u]];
          if (u < PT) tok[u < PT ? u : 0][0] = 0;
          st.b_input[b] = inp[u];
          st.b_steps[b] = 0;
          st.b_par[b] = 0;
          st.b_ml[b] = st.q_ml[inp[u]];
          st.b_nout[b] = 0;
          if (cap) cs.ord[live + rank] = b;   // admitted beams follow the live ones
          for (int j = 0; j < k; ++j) {
            st.s_status[b * k + j] = j == 0 ? SLOT_ACTIVE : SLOT_EMPTY;
            st.s_score[b * k + j] = 0.0;
            st.s_tok[b * k + j] = 0;   // start symbol
          }
        }
        ++rank;
      }
    }
  }

  // Selection: the live beams with the fewest steps taken (an admitted beam
  // has taken none), or every live beam (Var-Str-FIFO: the capacity n, from
  // the beam with the most steps down, covers all of them), or the
  // capacity-constrained prefix.
  const int mn = admit > 0 ? 0 : mn0;
  if (cap) cap_select<PER>(st, cs, sm, inp, stp, amask, orec, b0, nb, live + admit);

  bool sel[PER];
  int act_l = 0, term_l = 0, sel_l = 0, pos_l = 0;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    sel[u] = u < nb && inp[u] >= 0 && (cap ? cs.sel[b0 + u] != 0 : (st.select_all || stp[u] == mn));
    if (sel[u]) {
      ++sel_l;
      act_l += __popc(amask[u]);
      term_l += __popc(tmask[u]);
      pos_l += __popc(amask[u]) * (stp[u] + 1);
    } else {
      amask[u] = 0u;
    }
  }
  // Phase 2: row offsets (exclusive scan of active candidates) and the
  // step's totals of rows, no-ops, selected beams and output positions.
  int row, R, noops, nsel, npos;
  {
    int x = act_l, a = term_l, b = sel_l, q = pos_l;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
      a += __shfl_xor(a, o, 64);
      b += __shfl_xor(b, o, 64);
      q += __shfl_xor(q, o, 64);
    }
    if (lane == 63) ph2[0][w] = x;
    if (lane == 0) {
      ph2[1][w] = a;
      ph2[2][w] = b;
      ph2[3][w] = q;
    }
    __syncthreads();
    if (tid == 0) {
      int acc = 0, ta = 0, tb = 0, tq = 0;
      for (int i = 0; i < NW; ++i) {
        const int t = ph2[0][i];
        ph2[0][i] = acc;
        acc += t;
        ta += ph2[1][i];
        tb += ph2[2][i];
        tq += ph2[3][i];
      }
      ph2[0][NW] = acc;
      ph2[1][NW] = ta;
      ph2[2][NW] = tb;
      ph2[3][NW] = tq;
    }
    __syncthreads();
    row = ph2[0][w] + x - act_l;
    R = ph2[0][NW];
    noops = ph2[1][NW];
    nsel = ph2[2][NW];
    npos = ph2[3][NW];
  }

#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (u < nb) {
      const int b = b0 + u;
      st.b_sel[b] = sel[u];
      const int lx = sel[u] ? lxv[u] : 0;
#pragma unroll
      for (int j = 0; j < KMAX_SUPPORTED; ++j) {
        if (j >= k) break;
        const int s = b * k + j;
        if ((amask[u] >> j) & 1u) {
          int y;
          if (u < PT) y = tok[u < PT ? u : 0][j];
          else y = st.s_tok[s];
          st.r_slot[row] = s;
          st.r_hsrc[row] = stp[u] == 0 ? -1 - inp[u] : s;   // a fresh beam reads its encoding h0
          if (st.rec_i8) {
            st.haux[row].F = 1;
            st.haux[row].n = 0;
          }
          st.r_y[row] = y;
          st.r_t[row] = stp[u] + 1;
          st.r_Lx[row] = lx;
          st.s_row[s] = row;
          ++row;
        } else {
          st.s_row[s] = -1;
        }
      }
    }
  }

  if (tid == 0) {
    c->cursor = cursor + admit;
    c->live = live + admit;
    c->R = R;
    c->n_sel = nsel;
    c->t_sel = R > 0 ? mn + 1 : 0;
    c->done = R == 0 ? 1 : 0;
    // Counters by atomic adds whose results are not read (no wait).
    typedef unsigned long long u64;
    if (R > 0) {
      atomicAdd(reinterpret_cast<u64 *>(&c->rows_hist[min(63, R / st.hist_width)]), 1ull);
      atomicAdd(reinterpret_cast<u64 *>(&c->timesteps), 1ull);
      atomicAdd(reinterpret_cast<u64 *>(&c->expansions), (u64)R);
      atomicAdd(reinterpret_cast<u64 *>(&c->noops), (u64)noops);
      atomicAdd(reinterpret_cast<u64 *>(&c->positions), (u64)npos);
    }
    if (admit > 0) {
      atomicAdd(reinterpret_cast<u64 *>(&c->refills), 1ull);
      atomicAdd(reinterpret_cast<u64 *>(&c->admitted), (u64)admit);
    }
  }
}

// Reset of every beam, slot, output count and the control block.
__global__ void k_init(DevState st) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < st.n) {
    st.b_input[i] = -1;
    st.b_steps[i] = 0;
    st.b_sel[i] = 0;
    st.b_par[i] = 0;
    st.b_nout[i] = 0;
  }
  if (i < st.n * st.k) {
    st.s_status[i] = SLOT_EMPTY;
    st.s_row[i] = -1;
  }
  if (i < st.max_inputs) st.o_count[i] = 0;
  if (i == 0) {
    DevCtrl z = {};
    z.done = 1;
    *st.ctrl = z;
  }
}

}  // namespace

hipError_t launch_sched(const DevState &st, hipStream_t s) {
  const int per = (st.n + SCHED_THREADS - 1) / SCHED_THREADS;
  // One wave per 64 x PER beam records (cross-wave scans and barriers then
  // span only the waves that hold beams).
  const int p = per <= 1 ? 1 : per == 2 ? 2 : 4;
  const int threads = std::min(SCHED_THREADS, (st.n + 64 * p - 1) / (64 * p) * 64);
  if (p == 1) hipLaunchKernelGGL(k_sched<1>, dim3(1), dim3(threads), 0, s, st);
  else if (p == 2) hipLaunchKernelGGL(k_sched<2>, dim3(1), dim3(threads), 0, s, st);
  else hipLaunchKernelGGL(k_sched<4>, dim3(1), dim3(threads), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_init(const DevState &st, hipStream_t s) {
  int m = st.n * st.k;
  if (st.max_inputs > m) m = st.max_inputs;
  hipLaunchKernelGGL(k_init, dim3((m + 255) / 256), dim3(256), 0, s, st);
  return hipGetLastError();
}

}  // namespace sb
