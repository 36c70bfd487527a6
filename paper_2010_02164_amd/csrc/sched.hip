// Scheduler kernel: refill/admission, beam selection by minimal l_t and
// compaction of the active candidates of the selected beams into a dense
// row list (Alg. 1: the refill branch, "select E_s, B_s with min l_t", and
// the candidate loop's iteration space). One workgroup; the step's
// decisions are taken on the device so no host round trip is needed.
#include "sb_internal.h"

namespace sb {

namespace {

constexpr int SCHED_THREADS = 1024;

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

__device__ int block_min(int v, int *sm) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  if (lane == 0) sm[w] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int m = sm[0];
    for (int i = 1; i < nw; ++i) m = min(m, sm[i]);
    sm[nw] = m;
  }
  __syncthreads();
  int r = sm[nw];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(SCHED_THREADS) void k_sched(DevState st) {
  __shared__ int sm[SCHED_THREADS / 64 + 1];
  DevCtrl *c = st.ctrl;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int n = st.n, k = st.k;
  const int nq = c->n_queued, cursor = c->cursor;

  // Live beams before admission (|B| in Alg. 1).
  int lc = 0;
  for (int b = tid; b < n; b += nt) lc += (st.b_input[b] >= 0);
  int live;
  block_excl_scan(lc, sm, &live);

  // Refill: if inputs remain and |B| <= eps*n, admit m = min(n - |B|, left)
  // new inputs, in index order, into the free beam records in index order.
  int admit = 0;
  if (cursor < nq && live <= st.refill_thr) admit = min(n - live, nq - cursor);
  if (admit > 0) {
    const int per = (n + nt - 1) / nt;
    const int b0 = min(n, tid * per), b1 = min(n, b0 + per);
    int fc = 0;
    for (int b = b0; b < b1; ++b) fc += (st.b_input[b] < 0);
    int tot;
    int rank = block_excl_scan(fc, sm, &tot);
    for (int b = b0; b < b1; ++b) {
      if (st.b_input[b] >= 0) continue;
      if (rank < admit) {
        st.b_input[b] = cursor + rank;
        st.b_steps[b] = 0;
        st.b_par[b] = 0;
        for (int j = 0; j < k; ++j) {
          st.s_status[b * k + j] = j == 0 ? SLOT_ACTIVE : SLOT_EMPTY;
          st.s_score[b * k + j] = 0.0;
          st.s_tok[b * k + j] = 0;   // start symbol
        }
      }
      ++rank;
    }
  }
  __syncthreads();

  // Selection: the live beams with the fewest steps taken.
  int mn = INT_MAX;
  for (int b = tid; b < n; b += nt)
    if (st.b_input[b] >= 0) mn = min(mn, st.b_steps[b]);
  mn = block_min(mn, sm);

  // Compaction of the selected beams' active candidates, in slot order.
  const int nslots = n * k;
  const int per = (nslots + nt - 1) / nt;
  const int s0 = min(nslots, tid * per), s1 = min(nslots, s0 + per);
  int ac = 0, tc = 0;
  for (int s = s0; s < s1; ++s) {
    const int b = s / k;
    const bool sel = st.b_input[b] >= 0 && st.b_steps[b] == mn;
    const int status = st.s_status[s];
    ac += (sel && status == SLOT_ACTIVE);
    tc += (sel && (status == SLOT_EOS || status == SLOT_MAXLEN));
  }
  int R;
  int row = block_excl_scan(ac, sm, &R);
  int noops;
  block_excl_scan(tc, sm, &noops);
  for (int s = s0; s < s1; ++s) {
    const int b = s / k;
    const bool sel = st.b_input[b] >= 0 && st.b_steps[b] == mn;
    if (sel && st.s_status[s] == SLOT_ACTIVE) {
      const int q = st.b_input[b];
      st.r_slot[row] = s;
      st.r_hsrc[row] = mn == 0 ? -1 - q : s;   // a fresh beam reads its encoding h0
      st.r_y[row] = st.s_tok[s];
      st.r_t[row] = mn + 1;
      st.r_Lx[row] = st.q_Lx[q];
      st.s_row[s] = row;
      ++row;
    } else {
      st.s_row[s] = -1;
    }
  }
  int ns = 0;
  for (int b = tid; b < n; b += nt) {
    const int sel = st.b_input[b] >= 0 && st.b_steps[b] == mn;
    st.b_sel[b] = sel;
    ns += sel;
  }
  int nsel;
  block_excl_scan(ns, sm, &nsel);

  if (tid == 0) {
    c->cursor = cursor + admit;
    c->live = live + admit;
    c->R = R;
    c->n_sel = nsel;
    c->t_sel = R > 0 ? mn + 1 : 0;
    c->done = R == 0 ? 1 : 0;
    if (R > 0) {
      c->rows_hist[min(63, R / st.hist_width)] += 1;
      c->timesteps += 1;
      c->expansions += R;
      c->noops += noops;
    }
    if (admit > 0) {
      c->refills += 1;
      c->admitted += admit;
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
  }
  if (i < st.n * st.k) {
    st.s_status[i] = SLOT_EMPTY;
    st.s_row[i] = -1;
    st.s_prow[i] = -1;
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
  hipLaunchKernelGGL(k_sched, dim3(1), dim3(SCHED_THREADS), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_init(const DevState &st, hipStream_t s) {
  int m = st.n * st.k;
  if (st.max_inputs > m) m = st.max_inputs;
  hipLaunchKernelGGL(k_init, dim3((m + 255) / 256), dim3(256), 0, s, st);
  return hipGetLastError();
}

}  // namespace sb
