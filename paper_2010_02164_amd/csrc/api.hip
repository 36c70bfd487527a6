// Host side of the streambeam C ABI: validation, workspace carve-up, the
// per-timestep launch sequence of Alg. 1 and result collection.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/streambeam.h"
#include "sb_internal.h"
#include "topk.h"

using namespace sb;

struct sb_decoder {
  sb_model model;
  sb_params params;
  DevState st;
  hipStream_t stream;
  unsigned char *ws;
  size_t ws_bytes;
  int32_t n_queued = 0;
  int32_t collected = 0;       // inputs already returned by sb_collect
  int32_t *pinned_len = nullptr;   // [2][max_inputs] L_x and max_len staging (none: noalloc)
  int32_t *pinned_flag = nullptr;  // [2] done-flag readback (noalloc: host_flag below)
  int32_t host_flag[2] = {0, 0};   // done-flag readback of a decoder that allocates nothing
  int device = 0;
  bool noalloc = false;            // lives in the library's static storage (sb_create_noalloc)
  hipEvent_t poll_ev[2] = {nullptr, nullptr};
  bool timing = false;
  double proj_ms = 0.0;
  int64_t proj_launches = 0;
  // A burst of timesteps captured once as a HIP graph (untimed runs).
  hipStream_t cap_stream = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t graph_exec = nullptr;
  // Timed runs launch kernel by kernel with an event pair around every
  // projection launch, taken from this pool.
  std::vector<hipEvent_t> tev;
  int tev_used = 0;
  std::vector<int64_t> ids;   // caller id per queue position
  std::string err;
};

namespace {

constexpr size_t ALIGN = 256;

struct Layout {
  size_t ctrl, q_h0, q_Lx, q_ml, b_input, b_steps, b_sel, b_par, b_ml, b_nout, b_order, s_status, s_score, s_tok, s_h,
      s_row, bp, r_slot, r_hsrc, r_y, r_t, r_Lx, r_lse, hbuf, part, top_lp, top_tok,
      o_count, o_hyp, o_tok, o_pack, o_off, wh_t, kvs, anc, wkv_t, xbuf, attn_part, wout_t, wd3, w_exp, w_ln, w_li,
      w_lv, wt_off, wt_col, wt_val, hd, s_hd, q_hd, haux, s_haux, q_haux, total;
};

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// The exact bf16 recurrence: its K loop takes 4 waves x 2 blocks x 32
// values per pass and its digit sums stay exact in fp64 up to 2048 state
// values.
bool rec_i8_eligible(const sb_model &m) { return m.dtype == SB_BF16 && m.d % 256 == 0 && m.d <= 2048; }

int kbucket_of(int k) { return k <= 4 ? 4 : (k <= 8 ? 8 : 16); }

// Keys per partial record: the short list when the vocabulary spans at
// least 64 projection tiles (a tile then rarely holds 4 of a row's best k,
// and the row merge recomputes the ones that do), else the k-bucket.
int tile_keys_of(const sb_model &m, const sb_params &p) {
  const int kb = kbucket_of(p.k + (p.finalize_rule == SB_RULE_FAIRSEQ ? 1 : 0));
  return proj_tiles(m.vocab) >= 64 ? TILE_KEYS_SHORT : kb;
}

// Beam records held by the decoder: the cached pool (0 means n).
int pool_of(const sb_params &p) { return p.pool > 0 ? p.pool : p.n; }

Layout layout_of(const sb_model &m, const sb_params &p) {
  Layout L{};
  const size_t es = m.dtype == SB_BF16 ? 2 : 4;
  // Beams and candidate slots are sized by the pool of cached beams; the
  // per-row buffers by the n*k rows a timestep may expand.
  const size_t n = pool_of(p), k = p.k, d = m.d, nk = n * k, Rm = (size_t)p.n * k;
  const size_t S = proj_tiles(m.vocab);
  const size_t bpw = p.finalize_rule == SB_RULE_FAIRSEQ ? 2 * (size_t)p.k : (size_t)p.k;
  const size_t Q = p.max_inputs, MLC = p.max_len_cap;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += up(bytes);
    return o;
  };
  L.ctrl = take(sizeof(DevCtrl));
  L.q_h0 = take(Q * d * es);
  L.q_Lx = take(Q * 4);
  L.q_ml = take(Q * 4);
  L.b_input = take(n * 4);
  L.b_steps = take(n * 4);
  L.b_sel = take(n * 4);
  L.b_par = take(n * 4);
  L.b_ml = take(n * 4);
  L.b_nout = take(n * 4);
  L.b_order = take(n * 4);
  L.s_status = take(nk * 4);
  L.s_score = take(nk * 8);
  L.s_tok = take(nk * 4);
  L.s_h = take(nk * d * es);
  L.s_row = take(nk * 4);
  L.bp = take(Q * MLC * bpw * 4);
  L.r_slot = take(Rm * 4);
  L.r_hsrc = take(Rm * 4);
  L.r_y = take(Rm * 4);
  L.r_t = take(Rm * 4);
  L.r_Lx = take(Rm * 4);
  L.r_lse = take(Rm * 8);
  L.hbuf = take(Rm * d * es);
  L.part = take(Rm * S * part_width(tile_keys_of(m, p)) * 4);
  L.top_lp = take(Rm * k * 8);
  L.top_tok = take(Rm * k * 4);
  L.o_count = take(Q * 4);
  L.o_hyp = take(Q * k * sizeof(OutHyp));
  L.o_tok = take(Q * k * MLC * 4);
  L.o_pack = take(Q * k * MLC * 4);
  L.o_off = take(Q * k * 8);
  L.wout_t = take(S * 128 * d * es);
  L.wh_t = take(d * d * es);   // W_h in the recurrence's fragment order
  if (m.kv_layers > 0) {
    const size_t planes = (size_t)m.kv_layers * 2;
    L.kvs = take(nk * MLC * planes * d * 2);
    L.anc = take(2 * nk * ((MLC + 3) / 4 * 4));
    L.wkv_t = take(planes * d * d * 2);
  }
  if (m.attn) {
    L.xbuf = take(Rm * d * 2);
    L.attn_part = take(Rm * (size_t)m.kv_layers * d * 8);
  }
  if (rec_i8_eligible(m)) {
    L.wd3 = take(3 * d * d);
    L.w_exp = take(d * 4);
    L.w_ln = take((d + 1) * 4);
    L.w_li = take(d * REC_WLIST * 4);
    L.w_lv = take(d * REC_WLIST * 4);
    L.wt_off = take(d / 32 * 33 * 4);
    L.wt_col = take(d / 32 * REC_WTILE * 4);
    L.wt_val = take(d / 32 * REC_WTILE * 4);
    L.hd = take(Rm * rec_dig_row_bytes(d));
    L.s_hd = take(nk * rec_dig_row_bytes(d));
    L.q_hd = take(Q * rec_dig_row_bytes(d));
    L.haux = take(Rm * sizeof(RowAux));
    L.s_haux = take(nk * sizeof(RowAux));
    L.q_haux = take(Q * sizeof(RowAux));
  }
  L.total = off;
  return L;
}

sb_status check(const sb_model *m, const sb_params *p, std::string *why) {
  auto bad = [&](sb_status s, const char *msg) {
    if (why) *why = msg;
    return s;
  };
  if (!m || !p) return bad(SB_E_INVALID_ARG, "null model or params");
  if (m->dtype != SB_F32 && m->dtype != SB_BF16) return bad(SB_E_INVALID_ARG, "unknown dtype");
  if (m->d < 64 || m->d > 4096 || m->d % 64) return bad(SB_E_UNSUPPORTED, "d must be a multiple of 64 in [64, 4096]");
  if (m->dtype == SB_BF16 && m->d % 128) return bad(SB_E_UNSUPPORTED, "bf16 needs d a multiple of 128");
  if (p->k < 1 || p->k > KMAX_SUPPORTED) return bad(SB_E_UNSUPPORTED, "k must be in [1, 16]");
  if (m->vocab < 2 || m->vocab < p->k || m->vocab > (1 << 23)) return bad(SB_E_INVALID_ARG, "vocab must be in [max(2,k), 2^23]");
  if (!(p->n >= 1 && p->n <= 4096)) return bad(SB_E_UNSUPPORTED, "n must be in [1, 4096]");  // 4 beams per scheduler thread
  if ((int64_t)p->n * p->k > 65536) return bad(SB_E_UNSUPPORTED, "n*k must be <= 65536");
  if (!(p->eps >= 0.0 && p->eps < 1.0)) return bad(SB_E_INVALID_ARG, "eps must be in [0, 1)");
  if (!(p->delta > 0.0)) return bad(SB_E_INVALID_ARG, "delta must be > 0 (use +inf to disable)");
  if (p->max_per_node < 1 || p->max_per_node > p->k) return bad(SB_E_INVALID_ARG, "max_per_node must be in [1, k]");
  if (p->sched < SB_FIXED || p->sched > SB_VAR_CAP) return bad(SB_E_INVALID_ARG, "unknown scheduler");
  if (p->pool != 0 && p->pool != p->n && p->sched != SB_VAR_CAP)
    return bad(SB_E_INVALID_ARG, "a pool other than n needs SB_VAR_CAP");
  if (p->pool != 0 && (p->pool < p->n || p->pool > 4096)) return bad(SB_E_INVALID_ARG, "pool must be 0 or in [n, 4096]");
  if ((int64_t)pool_of(*p) * p->k > 65536) return bad(SB_E_UNSUPPORTED, "pool*k must be <= 65536");
  if (p->finalize_rule != SB_RULE_PAPER && p->finalize_rule != SB_RULE_FAIRSEQ)
    return bad(SB_E_INVALID_ARG, "unknown finalization rule");
  if (p->finalize_rule == SB_RULE_FAIRSEQ && p->k > KMAX_SUPPORTED - 1)
    return bad(SB_E_UNSUPPORTED, "the Fairseq rule needs k <= 15");
  if (p->max_len_cap < 1 || p->max_len_cap > 4096) return bad(SB_E_INVALID_ARG, "max_len_cap must be in [1, 4096]");
  if (p->max_inputs < 1) return bad(SB_E_INVALID_ARG, "max_inputs must be >= 1");
  const int64_t es = m->dtype == SB_BF16 ? 2 : 4;
  if ((int64_t)(m->vocab + 127) / 128 * 128 * m->d * es >= (1ll << 32) ||
      (int64_t)pool_of(*p) * p->k * m->d * es >= (1ll << 32))
    return bad(SB_E_UNSUPPORTED, "W_out and the candidate-state buffer must each be under 4 GiB");
  if (m->kv_layers < 0 || m->kv_layers > 8) return bad(SB_E_UNSUPPORTED, "kv_layers must be in [0, 8]");
  if (m->kv_layers > 0 && m->dtype != SB_BF16) return bad(SB_E_UNSUPPORTED, "KV state requires bf16");
  if (m->kv_layers > 0 && !m->W_kv) return bad(SB_E_INVALID_ARG, "W_kv is NULL");
  if (m->attn != 0 && m->attn != 1) return bad(SB_E_INVALID_ARG, "attn must be 0 or 1");
  if (m->attn && m->kv_layers == 0) return bad(SB_E_INVALID_ARG, "attention needs a KV state");
  if (m->attn && m->d != 256 && m->d != 512 && m->d != 1024 && m->d != 2048)
    return bad(SB_E_UNSUPPORTED, "attention needs d in {256, 512, 1024, 2048}");
  return SB_OK;
}

// Effective search parameters of a scheduler (Sec. 3; App. A.1).
sb_params effective(const sb_params &p) {
  sb_params e = p;
  if (p.sched == SB_FIXED) {
    e.eps = 0.0;
    e.delta = INFINITY;
    e.max_per_node = p.k;
  } else if (p.sched == SB_VAR_BATCH) {
    e.eps = 0.0;
  } else if (p.sched == SB_FIXED_STREAM) {
    e.delta = INFINITY;
    e.max_per_node = p.k;
  }
  if (p.finalize_rule == SB_RULE_FAIRSEQ) {
    e.delta = INFINITY;
    e.max_per_node = p.k;
  }
  return e;
}

#define HIPCHK(expr)                                                       \
  do {                                                                     \
    hipError_t _e = (expr);                                                \
    if (_e != hipSuccess) {                                                \
      dec->err = std::string(#expr) + ": " + hipGetErrorString(_e);        \
      return SB_E_HIP;                                                     \
    }                                                                      \
  } while (0)

__global__ void k_set_queued(DevCtrl *c, int32_t nq) {
  c->n_queued = nq;
  if (c->cursor < nq) c->done = 0;
}

__global__ void k_set_rows(DevCtrl *c, int32_t R) { c->R = R; }

constexpr int BURST = 8;   // timesteps per graph launch / per done-flag poll

// One timestep of Alg. 1. With e0/e1 given, HIP events bracket the
// projection kernel.
sb_status launch_step(sb_decoder *dec, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
  const DevState &st = dec->st;
  HIPCHK(launch_sched(st, s));
  HIPCHK(launch_rec(st, s));
  if (st.kv_layers > 0) HIPCHK(launch_kv_append(st, s));
  if (st.attn) HIPCHK(launch_attn(st, s));
  if (e0) HIPCHK(hipEventRecord(e0, s));
  HIPCHK(launch_proj(st, s));
  if (e1) HIPCHK(hipEventRecord(e1, s));
  HIPCHK(launch_beam(st, s));
  return SB_OK;
}

// Capture BURST timesteps as a graph on a private stream (the caller's
// stream may be the legacy default stream, which cannot be captured).
sb_status capture(sb_decoder *dec, hipGraph_t *g_out, hipGraphExec_t *exec_out) {
  if (!dec->cap_stream) HIPCHK(hipStreamCreateWithFlags(&dec->cap_stream, hipStreamNonBlocking));
  HIPCHK(hipStreamBeginCapture(dec->cap_stream, hipStreamCaptureModeThreadLocal));
  sb_status st = SB_OK;
  for (int i = 0; i < BURST && st == SB_OK; ++i) st = launch_step(dec, dec->cap_stream);
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(dec->cap_stream, &g);
  if (st != SB_OK) {
    if (g) (void)hipGraphDestroy(g);
    return st;
  }
  HIPCHK(e);
  *g_out = g;
  HIPCHK(hipGraphInstantiate(exec_out, g, nullptr, nullptr, 0));
  return SB_OK;
}

// Add the projection times of the used part of the event pool.
sb_status harvest(sb_decoder *dec) {
  for (int i = 0; i + 1 < dec->tev_used; i += 2) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, dec->tev[i], dec->tev[i + 1]));
    dec->proj_ms += ms;
    dec->proj_launches += 1;
  }
  dec->tev_used = 0;
  return SB_OK;
}

// One timed timestep: events from the pool bracket the projection.
sb_status launch_timed_step(sb_decoder *dec) {
  if (dec->tev_used + 2 > (int)dec->tev.size()) {
    HIPCHK(hipStreamSynchronize(dec->stream));
    sb_status s = harvest(dec);
    if (s != SB_OK) return s;
  }
  hipEvent_t e0 = dec->tev[dec->tev_used], e1 = dec->tev[dec->tev_used + 1];
  dec->tev_used += 2;
  return launch_step(dec, dec->stream, e0, e1);
}

}  // namespace

// Workspace of the allocation-free decoders (below).
static __device__ __align__(256) unsigned char scratch[SB_NOALLOC_SCRATCH_BYTES];

namespace {

// ---------------------------------------------------------------------------
// Allocation-free decoders (sb_create_noalloc). The workspace is a static
// device array, one copy per GPU the library runs on, held until the process
// ends; the decoder object is static host storage, one per GPU. In host code
// `scratch` names a host-side stand-in: kernels and copies get the device
// address that hipGetSymbolAddress returns for the current device.
constexpr int NOALLOC_MAX_DEVICES = 64;

struct NoallocSlot {
  unsigned char *ptr = nullptr;   // device address of `scratch` on this GPU
  bool in_use = false;            // a noalloc decoder on this GPU is alive
  alignas(sb_decoder) unsigned char obj[sizeof(sb_decoder)];
};
NoallocSlot g_noalloc[NOALLOC_MAX_DEVICES];
std::mutex g_noalloc_mu;
thread_local char g_create_err[256] = "";

void set_create_err(const char *msg) {
  snprintf(g_create_err, sizeof g_create_err, "%s", msg);
}

}  // namespace

extern "C" {

const char *sb_status_string(sb_status s) {
  switch (s) {
    case SB_OK: return "ok";
    case SB_E_INVALID_ARG: return "invalid argument";
    case SB_E_WORKSPACE: return "workspace too small or misaligned";
    case SB_E_STATE: return "invalid state";
    case SB_E_QUEUE_FULL: return "input queue full";
    case SB_E_TRUNCATED: return "output truncated";
    case SB_E_HIP: return "HIP runtime error";
    case SB_E_UNSUPPORTED: return "unsupported shape or option";
  }
  return "unknown status";
}

sb_status sb_validate(const sb_model *model, const sb_params *params) {
  return check(model, params, nullptr);
}

size_t sb_workspace_bytes(const sb_model *model, const sb_params *params) {
  if (check(model, params, nullptr) != SB_OK) return 0;
  return layout_of(*model, *params).total;
}

const char *sb_last_error(const sb_decoder *dec) {
  if (dec) return dec->err.c_str();
  return g_create_err[0] ? g_create_err : "null decoder";
}

}  // extern "C"

namespace {

// Set up `dec` over `workspace` (already checked to hold the layout) and
// initialise the device state on `stream`. On failure the caller disposes of
// the decoder with sb_destroy.
sb_status init_decoder(sb_decoder *dec, const sb_model *model, const sb_params *params, void *workspace,
                       size_t bytes, void *stream) {
  const Layout L = layout_of(*model, *params);
  dec->model = *model;
  dec->params = effective(*params);
  dec->stream = static_cast<hipStream_t>(stream);
  dec->ws = static_cast<unsigned char *>(workspace);
  dec->ws_bytes = bytes;
  DevState &st = dec->st;
  unsigned char *w = dec->ws;
  st.ctrl = reinterpret_cast<DevCtrl *>(w + L.ctrl);
  st.q_h0 = w + L.q_h0;
  st.q_Lx = reinterpret_cast<int32_t *>(w + L.q_Lx);
  st.q_ml = reinterpret_cast<int32_t *>(w + L.q_ml);
  st.b_input = reinterpret_cast<int32_t *>(w + L.b_input);
  st.b_steps = reinterpret_cast<int32_t *>(w + L.b_steps);
  st.b_sel = reinterpret_cast<int32_t *>(w + L.b_sel);
  st.b_par = reinterpret_cast<int32_t *>(w + L.b_par);
  st.b_ml = reinterpret_cast<int32_t *>(w + L.b_ml);
  st.b_nout = reinterpret_cast<int32_t *>(w + L.b_nout);
  st.b_order = reinterpret_cast<int32_t *>(w + L.b_order);
  st.s_status = reinterpret_cast<int32_t *>(w + L.s_status);
  st.s_score = reinterpret_cast<double *>(w + L.s_score);
  st.s_tok = reinterpret_cast<int32_t *>(w + L.s_tok);
  st.s_h = w + L.s_h;
  st.s_row = reinterpret_cast<int32_t *>(w + L.s_row);
  st.bp = reinterpret_cast<uint32_t *>(w + L.bp);
  st.r_slot = reinterpret_cast<int32_t *>(w + L.r_slot);
  st.r_hsrc = reinterpret_cast<int32_t *>(w + L.r_hsrc);
  st.r_y = reinterpret_cast<int32_t *>(w + L.r_y);
  st.r_t = reinterpret_cast<int32_t *>(w + L.r_t);
  st.r_Lx = reinterpret_cast<int32_t *>(w + L.r_Lx);
  st.r_lse = reinterpret_cast<double *>(w + L.r_lse);
  st.hbuf = w + L.hbuf;
  st.part = reinterpret_cast<float *>(w + L.part);
  st.top_lp = reinterpret_cast<double *>(w + L.top_lp);
  st.top_tok = reinterpret_cast<int32_t *>(w + L.top_tok);
  st.o_count = reinterpret_cast<int32_t *>(w + L.o_count);
  st.o_hyp = reinterpret_cast<OutHyp *>(w + L.o_hyp);
  st.o_tok = reinterpret_cast<int32_t *>(w + L.o_tok);
  st.o_pack = reinterpret_cast<int32_t *>(w + L.o_pack);
  st.o_off = reinterpret_cast<int64_t *>(w + L.o_off);
  if (model->kv_layers > 0) {
    st.kvs = reinterpret_cast<uint16_t *>(w + L.kvs);
    st.anc = reinterpret_cast<uint8_t *>(w + L.anc);
    st.wkv_t = w + L.wkv_t;
  }
  st.anc_stride = (dec->params.max_len_cap + 3) / 4 * 4;
  st.attn = model->attn;
  st.xbuf = model->attn ? w + L.xbuf : nullptr;
  st.attn_part = model->attn ? reinterpret_cast<double *>(w + L.attn_part) : nullptr;
  st.proj_in = model->attn ? st.xbuf : st.hbuf;
  st.rec_i8 = 0;
  if (rec_i8_eligible(*model)) {
    st.wd3 = reinterpret_cast<int8_t *>(w + L.wd3);
    st.w_exp = reinterpret_cast<int32_t *>(w + L.w_exp);
    st.w_ln = reinterpret_cast<int32_t *>(w + L.w_ln);
    st.w_li = reinterpret_cast<int32_t *>(w + L.w_li);
    st.w_lv = reinterpret_cast<float *>(w + L.w_lv);
    st.wt_off = reinterpret_cast<int32_t *>(w + L.wt_off);
    st.wt_col = reinterpret_cast<int32_t *>(w + L.wt_col);
    st.wt_val = reinterpret_cast<float *>(w + L.wt_val);
    st.hd = reinterpret_cast<int8_t *>(w + L.hd);
    st.s_hd = reinterpret_cast<int8_t *>(w + L.s_hd);
    st.q_hd = reinterpret_cast<int8_t *>(w + L.q_hd);
    st.haux = reinterpret_cast<RowAux *>(w + L.haux);
    st.s_haux = reinterpret_cast<RowAux *>(w + L.s_haux);
    st.q_haux = reinterpret_cast<RowAux *>(w + L.q_haux);
  }
  st.W_h = model->W_h;
  st.E = model->E;
  st.W_out = model->W_out;
  st.wout_t = w + L.wout_t;
  st.wh_t = model->dtype == SB_F32 ? reinterpret_cast<const float4 *>(w + L.wh_t) : nullptr;
  st.wh16_t = model->dtype == SB_BF16 ? reinterpret_cast<const uint2 *>(w + L.wh_t) : nullptr;
  const sb_params &p = dec->params;
  st.n = pool_of(p);
  st.k = p.k;
  st.d = model->d;
  st.V = model->vocab;
  st.M = p.max_per_node;
  st.max_len_cap = p.max_len_cap;
  st.refill_thr = (int32_t)floor(p.eps * (double)st.n);   // live <= eps*P  <=>  live <= floor(eps*P)
  st.S = proj_tiles(model->vocab);
  st.R_max = p.n * p.k;
  st.dtype = model->dtype;
  st.kv_layers = model->kv_layers;
  st.max_inputs = p.max_inputs;
  st.rule = p.finalize_rule;
  st.bpw = p.finalize_rule == SB_RULE_FAIRSEQ ? 2 * p.k : p.k;
  st.kbucket = kbucket_of(p.k + st.rule);   // the Fairseq rule draws k+1 children per parent
  st.tile_keys = tile_keys_of(*model, p);
  st.hist_width = std::max(16, (st.R_max + 63) / 64);
  st.select_all = p.sched == SB_VAR_FIFO ? 1 : 0;
  st.cap = p.sched == SB_VAR_CAP ? 1 : 0;
  st.row_budget = p.n * p.k;
  {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
      return SB_E_HIP;
    st.n_cu = ncu;
    dec->device = dev;
  }
  st.delta = p.delta;
  st.beta = model->eos_beta;

  if (dec->noalloc) {
    // No pinned staging: submits copy straight from the caller's arrays
    // and wait; the done flag is read back into the decoder object. The
    // poll events are made by the first sb_run.
    dec->pinned_flag = dec->host_flag;
  } else {
    if (hipHostMalloc(reinterpret_cast<void **>(&dec->pinned_len), sizeof(int32_t) * 2 * (size_t)p.max_inputs,
                      hipHostMallocDefault) != hipSuccess)
      return SB_E_HIP;
    if (hipHostMalloc(reinterpret_cast<void **>(&dec->pinned_flag), sizeof(int32_t) * 2, hipHostMallocDefault) !=
        hipSuccess)
      return SB_E_HIP;
    for (int i = 0; i < 2; ++i)
      if (hipEventCreateWithFlags(&dec->poll_ev[i], hipEventDisableTiming) != hipSuccess) return SB_E_HIP;
  }
  if (launch_init(st, dec->stream) != hipSuccess) return SB_E_HIP;
  if (launch_relayout_wout(st, dec->stream) != hipSuccess) return SB_E_HIP;
  if (launch_relayout_wh(st, dec->stream) != hipSuccess) return SB_E_HIP;
  if (model->kv_layers > 0 &&
      launch_relayout_wkv(st, static_cast<const uint16_t *>(model->W_kv), dec->stream) != hipSuccess)
    return SB_E_HIP;
  if (rec_i8_eligible(*model)) {
    // W_h's digit planes; a W_h with more small values in a row or a tile
    // than the lists hold keeps the fp64 recurrence.
    int32_t overflow = 1;
    if (launch_rec_prepare(st, dec->stream) != hipSuccess ||
        hipMemcpyAsync(&overflow, st.w_ln + st.d, sizeof(int32_t), hipMemcpyDeviceToHost, dec->stream) != hipSuccess ||
        hipStreamSynchronize(dec->stream) != hipSuccess)
      return SB_E_HIP;
    st.rec_i8 = overflow ? 0 : 1;
  }
  return SB_OK;
}

}  // namespace

extern "C" {

sb_status sb_create(const sb_model *model, const sb_params *params, void *workspace, size_t bytes,
                    void *stream, sb_decoder **out) {
  if (!out) return SB_E_INVALID_ARG;
  *out = nullptr;
  sb_status s = check(model, params, nullptr);
  if (s != SB_OK) return s;
  if (!model->W_h || !model->E || !model->W_out) return SB_E_INVALID_ARG;
  const Layout L = layout_of(*model, *params);
  if (!workspace || ((uintptr_t)workspace % ALIGN) != 0 || bytes < L.total) return SB_E_WORKSPACE;
  sb_decoder *dec = new (std::nothrow) sb_decoder();
  if (!dec) return SB_E_INVALID_ARG;
  s = init_decoder(dec, model, params, workspace, bytes, stream);
  if (s != SB_OK) {
    sb_destroy(dec);
    return s;
  }
  *out = dec;
  return SB_OK;
}

sb_status sb_create_noalloc(const sb_model *model, const sb_params *params, void *stream, sb_decoder **out) {
  if (!out) return SB_E_INVALID_ARG;
  *out = nullptr;
  std::string why;
  sb_status s = check(model, params, &why);
  if (s != SB_OK) {
    set_create_err(why.c_str());
    return s;
  }
  if (!model->W_h || !model->E || !model->W_out) {
    set_create_err("sb_create_noalloc: null weight pointer");
    return SB_E_INVALID_ARG;
  }
  const size_t need = layout_of(*model, *params).total;
  if (need > SB_NOALLOC_SCRATCH_BYTES) {
    char msg[256];
    snprintf(msg, sizeof msg,
             "sb_create_noalloc: these shapes need %zu bytes of workspace; the static scratch holds %zu "
             "(use sb_create with a caller workspace)",
             need, (size_t)SB_NOALLOC_SCRATCH_BYTES);
    set_create_err(msg);
    return SB_E_WORKSPACE;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= NOALLOC_MAX_DEVICES) {
    set_create_err("sb_create_noalloc: no usable current device");
    return SB_E_HIP;
  }
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  NoallocSlot &slot = g_noalloc[dev];
  if (slot.in_use) {
    set_create_err("sb_create_noalloc: a decoder over this GPU's static scratch is still alive");
    return SB_E_STATE;
  }
  if (!slot.ptr) {
    // Once per device, with that device current: the device address of
    // this GPU's copy of the array.
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      char msg[256];
      snprintf(msg, sizeof msg, "sb_create_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      set_create_err(msg);
      return SB_E_HIP;
    }
    slot.ptr = static_cast<unsigned char *>(p);
  }
  sb_decoder *dec = new (slot.obj) sb_decoder();
  dec->noalloc = true;
  slot.in_use = true;
  s = init_decoder(dec, model, params, slot.ptr, SB_NOALLOC_SCRATCH_BYTES, stream);
  if (s != SB_OK) {
    set_create_err(dec->err.empty() ? "sb_create_noalloc: HIP call failed" : dec->err.c_str());
    (void)hipStreamSynchronize(dec->stream);   // nothing enqueued may still write the scratch
    dec->~sb_decoder();
    slot.in_use = false;
    return s;
  }
  *out = dec;
  return SB_OK;
}

sb_status sb_reset(sb_decoder *dec) {
  if (!dec) return SB_E_INVALID_ARG;
  // Earlier submits may still be copying from the pinned length staging.
  HIPCHK(hipStreamSynchronize(dec->stream));
  HIPCHK(launch_init(dec->st, dec->stream));
  dec->n_queued = 0;
  dec->collected = 0;
  return SB_OK;
}

sb_status sb_submit(sb_decoder *dec, int32_t count, const int64_t *ids, const void *h0, const int32_t *L_x,
                    const int32_t *max_len) {
  if (!dec) return SB_E_INVALID_ARG;
  if (count < 0 || (count > 0 && (!h0 || !L_x || !max_len))) {
    dec->err = "sb_submit: bad count or null pointer";
    return SB_E_INVALID_ARG;
  }
  if (count == 0) return SB_OK;
  const sb_params &p = dec->params;
  if ((int64_t)dec->n_queued + count > p.max_inputs) {
    dec->err = "sb_submit: queue capacity exceeded";
    return SB_E_QUEUE_FULL;
  }
  for (int i = 0; i < count; ++i) {
    if (max_len[i] < 1 || max_len[i] > p.max_len_cap) {
      dec->err = "sb_submit: max_len out of [1, max_len_cap]";
      return SB_E_INVALID_ARG;
    }
  }
  const int q0 = dec->n_queued;
  if (dec->ids.size() < (size_t)p.max_inputs) dec->ids.resize(p.max_inputs);
  for (int i = 0; i < count; ++i) dec->ids[q0 + i] = ids ? ids[i] : (int64_t)(q0 + i);
  const size_t es = dec->model.dtype == SB_BF16 ? 2 : 4;
  const size_t rowbytes = (size_t)dec->model.d * es;
  // Lengths go through the pinned staging; a decoder without it (noalloc)
  // copies from the caller's arrays and waits below.
  const int32_t *lx = L_x, *ml = max_len;
  if (dec->pinned_len) {
    int32_t *slx = dec->pinned_len + q0, *sml = dec->pinned_len + p.max_inputs + q0;
    memcpy(slx, L_x, sizeof(int32_t) * count);
    memcpy(sml, max_len, sizeof(int32_t) * count);
    lx = slx;
    ml = sml;
  }
  HIPCHK(hipMemcpyAsync(static_cast<unsigned char *>(dec->st.q_h0) + q0 * rowbytes, h0, count * rowbytes,
                        hipMemcpyDeviceToDevice, dec->stream));
  if (dec->st.rec_i8)
    HIPCHK(launch_row_digits(dec->st, static_cast<unsigned char *>(dec->st.q_h0) + q0 * rowbytes, count,
                             dec->st.q_hd + (size_t)q0 * rec_dig_row_bytes(dec->model.d), dec->st.q_haux + q0, dec->stream));
  HIPCHK(hipMemcpyAsync(dec->st.q_Lx + q0, lx, sizeof(int32_t) * count, hipMemcpyHostToDevice, dec->stream));
  HIPCHK(hipMemcpyAsync(dec->st.q_ml + q0, ml, sizeof(int32_t) * count, hipMemcpyHostToDevice, dec->stream));
  dec->n_queued += count;
  hipLaunchKernelGGL(k_set_queued, dim3(1), dim3(1), 0, dec->stream, dec->st.ctrl, dec->n_queued);
  HIPCHK(hipGetLastError());
  if (!dec->pinned_len) HIPCHK(hipStreamSynchronize(dec->stream));
  return SB_OK;
}

sb_status sb_step(sb_decoder *dec, int32_t *done) {
  if (!dec) return SB_E_INVALID_ARG;
  sb_status s = launch_step(dec, dec->stream);
  if (s != SB_OK) return s;
  if (done) {
    HIPCHK(hipMemcpyAsync(dec->pinned_flag, &dec->st.ctrl->done, sizeof(int32_t), hipMemcpyDeviceToHost,
                          dec->stream));
    HIPCHK(hipStreamSynchronize(dec->stream));
    *done = dec->pinned_flag[0];
  }
  return SB_OK;
}

sb_status sb_run(sb_decoder *dec) {
  if (!dec) return SB_E_INVALID_ARG;
  // Every step either expands a live beam or is the final no-op, and a beam
  // takes at most max_len_cap steps, so this bounds any correct run.
  const int64_t limit = ((int64_t)dec->n_queued + pool_of(dec->params)) * (dec->params.max_len_cap + 1) + 64;
  const bool timed = dec->timing;
  for (int i = 0; i < 2; ++i)   // made here for decoders that allocate nothing at creation
    if (!dec->poll_ev[i]) HIPCHK(hipEventCreateWithFlags(&dec->poll_ev[i], hipEventDisableTiming));
  if (!timed && !dec->graph_exec) {
    sb_status s = capture(dec, &dec->graph, &dec->graph_exec);
    if (s != SB_OK) return s;
  }
  int64_t bursts = 0;
  while (true) {
    const int slot = (int)(bursts & 1);
    if (!timed) {
      HIPCHK(hipGraphLaunch(dec->graph_exec, dec->stream));
    } else {
      for (int i = 0; i < BURST; ++i) {
        sb_status s = launch_timed_step(dec);
        if (s != SB_OK) return s;
      }
    }
    HIPCHK(hipMemcpyAsync(dec->pinned_flag + slot, &dec->st.ctrl->done, sizeof(int32_t),
                          hipMemcpyDeviceToHost, dec->stream));
    HIPCHK(hipEventRecord(dec->poll_ev[slot], dec->stream));
    ++bursts;
    // Poll the previous burst's flag while this burst runs.
    if (bursts >= 2) {
      HIPCHK(hipEventSynchronize(dec->poll_ev[slot ^ 1]));
      if (dec->pinned_flag[slot ^ 1]) break;
    }
    if (bursts * BURST > limit) {
      dec->err = "sb_run: step limit exceeded without completion";
      return SB_E_STATE;
    }
  }
  // Rebuild the tokens of every finished hypothesis in device memory.
  HIPCHK(launch_backtrack(dec->st, dec->collected, dec->n_queued, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  return SB_OK;
}

sb_status sb_collect(sb_decoder *dec, sb_hyp *hyps, int64_t hyp_cap, int32_t *tokens, int64_t tok_cap,
                     int64_t *n_hyps, int64_t *n_tokens) {
  if (!dec || !n_hyps || !n_tokens || hyp_cap < 0 || tok_cap < 0 || (hyp_cap > 0 && !hyps) ||
      (tok_cap > 0 && !tokens))
    return SB_E_INVALID_ARG;
  *n_hyps = 0;
  *n_tokens = 0;
  const int q0 = dec->collected, q1 = dec->n_queued;
  if (q1 <= q0) return SB_OK;
  const int k = dec->params.k, MLC = dec->params.max_len_cap;
  HIPCHK(launch_backtrack(dec->st, q0, q1, dec->stream));
  const int nq = q1 - q0;
  std::vector<int32_t> cnt(nq);
  std::vector<OutHyp> oh((size_t)nq * k);
  HIPCHK(hipMemcpyAsync(cnt.data(), dec->st.o_count + q0, sizeof(int32_t) * nq, hipMemcpyDeviceToHost,
                        dec->stream));
  HIPCHK(hipMemcpyAsync(oh.data(), dec->st.o_hyp + (size_t)q0 * k, sizeof(OutHyp) * nq * k,
                        hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  // Finished prefix and the part of it that fits the buffers.
  int q_end = q0;
  int64_t nh = 0, nt = 0;
  bool truncated = false;
  for (int q = q0; q < q1; ++q) {
    const int c = cnt[q - q0];
    if (c <= 0) break;
    int64_t toks = 0;
    for (int r = 0; r < c; ++r) toks += oh[(size_t)(q - q0) * k + r].length;
    if (nh + c > hyp_cap || nt + toks > tok_cap) {
      truncated = true;
      break;
    }
    nh += c;
    nt += toks;
    q_end = q + 1;
  }
  if (q_end > q0) {
    // Records on the host; the tokens are packed on the device in the same
    // order and copied in one piece (only the tokens the hypotheses hold).
    std::vector<int64_t> off((size_t)(q_end - q0) * k, -1);
    int64_t h = 0, t = 0;
    for (int q = q0; q < q_end; ++q) {
      const int c = cnt[q - q0];
      for (int r = 0; r < c; ++r) {
        const OutHyp &o = oh[(size_t)(q - q0) * k + r];
        sb_hyp &y = hyps[h++];
        y.input = dec->ids[q];
        y.rank = r;
        y.length = o.length;
        y.status = o.status;
        y.finalize_step = o.finalize_step;
        y.score = o.score;
        y.tok_offset = t;
        off[(size_t)(q - q0) * k + r] = t;
        t += o.length;
      }
    }
    HIPCHK(hipMemcpyAsync(dec->st.o_off, off.data(), sizeof(int64_t) * off.size(), hipMemcpyHostToDevice,
                          dec->stream));
    HIPCHK(launch_pack(dec->st, q0, q_end, dec->stream));
    if (t > 0)
      HIPCHK(hipMemcpyAsync(tokens, dec->st.o_pack, sizeof(int32_t) * t, hipMemcpyDeviceToHost, dec->stream));
    HIPCHK(hipStreamSynchronize(dec->stream));
  }
  *n_hyps = nh;
  *n_tokens = nt;
  dec->collected = q_end;
  return truncated ? SB_E_TRUNCATED : SB_OK;
}

sb_status sb_stats(sb_decoder *dec, sb_stats_t *out) {
  if (!dec || !out) return SB_E_INVALID_ARG;
  DevCtrl c;
  HIPCHK(hipMemcpyAsync(&c, dec->st.ctrl, sizeof(DevCtrl), hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  out->timesteps = c.timesteps;
  out->expansions = c.expansions;
  out->noops = c.noops;
  out->refills = c.refills;
  out->admitted = c.admitted;
  out->hyps = c.hyps;
  out->finished = c.finished;
  out->positions = c.positions;
  out->tile_recomputes = c.tile_recomputes;
  return SB_OK;
}

sb_status sb_rows_histogram(sb_decoder *dec, int64_t *counts, int32_t *bucket_width) {
  if (!dec || !counts || !bucket_width) return SB_E_INVALID_ARG;
  DevCtrl c;
  HIPCHK(hipMemcpyAsync(&c, dec->st.ctrl, sizeof(DevCtrl), hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  for (int i = 0; i < 64; ++i) counts[i] = c.rows_hist[i];
  *bucket_width = dec->st.hist_width;
  return SB_OK;
}

sb_status sb_set_timing(sb_decoder *dec, int32_t enable) {
  if (!dec) return SB_E_INVALID_ARG;
  if (enable && dec->tev.empty()) {
    dec->tev.resize(2 * 1024, nullptr);
    // Timing only: no system-scope fences (nothing the host reads depends
    // on them; the done-flag poll keeps its own fenced events).
    for (auto &e : dec->tev) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
  }
  dec->timing = enable != 0;
  dec->tev_used = 0;
  dec->proj_ms = 0.0;
  dec->proj_launches = 0;
  return SB_OK;
}

sb_status sb_timing(sb_decoder *dec, double *proj_ms, int64_t *proj_launches) {
  if (!dec || !proj_ms || !proj_launches) return SB_E_INVALID_ARG;
  HIPCHK(hipStreamSynchronize(dec->stream));
  sb_status s = harvest(dec);
  if (s != SB_OK) return s;
  *proj_ms = dec->proj_ms;
  *proj_launches = dec->proj_launches;
  return SB_OK;
}

sb_status sb_debug_expand(sb_decoder *dec, int32_t R, const void *h_prev, const int32_t *y, const int32_t *t,
                          const int32_t *L_x, void *h_out, double *lse, double *top_lp, int32_t *top_tok) {
  if (!dec) return SB_E_INVALID_ARG;
  const DevState &st = dec->st;
  if (R < 1 || R > st.R_max || !h_prev || !y || !t || !L_x || !h_out || !lse || !top_lp || !top_tok)
    return SB_E_INVALID_ARG;
  if (st.attn) return SB_E_UNSUPPORTED;
  const size_t es = st.dtype == 1 ? 2 : 4;
  const size_t rowbytes = (size_t)st.d * es;
  std::vector<int32_t> src(R);
  for (int r = 0; r < R; ++r) src[r] = r;   // states placed in slots 0..R-1
  HIPCHK(hipMemcpyAsync(st.s_h, h_prev, R * rowbytes, hipMemcpyDeviceToDevice, dec->stream));
  if (st.rec_i8) {
    HIPCHK(launch_row_digits(st, st.s_h, R, st.s_hd, st.s_haux, dec->stream));
    HIPCHK(launch_aux_reset(st.haux, R, dec->stream));
  }
  HIPCHK(hipMemcpyAsync(st.r_hsrc, src.data(), sizeof(int32_t) * R, hipMemcpyHostToDevice, dec->stream));
  HIPCHK(hipMemcpyAsync(st.r_y, y, sizeof(int32_t) * R, hipMemcpyHostToDevice, dec->stream));
  HIPCHK(hipMemcpyAsync(st.r_t, t, sizeof(int32_t) * R, hipMemcpyHostToDevice, dec->stream));
  HIPCHK(hipMemcpyAsync(st.r_Lx, L_x, sizeof(int32_t) * R, hipMemcpyHostToDevice, dec->stream));
  hipLaunchKernelGGL(k_set_rows, dim3(1), dim3(1), 0, dec->stream, st.ctrl, R);
  HIPCHK(hipGetLastError());
  HIPCHK(launch_rec(st, dec->stream));
  HIPCHK(launch_proj(st, dec->stream));
  HIPCHK(launch_rowmerge(st, dec->stream));
  HIPCHK(hipMemcpyAsync(h_out, st.hbuf, R * rowbytes, hipMemcpyDeviceToDevice, dec->stream));
  HIPCHK(hipMemcpyAsync(lse, st.r_lse, sizeof(double) * R, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(top_lp, st.top_lp, sizeof(double) * R * st.k, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(top_tok, st.top_tok, sizeof(int32_t) * R * st.k, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  return sb_reset(dec);
}

sb_status sb_debug_slot(sb_decoder *dec, int32_t beam, int32_t rank, int32_t *status, double *score,
                        int64_t *input, int32_t *steps, int32_t *tokens, int32_t tok_cap, int32_t *n_tokens,
                        uint16_t *kv, int64_t kv_cap) {
  if (!dec || !status || !score || !input || !steps || !n_tokens) return SB_E_INVALID_ARG;
  const DevState &st = dec->st;
  if (beam < 0 || beam >= st.n || rank < 0 || rank >= st.k) return SB_E_INVALID_ARG;
  const int slot = beam * st.k + rank;
  int32_t bin = -1, bst = 0, bpar = 0, sst = 0;
  double ssc = 0.0;
  HIPCHK(hipMemcpyAsync(&bin, st.b_input + beam, 4, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(&bst, st.b_steps + beam, 4, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(&bpar, st.b_par + beam, 4, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(&sst, st.s_status + slot, 4, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipMemcpyAsync(&ssc, st.s_score + slot, 8, hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  *status = bin >= 0 ? sst : SLOT_EMPTY;
  *score = ssc;
  *input = bin;
  *steps = bst;
  *n_tokens = 0;
  if (bin < 0 || sst == SLOT_EMPTY) return SB_OK;
  // Tokens: walk this input's backpointers from level `steps`.
  std::vector<uint32_t> bp((size_t)st.max_len_cap * st.bpw);
  HIPCHK(hipMemcpyAsync(bp.data(), st.bp + (size_t)bin * st.max_len_cap * st.bpw, bp.size() * 4,
                        hipMemcpyDeviceToHost, dec->stream));
  HIPCHK(hipStreamSynchronize(dec->stream));
  std::vector<int32_t> rev;
  int pos = rank;
  for (int lev = bst; lev >= 1; --lev) {
    const uint32_t e = bp[(size_t)(lev - 1) * st.bpw + pos];
    if ((e & 0xFFFFFFu) != BP_NOOP) rev.push_back((int32_t)(e & 0xFFFFFFu));
    pos = (int)(e >> 24);
  }
  *n_tokens = (int32_t)rev.size();
  if (tokens)
    for (int i = 0; i < (int)rev.size() && i < tok_cap; ++i) tokens[i] = rev[rev.size() - 1 - i];
  if (kv && st.kv_layers > 0 && sst == SLOT_ACTIVE && bst > 0) {
    // Rows of levels 0 .. steps-1, found through the slot's ancestor ranks.
    const int planes = st.kv_layers * 2;
    std::vector<uint8_t> anc((size_t)bst);
    HIPCHK(hipMemcpyAsync(anc.data(), st.anc + ((size_t)bpar * st.n * st.k + slot) * st.anc_stride, (size_t)bst,
                          hipMemcpyDeviceToHost, dec->stream));
    HIPCHK(hipStreamSynchronize(dec->stream));
    for (int lev = 0; lev < bst; ++lev)
      if (anc[lev] >= st.k) {
        dec->err = "sb_debug_slot: corrupt KV ancestry";
        return SB_E_STATE;
      }
    for (int pl = 0; pl < planes; ++pl) {
      const int64_t need = (int64_t)(pl + 1) * bst * st.d;
      if (need > kv_cap) break;
      for (int lev = 0; lev < bst; ++lev) {
        const size_t src = ((((size_t)beam * st.max_len_cap + lev) * st.k + anc[lev]) * planes + pl) * st.d;
        HIPCHK(hipMemcpyAsync(kv + ((size_t)pl * bst + lev) * st.d, st.kvs + src, (size_t)st.d * 2,
                              hipMemcpyDeviceToHost, dec->stream));
      }
    }
    HIPCHK(hipStreamSynchronize(dec->stream));
  }
  return SB_OK;
}

sb_status sb_destroy(sb_decoder *dec) {
  if (!dec) return SB_E_INVALID_ARG;
  (void)hipStreamSynchronize(dec->stream);
  for (auto e : dec->tev)
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < 2; ++i)
    if (dec->poll_ev[i]) (void)hipEventDestroy(dec->poll_ev[i]);
  if (dec->pinned_len) (void)hipHostFree(dec->pinned_len);
  if (dec->pinned_flag && dec->pinned_flag != dec->host_flag) (void)hipHostFree(dec->pinned_flag);
  if (dec->graph_exec) (void)hipGraphExecDestroy(dec->graph_exec);
  if (dec->graph) (void)hipGraphDestroy(dec->graph);
  if (dec->cap_stream) (void)hipStreamDestroy(dec->cap_stream);
  if (dec->noalloc) {
    // Static storage: end the object's lifetime and free the GPU's slot.
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    const int dev = dec->device;
    dec->~sb_decoder();
    g_noalloc[dev].in_use = false;
    return SB_OK;
  }
  delete dec;
  return SB_OK;
}

}  // extern "C"
