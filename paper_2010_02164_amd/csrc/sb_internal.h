// Internal device-state layout and kernel launchers of the streambeam library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sb {

enum : int32_t { SLOT_EMPTY = 0, SLOT_ACTIVE = 1, SLOT_EOS = 2, SLOT_MAXLEN = 3 };

// Backpointer entry of the per-beam history table: parent rank in the
// previous beam (bits 24..31) and the emitted token (bits 0..23); a no-op
// expansion of a terminated candidate stores BP_NOOP as its token.
constexpr uint32_t BP_NOOP = 0xFFFFFFu;
constexpr int KMAX_SUPPORTED = 16;

// Exact bf16 recurrence: a state row's bf16 values, scaled by 2^(21 - F),
// as three signed 7-bit digit planes (int8), plus the values of the row too
// small for that window (|x| < 2^(F - 13)), kept as (column, value).
constexpr int REC_HL = 15;
struct RowAux {
  int32_t F;                 // row exponent: every |x| < 2^F
  int32_t n;                 // out-of-window values (> REC_HL: not all kept)
  int32_t col[REC_HL];
  float val[REC_HL];
};
static_assert(sizeof(RowAux) == 128, "RowAux is copied as 8 x 16 bytes");

// Device-side control block: the scheduler state of Alg. 1 and the counters.
struct DevCtrl {
  int32_t n_queued;   // inputs submitted so far
  int32_t cursor;     // next input to admit (Alg. 1's c)
  int32_t R;          // rows (active candidates) expanded this step
  int32_t t_sel;      // smallest 1-based output position among the selected beams
  int32_t live;       // live beams after admission
  int32_t done;       // 1: nothing queued and no beam live
  int32_t n_sel;      // beams selected this step
  int32_t pad0;
  int64_t timesteps, expansions, noops, refills, admitted, hyps, finished;
  int64_t positions;       // output positions t of the expanded rows, summed
  int64_t tile_recomputes; // (row, tile) pairs recomputed by the row merge
  int64_t rows_hist[64];   // timesteps by rows expanded, bucket = R / hist_width
};

// A finalized hypothesis. The beam kernel records where its history ends
// (level = steps taken, rank = position in the final beam); the backtrack
// kernel later walks the backpointers to fill `length` and the tokens.
struct OutHyp {
  double score;
  int32_t length, status, finalize_step, level;
  int32_t pos;         // its backpointer entry at `level` (position in that row)
  int32_t pad;
};

// All device pointers and sizes a kernel may need, passed by value.
struct DevState {
  DevCtrl *ctrl;
  // input queue
  void *q_h0;          // [max_inputs][d]
  int32_t *q_Lx, *q_ml;
  // beams [n] (n = the pool of cached beams)
  int32_t *b_input;    // queue position, -1 = free
  int32_t *b_steps;    // l_t: steps taken
  int32_t *b_sel;      // 1 if expanded this step
  int32_t *b_par;      // which KV buffer holds this beam's state
  int32_t *b_ml;       // max_len of the beam's input
  int32_t *b_nout;     // outputs already finalized (Fairseq rule)
  int32_t *b_order;    // capacity mode: records of the live beams in admission order
  // candidate slots [n*k], slot = beam*k + rank
  int32_t *s_status;
  double *s_score;
  int32_t *s_tok;      // last token (0 for a fresh beam: the start symbol)
  void *s_h;           // [n*k][d] state after consuming the candidate's tokens
  int32_t *s_row;      // row of the slot this step, -1 if not expanded
  uint32_t *bp;        // [max_inputs][max_len_cap][bpw] backpointers, by queue position
  // rows [R_max]: per-row metadata written by the scheduler
  int32_t *r_slot;     // slot of the expanded candidate
  int32_t *r_hsrc;     // state source: >= 0 slot index into s_h, < 0 queue row (-1 - q) of q_h0
  int32_t *r_y;        // last token, consumed by the recurrence
  int32_t *r_t;        // 1-based index of the token being emitted (EOS bias, max length)
  int32_t *r_Lx;       // L_x of the row's input (EOS bias)
  double *r_lse;       // log-sum-exp of the row's logits
  void *hbuf;          // [R_max][d] new states of the expanded rows
  float *part;         // [R_max][S][2 + 2k] per-tile (max, sumexp, top-k vals, top-k ids)
  double *top_lp;      // [R_max][k] log-probs of each row's best k tokens
  int32_t *top_tok;    // [R_max][k]
  // outputs, indexed by queue position
  int32_t *o_count;    // [max_inputs] |Y[i]| (0 = unfinished)
  OutHyp *o_hyp;       // [max_inputs][k]
  int32_t *o_tok;      // [max_inputs][k][max_len_cap]
  int32_t *o_pack;     // [max_inputs * k * max_len_cap] collected tokens, packed back to back
  int64_t *o_off;      // [max_inputs][k] offset of each collected hypothesis in o_pack (-1: none)
  // KV-like state (bf16 bits). The row produced by expanding the candidate
  // at (beam, level, rank) is stored once, at kvs[beam][level][rank]; a
  // candidate's rows are those of its ancestors, whose ranks per level it
  // keeps in anc (two buffers, the beam's parity picks the current one).
  uint16_t *kvs;       // [n][max_len_cap][k][L*2][d]
  uint8_t *anc;        // [2][n*k][anc_stride]: rank of the ancestor at each level
  unsigned char *wkv_t; // W_kv in the fragment order of wout_t: output v = plane*d + o as vocabulary row
  // attention read-out (attn models): projection input x [R_max][d] bf16
  void *xbuf;
  double *attn_part;   // [R_max][L][d] per-layer read-outs a_l
  const void *proj_in; // rows the projection reads: xbuf (attn) or hbuf
  // Exact bf16 recurrence (rec_i8 = 1, bf16, d a multiple of 256, <= 2048): W_h
  // as three signed 7-bit digit planes of W_h[o][i] * 2^(21 - w_exp[o]) in
  // MFMA fragment order, per row the values outside that window, and state
  // rows as digit planes (rec_dig_off) with their RowAux: the new states of the
  // step (hd), the candidate slots (s_hd) and the queued encodings (q_hd).
  int32_t rec_i8;
  int8_t *wd3;         // [d/32][d/32][3 planes][64 lanes][16 bytes]
  int32_t *w_exp;      // [d] smallest e with |W_h[o][i]| < 2^e
  int32_t *w_ln;       // [d + 1] out-of-window values per row; [d]: 1 if a list overflowed
  int32_t *w_li;       // [d][REC_WLIST] their columns
  float *w_lv;         // [d][REC_WLIST] their values
  int32_t *wt_off;     // [d/32][33] the lists of an output tile, concatenated: row starts
  int32_t *wt_col;     // [d/32][REC_WTILE] columns (ascending within a row)
  float *wt_val;       // [d/32][REC_WTILE] values
  int8_t *hd, *s_hd, *q_hd;     // [rows][4d bytes]: digit (k, a) at rec_dig_off(k, a)
  RowAux *haux, *s_haux, *q_haux;
  // fp32 W_h in the recurrence's A-fragment order: [d/32][d/8][64 lanes][16 B],
  // lane (h, l) of output tile vt at K step s holding W_h[32 vt + l][8 s + 4h .. +3]
  // bf16 W_h likewise for the fp64 recurrence: [d/32][d/16][2 row halves][64 lanes][8 B],
  // lane (g, l) of half x at K step s holding W_h[32 vt + 16 x + l][16 s + 4g .. +3]
  const float4 *wh_t;
  const uint2 *wh16_t;
  // model
  const void *W_h, *E, *W_out;
  // W_out re-laid out tile-contiguous: [S][nk][128 rows][128 bytes], one
  // 16 KB block per (128-row vocabulary tile, 128-byte K chunk); rows >= V
  // are zero.
  unsigned char *wout_t;
  // sizes and parameters
  int32_t n, k, d, V, M, max_len_cap, refill_thr, S, R_max, dtype, kv_layers, max_inputs;
  int32_t attn;        // 1: projection input = h + layer-mean attention read-out
  int32_t anc_stride;  // bytes per slot of anc: max_len_cap rounded up to 4
  int32_t kbucket;     // top-k list length used by the kernels: 4, 8 or 16 (>= k)
  int32_t tile_keys;   // keys per (row, vocabulary tile) partial record: 4 or kbucket
  int32_t hist_width;  // rows per bucket of DevCtrl::rows_hist
  int32_t n_cu;        // compute units of the device (persistent launches)
  int32_t select_all;  // 1: expand every live beam (Var-Str-FIFO), 0: minimal l_t only
  int32_t cap;         // 1: capacity-constrained selection (row_budget rows, (l_t, admission) order)
  int32_t row_budget;  // rows a timestep may expand (batch size times k)
  int32_t rule;        // finalization rule: 0 paper (App. A.1), 1 Fairseq
  int32_t bpw;         // backpointer entries per level: k (paper), 2k (Fairseq: beam + outputs)
  double delta;
  float beta;
};

// Out-of-window values kept per W_h row by the exact bf16 recurrence, and
// per tile of 32 rows; a W_h with more uses the fp64 recurrence.
constexpr int REC_WLIST = 16;
constexpr int REC_WTILE = 64;

// A state row's digit planes, 128 bytes per 32 values: for value k and
// plane a, byte 48 ((k / 16) % 2) + 16 a + k % 16 of block k / 32 (the last
// 32 bytes of a block unused), so that one lane's three 16-byte MFMA
// operands lie together and a block is one 128-byte line.
__host__ __device__ constexpr int rec_dig_off(int k, int a) { return (k >> 5) * 128 + ((k >> 4) & 1) * 48 + a * 16 + (k & 15); }
constexpr size_t rec_dig_row_bytes(size_t d) { return 4 * d; }

// Tile sizes of the projection/recurrence GEMMs.
constexpr int GEMM_BV = 128;   // out features (vocab / hidden) per workgroup
constexpr int GEMM_BR = 64;    // batch rows per workgroup

inline int proj_tiles(int V) { return (V + GEMM_BV - 1) / GEMM_BV; }

// Launchers (each returns the launch status).
hipError_t launch_sched(const DevState &st, hipStream_t s);
hipError_t launch_rec(const DevState &st, hipStream_t s);
hipError_t launch_relayout_wh(const DevState &st, hipStream_t s);
hipError_t launch_rec_prepare(const DevState &st, hipStream_t s);
hipError_t launch_row_digits(const DevState &st, const void *rows, int count, int8_t *dig, RowAux *aux, hipStream_t s);
hipError_t launch_aux_reset(RowAux *aux, int count, hipStream_t s);
hipError_t launch_proj(const DevState &st, hipStream_t s);
hipError_t launch_rowmerge(const DevState &st, hipStream_t s);
hipError_t launch_beam(const DevState &st, hipStream_t s);
hipError_t launch_kv_append(const DevState &st, hipStream_t s);
hipError_t launch_attn(const DevState &st, hipStream_t s);
hipError_t launch_backtrack(const DevState &st, int q0, int q1, hipStream_t s);
hipError_t launch_pack(const DevState &st, int q0, int q1, hipStream_t s);
hipError_t launch_init(const DevState &st, hipStream_t s);
hipError_t launch_relayout_wout(const DevState &st, hipStream_t s);
hipError_t launch_relayout_wkv(const DevState &st, const uint16_t *W_kv, hipStream_t s);

}  // namespace sb
