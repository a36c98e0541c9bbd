// Where one workgroup's work lives: its sequence, lengths, tensor rows and
// window, for fixed-length and ragged batches alike.
//
// Grids run over (block row) x (unit) x (head group): in a fixed-length batch
// the row is the block within the sequence and unit = b H_k + h_k; in a ragged
// batch the row is the block over the whole batch (sequence b's blocks follow
// those of b - 1) and unit = h_k, the sequence coming from the block-to-
// sequence map of the schedule.
#pragma once

#include "internal.h"
#include "window_rule.h"

namespace cowa {

struct SeqCtx {
  int32_t b;         // sequence
  int32_t tile;      // block within the sequence
  int32_t n_q, n_k;  // its lengths
  int64_t q0, qh;    // row (of d elements) of query 0 of QO head 0; + qh per QO head (Q, O, dO, dQ, LSE, D)
  int64_t k0, kh;    // row of key 0 of KV head 0; + kh per KV head (K, V, dK, dV)
  int32_t sched;     // schedule row (QO side) or column (KV side) of (h_k, block)
  Geo32 g;           // window of (b, h_k), bounds clamped to n_k
};

// Units of the grid: B H_k for fixed lengths, H_k for a ragged batch.
__host__ __device__ inline int grid_units(const cowa_params& p, const SchedView& sv) {
  return sv.ragged ? p.h_k : p.batch * p.h_k;
}

// qside: the row counts QO blocks (forward, dQ pass), else KV blocks (dK/dV pass).
__device__ inline SeqCtx seq_ctx(const cowa_params& p, const SchedView& sv, int row, int unit, bool qside,
                                 int& hk) {
  SeqCtx c;
  const WinDesc* wd;
  if (!sv.ragged) {
    c.b = unit / p.h_k;
    hk = unit % p.h_k;
    c.tile = row;
    c.n_q = p.n_q;
    c.n_k = p.n_k;
    c.q0 = (int64_t)c.b * p.h_q * p.n_q;
    c.qh = p.n_q;
    c.k0 = (int64_t)c.b * p.h_k * p.n_k;
    c.kh = p.n_k;
    wd = sv.win + hk;
  } else {
    hk = unit;
    c.b = (qside ? sv.qt_seq : sv.kt_seq)[row];
    const SeqDesc sd = sv.seq[c.b];
    c.tile = row - (qside ? sd.qt_off : sd.kt_off);
    c.n_q = sd.n_q;
    c.n_k = sd.n_k;
    c.q0 = sd.q_start;
    c.qh = p.n_q;
    c.k0 = sd.k_start;
    c.kh = p.n_k;
    wd = sv.win + (sv.per_seq_win ? c.b * p.h_k : 0) + hk;
  }
  c.sched = hk * (qside ? sv.n_qt : sv.n_kt) + row;
  const WinDesc w = *wd;
  c.g.off = c.n_k - c.n_q;
  c.g.w_near = w.near < c.n_k ? w.near : c.n_k;
  c.g.w_sink = w.sink < c.n_k ? w.sink : c.n_k;
  c.g.lo = w.lo < c.n_k ? w.lo : c.n_k;
  c.g.hi = w.hi < c.n_k ? w.hi : c.n_k;
  c.g.n_q = c.n_q;
  c.g.n_k = c.n_k;
  return c;
}

}  // namespace cowa
