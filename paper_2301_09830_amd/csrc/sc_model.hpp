// Host-side model behind selective stage compression (Sec. 7).
//
// With pipeline parallelism the stages finish their backward passes at
// different times: the later stages finish first and start their
// data-parallel gradient exchange while the earlier stages still compute, so
// the exchange of the earliest stage is the one left exposed at the end of
// the iteration.  Sec. 7 compresses the exchange of a selected set of stages,
// starting from the earliest, each choice moving the bottleneck to the next
// stage.  Two pieces:
//
//   pipeline_1f1b  event simulation of the one-forward-one-backward schedule
//                  (Sec. 2.2) on S uniform stages: when each stage's last
//                  backward pass ends (the paper trains with the interleaved
//                  form of this schedule, Sec. 8, in which the devices finish
//                  in the same order: the backward of the last micro-batch
//                  still ends on the later devices first);
//   sc_select      given each stage's backward end, its exchange time
//                  uncompressed and compressed and its compression time (the
//                  measured time of the compressor on the stage's matrices),
//                  compress the current bottleneck stage while that shortens
//                  it and the budget allows.
#pragma once

#include <cmath>
#include <cstdint>
#include <vector>

namespace occ {

// Schedule of one stage under 1F1B: `warm` forward passes, then alternating
// forward/backward, then the remaining backward passes.
struct PipeOp {
  bool fwd;
  int mb;   // micro-batch
};

inline std::vector<PipeOp> one_f_one_b_order(int S, int m, int s) {
  const int warm = std::min(S - s - 1, m);
  std::vector<PipeOp> ops;
  ops.reserve(2 * (size_t)m);
  for (int i = 0; i < warm; ++i) ops.push_back({true, i});
  for (int i = 0; i < m - warm; ++i) {
    ops.push_back({true, warm + i});
    ops.push_back({false, i});
  }
  for (int i = m - warm; i < m; ++i) ops.push_back({false, i});
  return ops;
}

// Simulates the schedule: an operation starts when its stage is free and its
// input has arrived (forward of micro-batch i on stage s after stage s - 1's,
// backward after stage s + 1's, each hop taking t_p2p); a forward takes t_fwd
// and a backward t_bwd.  bwd_done[s] = end of stage s's last operation (its
// last backward pass).  Returns false if the schedule cannot complete (it
// always can for valid arguments).
inline bool pipeline_1f1b(int S, int m, double F, double B, double p, double* bwd_done,
                          double* t_end) {
  std::vector<std::vector<PipeOp>> ops(S);
  std::vector<std::vector<double>> f_end(S, std::vector<double>(m, -1.0)),
      b_end(S, std::vector<double>(m, -1.0));
  for (int s = 0; s < S; ++s) ops[s] = one_f_one_b_order(S, m, s);
  std::vector<size_t> next(S, 0);
  std::vector<double> free_at(S, 0.0);
  size_t left = 2 * (size_t)m * S;
  while (left > 0) {
    bool progress = false;
    for (int s = 0; s < S; ++s) {
      while (next[s] < ops[s].size()) {
        const PipeOp op = ops[s][next[s]];
        double ready;
        if (op.fwd) {
          if (s == 0) ready = 0.0;
          else if (f_end[s - 1][op.mb] < 0) break;
          else ready = f_end[s - 1][op.mb] + p;
        } else {
          if (s == S - 1) {
            if (f_end[s][op.mb] < 0) break;
            ready = f_end[s][op.mb];
          } else if (b_end[s + 1][op.mb] < 0) {
            break;
          } else {
            ready = b_end[s + 1][op.mb] + p;
          }
        }
        const double start = std::max(ready, free_at[s]);
        const double end = start + (op.fwd ? F : B);
        (op.fwd ? f_end : b_end)[s][op.mb] = end;
        free_at[s] = end;
        ++next[s];
        --left;
        progress = true;
      }
    }
    if (!progress) return false;
  }
  double last = 0.0;
  for (int s = 0; s < S; ++s) {
    bwd_done[s] = free_at[s];
    last = std::max(last, free_at[s]);
  }
  if (t_end) *t_end = last;
  return true;
}

struct StageTimes {
  double bwd_done, comm, comm_compressed, compress;
};

inline double stage_end(const StageTimes& t, bool compressed) {
  return t.bwd_done + (compressed ? t.compress + t.comm_compressed : t.comm);
}

// Greedy bottleneck selection: starting with no stage compressed, while fewer
// than max_compressed stages are compressed, take the stage whose exchange
// ends last (the earliest stage among equal ends); if it is already
// compressed, or compressing it does not end its exchange earlier, stop;
// otherwise compress it.  Returns the end of the last exchange, which is the
// least last end any choice of at most max_compressed stages reaches: a
// stopping bottleneck cannot end earlier under any choice, and while it is
// uncompressed the stages with later uncompressed ends are compressed
// already.
inline double sc_select(const StageTimes* st, int S, int max_compressed, uint8_t* selected,
                        int* n_selected) {
  for (int s = 0; s < S; ++s) selected[s] = 0;
  int k = 0;
  for (;;) {
    int bot = 0;
    double worst = stage_end(st[0], selected[0]);
    for (int s = 1; s < S; ++s) {
      const double e = stage_end(st[s], selected[s]);
      if (e > worst) {
        worst = e;
        bot = s;
      }
    }
    if (k >= max_compressed || selected[bot] || !(stage_end(st[bot], true) < worst)) {
      if (n_selected) *n_selected = k;
      return worst;
    }
    selected[bot] = 1;
    ++k;
  }
}

}  // namespace occ
