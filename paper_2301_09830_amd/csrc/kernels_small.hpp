// Fused small-rank path of liboptcc (padded rank RP <= 16): helpers, the
// orthogonalisation factor, the finishing kernel and the reconstruction pass.
//
// One power-iteration round is three launches; kernel boundaries are the
// only device-wide synchronisation (an agent-scope release fence in every
// block of a streaming kernel writes back the XCD's L2 and costs more than a
// launch):
//   k_pm     left product P = A Q on the matrix cores (kernels_mfma16.hpp);
//            each block owns whole rows, so it stores final rows of P and
//            their fp64 Gram partial.
//   k_qm     right product partials Q' = A^T P on the raw P over row splits
//            (fp64 matrix cores, kernels_mfma16.hpp); its first block per
//            matrix sums the Gram partials, runs the Cholesky G = R^T R
//            (CholeskyQR first pass; the second only when the first found the
//            Gram badly conditioned) and stores T = R^-1, so that P_hat = P T
//            and A^T P_hat = Q' T.
//   k_qfin16 Q = (sum of the split partials) T and P_hat = P T.
// and after the last round
//   k_mh16   reconstruction and residual, M_hat = P_hat Q^T and
//            err = A - M_hat (matrix cores, kernels_mfma16.hpp).
#pragma once

#include "kernels.hpp"

namespace occ {

// -------------------------------------------------------------------------
// A = M + err_prev in 4-column chunks, split into "issue" and "value" so that
// loads of the next sub-tile can be in flight while the current one is used.
// -------------------------------------------------------------------------
template <int DT> struct MVec { using T = float4; };
template <> struct MVec<DT_BF16> { using T = uint2; };

template <int DT>
struct AChunk {
  typename MVec<DT>::T m;
  float4 e;
};

template <int DT>
__device__ __forceinline__ typename MVec<DT>::T neg_zero_m() {
  if constexpr (DT == DT_F32) return make_float4(-0.f, -0.f, -0.f, -0.f);
  else return make_uint2(0x80008000u, 0x80008000u);
}

// Fast path: whole chunk in bounds and VEC layout; otherwise the exact
// element-wise A is stored in `e` and `m` holds -0 (x + -0 == x for all x).
template <int DT, bool VEC, bool RM = false>
__device__ __forceinline__ void chunk_issue(const Desc& d, int row, int col, int c_hi,
                                            AChunk<DT>& x) {
  if (VEC && row < d.m && col + 4 <= c_hi) {
    const int64_t pr = prow<RM>(d, row);
    const int64_t mo = pr * d.ldm + col;
    x.m = *(const typename MVec<DT>::T*)((const char*)d.M + mo * (DT == DT_F32 ? 4 : 2));
    x.e = d.err_in ? *(const float4*)(d.err_in + pr * d.lde_in + col)
                   : make_float4(-0.f, -0.f, -0.f, -0.f);
  } else {
    float a[4];
    load_a4<DT, false, RM>(d, row, col, c_hi, a);
    x.m = neg_zero_m<DT>();
    x.e = make_float4(a[0], a[1], a[2], a[3]);
  }
}

template <int DT>
__device__ __forceinline__ void chunk_value(const AChunk<DT>& x, float a[4]) {
  if constexpr (DT == DT_F32) {
    a[0] = x.m.x + x.e.x; a[1] = x.m.y + x.e.y; a[2] = x.m.z + x.e.z; a[3] = x.m.w + x.e.w;
  } else {
    a[0] = bf16_lo(x.m.x) + x.e.x;
    a[1] = bf16_hi(x.m.x) + x.e.y;
    a[2] = bf16_lo(x.m.y) + x.e.z;
    a[3] = bf16_hi(x.m.y) + x.e.w;
  }
}

// Source of the warm-start or previous round's Q: the caller's Q when
// rank == RP (same layout), else the padded workspace copy.
template <int RP>
__device__ __forceinline__ const float* q_src(const Desc& d) { return d.r == RP ? d.Q : d.qpad; }

// Packed upper triangle of an RP x RP symmetric matrix: entry p < NP
// (NP = RP (RP + 1) / 2) is (k, l) with k <= l, row by row.
template <int RP>
__device__ __forceinline__ void upper_entry(int p, int& k, int& l) {
  int kk = 0, rem = p;
  while (rem >= RP - kk) { rem -= RP - kk; ++kk; }
  k = kk;
  l = kk + rem;
}

// -------------------------------------------------------------------------
// Orthogonalisation of the small-rank path (Sec. 2.3 CholeskyQR; the second
// pass only when the first lost orthogonality).  P_hat = P T with
// T = R1^-1 (R2^-1), so A^T P_hat = (A^T P) T: the right product runs on the
// raw P, and T is formed by one block per matrix that runs beside it (the
// first blocks of k_qm): Gram = sum of the row-block partials (slice
// (entry, group) per thread pair, loads in flight, slices added in LDS in
// order), Cholesky by wave 0 with one matrix entry per lane slot, T stored
// to d.t1.  k_qfin16 then applies T to the summed right-product partials
// and to P.  The chain Gram -> Cholesky -> T thus overlaps the streaming
// pass instead of running between the two products.
// -------------------------------------------------------------------------
constexpr int CH_SLICES_MAX = 1024;  // thread pairs the Gram sum is sliced for (fixes its order)
constexpr int CH_CHUNK = 256;     // rows per chunk of the second-pass Gram
constexpr int CH_BATCH = 20;      // partial loads in flight per thread

struct CholSmem {
  double part[8][16 * 17 / 2];
  double G[16 * 16];
  double R[2][16 * 16];       // factors of the two passes (upper triangle, row-major)
  double inv[2][16];          // 1 / R[k][k], zero for a dependent column
  double rows[CH_CHUNK * 16];
  double T[16 * 16];          // P_hat = P T (row-major)
  uint32_t need;
};

// 1/sqrt(v) for v > 0: hardware estimate refined by two Newton steps
// (y <- y + y (1 - v y^2) / 2), accurate to an ulp or two.
__device__ __forceinline__ double rsqrt_nr(double v) {
  double y = __builtin_amdgcn_rsq(v);
  double e = fma(-v * y, y, 1.0);
  y = fma(0.5 * y, e, y);
  e = fma(-v * y, y, 1.0);
  return fma(0.5 * y, e, y);
}

struct CholInfo {
  uint32_t defmask;   // dependent columns
  double pmax, pmin;  // extreme pivots (squared diagonal of R) over independent columns
};

// Cholesky G = R^T R of the leading RP x RP block of the symmetric G (LDS,
// row-major), by one wave; R (upper triangle, zero below) and the inverse
// diagonal go to LDS.  Right-looking on the upper triangle: lane slot
// (lane, q) owns entry e = lane + 64 q = (i, j) of the Schur complement; at
// step k every slot reads the pivot and its two row-k factors straight from
// the registers of the lanes owning row k (cross-lane shuffles: row k is
// slot k RP / 64 of lanes k RP % 64 .. + RP - 1), and entries with
// k < i <= j are updated.  Columns >= r
// are padding; a pivot <= kPivotTol * max diag(G) marks its column
// dependent: that row of R is the unit row, its inverse diagonal is zero (the
// column of P_hat is zero) and later steps ignore it.  NaN pivots are not
// dependent: they propagate like the data.
template <int RP>
__device__ __forceinline__ CholInfo chol_lanes(const double* G, int r, double* R, double* inv,
                                              uint32_t* flags) {
  static_assert(64 % RP == 0, "a row of the Schur complement lies in one slot");
  constexpr int NE = (RP * RP + kWave - 1) / kWave;
  const int lane = threadIdx.x & 63;
  double w[NE];
  int ei[NE], ej[NE];
  bool up[NE];
#pragma unroll
  for (int q = 0; q < NE; ++q) {
    const int e = lane + kWave * q;
    ei[q] = e / RP;
    ej[q] = e % RP;
    up[q] = e < RP * RP && ei[q] <= ej[q];
    w[q] = up[q] ? G[e] : 0.0;
  }
  double maxdiag = 0.0;
  bool nonfinite = false;
#pragma unroll
  for (int k = 0; k < RP; ++k) {
    const double gkk = G[k * RP + k];
    nonfinite = nonfinite || !isfinite(gkk);
    maxdiag = gkk > maxdiag ? gkk : maxdiag;
  }
  const double thr = kPivotTol * maxdiag;
  CholInfo o;
  o.defmask = 0;
  o.pmax = 0.0;
  o.pmin = 1e308;
#pragma unroll
  for (int k = 0; k < RP; ++k) {
    // entry (k, x) of the Schur complement: slot k RP / 64 of lane k RP % 64 + x
    const double wk = w[(k * RP) / kWave];
    const int base = (k * RP) % kWave;
    const double piv = __shfl(wk, base + k);
    double ri[NE], rj[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      ri[q] = __shfl(wk, base + (ei[q] < RP ? ei[q] : 0));
      rj[q] = __shfl(wk, base + ej[q]);
    }
    const bool dep = (k >= r) || (piv <= thr);
    o.defmask |= dep ? (1u << k) : 0u;
    if (!dep) {
      o.pmax = piv > o.pmax ? piv : o.pmax;
      o.pmin = piv < o.pmin ? piv : o.pmin;
    }
    const double ik = dep ? 0.0 : rsqrt_nr(piv);
    if (lane == 0) inv[k] = ik;
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      if (up[q] && ei[q] == k)
        R[k * RP + ej[q]] = (ej[q] == k) ? (dep ? 1.0 : piv * ik) : (dep ? 0.0 : w[q] * ik);
      if (!dep && up[q] && ei[q] > k) w[q] = fma(-(ri[q] * ik), rj[q] * ik, w[q]);
    }
  }
#pragma unroll
  for (int q = 0; q < NE; ++q) {
    const int e = lane + kWave * q;
    if (e < RP * RP && ei[q] > ej[q]) R[e] = 0.0;
  }
  const uint32_t live = r >= 32 ? 0xffffffffu : ((1u << r) - 1u);
  if (lane == 0 && flags) {
    if (nonfinite) atomicOr(flags, FLAG_NONFINITE);
    if (o.defmask & live) atomicOr(flags, FLAG_RANK_DEFICIENT);
  }
  return o;
}

// The first pass lost orthogonality when diag(R) spans more than
// kSecondPassCond, i.e. the pivots span more than its square.
__device__ __forceinline__ uint32_t needs_second_pass(const CholInfo& o) {
  return (o.pmax > 0.0 && o.pmax > kSecondPassCond * kSecondPassCond * o.pmin) ? 1u : 0u;
}

// x <- x R^-1 for one row (forward substitution, fp64), R upper triangular
// with inverse diagonal inv (zero for a dependent column, which zeroes it).
template <int RP>
__device__ __forceinline__ void solve_row(double* x, const double* R, const double* inv) {
#pragma unroll
  for (int j = 0; j < RP; ++j) {
    // one column of R in flight at a time: hoisting all of its LDS reads out
    // of the loop would take about 270 VGPRs
    asm volatile("" ::: "memory");
    double v = x[j];
#pragma unroll
    for (int k = 0; k < j; ++k) v = fma(-x[k], R[k * RP + j], v);
    x[j] = v * inv[j];
  }
}

// Gram (upper triangle, fp64) of `nsrc` stacked packed partials, by NT
// threads; result (full symmetric) in G.  The partials are cut into NG
// consecutive slices, each summed in order, and the slices are added in
// order (NG depends on the rank only, so the sum does not depend on NT).
template <int RP, int NT>
__device__ __forceinline__ void gram_sum_all(const double* src, int nsrc, CholSmem& sm, double* G) {
  constexpr int NP = RP * (RP + 1) / 2;
  constexpr int NG = CH_SLICES_MAX / NP < 8 ? CH_SLICES_MAX / NP : 8;
  static_assert(NP <= NT, "one thread per entry for the slice sum");
  const int t = threadIdx.x;
  for (int pr = t; pr < NG * NP; pr += NT) {
    const int p = pr % NP, q = pr / NP;
    const int per = (nsrc + NG - 1) / NG;
    const int g0 = min(nsrc, q * per), g1 = min(nsrc, g0 + per);
    double s = 0.0;
    for (int gb = g0; gb < g1; gb += CH_BATCH) {
      double v[CH_BATCH];
#pragma unroll
      for (int u = 0; u < CH_BATCH; ++u) v[u] = (gb + u < g1) ? src[(int64_t)(gb + u) * NP + p] : 0.0;
#pragma unroll
      for (int u = 0; u < CH_BATCH; ++u)
        if (gb + u < g1) s = (gb + u == g0) ? v[u] : s + v[u];
    }
    sm.part[q][p] = s;
  }
  __syncthreads();
  if (t < NP) {
    double s = sm.part[0][t];
    for (int qq = 1; qq < NG; ++qq) s += sm.part[qq][t];
    int k, l;
    upper_entry<RP>(t, k, l);
    G[k * RP + l] = s;
    G[l * RP + k] = s;
  }
  __syncthreads();
}

// Row of P (fp64) from the unorthogonalised P.
template <int RP>
__device__ __forceinline__ void p_row(const Desc& d, int64_t row, double* x) {
#pragma unroll
  for (int k = 0; k < RP; k += 4) {
    const float4 v = *(const float4*)(d.praw + row * RP + k);
    x[k] = v.x; x[k + 1] = v.y; x[k + 2] = v.z; x[k + 3] = v.w;
  }
}

// T of one matrix by one block of NT threads (see above); also stores the
// second-pass decision (d.info[0]) and the numeric flags.
template <int RP, int NT>
__device__ __forceinline__ void orth_t_body(const Desc& d, uint32_t* flags, CholSmem& sm) {
  const int t = threadIdx.x;
  gram_sum_all<RP, NT>(d.gpart, d.ng, sm, sm.G);
  if (t < kWave) {
    const CholInfo o = chol_lanes<RP>(sm.G, d.r, sm.R[0], sm.inv[0], flags);
    const uint32_t need = needs_second_pass(o);
    if (t == 0) {
      d.info[0] = need;
      sm.need = need;
    }
  }
  __syncthreads();
  const uint32_t need = sm.need;
  if (need) {
    // Second pass: Gram of P_hat1 = P R1^-1 (fp64) over all rows, in chunks.
    constexpr int NP = RP * (RP + 1) / 2;
    constexpr int NG = NT / NP < 8 ? NT / NP : 8;
    static_assert(CH_CHUNK <= NT, "one row of a chunk per thread");
    const int p = t % NP, q = t / NP;
    int pk_, pl_;
    upper_entry<RP>(p, pk_, pl_);
    double acc = 0.0;
    const int per = (CH_CHUNK + NG - 1) / NG;
    for (int c0 = 0; c0 < d.m; c0 += CH_CHUNK) {
      if (t < CH_CHUNK) {
        const int row = c0 + t;
        double v[RP];
#pragma unroll
        for (int k = 0; k < RP; ++k) v[k] = 0.0;
        if (row < d.m) {
          p_row<RP>(d, row, v);
          solve_row<RP>(v, sm.R[0], sm.inv[0]);
        }
#pragma unroll
        for (int k = 0; k < RP; ++k) sm.rows[t * RP + k] = v[k];
      }
      __syncthreads();
      if (q < NG) {
        const int i0 = min(CH_CHUNK, q * per), i1 = min(CH_CHUNK, i0 + per);
        for (int i = i0; i < i1; ++i) acc = fma(sm.rows[i * RP + pk_], sm.rows[i * RP + pl_], acc);
      }
      __syncthreads();
    }
    if (q < NG) sm.part[q][p] = acc;
    __syncthreads();
    if (t < NP) {
      double sacc = sm.part[0][t];
      for (int qq = 1; qq < NG; ++qq) sacc += sm.part[qq][t];
      sm.G[pk_ * RP + pl_] = sacc;
      sm.G[pl_ * RP + pk_] = sacc;
    }
    __syncthreads();
    if (t < kWave) chol_lanes<RP>(sm.G, d.r, sm.R[1], sm.inv[1], flags);
    __syncthreads();
  }
  // The substitution x -> x R1^-1 (R2^-1) is linear, so P_hat = P T with row
  // i of T the image of the unit row e_i (upper triangular; a dependent
  // column's inverse diagonal is zero, so its column of T is zero).
  if (t < RP) {
    double x[RP];
#pragma unroll
    for (int k = 0; k < RP; ++k) x[k] = (k == t) ? 1.0 : 0.0;
    solve_row<RP>(x, sm.R[0], sm.inv[0]);
    if (need) solve_row<RP>(x, sm.R[1], sm.inv[1]);
#pragma unroll
    for (int k = 0; k < RP; ++k) d.t1[t * RP + k] = x[k];
  }
}

// -------------------------------------------------------------------------
// k_qfin16: the factor T applied.  Blocks [0, nq) (kind K_QRED): for
// kBlock / (S RP) columns c each, Q'[c][k] = sum over the sq row splits of
// the fp64 qpart[s][c][k] -- S = qfin_slices(sq) threads per element each
// summing a consecutive slice of the splits in order, the slices then added
// in order -- then Q[c][j] = sum_k Q'[c][k] T[k][j] (fp64, k ascending),
// written to the caller's Q and the padded copy.
// Blocks [nq, ...) (kind K_APPLY): for kBlock / (RP / 4) rows each,
// P_hat[i][j] = sum_k P[i][k] T[k][j] (fp64, k ascending), four columns j per
// thread, written to the caller's P and the padded copy.
// -------------------------------------------------------------------------
template <int RP>
__device__ __forceinline__ void load_t(const Desc& d, double* Ts) {
  for (int e = threadIdx.x; e < RP * RP; e += kBlock) Ts[e] = d.t1[e];
}

template <int RP>
__device__ __forceinline__ void qfin_q_body(const Desc& d, int b, double* Ts, double* qs,
                                            double* part) {
  const int S = qfin_slices(d.sq);
  const int t = threadIdx.x, o = t / S, sl = t % S;   // element o of the block, slice sl
  const int cl = o / RP, k = o % RP;
  load_t<RP>(d, Ts);
  const double* qp = (const double*)d.qpart;
  const int64_t c = (int64_t)b * (kBlock / (S * RP)) + cl;
  const int64_t idx = c * RP + k;
  const int per = (d.sq + S - 1) / S;
  const int s0 = min(d.sq, sl * per), s1 = min(d.sq, s0 + per);
  double acc = 0.0;
  if (c < d.n) {
    for (int t0 = s0; t0 < s1; t0 += 16) {
      double v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = (t0 + u < s1) ? qp[(int64_t)(t0 + u) * d.n * RP + idx] : 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (t0 + u < s1) acc = (t0 + u == s0) ? v[u] : acc + v[u];
    }
  }
  part[t] = acc;
  __syncthreads();
  if (sl == 0) {
    double q = part[t];
    for (int x = 1; x < S; ++x) q = q + part[t + x];
    qs[o] = q;
  }
  __syncthreads();
  if (sl != 0 || c >= d.n) return;
  double q = 0.0;
#pragma unroll
  for (int kk = 0; kk < RP; ++kk) q = fma(qs[cl * RP + kk], Ts[kk * RP + k], q);
  const float v = (float)q;
  d.qpad[idx] = v;   // always: the next left product and the reconstruction read the padded copy
  if (k < d.r) d.Q[c * d.r + k] = v;
}

template <int RP>
__device__ __forceinline__ void qfin_p_body(const Desc& d, int b, double* Ts) {
  constexpr int TPR = RP / 4;               // threads per row
  constexpr int RPB = kBlock / TPR;
  const int t = threadIdx.x, j0 = 4 * (t % TPR);
  load_t<RP>(d, Ts);
  __syncthreads();
  const int64_t row = (int64_t)b * RPB + t / TPR;
  if (row >= d.m) return;
  double x[RP];
  p_row<RP>(d, row, x);
  float out[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < RP; ++k) acc = fma(x[k], Ts[k * RP + j0 + q], acc);
    out[q] = (float)acc;
  }
  // the padded copy is always written: the reconstruction pass reads it
  // with 16-byte loads (the caller's P has no alignment guarantee)
  *(float4*)(d.phat + row * RP + j0) = make_float4(out[0], out[1], out[2], out[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (j0 + q < d.r) d.P[row * d.r + j0 + q] = out[q];
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qfin16(OCC_KARGS, int nq) {
  __shared__ double Ts[RP * RP];
  __shared__ double qs[kBlock];
  __shared__ double part[kBlock];
  const int b = (int)blockIdx.x;
  if (b < nq) {
#define B_(d, bb) qfin_q_body<RP>(d, bb, Ts, qs, part)
    OCC_DISPATCH_AT(K_QRED, B_, b)
#undef B_
  } else {
#define B_(d, bb) qfin_p_body<RP>(d, bb, Ts)
    OCC_DISPATCH_AT(K_APPLY, B_, b - nq)
#undef B_
  }
}

}  // namespace occ
