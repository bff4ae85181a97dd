// Fused small-rank path of liboptcc (padded rank RP <= 16): helpers, the
// Cholesky, P_hat and Q-reduction kernels and the reconstruction pass.
//
// One power-iteration round is four launches; kernel boundaries are the only
// device-wide synchronisation on the streaming passes (an agent-scope
// release fence in every block of a streaming kernel writes back the XCD's
// L2 and costs more than a launch):
//   k_pm     left product P = A Q on the matrix cores (kernels_mfma16.hpp);
//            each block owns whole rows, so it stores final rows of P and
//            their fp64 Gram partial.
//   k_orth16 every block sums the Gram partials and runs the Cholesky
//            factorisation (CholeskyQR first pass; the second pass only when
//            the first found the Gram badly conditioned) -- the same
//            deterministic computation in each block, so no hand-off is
//            needed -- then forms P_hat = P T for its own 128 rows.
//   k_qm     right product partials A^T P_hat over row splits (matrix cores).
//   k_qred16 Q = sum of the row-split partials.
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
template <int DT, bool VEC>
__device__ __forceinline__ void chunk_issue(const Desc& d, int row, int col, int c_hi,
                                            AChunk<DT>& x) {
  if (VEC && row < d.m && col + 4 <= c_hi) {
    const int64_t mo = (int64_t)row * d.ldm + col;
    x.m = *(const typename MVec<DT>::T*)((const char*)d.M + mo * (DT == DT_F32 ? 4 : 2));
    x.e = d.err_in ? *(const float4*)(d.err_in + (int64_t)row * d.lde_in + col)
                   : make_float4(-0.f, -0.f, -0.f, -0.f);
  } else {
    float a[4];
    load_a4<DT, false>(d, row, col, c_hi, a);
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

// Source of the factors: the caller's P/Q when rank == RP (same layout),
// else the padded workspace copies.
template <int RP>
__device__ __forceinline__ const float* q_src(const Desc& d) { return d.r == RP ? d.Q : d.qpad; }
template <int RP>
__device__ __forceinline__ const float* p_src(const Desc& d) { return d.r == RP ? d.P : d.phat; }

// dst[e] = sum_{g < parts} src[g][e] for e < RP*RP (fixed order); loads are
// issued in batches of 16 so a thread waits for memory once per batch.
template <int RP>
__device__ __forceinline__ void sum_partials(const double* src, int parts, double* dst) {
  for (int e = threadIdx.x; e < RP * RP; e += kBlock) {
    double s = 0.0;
    for (int g0 = 0; g0 < parts; g0 += 16) {
      double v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        v[u] = (g0 + u < parts) ? src[(int64_t)(g0 + u) * RP * RP + e] : 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (g0 + u < parts) s = (g0 + u == 0) ? v[u] : s + v[u];
    }
    dst[e] = s;
  }
}


// Gram of `nr` rows held in LDS as doubles (row pitch RP), full matrix.
template <int RP, int NT = kBlock>
__device__ __forceinline__ void gram_rows_store(const double* rows, int nr, double* dst) {
  for (int e = threadIdx.x; e < RP * RP; e += NT) {
    const int k = e / RP, l = e % RP;
    double s = 0.0;
    for (int i = 0; i < nr; ++i) s = fma(rows[i * RP + k], rows[i * RP + l], s);
    dst[e] = s;
  }
}

// -------------------------------------------------------------------------
// k_orth16: Gram = sum of the row-block partials, Cholesky, T = L^-T
// (CholeskyQR first pass) and, only when the first pass lost orthogonality,
// the second pass; then P_hat = P T.  Blocks of 1024 threads: thread
// (pair, group) sums a slice of the upper-triangle partials with all its
// loads in flight, the slices are added in LDS in order, and wave 0
// factorises with the matrix in registers.
// -------------------------------------------------------------------------
constexpr int CH_THREADS = 1024;
static_assert(F_ORTHROWS <= CH_THREADS, "k_orth16 forms one P_hat row per thread");
constexpr int CH_CHUNK = 256;     // rows per chunk of the second-pass Gram
constexpr int CH_BATCH = 20;      // partial loads in flight per thread

struct CholSmem {
  double part[8][16 * 17 / 2];
  double G[16 * 16];
  double T1[16 * 16];
  double rows[CH_CHUNK * 16];
  uint32_t need;
};

__device__ __forceinline__ double readlane_d(double v, int lane) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), lane);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

template <int RP>
struct CholOut {
  double x[RP];       // lane c: column c of X = L^-1 (dependent rows zero)
  uint32_t defmask;   // dependent columns
  double pmax, pmin;  // extreme pivots (squared diagonal of L) over independent columns < r
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

// Cholesky G = L L^T of the leading RP x RP block of G (rows/columns >= r
// are padding and count as dependent).  A pivot <= kPivotTol * max diag(G)
// marks its column dependent: the column of L is zero below a unit
// diagonal and later columns ignore it.  Executed by one wave with the
// matrix in registers: lane i holds row i, and values of other rows are
// broadcast with v_readlane (compile-time indices), so the sequential
// factorisation has no memory latency.  Only reciprocals of the diagonal
// are formed (one refined rsqrt per pivot; no divides).
template <int RP>
__device__ __forceinline__ CholOut<RP> chol_regs(const double* G, int r, uint32_t* flags) {
  const int lane = threadIdx.x & 63;
  CholOut<RP> o;
  double a[RP];
#pragma unroll
  for (int k = 0; k < RP; ++k) a[k] = (lane < RP) ? G[lane * RP + k] : 0.0;
  double maxdiag = 0.0;
  bool nonfinite = false;
#pragma unroll
  for (int j = 0; j < RP; ++j) {
    const double gjj = readlane_d(a[j], j);
    nonfinite = nonfinite || !isfinite(gjj);
    maxdiag = gjj > maxdiag ? gjj : maxdiag;
  }
  if (lane == 0 && nonfinite && flags) atomicOr(flags, FLAG_NONFINITE);
  const double thr = kPivotTol * maxdiag;
  uint32_t defmask = 0;
  bool any_dep = false;
  double invd[RP];
  o.pmax = 0.0;
  o.pmin = 1e308;
#pragma unroll
  for (int j = 0; j < RP; ++j) {
    const double piv = readlane_d(a[j], j);
    const bool dep = (j >= r) || (piv <= thr);
    any_dep = any_dep || (dep && j < r);
    defmask |= dep ? (1u << j) : 0u;
    if (!dep) {
      o.pmax = piv > o.pmax ? piv : o.pmax;
      o.pmin = piv < o.pmin ? piv : o.pmin;
    }
    // NaN pivots are not "dependent": they propagate into T like the data
    const double inv = dep ? 1.0 : rsqrt_nr(piv);
    invd[j] = inv;
    if (lane == j) a[j] = dep ? 1.0 : piv * inv;
    else if (lane > j) a[j] = dep ? 0.0 : a[j] * inv;
#pragma unroll
    for (int k = j + 1; k < RP; ++k) {
      const double lkj = readlane_d(a[j], k);
      if (lane >= k) a[k] -= a[j] * lkj;
    }
  }
  if (lane == 0 && any_dep && flags) atomicOr(flags, FLAG_RANK_DEFICIENT);
#pragma unroll
  for (int i = 0; i < RP; ++i) {
    double s = (lane == i) ? 1.0 : 0.0;
#pragma unroll
    for (int k = 0; k < i; ++k) s -= readlane_d(a[k], i) * o.x[k];
    o.x[i] = (i >= lane && !((defmask >> i) & 1u)) ? s * invd[i] : 0.0;
  }
  o.defmask = defmask;
  return o;
}

// The first pass lost orthogonality when diag(L) spans more than
// kSecondPassCond, i.e. the pivots span more than its square.
template <int RP>
__device__ __forceinline__ uint32_t needs_second_pass(const CholOut<RP>& o) {
  return (o.pmax > 0.0 && o.pmax > kSecondPassCond * kSecondPassCond * o.pmin) ? 1u : 0u;
}

// Gram (upper triangle, fp64) of `nsrc` stacked RP x RP partials, by all
// CH_THREADS threads; result (full symmetric) in G.
template <int RP>
__device__ __forceinline__ void gram_sum_all(const double* src, int nsrc, CholSmem& sm, double* G) {
  constexpr int NP = RP * (RP + 1) / 2;
  constexpr int NG = CH_THREADS / NP < 8 ? CH_THREADS / NP : 8;
  const int t = threadIdx.x;
  const int p = t % NP, q = t / NP;
  if (q < NG) {
    int k = 0, rem = p;
    while (rem >= RP - k) { rem -= RP - k; ++k; }
    const int e = k * RP + (k + rem);
    const int per = (nsrc + NG - 1) / NG;
    const int g0 = min(nsrc, q * per), g1 = min(nsrc, g0 + per);
    double s = 0.0;
    for (int gb = g0; gb < g1; gb += CH_BATCH) {
      double v[CH_BATCH];
#pragma unroll
      for (int u = 0; u < CH_BATCH; ++u) v[u] = (gb + u < g1) ? src[(int64_t)(gb + u) * RP * RP + e] : 0.0;
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
    int k = 0, rem = t;
    while (rem >= RP - k) { rem -= RP - k; ++k; }
    const int l = k + rem;
    G[k * RP + l] = s;
    G[l * RP + k] = s;
  }
  __syncthreads();
}

// P_hat row = P row * T (fp64), written to the caller's P and the padded
// copy.
template <int RP>
__device__ __forceinline__ void phat_row(const Desc& d, int64_t row, const double* T) {
  // keep the T reads here: hoisting all of them out of a row loop costs ~270 VGPRs
  asm volatile("" ::: "memory");
  float p[RP];
#pragma unroll
  for (int k = 0; k < RP; k += 4) {
    const float4 v = *(const float4*)(d.praw + row * RP + k);
    p[k] = v.x; p[k + 1] = v.y; p[k + 2] = v.z; p[k + 3] = v.w;
  }
  float out[RP];
#pragma unroll
  for (int k = 0; k < RP; ++k) {
    asm volatile("" ::: "memory");   // one column of T in flight at a time
    double v = 0.0;
#pragma unroll
    for (int l = 0; l <= k; ++l) v = fma((double)p[l], T[l * RP + k], v);
    out[k] = (float)v;
  }
  // the padded copy is always written: the reconstruction pass reads it with
  // 16-byte loads (the caller's P has no alignment guarantee)
#pragma unroll
  for (int k = 0; k < RP; k += 4)
    *(float4*)(d.phat + row * RP + k) = make_float4(out[k], out[k + 1], out[k + 2], out[k + 3]);
#pragma unroll
  for (int k = 0; k < RP; ++k)
    if (k < d.r) d.P[row * d.r + k] = out[k];
}

// k_orth16 block b: full Gram, Cholesky (and the second pass when needed),
// computed identically in every block, then P_hat for rows
// [b * F_ORTHROWS, (b + 1) * F_ORTHROWS).  Block 0 also stores T1, Tm, the
// second-pass decision and the numeric flags.
template <int RP>
__device__ __forceinline__ void orth16_body(const Desc& d, int b, uint32_t* flags, CholSmem& sm) {
  const int t = threadIdx.x;
  uint32_t* fl = (b == 0) ? flags : nullptr;
  gram_sum_all<RP>(d.gpart, d.ng, sm, sm.G);
  if (t < kWave) {
    const CholOut<RP> o = chol_regs<RP>(sm.G, d.r, fl);
    const uint32_t need = needs_second_pass<RP>(o);
    if (t < RP) {
#pragma unroll
      for (int i = 0; i < RP; ++i) {
        sm.T1[t * RP + i] = o.x[i];
        if (b == 0) {
          d.t1[t * RP + i] = o.x[i];
          if (!need) d.tm[t * RP + i] = o.x[i];
        }
      }
    }
    if (t == 0) {
      if (b == 0) d.info[0] = need;
      sm.need = need;
    }
  }
  __syncthreads();
  const double* T = sm.T1;
  if (sm.need) {
    // Second pass: Gram of P_hat1 = P T1 (fp64) over all rows, in chunks.
    constexpr int NP = RP * (RP + 1) / 2;
    constexpr int NG = CH_THREADS / NP < 8 ? CH_THREADS / NP : 8;
    const int p = t % NP, q = t / NP;
    int pk_ = 0, rem = p;
    while (rem >= RP - pk_) { rem -= RP - pk_; ++pk_; }
    const int pl_ = pk_ + rem;
    double acc = 0.0;
    const int per = (CH_CHUNK + NG - 1) / NG;
    for (int c0 = 0; c0 < d.m; c0 += CH_CHUNK) {
      if (t < CH_CHUNK) {
        const int row = c0 + t;
        double v[RP];
#pragma unroll
        for (int k = 0; k < RP; ++k) v[k] = 0.0;
        if (row < d.m) {
          asm volatile("" ::: "memory");
#pragma unroll
          for (int k = 0; k < RP; ++k) {
            double sacc = 0.0;
#pragma unroll
            for (int l = 0; l <= k; ++l)
              sacc = fma((double)d.praw[(int64_t)row * RP + l], sm.T1[l * RP + k], sacc);
            v[k] = sacc;
          }
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
    if (t < kWave) {
      const CholOut<RP> o2 = chol_regs<RP>(sm.G, d.r, fl);
      // Tm = T1 T2 with T2 = X2^T: Tm[l][k] = sum_{l <= p <= k} T1[l][p] X2[k][p];
      // lane p holds X2[k][p] in o2.x[k].  G is no longer read (chol_regs
      // loaded it into registers first), so Tm overwrites it row by row.
#pragma unroll
      for (int k = 0; k < RP; ++k) {
        double sacc = 0.0;
#pragma unroll
        for (int pp = 0; pp < RP; ++pp) {
          const double x2 = readlane_d(o2.x[k], pp);
          if (t < RP && pp >= t && pp <= k) sacc = fma(sm.T1[t * RP + pp], x2, sacc);
        }
        if (t < RP) {
          sm.G[t * RP + k] = sacc;
          if (b == 0) d.tm[t * RP + k] = sacc;
        }
      }
    }
    __syncthreads();
    T = sm.G;
  }
  const int64_t row = (int64_t)b * F_ORTHROWS + t;
  if (t < F_ORTHROWS && row < d.m) phat_row<RP>(d, row, T);
}

template <int RP>
__global__ __launch_bounds__(CH_THREADS) void k_orth16(OCC_KARGS, uint32_t* flags) {
  __shared__ CholSmem sm;
#define B_(d, b) orth16_body<RP>(d, b, flags, sm)
  OCC_DISPATCH(K_PGRAM, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_qred16: Q[c][k] = sum over row splits of qpart[s][c][k] (fixed order),
// written to the caller's Q and the padded copy.
// -------------------------------------------------------------------------
template <int RP>
__device__ __forceinline__ void qred16_body(const Desc& d, int b) {
  const int64_t idx = (int64_t)b * kBlock + threadIdx.x;
  if (idx >= (int64_t)d.n * RP) return;
  const int c = (int)(idx / RP), k = (int)(idx % RP);
  float acc = 0.f;
  for (int t0 = 0; t0 < d.sq; t0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (t0 + u < d.sq) ? d.qpart[(int64_t)(t0 + u) * d.n * RP + idx] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (t0 + u < d.sq) acc = (t0 + u == 0) ? v[u] : acc + v[u];
  }
  d.qpad[idx] = acc;   // always: the reconstruction pass reads the padded copy
  if (k < d.r) d.Q[(int64_t)c * d.r + k] = acc;
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qred16(OCC_KARGS) {
#define B_(d, b) qred16_body<RP>(d, b)
  OCC_DISPATCH(K_QRED, B_)
#undef B_
}

}  // namespace occ
