// Small-rank products on the matrix cores (padded rank RP <= 16).
//
// Both tall-skinny products of a power-iteration round are dense
// contractions with a 16-wide output dimension; the 16x16x4 MFMA forms take
// their two operands spread over the 64 lanes (one value per lane), so the
// 16-wide factor (Q rows in the left product, P rows in the right one) never
// has to be broadcast, and A goes straight from 16-byte global loads into
// the instruction.  The left product and the reconstruction are fp32
// products with fp32 accumulation; the right product runs in fp64 (see
// k_qm).
//
// Lane layout of v_mfma_f32_16x16x4_f32 (lane l = 16*g + li):
//   A operand  a = A[i = li][k = g]      B operand  b = B[k = g][j = li]
//   result     D[i = 4*g + v][j = li] in component v of the float4.
//
//   k_pm   P = A Q.  A block owns 32 whole rows (two 16-row MFMA tiles);
//          each wave walks 32-column K-steps: lane (g, li) loads 8
//          consecutive columns 8g..8g+7 of row li (a full 128-byte line of err
//          per 4 lanes) and feeds them to 8 MFMAs whose K index is column
//          8g+j.  The B operand is Q[8g+j][li].  The next K-step's A and Q are
//          loaded before the current one is used.
//   k_qm   Q' = A^T P partials (fp64).  A block owns 128 columns and a row
//          split; each wave takes an eighth of the rows in 4-row K-steps:
//          lane (g, li) loads columns 8li..8li+7 of row g and feeds 8 MFMAs,
//          MFMA t producing the interleaved column tile {8m + t}.  The B
//          operand is P[row g][li].
//   k_mh16 M_hat = P_hat Q^T and err = A - M_hat (see below).
#pragma once

#include "kernels_small.hpp"

namespace occ {

typedef float f4v __attribute__((ext_vector_type(4)));

// LDS reads of W floats issued as inline assembly, for loops with LDS DMA of
// other stages still in flight (the compiler cannot tell those apart from the
// stage being read and would wait for them).  The caller ends a batch of them
// with s_waitcnt lgkmcnt(0), taking the read values as "+v" operands so that
// no use moves above the wait.
template <int W> struct LdsVec;
template <> struct LdsVec<1> { typedef float T; };
template <> struct LdsVec<2> { typedef float T __attribute__((ext_vector_type(2))); };
template <> struct LdsVec<4> { typedef f4v T; };

template <int W>
__device__ __forceinline__ void ds_read_asm(typename LdsVec<W>::T& v, uint32_t addr) {
  if constexpr (W == 1) asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  else if constexpr (W == 2) asm volatile("ds_read_b64 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  else asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
}

template <int W>
__device__ __forceinline__ float lds_elem(const typename LdsVec<W>::T& v, int j) {
  if constexpr (W == 1) return v;
  else return v[j];
}

constexpr int PM_RB = 2;                  // 16-row MFMA tiles per block in k_pm
constexpr int PM_ROWS = 16 * PM_RB;       // rows per block (== F_PROWS)
constexpr int PM_WAVES = F_PM_WAVES;      // waves per block in k_pm
constexpr int PM_THREADS = PM_WAVES * kWave;
static_assert(PM_ROWS == F_PROWS, "k_pm block rows must match the plan");
constexpr int QM_COLS = F_QCOLS;          // columns per block in k_qm
constexpr int QM_WAVES = 8;               // waves per block in k_qm (each a contiguous share of the split's rows)
constexpr int QM_THREADS = QM_WAVES * kWave;

__device__ __forceinline__ f4v mfma4(float a, float b, f4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// v_mfma_f64_16x16x4_f64: the operands as in the fp32 form (lane (g, li)
// supplies A[i = li][k = g] and B[k = g][j = li]), but component v of the
// result holds D[i = 4 v + g][j = li] (rows interleaved across the four lane
// groups; checked with an in-bounds probe on the MI355X).
typedef double d4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ d4v mfma4d(double a, double b, d4v c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Eight consecutive elements of A = M + err_prev (columns c..c+7 of one row),
// kept as raw loads until used.  Out-of-range or unaligned chunks hold the
// exact element-wise A in e0/e1 and -0 in m (x + -0 == x for every x).
template <int DT> struct Ch8;
template <> struct Ch8<DT_BF16> { uint4 m; float4 e0, e1; };
template <> struct Ch8<DT_F32> { float4 m0, m1; float4 e0, e1; };

template <int DT>
__device__ __forceinline__ void ch8_neg_zero(Ch8<DT>& x) {
  if constexpr (DT == DT_BF16) {
    x.m = make_uint4(0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u);
  } else {
    x.m0 = make_float4(-0.f, -0.f, -0.f, -0.f);
    x.m1 = x.m0;
  }
}

template <int DT, bool VEC, bool RM = false>
__device__ __forceinline__ Ch8<DT> ch8_load(const Desc& d, int row, int c, int c_hi) {
  Ch8<DT> x;
  if (VEC && row < d.m && c + 8 <= c_hi) {
    const int64_t pr = prow<RM>(d, row);
    const int64_t mo = pr * d.ldm + c;
    if constexpr (DT == DT_BF16) {
      x.m = *(const uint4*)((const uint16_t*)d.M + mo);
    } else {
      x.m0 = *(const float4*)((const float*)d.M + mo);
      x.m1 = *(const float4*)((const float*)d.M + mo + 4);
    }
    if (d.err_in) {
      const float* e = d.err_in + pr * d.lde_in + c;
      x.e0 = *(const float4*)e;
      x.e1 = *(const float4*)(e + 4);
    } else {
      x.e0 = make_float4(-0.f, -0.f, -0.f, -0.f);
      x.e1 = x.e0;
    }
  } else {
    float lo[4], hi[4];
    load_a4<DT, false, RM>(d, row, c, c_hi, lo);
    load_a4<DT, false, RM>(d, row, c + 4, c_hi, hi);
    ch8_neg_zero<DT>(x);
    x.e0 = make_float4(lo[0], lo[1], lo[2], lo[3]);
    x.e1 = make_float4(hi[0], hi[1], hi[2], hi[3]);
  }
  return x;
}

// The eight A values of a chunk.
template <int DT>
__device__ __forceinline__ void ch8_values(const Ch8<DT>& x, float a[8]) {
  if constexpr (DT == DT_BF16) {
    a[0] = bf16_lo(x.m.x) + x.e0.x; a[1] = bf16_hi(x.m.x) + x.e0.y;
    a[2] = bf16_lo(x.m.y) + x.e0.z; a[3] = bf16_hi(x.m.y) + x.e0.w;
    a[4] = bf16_lo(x.m.z) + x.e1.x; a[5] = bf16_hi(x.m.z) + x.e1.y;
    a[6] = bf16_lo(x.m.w) + x.e1.z; a[7] = bf16_hi(x.m.w) + x.e1.w;
  } else {
    a[0] = x.m0.x + x.e0.x; a[1] = x.m0.y + x.e0.y; a[2] = x.m0.z + x.e0.z; a[3] = x.m0.w + x.e0.w;
    a[4] = x.m1.x + x.e1.x; a[5] = x.m1.y + x.e1.y; a[6] = x.m1.z + x.e1.z; a[7] = x.m1.w + x.e1.w;
  }
}

// Eight Q values Q[c..c+7][li] (zero past n or past the padded rank).
struct Q8v { float4 a, b; };

template <int RP>
__device__ __forceinline__ Q8v q8_load(const float* qs, int n, int c, int li) {
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (li < RP && c + j < n) ? qs[(int64_t)(c + j) * RP + li] : 0.f;
  Q8v q;
  q.a = make_float4(v[0], v[1], v[2], v[3]);
  q.b = make_float4(v[4], v[5], v[6], v[7]);
  return q;
}

// -------------------------------------------------------------------------
// k_pm: left product on MFMA.  A block owns PM_ROWS whole rows at a time;
// its PM_WAVES waves take interleaved 32-column K-steps of those rows (so
// together they stream contiguous column ranges; a matrix with fewer K-steps
// than waves has the spare waves take the next row blocks) and their partial
// tiles are summed in LDS in wave order.  The block stores the final rows of
// P and accumulates the fp64 Gram partial of all its rows.
//
// The MFMA operand layout gives each of a load's 64 lanes a different row
// out of 16 (4 lanes x 16 bytes per row), so a load straight into registers
// touches 16 cache lines per instruction, half of each, and the other half
// comes with the next instruction; the L1 address path then stalls the
// texture addresser for about half of the kernel.  With 16-byte aligned
// rows the tiles are instead brought in by global_load_lds_dwordx4, which
// writes lane l's 16 bytes to LDS at base + 16 l and so lets every
// instruction read whole 128-byte lines (8 rows of err, 16 rows of bf16 M);
// lanes fetch their chunks in an XOR-swizzled order so that the operand
// reads from LDS are free of bank conflicts.  Each wave owns PM_STAGES tile
// stages, two K-steps in flight while it works on a third: with one block of
// four waves per compute unit that measured faster (40.5-41 us vs 42.5 us on
// 8192 x 4096) than eight waves with one K-step in flight each, which is
// what the LDS allows for eight.
// -------------------------------------------------------------------------
constexpr int PM_ESLOT = 1024 + 128;   // LDS bytes per 8-row fp32 load; the pad shifts banks by 32 words
constexpr int PM_BSLOT = 1024;         // LDS bytes per 16-row bf16 M load
constexpr int PM_QBYTES = 32 * 16 * 4; // Q rows of a K-step (rank padded to at most 16)
// one K-step, 32 rows x 32 columns: err, then M (bf16: two 16-row slots;
// fp32: four 8-row slots laid out like err), then the Q rows
template <int DT>
constexpr int pm_mbytes() { return DT == DT_BF16 ? 2 * PM_BSLOT : 4 * PM_ESLOT; }
template <int DT>
constexpr int pm_stage() { return 4 * PM_ESLOT + pm_mbytes<DT>() + PM_QBYTES; }

constexpr int PM_STAGES = 3;             // K-step stages per wave (two in flight)

union PMSmem {
  struct {
    float red[PM_WAVES][PM_ROWS * 16];   // per-wave partial tiles
    double rows[PM_WAVES * PM_ROWS * 16];   // final P rows of the group as doubles (Gram)
  } e;
  uint8_t tile[PM_WAVES][PM_STAGES][pm_stage<DT_F32>()];   // per wave, the K-step stages
};

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// load instructions pm_tile_issue issues per K-step (the same in every wave)
template <int DT, int RP>
constexpr int pm_tile_loads() { return 4 + (DT == DT_BF16 ? 2 : 4) + (32 * RP * 4 + 1023) / 1024; }

// K-step columns [c0, c0 + 32) of the block's 32 rows of err and M, and Q
// rows c0 .. c0+31, into `dst` (rows past m repeat row m-1; their results
// are never stored).
template <int DT, int RP>
__device__ __forceinline__ void pm_tile_issue(const Desc& d, const float* qs, int row0, int c0,
                                              uint8_t* dst) {
  const int lane = threadIdx.x & 63;
  const int last = d.m - 1;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    // err rows 8q .. 8q+7: lane l takes row l / 8, chunk (l % 8) ^ (l / 8)
    const int rr = lane >> 3, ch = (lane & 7) ^ rr;
    const int row = min(row0 + 8 * q + rr, last);
    __builtin_amdgcn_global_load_lds((gvoid_t*)(d.err_in + (int64_t)row * d.lde_in + c0 + 4 * ch),
                                     (lvoid_t*)(dst + q * PM_ESLOT), 16, 0, 0);
  }
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      // bf16 M rows 16q .. 16q+15: lane l takes row l / 4, chunk (l % 4) ^ (l / 16)
      const int rr = lane >> 2, ch = (lane & 3) ^ (rr >> 2);
      const int row = min(row0 + 16 * q + rr, last);
      __builtin_amdgcn_global_load_lds((gvoid_t*)((const uint16_t*)d.M + (int64_t)row * d.ldm + c0 + 8 * ch),
                                       (lvoid_t*)(dst + 4 * PM_ESLOT + q * PM_BSLOT), 16, 0, 0);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // fp32 M: the err layout
      const int rr = lane >> 3, ch = (lane & 7) ^ rr;
      const int row = min(row0 + 8 * q + rr, last);
      __builtin_amdgcn_global_load_lds((gvoid_t*)((const float*)d.M + (int64_t)row * d.ldm + c0 + 4 * ch),
                                       (lvoid_t*)(dst + 4 * PM_ESLOT + q * PM_ESLOT), 16, 0, 0);
    }
  }
  // Q rows c0 .. c0+31 (32 RP floats, contiguous) as they are
#pragma unroll
  for (int q = 0; q < (32 * RP * 4 + 1023) / 1024; ++q)
    if (1024 * q + 16 * lane < 32 * RP * 4)
      __builtin_amdgcn_global_load_lds((gvoid_t*)(qs + (int64_t)c0 * RP + 256 * q + 4 * lane),
                                       (lvoid_t*)(dst + 4 * PM_ESLOT + pm_mbytes<DT>() + 1024 * q), 16, 0, 0);
}

// RM (row-sparse step): rows through the row map, register loads only (the
// tile path's wait counts assume its DMA instructions alone are in flight).
// Row group grp of P: row blocks grp * rpg .. grp * rpg + rpg - 1 (rpg =
// PM_WAVES / wk), wave w taking row block grp * rpg + w / wk and its K-steps
// w % wk, w % wk + wk, ... (wk = pm_waves_per_rb(n) waves per row block).
// The rows are stored to praw, and as doubles to sm.e.rows (zero past m)
// for the Gram partial; ends with a barrier.
template <int DT, bool VEC, int RP, bool RM, int WK>
__device__ __forceinline__ void pm_rows(const Desc& d, int grp, PMSmem& sm) {
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 15, g = lane >> 4;
  const int nk = (d.n + 31) / 32;
  constexpr int wk = WK, rpg = PM_WAVES / WK;
  const int row_blocks = (d.m + PM_ROWS - 1) / PM_ROWS;
  const int rb = grp * rpg + wave / wk, kw = wave % wk;
  const bool live = rb < row_blocks;
  const int row0 = rb * PM_ROWS;
  const float* qs = q_src<RP>(d);

  // Row blocks start their walk at staggered K-steps (and wrap around), so
  // that at any moment the device reads many column ranges instead of one
  // stripe of every row (which lands on a few HBM channels).
  const int ks0 = (int)(((int64_t)rb * wk) % nk);
  auto kcol = [&](int it) {
    int k = ks0 + it;
    if (k >= nk) k -= nk;
    return 32 * k + 8 * g;
  };

  f4v acc[PM_RB];
#pragma unroll
  for (int r = 0; r < PM_RB; ++r) acc[r] = f4v{0.f, 0.f, 0.f, 0.f};

  auto mfma_step = [&](const Ch8<DT>* x, const Q8v& cq) {
    const float qv[8] = {cq.a.x, cq.a.y, cq.a.z, cq.a.w, cq.b.x, cq.b.y, cq.b.z, cq.b.w};
#pragma unroll
    for (int r = 0; r < PM_RB; ++r) {
      float a[8];
      ch8_values<DT>(x[r], a);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[r] = mfma4(a[j], qv[j], acc[r]);
    }
  };

  // 16-byte aligned rows, whole 32-column K-steps, an error buffer and a
  // 16-byte aligned Q: tiles through LDS (the condition is the same for the
  // whole launch); otherwise loads straight into registers.
  bool dma = false;
  if constexpr (VEC && !RM) {
    dma = d.err_in != nullptr && (d.n & 31) == 0 && ((uintptr_t)qs & 15) == 0;
    if (dma) {
      // This wave's K-steps ks = kw + wk * it; step it lives in stage
      // it % PM_STAGES.  Per step: wait until only the steps issued after it
      // may be in flight, read its operands (inline ds_read, see above),
      // issue the step PM_STAGES - 1 ahead into the stage just freed, run the
      // products.
      constexpr int NI = pm_tile_loads<DT, RP>();
      constexpr int STAGE = pm_stage<DT>();
      static_assert(PM_STAGES <= 4 && 2 * NI <= 63, "vmcnt immediates");
      uint8_t* const tiles = sm.tile[wave][0];
      const uint32_t tbase = (uint32_t)(size_t)(lvoid_t*)tiles;
      const int nmine = live && kw < nk ? (nk - kw + wk - 1) / wk : 0;
#pragma unroll
      for (int y = 0; y + 1 < PM_STAGES; ++y)
        if (y < nmine) pm_tile_issue<DT, RP>(d, qs, row0, kcol(kw + wk * y) - 8 * g, tiles + y * STAGE);
      int st = 0;
      for (int it = 0; it < nmine; ++it) {
        const int after = min(it + PM_STAGES - 2, nmine - 1) - it;
        if (after <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        else if (after == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(NI) : "memory");
        else asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * NI) : "memory");
        const uint32_t cb = tbase + st * STAGE;
        // err (and fp32 M) of row tile r: row 16 r + li is slot 2r + li/8,
        // row li % 8 of it; chunk c of that row sits at c ^ (li % 8)
        f4v e0[PM_RB], e1[PM_RB], m0[PM_RB], m1[PM_RB];
        float qv[8];
#pragma unroll
        for (int r = 0; r < PM_RB; ++r) {
          const int q = 2 * r + (li >> 3), rr = li & 7;
          const uint32_t e = cb + q * PM_ESLOT + rr * 128;
          ds_read_asm<4>(e0[r], e + 16 * ((2 * g) ^ rr));
          ds_read_asm<4>(e1[r], e + 16 * ((2 * g + 1) ^ rr));
          if constexpr (DT == DT_BF16) {
            ds_read_asm<4>(m0[r], cb + 4 * PM_ESLOT + r * PM_BSLOT + li * 64 + 16 * (g ^ (li >> 2)));
          } else {
            ds_read_asm<4>(m0[r], e + 4 * PM_ESLOT + 16 * ((2 * g) ^ rr));
            ds_read_asm<4>(m1[r], e + 4 * PM_ESLOT + 16 * ((2 * g + 1) ^ rr));
          }
        }
        const int lq = li < RP ? li : 0;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          ds_read_asm<1>(qv[j], cb + 4 * PM_ESLOT + pm_mbytes<DT>() + ((8 * g + j) * RP + lq) * 4);
        static_assert(PM_RB == 2, "the waits below name the operands of two row tiles");
        if constexpr (DT == DT_BF16) {
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(e0[0]), "+v"(e1[0]), "+v"(m0[0]), "+v"(e0[1]), "+v"(e1[1]), "+v"(m0[1]),
                         "+v"(qv[0]), "+v"(qv[1]), "+v"(qv[2]), "+v"(qv[3]), "+v"(qv[4]), "+v"(qv[5]),
                         "+v"(qv[6]), "+v"(qv[7]));
        } else {
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(e0[0]), "+v"(e1[0]), "+v"(m0[0]), "+v"(m1[0]), "+v"(e0[1]), "+v"(e1[1]),
                         "+v"(m0[1]), "+v"(m1[1]), "+v"(qv[0]), "+v"(qv[1]), "+v"(qv[2]), "+v"(qv[3]),
                         "+v"(qv[4]), "+v"(qv[5]), "+v"(qv[6]), "+v"(qv[7]));
        }
        if (it + PM_STAGES - 1 < nmine) {
          const int sn = st == 0 ? PM_STAGES - 1 : st - 1;
          pm_tile_issue<DT, RP>(d, qs, row0, kcol(kw + wk * (it + PM_STAGES - 1)) - 8 * g,
                                tiles + sn * STAGE);
        }
        st = st + 1 == PM_STAGES ? 0 : st + 1;
        Ch8<DT> x[PM_RB];
#pragma unroll
        for (int r = 0; r < PM_RB; ++r) {
          x[r].e0 = make_float4(e0[r][0], e0[r][1], e0[r][2], e0[r][3]);
          x[r].e1 = make_float4(e1[r][0], e1[r][1], e1[r][2], e1[r][3]);
          if constexpr (DT == DT_BF16) {
            x[r].m = make_uint4(__float_as_uint(m0[r][0]), __float_as_uint(m0[r][1]),
                                __float_as_uint(m0[r][2]), __float_as_uint(m0[r][3]));
          } else {
            x[r].m0 = make_float4(m0[r][0], m0[r][1], m0[r][2], m0[r][3]);
            x[r].m1 = make_float4(m1[r][0], m1[r][1], m1[r][2], m1[r][3]);
          }
        }
        Q8v cq;
        const bool qin = li < RP;
        cq.a = make_float4(qin ? qv[0] : 0.f, qin ? qv[1] : 0.f, qin ? qv[2] : 0.f, qin ? qv[3] : 0.f);
        cq.b = make_float4(qin ? qv[4] : 0.f, qin ? qv[5] : 0.f, qin ? qv[6] : 0.f, qin ? qv[7] : 0.f);
        mfma_step(x, cq);
      }
    }
  }
  if (!dma) {
    Ch8<DT> cur[PM_RB], nxt[PM_RB];
    Q8v cq, nq;
    int ks = live ? kw : nk;
    if (ks < nk) {
      const int c = kcol(ks);
      cq = q8_load<RP>(qs, d.n, c, li);
#pragma unroll
      for (int r = 0; r < PM_RB; ++r) cur[r] = ch8_load<DT, VEC, RM>(d, row0 + 16 * r + li, c, d.n);
    }
    for (; ks < nk; ks += wk) {
      const bool more = ks + wk < nk;
      const int cn = more ? kcol(ks + wk) : 0;
      if (more) {
        nq = q8_load<RP>(qs, d.n, cn, li);
#pragma unroll
        for (int r = 0; r < PM_RB; ++r) nxt[r] = ch8_load<DT, VEC, RM>(d, row0 + 16 * r + li, cn, d.n);
      }
      mfma_step(cur, cq);
      if (more) {
        cq = nq;
#pragma unroll
        for (int r = 0; r < PM_RB; ++r) cur[r] = nxt[r];
      }
    }
  }
  __syncthreads();   // every wave is done with its tiles before they turn into the reduction buffer

  // acc[r][v] = partial P[row0 + 16r + 4g + v][li] of this wave.
#pragma unroll
  for (int r = 0; r < PM_RB; ++r)
#pragma unroll
    for (int v = 0; v < 4; ++v) sm.e.red[wave][(16 * r + 4 * g + v) * 16 + li] = acc[r][v];
  __syncthreads();
  // row block r of the group: the partial tiles of waves r wk .. r wk + wk - 1, in order
  for (int e = threadIdx.x; e < rpg * PM_ROWS * RP; e += PM_THREADS) {
    const int r = e / (PM_ROWS * RP), i = (e / RP) % PM_ROWS, k = e % RP;
    float s = sm.e.red[r * wk][i * 16 + k];
#pragma unroll
    for (int w = 1; w < wk; ++w) s = s + sm.e.red[r * wk + w][i * 16 + k];
    const int64_t row = (int64_t)(grp * rpg + r) * PM_ROWS + i;
    if (row < d.m) d.praw[row * RP + k] = s;
    sm.e.rows[(r * PM_ROWS + i) * RP + k] = row < d.m ? (double)s : 0.0;
  }
  __syncthreads();
}

// Block b takes row groups b, b + ng, b + 2 ng, ... (ng = d.ng blocks, at
// most F_PM_MAXBLOCKS, so that the Gram partials stay few for tall
// matrices) and stores one packed fp64 Gram partial of all its rows
// (entry p accumulated by thread p, rows in order).  NARROW: some matrix of
// the launch has fewer K-steps than waves (each matrix's row grouping is
// chosen at run time); otherwise every matrix takes one row block at a time.
template <int DT, bool VEC, int RP, bool RM = false, bool NARROW = false>
__device__ __forceinline__ void pm_body(const Desc& d, int b, PMSmem& sm) {
  constexpr int NP = RP * (RP + 1) / 2;
  static_assert(NP <= PM_THREADS, "one Gram entry per thread");
  const int t = threadIdx.x;
  int gk = 0, gl = 0;
  if (t < NP) upper_entry<RP>(t, gk, gl);
  double gacc = 0.0;
  const int wk = NARROW ? pm_waves_per_rb(d.n) : PM_WAVES, rpg = PM_WAVES / wk;
  const int row_groups = ((d.m + PM_ROWS - 1) / PM_ROWS + rpg - 1) / rpg;
  for (int grp = b; grp < row_groups; grp += d.ng) {
    if (grp != b) __syncthreads();   // the rows are read before the next tiles land there
    if (!NARROW || wk == PM_WAVES) pm_rows<DT, VEC, RP, RM, PM_WAVES>(d, grp, sm);
    else if (wk == 2) pm_rows<DT, VEC, RP, RM, 2>(d, grp, sm);
    else pm_rows<DT, VEC, RP, RM, 1>(d, grp, sm);
    const int nr = min(rpg * PM_ROWS, d.m - grp * rpg * PM_ROWS);
    if (t < NP)
      for (int i = 0; i < nr; ++i) gacc = fma(sm.e.rows[i * RP + gk], sm.e.rows[i * RP + gl], gacc);
  }
  if (t < NP) d.gpart[(int64_t)b * NP + t] = gacc;
}

template <int DT, bool VEC, int RP, bool RM = false, bool NARROW = false>
__global__ __launch_bounds__(PM_THREADS) void k_pm(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) PMSmem sm;
#define B_(d, b) pm_body<DT, VEC, RP, RM, NARROW>(d, b, sm)
  OCC_DISPATCH(K_PASS_P, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_qm: right product partials on the fp64 matrix cores, Q' = A^T P on the
// raw P (A^T P_hat = Q' T, with T applied by k_qfin16).  T cancels the
// disparate scales and near-parallel directions of P's columns, so Q' is
// accumulated in fp64 (A and P enter exactly): in fp32 the cancellation
// amplified its rounding by up to the condition of P.  At rank 16 the fp64
// products take about 14 us of matrix-core time on 8192 x 4096 against
// about 25 us of memory time, so the pass stays memory-bound.
//
// A block owns 128 columns and a row split; each of its QM_WAVES waves takes
// a contiguous share of the split's rows in 4-row K-steps.  The B operand is
// P[row][li], read from the padded raw P.  The waves' partial tiles are
// summed in LDS in a fixed order and stored (fp64) to qpart[split].  The
// first `count` blocks of the grid instead form the orthogonalisation factor
// T of one matrix each (orth_t_body): they are dispatched first and finish
// while the streaming blocks run.
// -------------------------------------------------------------------------
struct QMSmem {
  double red[QM_WAVES / 2][QM_COLS * 16];   // partial tiles of wave pairs (w, w + QM_WAVES / 2)
};

template <int DT, bool VEC, int RP, bool RM = false>
__device__ __forceinline__ void qm_body(const Desc& d, int b, QMSmem& sm) {
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 15, g = lane >> 4;
  const int col_tiles = (d.n + QM_COLS - 1) / QM_COLS;
  const int ct = b % col_tiles, s = b / col_tiles;
  const int r_lo = s * d.q_rows;
  const int r_hi = min(d.m, r_lo + d.q_rows);
  const int nr = r_hi - r_lo;
  const int c0 = ct * QM_COLS;

  const float* ps = d.praw;

  const int wr = (nr + QM_WAVES - 1) / QM_WAVES;
  const int w_lo = r_lo + min(nr, wave * wr), w_hi = r_lo + min(nr, wave * wr + wr);
  const int nk = (w_hi - w_lo + 3) / 4;
  const int col = c0 + 8 * li;
  d4v acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = d4v{0.0, 0.0, 0.0, 0.0};
  Ch8<DT> cur, nxt;
  float cp = 0.f, np = 0.f;
  {
    const int row = w_lo + g;
    const bool ok = row < w_hi;
    cur = ch8_load<DT, VEC, RM>(d, ok ? row : d.m, col, d.n);
    cp = (ok && li < RP) ? ps[(int64_t)row * RP + li] : 0.f;
  }
  for (int ks = 0; ks < nk; ++ks) {
    const bool more = ks + 1 < nk;
    if (more) {
      const int row = w_lo + 4 * (ks + 1) + g;
      const bool ok = row < w_hi;
      nxt = ch8_load<DT, VEC, RM>(d, ok ? row : d.m, col, d.n);
      np = (ok && li < RP) ? ps[(int64_t)row * RP + li] : 0.f;
    }
    float a[8];
    ch8_values<DT>(cur, a);
    const double pd = (double)cp;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = mfma4d((double)a[t], pd, acc[t]);
    if (more) {
      cur = nxt;
      cp = np;
    }
  }

  // acc[t][v] = partial Q'[c0 + 8(4v + g) + t][li] of this wave.  Waves
  // w < QM_WAVES / 2 store theirs, waves w + QM_WAVES / 2 add theirs to
  // them, and the pair sums are added in pair order.
  constexpr int HW = QM_WAVES / 2;
  double* red = sm.red[wave % HW];
  if (wave < HW) {
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[(8 * (4 * v + g) + t) * 16 + li] = acc[t][v];
  }
  __syncthreads();
  if (wave >= HW) {
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = (8 * (4 * v + g) + t) * 16 + li;
        red[i] = red[i] + acc[t][v];
      }
  }
  __syncthreads();
  double* qp = (double*)d.qpart;
  for (int e = threadIdx.x; e < QM_COLS * RP; e += QM_THREADS) {
    const int cl = e / RP, k = e % RP;
    const int gcol = c0 + cl;
    if (gcol >= d.n) continue;
    double v = sm.red[0][cl * 16 + k];
#pragma unroll
    for (int w = 1; w < HW; ++w) v = v + sm.red[w][cl * 16 + k];
    qp[((int64_t)s * d.n + gcol) * RP + k] = v;
  }
}

union QMOSmem {
  QMSmem q;
  CholSmem c;
};

template <int DT, bool VEC, int RP, bool RM = false>
__global__ __launch_bounds__(QM_THREADS) void k_qm(OCC_KARGS, uint32_t* flags) {
  __shared__ __attribute__((aligned(16))) QMOSmem sm;
  const int b = (int)blockIdx.x;
  if (b < count) {
    orth_t_body<RP, QM_THREADS>(count == 1 ? single : table[b], flags, sm.c);
    return;
  }
#define B_(d, bb) qm_body<DT, VEC, RP, RM>(d, bb, sm.q)
  OCC_DISPATCH_AT(K_PASS_Q, B_, b - count)
#undef B_
}

// -------------------------------------------------------------------------
// k_mh16: reconstruction and residual, M_hat = P_hat Q^T and
// err = A - M_hat.  The products run on v_mfma_f32_16x16x4_f32 in the
// transposed form M_hat^T = Q P_hat^T: for a 16-row group and a 16-column
// tile, lane (g, li) supplies Q[col li][k] and P_hat[row li][k] for its
// K-steps' rank indices k = S g + s (S = RP / 4, MFMA s) and receives
// M_hat[row li][cols 4g..4g+3].  That layout would write 16 rows x 64 bytes
// per instruction, so each wave passes its 16 x F_MHCOLS tile through LDS
// and then reads A, writes M_hat and writes err row-contiguously (32 lanes x
// 16 bytes per row).  A block is four waves; wave w takes the 16-row groups
// w, w + 4, ... of the block's d.mr rows, and loads that group's A before
// its MFMAs so the loads are in flight during them.
//
// SRC 0: factors from the step's padded workspace copies (row pitch RP,
//        read with 16-byte loads).
// SRC 1: the caller's P (m x r) and Q (n x r) (stand-alone decompression).
// WRITE_ERR also reads A and writes err; without it only M_hat is written.
// Both entry points run this same code, so their M_hat agree bitwise.
// -------------------------------------------------------------------------
constexpr int MX_LDW = F_MHCOLS + 4;          // LDS row pitch (floats), 16-byte skew per row
constexpr int MX_LPR = F_MHCOLS / 4;          // lanes per row in the row-contiguous phase
constexpr int MX_RPI = kWave / MX_LPR;        // rows per instruction in that phase
constexpr int MX_NCH = 16 / MX_RPI;           // row chunks per lane per 16-row group
static_assert(F_MHGROUP == 4 * 16, "four waves of 16-row groups per block step");

struct MXSmem {
  float t[4][16 * MX_LDW];
};

// Factor values [row][S g .. S g + S - 1] of a lane: from the padded
// workspace copy (row pitch RP, 256-byte aligned base) with one vector load,
// or from a caller's m x r array element by element (zero past rank r).
template <int S>
__device__ __forceinline__ void factor_vec(const float* p, float v[S]) {
  if constexpr (S % 4 == 0) {
#pragma unroll
    for (int j = 0; j < S; j += 4) {
      const float4 x = *(const float4*)(p + j);
      v[j] = x.x; v[j + 1] = x.y; v[j + 2] = x.z; v[j + 3] = x.w;
    }
  } else if constexpr (S == 2) {
    const float2 x = *(const float2*)p;
    v[0] = x.x; v[1] = x.y;
  } else {
    v[0] = *p;
  }
}

template <int RP, int SRC>
__device__ __forceinline__ void factor_load(const float* base, int r, int row, bool ok, int k0,
                                            float v[RP / 4]) {
  constexpr int S = RP / 4;
  if (!ok) {
#pragma unroll
    for (int s = 0; s < S; ++s) v[s] = 0.f;
  } else if (SRC == 0) {
    factor_vec<S>(base + (int64_t)row * RP + k0, v);
  } else {
#pragma unroll
    for (int s = 0; s < S; ++s) v[s] = (k0 + s < r) ? base[(int64_t)row * r + k0 + s] : 0.f;
  }
}

// OUTBF (stand-alone decompression only): M_hat is stored as bf16, each
// element rounded to nearest even from the fp32 result.
template <int DT, bool VEC, int RP, int SRC, bool WRITE_MHAT, bool WRITE_ERR, bool OUTBF = false,
          bool RM = false>
__device__ __forceinline__ void mh16_body(const Desc& d, int b, MXSmem& sm) {
  constexpr int S = RP / 4;        // MFMA K-steps (rank indices per lane group)
  constexpr int NTILE = F_MHCOLS / 16;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 15, g = lane >> 4;
  const int col_tiles = (d.n + F_MHCOLS - 1) / F_MHCOLS;
  const int ct = b % col_tiles, rb = b / col_tiles;
  const int c0 = ct * F_MHCOLS;
  const int r_lo = rb * d.mr, r_hi = min(d.m, r_lo + d.mr);
  const float* qs = (SRC == 0) ? d.qpad : d.Q;
  const float* ps = (SRC == 0) ? d.phat : d.P;

  // A operand of tile t: Q[c0 + 16t + li][S g + s]
  float qa[NTILE][S];
#pragma unroll
  for (int t = 0; t < NTILE; ++t) {
    const int c = c0 + 16 * t + li;
    factor_load<RP, SRC>(qs, d.r, c, c < d.n, S * g, qa[t]);
  }
  const int cl = 4 * (lane % MX_LPR), rl = lane / MX_LPR;
  const int col = c0 + cl;
  const bool vec_col = VEC && col + 4 <= d.n;
  float* tile = sm.t[wave];
  for (int r0 = r_lo + 16 * wave; r0 < r_hi; r0 += F_MHGROUP) {
    AChunk<DT> x[MX_NCH];
    if (WRITE_ERR) {
#pragma unroll
      for (int k = 0; k < MX_NCH; ++k) {
        const int row = r0 + rl + MX_RPI * k;
        chunk_issue<DT, VEC, RM>(d, row < r_hi ? row : d.m, col, d.n, x[k]);
      }
    }
    // B operand: P_hat[r0 + li][S g + s]
    const int rowb = r0 + li;
    float pb[S];
    factor_load<RP, SRC>(ps, d.r, rowb, rowb < r_hi, S * g, pb);
#pragma unroll
    for (int t = 0; t < NTILE; ++t) {
      f4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < S; ++s) acc = mfma4(qa[t][s], pb[s], acc);
      *(float4*)(tile + li * MX_LDW + 16 * t + 4 * g) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
    // the tile is written and read by this wave only; LDS keeps a wave's
    // operations in order, and the wait also orders them for the compiler
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int k = 0; k < MX_NCH; ++k) {
      const int rr = rl + MX_RPI * k;
      const int row = r0 + rr;
      const float4 mh4 = *(const float4*)(tile + rr * MX_LDW + cl);
      if (row >= r_hi) continue;
      const int64_t pr = prow<RM>(d, row);
      const float mh[4] = {mh4.x, mh4.y, mh4.z, mh4.w};
      float e[4] = {0.f, 0.f, 0.f, 0.f};
      if (WRITE_ERR) {
        float a[4];
        chunk_value<DT>(x[k], a);
#pragma unroll
        for (int j = 0; j < 4; ++j) e[j] = a[j] - mh[j];
      }
      if (vec_col) {
        // streaming outputs: nontemporal stores (the dirty lines would
        // otherwise be written back during the next step's first pass)
        typedef float nt4 __attribute__((ext_vector_type(4)));
        typedef uint32_t nu2 __attribute__((ext_vector_type(2)));
        if (WRITE_MHAT && OUTBF)
          __builtin_nontemporal_store(nu2{bf16_pack2(mh[0], mh[1]), bf16_pack2(mh[2], mh[3])},
                                      (nu2*)((uint16_t*)d.Mhat + pr * d.ldh + col));
        else if (WRITE_MHAT)
          __builtin_nontemporal_store(nt4{mh[0], mh[1], mh[2], mh[3]},
                                      (nt4*)(d.Mhat + pr * d.ldh + col));
        if (WRITE_ERR)
          __builtin_nontemporal_store(nt4{e[0], e[1], e[2], e[3]},
                                      (nt4*)(d.err_out + pr * d.lde_out + col));
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (col + j < d.n) {
            if (WRITE_MHAT) store_mhat1<OUTBF>(d, pr * d.ldh + col + j, mh[j]);
            if (WRITE_ERR) d.err_out[pr * d.lde_out + col + j] = e[j];
          }
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

template <int DT, bool VEC, int RP, int SRC, bool WRITE_MHAT, bool WRITE_ERR, bool OUTBF = false,
          bool RM = false>
__global__ __launch_bounds__(kBlock) void k_mh16(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) MXSmem sm;
#define B_(d, b) mh16_body<DT, VEC, RP, SRC, WRITE_MHAT, WRITE_ERR, OUTBF, RM>(d, b, sm)
  OCC_DISPATCH(K_MHAT, B_)
#undef B_
}

}  // namespace occ
