// liboptcc C ABI: argument validation, workspace carving and launch sequencing.
//
// Everything here runs on the host.  Arguments are checked before anything
// is enqueued; a call either returns an error code with the device untouched
// or enqueues its whole kernel sequence on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <type_traits>
#include <vector>

#include "optcc.h"
#include "plan.hpp"
#include "kernels.hpp"
#include "kernels_small.hpp"
#include "kernels_mfma16.hpp"
#include "kernels_large.hpp"
#include "sc_model.hpp"

using namespace occ;

// Workspace of occ_step_batched_noalloc: one array per GPU, resident for the
// life of the process.  Host code never uses this name as an address (it is
// a host-side stand-in); it takes each device's address from
// hipGetSymbolAddress once per device (noalloc_scratch below).
static __device__ __align__(256) uint8_t scratch[OCC_NOALLOC_MAX_BYTES];

namespace {

// ----------------------------------------------------------------------------
// optional per-kernel event timing
// ----------------------------------------------------------------------------
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};

struct Profiler {
  bool on = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> free_events;

  hipEvent_t take() {
    if (!free_events.empty()) {
      hipEvent_t e = free_events.back();
      free_events.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

Profiler g_prof;

template <typename F>
occ_status_t launch(const char* name, hipStream_t s, F&& f) {
  hipEvent_t a = nullptr;
  if (g_prof.on) {
    a = g_prof.take();
    if (a) (void)hipEventRecord(a, s);
  }
  f();
  const hipError_t e = hipGetLastError();
  if (g_prof.on && a) {
    hipEvent_t b = g_prof.take();
    if (b) {
      (void)hipEventRecord(b, s);
      g_prof.recs.push_back({name, a, b});
    }
  }
  return e == hipSuccess ? OCC_OK : OCC_E_HIP;
}

#define OCC_TRY(x)                       \
  do {                                   \
    const occ_status_t st_ = (x);        \
    if (st_ != OCC_OK) return st_;       \
  } while (0)

template <typename F>
void with_rp(int rp, F&& f) {
  switch (rp) {
    case 4: f(std::integral_constant<int, 4>{}); break;
    case 8: f(std::integral_constant<int, 8>{}); break;
    case 16: f(std::integral_constant<int, 16>{}); break;
    case 32: f(std::integral_constant<int, 32>{}); break;
    case 64: f(std::integral_constant<int, 64>{}); break;
    default: f(std::integral_constant<int, 128>{}); break;
  }
}

template <typename F>
void with_dt_vec(int dt, bool vec, F&& f) {
  if (dt == DT_F32) {
    if (vec) f(std::integral_constant<int, DT_F32>{}, std::true_type{});
    else f(std::integral_constant<int, DT_F32>{}, std::false_type{});
  } else {
    if (vec) f(std::integral_constant<int, DT_BF16>{}, std::true_type{});
    else f(std::integral_constant<int, DT_BF16>{}, std::false_type{});
  }
}

// ----------------------------------------------------------------------------
// validation helpers
// ----------------------------------------------------------------------------
struct Span {
  uintptr_t lo, hi;
  bool writable;
};

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t elem_size(int dt) { return dt == OCC_BF16 ? 2 : 4; }

Span span2d(const void* p, int64_t rows, int64_t cols, int64_t ld, size_t es, bool w) {
  const uintptr_t lo = (uintptr_t)p;
  return {lo, lo + (uintptr_t)(((rows - 1) * ld + cols) * (int64_t)es), w};
}

bool overlaps(std::vector<Span> v) {
  std::sort(v.begin(), v.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
  // any writable interval must be disjoint from every other interval
  for (size_t i = 0; i < v.size(); ++i) {
    for (size_t j = i + 1; j < v.size() && v[j].lo < v[i].hi; ++j) {
      if (v[i].writable || v[j].writable) return true;
    }
  }
  return false;
}

constexpr int64_t kMaxDim = (int64_t)1 << 31;

occ_status_t check_rank_iters(int rank, int iters, int64_t m, int64_t n) {
  if (rank < 1 || rank > OCC_MAX_RANK || rank > m || rank > n) return OCC_E_RANK;
  if (iters < 1 || iters > OCC_MAX_ITERS) return OCC_E_ITERS;
  return OCC_OK;
}

occ_status_t check_shape(int64_t m, int64_t n, int64_t ld) {
  if (m < 1 || n < 1 || m >= kMaxDim || n >= kMaxDim) return OCC_E_SHAPE;
  if (ld < n || ld >= kMaxDim) return OCC_E_SHAPE;
  if (m * ld >= ((int64_t)1 << 46)) return OCC_E_SHAPE;
  return OCC_OK;
}

// ----------------------------------------------------------------------------
// batch plan
// ----------------------------------------------------------------------------
struct Batch {
  std::vector<Desc> descs;
  int rp = 4, dt = 0, iters = 1;
  bool vec = false;
  bool fused = false;
  int64_t blocks[K_NUM] = {};
  size_t ws_needed = 0;
};

// ----------------------------------------------------------------------------
// resident blocks of the large-rank streaming kernels
// ----------------------------------------------------------------------------
// From the HIP occupancy calculator for the kernel instances of a fused step
// on the current device.  When no device answers (a host without a GPU) the
// defaults of Slots apply, so workspace sizes stay computable there; a
// workspace sized on one device type may be too small on another, which the
// call reports as OCC_E_WORKSPACE.
template <int DT, int RP>
Slots device_slots_for(int dev) {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1) {
    (void)hipGetLastError();
    return Slots{};
  }
  constexpr bool X3 = DT == DT_BF16;
  int bp = 0, bq = 0, bm = 0;
  bool ok = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                 &bp, k_lp<DT, RP, SA_MERR_SAVE, X3, true>, lp_block_rows(RP, X3) / 32 * kWave,
                 0) == hipSuccess;
  if constexpr (X3)
    ok = ok && hipOccupancyMaxActiveBlocksPerMultiprocessor(&bq, k_lqx<DT_F32, RP, SA_SAVED, true>,
                                                            lqx_waves(RP) * kWave, 0) == hipSuccess;
  else
    ok = ok && hipOccupancyMaxActiveBlocksPerMultiprocessor(&bq, k_lq<DT_F32, RP, SA_SAVED, true>,
                                                            kBlock, 0) == hipSuccess;
  if constexpr (X3)
    ok = ok && hipOccupancyMaxActiveBlocksPerMultiprocessor(&bm, k_mlx<RP, 0, true, true>, kBlock,
                                                            0) == hipSuccess;
  else
    ok = ok && hipOccupancyMaxActiveBlocksPerMultiprocessor(
                   &bm, k_ml<DT_F32, RP, SA_SAVED, 0, true, true>, kBlock, 0) == hipSuccess;
  if (!ok || bp < 1 || bq < 1 || bm < 1) {
    (void)hipGetLastError();
    return Slots{};
  }
  Slots sl;
  sl.p = (int64_t)cus * bp;
  sl.q = (int64_t)cus * bq;
  sl.m = (int64_t)cus * bm;
  return sl;
}

Slots device_slots(int dt, int rp) {
  if (rp <= kFusedMaxRank) return Slots{};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return Slots{};
  }
  static std::mutex mu;
  static std::map<std::tuple<int, int, int>, Slots> cache;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(dev, dt, rp);
  const auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  Slots sl;
  with_rp(rp, [&](auto RPc) {
    constexpr int RP = decltype(RPc)::value;
    if constexpr (RP > kFusedMaxRank)
      sl = dt == DT_F32 ? device_slots_for<DT_F32, RP>(dev) : device_slots_for<DT_BF16, RP>(dev);
  });
  cache[key] = sl;
  return sl;
}

size_t table_bytes(int count) { return count > 1 ? align_up((size_t)count * sizeof(Desc)) : 0; }

// Turn the workspace offsets stored in the descriptors into device addresses.
void finalize_regions(Batch& b, void* ws) {
  const uintptr_t base = (uintptr_t)ws;
  for (Desc& d : b.descs) {
    d.qpad = (float*)(base + (uintptr_t)d.qpad);
    d.phat = (float*)(base + (uintptr_t)d.phat);
    d.praw = (float*)(base + (uintptr_t)d.praw);
    d.ppart = (float*)(base + (uintptr_t)d.ppart);
    d.qpart = (float*)(base + (uintptr_t)d.qpart);
    d.gpart = (double*)(base + (uintptr_t)d.gpart);
    d.gsum = (double*)(base + (uintptr_t)d.gsum);
    d.t1 = (double*)(base + (uintptr_t)d.t1);
    d.tm = (double*)(base + (uintptr_t)d.tm);
    d.info = (uint32_t*)(base + (uintptr_t)d.info);
    d.phat_t = (float*)(base + (uintptr_t)d.phat_t);
    d.qbf = (uint16_t*)(base + (uintptr_t)d.qbf);
  }
}

// Validate a batch and compute its plan.  With ws == nullptr only the
// workspace size is computed (pointers are not checked).
occ_status_t plan_batch(const occ_mat_t* mats, int count, int rank, int iters, unsigned flags,
                        void* ws, size_t ws_bytes, bool size_only, Batch& b) {
  if (count < 1) return OCC_E_SHAPE;
  if (!mats) return OCC_E_NULL;
  if (flags & ~(unsigned)OCC_NO_MHAT) return OCC_E_FLAGS;
  const bool write_mhat = !(flags & OCC_NO_MHAT);
  const int dt = mats[0].m_dtype;
  for (int j = 0; j < count; ++j) {
    const occ_mat_t& a = mats[j];
    if (a.m_dtype != OCC_F32 && a.m_dtype != OCC_BF16) return OCC_E_DTYPE;
    if (a.m_dtype != dt) return OCC_E_DTYPE;
    OCC_TRY(check_shape(a.rows, a.cols, a.ldm));
    if (!size_only) {
      OCC_TRY(check_shape(a.rows, a.cols, a.lde));
      if (write_mhat) OCC_TRY(check_shape(a.rows, a.cols, a.ldh));
    }
    OCC_TRY(check_rank_iters(rank, iters, a.rows, a.cols));
  }
  b.rp = padded_rank(rank);
  b.dt = dt;
  b.iters = iters;
  b.fused = b.rp <= kFusedMaxRank;
  size_t off = kHeaderBytes + table_bytes(count);
  double total_elems = 0.0;
  for (int j = 0; j < count; ++j) total_elems += (double)mats[j].rows * (double)mats[j].cols;
  const Slots slots = device_slots(dt, b.rp);
  b.descs.assign(count, Desc{});
  for (int k = 0; k < K_NUM; ++k) b.blocks[k] = 0;
  for (int j = 0; j < count; ++j) {
    const occ_mat_t& a = mats[j];
    const Tiling t =
        make_tiling(a.rows, a.cols, b.rp, (double)a.rows * (double)a.cols / total_elems, slots,
                    dt == OCC_BF16);
    const Regions g = matrix_regions(a.rows, a.cols, b.rp, t);
    Desc& d = b.descs[j];
    d.m = (int32_t)a.rows;
    d.n = (int32_t)a.cols;
    d.r = rank;
    d.n_pad = t.n_pad;
    d.sp = t.sp;
    d.p_cols = t.p_cols;
    d.ng = t.ng;
    d.grows = t.grows;
    d.sq = t.sq;
    d.q_rows = t.q_rows;
    d.m_pad = t.m_pad;
    d.mr = t.mr;
    d.qr_cols = t.qr_cols;
    d.fused = b.fused ? 1 : 0;
    for (int k = 0; k < K_NUM; ++k) {
      d.blk[k] = (int32_t)b.blocks[k];
      b.blocks[k] += t.blocks[k];
      if (b.blocks[k] >= ((int64_t)1 << 31)) return OCC_E_SHAPE;
    }
    // remember region offsets (converted to pointers below)
    d.qpad = (float*)(uintptr_t)(off + g.qpad);
    d.phat = (float*)(uintptr_t)(off + g.phat);
    d.praw = (float*)(uintptr_t)(off + g.praw);
    d.ppart = (float*)(uintptr_t)(off + g.ppart);
    d.qpart = (float*)(uintptr_t)(off + g.qpart);
    d.gpart = (double*)(uintptr_t)(off + g.gpart);
    d.gsum = (double*)(uintptr_t)(off + g.gsum);
    d.t1 = (double*)(uintptr_t)(off + g.t1);
    d.tm = (double*)(uintptr_t)(off + g.tm);
    d.info = (uint32_t*)(uintptr_t)(off + g.info);
    d.phat_t = (float*)(uintptr_t)(off + g.phat_t);
    d.qbf = (uint16_t*)(uintptr_t)(off + g.qbf);
    off += g.total;
  }
  b.ws_needed = off;
  if (size_only) return OCC_OK;

  // pointers, alignment, aliasing, workspace
  if (!ws) return OCC_E_WORKSPACE;
  bool vec = true;
  std::vector<Span> spans;
  for (int j = 0; j < count; ++j) {
    const occ_mat_t& a = mats[j];
    if (!a.M || !a.err || !a.P || !a.Q || (write_mhat && !a.M_hat)) return OCC_E_NULL;
    const size_t es = elem_size(dt);
    if (!aligned(a.M, es) || !aligned(a.err, 4) || !aligned(a.P, 4) || !aligned(a.Q, 4) ||
        (write_mhat && !aligned(a.M_hat, 4)))
      return OCC_E_ALIGN;
    vec = vec && aligned(a.M, 16) && a.ldm % (dt == OCC_BF16 ? 8 : 4) == 0 &&
          aligned(a.err, 16) && a.lde % 4 == 0 &&
          (!write_mhat || (aligned(a.M_hat, 16) && a.ldh % 4 == 0));
    spans.push_back(span2d(a.M, a.rows, a.cols, a.ldm, es, false));
    spans.push_back(span2d(a.err, a.rows, a.cols, a.lde, 4, true));
    spans.push_back(span2d(a.P, a.rows, rank, rank, 4, true));
    spans.push_back(span2d(a.Q, a.cols, rank, rank, 4, true));
    if (write_mhat) spans.push_back(span2d(a.M_hat, a.rows, a.cols, a.ldh, 4, true));
  }
  if (!aligned(ws, kAlign)) return OCC_E_WORKSPACE;
  if (ws_bytes < b.ws_needed) return OCC_E_WORKSPACE;
  spans.push_back({(uintptr_t)ws, (uintptr_t)ws + b.ws_needed, true});
  if (overlaps(spans)) return OCC_E_ALIAS;
  b.vec = vec;

  finalize_regions(b, ws);
  for (int j = 0; j < count; ++j) {
    const occ_mat_t& a = mats[j];
    Desc& d = b.descs[j];
    if (dt != OCC_BF16) d.qbf = nullptr;   // the bf16 Q parts serve bf16 M only
    d.M = a.M;
    d.err_in = a.err;
    d.err_out = a.err;
    d.P = a.P;
    d.Q = a.Q;
    d.Mhat = write_mhat ? a.M_hat : nullptr;
    d.ldm = (int32_t)a.ldm;
    d.lde_in = (int32_t)a.lde;
    d.lde_out = (int32_t)a.lde;
    d.ldh = write_mhat ? (int32_t)a.ldh : 0;
    d.vec = vec ? 1 : 0;
  }
  return OCC_OK;
}

unsigned grid_of(int64_t blocks) { return (unsigned)std::max<int64_t>(blocks, 1); }

// Enqueue the compression passes (and, with `finish`, the fused
// reconstruction/residual pass) for a planned batch; numeric flags go to
// `flags`.  RM: row-sparse step (rows of M, err and M_hat through each
// descriptor's row map), on the register-load forms of the streaming kernels.
template <bool RM>
occ_status_t run_batch_t(const Batch& b, void* ws, uint32_t* flags, bool finish, bool write_mhat,
                         hipStream_t s) {
  const int count = (int)b.descs.size();
  const Desc* table = nullptr;
  Desc single = b.descs[0];
  if (count > 1) {
    Desc* dst = (Desc*)((char*)ws + kHeaderBytes);
    table = dst;
    for (int j0 = 0; j0 < count; j0 += kTableChunk) {
      TableChunk c{};
      const int nj = std::min(kTableChunk, count - j0);
      for (int j = 0; j < nj; ++j) c.d[j] = b.descs[j0 + j];
      OCC_TRY(launch("write_table", s, [&] {
        hipLaunchKernelGGL(k_write_table, dim3(1), dim3(256), 0, s, dst + j0, c, nj);
      }));
    }
  }
  occ_status_t st = OCC_OK;
  with_rp(b.rp, [&](auto RPc) {
    constexpr int RP = decltype(RPc)::value;
    with_dt_vec(b.dt, b.vec, [&](auto DTc, auto VECc) {
      constexpr int DT = decltype(DTc)::value;
      constexpr bool VEC = decltype(VECc)::value;
      auto LB = [&](const char* name, auto kern, int64_t blocks, int threads, auto... extra) {
        if (st != OCC_OK) return;
        st = launch(name, s, [&] {
          hipLaunchKernelGGL(kern, dim3(grid_of(blocks)), dim3(threads), 0, s, table, count,
                             single, extra...);
        });
      };
      auto L = [&](const char* name, auto kern, int64_t blocks, auto... extra) {
        LB(name, kern, blocks, kBlock, extra...);
      };
      if constexpr (RP <= kFusedMaxRank) {
        if (b.fused) {
          if (b.descs[0].r != RP) L("qpad", k_qpad<RP>, b.blocks[K_QPAD]);
          for (int it = 0; it < b.iters; ++it) {
            bool narrow = false;   // a matrix with fewer 32-column K-steps than waves
            for (const Desc& dd : b.descs) narrow = narrow || pm_waves_per_rb(dd.n) < PM_WAVES;
            if (narrow)
              LB("pass_p", k_pm<DT, VEC, RP, RM, true>, b.blocks[K_PASS_P], PM_THREADS);
            else
              LB("pass_p", k_pm<DT, VEC, RP, RM>, b.blocks[K_PASS_P], PM_THREADS);
            // T of each matrix (first `count` blocks) beside Q' = A^T P
            LB("pass_q", k_qm<DT, VEC, RP, RM>, count + b.blocks[K_PASS_Q], QM_THREADS, flags);
            L("q_finish", k_qfin16<RP>, b.blocks[K_QRED] + b.blocks[K_APPLY],
              (int)b.blocks[K_QRED]);
          }
          if (finish) {
            if (write_mhat)
              L("mhat_err", k_mh16<DT, VEC, RP, 0, true, true, false, RM>, b.blocks[K_MHAT]);
            else
              L("err_only", k_mh16<DT, VEC, RP, 0, false, true, false, RM>, b.blocks[K_MHAT]);
          }
          return;
        }
      }
      if constexpr (RP > kFusedMaxRank) {
        // Large-rank path.  With an error buffer to write (fused step) the
        // first left product stores A over it and every later pass reads A
        // back from there; a compress-only call re-reads M and err_prev.
        const bool saved = b.descs[0].err_out != nullptr;
        // bf16 M: left products on bf16 matrix cores with split operands
        constexpr bool X3 = DT == DT_BF16;
        // left products with their A tiles through LDS when every row is
        // 16-byte aligned, every 32-column K-step whole and A has a source.
        // With a row map only the first left product (M and err_prev rows)
        // and the reconstruction (err and M_hat rows) use it: the stored A is
        // compact, so every pass in between is the dense kernel.
        constexpr bool TL = true;
        constexpr int LPT = lp_block_rows(RP, X3) / 32 * kWave;   // threads of a left-product block
        bool whole = VEC;
        for (const Desc& dd : b.descs) whole = whole && dd.n % 32 == 0;
        const bool tiles_merr = whole && b.descs[0].err_in != nullptr;
        L("qpad", k_qpadl<RP>, b.blocks[K_QPAD]);
        for (int it = 0; it < b.iters; ++it) {
          if (!saved) {
            if (tiles_merr)
              LB("pass_p", k_lp<DT, RP, SA_MERR, X3, TL, RM>, b.blocks[K_PASS_P], LPT);
            else
              LB("pass_p", k_lp<DT, RP, SA_MERR, X3, false, RM>, b.blocks[K_PASS_P], LPT);
          } else if (it == 0) {
            if (tiles_merr)
              LB("pass_p_first", k_lp<DT, RP, SA_MERR_SAVE, X3, TL, RM>, b.blocks[K_PASS_P], LPT);
            else
              LB("pass_p_first", k_lp<DT, RP, SA_MERR_SAVE, X3, false, RM>, b.blocks[K_PASS_P], LPT);
          } else {
            if (whole)
              LB("pass_p_a", k_lp<DT_F32, RP, SA_SAVED, X3, TL>, b.blocks[K_PASS_P], LPT);
            else
              LB("pass_p_a", k_lp<DT_F32, RP, SA_SAVED, X3, false>, b.blocks[K_PASS_P], LPT);
          }
          L("gram", k_lg<RP, 0>, b.blocks[K_PGRAM]);
          L("gram_sum", k_gsum<RP, 0>, b.blocks[K_GSUM]);
          LB("chol", k_lchol<RP, 0>, count, LC_THREADS, flags);
          L("apply", k_lapply<RP, 0>, b.blocks[K_APPLY]);
          L("gram2", k_lg<RP, 1>, b.blocks[K_GRAM2]);
          L("gram_sum2", k_gsum<RP, 1>, b.blocks[K_GSUM]);
          LB("chol2", k_lchol<RP, 1>, count, LC_THREADS, flags);
          L("apply2", k_lapply<RP, 1>, b.blocks[K_APPLY]);
          if constexpr (X3) {
            // the stored A through LDS tiles under the same conditions
            constexpr int QXT = lqx_waves(RP) * kWave;
            if (saved && whole)
              LB("pass_q_a", k_lqx<DT_F32, RP, SA_SAVED, TL>, b.blocks[K_PASS_Q], QXT);
            else if (saved)
              LB("pass_q_a", k_lqx<DT_F32, RP, SA_SAVED, false>, b.blocks[K_PASS_Q], QXT);
            else
              LB("pass_q", k_lqx<DT, RP, SA_MERR, false, RM>, b.blocks[K_PASS_Q], QXT);
          } else {
            if (saved && whole)
              L("pass_q_a", k_lq<DT_F32, RP, SA_SAVED, TL>, b.blocks[K_PASS_Q]);
            else if (saved)
              L("pass_q_a", k_lq<DT_F32, RP, SA_SAVED, false>, b.blocks[K_PASS_Q]);
            else
              L("pass_q", k_lq<DT, RP, SA_MERR, false, RM>, b.blocks[K_PASS_Q]);
          }
          L("q_reduce", k_qredl<RP>, b.blocks[K_QRED]);
        }
        if (finish) {
          // bf16 M: the reconstruction on bf16 matrix cores with split operands
          if constexpr (X3) {
            if (write_mhat)
              L("mhat_err_a", k_mlx<RP, 0, true, true, false, RM>, b.blocks[K_MHAT]);
            else
              L("err_only_a", k_mlx<RP, 0, false, true, false, RM>, b.blocks[K_MHAT]);
          } else {
            if (write_mhat)
              L("mhat_err_a", k_ml<DT_F32, RP, SA_SAVED, 0, true, true, false, RM>, b.blocks[K_MHAT]);
            else
              L("err_only_a", k_ml<DT_F32, RP, SA_SAVED, 0, false, true, false, RM>, b.blocks[K_MHAT]);
          }
        }
      }
    });
  });
  return st;
}

occ_status_t run_batch(const Batch& b, void* ws, uint32_t* flags, bool finish, bool write_mhat,
                       hipStream_t s) {
  return b.descs[0].rmap ? run_batch_t<true>(b, ws, flags, finish, write_mhat, s)
                         : run_batch_t<false>(b, ws, flags, finish, write_mhat, s);
}

}  // namespace

namespace {

// Stand-alone decompression: M_hat = P Q^T with the reconstruction kernels of
// the fused step (SRC 1: factors from the caller's P and Q).
template <bool OUTBF>
occ_status_t decompress_impl(const float* P, const float* Q, int64_t m, int64_t n, int rank,
                             bool split, void* M_hat, int64_t ldh, hipStream_t s) {
  OCC_TRY(check_shape(m, n, ldh));
  if (rank < 1 || rank > OCC_MAX_RANK || rank > m || rank > n) return OCC_E_RANK;
  if (!P || !Q || !M_hat) return OCC_E_NULL;
  const size_t es = OUTBF ? 2 : 4;
  if (!aligned(P, 4) || !aligned(Q, 4) || !aligned(M_hat, es)) return OCC_E_ALIGN;
  std::vector<Span> spans = {span2d(P, m, rank, rank, 4, false), span2d(Q, n, rank, rank, 4, false),
                             span2d(M_hat, m, n, ldh, es, true)};
  if (overlaps(spans)) return OCC_E_ALIAS;
  const int rp = padded_rank(rank);
  const Tiling t = make_tiling(m, n, rp);
  Desc d{};
  d.m = (int32_t)m;
  d.n = (int32_t)n;
  d.r = rank;
  d.P = const_cast<float*>(P);
  d.Q = const_cast<float*>(Q);
  d.Mhat = (float*)M_hat;
  d.ldh = (int32_t)ldh;
  d.mr = t.mr;
  // 4 consecutive elements per vector store: 16 bytes (fp32) or 8 (bf16)
  const bool vec = aligned(M_hat, 4 * es) && ldh % 4 == 0;
  d.vec = vec ? 1 : 0;
  occ_status_t st = OCC_OK;
  with_rp(rp, [&](auto RPc) {
    constexpr int RP = decltype(RPc)::value;
    st = launch(OUTBF ? "decompress_bf16" : "decompress", s, [&] {
      const dim3 grid(grid_of(t.blocks[K_MHAT]));
      if constexpr (RP > kFusedMaxRank) {
        if (split)
          hipLaunchKernelGGL((k_mlx<RP, 1, true, false, OUTBF>), grid, dim3(kBlock), 0, s,
                             (const Desc*)nullptr, 1, d);
        else
          hipLaunchKernelGGL((k_ml<DT_F32, RP, SA_SAVED, 1, true, false, OUTBF>), grid,
                             dim3(kBlock), 0, s, (const Desc*)nullptr, 1, d);
      } else if (vec) {
        // same code as the fused step's reconstruction pass
        hipLaunchKernelGGL((k_mh16<DT_F32, true, RP, 1, true, false, OUTBF>), grid, dim3(kBlock),
                           0, s, (const Desc*)nullptr, 1, d);
      } else {
        hipLaunchKernelGGL((k_mh16<DT_F32, false, RP, 1, true, false, OUTBF>), grid,
                           dim3(kBlock), 0, s, (const Desc*)nullptr, 1, d);
      }
    });
  });
  return st;
}

}  // namespace

namespace {

// Leading dimension of the compact stored A of a row-sparse step: whole
// 128-byte lines per row.
int64_t compact_ld(int64_t cols) { return round_up(cols, 32); }

// Plan of a row-sparse step: the compressed matrix is the n_rows x cols
// matrix of the listed rows; its workspace regions are those of a dense
// matrix of that shape, followed by the validated copy of the row list.
occ_status_t plan_rows(const occ_mat_t* mat, int64_t n_rows, int rank, int iters, unsigned flags,
                       Batch& b, size_t& rows_off) {
  if (!mat) return OCC_E_NULL;
  if (flags & ~(unsigned)OCC_NO_MHAT) return OCC_E_FLAGS;
  if (mat->m_dtype != OCC_F32 && mat->m_dtype != OCC_BF16) return OCC_E_DTYPE;
  OCC_TRY(check_shape(mat->rows, mat->cols, mat->ldm));
  if (n_rows < 0 || n_rows > mat->rows) return OCC_E_SHAPE;
  if (n_rows == 0) {
    if (rank < 1 || rank > OCC_MAX_RANK || rank > mat->cols) return OCC_E_RANK;
    if (iters < 1 || iters > OCC_MAX_ITERS) return OCC_E_ITERS;
    b = Batch{};
    b.ws_needed = kHeaderBytes;
    rows_off = 0;
    return OCC_OK;
  }
  occ_mat_t a = *mat;
  a.rows = n_rows;
  OCC_TRY(plan_batch(&a, 1, rank, iters, flags, nullptr, 0, true, b));
  rows_off = b.ws_needed;
  b.ws_needed += align_up((size_t)n_rows * 4);
  if (!b.fused) {
    // large-rank path: the first left product stores A = M + err_prev of the
    // listed rows here (n_rows x compact_ld), every later pass reads it back
    b.ws_needed += align_up((size_t)n_rows * compact_ld(mat->cols) * 4);
  }
  return OCC_OK;
}

}  // namespace

namespace {

// Device address of `scratch` on the current device, looked up once per device
// with that device current; nullptr if the runtime cannot provide it.
void* noalloc_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return nullptr;
  }
  static std::mutex mu;
  static std::map<int, void*> addr;
  std::lock_guard<std::mutex> lock(mu);
  const auto it = addr.find(dev);
  if (it != addr.end()) return it->second;
  void* p = nullptr;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
    (void)hipGetLastError();
    return nullptr;
  }
  addr[dev] = p;
  return p;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================
extern "C" {

int occ_abi_version(void) { return OCC_ABI_VERSION; }

const char* occ_status_str(int status) {
  switch (status) {
    case OCC_OK: return "ok";
    case OCC_E_NULL: return "a required pointer is NULL";
    case OCC_E_SHAPE: return "invalid shape or leading dimension";
    case OCC_E_RANK: return "rank out of range (1 <= rank <= min(rows, cols), rank <= 128)";
    case OCC_E_ITERS: return "iters out of range (1 <= iters <= 64)";
    case OCC_E_DTYPE: return "unknown or mixed M dtype";
    case OCC_E_ALIGN: return "pointer not aligned to its element size";
    case OCC_E_ALIAS: return "buffers overlap";
    case OCC_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case OCC_E_HIP: return "HIP runtime or kernel launch failure";
    case OCC_E_FLAGS: return "unknown flag bit";
    default: return "unknown status";
  }
}

size_t occ_workspace_bytes(const occ_mat_t* mats, int count, int rank, int iters) {
  Batch b;
  if (plan_batch(mats, count, rank, iters, 0, nullptr, 0, true, b) != OCC_OK) return 0;
  return b.ws_needed;
}

size_t occ_compress_workspace_bytes(int64_t m, int64_t n, int m_dtype, int rank, int iters) {
  occ_mat_t a{};
  a.rows = m;
  a.cols = n;
  a.ldm = n;
  a.m_dtype = m_dtype;
  return occ_workspace_bytes(&a, 1, rank, iters);
}

occ_status_t occ_workspace_init(void* ws, size_t ws_bytes, occ_stream_t stream) {
  if (!ws) return OCC_E_NULL;
  if (!aligned(ws, kAlign) || ws_bytes < kHeaderBytes) return OCC_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  return launch("ws_init", s, [&] {
    hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(256), 0, s, (uint32_t*)ws,
                       (int)(kHeaderBytes / 4));
  });
}

occ_status_t occ_step_batched(const occ_mat_t* mats, int count, int rank, int iters,
                              unsigned flags, void* ws, size_t ws_bytes, occ_stream_t stream) {
  Batch b;
  OCC_TRY(plan_batch(mats, count, rank, iters, flags, ws, ws_bytes, false, b));
  return run_batch(b, ws, (uint32_t*)ws, true, !(flags & OCC_NO_MHAT), (hipStream_t)stream);
}

occ_status_t occ_step_batched_noalloc(const occ_mat_t* mats, int count, int rank, int iters,
                                      unsigned flags, uint32_t* flags_out, occ_stream_t stream) {
  Batch b;
  OCC_TRY(plan_batch(mats, count, rank, iters, flags, nullptr, 0, true, b));
  if (b.ws_needed > OCC_NOALLOC_MAX_BYTES) return OCC_E_WORKSPACE;
  if (flags_out && !aligned(flags_out, 4)) return OCC_E_ALIGN;
  void* ws = noalloc_scratch();
  if (!ws) return OCC_E_HIP;
  OCC_TRY(plan_batch(mats, count, rank, iters, flags, ws, OCC_NOALLOC_MAX_BYTES, false, b));
  // the scratch header is the flag word when the caller passes none; nothing
  // else in it needs to start at zero (every region is written before it is read)
  uint32_t* fl = flags_out ? flags_out : (uint32_t*)ws;
  return run_batch(b, ws, fl, true, !(flags & OCC_NO_MHAT), (hipStream_t)stream);
}

occ_status_t occ_step(const occ_mat_t* mat, int rank, int iters, unsigned flags, void* ws,
                      size_t ws_bytes, occ_stream_t stream) {
  if (!mat) return OCC_E_NULL;
  return occ_step_batched(mat, 1, rank, iters, flags, ws, ws_bytes, stream);
}

size_t occ_step_rows_workspace_bytes(int64_t n_rows, int64_t cols, int m_dtype, int rank,
                                     int iters) {
  occ_mat_t a{};
  a.rows = std::max<int64_t>(n_rows, 1);
  a.cols = cols;
  a.ldm = cols;
  a.m_dtype = m_dtype;
  Batch b;
  size_t rows_off = 0;
  if (plan_rows(&a, n_rows, rank, iters, 0, b, rows_off) != OCC_OK) return 0;
  return b.ws_needed;
}

occ_status_t occ_step_rows(const occ_mat_t* mat, const int32_t* rows, int64_t n_rows, int rank,
                           int iters, unsigned flags, void* ws, size_t ws_bytes,
                           occ_stream_t stream) {
  Batch b;
  size_t rows_off = 0;
  OCC_TRY(plan_rows(mat, n_rows, rank, iters, flags, b, rows_off));
  const occ_mat_t& a = *mat;
  const bool write_mhat = !(flags & OCC_NO_MHAT);
  OCC_TRY(check_shape(a.rows, a.cols, a.lde));
  if (write_mhat) OCC_TRY(check_shape(a.rows, a.cols, a.ldh));
  if (!a.M || !a.err || !a.Q || (n_rows > 0 && (!a.P || !rows)) || (write_mhat && !a.M_hat))
    return OCC_E_NULL;
  if (!ws) return OCC_E_WORKSPACE;
  if (!aligned(ws, kAlign) || ws_bytes < b.ws_needed) return OCC_E_WORKSPACE;
  const int dt = a.m_dtype;
  const size_t es = elem_size(dt);
  if (!aligned(a.M, es) || !aligned(a.err, 4) || !aligned(a.Q, 4) || (a.P && !aligned(a.P, 4)) ||
      (rows && !aligned(rows, 4)) || (write_mhat && !aligned(a.M_hat, 4)))
    return OCC_E_ALIGN;
  std::vector<Span> spans = {span2d(a.M, a.rows, a.cols, a.ldm, es, false),
                             span2d(a.err, a.rows, a.cols, a.lde, 4, true),
                             span2d(a.Q, a.cols, rank, rank, 4, true),
                             {(uintptr_t)ws, (uintptr_t)ws + b.ws_needed, true}};
  if (n_rows > 0) {
    spans.push_back(span2d(a.P, n_rows, rank, rank, 4, true));
    spans.push_back(span2d(rows, 1, n_rows, n_rows, 4, false));
  }
  if (write_mhat) spans.push_back(span2d(a.M_hat, a.rows, a.cols, a.ldh, 4, true));
  if (overlaps(spans)) return OCC_E_ALIAS;
  hipStream_t s = (hipStream_t)stream;
  uint32_t* fl = (uint32_t*)ws;
  if (n_rows == 0) {
    const int64_t nq = a.cols * rank;
    return launch("rows_empty", s, [&] {
      hipLaunchKernelGGL(k_rows_empty, dim3((unsigned)std::min<int64_t>(cdiv(nq, kBlock), 1024)),
                         dim3(kBlock), 0, s, a.Q, nq, fl);
    });
  }
  int32_t* rmap = (int32_t*)((char*)ws + rows_off);
  OCC_TRY(launch("rows_check", s, [&] {
    hipLaunchKernelGGL(k_rows_check, dim3((unsigned)std::min<int64_t>(cdiv(n_rows, kBlock), 1024)),
                       dim3(kBlock), 0, s, rows, n_rows, (int32_t)a.rows, rmap, fl);
  }));
  finalize_regions(b, ws);
  Desc& d = b.descs[0];
  if (dt != OCC_BF16) d.qbf = nullptr;
  d.M = a.M;
  d.err_in = a.err;
  d.err_out = a.err;
  d.P = a.P;
  d.Q = a.Q;
  d.Mhat = write_mhat ? a.M_hat : nullptr;
  d.ldm = (int32_t)a.ldm;
  d.lde_in = (int32_t)a.lde;
  d.lde_out = (int32_t)a.lde;
  d.ldh = write_mhat ? (int32_t)a.ldh : 0;
  d.rmap = rmap;
  if (!b.fused) {
    // stored A compact in the workspace; the reconstruction writes err
    d.err_out = (float*)((char*)ws + rows_off + align_up((size_t)n_rows * 4));
    d.lde_out = (int32_t)compact_ld(a.cols);
    d.err_fin = a.err;
    d.lde_fin = (int32_t)a.lde;
  }
  b.vec = aligned(a.M, 16) && a.ldm % (dt == OCC_BF16 ? 8 : 4) == 0 && aligned(a.err, 16) &&
          a.lde % 4 == 0 && (!write_mhat || (aligned(a.M_hat, 16) && a.ldh % 4 == 0));
  d.vec = b.vec ? 1 : 0;
  return run_batch(b, ws, fl, true, write_mhat, s);
}

occ_status_t occ_compress(const void* M, int m_dtype, int64_t m, int64_t n, int64_t ldm,
                          const float* err_prev, int64_t lde, float* P, float* Q, int rank,
                          int iters, void* ws, size_t ws_bytes, occ_stream_t stream) {
  if (m_dtype != OCC_F32 && m_dtype != OCC_BF16) return OCC_E_DTYPE;
  OCC_TRY(check_shape(m, n, ldm));
  if (err_prev) OCC_TRY(check_shape(m, n, lde));
  OCC_TRY(check_rank_iters(rank, iters, m, n));
  if (!M || !P || !Q) return OCC_E_NULL;
  occ_mat_t a{};
  a.M = M;
  a.m_dtype = m_dtype;
  a.rows = m;
  a.cols = n;
  a.ldm = ldm;
  a.lde = err_prev ? lde : n;
  a.P = P;
  a.Q = Q;
  Batch b;
  OCC_TRY(plan_batch(&a, 1, rank, iters, OCC_NO_MHAT, nullptr, 0, true, b));
  if (!ws) return OCC_E_WORKSPACE;
  if (!aligned(ws, kAlign) || ws_bytes < b.ws_needed) return OCC_E_WORKSPACE;
  const size_t es = elem_size(m_dtype);
  if (!aligned(M, es) || !aligned(P, 4) || !aligned(Q, 4) || (err_prev && !aligned(err_prev, 4)))
    return OCC_E_ALIGN;
  std::vector<Span> spans = {span2d(M, m, n, ldm, es, false), span2d(P, m, rank, rank, 4, true),
                             span2d(Q, n, rank, rank, 4, true),
                             {(uintptr_t)ws, (uintptr_t)ws + b.ws_needed, true}};
  if (err_prev) spans.push_back(span2d(err_prev, m, n, lde, 4, false));
  if (overlaps(spans)) return OCC_E_ALIAS;
  finalize_regions(b, ws);
  Desc& d = b.descs[0];
  if (m_dtype != OCC_BF16) d.qbf = nullptr;
  d.M = M;
  d.P = P;
  d.Q = Q;
  d.ldm = (int32_t)ldm;
  d.err_in = err_prev;
  d.lde_in = err_prev ? (int32_t)lde : 0;
  d.err_out = nullptr;
  d.Mhat = nullptr;
  b.vec = aligned(M, 16) && ldm % (m_dtype == OCC_BF16 ? 8 : 4) == 0 &&
          (!err_prev || (aligned(err_prev, 16) && lde % 4 == 0));
  d.vec = b.vec ? 1 : 0;
  return run_batch(b, ws, (uint32_t*)ws, false, false, (hipStream_t)stream);
}

occ_status_t occ_decompress(const float* P, const float* Q, int64_t m, int64_t n, int rank,
                            float* M_hat, int64_t ldh, occ_stream_t stream) {
  return decompress_impl<false>(P, Q, m, n, rank, false, M_hat, ldh, (hipStream_t)stream);
}

occ_status_t occ_decompress_ex(const float* P, const float* Q, int64_t m, int64_t n, int rank,
                               unsigned flags, void* M_hat, int64_t ldh, occ_stream_t stream) {
  if (flags & ~(unsigned)(OCC_DEC_SPLIT_BF16 | OCC_DEC_OUT_BF16)) return OCC_E_FLAGS;
  const bool split = (flags & OCC_DEC_SPLIT_BF16) != 0;
  if (flags & OCC_DEC_OUT_BF16)
    return decompress_impl<true>(P, Q, m, n, rank, split, M_hat, ldh, (hipStream_t)stream);
  return decompress_impl<false>(P, Q, m, n, rank, split, M_hat, ldh, (hipStream_t)stream);
}

occ_status_t occ_err_update(const void* M, int m_dtype, int64_t m, int64_t n, int64_t ldm,
                            const float* err_prev, int64_t lde, const float* M_hat, int64_t ldh,
                            float* err_new, occ_stream_t stream) {
  if (m_dtype != OCC_F32 && m_dtype != OCC_BF16) return OCC_E_DTYPE;
  OCC_TRY(check_shape(m, n, ldm));
  OCC_TRY(check_shape(m, n, ldh));
  OCC_TRY(check_shape(m, n, lde));
  if (!M || !M_hat || !err_new) return OCC_E_NULL;
  const size_t es = elem_size(m_dtype);
  if (!aligned(M, es) || !aligned(M_hat, 4) || !aligned(err_new, 4) ||
      (err_prev && !aligned(err_prev, 4)))
    return OCC_E_ALIGN;
  const int64_t lde_new = lde;
  std::vector<Span> spans = {span2d(M, m, n, ldm, es, false), span2d(M_hat, m, n, ldh, 4, false),
                             span2d(err_new, m, n, lde_new, 4, true)};
  const bool inplace = err_prev && (const void*)err_prev == (const void*)err_new;
  if (err_prev && !inplace) spans.push_back(span2d(err_prev, m, n, lde, 4, false));
  if (overlaps(spans)) return OCC_E_ALIAS;
  Desc d{};
  d.M = M;
  d.m = (int32_t)m;
  d.n = (int32_t)n;
  d.ldm = (int32_t)ldm;
  d.err_in = err_prev;
  d.lde_in = err_prev ? (int32_t)lde : 0;
  d.Mhat = const_cast<float*>(M_hat);
  d.ldh = (int32_t)ldh;
  d.err_out = err_new;
  d.lde_out = (int32_t)lde_new;
  const int64_t total = m * n;
  const unsigned grid = (unsigned)std::min<int64_t>((total + kBlock - 1) / kBlock, 16384);
  hipStream_t s = (hipStream_t)stream;
  return launch("err_update", s, [&] {
    if (m_dtype == OCC_BF16)
      hipLaunchKernelGGL(k_err_update<DT_BF16>, dim3(grid), dim3(kBlock), 0, s, d);
    else
      hipLaunchKernelGGL(k_err_update<DT_F32>, dim3(grid), dim3(kBlock), 0, s, d);
  });
}

occ_status_t occ_get_flags(void* ws, uint32_t* flags_out, int clear, occ_stream_t stream) {
  if (!ws || !flags_out) return OCC_E_NULL;
  if (!aligned(ws, kAlign)) return OCC_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint32_t v = 0;
  if (hipMemcpyAsync(&v, ws, sizeof(v), hipMemcpyDeviceToHost, s) != hipSuccess) return OCC_E_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return OCC_E_HIP;
  *flags_out = v;
  if (clear) {
    return launch("flags_clear", s, [&] {
      hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(64), 0, s, (uint32_t*)ws, 1);
    });
  }
  return OCC_OK;
}

occ_status_t occ_pipeline_1f1b(int n_stages, int n_micro, double t_fwd, double t_bwd,
                               double t_p2p, double* bwd_done, double* t_end) {
  if (!bwd_done) return OCC_E_NULL;
  if (n_stages < 1 || n_micro < 1 || n_stages > 4096 || n_micro > (1 << 20)) return OCC_E_SHAPE;
  for (double t : {t_fwd, t_bwd, t_p2p})
    if (!(t >= 0.0) || !std::isfinite(t)) return OCC_E_SHAPE;
  return pipeline_1f1b(n_stages, n_micro, t_fwd, t_bwd, t_p2p, bwd_done, t_end) ? OCC_OK
                                                                               : OCC_E_SHAPE;
}

occ_status_t occ_sc_select(const occ_stage_t* stages, int n_stages, int max_compressed,
                           uint8_t* selected, int* n_selected, double* t_end) {
  if (!stages || !selected) return OCC_E_NULL;
  if (n_stages < 1 || max_compressed < 0) return OCC_E_SHAPE;
  std::vector<StageTimes> st(n_stages);
  for (int s = 0; s < n_stages; ++s) {
    const occ_stage_t& x = stages[s];
    for (double t : {x.bwd_done, x.comm, x.comm_compressed, x.compress})
      if (!(t >= 0.0) || !std::isfinite(t)) return OCC_E_SHAPE;
    st[s] = {x.bwd_done, x.comm, x.comm_compressed, x.compress};
  }
  const double end = sc_select(st.data(), n_stages, max_compressed, selected, n_selected);
  if (t_end) *t_end = end;
  return OCC_OK;
}

occ_status_t occ_profile_begin(void) {
  for (auto& r : g_prof.recs) {
    g_prof.free_events.push_back(r.a);
    g_prof.free_events.push_back(r.b);
  }
  g_prof.recs.clear();
  g_prof.on = true;
  return OCC_OK;
}

occ_status_t occ_profile_end(occ_kernel_time_t* out, int max, int* n_out) {
  g_prof.on = false;
  std::vector<occ_kernel_time_t> agg;
  for (auto& r : g_prof.recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return OCC_E_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return OCC_E_HIP;
    auto it = std::find_if(agg.begin(), agg.end(),
                           [&](const occ_kernel_time_t& k) { return std::strcmp(k.name, r.name) == 0; });
    if (it == agg.end()) {
      occ_kernel_time_t k{};
      std::snprintf(k.name, sizeof(k.name), "%s", r.name);
      agg.push_back(k);
      it = agg.end() - 1;
    }
    it->launches += 1;
    it->total_ms += ms;
  }
  for (auto& r : g_prof.recs) {
    g_prof.free_events.push_back(r.a);
    g_prof.free_events.push_back(r.b);
  }
  g_prof.recs.clear();
  if (n_out) *n_out = (int)agg.size();
  if (out)
    for (int i = 0; i < (int)agg.size() && i < max; ++i) out[i] = agg[i];
  return OCC_OK;
}

}  // extern "C"
