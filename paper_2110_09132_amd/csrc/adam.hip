// Row-wise (lazy) Adam on the rows a shard owns (Sec. 4.1.1, Sec. 5.7;
// Kingma & Ba, Algorithm 1).  One pass over the listed rows: for each element
// read g, w, m, v once and write w, m, v once; rows not listed are not touched.
// Rows are mapped to lanes as in the gather (L lanes per row); table rows are
// random 4*D-byte blocks, gradient rows are contiguous.  W, m, v go back with
// streaming stores and m, v come in with streaming loads (nothing else in the
// step touches them); the loads of W and of the gradient rows are plain (the
// table rows were just read by the lookup, the gradient rows just written by
// the reduction, and both are often still cached).
#include <cmath>

#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
// Row steps per tile: two (the loads of the next tile are in flight while the
// current one is stored); with rows of one column step each wave takes four
// tiles' worth of rows.  Measured in the overlapped steps (update beside the
// next step's reduction): the low-duplication workload (63.5k rows of 1 KB)
// 144.0 us per step with four-row tiles and one tile's worth of rows per wave,
// 138.3 us with two-row tiles and four (eight, sixteen or three-row variants
// in between); the shared-vocabulary workload (7.1k rows of 2 KB) 56.1 -> 53.7
// us with two-row tiles for wide rows too, the 4 KB-row workloads unchanged.
//
// The grid is sized for the row capacity; the rows actually listed (known
// only on the device) are spread over enough waves that each takes at most
// four tiles, and over no fewer than the resident waves: a short list (6.3k
// rows of 1 KB) then runs in one round of resident workgroups instead of
// being packed into the first of several (update alone 15.0 -> 13.5 us, its
// overlapped step 47.3 -> 45.7 us; 63.5k rows unchanged).
constexpr int kRowsInFlight = 2;
constexpr int kNarrowTilesPerWave = 4;

__device__ __forceinline__ float adam_elem(float g, float& w, float& m, float& v, const AdamCoeffs& c) {
  m = c.beta1 * m + c.one_minus_beta1 * g;
  v = c.beta2 * v + c.one_minus_beta2 * (g * g);
  const float denom = sqrtf(v * c.inv_bc2) + c.eps;
  w = w - c.step_size * (m / denom);
  return w;
}

__device__ __forceinline__ void adam_vec(const float4& g, float4& w, float4& m, float4& v, const AdamCoeffs& c) {
  adam_elem(g.x, w.x, m.x, v.x, c);
  adam_elem(g.y, w.y, m.y, v.y, c);
  adam_elem(g.z, w.z, m.z, v.z, c);
  adam_elem(g.w, w.w, m.w, v.w, c);
}
__device__ __forceinline__ void adam_vec(const float& g, float& w, float& m, float& v, const AdamCoeffs& c) {
  adam_elem(g, w, m, v, c);
}

// Waves of this kernel that can be resident at once: 256 CUs x 4 SIMDs x 2
// waves (its register use allows two per SIMD).
constexpr int kResidentWaves = 2048;

// LDS reserved (and not used) by each workgroup of the narrow-row update with
// vector rows (the scalar path, for odd D, uses few registers and is left alone): with
// 160 KB of LDS per CU, at most two of its workgroups, two waves per SIMD,
// share a CU.  Its registers alone would allow three; at three the update
// crowds out the reduction of the next step that runs beside it on another
// stream, and the step gets slower (measured: 167 -> 200 us per step with
// coalesce and pack as separate calls, 147 -> 149 us with the owner-major call).
constexpr size_t kNarrowOccupancyLds = 56 * 1024;

// Row ranges of few wide rows are shared by cs waves, each taking every cs-th
// column step, so that about kResidentWaves waves have work; each wave keeps
// at least two column steps where the rows allow it, so that its loads of the
// next step are in flight while the current one is stored.
__device__ __forceinline__ int column_share(int rows, int step_rows, int ncols, int all_waves) {
  const int ranges = max((rows + step_rows - 1) / step_rows, 1);
  const float want = static_cast<float>(kResidentWaves) / static_cast<float>(ranges);
  return static_cast<int>(fminf(fmaxf(rintf(want), 1.0f), static_cast<float>(min(ncols, all_waves))));
}

// Each wave owns a contiguous range of the listed rows (with wide rows, every
// cs-th column step of one).  The row ids of 64 rows come in one coalesced
// load and reach their lanes by shuffle; rows are processed in tiles of
// kRowsInFlight row steps, and the loads (g, w, m, v) of the next tile are
// issued before the current tile is computed and stored.  kWide: rows of more
// than one column step (Dv > 64); the tiles then run over the wave's column
// steps as well, one sequence.
template <typename VecT, bool kWide>
__global__ __launch_bounds__(kThreads) void adam_kernel(VecT* __restrict__ W, VecT* __restrict__ M,
                                                        VecT* __restrict__ S, int64_t V, int Dv, int log2L,
                                                        const int32_t* __restrict__ row_ids,
                                                        const VecT* __restrict__ rows,
                                                        const int32_t* __restrict__ offsets, int sb, int se, int cap,
                                                        AdamCoeffs cval, const AdamCoeffs* __restrict__ coeffs_dev,
                                                        int32_t* status) {
  const AdamCoeffs c = coeffs_dev != nullptr ? *coeffs_dev : cval;
  int lo = offsets[sb], hi = offsets[se];
  lo = max(0, min(lo, cap));
  hi = max(lo, min(hi, cap));
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int lane = static_cast<int>(lane_id());
  const int sub = lane >> log2L;
  const int cl = lane & (L - 1);
  const int step_rows = rpw * kRowsInFlight;
  const int all_waves = static_cast<int>(gridDim.x) * (kThreads / kWave);
  const int wave_all = uniform(static_cast<int>(blockIdx.x) * (kThreads / kWave) + static_cast<int>(threadIdx.x / kWave));
  const int ncols = kWide ? (Dv + L - 1) / L : 1;
  int cs = 1, wave = wave_all, part = 0, nwaves = all_waves;
  if (kWide) {
    cs = uniform(column_share(hi - lo, step_rows, ncols, all_waves));  // 1 <= cs <= all_waves
    wave = wave_all / cs;  // row range (waves past the last range find it empty)
    part = wave_all - wave * cs;
    nwaves = all_waves / cs;
  }
  if (!kWide)  // the listed rows over at least the resident waves, at most kNarrowTilesPerWave tiles each
    nwaves = min(all_waves, max(kResidentWaves, (hi - lo + kNarrowTilesPerWave * step_rows - 1) /
                                                    (kNarrowTilesPerWave * step_rows)));
  int per = (hi - lo + nwaves - 1) / nwaves;
  per = (per + step_rows - 1) / step_rows * step_rows;
  const long long r0 = lo + static_cast<long long>(wave) * per;
  const long long r1 = min(static_cast<long long>(hi), r0 + per);
  // two register buffers used in turn; every index below is a compile-time constant
  struct Buf {
    VecT g[kRowsInFlight], w[kRowsInFlight], m[kRowsInFlight], s[kRowsInFlight];
    int rid[kRowsInFlight];
    int col;
    bool cok;
  } A, B;
  bool bad = false;
  for (long long c0 = r0; c0 < r1; c0 += kWave) {  // 64 rows per id load
    const int n = static_cast<int>(min(static_cast<long long>(kWave), r1 - c0));
    const int32_t ridreg = row_ids[min(c0 + lane, static_cast<long long>(hi) - 1)];
    bad |= lane < n && (ridreg < 0 || ridreg >= V);
    const int ngroups = (n + step_rows - 1) / step_rows;
    auto apply = [&](Buf& x, int col, bool cok) {
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        if (x.rid[u] >= 0 && cok) {
          adam_vec(x.g[u], x.w[u], x.m[u], x.s[u], c);
          const size_t e = static_cast<size_t>(x.rid[u]) * Dv + col;
          store_stream(&W[e], x.w[u]);
          store_stream(&M[e], x.m[u]);
          store_stream(&S[e], x.s[u]);
        }
      }
    };
    // Loads are unconditional (a group or tile past the last one reads row 0 of
    // the table, one cached line for every wave, and stores nothing): with a
    // branch around them the compiler could not count the loads in flight and
    // would wait for all of them.  (Re-reading real rows instead would fetch
    // the moments twice: they come in with streaming loads.)
    if constexpr (!kWide) {  // one column step: the row groups in turn
      const int col = min(cl, Dv - 1);
      const bool cok = cl < Dv;
      auto load = [&](int grp, Buf& x) {
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          const int j = grp * step_rows + u * rpw + sub;
          const int r = __shfl(ridreg, min(j, kWave - 1), kWave);
          x.rid[u] = (j < n && r >= 0 && r < V) ? r : -1;
          const size_t e = static_cast<size_t>(x.rid[u] < 0 ? 0 : x.rid[u]) * Dv + col;
          x.g[u] = rows[static_cast<size_t>(c0 + min(j, n - 1)) * Dv + col];
          x.w[u] = W[e];
          x.m[u] = load_stream(&M[e]);
          x.s[u] = load_stream(&S[e]);
        }
      };
      load(0, A);
      for (int grp = 0; grp < ngroups; grp += 2) {
        load(grp + 1, B);
        apply(A, col, cok);
        load(grp + 2, A);
        apply(B, col, cok);
      }
    } else {  // tiles (column step k: cb = (part + k * cs) * L; row group grp) in one sequence
      const int nsteps = (ncols - part + cs - 1) / cs;
      const int ntiles = nsteps * ngroups;
      int lk = 0, lg = 0, lq = 0;  // the next tile to load
      auto load = [&](Buf& x) {
        const bool live = lq < ntiles;
        const int k = live ? lk : nsteps - 1;
        const int grp = live ? lg : ngroups - 1;
        const int cb = (part + k * cs) * L;
        x.col = min(cb + cl, Dv - 1);
        x.cok = live && cb + cl < Dv;
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          const int j = grp * step_rows + u * rpw + sub;
          const int r = __shfl(ridreg, min(j, kWave - 1), kWave);
          x.rid[u] = (live && j < n && r >= 0 && r < V) ? r : -1;
          const size_t e = static_cast<size_t>(x.rid[u] < 0 ? 0 : x.rid[u]) * Dv + x.col;
          x.g[u] = rows[static_cast<size_t>(c0 + min(j, n - 1)) * Dv + x.col];
          x.w[u] = W[e];
          x.m[u] = load_stream(&M[e]);
          x.s[u] = load_stream(&S[e]);
        }
        ++lq;
        if (++lg == ngroups) {
          lg = 0;
          ++lk;
        }
      };
      load(A);
      for (int q = 0; q < ntiles; q += 2) {
        load(B);
        apply(A, A.col, A.cok);
        load(A);
        apply(B, B.col, B.cok);
      }
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

}  // namespace

hipError_t launch_adam(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int D, const int32_t* row_ids,
                       const float* rows, const int32_t* offsets, int shard_begin, int shard_end, int cap_rows,
                       const AdamCoeffs& c, const AdamCoeffs* coeffs_dev, int32_t* status, hipStream_t stream,
                       hipEvent_t start, hipEvent_t stop) {
  if (cap_rows == 0 || shard_begin == shard_end) return hipSuccess;
  const auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  const bool vec4 = (D % 4 == 0) && al16(table) && al16(exp_avg) && al16(exp_avg_sq) && al16(rows);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const bool wide = Dv > kWave;  // more than one column step per row
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * (kThreads / kWave) * kRowsInFlight *
                                   (wide ? 1 : kNarrowTilesPerWave);
  const unsigned grid = grid_for((cap_rows + rows_per_block - 1) / rows_per_block, kMaxBlocks);
  // Both events are attached to the dispatch, so they time the kernel itself
  // (an attached start event idles the stream a few microseconds longer than a
  // marker before the launch, which would also count the dispatch latency).
#define EMB_ADAM(VT, WIDE)                                                                                        \
  hipExtLaunchKernelGGL((adam_kernel<VT, WIDE>), dim3(grid), dim3(kThreads),                                      \
                        (WIDE) || sizeof(VT) != 16 ? 0 : kNarrowOccupancyLds, stream, start, stop, 0,              \
                        reinterpret_cast<VT*>(table), reinterpret_cast<VT*>(exp_avg),                              \
                        reinterpret_cast<VT*>(exp_avg_sq), V, Dv, rl.log2_lanes, row_ids,                          \
                        reinterpret_cast<const VT*>(rows), offsets, shard_begin, shard_end, cap_rows, c, coeffs_dev, status)
  if (vec4) {
    if (wide)
      EMB_ADAM(float4, true);
    else
      EMB_ADAM(float4, false);
  } else {
    if (wide)
      EMB_ADAM(float, true);
    else
      EMB_ADAM(float, false);
  }
#undef EMB_ADAM
  return hipGetLastError();
}

}  // namespace emb
