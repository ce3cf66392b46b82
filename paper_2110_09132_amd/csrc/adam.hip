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
constexpr int kRowsInFlight = 4;

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

// Each wave owns a contiguous range of the listed rows (or, for few wide rows,
// every cs-th column step of one).  The row ids of 64 rows come in one
// coalesced load and reach their lanes by shuffle; rows are processed in
// groups of kRowsInFlight steps, and the loads (g, w, m, v) of the next group
// are issued before the current group is computed and stored.
template <typename VecT>
__global__ __launch_bounds__(kThreads) void adam_kernel(VecT* __restrict__ W, VecT* __restrict__ M,
                                                        VecT* __restrict__ S, int64_t V, int Dv, int log2L,
                                                        const int32_t* __restrict__ row_ids,
                                                        const VecT* __restrict__ rows,
                                                        const int32_t* __restrict__ offsets, int sb, int se, int cap,
                                                        AdamCoeffs c, int32_t* status) {
  int lo = offsets[sb], hi = offsets[se];
  lo = max(0, min(lo, cap));
  hi = max(lo, min(hi, cap));
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int lane = static_cast<int>(lane_id());
  const int sub = lane >> log2L;
  const int cl = lane & (L - 1);
  const int step_rows = rpw * kRowsInFlight;
  // With few rows (a batch with many repeats) and wide rows, cs waves share a
  // row range, each taking every cs-th column step, so that about every wave
  // of the launch has work.
  const int all_waves = static_cast<int>(gridDim.x) * (kThreads / kWave);
  const int ncols = (Dv + L - 1) / L;
  const int wave_all = uniform(static_cast<int>(blockIdx.x) * (kThreads / kWave) + static_cast<int>(threadIdx.x / kWave));
  int cs = 1, wave = wave_all, part = 0, nwaves = all_waves;
  if (ncols > 1) {
    const float want = static_cast<float>(all_waves) * step_rows / static_cast<float>(max(hi - lo, 1));
    // at most all_waves, so that at least one wave takes each row range
    cs = uniform(static_cast<int>(fminf(fmaxf(want, 1.0f), static_cast<float>(min(ncols, all_waves)))));
    wave = wave_all / cs;  // row range (waves past the last range find it empty)
    part = wave_all - wave * cs;
    nwaves = all_waves / cs;
  }
  int per = (hi - lo + nwaves - 1) / nwaves;
  per = (per + step_rows - 1) / step_rows * step_rows;
  const long long r0 = lo + static_cast<long long>(wave) * per;
  const long long r1 = min(static_cast<long long>(hi), r0 + per);
  bool bad = false;
  for (long long c0 = r0; c0 < r1; c0 += kWave) {  // 64 rows per id load
    const int n = static_cast<int>(min(static_cast<long long>(kWave), r1 - c0));
    const int32_t ridreg = row_ids[min(c0 + lane, static_cast<long long>(hi) - 1)];
    bad |= lane < n && (ridreg < 0 || ridreg >= V);
    const int ngroups = (n + step_rows - 1) / step_rows;
    for (int cb = part * L; cb < Dv; cb += cs * L) {  // uniform column steps (the shuffles need every lane)
      const int col = min(cb + cl, Dv - 1);
      const bool cok = cb + cl < Dv;
      // two register buffers used in turn; every index below is a compile-time constant
      struct Buf {
        VecT g[kRowsInFlight], w[kRowsInFlight], m[kRowsInFlight], s[kRowsInFlight];
        int rid[kRowsInFlight];
      } A, B;
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
      auto apply = [&](Buf& x) {
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
      // Loads are unconditional (a group past the last one reads clamped
      // addresses and stores nothing): with a branch around them the compiler
      // could not count the loads in flight and would wait for all of them.
      load(0, A);
      for (int grp = 0; grp < ngroups; grp += 2) {
        load(grp + 1, B);
        apply(A);
        load(grp + 2, A);
        apply(B);
      }
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

}  // namespace

hipError_t launch_adam(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int D, const int32_t* row_ids,
                       const float* rows, const int32_t* offsets, int shard_begin, int shard_end, int cap_rows,
                       const AdamCoeffs& c, int32_t* status, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  if (cap_rows == 0 || shard_begin == shard_end) return hipSuccess;
  const auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  const bool vec4 = (D % 4 == 0) && al16(table) && al16(exp_avg) && al16(exp_avg_sq) && al16(rows);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((cap_rows + rows_per_block - 1) / rows_per_block, kMaxBlocks);
  // Both events are attached to the dispatch, so they time the kernel itself
  // (an attached start event idles the stream a few microseconds longer than a
  // marker before the launch, which would also count the dispatch latency).
  if (vec4)
    hipExtLaunchKernelGGL(adam_kernel<float4>, dim3(grid), dim3(kThreads), 0, stream, start, stop, 0,
                          reinterpret_cast<float4*>(table), reinterpret_cast<float4*>(exp_avg),
                          reinterpret_cast<float4*>(exp_avg_sq), V, Dv, rl.log2_lanes, row_ids,
                          reinterpret_cast<const float4*>(rows), offsets, shard_begin, shard_end, cap_rows, c, status);
  else
    hipExtLaunchKernelGGL(adam_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, start, stop, 0, table, exp_avg,
                          exp_avg_sq, V, Dv, rl.log2_lanes, row_ids, rows, offsets, shard_begin, shard_end, cap_rows, c,
                          status);
  return hipGetLastError();
}

}  // namespace emb
