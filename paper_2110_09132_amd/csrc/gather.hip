// Forward lookup (Sec. 4.1.1): out[t][:] = table[ids[t]][:].
//
// Each wave owns a contiguous range of output rows.  A row is handled by
// L = min(64, 2^ceil(log2(D / VEC))) lanes, so a wave covers 64 / L rows per
// step.  The ids of 64 rows come in one coalesced load (lane l holds the id of
// row l) and reach their lanes by shuffle; rows are processed in groups of
// kRowsInFlight steps, and the table loads of the next group are issued before
// the current group is stored (two register buffers used in turn), so each
// lane keeps two groups of independent 16-byte loads in flight.  Reads are whole table rows (cached: the
// update of the same step reads most of them again), writes contiguous rows (streaming stores).
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsInFlight = 8;

// kWide: rows of more than one column step (Dv > 64).  The wave's column steps
// and row groups then run as one sequence of tiles, so that the loads of the
// next column step are in flight while the current one is stored (with few
// rows per wave, a single group per column step would otherwise wait for its
// loads step after step).
template <typename VecT, bool kWide>
__global__ __launch_bounds__(kThreads) void gather_kernel(const VecT* __restrict__ table, int64_t V, int Dv,
                                                          int log2L, const int32_t* __restrict__ ids, int T,
                                                          VecT* __restrict__ out, int32_t* status) {
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int lane = static_cast<int>(lane_id());
  const int sub = lane >> log2L;
  const int cl = lane & (L - 1);
  const int wave = uniform(static_cast<int>(blockIdx.x) * (kThreads / kWave) + static_cast<int>(threadIdx.x / kWave));
  const int nwaves = static_cast<int>(gridDim.x) * (kThreads / kWave);
  // rows of this wave: [r0, r1), a multiple of the rows one step covers
  const long long step_rows = static_cast<long long>(rpw) * kRowsInFlight;
  long long per = (static_cast<long long>(T) + nwaves - 1) / nwaves;
  per = (per + step_rows - 1) / step_rows * step_rows;
  const long long r0 = static_cast<long long>(wave) * per;
  const long long r1 = min(static_cast<long long>(T), r0 + per);
  bool bad = false;
  for (long long c0 = r0; c0 < r1; c0 += kWave) {  // 64 rows per id load
    const int n = static_cast<int>(min(static_cast<long long>(kWave), r1 - c0));
    const int32_t idreg = ids[min(c0 + lane, static_cast<long long>(T) - 1)];
    bad |= lane < n && (idreg < 0 || idreg >= V);
    // group g covers chunk rows [g * step_rows, (g + 1) * step_rows)
    const int ngroups = static_cast<int>((n + step_rows - 1) / step_rows);
    auto row_id = [&](int g, int u) {  // table row of this lane's row u of group g, -1 if none
      const int j = g * static_cast<int>(step_rows) + u * rpw + sub;
      const int id = __shfl(idreg, min(j, kWave - 1), kWave);
      return (j < n && id >= 0 && id < V) ? id : -1;
    };
    if constexpr (kWide) {
      // tiles (column step k: cb = k * L; row group g) in one sequence, two buffers in turn
      struct Tile {
        VecT v[kRowsInFlight];
        int id[kRowsInFlight];
        int c, g;
        bool live;
      } A, B;
      const int nsteps = (Dv + L - 1) / L;
      const int ntiles = nsteps * ngroups;
      int lk = 0, lg = 0, lq = 0;  // the next tile to load
      // a tile past the last one reads row 0 (one cached line) and is not stored
      auto load = [&](Tile& x) {
        x.live = lq < ntiles;
        x.g = x.live ? lg : 0;
        const int cb = (x.live ? lk : 0) * L;
        x.c = min(cb + cl, Dv - 1);
        const bool cok = cb + cl < Dv;
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          x.id[u] = x.live ? row_id(x.g, u) : -1;
          x.v[u] = table[static_cast<size_t>(x.id[u] < 0 ? 0 : x.id[u]) * Dv + x.c];
        }
        x.live = x.live && cok;
        ++lq;
        if (++lg == ngroups) {
          lg = 0;
          ++lk;
        }
      };
      auto store = [&](const Tile& x) {
        if (!x.live) return;
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          const int j = x.g * static_cast<int>(step_rows) + u * rpw + sub;
          if (j < n) store_stream(&out[static_cast<size_t>(c0 + j) * Dv + x.c], x.id[u] < 0 ? VecT{} : x.v[u]);
        }
      };
      load(A);
      for (int q = 0; q < ntiles; q += 2) {
        load(B);
        store(A);
        load(A);
        store(B);
      }
      continue;
    }
    // column steps are uniform across the wave (the shuffles need every lane)
    for (int cb = 0; cb < Dv; cb += L) {
      const int c = min(cb + cl, Dv - 1);
      const bool cok = cb + cl < Dv;
      // two register buffers used in turn (every index is a compile-time
      // constant, and no loaded value is copied, so loads stay in flight)
      struct Group {
        VecT v[kRowsInFlight];
        int id[kRowsInFlight];
      } A, B;
      // loads are unconditional: past the last group they read row 0 and are not stored
      auto load = [&](int g, Group& x) {
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          x.id[u] = row_id(g, u);
          x.v[u] = table[static_cast<size_t>(x.id[u] < 0 ? 0 : x.id[u]) * Dv + c];
        }
      };
      auto store = [&](int g, const Group& x) {
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
          const int j = g * static_cast<int>(step_rows) + u * rpw + sub;
          if (j < n && cok) store_stream(&out[static_cast<size_t>(c0 + j) * Dv + c], x.id[u] < 0 ? VecT{} : x.v[u]);
        }
      };
      load(0, A);
      for (int g = 0; g < ngroups; g += 2) {
        load(g + 1, B);
        store(g, A);
        load(g + 2, A);
        store(g + 1, B);
      }
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

}  // namespace

hipError_t launch_gather(const float* table, int64_t V, int D, const int32_t* ids, int T, float* out,
                         int32_t* status, hipStream_t stream, hipEvent_t done) {
  if (T == 0) return done != nullptr ? hipEventRecord(done, stream) : hipSuccess;
  const bool vec4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(table) % 16 == 0) &&
                    (reinterpret_cast<uintptr_t>(out) % 16 == 0);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((T + rows_per_block - 1) / rows_per_block, kMaxBlocks);
  const bool wide = Dv > kWave;
  if (vec4) {
    const auto* tv = reinterpret_cast<const float4*>(table);
    auto* ov = reinterpret_cast<float4*>(out);
    if (wide)
      hipExtLaunchKernelGGL((gather_kernel<float4, true>), dim3(grid), dim3(kThreads), 0, stream, nullptr, done, 0, tv,
                            V, Dv, rl.log2_lanes, ids, T, ov, status);
    else
      hipExtLaunchKernelGGL((gather_kernel<float4, false>), dim3(grid), dim3(kThreads), 0, stream, nullptr, done, 0, tv,
                            V, Dv, rl.log2_lanes, ids, T, ov, status);
  } else {
    if (wide)
      hipExtLaunchKernelGGL((gather_kernel<float, true>), dim3(grid), dim3(kThreads), 0, stream, nullptr, done, 0,
                            table, V, Dv, rl.log2_lanes, ids, T, out, status);
    else
      hipExtLaunchKernelGGL((gather_kernel<float, false>), dim3(grid), dim3(kThreads), 0, stream, nullptr, done, 0,
                            table, V, Dv, rl.log2_lanes, ids, T, out, status);
  }
  return hipGetLastError();
}

}  // namespace emb
