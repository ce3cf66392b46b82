// Forward lookup (Sec. 4.1.1): out[t][:] = table[ids[t]][:].
//
// A row is handled by L = min(64, 2^ceil(log2(D / VEC))) lanes; a wave covers
// 64 / L rows per step and keeps kRowsInFlight steps of loads in flight before
// storing, so every lane has several independent 16-byte loads outstanding.
// Reads are whole table rows (contiguous), writes are contiguous output rows.
#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsInFlight = 8;

template <typename VecT>
__global__ __launch_bounds__(kThreads) void gather_kernel(const VecT* __restrict__ table, int64_t V, int Dv,
                                                          int log2L, const int32_t* __restrict__ ids, int T,
                                                          VecT* __restrict__ out, int32_t* status) {
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int sub = lane_id() >> log2L;
  const int cl = lane_id() & (L - 1);
  const long long wave = (static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x) / kWave;
  const long long nwaves = static_cast<long long>(gridDim.x) * (kThreads / kWave);
  const long long rows_per_step = static_cast<long long>(rpw) * kRowsInFlight;
  bool bad = false;
  for (long long r0 = wave * rows_per_step; r0 < T; r0 += nwaves * rows_per_step) {
    // Loads are issued unconditionally from clamped, always-valid addresses so
    // that all of them are in flight together; only the stores are predicated.
    int32_t id[kRowsInFlight];
    bool live[kRowsInFlight];
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const long long row = r0 + u * rpw + sub;
      live[u] = row < T;
      id[u] = ids[live[u] ? row : T - 1];
    }
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const bool ok = id[u] >= 0 && id[u] < V;
      bad |= live[u] && !ok;
      if (!ok) id[u] = -1;
    }
    for (int c = cl; c < Dv; c += L) {
      VecT v[kRowsInFlight];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u)
        v[u] = table[static_cast<size_t>(id[u] < 0 ? 0 : id[u]) * Dv + c];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        const long long row = r0 + u * rpw + sub;
        if (live[u]) out[static_cast<size_t>(row) * Dv + c] = id[u] < 0 ? VecT{} : v[u];
      }
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

}  // namespace

hipError_t launch_gather(const float* table, int64_t V, int D, const int32_t* ids, int T, float* out,
                         int32_t* status, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const bool vec4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(table) % 16 == 0) &&
                    (reinterpret_cast<uintptr_t>(out) % 16 == 0);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((T + rows_per_block - 1) / rows_per_block, 4096);
  if (vec4) {
    hipLaunchKernelGGL(gather_kernel<float4>, dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<const float4*>(table), V, Dv, rl.log2_lanes, ids, T,
                       reinterpret_cast<float4*>(out), status);
  } else {
    hipLaunchKernelGGL(gather_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, table, V, Dv, rl.log2_lanes,
                       ids, T, out, status);
  }
  return hipGetLastError();
}

}  // namespace emb
