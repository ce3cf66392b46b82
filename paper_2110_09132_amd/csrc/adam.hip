// Row-wise (lazy) Adam on the rows a shard owns (Sec. 4.1.1, Sec. 5.7;
// Kingma & Ba, Algorithm 1).  One pass over the listed rows: for each element
// read g, w, m, v once and write w, m, v once; rows not listed are not touched.
// Rows are mapped to lanes as in the gather (L lanes per row, several rows in
// flight per wave); table rows are random 4*D-byte blocks, gradient rows are
// contiguous.
#include <cmath>

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
  const int sub = lane_id() >> log2L;
  const int cl = lane_id() & (L - 1);
  const long long wave = (static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x) / kWave;
  const long long nwaves = static_cast<long long>(gridDim.x) * (kThreads / kWave);
  const long long step = static_cast<long long>(rpw) * kRowsInFlight;
  bool bad = false;
  for (long long r0 = lo + wave * step; r0 < hi; r0 += nwaves * step) {
    // All loads come from clamped, always-valid addresses and are issued
    // together; only rows that exist and are valid are stored.
    int32_t rid[kRowsInFlight];
    long long src[kRowsInFlight];
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const long long i = r0 + u * rpw + sub;
      src[u] = i < hi ? i : hi - 1;
      rid[u] = row_ids[src[u]];
    }
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const bool live = r0 + u * rpw + sub < hi;
      const bool ok = rid[u] >= 0 && rid[u] < V;
      bad |= live && !ok;
      if (!live || !ok) rid[u] = -1;
    }
    for (int col = cl; col < Dv; col += L) {
      VecT g[kRowsInFlight], w[kRowsInFlight], m[kRowsInFlight], s[kRowsInFlight];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        const size_t e = static_cast<size_t>(rid[u] < 0 ? 0 : rid[u]) * Dv + col;
        g[u] = rows[static_cast<size_t>(src[u]) * Dv + col];
        w[u] = W[e];
        m[u] = M[e];
        s[u] = S[e];
      }
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        if (rid[u] >= 0) {
          adam_vec(g[u], w[u], m[u], s[u], c);
          const size_t e = static_cast<size_t>(rid[u]) * Dv + col;
          W[e] = w[u];
          M[e] = m[u];
          S[e] = s[u];
        }
      }
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

}  // namespace

hipError_t launch_adam(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int D, const int32_t* row_ids,
                       const float* rows, const int32_t* offsets, int shard_begin, int shard_end, int cap_rows,
                       const AdamCoeffs& c, int32_t* status, hipStream_t stream) {
  if (cap_rows == 0 || shard_begin == shard_end) return hipSuccess;
  const auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  const bool vec4 = (D % 4 == 0) && al16(table) && al16(exp_avg) && al16(exp_avg_sq) && al16(rows);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((cap_rows + rows_per_block - 1) / rows_per_block, 8192);
  if (vec4)
    hipLaunchKernelGGL(adam_kernel<float4>, dim3(grid), dim3(kThreads), 0, stream, reinterpret_cast<float4*>(table),
                       reinterpret_cast<float4*>(exp_avg), reinterpret_cast<float4*>(exp_avg_sq), V, Dv,
                       rl.log2_lanes, row_ids, reinterpret_cast<const float4*>(rows), offsets, shard_begin, shard_end,
                       cap_rows, c, status);
  else
    hipLaunchKernelGGL(adam_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, table, exp_avg, exp_avg_sq, V, Dv,
                       rl.log2_lanes, row_ids, rows, offsets, shard_begin, shard_end, cap_rows, c, status);
  return hipGetLastError();
}

}  // namespace emb
