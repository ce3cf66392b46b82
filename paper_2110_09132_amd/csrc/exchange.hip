// The receiver side of the sparse-gradient exchange (Sec. 4.1.1 / 4.1.2: the
// coalesced rows go to their owners with an AlltoAll; an owner sums what it
// receives for the same row), simulated on one device for P workers.
//
//  1. exchange_offsets: from the P send layouts (worker w's rows for owner p
//     at [send_offsets[w][p], send_offsets[w][p + 1])), where each block lands
//     at its receiver: owner-major, senders in order inside an owner.  One
//     workgroup; P <= 1024.
//  2. exchange_rows: a P x P block transpose of ids and rows.  Each row finds
//     its owner block by binary search over its sender's offsets, which each
//     workgroup first copies to LDS with the receivers' destinations.
// The merge of the received runs is the owner-major coalesce with a token
// count read on the device (the received total), in coalesce.hip.
#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 1024;       // one thread per owner in exchange_offsets
constexpr int kRowThreads = 256;
constexpr int kRowsInFlight = 8;

// counts[w][p], from the offsets of sender w, clamped into [0, cap] and made monotone
__device__ __forceinline__ int block_count(const int32_t* __restrict__ offs, int P, int cap, int w, int p) {
  const int32_t* o = offs + static_cast<size_t>(w) * (P + 1);
  const int a = min(max(o[p], 0), cap);
  const int b = min(max(o[p + 1], a), cap);
  return b - a;
}

__global__ __launch_bounds__(kThreads) void exchange_offsets_kernel(const int32_t* __restrict__ send_offsets, int P,
                                                                    int cap, int32_t* __restrict__ recv_offsets,
                                                                    int32_t* __restrict__ recv_total) {
  __shared__ uint32_t base[kThreads];
  __shared__ uint32_t wsum[kThreads / kWave];
  const int p = threadIdx.x;
  uint32_t total = 0;
  if (p < P)
    for (int w = 0; w < P; ++w) total += static_cast<uint32_t>(block_count(send_offsets, P, cap, w, p));
  base[p] = total;
  __syncthreads();
  const uint32_t all = block_exclusive_scan<kThreads>(base, P, wsum);
  if (p < P) {
    uint32_t run = base[p];
    int32_t* r = recv_offsets + static_cast<size_t>(p) * (P + 1);
    for (int w = 0; w < P; ++w) {
      r[w] = static_cast<int32_t>(run);
      run += static_cast<uint32_t>(block_count(send_offsets, P, cap, w, p));
    }
    r[P] = static_cast<int32_t>(run);
  }
  if (p == 0) *recv_total = static_cast<int32_t>(all);
}

// Row k of sender w (k < its sent rows) goes to receiver p, the owner block
// holding k, at recv_offsets[p][w] + (k - send_offsets[w][p]).  L lanes per row.
template <typename VecT>
__global__ __launch_bounds__(kRowThreads) void exchange_rows_kernel(
    const int32_t* __restrict__ send_ids, const VecT* __restrict__ send_rows, const int32_t* __restrict__ send_offsets,
    int P, int cap, int Dv, int log2L, const int32_t* __restrict__ recv_offsets, int32_t* __restrict__ recv_ids,
    VecT* __restrict__ recv_rows) {
  // the sender's offsets, block sizes and destinations, once per workgroup in LDS
  // (a row then finds its block by a binary search in LDS, not in memory)
  __shared__ int32_t s_o[kThreads + 1];   // send_offsets[w][p]
  __shared__ int32_t s_cnt[kThreads];     // rows of block p (clamped)
  __shared__ int32_t s_dst[kThreads];     // where receiver p puts them: recv_offsets[p][w]
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int sub = static_cast<int>(lane_id()) >> log2L;
  const int cl = static_cast<int>(lane_id()) & (L - 1);
  const int w = blockIdx.y;  // the sender
  const int32_t* o = send_offsets + static_cast<size_t>(w) * (P + 1);
  for (int p = threadIdx.x; p <= P; p += kRowThreads) {
    s_o[p] = o[p];
    if (p < P) {
      s_cnt[p] = block_count(send_offsets, P, cap, w, p);
      s_dst[p] = recv_offsets[static_cast<size_t>(p) * (P + 1) + w];
    }
  }
  __syncthreads();
  const int sent = min(max(s_o[P], 0), cap);
  const long long wave = (static_cast<long long>(blockIdx.x) * kRowThreads + threadIdx.x) / kWave;
  const long long nwaves = static_cast<long long>(gridDim.x) * (kRowThreads / kWave);
  const long long step = static_cast<long long>(rpw) * kRowsInFlight;
  for (long long r0 = wave * step; r0 < sent; r0 += nwaves * step) {
    int64_t dst[kRowsInFlight];
    int64_t src[kRowsInFlight];
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const long long k = r0 + u * rpw + sub;
      const int kc = static_cast<int>(k < sent ? k : sent - 1);
      // owner block of row kc: the last p with o[p] <= kc (offsets are ascending)
      int lo = 0, hi = P - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_o[mid] <= kc) lo = mid; else hi = mid - 1;
      }
      const int a = min(max(s_o[lo], 0), cap);
      const int off = kc - a;  // inside the block unless the offsets are malformed
      src[u] = static_cast<int64_t>(w) * cap + kc;
      dst[u] = (k < sent && off >= 0 && off < s_cnt[lo]) ? static_cast<int64_t>(s_dst[lo]) + off : -1;
    }
    if (cl == 0) {
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u)
        if (dst[u] >= 0) recv_ids[dst[u]] = send_ids[src[u]];
    }
    for (int c = cl; c < Dv; c += L) {
      VecT v[kRowsInFlight];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) v[u] = send_rows[static_cast<size_t>(src[u]) * Dv + c];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u)
        if (dst[u] >= 0) recv_rows[static_cast<size_t>(dst[u]) * Dv + c] = v[u];
    }
  }
}

}  // namespace

hipError_t launch_exchange(const int32_t* send_ids, const float* send_rows, const int32_t* send_offsets, int P,
                           int cap, int D, int32_t* recv_ids, float* recv_rows, int32_t* recv_offsets,
                           int32_t* recv_total, hipStream_t stream) {
  hipLaunchKernelGGL(exchange_offsets_kernel, dim3(1), dim3(kThreads), 0, stream, send_offsets, P, cap, recv_offsets,
                     recv_total);
  if (cap == 0) return hipGetLastError();
  const auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  const bool vec4 = (D % 4 == 0) && al16(send_rows) && al16(recv_rows);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kRowThreads / kWave);
  const dim3 grid(grid_for((cap + rows_per_block - 1) / rows_per_block, 65535), P);
  if (vec4)
    hipLaunchKernelGGL(exchange_rows_kernel<float4>, grid, dim3(kRowThreads), 0, stream, send_ids,
                       reinterpret_cast<const float4*>(send_rows), send_offsets, P, cap, Dv, rl.log2_lanes,
                       recv_offsets, recv_ids, reinterpret_cast<float4*>(recv_rows));
  else
    hipLaunchKernelGGL(exchange_rows_kernel<float>, grid, dim3(kRowThreads), 0, stream, send_ids, send_rows,
                       send_offsets, P, cap, Dv, rl.log2_lanes, recv_offsets, recv_ids, recv_rows);
  return hipGetLastError();
}

}  // namespace emb
