// Pack the coalesced rows by owner shard (Sec. 4.1.1 / 4.1.2): the layout an
// AlltoAll of sparse gradients sends, one contiguous block per owner.
//
// A stable partition by owner is one radix pass whose digit is the owner
// (P <= 1024 owners plus one bin for rows that are not sent):
//  1. per-tile owner histograms (LDS atomics); the owner digit of every row
//     is kept, so the owner table is read once,
//  2. per tile: global base of each owner (sum of earlier tiles and owners) +
//     stable rank inside the tile (wave ballots, as in the sort) -> the send
//     slot of every row; ids are written there, the slot is kept for step 3;
//     tile 0 writes send_counts / send_offsets,
//  3. the rows are copied to their slots (contiguous row reads and writes).
#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 4;
constexpr int kTile = kThreads * kItems;  // rows per tile
constexpr int kMaxOwners = 1024;
constexpr int kBinsMax = kMaxOwners + 1;
constexpr int kRowsInFlight = 8;

__device__ __forceinline__ int clamp_rows(const int32_t* num_unique, int cap) {
  const int u = num_unique[0];
  return u < 0 ? 0 : (u > cap ? cap : u);
}

// Owner of a row, or P when the row is not sent.  The owner table is read
// at a clamped index so the load never depends on a branch.
__device__ __forceinline__ uint32_t owner_of(int32_t id, const int32_t* __restrict__ row_owner, int64_t V, int P,
                                             int& flags) {
  const bool id_ok = id >= 0 && id < V;
  const int32_t o = row_owner[id_ok ? id : 0];
  if (!id_ok) {
    flags |= EMB_DEV_ID_OUT_OF_RANGE;
    return static_cast<uint32_t>(P);
  }
  if (o < 0 || o >= P) {
    flags |= EMB_DEV_OWNER_OUT_OF_RANGE;
    return static_cast<uint32_t>(P);
  }
  return static_cast<uint32_t>(o);
}

__global__ __launch_bounds__(kThreads) void pack_hist_kernel(const int32_t* __restrict__ uniq_ids,
                                                             const int32_t* __restrict__ num_unique, int cap,
                                                             const int32_t* __restrict__ row_owner, int64_t V, int P,
                                                             uint32_t* __restrict__ tile_hist,
                                                             uint16_t* __restrict__ digit_of, int32_t* status) {
  __shared__ uint32_t h[kBinsMax];
  const int bins = P + 1;
  for (int i = threadIdx.x; i < bins; i += kThreads) h[i] = 0;
  __syncthreads();
  const int U = clamp_rows(num_unique, cap);
  const int base = blockIdx.x * kTile;
  int flags = 0;
  if (base < U) {
    int32_t id[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) id[r] = uniq_ids[min(base + r * kThreads + static_cast<int>(threadIdx.x), U - 1)];
    uint32_t d[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) d[r] = owner_of(id[r], row_owner, V, P, flags);
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
      const int k = base + r * kThreads + static_cast<int>(threadIdx.x);
      if (k < U) {
        atomicAdd(&h[d[r]], 1u);
        digit_of[k] = static_cast<uint16_t>(d[r]);
      }
    }
  }
  if (flags != 0) raise_flag(status, flags);
  __syncthreads();
  for (int i = threadIdx.x; i < bins; i += kThreads) tile_hist[static_cast<size_t>(blockIdx.x) * bins + i] = h[i];
}

__global__ __launch_bounds__(kThreads) void pack_scatter_kernel(
    const int32_t* __restrict__ uniq_ids, const int32_t* __restrict__ num_unique, int cap,
    const uint16_t* __restrict__ digit_of, int P, int owner_bits, const uint32_t* __restrict__ tile_hist,
    int ntiles, int32_t* __restrict__ send_ids, int32_t* __restrict__ slot_of, int32_t* __restrict__ send_counts,
    int32_t* __restrict__ send_offsets) {
  __shared__ uint32_t cnt[(kThreads / kWave) * kBinsMax];
  __shared__ uint32_t dstart[kBinsMax], colall[kBinsMax], gbase[kBinsMax];
  __shared__ uint32_t red_all[kBinsMax], red_bef[kBinsMax];
  __shared__ uint32_t wsum[kThreads / kWave];
  const int bins = P + 1;
  const int tile = blockIdx.x;
  const int base = tile * kTile;
  const int w = threadIdx.x / kWave;
  const int U = clamp_rows(num_unique, cap);

  int32_t id[kItems];
  uint32_t dig[kItems], lpos[kItems];
  bool valid[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int k = base + w * kItems * kWave + r * kWave + static_cast<int>(lane_id());
    const int kc = max(min(k, U - 1), 0);
    valid[r] = k < U;
    id[r] = uniq_ids[kc];
    dig[r] = digit_of[kc];
    if (!valid[r]) dig[r] = 0u;
  }
  const uint32_t total =
      tile_global_bases<kThreads>(tile_hist, ntiles, tile, bins, colall, gbase, red_all, red_bef, wsum);
  tile_stable_rank<kThreads, kItems>(dig, valid, bins, owner_bits, cnt, dstart, wsum, lpos);
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int k = base + w * kItems * kWave + r * kWave + static_cast<int>(lane_id());
    if (!valid[r]) continue;
    const uint32_t d = dig[r];
    if (d == static_cast<uint32_t>(P)) {
      slot_of[k] = -1;
    } else {
      const uint32_t dest = gbase[d] + (lpos[r] - dstart[d]);
      send_ids[dest] = id[r];
      slot_of[k] = static_cast<int32_t>(dest);
    }
  }
  if (tile == 0) {
    for (int p = threadIdx.x; p < P; p += kThreads) {
      send_counts[p] = static_cast<int32_t>(colall[p]);
      send_offsets[p] = static_cast<int32_t>(gbase[p]);  // tile 0: nothing before it
    }
    if (threadIdx.x == 0) send_offsets[P] = static_cast<int32_t>(total - colall[P]);
  }
}

template <typename VecT>
__global__ __launch_bounds__(kThreads) void pack_rows_kernel(const VecT* __restrict__ uniq_grad,
                                                             const int32_t* __restrict__ num_unique, int cap,
                                                             const int32_t* __restrict__ slot_of, int Dv, int log2L,
                                                             VecT* __restrict__ send_rows) {
  const int U = clamp_rows(num_unique, cap);
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int sub = lane_id() >> log2L;
  const int cl = lane_id() & (L - 1);
  const long long wave = (static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x) / kWave;
  const long long nwaves = static_cast<long long>(gridDim.x) * (kThreads / kWave);
  const long long step = static_cast<long long>(rpw) * kRowsInFlight;
  for (long long r0 = wave * step; r0 < U; r0 += nwaves * step) {
    int32_t dst[kRowsInFlight];
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const long long k = r0 + u * rpw + sub;
      dst[u] = slot_of[k < U ? k : U - 1];
      if (k >= U) dst[u] = -1;
    }
    for (int c = cl; c < Dv; c += L) {
      VecT v[kRowsInFlight];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        const long long k = r0 + u * rpw + sub;
        v[u] = uniq_grad[static_cast<size_t>(k < U ? k : U - 1) * Dv + c];
      }
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u)
        if (dst[u] >= 0) send_rows[static_cast<size_t>(dst[u]) * Dv + c] = v[u];
    }
  }
}

struct PackWs {
  uint32_t* tile_hist;
  int32_t* slot_of;
  uint16_t* digit_of;
  size_t bytes;
};

PackWs carve(void* base, int cap, int P) {
  Carver cv{static_cast<char*>(base)};
  const size_t ntiles = (static_cast<size_t>(cap) + kTile - 1) / kTile;
  PackWs w;
  w.tile_hist = cv.take<uint32_t>((ntiles > 0 ? ntiles : 1) * static_cast<size_t>(P + 1));
  w.slot_of = cv.take<int32_t>(static_cast<size_t>(cap > 0 ? cap : 1));
  w.digit_of = cv.take<uint16_t>(static_cast<size_t>(cap > 0 ? cap : 1));
  w.bytes = cv.size();
  return w;
}

__global__ void empty_pack_kernel(int P, int32_t* send_counts, int32_t* send_offsets) {
  for (int p = threadIdx.x; p <= P; p += blockDim.x) {
    if (p < P) send_counts[p] = 0;
    send_offsets[p] = 0;
  }
}

}  // namespace

size_t pack_workspace_bytes(int cap_rows, int P) { return carve(nullptr, cap_rows, P).bytes; }

hipError_t launch_pack(const int32_t* uniq_ids, const float* uniq_grad, const int32_t* num_unique, int cap_rows,
                       int D, const int32_t* row_owner, int64_t V, int P, int32_t* send_ids, float* send_rows,
                       int32_t* send_counts, int32_t* send_offsets, void* workspace, int32_t* status,
                       hipStream_t stream) {
  if (cap_rows == 0) {
    hipLaunchKernelGGL(empty_pack_kernel, dim3(1), dim3(256), 0, stream, P, send_counts, send_offsets);
    return hipGetLastError();
  }
  PackWs ws = carve(workspace, cap_rows, P);
  const int ntiles = (cap_rows + kTile - 1) / kTile;
  int owner_bits = 0;
  while ((1 << owner_bits) <= P) ++owner_bits;  // digits 0..P
  hipLaunchKernelGGL(pack_hist_kernel, dim3(ntiles), dim3(kThreads), 0, stream, uniq_ids, num_unique, cap_rows,
                     row_owner, V, P, ws.tile_hist, ws.digit_of, status);
  hipLaunchKernelGGL(pack_scatter_kernel, dim3(ntiles), dim3(kThreads), 0, stream, uniq_ids, num_unique, cap_rows,
                     ws.digit_of, P, owner_bits, ws.tile_hist, ntiles, send_ids, ws.slot_of, send_counts,
                     send_offsets);
  const bool vec4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(uniq_grad) % 16 == 0) &&
                    (reinterpret_cast<uintptr_t>(send_rows) % 16 == 0);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((cap_rows + rows_per_block - 1) / rows_per_block, kMaxBlocks);
  if (vec4)
    hipLaunchKernelGGL(pack_rows_kernel<float4>, dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<const float4*>(uniq_grad), num_unique, cap_rows, ws.slot_of, Dv,
                       rl.log2_lanes, reinterpret_cast<float4*>(send_rows));
  else
    hipLaunchKernelGGL(pack_rows_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, uniq_grad, num_unique,
                       cap_rows, ws.slot_of, Dv, rl.log2_lanes, send_rows);
  return hipGetLastError();
}

}  // namespace emb
