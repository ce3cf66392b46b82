// Column-wise partition of the embedding table (Sec. 4.1.1: every process
// holds the whole vocabulary for a slice of the embedding columns, so every
// owner gets the same number of rows; the lookup results travel with a first
// AlltoAll, the sparse gradients with a second one).
//
// Owner p holds float columns [off(p), off(p + 1)), off(p) = floor(p * D / P).
// The column-block layout of capacity C stores block p, the [C][w(p)] slice of
// p's columns (w(p) = off(p + 1) - off(p)), row-major at float offset
// C * off(p); together the blocks fill C * D floats.  With C = V this is the
// partitioned table, one shard per owner.
//
//  column_pack:     rows [R][D]          -> blocks of capacity C  (the gradient
//                   payload: every owner gets all R coalesced ids)
//  column_gather:   shards (C = V), ids  -> blocks of capacity T  (each owner's
//                   lookup of the tokens of every worker)
//  column_assemble: blocks, rows [row0, row0 + R) -> rows [R][D]  (what a
//                   worker holds after the lookup-result AlltoAll)
// All are bit copies.  The default kernels work on tiles of rows staged
// through LDS (column_tile_kernel, below), so that both sides move long
// contiguous runs.  Rows too wide for a tile take column_kernel: a row is
// handled by L lanes; lane l moves the vectors c = l, l + L, ... of its row, so
// the reads and writes of one owner's slice are contiguous; a wave moves
// kRowsInFlight steps of 64 / L rows, all loads before any store.
// When D is a multiple of 4P, every slice is a whole number of float4 and the
// kernels move float4; otherwise single floats.
#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsInFlight = 8;

enum ColumnMode { kPack = 0, kGather = 1, kAssemble = 2 };

// First vector column of owner p (Dv vectors per row).  32-bit: the boundary
// requires D * P < 2^31, so p * Dv and c * P fit.
__device__ __forceinline__ int col_begin(int p, int Dv, int P) {
  return static_cast<int>(static_cast<uint32_t>(p * Dv) / static_cast<uint32_t>(P));
}

// Owner of vector column c: the p with col_begin(p) <= c < col_begin(p + 1).
__device__ __forceinline__ int col_owner(int c, int Dv, int P) {
  int p = static_cast<int>(static_cast<uint32_t>(c * P) / static_cast<uint32_t>(Dv));
  p = min(max(p, 0), P - 1);
  while (p + 1 < P && col_begin(p + 1, Dv, P) <= c) ++p;
  while (p > 0 && col_begin(p, Dv, P) > c) --p;
  return p;
}

// Rows handled: kPack R = *count clamped to [0, cap] (cap if count is null);
// kGather R = cap = T; kAssemble R = cap.  src_cap: capacity of the source
// blocks (kGather: V, kAssemble: the blocks' C); dst_cap: capacity of the
// destination blocks (kPack, kGather).
template <typename VecT, int kMode>
__global__ __launch_bounds__(kThreads) void column_kernel(const VecT* __restrict__ src, VecT* __restrict__ dst,
                                                          const int32_t* __restrict__ ids,
                                                          const int32_t* __restrict__ count, int cap,
                                                          int64_t src_cap, int64_t dst_cap, int64_t row0, int Dv,
                                                          int P, int log2L, int32_t* status) {
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int lane = static_cast<int>(lane_id());
  const int sub = lane >> log2L;
  const int cl = lane & (L - 1);
  const int R = (kMode == kPack && count != nullptr) ? min(max(*count, 0), cap) : cap;
  if (R == 0) return;
  const int64_t group_rows = static_cast<int64_t>(rpw) * kRowsInFlight;
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kThreads / kWave);
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * (kThreads / kWave) + threadIdx.x / kWave;
  bool bad = false;
  for (int64_t g0 = wave * group_rows; g0 < R; g0 += nwaves * group_rows) {
    int64_t row[kRowsInFlight];  // this lane's rows, clamped into [0, R)
    bool live[kRowsInFlight];
    int64_t key[kRowsInFlight];  // kGather: table row (0 for a bad id); else the row
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) {
      const int64_t r = g0 + u * rpw + sub;
      live[u] = r < R;
      row[u] = live[u] ? r : R - 1;
      key[u] = row[u];
      if (kMode == kGather) {
        const int32_t id = ids[row[u]];
        const bool ok = id >= 0 && id < src_cap;
        bad |= live[u] && !ok;
        key[u] = ok ? id : -1;
      }
    }
    for (int c = cl; c < Dv; c += L) {
      const int p = col_owner(c, Dv, P);
      const int a = col_begin(p, Dv, P);
      const int64_t w = col_begin(p + 1, Dv, P) - a;
      const int64_t k = c - a;
      VecT v[kRowsInFlight];
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        size_t s;
        if (kMode == kPack) s = static_cast<size_t>(row[u]) * Dv + c;
        else if (kMode == kGather) s = static_cast<size_t>(src_cap * a + (key[u] < 0 ? 0 : key[u]) * w + k);
        else s = static_cast<size_t>(src_cap * a + (row0 + row[u]) * w + k);
        v[u] = src[s];
      }
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) {
        if (!live[u]) continue;
        size_t d;
        if (kMode == kAssemble) d = static_cast<size_t>(row[u]) * Dv + c;
        else d = static_cast<size_t>(dst_cap * a + row[u] * w + k);
        dst[d] = (kMode == kGather && key[u] < 0) ? VecT{} : v[u];
      }
    }
  }
  if (kMode == kGather && __any(bad) && lane == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
}

// Tiled form (the default): a workgroup takes a tile of n <= TR consecutive
// rows.  Each owner's part of the tile is one contiguous run of n * w(p) units
// in block p (rows r0 .. r0 + n - 1 of the block), and each row one contiguous
// run of Dv units on the row-major side:
// pack:   rows -> LDS in row order (whole tile rows), LDS -> blocks in owner order;
// join:   blocks -> LDS in owner order, LDS -> rows in row order;
// lookup: owner order on both sides, no LDS (the shard rows are random anyway;
//         the block runs are written contiguously).
// In owner order wave v takes owners v, v + 4, ...; its lanes walk the owner's
// run (unit k is row k / w, column k % w of the owner's slice), so the owner's
// start and width are wave-uniform.  LDS rows are padded by one unit so that
// the rows of a tile start in different banks.  Threads issue kUnroll loads
// before they store.
constexpr int kTileUnits = 1024;  // units per tile (16 KB of float4)
constexpr int kUnroll = 4;
constexpr int kLdsPad = 1;

template <typename VecT, int kMode>
__global__ __launch_bounds__(kThreads) void column_tile_kernel(const VecT* __restrict__ src, VecT* __restrict__ dst,
                                                               const int32_t* __restrict__ ids,
                                                               const int32_t* __restrict__ count, int cap,
                                                               int64_t src_cap, int64_t dst_cap, int64_t row0,
                                                               int Dv, int P, int TR, int32_t* status) {
  extern __shared__ __align__(16) unsigned char column_lds[];
  VecT* tile = reinterpret_cast<VecT*>(column_lds);
  const int ld = Dv + kLdsPad;
  const int R = (kMode == kPack && count != nullptr) ? min(max(*count, 0), cap) : cap;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * TR;
  if (r0 >= R) return;
  const int n = static_cast<int>(min(static_cast<int64_t>(TR), R - r0));
  const int units = n * Dv;
  const int wv = static_cast<int>(threadIdx.x) / kWave;
  const int lane = static_cast<int>(lane_id());
  bool bad = false;
  if (kMode != kPack) {
    // owner order from the source: blocks (join) or shard rows (lookup)
    for (int p = wv; p < P; p += kThreads / kWave) {
      const int a = uniform(col_begin(p, Dv, P));
      const int w = uniform(col_begin(p + 1, Dv, P) - a);
      const int run = n * w;
      for (int k0 = lane; k0 < run; k0 += kWave * kUnroll) {
        VecT v[kUnroll];
        int rr[kUnroll], jj[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int k = min(k0 + u * kWave, run - 1);  // clamped: past the run re-reads its last unit
          rr[u] = k / w;
          jj[u] = k - rr[u] * w;
          if (kMode == kGather) {
            const int32_t id = ids[r0 + rr[u]];
            const bool ok = id >= 0 && id < src_cap;
            bad |= !ok && k0 + u * kWave < run;
            v[u] = src[static_cast<size_t>(src_cap * a + static_cast<int64_t>(ok ? id : 0) * w + jj[u])];
            if (!ok) v[u] = VecT{};
          } else {
            v[u] = src[static_cast<size_t>(src_cap * a + (row0 + r0 + rr[u]) * w + jj[u])];
          }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          if (k0 + u * kWave >= run) continue;
          if (kMode == kGather) dst[static_cast<size_t>(dst_cap * a + (r0 + rr[u]) * w + jj[u])] = v[u];
          else tile[rr[u] * ld + a + jj[u]] = v[u];
        }
      }
    }
    if (kMode == kGather) {
      if (__any(bad) && lane == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
      return;
    }
  } else {
    // row order from the rows
    for (int i0 = threadIdx.x; i0 < units; i0 += kThreads * kUnroll) {
      VecT v[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        v[u] = src[static_cast<size_t>(r0) * Dv + min(i0 + u * kThreads, units - 1)];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = i0 + u * kThreads;
        if (i < units) {
          const int r = i / Dv;
          tile[r * ld + (i - r * Dv)] = v[u];
        }
      }
    }
  }
  __syncthreads();
  if (kMode == kPack) {
    // owner order to the blocks
    for (int p = wv; p < P; p += kThreads / kWave) {
      const int a = uniform(col_begin(p, Dv, P));
      const int w = uniform(col_begin(p + 1, Dv, P) - a);
      const int run = n * w;
      for (int k = lane; k < run; k += kWave) {
        const int r = k / w;
        const int j = k - r * w;
        dst[static_cast<size_t>(dst_cap * a + (r0 + r) * w + j)] = tile[r * ld + a + j];
      }
    }
  } else {
    // row order to the rows
    for (int i = threadIdx.x; i < units; i += kThreads) {
      const int r = i / Dv;
      dst[static_cast<size_t>(r0) * Dv + i] = tile[r * ld + (i - r * Dv)];
    }
  }
}

__global__ void column_counts_kernel(const int32_t* __restrict__ count, int cap, int P,
                                     int32_t* __restrict__ send_counts) {
  const int R = count != nullptr ? min(max(*count, 0), cap) : cap;
  for (int p = threadIdx.x; p < P; p += blockDim.x) send_counts[p] = R;
}

template <int kMode>
hipError_t launch_column(const float* src, float* dst, const int32_t* ids, const int32_t* count, int cap,
                         int64_t src_cap, int64_t dst_cap, int64_t row0, int D, int P, int32_t* status,
                         hipStream_t stream) {
  if (cap == 0) return hipSuccess;
  const auto al16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
  const bool vec4 = D % (4 * P) == 0 && al16(src) && al16(dst);
  const int Dv = vec4 ? D / 4 : D;
  const RowLanes rl = row_lanes_for(Dv);
  const long long rows_per_block = static_cast<long long>(rl.rows_per_wave()) * kRowsInFlight * (kThreads / kWave);
  const unsigned grid = grid_for((cap + rows_per_block - 1) / rows_per_block, kMaxBlocks);
  // tiles of up to kTileUnits units (at least one row); rows too wide for a
  // 32 KB tile take the row-per-lanes kernel
  const size_t unit = vec4 ? sizeof(float4) : sizeof(float);
  const int TR = max(1, kTileUnits / Dv);
  const size_t lds = static_cast<size_t>(TR) * (Dv + kLdsPad) * unit;
  if (lds <= 32768) {
    const unsigned tiles = static_cast<unsigned>((static_cast<long long>(cap) + TR - 1) / TR);
    const size_t shm = kMode == kGather ? 0 : lds;
    if (vec4)
      hipLaunchKernelGGL((column_tile_kernel<float4, kMode>), dim3(tiles), dim3(kThreads), shm, stream,
                         reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), ids, count, cap,
                         src_cap, dst_cap, row0, Dv, P, TR, status);
    else
      hipLaunchKernelGGL((column_tile_kernel<float, kMode>), dim3(tiles), dim3(kThreads), shm, stream, src, dst, ids,
                         count, cap, src_cap, dst_cap, row0, Dv, P, TR, status);
    return hipGetLastError();
  }
  if (vec4)
    hipLaunchKernelGGL((column_kernel<float4, kMode>), dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), ids, count, cap,
                       src_cap, dst_cap, row0, Dv, P, rl.log2_lanes, status);
  else
    hipLaunchKernelGGL((column_kernel<float, kMode>), dim3(grid), dim3(kThreads), 0, stream, src, dst, ids, count,
                       cap, src_cap, dst_cap, row0, Dv, P, rl.log2_lanes, status);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_column_pack(const float* rows, const int32_t* num_rows, int cap, int D, int P, float* blocks,
                              int32_t* send_counts, hipStream_t stream) {
  if (send_counts != nullptr)
    hipLaunchKernelGGL(column_counts_kernel, dim3(1), dim3(kThreads), 0, stream, num_rows, cap, P, send_counts);
  return launch_column<kPack>(rows, blocks, nullptr, num_rows, cap, 0, cap, 0, D, P, nullptr, stream);
}

hipError_t launch_column_gather(const float* shards, int64_t V, int D, int P, const int32_t* ids, int T,
                                float* blocks, int32_t* status, hipStream_t stream) {
  return launch_column<kGather>(shards, blocks, ids, nullptr, T, V, T, 0, D, P, status, stream);
}

hipError_t launch_column_assemble(const float* blocks, int64_t C, int64_t row0, int R, int D, int P, float* rows,
                                  hipStream_t stream) {
  return launch_column<kAssemble>(blocks, rows, nullptr, nullptr, R, C, 0, row0, D, P, nullptr, stream);
}

}  // namespace emb
