// Device helpers shared by the kernels of the library (wave64, gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "emb.h"

namespace emb {

constexpr int kWave = 64;

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// Mask of the lanes below this one.
__device__ __forceinline__ uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

__device__ __forceinline__ void raise_flag(int32_t* status, int32_t flag) {
  if (status != nullptr) atomicOr(status, flag);
}

// Streaming (non-temporal) accesses, for data a step touches once: the
// lookup's output rows, the update's stores of W, m, v, the reduction's reads
// of the per-token gradients.  Marking them keeps the caches for what a step
// reads twice (the table rows that its lookup and its update both touch, and
// the reduced rows that the update reads right after the reduction).
typedef float stream_f4 __attribute__((ext_vector_type(4)));
typedef uint32_t stream_u2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_stream(float4* p, const float4& v) {
  __builtin_nontemporal_store(*reinterpret_cast<const stream_f4*>(&v), reinterpret_cast<stream_f4*>(p));
}
__device__ __forceinline__ void store_stream(float* p, float v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ float4 load_stream(const float4* p) {
  const stream_f4 v = __builtin_nontemporal_load(reinterpret_cast<const stream_f4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float load_stream(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ uint2 load_stream(const uint2* p) {
  const stream_u2 v = __builtin_nontemporal_load(reinterpret_cast<const stream_u2*>(p));
  return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint16_t load_stream(const uint16_t* p) { return __builtin_nontemporal_load(p); }

// Wave-uniform value as an SGPR (lets the compiler use scalar loads).
__device__ __forceinline__ int32_t uniform(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// Inclusive prefix sum across the 64 lanes of a wave, with DPP moves (no LDS
// traffic, unlike lane shuffles): shifts by 1, 2, 4 and 8 lanes inside each row
// of 16, then each row's total broadcast to the rows above it (row_bcast:15 to
// rows 1 and 3, row_bcast:31 to rows 2 and 3).  Lanes a move does not reach
// read 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kCtrl, kRowMask, 0xf, false));
}
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += dpp_move<0x111, 0xf>(x);  // row_shr:1
  x += dpp_move<0x112, 0xf>(x);  // row_shr:2
  x += dpp_move<0x114, 0xf>(x);  // row_shr:4
  x += dpp_move<0x118, 0xf>(x);  // row_shr:8
  x += dpp_move<0x142, 0xa>(x);  // row_bcast:15, into rows 1 and 3
  x += dpp_move<0x143, 0xc>(x);  // row_bcast:31, into rows 2 and 3
  return x;
}

// Sum over the 64 lanes of a wave, in every lane.
__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(wave_inclusive_scan(x)), kWave - 1));
}

// Exclusive scan, in place, of a[0..n) in LDS by a block of NT threads.
// `wsum` is LDS scratch of NT/64 words.  Returns the total.  Ends with a barrier.
template <int NT>
__device__ uint32_t block_exclusive_scan(uint32_t* a, int n, uint32_t* wsum) {
  const int per = (n + NT - 1) / NT;
  const int beg = min(static_cast<int>(threadIdx.x) * per, n);
  const int end = min(beg + per, n);
  uint32_t s = 0;
  for (int i = beg; i < end; ++i) s += a[i];
  const uint32_t inc = wave_inclusive_scan(s);
  const int w = threadIdx.x / kWave;
  if (lane_id() == kWave - 1) wsum[w] = inc;
  __syncthreads();
  uint32_t base = 0, total = 0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) {
    const uint32_t v = wsum[i];
    base += (i < w) ? v : 0u;
    total += v;
  }
  uint32_t run = base + inc - s;
  for (int i = beg; i < end; ++i) {
    const uint32_t v = a[i];
    a[i] = run;
    run += v;
  }
  __syncthreads();
  return total;
}

// Stable ranking of small integer digits inside one tile of NT*ITEMS keys.
//
// Key (wave w, round r, lane l) of the tile is input element
// w*ITEMS*64 + r*64 + l, so walking waves, then rounds, then lanes visits the
// keys in input order.  Within a round, lanes holding the same digit are found
// with one ballot per digit bit; the lowest such lane advances the wave's
// counter for that digit.  After all rounds the per-wave counters are turned
// into exclusive offsets across waves and digits, which gives each key its
// position in the tile's stable digit order.
//
// cnt: LDS [NT/64][bins]; dstart: LDS [bins]; wsum: LDS [NT/64].
// On return dstart[d] is the tile-local start of digit d, lpos[] the tile
// position of each valid key, and the function returns the number of valid keys.
// MAXBITS > 0: digits have at most MAXBITS bits, and the ballots run over all
// MAXBITS of them, unrolled (the bits above `bits` are 0 in every lane, so
// their ballots leave the peers unchanged); 0: a loop over `bits`.
template <int NT, int ITEMS, int MAXBITS = 0>
__device__ uint32_t tile_stable_rank(const uint32_t (&dig)[ITEMS], const bool (&valid)[ITEMS], int bins,
                                     int bits, uint32_t* cnt, uint32_t* dstart, uint32_t* wsum,
                                     uint32_t (&lpos)[ITEMS]) {
  constexpr int NW = NT / kWave;
  const int w = threadIdx.x / kWave;
  for (int i = threadIdx.x; i < NW * bins; i += NT) cnt[i] = 0;
  __syncthreads();
  uint32_t* mine = cnt + w * bins;
  uint32_t rank[ITEMS];
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const uint32_t d = dig[r];
    uint64_t peers = __ballot(valid[r]);
    if constexpr (MAXBITS > 0) {
#pragma unroll
      for (int b = 0; b < MAXBITS; ++b) {
        const bool set = (d >> b) & 1u;
        const uint64_t m = __ballot(set);
        peers &= set ? m : ~m;
      }
    } else {
      for (int b = 0; b < bits; ++b) {
        const bool set = (d >> b) & 1u;
        const uint64_t m = __ballot(set);
        peers &= set ? m : ~m;
      }
    }
    const uint32_t below = __popcll(peers & lanemask_lt());
    const uint32_t old = valid[r] ? mine[d] : 0u;
    // all lanes have read the counter before the group leader writes it
    __builtin_amdgcn_wave_barrier();
    if (valid[r] && below == 0) mine[d] = old + static_cast<uint32_t>(__popcll(peers));
    __builtin_amdgcn_wave_barrier();
    rank[r] = old + below;
  }
  __syncthreads();
  for (int d = threadIdx.x; d < bins; d += NT) {
    uint32_t s = 0;
    for (int ww = 0; ww < NW; ++ww) {
      const uint32_t v = cnt[ww * bins + d];
      cnt[ww * bins + d] = s;
      s += v;
    }
    dstart[d] = s;
  }
  __syncthreads();
  const uint32_t total = block_exclusive_scan<NT>(dstart, bins, wsum);
#pragma unroll
  for (int r = 0; r < ITEMS; ++r)
    lpos[r] = valid[r] ? dstart[dig[r]] + cnt[w * bins + dig[r]] + rank[r] : 0xFFFFFFFFu;
  return total;
}

// For each digit d < bins, over the per-tile histograms hist[ntiles][bins]:
//   colall[d] = sum over all tiles of hist[t][d]
//   gbase[d]  = sum over all tiles of digits d' < d  +  sum over tiles t < tile of hist[t][d]
// i.e. where this tile's keys of digit d start in the stably sorted output.
// When bins < NT, NT / bins threads share a digit, each summing every G-th
// tile; loads are issued 8 at a time from clamped addresses so they overlap.
// red_all, red_bef: LDS scratch of max(NT, bins) words each.
// Returns the grand total.  Ends with a barrier.
template <int NT>
__device__ uint32_t tile_global_bases(const uint32_t* __restrict__ hist, int ntiles, int tile, int bins,
                                      uint32_t* colall, uint32_t* gbase, uint32_t* red_all, uint32_t* red_bef,
                                      uint32_t* wsum) {
  constexpr int kBatch = 8;
  const int G = bins <= NT ? NT / bins : 1;
  for (int item = threadIdx.x; item < G * bins; item += NT) {
    const int d = item % bins;
    const int g = item / bins;
    uint32_t all = 0, bef = 0;
    for (int t0 = g; t0 < ntiles; t0 += kBatch * G) {
      uint32_t v[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int t = min(t0 + k * G, ntiles - 1);
        v[k] = hist[static_cast<size_t>(t) * bins + d];
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int t = t0 + k * G;
        const uint32_t x = t < ntiles ? v[k] : 0u;
        all += x;
        bef += t < tile ? x : 0u;
      }
    }
    red_all[item] = all;
    red_bef[item] = bef;
  }
  __syncthreads();
  for (int d = threadIdx.x; d < bins; d += NT) {
    uint32_t all = 0, bef = 0;
    for (int g = 0; g < G; ++g) {
      all += red_all[g * bins + d];
      bef += red_bef[g * bins + d];
    }
    colall[d] = all;
    gbase[d] = all;
    red_bef[d] = bef;  // item d belongs to this thread: no other thread reads it now
  }
  __syncthreads();
  const uint32_t total = block_exclusive_scan<NT>(gbase, bins, wsum);
  for (int d = threadIdx.x; d < bins; d += NT) gbase[d] += red_bef[d];
  __syncthreads();
  return total;
}

// Rows of D elements are processed by groups of lanes: a row gets
// L = min(64, 2^ceil(log2(ncols))) lanes and a wave covers 64 / L rows at once.
struct RowLanes {
  int log2_lanes;  // log2 L
  __host__ __device__ int lanes() const { return 1 << log2_lanes; }
  __host__ __device__ int rows_per_wave() const { return kWave >> log2_lanes; }
};

inline RowLanes row_lanes_for(int ncols) {
  int l = 0;
  while ((1 << l) < ncols && l < 6) ++l;
  return RowLanes{l};
}

}  // namespace emb
