// COALESCE + UNIQUE of Algorithm 1 (Sec. 4.2.2): sum the gradient rows of
// tokens with equal id, output the distinct ids in ascending order.
//
// Stages (all enqueued on one stream, no host synchronisation):
//  1. LSD radix sort of (id, token position) pairs, stable, digits of <= 8 bits
//     over bitwidth(V) key bits.  Ids outside [0, V) become the key V, which
//     sorts after every valid id and is then ignored.  Each pass is two
//     kernels: per-tile digit histograms, then a tile-local stable ranking in
//     LDS (wave ballots) plus the tile's global digit bases, staged through LDS
//     so that runs of one digit are written contiguously.
//  2. Segment discovery over the sorted keys: per-tile head counts, then the
//     unique index of every sorted element, uniq_ids, seg_offsets, num_unique.
//  3. Deterministic segmented reduction: the sorted order is cut into chunks
//     of kChunk tokens, one wave per chunk, summing rows in sorted order.
//     Segments inside one chunk are written directly; the pieces of a segment
//     that crosses chunk boundaries go to a partials buffer, and a combine
//     kernel adds them in chunk order (4 waves per segment, each summing a
//     contiguous range of pieces, then the 4 results in wave order).  The
//     order of every addition depends only on the ids, never on scheduling.
#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 8;
constexpr int kTile = kThreads * kItems;  // keys per sort / segment tile
constexpr int kRadixBitsMax = 8;
constexpr int kBinsMax = 1 << kRadixBitsMax;
constexpr int kChunk = 32;       // sorted tokens per reduction wave
constexpr int kLoadsInFlight = 8;
constexpr int kCombineWaves = kThreads / kWave;

__device__ __forceinline__ uint32_t sanitize(int32_t id, uint32_t V) {
  return (id >= 0 && static_cast<uint32_t>(id) < V) ? static_cast<uint32_t>(id) : V;
}

// ---------------------------------------------------------------- radix sort
__global__ __launch_bounds__(kThreads) void radix_hist_kernel(const uint32_t* __restrict__ keys,
                                                              const int32_t* __restrict__ raw_ids, uint32_t V,
                                                              int T, int shift, int bits,
                                                              uint32_t* __restrict__ tile_hist, int32_t* status) {
  __shared__ uint32_t h[kBinsMax];
  const int bins = 1 << bits;
  for (int i = threadIdx.x; i < bins; i += kThreads) h[i] = 0;
  __syncthreads();
  const int base = blockIdx.x * kTile;
  bool bad = false;
  uint32_t k[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int g = min(base + r * kThreads + static_cast<int>(threadIdx.x), T - 1);
    k[r] = raw_ids != nullptr ? sanitize(raw_ids[g], V) : keys[g];
  }
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    if (base + r * kThreads + static_cast<int>(threadIdx.x) < T) {
      bad |= (k[r] == V);
      atomicAdd(&h[(k[r] >> shift) & (bins - 1)], 1u);
    }
  }
  if (__any(bad) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
  __syncthreads();
  for (int i = threadIdx.x; i < bins; i += kThreads) tile_hist[static_cast<size_t>(blockIdx.x) * bins + i] = h[i];
}

__global__ __launch_bounds__(kThreads) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const int32_t* __restrict__ raw_ids, const int32_t* __restrict__ vals_in,
    uint32_t V, int T, int shift, int bits, const uint32_t* __restrict__ tile_hist, int ntiles,
    uint32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out) {
  __shared__ uint32_t cnt[(kThreads / kWave) * kBinsMax];
  __shared__ uint32_t dstart[kBinsMax], colall[kBinsMax], gbase[kBinsMax];
  __shared__ uint32_t red_all[kThreads], red_bef[kThreads];
  __shared__ uint32_t wsum[kThreads / kWave];
  __shared__ uint32_t skeys[kTile];
  __shared__ int32_t svals[kTile];
  const int bins = 1 << bits;
  const int tile = blockIdx.x;
  const int base = tile * kTile;
  const int w = threadIdx.x / kWave;

  uint32_t key[kItems], dig[kItems], lpos[kItems];
  int32_t val[kItems];
  bool valid[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int g = base + w * kItems * kWave + r * kWave + static_cast<int>(lane_id());
    const int gc = min(g, T - 1);  // clamped: every load is issued unconditionally
    valid[r] = g < T;
    key[r] = raw_ids != nullptr ? sanitize(raw_ids[gc], V) : keys_in[gc];
    val[r] = vals_in != nullptr ? vals_in[gc] : g;
    dig[r] = (key[r] >> shift) & (bins - 1);
  }
  tile_global_bases<kThreads>(tile_hist, ntiles, tile, bins, colall, gbase, red_all, red_bef, wsum);
  tile_stable_rank<kThreads, kItems>(dig, valid, bins, bits, cnt, dstart, wsum, lpos);
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    if (valid[r]) {
      skeys[lpos[r]] = key[r];
      svals[lpos[r]] = val[r];
    }
  }
  __syncthreads();
  const int n = min(kTile, T - base);
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const uint32_t k = skeys[i];
    const uint32_t d = (k >> shift) & (bins - 1);
    const uint32_t dest = gbase[d] + (static_cast<uint32_t>(i) - dstart[d]);
    keys_out[dest] = k;
    vals_out[dest] = svals[i];
  }
}

// ------------------------------------------------------- segment discovery
// Each thread owns kItems consecutive sorted keys; it loads them together with
// the key before (head test) and the key after (last-valid test).
struct KeyWindow {
  uint32_t k[kItems + 2];  // k[j] = skeys[base - 1 + j], clamped to [0, T)
  __device__ KeyWindow(const uint32_t* __restrict__ skeys, int base, int T) {
#pragma unroll
    for (int j = 0; j < kItems + 2; ++j) k[j] = skeys[min(max(base - 1 + j, 0), T - 1)];
  }
  // sorted element base + j is the first of its id (j < kItems)
  __device__ bool head(int base, int j, int T, uint32_t V) const {
    const int i = base + j;
    return i < T && k[j + 1] < V && (i == 0 || k[j] != k[j + 1]);
  }
};

__global__ __launch_bounds__(kThreads) void seg_count_kernel(const uint32_t* __restrict__ skeys, uint32_t V, int T,
                                                             uint32_t* __restrict__ tile_heads) {
  __shared__ uint32_t wsum[kThreads / kWave];
  const int base = blockIdx.x * kTile + threadIdx.x * kItems;
  const KeyWindow win(skeys, base, T);
  uint32_t c = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) c += win.head(base, j, T, V) ? 1u : 0u;
  c = wave_sum(c);
  if (lane_id() == 0) wsum[threadIdx.x / kWave] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int i = 0; i < kThreads / kWave; ++i) s += wsum[i];
    tile_heads[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(kThreads) void seg_emit_kernel(const uint32_t* __restrict__ skeys, uint32_t V, int T,
                                                            const uint32_t* __restrict__ tile_heads,
                                                            int32_t* __restrict__ uniq_ids,
                                                            int32_t* __restrict__ seg_offsets,
                                                            int32_t* __restrict__ num_unique,
                                                            int32_t* __restrict__ seg_of,
                                                            int32_t* __restrict__ span_count) {
  __shared__ uint32_t wsum[kThreads / kWave];
  __shared__ uint32_t tile_base;
  const int base = blockIdx.x * kTile + threadIdx.x * kItems;
  const KeyWindow win(skeys, base, T);
  // heads in earlier tiles (8 loads in flight per thread)
  uint32_t s = 0;
  for (int t0 = threadIdx.x; t0 < static_cast<int>(blockIdx.x); t0 += 8 * kThreads) {
    uint32_t v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = tile_heads[min(t0 + k * kThreads, static_cast<int>(blockIdx.x) - 1)];
#pragma unroll
    for (int k = 0; k < 8; ++k) s += (t0 + k * kThreads < static_cast<int>(blockIdx.x)) ? v[k] : 0u;
  }
  s = wave_sum(s);
  if (lane_id() == 0) wsum[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = 0;
    for (int i = 0; i < kThreads / kWave; ++i) b += wsum[i];
    tile_base = b;
  }
  __syncthreads();
  // heads of this thread's items, exclusive scan over the block
  uint32_t c = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) c += win.head(base, j, T, V) ? 1u : 0u;
  const uint32_t inc = wave_inclusive_scan(c);
  if (lane_id() == kWave - 1) wsum[threadIdx.x / kWave] = inc;
  __syncthreads();
  uint32_t wbase = 0;
  for (int i = 0; i < static_cast<int>(threadIdx.x / kWave); ++i) wbase += wsum[i];
  // number of heads before the current item, over the whole sorted array
  uint32_t run = tile_base + wbase + inc - c;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int i = base + j;
    const uint32_t key = win.k[j + 1];
    if (i < T && key < V) {
      if (win.head(base, j, T, V)) {
        uniq_ids[run] = static_cast<int32_t>(key);
        seg_offsets[run] = i;
        ++run;
      }
      seg_of[i] = static_cast<int32_t>(run - 1);
      if (i + 1 == T || win.k[j + 2] >= V) {  // last valid token
        seg_offsets[run] = i + 1;
        num_unique[0] = static_cast<int32_t>(run);
      }
    } else if (i == 0 && T > 0) {  // no valid token at all
      seg_offsets[0] = 0;
      num_unique[0] = 0;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) span_count[0] = 0;
}

// --------------------------------------------------------- segmented reduction
template <bool BF16, int VEC>
struct GradRow;

template <>
struct GradRow<false, 4> {
  using Acc = float4;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return reinterpret_cast<const float4*>(g)[row * Dv + c];
  }
};
template <>
struct GradRow<false, 1> {
  using Acc = float;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return reinterpret_cast<const float*>(g)[row * Dv + c];
  }
};
template <>
struct GradRow<true, 4> {
  using Acc = float4;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    const uint2 h = reinterpret_cast<const uint2*>(g)[row * Dv + c];
    return make_float4(__uint_as_float(h.x << 16), __uint_as_float(h.x & 0xFFFF0000u), __uint_as_float(h.y << 16),
                       __uint_as_float(h.y & 0xFFFF0000u));
  }
};
template <>
struct GradRow<true, 1> {
  using Acc = float;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(g)[row * Dv + c]) << 16);
  }
};

template <bool BF16, int VEC>
__global__ __launch_bounds__(kThreads) void seg_reduce_kernel(
    const void* __restrict__ grad, int D, const int32_t* __restrict__ spos, const int32_t* __restrict__ seg_of,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ num_unique, int nchunks,
    float* __restrict__ uniq_grad, float* __restrict__ partial, int32_t* __restrict__ span_list,
    int32_t* __restrict__ span_count) {
  using Row = GradRow<BF16, VEC>;
  using Acc = typename Row::Acc;
  const int chunk = uniform(static_cast<int>(blockIdx.x) * (kThreads / kWave) + static_cast<int>(threadIdx.x / kWave));
  if (chunk >= nchunks) return;
  const int nvalid = seg_offsets[num_unique[0]];
  const int a = chunk * kChunk;
  const int b = min(a + kChunk, nvalid);
  if (a >= b) return;
  const int Dv = D / VEC;
  Acc* out_rows = reinterpret_cast<Acc*>(uniq_grad);
  Acc* part_rows = reinterpret_cast<Acc*>(partial);

  for (int cb = 0; cb < Dv; cb += kWave) {
    const int c = cb + static_cast<int>(lane_id());
    const bool colok = c < Dv;
    const int cc = min(c, Dv - 1);  // clamped column: loads are unconditional
    Acc acc = Acc{};
    int cur = seg_of[a];
    int rs = a;
    auto flush = [&](int u, int s, int e) {
      const int S = seg_offsets[u];
      const int E = seg_offsets[u + 1];
      if (S == s && E == e) {
        if (colok) out_rows[static_cast<size_t>(u) * Dv + c] = acc;
      } else {
        const int slot = (s == a) ? 0 : 1;
        if (colok) part_rows[(static_cast<size_t>(chunk) * 2 + slot) * Dv + c] = acc;
        if (s == S && cb == 0 && lane_id() == 0) span_list[atomicAdd(span_count, 1)] = u;
      }
    };
    for (int i0 = a; i0 < b; i0 += kLoadsInFlight) {
      int u[kLoadsInFlight];
      Acc g[kLoadsInFlight];
#pragma unroll
      for (int k = 0; k < kLoadsInFlight; ++k) {
        const int ic = min(i0 + k, b - 1);
        u[k] = seg_of[ic];
        g[k] = Row::load(grad, static_cast<size_t>(spos[ic]), Dv, cc);
      }
#pragma unroll
      for (int k = 0; k < kLoadsInFlight; ++k) {
        const int i = i0 + k;
        if (i < b) {
          if (u[k] != cur) {
            flush(cur, rs, i);
            acc = Acc{};
            cur = u[k];
            rs = i;
          }
          acc += g[k];
        }
      }
    }
    flush(cur, rs, b);
  }
}

template <int VEC>
__global__ __launch_bounds__(kThreads) void seg_combine_kernel(const float* __restrict__ partial, int D,
                                                               const int32_t* __restrict__ seg_offsets,
                                                               const int32_t* __restrict__ span_list,
                                                               const int32_t* __restrict__ span_count,
                                                               float* __restrict__ uniq_grad) {
  using Acc = typename GradRow<false, VEC>::Acc;
  __shared__ Acc red[kCombineWaves][kWave];
  const int n = span_count[0];
  const int Dv = D / VEC;
  const int w = threadIdx.x / kWave;
  const Acc* part_rows = reinterpret_cast<const Acc*>(partial);
  Acc* out_rows = reinterpret_cast<Acc*>(uniq_grad);
  for (int j = blockIdx.x; j < n; j += gridDim.x) {
    const int u = span_list[j];
    const int S = seg_offsets[u];
    const int E = seg_offsets[u + 1];
    const int c0 = S / kChunk;
    const int np = (E - 1) / kChunk - c0 + 1;
    const int first_slot = (S == c0 * kChunk) ? 0 : 1;
    const int p_beg = static_cast<int>((static_cast<long long>(w) * np) / kCombineWaves);
    const int p_end = static_cast<int>((static_cast<long long>(w + 1) * np) / kCombineWaves);
    for (int cb = 0; cb < Dv; cb += kWave) {
      const int c = cb + static_cast<int>(lane_id());
      const bool colok = c < Dv;
      const int cc = min(c, Dv - 1);
      Acc acc = Acc{};
      for (int p0 = p_beg; p0 < p_end; p0 += kLoadsInFlight) {
        Acc g[kLoadsInFlight];
#pragma unroll
        for (int k = 0; k < kLoadsInFlight; ++k) {
          const int p = min(p0 + k, p_end - 1);
          const int slot = (p == 0) ? first_slot : 0;
          g[k] = part_rows[(static_cast<size_t>(c0 + p) * 2 + slot) * Dv + cc];
        }
#pragma unroll
        for (int k = 0; k < kLoadsInFlight; ++k)
          if (p0 + k < p_end) acc += g[k];
      }
      red[w][lane_id()] = acc;
      __syncthreads();
      if (w == 0 && colok) {
        Acc t = red[0][lane_id()];
#pragma unroll
        for (int q = 1; q < kCombineWaves; ++q) t += red[q][lane_id()];
        out_rows[static_cast<size_t>(u) * Dv + c] = t;
      }
      __syncthreads();
    }
  }
}

__global__ void empty_batch_kernel(int32_t* seg_offsets, int32_t* num_unique) {
  seg_offsets[0] = 0;
  num_unique[0] = 0;
}

int key_bits(int64_t V) {  // bits needed for keys 0..V (V is the invalid-id key)
  int b = 0;
  while ((int64_t{1} << b) <= V) ++b;
  return b;
}

struct CoalesceWs {
  uint32_t *keys_a, *keys_b;
  int32_t *vals_a, *vals_b;
  uint32_t* tile_hist;
  uint32_t* tile_heads;
  int32_t* seg_of;
  int32_t* span_list;
  int32_t* span_count;
  float* partial;
  size_t bytes;
};

CoalesceWs carve(void* base, int T, int D) {
  Carver cv{static_cast<char*>(base)};
  const size_t n = static_cast<size_t>(T);
  const size_t ntiles = (n + kTile - 1) / kTile;
  const size_t nchunks = (n + kChunk - 1) / kChunk;
  CoalesceWs w;
  w.keys_a = cv.take<uint32_t>(n);
  w.keys_b = cv.take<uint32_t>(n);
  w.vals_a = cv.take<int32_t>(n);
  w.vals_b = cv.take<int32_t>(n);
  w.tile_hist = cv.take<uint32_t>(ntiles * kBinsMax);
  w.tile_heads = cv.take<uint32_t>(ntiles);
  w.seg_of = cv.take<int32_t>(n);
  w.span_list = cv.take<int32_t>(nchunks);
  w.span_count = cv.take<int32_t>(1);
  w.partial = cv.take<float>(nchunks * 2 * static_cast<size_t>(D));
  w.bytes = cv.size();
  return w;
}

}  // namespace

size_t coalesce_workspace_bytes(int T, int64_t /*V*/, int D) { return carve(nullptr, T, D).bytes; }

hipError_t launch_coalesce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                           int32_t* uniq_ids, int32_t* seg_offsets, float* uniq_grad, int32_t* num_unique,
                           void* workspace, int32_t* status, hipStream_t stream) {
  if (T == 0) {
    hipLaunchKernelGGL(empty_batch_kernel, dim3(1), dim3(1), 0, stream, seg_offsets, num_unique);
    return hipGetLastError();
  }
  CoalesceWs ws = carve(workspace, T, D);
  const uint32_t Vk = static_cast<uint32_t>(V);
  const int ntiles = (T + kTile - 1) / kTile;
  const int nchunks = (T + kChunk - 1) / kChunk;

  // 1. radix sort of (key, position)
  const int B = key_bits(V);
  const int npass = (B + kRadixBitsMax - 1) / kRadixBitsMax;
  const int per = (B + npass - 1) / npass;
  const uint32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  uint32_t* kout = ws.keys_a;
  int32_t* vout = ws.vals_a;
  for (int p = 0; p < npass; ++p) {
    const int shift = p * per;
    const int bits = min(per, B - shift);
    const int32_t* raw = (p == 0) ? ids : nullptr;
    hipLaunchKernelGGL(radix_hist_kernel, dim3(ntiles), dim3(kThreads), 0, stream, kin, raw, Vk, T, shift, bits,
                       ws.tile_hist, status);
    hipLaunchKernelGGL(radix_scatter_kernel, dim3(ntiles), dim3(kThreads), 0, stream, kin, raw, vin, Vk, T, shift,
                       bits, ws.tile_hist, ntiles, kout, vout);
    kin = kout;
    vin = vout;
    kout = (kout == ws.keys_a) ? ws.keys_b : ws.keys_a;
    vout = (vout == ws.vals_a) ? ws.vals_b : ws.vals_a;
  }
  const uint32_t* skeys = kin;
  const int32_t* spos = vin;

  // 2. segments
  hipLaunchKernelGGL(seg_count_kernel, dim3(ntiles), dim3(kThreads), 0, stream, skeys, Vk, T, ws.tile_heads);
  hipLaunchKernelGGL(seg_emit_kernel, dim3(ntiles), dim3(kThreads), 0, stream, skeys, Vk, T, ws.tile_heads,
                     uniq_ids, seg_offsets, num_unique, ws.seg_of, ws.span_count);

  // 3. reduction
  const bool vec4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(grad) % (grad_bf16 ? 8 : 16) == 0) &&
                    (reinterpret_cast<uintptr_t>(uniq_grad) % 16 == 0);
  const dim3 rgrid((nchunks + kThreads / kWave - 1) / (kThreads / kWave));
  const dim3 cgrid(grid_for(nchunks, 1024));
  if (vec4) {
    if (grad_bf16)
      hipLaunchKernelGGL((seg_reduce_kernel<true, 4>), rgrid, dim3(kThreads), 0, stream, grad, D, spos, ws.seg_of,
                         seg_offsets, num_unique, nchunks, uniq_grad, ws.partial, ws.span_list, ws.span_count);
    else
      hipLaunchKernelGGL((seg_reduce_kernel<false, 4>), rgrid, dim3(kThreads), 0, stream, grad, D, spos, ws.seg_of,
                         seg_offsets, num_unique, nchunks, uniq_grad, ws.partial, ws.span_list, ws.span_count);
    hipLaunchKernelGGL(seg_combine_kernel<4>, cgrid, dim3(kThreads), 0, stream, ws.partial, D, seg_offsets,
                       ws.span_list, ws.span_count, uniq_grad);
  } else {
    if (grad_bf16)
      hipLaunchKernelGGL((seg_reduce_kernel<true, 1>), rgrid, dim3(kThreads), 0, stream, grad, D, spos, ws.seg_of,
                         seg_offsets, num_unique, nchunks, uniq_grad, ws.partial, ws.span_list, ws.span_count);
    else
      hipLaunchKernelGGL((seg_reduce_kernel<false, 1>), rgrid, dim3(kThreads), 0, stream, grad, D, spos, ws.seg_of,
                         seg_offsets, num_unique, nchunks, uniq_grad, ws.partial, ws.span_list, ws.span_count);
    hipLaunchKernelGGL(seg_combine_kernel<1>, cgrid, dim3(kThreads), 0, stream, ws.partial, D, seg_offsets,
                       ws.span_list, ws.span_count, uniq_grad);
  }
  return hipGetLastError();
}

}  // namespace emb
