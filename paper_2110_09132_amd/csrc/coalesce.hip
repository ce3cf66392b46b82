// COALESCE + UNIQUE of Algorithm 1 (Sec. 4.2.2): sum the gradient rows of
// tokens with equal id, output the distinct ids in ascending order.  The
// owner-major variant sorts by the key (owner, id) instead, which puts the
// distinct ids straight into the per-owner send layout of Sec. 4.1.2 (owner
// p's rows contiguous, ascending id inside): coalesce and pack in one pass
// over the gradient rows.
//
// Kernels (one stream, no host synchronisation):
//  1. sort_keys_upsweep: the sort key of every token (owner and next-batch
//     lookups done once) and the digit histograms of every radix pass at once
//     (the digit totals do not depend on the order of the keys); it also
//     clears the look-back state used by the later kernels.  Tokens whose id
//     (or owner) is out of range take no part: they are left out of the
//     histograms and so out of the sorted sequence.
//  2. sort_pass, once per digit of the key bits (<= 8 bits each, 9 where that
//     saves a pass): a stable LSD radix pass over (key, token position).
//     Each tile ranks its keys in LDS with wave ballots, publishes its
//     per-digit counts (before the ranking, so that the tiles after it find
//     them early) and reads the counts of the tiles before it (decoupled
//     look-back, Merrill & Garland 2016), so one launch per pass suffices.
//     Pass 0 sums the key build's histograms into digit totals; its first
//     tiles, once done, leave the digit starts of the later passes, which then
//     read one word per digit instead of every histogram.
//     Tiles take their index from a ticket counter, so a tile only waits for
//     tiles that are already running.  The sorted sequence holds the n_valid
//     tokens that take part.
//  3. seg_count: the number of first tokens of an id (heads) in each run of
//     128 sorted tokens.
//  4. seg_reduce: each wave owns 32 consecutive sorted tokens (for batches of
//     few tokens with wide rows, several workgroups share them, each summing
//     a slice of the columns).  It finds the
//     heads with lane shuffles, adds up the head counts of the earlier
//     workgroups, writes uniq_ids / seg_offsets / num_unique (and, by owner,
//     where each owner's rows start), and sums the
//     gradient rows of its tokens in sorted order.  The sums of an id that
//     crosses chunk boundaries inside the workgroup are added in LDS, in chunk
//     order; only an id that crosses a boundary between workgroups leaves its
//     pieces (one per workgroup) in a partials buffer.
//  5. seg_combine: adds the pieces of each such id in workgroup order
//     (16 waves per id, each summing a contiguous range of pieces, then the
//     results in wave order); by owner, it also forms the per-owner counts.
// The lookup requests of the row-wise forward exchange reuse kernels 1-3 on
// the owner-major keys and replace 4-5 by request_kernel (no rows to sum).
// Batches of at most 2048 tokens take one kernel instead of all five
// (small_coalesce_kernel: the same keys, sort and sums in one workgroup).
// The order of every floating-point addition depends only on the ids, never
// on scheduling, so results are bitwise reproducible.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace emb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxPasses = 4;  // up to 31 key bits

// Radix configuration: sort tiles on 512 threads, of 1024 keys (two per
// thread), or of 1536 keys (three per thread) for batches of more than 32768
// tokens; key-build tiles of 1024 tokens (two per thread); digits of at most
// 8 bits, or 9 bits where that saves a pass (keys of 9, 17-18 or 25-27 bits:
// one, two or three passes instead of two, three or four).  The passes are
// latency-bound (a few dozen tiles on 256 CUs), so short per-thread chains win:
// measured per owner-major call against 256-thread tiles of 2048 keys with
// 2048-token key-build tiles, 4.5 to 8.8 us less on every workload (72.6 ->
// 68.2 us for 65536 tokens of 24-bit keys); 1024 threads, or 4096- and
// 8192-token key-build tiles, were slower.  Once only pass 0 summed the key
// build's histograms, 1024-token key-build tiles gained up to 1.8 us more.
// The look-back of a tile reads its predecessors 16 at a time from beyond
// L2, so on 65536 tokens fewer, larger tiles pay (three keys per thread: 60.5
// -> 58.7 us; four: 59.0), while on 16384 tokens they cost 1 to 2 us.  (Two
// passes of 11-bit digits were measured slower than three of 8 bits for
// 24-bit keys: the 2048-bin ranking is LDS-bound and runs on half as many
// tiles.)
template <int NT, int BITS, int ITEMS>
struct SortCfg {
  static constexpr int kNT = NT;
  static constexpr int kBits = BITS;
  static constexpr int kBins = 1 << BITS;
  static constexpr int kItems = ITEMS;           // keys per thread of a sort tile
  static constexpr int kTile = NT * kItems;      // keys per sort tile
  static constexpr int kUpTile = 1024;           // tokens per key-build (histogram) tile
  static constexpr int kPasses = kMaxPasses;     // most passes this configuration runs
  static_assert(kUpTile % NT == 0, "whole key-build rounds");
};
using Narrow = SortCfg<512, 8, 2>;
using Wide9 = SortCfg<512, 9, 2>;
using NarrowBig = SortCfg<512, 8, 3>;
using Wide9Big = SortCfg<512, 9, 3>;
constexpr int kBigTileAbove = 32768;  // batches of more tokens take the 1536-key tiles
constexpr int kWide9Passes = 3;  // most passes of 9-bit digits
// Histogram and look-back words per tile, for every pass of either configuration.
constexpr int kHistPerTile = kMaxPasses * Narrow::kBins > kWide9Passes * Wide9::kBins ? kMaxPasses * Narrow::kBins
                                                                                      : kWide9Passes * Wide9::kBins;
// The workspace is laid out for the configuration with the most tiles.
static_assert(Narrow::kTile == Wide9::kTile && Narrow::kTile <= NarrowBig::kTile && Narrow::kTile <= Wide9Big::kTile,
              "the workspace's tile count is the largest");
static_assert(Narrow::kUpTile == Wide9::kUpTile && Narrow::kUpTile == NarrowBig::kUpTile &&
              Narrow::kUpTile == Wide9Big::kUpTile, "one key-build tiling");
constexpr int kChunk = 32;                    // sorted tokens per reduction wave
constexpr int kRedTile = kChunk * kWaves;     // sorted tokens per reduction workgroup
constexpr int kLoadsInFlight = 8;
// The combine of ids that cross reduction workgroups: one workgroup per such
// id, its waves splitting the id's pieces (one per reduction workgroup it
// touches); wide, so that a hot id's many pieces are summed by many waves at
// once.
constexpr int kCombineThreads = 1024;
constexpr int kCombineWaves = kCombineThreads / kWave;
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kTotalsBatch = 32;     // digit-total loads in flight per thread (tiles of the key build)
constexpr int kLookBackWindow = 16;  // look-back status words in flight per thread

// Look-back status word: value in the low 30 bits, state in the top 2 bits.
constexpr uint32_t kAggregate = 1u << 30;  // the tile's own count
constexpr uint32_t kInclusive = 2u << 30;  // the count of this and every earlier tile
constexpr uint32_t kStateMask = 3u << 30;
constexpr uint32_t kValueMask = ~kStateMask;

__device__ __forceinline__ void publish(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t peek(uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// How a token's id becomes its sort key: the id itself; with row owners,
// owner << ib | id, which orders tokens by owner shard and by id inside it;
// with the vertical split as well, class << (ib + ob) | owner << ib | id, where
// class 0 marks the prior rows (the id occurs in the next batch) and 1 the
// delayed ones, so that the prior rows of every owner come first.
struct KeySpec {
  uint32_t V;                // ids in [0, V) take part
  const int32_t* row_owner;  // nullptr: the key is the id
  int32_t P;                 // owners in [0, P) take part
  int ib, ob;                // id bits and owner bits of a composite key
  uint32_t id_mask;          // key -> id
  uint32_t omask;            // (key >> ib) & omask -> owner
  int cls_shift;             // key >> cls_shift -> class (32: no class bit)
  const uint32_t* next_tab;  // set of the next batch's ids (nullptr: no split): one byte per
                             // row of [0, V) (next_bytemap), else a hash set of 2^(32 - tab_shift) slots
  bool next_bytemap;
  int tab_shift;
  int G;                     // groups of the output: owners, times 2 with the split
  const int32_t* count_dev;  // if given: only the first *count_dev tokens take part
};

__device__ __forceinline__ int group_of(uint32_t key, const KeySpec& ks) {
  const int cls = static_cast<int>(static_cast<uint64_t>(key) >> ks.cls_shift);
  return cls * ks.P + static_cast<int>((key >> ks.ib) & ks.omask);
}

// Open-addressing hash set of ids (slot value id + 1, 0 = empty, linear probing).
__device__ __forceinline__ uint32_t tab_slot(uint32_t id, int shift) { return (id * 0x9E3779B1u) >> shift; }

__device__ __forceinline__ bool in_next(uint32_t id, const KeySpec& ks) {
  if (ks.next_bytemap) return reinterpret_cast<const uint8_t*>(ks.next_tab)[id] != 0;
  const uint32_t mask = 0xFFFFFFFFu >> ks.tab_shift;
  uint32_t slot = tab_slot(id, ks.tab_shift);
  for (uint32_t probe = 0; probe <= mask; ++probe) {
    const uint32_t v = ks.next_tab[slot];
    if (v == id + 1) return true;
    if (v == 0) return false;
    slot = (slot + 1) & mask;
  }
  return false;
}

__global__ __launch_bounds__(kThreads) void tab_clear_kernel(uint32_t* __restrict__ tab, int n) {
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads) tab[i] = 0;
}

// Inserts the in-range ids of the next batch.  Byte map: a plain byte store
// per id (setting a byte needs no read-modify-write, so repeated ids, the hot
// rows of a skewed batch, do not queue on one atomic).  Hash set (at most half
// full, so every insertion finds a free slot): each workgroup first drops the
// repeats among its own ids with a small LDS set, so that hot ids do not pile
// their atomics onto one slot.
constexpr int kLdsSlots = 1024;  // a power of two, 4x the ids of a workgroup (slot = 10 hash bits)
static_assert(kLdsSlots == 4 * kThreads, "the LDS set holds four slots per id");

__global__ __launch_bounds__(kThreads) void tab_insert_kernel(const int32_t* __restrict__ next_ids, int T_next,
                                                              uint32_t V, uint32_t* __restrict__ tab, bool bytemap,
                                                              int shift) {
  __shared__ uint32_t local[kLdsSlots];
  const int t = blockIdx.x * kThreads + threadIdx.x;
  const int32_t id = next_ids[min(t, T_next - 1)];
  bool first = t < T_next && id >= 0 && static_cast<uint32_t>(id) < V;
  if (bytemap) {
    if (first) reinterpret_cast<uint8_t*>(tab)[id] = 1;
    return;
  }
  for (int i = threadIdx.x; i < kLdsSlots; i += kThreads) local[i] = 0;
  __syncthreads();
  if (first) {  // the first thread of the workgroup to insert this id carries it on
    const uint32_t key = static_cast<uint32_t>(id) + 1u;
    uint32_t slot = tab_slot(static_cast<uint32_t>(id), 32 - 10) & (kLdsSlots - 1);
    for (int probe = 0; probe < kLdsSlots; ++probe) {
      const uint32_t old = atomicCAS(&local[slot], 0u, key);
      if (old == 0u) break;
      if (old == key) {
        first = false;
        break;
      }
      slot = (slot + 1) & (kLdsSlots - 1);
    }
  }
  if (!first) return;
  const uint32_t mask = 0xFFFFFFFFu >> shift;
  uint32_t slot = tab_slot(static_cast<uint32_t>(id), shift);
  for (uint32_t probe = 0; probe <= mask; ++probe) {
    const uint32_t old = atomicCAS(&tab[slot], 0u, static_cast<uint32_t>(id) + 1u);
    if (old == 0u || old == static_cast<uint32_t>(id) + 1u) return;
    slot = (slot + 1) & mask;
  }
}

// Exclusive prefix of one digit's counts over tiles 0 .. tile-1, read from
// status words lb[t * stride] (nearest first, kWindow at a time) until a tile with
// an inclusive count is found.  Every tile publishes its aggregate before it
// waits, so the wait ends; it is bounded anyway and reports EMB_DEV_STALLED.
// The status words of tiles on other XCDs are read from beyond their L2: a
// window costs about a microsecond, and wider windows (32, 64 words per thread)
// were measured slower than 16.
template <int kWindow>
__device__ uint32_t digit_look_back(uint32_t* lb, int tile, int stride, int32_t* status) {
  uint32_t excl = 0;
  int j = tile - 1;
  uint32_t spins = 0;
  while (j >= 0) {
    uint32_t s[kWindow];
#pragma unroll
    for (int k = 0; k < kWindow; ++k) s[k] = peek(lb + static_cast<size_t>(max(j - k, 0)) * stride);
    uint32_t acc = 0;
    bool blocked = false, done = false;
#pragma unroll
    for (int k = 0; k < kWindow; ++k) {
      if (done || blocked) continue;
      if (j - k < 0) {
        done = true;
        continue;
      }
      const uint32_t st = s[k] & kStateMask;
      if (st == 0) {
        blocked = true;
        continue;
      }
      acc += s[k] & kValueMask;
      done = (st == kInclusive);
    }
    if (blocked) {
      if (++spins > kSpinLimit) {
        raise_flag(status, EMB_DEV_STALLED);
        return excl;
      }
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    excl += acc;
    if (done) return excl;
    j -= kWindow;
  }
  return excl;
}

struct RadixPlan {
  int npass;  // number of passes
  int per;    // bits per pass (<= the digit width)
  int B;      // key bits
  int digit;  // digit width of the configuration: 8 (Narrow) or 9 (Wide9)
  __host__ __device__ int shift(int p) const { return p * per; }
  __host__ __device__ int bits(int p) const { return min(per, B - p * per); }
};

int bits_for(int64_t n) {  // bits of the values 0 .. n - 1
  int B = 0;
  while ((int64_t{1} << B) < n) ++B;
  return B;
}

// Key bits: bits(V) for the id, plus bits(P) for the owner of a composite key,
// plus one for the class bit of the vertical split.
int key_bits(int64_t V, bool by_owner, int P, bool split) {
  return bits_for(V) + (by_owner ? bits_for(P) : 0) + (split ? 1 : 0);
}

RadixPlan plan_for(int B) {
  B = max(B, 1);  // one pass even when every key is 0
  const int digit = ((B + 8) / 9 < (B + 7) / 8 && (B + 8) / 9 <= kWide9Passes) ? 9 : 8;
  const int npass = (B + digit - 1) / digit;
  return RadixPlan{npass, (B + npass - 1) / npass, B, digit};
}

KeySpec key_spec(int64_t V, const int32_t* row_owner, int P, bool split) {
  KeySpec ks;
  ks.V = static_cast<uint32_t>(V);
  ks.row_owner = row_owner;
  const bool own = row_owner != nullptr;
  ks.P = own ? P : 1;
  ks.ib = own ? bits_for(V) : 0;
  ks.ob = own ? bits_for(P) : 0;
  ks.id_mask = own ? static_cast<uint32_t>((uint64_t{1} << ks.ib) - 1) : ~0u;
  ks.omask = static_cast<uint32_t>((uint64_t{1} << ks.ob) - 1);
  ks.cls_shift = (own && split) ? ks.ib + ks.ob : 32;
  ks.next_tab = nullptr;
  ks.next_bytemap = false;
  ks.tab_shift = 32;
  ks.G = (own && split) ? 2 * P : ks.P;
  ks.count_dev = nullptr;
  return ks;
}

// ---------------------------------------------------------------- radix sort
// The sort key of every token and the digit histograms of every pass, in one
// kernel per tile of kUpTile tokens: keys[t], and vals[t] = t for a token that
// takes part, -1 for one that does not (id outside [0, V), owner outside
// [0, P), or t beyond the device-side token count).  The owner and next-batch
// lookups are done here once, so the passes read plain keys.  The workgroups
// also clear the look-back words and tickets of the passes.
template <class C>
__global__ __launch_bounds__(C::kNT) void sort_keys_upsweep_kernel(const int32_t* __restrict__ ids, int T, KeySpec ks,
                                                                   RadixPlan plan, uint32_t* __restrict__ keys,
                                                                   int32_t* __restrict__ vals,
                                                                   uint32_t* __restrict__ up_hist,
                                                                   uint32_t* __restrict__ zero_begin, int zero_words,
                                                                   int32_t* status) {
  constexpr int NT = C::kNT, kBins = C::kBins, kPer = C::kUpTile / NT;
  __shared__ uint32_t h[C::kPasses * kBins];
  for (int i = threadIdx.x; i < plan.npass * kBins; i += NT) h[i] = 0;
  const int base = blockIdx.x * C::kUpTile;
  const int Tc = ks.count_dev != nullptr ? min(max(*ks.count_dev, 0), T) : T;  // tokens that exist
  int32_t id[kPer];
  bool idok[kPer];
  uint32_t own[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) id[r] = ids[min(base + r * NT + static_cast<int>(threadIdx.x), T - 1)];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    idok[r] = id[r] >= 0 && static_cast<uint32_t>(id[r]) < ks.V;
    own[r] = 0;
  }
  if (ks.row_owner != nullptr) {
#pragma unroll
    for (int r = 0; r < kPer; ++r) own[r] = static_cast<uint32_t>(ks.row_owner[idok[r] ? id[r] : 0]);
  }
  __syncthreads();  // the histograms are cleared
  bool bad_id = false, bad_owner = false;
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int t = base + r * NT + static_cast<int>(threadIdx.x);
    const bool inb = t < Tc;
    const bool ownok = own[r] < static_cast<uint32_t>(ks.P);
    const bool take = inb && idok[r] && ownok;
    bad_id |= inb && !idok[r];
    bad_owner |= inb && idok[r] && !ownok;
    uint32_t key = (own[r] << ks.ib) | static_cast<uint32_t>(id[r]);
    if (ks.next_tab != nullptr && take && !in_next(static_cast<uint32_t>(id[r]), ks)) key |= 1u << ks.cls_shift;
    if (t < T) {
      keys[t] = key;
      vals[t] = take ? t : -1;
    }
    if (take)
      for (int p = 0; p < plan.npass; ++p)
        atomicAdd(&h[p * kBins + ((key >> plan.shift(p)) & ((1u << plan.bits(p)) - 1u))], 1u);
  }
  if (__any(bad_id) && lane_id() == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
  if (__any(bad_owner) && lane_id() == 0) raise_flag(status, EMB_DEV_OWNER_OUT_OF_RANGE);
  __syncthreads();
  for (int i = threadIdx.x; i < plan.npass * kBins; i += NT)
    up_hist[static_cast<size_t>(blockIdx.x) * plan.npass * kBins + i] = h[i];
  for (int i = blockIdx.x * NT + threadIdx.x; i < zero_words; i += gridDim.x * NT) zero_begin[i] = 0;
}

// Digit totals of pass p over the key build's nup histograms, by NT = G * kBins
// threads: thread i sums digit i mod kBins over histograms g, g + G, ... where
// g = i / kBins (kTotalsBatch loads in flight), so that with 8-bit digits both
// halves of the workgroup load; digit_totals_combine adds the G parts up.
template <int NT, int kBins>
__device__ __forceinline__ uint32_t digit_total_part(const uint32_t* __restrict__ up_hist, int nup, int npass, int p) {
  static_assert(NT % kBins == 0, "whole groups of digits");
  constexpr int G = NT / kBins;
  const int d = static_cast<int>(threadIdx.x) % kBins;
  const int g = static_cast<int>(threadIdx.x) / kBins;
  uint32_t tot = 0;
  for (int u0 = g; u0 < nup; u0 += kTotalsBatch * G) {
    uint32_t v[kTotalsBatch];
#pragma unroll
    for (int z = 0; z < kTotalsBatch; ++z)
      v[z] = up_hist[(static_cast<size_t>(min(u0 + z * G, nup - 1)) * npass + p) * kBins + d];
#pragma unroll
    for (int z = 0; z < kTotalsBatch; ++z) tot += (u0 + z * G < nup) ? v[z] : 0u;
  }
  return tot;
}

// out[d] = the sum of the G parts of digit d for d < bins, 0 for bins <= d <
// kBins; scratch: LDS of NT words, written before the first barrier (no thread
// may still read it), out after it.  Ends with a barrier.
template <int NT, int kBins>
__device__ __forceinline__ void digit_totals_combine(uint32_t part, uint32_t* scratch, uint32_t* out, int bins) {
  constexpr int G = NT / kBins;
  scratch[threadIdx.x] = part;
  __syncthreads();
  for (int d = threadIdx.x; d < kBins; d += NT) {
    uint32_t t = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) t += scratch[g * kBins + d];
    out[d] = d < bins ? t : 0u;
  }
  __syncthreads();
}

// kFirst: pass 0 (sums the key build's histograms); else a later pass (reads
// the starts pass 0 left).  Two kernels rather than a branch, so that the
// compiler keeps the ticket in flight beside the loads of either.
template <class C, bool kFirst>
__global__ __launch_bounds__(C::kNT) void sort_pass_kernel(
    const uint32_t* __restrict__ keys_in, const int32_t* __restrict__ vals_in, int T, RadixPlan plan, int pass,
    const uint32_t* __restrict__ up_hist, int nup, uint32_t* lookback,
    uint32_t* ticket, int ntiles, uint32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out,
    uint32_t* __restrict__ n_valid, uint32_t* __restrict__ starts, int32_t* status) {
  constexpr int NT = C::kNT, kBins = C::kBins, kTile = C::kTile, NW = NT / kWave, kItems = C::kItems;
  constexpr int kDigitsPerThread = (kBins + NT - 1) / NT;
  __shared__ uint32_t cnt[NW * kBins];
  __shared__ uint32_t dstart[kBins], gbase[kBins], thist[kBins];
  __shared__ uint32_t wsum[NW];
  __shared__ uint32_t skeys[kTile];
  __shared__ int32_t svals[kTile];
  __shared__ int tile_s;
  // The ticket's round trip overlaps the loads below, which do not depend on
  // the tile (this file is built without the compiler's atomic optimizer, whose
  // wave-wide form of an atomic waits for the result right away).
  uint32_t ticket_v = 0;
  if (threadIdx.x == 0) ticket_v = atomicAdd(ticket, 1u);
  const int shift = plan.shift(pass);
  const int bits = plan.bits(pass);
  const int bins = 1 << bits;
  // where each digit starts in the sorted output: pass 0 sums the digit totals
  // of the key build's histograms and scans them; the later passes read the
  // starts that pass 0 left, and the number of tokens that take part
  static_assert(NT % kBins == 0, "a whole number of threads per digit");
  uint32_t tot;  // pass 0: this thread's part of its digit's total; later passes: its digit's start
  uint32_t tv_later = 0;
  if constexpr (kFirst) {
    tot = digit_total_part<NT, kBins>(up_hist, nup, plan.npass, pass);
  } else {
    tot = starts[pass * kBins + static_cast<int>(threadIdx.x) % kBins];
    tv_later = *n_valid;
  }

  for (int i = threadIdx.x; i < kBins; i += NT) thist[i] = 0;
  if (threadIdx.x == 0) tile_s = static_cast<int>(ticket_v);
  __syncthreads();
  const int tile = tile_s;
  if (tile < 0 || tile >= ntiles) {  // the ticket counter was not cleared: never index with it
    if (threadIdx.x == 0) raise_flag(status, EMB_DEV_STALLED);
    return;
  }
  const int base = tile * kTile;
  const int w = threadIdx.x / kWave;

  // keys of this tile, in (wave, round, lane) order = input order
  uint32_t key[kItems], dig[kItems], lpos[kItems];
  int32_t val[kItems];
  bool valid[kItems];
  int idx[kItems];
  bool inb[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int g = base + w * kItems * kWave + r * kWave + static_cast<int>(lane_id());
    inb[r] = g < T;
    idx[r] = min(g, T - 1);
    val[r] = vals_in[idx[r]];
    key[r] = keys_in[idx[r]];
  }
  // the sorted sequence holds the tokens that take part: the sum of the totals
  uint32_t tv = tv_later;
  if constexpr (kFirst) {
    digit_totals_combine<NT, kBins>(tot, cnt, gbase, bins);
    tv = block_exclusive_scan<NT>(gbase, bins, wsum);
  } else {
    if (threadIdx.x < kBins) gbase[threadIdx.x] = threadIdx.x < static_cast<unsigned>(bins) ? tot : 0u;
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < kItems; ++r) dig[r] = (key[r] >> shift) & (bins - 1);
  // the first pass reads every token (those that take part have a position);
  // later passes read the tv sorted tokens
#pragma unroll
  for (int r = 0; r < kItems; ++r)
    valid[r] = inb[r] && (kFirst ? val[r] >= 0 : static_cast<uint32_t>(idx[r]) < tv);
  if (tile == 0 && threadIdx.x == 0) *n_valid = tv;
  // This tile's count of each digit, published before the ranking so that the
  // tiles after it find it when they look back.
#pragma unroll
  for (int r = 0; r < kItems; ++r)
    if (valid[r]) atomicAdd(&thist[dig[r]], 1u);
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kDigitsPerThread; ++q) {
    const int d = static_cast<int>(threadIdx.x) + q * NT;
    if (d < bins)
      publish(lookback + static_cast<size_t>(tile) * kBins + d, (tile == 0 ? kInclusive : kAggregate) | thist[d]);
  }

  const uint32_t nvalid = tile_stable_rank<NT, kItems, C::kBits>(dig, valid, bins, bits, cnt, dstart, wsum, lpos);
#pragma unroll
  for (int q = 0; q < kDigitsPerThread; ++q) {
    const int d = static_cast<int>(threadIdx.x) + q * NT;
    if (d < bins && tile > 0) {
      const uint32_t mine = thist[d];
      const uint32_t excl = digit_look_back<kLookBackWindow>(lookback + d, tile, kBins, status);
      publish(lookback + static_cast<size_t>(tile) * kBins + d, kInclusive | (excl + mine));
      gbase[d] += excl;
    }
  }
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    if (valid[r]) {
      skeys[lpos[r]] = key[r];
      svals[lpos[r]] = val[r];
    }
  }
  __syncthreads();
  const int n = static_cast<int>(nvalid);
  for (int i = threadIdx.x; i < n; i += NT) {
    const uint32_t k = skeys[i];
    const uint32_t dd = (k >> shift) & (bins - 1);
    const uint32_t dest = gbase[dd] + (static_cast<uint32_t>(i) - dstart[dd]);
    if (dest < static_cast<uint32_t>(T)) {  // always, unless the histograms were overwritten meanwhile
      keys_out[dest] = k;
      vals_out[dest] = svals[i];
    }
  }
  // After its own tile, tile t of pass 0 scans the digit totals of passes
  // t + 1, t + 1 + ntiles, ... (off the look-back chain: the first tiles finish
  // first).
  if constexpr (!kFirst) return;
  for (int later = tile + 1; later < plan.npass; later += ntiles) {
    const int lbins = 1 << plan.bits(later);
    const uint32_t part = digit_total_part<NT, kBins>(up_hist, nup, plan.npass, later);
    // cnt was last read by the ranking (before the scatter's barrier), gbase by
    // the scatter or the previous round's stores (before the combine's barrier)
    digit_totals_combine<NT, kBins>(part, cnt, gbase, lbins);
    block_exclusive_scan<NT>(gbase, lbins, wsum);
    for (int d = threadIdx.x; d < kBins; d += NT) starts[later * kBins + d] = gbase[d];
  }
}

// --------------------------------------------- segments + segmented reduction
template <bool BF16, int VEC>
struct GradRow;

template <>
struct GradRow<false, 4> {
  using Acc = float4;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return load_stream(reinterpret_cast<const float4*>(g) + row * Dv + c);
  }
};
template <>
struct GradRow<false, 1> {
  using Acc = float;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return load_stream(reinterpret_cast<const float*>(g) + row * Dv + c);
  }
};
template <>
struct GradRow<true, 4> {
  using Acc = float4;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    const uint2 h = load_stream(reinterpret_cast<const uint2*>(g) + row * Dv + c);
    return make_float4(__uint_as_float(h.x << 16), __uint_as_float(h.x & 0xFFFF0000u), __uint_as_float(h.y << 16),
                       __uint_as_float(h.y & 0xFFFF0000u));
  }
};
template <>
struct GradRow<true, 1> {
  using Acc = float;
  __device__ static Acc load(const void* g, size_t row, int Dv, int c) {
    return __uint_as_float(static_cast<uint32_t>(load_stream(reinterpret_cast<const uint16_t*>(g) + row * Dv + c)) << 16);
  }
};

// Number of heads (first sorted token of an id: its key differs from the
// previous one) among the kRedTile sorted tokens of each reduction workgroup.
__global__ __launch_bounds__(kThreads) void seg_count_kernel(const uint32_t* __restrict__ skeys,
                                                             const uint32_t* __restrict__ n_valid,
                                                             uint32_t* __restrict__ tile_heads, int ntiles) {
  const int tile = blockIdx.x * kWaves + threadIdx.x / kWave;  // one wave per reduction workgroup
  if (tile >= ntiles) return;
  const int tv = static_cast<int>(min(*n_valid, static_cast<uint32_t>(ntiles) * kRedTile));
  uint32_t c = 0;
  for (int k = static_cast<int>(lane_id()); k < kRedTile; k += kWave) {
    const int e = tile * kRedTile + k;
    const int ec = max(min(e, tv - 1), 0);  // loads stay inside the T sorted keys
    const bool head = e < tv && (e == 0 || skeys[max(ec - 1, 0)] != skeys[ec]);
    c += head ? 1u : 0u;
  }
  c = wave_sum(c);
  if (lane_id() == 0) tile_heads[tile] = c;
}

template <bool BF16, int VEC>
__global__ __launch_bounds__(kThreads) void seg_reduce_kernel(
    const uint32_t* __restrict__ skeys, const int32_t* __restrict__ spos, const uint32_t* __restrict__ n_valid, int T,
    const void* __restrict__ grad, int D, const uint32_t* __restrict__ tile_heads, KeySpec ks,
    int32_t* __restrict__ uniq_ids, int32_t* __restrict__ seg_offsets, int32_t* __restrict__ num_unique,
    float* __restrict__ uniq_grad, int32_t* __restrict__ owner_offsets, float* __restrict__ partial,
    int32_t* __restrict__ span_list, int32_t* __restrict__ span_count, int max_spans) {
  __shared__ uint32_t wave_heads[kWaves];
  __shared__ uint32_t red[kWaves];
  __shared__ uint32_t wave_flags[kWaves];
  const int tile = blockIdx.x;
  const int w = threadIdx.x / kWave;
  const int lane = static_cast<int>(lane_id());
  const int chunk = tile * kWaves + w;
  const int a = chunk * kChunk;
  // column blocks of kWave vectors: this workgroup sums blocks cb0, cb0 + cstep, ...
  // (several workgroups share a chunk's columns when the batch has few chunks
  // and wide rows); the segment bookkeeping is written by the cb0 == 0 one
  const int cb0 = static_cast<int>(blockIdx.y) * kWave;
  const int cstep = static_cast<int>(gridDim.y) * kWave;
  const bool meta = blockIdx.y == 0;

  // lane L holds sorted element e = a - 1 + L, for L = 0 .. kChunk + 1
  // (workspace values are clamped so that no index can leave its array)
  const int tv = static_cast<int>(min(*n_valid, static_cast<uint32_t>(T)));
  const int e = a - 1 + lane;
  const int ec = min(max(e, 0), T - 1);
  const uint32_t key = skeys[ec];
  const int32_t pos = min(max(spos[ec], 0), T - 1);
  // head counts of the earlier workgroups: the first kThreads * 4 are loaded
  // together with the keys (independent loads, one round trip for both)
  uint32_t hv[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) hv[q] = tile_heads[min(q * kThreads + static_cast<int>(threadIdx.x), max(tile - 1, 0))];
  const bool valid = e >= 0 && e < tv && lane <= kChunk + 1;
  const uint32_t key_prev = __shfl_up(key, 1, kWave);
  // element e does not continue the id of element e - 1
  const bool starts_new = !valid || e == 0 || key_prev != key;
  const bool in_chunk = lane >= 1 && lane <= kChunk;
  const bool head = in_chunk && valid && starts_new;
  const uint64_t heads = __ballot(head);
  const uint64_t brk = __ballot(starts_new);
  const int nv = __popcll(__ballot(in_chunk && valid));  // valid tokens of the chunk (a prefix of it)
  const bool open_lo = ((brk >> 1) & 1ull) == 0;             // element a continues the id of a - 1
  const bool open_hi = ((brk >> (kChunk + 1)) & 1ull) == 0;  // element a + kChunk continues the chunk's last id
  const uint64_t inner = nv >= 1 ? (((1ull << (nv - 1)) - 1ull) << 2) : 0ull;
  const bool one_run = nv >= 1 && (brk & inner) == 0;  // no head after the chunk's first token
  if (lane == 0) {
    wave_heads[w] = static_cast<uint32_t>(__popcll(heads));
    wave_flags[w] = (open_hi ? 1u : 0u) | (one_run ? 2u : 0u);
  }
  // The rows do not depend on the unique indices: the loads of the first
  // column block of all kChunk rows are issued before the workgroup combines
  // its counts.  Loads are unconditional, from clamped rows (a chunk with
  // fewer valid tokens re-reads its last row), so they stay in flight together.
  using Row = GradRow<BF16, VEC>;
  using Acc = typename Row::Acc;
  const int Dv = D / VEC;
  const int last = max(nv, 1) - 1;
  Acc g[kChunk];
#pragma unroll
  for (int k = 0; k < kChunk; ++k)
    g[k] = Row::load(grad, static_cast<size_t>(__builtin_amdgcn_readlane(pos, min(k, last) + 1)), Dv,
                     min(cb0 + lane, Dv - 1));
  // heads before this workgroup: the sum of the earlier workgroups' counts
  uint32_t before = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) before += (q * kThreads + static_cast<int>(threadIdx.x) < tile) ? hv[q] : 0u;
  for (int t0 = kThreads * 4; t0 < tile; t0 += kThreads * 4) {  // more than 1024 earlier workgroups
    uint32_t v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = tile_heads[min(t0 + q * kThreads + static_cast<int>(threadIdx.x), tile - 1)];
#pragma unroll
    for (int q = 0; q < 4; ++q) before += (t0 + q * kThreads + static_cast<int>(threadIdx.x) < tile) ? v[q] : 0u;
  }
  before = wave_sum(before);
  if (lane == 0) red[w] = before;
  __syncthreads();
  uint32_t ubase = 0;
#pragma unroll
  for (int q = 0; q < kWaves; ++q) ubase += red[q];
  for (int q = 0; q < w; ++q) ubase += wave_heads[q];
  const uint64_t upto = (lane == kWave - 1) ? ~0ull : ((2ull << lane) - 1ull);
  const int u = static_cast<int>(ubase + __popcll(heads & upto)) - 1;  // unique index of element e
  const bool u_ok = u >= 0 && u < T;
  if (meta && head && u_ok) {
    uniq_ids[u] = static_cast<int32_t>(key & ks.id_mask);
    seg_offsets[u] = e;
    if (owner_offsets != nullptr) {  // groups o' < p <= o start at this row
      const int o = min(group_of(key, ks), ks.G);
      const int o_prev = e == 0 ? -1 : group_of(key_prev, ks);
      for (int p = o_prev + 1; p <= o; ++p) owner_offsets[p] = u;
    }
  }
  const bool next_valid = __shfl_down(valid ? 1 : 0, 1, kWave) != 0;
  if (meta && in_chunk && valid && u_ok && (e + 1 == T || !next_valid)) {
    seg_offsets[u + 1] = e + 1;  // the last valid token of the whole batch
    num_unique[0] = u + 1;
    if (owner_offsets != nullptr)
      for (int p = min(group_of(key, ks), ks.G) + 1; p <= ks.G; ++p) owner_offsets[p] = u + 1;
  }
  if (meta && chunk == 0 && lane == 1 && !valid) {  // no valid token at all
    seg_offsets[0] = 0;
    num_unique[0] = 0;
    if (owner_offsets != nullptr)
      for (int p = 0; p <= ks.G; ++p) owner_offsets[p] = 0;
  }
  // from here on the waves of the workgroup meet at one barrier per column
  // block, so only a whole workgroup may leave early
  if (tile * kRedTile >= tv) return;

  // sum the rows of the chunk's tokens in sorted order, one run of equal ids
  // at a time.  A run that crosses chunk boundaries inside the workgroup is
  // finished by the wave where it starts (wave 0 for one that began before the
  // workgroup): it adds the first-run sums the later waves leave in LDS, in
  // chunk order.  Only runs that cross the workgroup's ends leave pieces for
  // seg_combine: slot 0 holds the run through the workgroup's first token,
  // slot 1 a run that starts later and goes on into the next workgroup.
  __shared__ Acc lds_piece[2][kWaves - 1][kWave];
  Acc* out_rows = reinterpret_cast<Acc*>(uniq_grad);
  Acc* part_rows = reinterpret_cast<Acc*>(partial);
  int buf = 0;
  for (int cb = cb0; cb < Dv; cb += cstep, buf ^= 1) {
    const int c = cb + lane;
    const bool colok = c < Dv;
    const int cc = min(c, Dv - 1);
    if (cb > cb0) {  // the next column block of the same rows
#pragma unroll
      for (int k = 0; k < kChunk; ++k)
        g[k] = Row::load(grad, static_cast<size_t>(__builtin_amdgcn_readlane(pos, min(k, last) + 1)), Dv, cc);
    }
    Acc acc = Acc{};
    int rs = 0;
    int cur = __builtin_amdgcn_readlane(u, 1);
    auto flush = [&](int uu, int s, int t) {  // run of chunk tokens [s, t)
      const bool lo = s == 0 && open_lo;
      const bool hi = t == kChunk && open_hi;
      if (hi && (w == 0 || !lo)) return;  // this wave finishes it after the barrier
      if (!lo) {
        if (colok && uu >= 0 && uu < T) out_rows[static_cast<size_t>(uu) * Dv + c] = acc;
      } else if (w > 0) {
        lds_piece[buf][w - 1][lane] = acc;
      } else if (colok) {  // the end of a run that began before the workgroup
        part_rows[(static_cast<size_t>(tile) * 2) * Dv + c] = acc;
      }
    };
    if (nv > 0) {
#pragma unroll
      for (int j = 0; j < kChunk; ++j) {
        if (j < nv) {
          if (j > rs && ((brk >> (j + 1)) & 1ull)) {
            flush(cur, rs, j);
            acc = Acc{};
            rs = j;
            cur = __builtin_amdgcn_readlane(u, j + 1);
          }
          acc += g[j];
        }
      }
      flush(cur, rs, nv);
    }
    __syncthreads();
    if (nv == kChunk && open_hi && (w == 0 || rs > 0 || !open_lo)) {
      int w1 = w;
      bool more = true;  // the run goes on past chunk w1
      while (more && w1 + 1 < kWaves) {
        ++w1;
        acc += lds_piece[buf][w1 - 1][lane];
        more = wave_flags[w1] == 3u;
      }
      const bool from_before = w == 0 && rs == 0 && open_lo;
      if (!more && !from_before) {
        if (colok && cur >= 0 && cur < T) out_rows[static_cast<size_t>(cur) * Dv + c] = acc;
      } else {
        const int slot = (w == 0 && rs == 0) ? 0 : 1;
        if (colok) part_rows[(static_cast<size_t>(tile) * 2 + slot) * Dv + c] = acc;
        if (more && !from_before && cb == 0 && lane == 0) {
          const int k = atomicAdd(span_count, 1);  // at most one per workgroup
          if (k < max_spans) span_list[k] = cur;
        }
      }
    }
  }
}

template <int VEC>
__global__ __launch_bounds__(kCombineThreads) void seg_combine_kernel(const float* __restrict__ partial, int D,
                                                               const int32_t* __restrict__ seg_offsets,
                                                               const int32_t* __restrict__ span_list,
                                                               const int32_t* __restrict__ span_count,
                                                               float* __restrict__ uniq_grad,
                                                               const int32_t* __restrict__ owner_offsets,
                                                               int32_t* __restrict__ owner_counts, int P, int T,
                                                               int max_spans) {
  using Acc = typename GradRow<false, VEC>::Acc;
  __shared__ Acc red[kCombineWaves][kWave];
  if (owner_counts != nullptr && blockIdx.x == 0 && blockIdx.y == 0)
    for (int p = threadIdx.x; p < P; p += kCombineThreads) owner_counts[p] = owner_offsets[p + 1] - owner_offsets[p];
  const int n = min(span_count[0], max_spans);
  const int Dv = D / VEC;
  const int w = threadIdx.x / kWave;
  const Acc* part_rows = reinterpret_cast<const Acc*>(partial);
  Acc* out_rows = reinterpret_cast<Acc*>(uniq_grad);
  for (int j = blockIdx.x; j < n; j += gridDim.x) {
    const int u = span_list[j];
    if (u < 0 || u >= T) continue;
    const int S = min(max(seg_offsets[u], 0), T);
    const int E = min(max(seg_offsets[u + 1], S), T);
    const int c0 = S / kRedTile;
    const int np = (E - 1) / kRedTile - c0 + 1;
    const int first_slot = (S == c0 * kRedTile) ? 0 : 1;
    const int p_beg = static_cast<int>((static_cast<long long>(w) * np) / kCombineWaves);
    const int p_end = static_cast<int>((static_cast<long long>(w + 1) * np) / kCombineWaves);
    // column blocks of kWave vectors, split over gridDim.y workgroups as in seg_reduce
    for (int cb = static_cast<int>(blockIdx.y) * kWave; cb < Dv; cb += static_cast<int>(gridDim.y) * kWave) {
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

// ------------------------------------------------------- one-workgroup path
// Batches of at most kSmallMax tokens are coalesced by one workgroup in one
// launch: the keys (built as in sort_keys_upsweep) are compacted to the
// tokens that take part, sorted by an LSD radix sort in LDS (8-bit digits,
// stable ranking as in the radix passes), and the segments are summed, each
// by a group of lanes, over its tokens in sorted order.  The outputs are those
// of the multi-kernel path; the fp32 sums of segments that would cross a
// 32-token chunk there are rounded in another order (a plain sorted-order sum
// here), within the same bound.  For small batches the launches and the gaps
// between them are most of the multi-kernel path's time.
constexpr int kSmallThreads = 1024;
constexpr int kSmallItems = 2;
constexpr int kSmallMax = kSmallThreads * kSmallItems;
constexpr int kSmallGroupsMax = 2 * 1024;  // owner groups, times two with the split

template <bool BF16, int VEC>
__global__ __launch_bounds__(kSmallThreads) void small_coalesce_kernel(
    const int32_t* __restrict__ ids, int T, KeySpec ks, int npass, const void* __restrict__ grad, int D, int log2L,
    int32_t* __restrict__ uniq_ids, int32_t* __restrict__ seg_offsets, int32_t* __restrict__ num_unique,
    float* __restrict__ uniq_grad, int32_t* __restrict__ group_counts, int32_t* __restrict__ group_offsets,
    int32_t* status) {
  constexpr int NT = kSmallThreads, NW = NT / kWave, IT = kSmallItems;
  __shared__ uint32_t key_s[2][kSmallMax];
  __shared__ int32_t pos_s[2][kSmallMax];
  __shared__ uint32_t cnt[NW * 256];
  __shared__ uint32_t dstart[256];
  __shared__ uint32_t wsum[NW];
  __shared__ uint32_t hs[kSmallMax];              // head flags, then their exclusive scan
  __shared__ int32_t sstart[kSmallMax + 1];       // first sorted token of each segment, and n
  __shared__ int32_t goff[kSmallGroupsMax + 1];   // group offsets
  const int w = threadIdx.x / kWave;
  const int lane = static_cast<int>(lane_id());
  const int Tc = ks.count_dev != nullptr ? min(max(*ks.count_dev, 0), T) : T;  // tokens that exist
  // 1. keys of the tokens, element e = (wave, round, lane) as the ranking walks them
  uint32_t key[IT], dig[IT], lpos[IT];
  bool inb[IT], take[IT];
  bool bad_id = false, bad_owner = false;
#pragma unroll
  for (int r = 0; r < IT; ++r) {
    const int e = w * IT * kWave + r * kWave + lane;
    inb[r] = e < Tc;
    const int32_t id = ids[min(e, T - 1)];
    const bool idok = id >= 0 && static_cast<uint32_t>(id) < ks.V;
    uint32_t own = 0;
    if (ks.row_owner != nullptr) own = static_cast<uint32_t>(ks.row_owner[idok ? id : 0]);
    const bool ownok = own < static_cast<uint32_t>(ks.P);
    take[r] = inb[r] && idok && ownok;
    bad_id |= inb[r] && !idok;
    bad_owner |= inb[r] && idok && !ownok;
    key[r] = (own << ks.ib) | static_cast<uint32_t>(idok ? id : 0);
    if (ks.next_tab != nullptr && take[r] && !in_next(static_cast<uint32_t>(id), ks)) key[r] |= 1u << ks.cls_shift;
    dig[r] = take[r] ? 0u : 1u;
  }
  if (__any(bad_id) && lane == 0) raise_flag(status, EMB_DEV_ID_OUT_OF_RANGE);
  if (__any(bad_owner) && lane == 0) raise_flag(status, EMB_DEV_OWNER_OUT_OF_RANGE);
  // 2. the tokens that take part, first and in token order
  (void)tile_stable_rank<NT, IT>(dig, inb, 2, 1, cnt, dstart, wsum, lpos);
  const int n = static_cast<int>(dstart[1]);  // tokens that take part
#pragma unroll
  for (int r = 0; r < IT; ++r) {
    if (take[r]) {
      key_s[0][lpos[r]] = key[r];
      pos_s[0][lpos[r]] = w * IT * kWave + r * kWave + lane;
    }
  }
  __syncthreads();
  // 3. LSD radix passes of 8-bit digits in LDS
  int cur = 0;
  for (int p = 0; p < npass; ++p) {
    bool valid[IT];
    int32_t pos[IT];
#pragma unroll
    for (int r = 0; r < IT; ++r) {
      const int e = w * IT * kWave + r * kWave + lane;
      valid[r] = e < n;
      key[r] = key_s[cur][min(e, kSmallMax - 1)];
      pos[r] = pos_s[cur][min(e, kSmallMax - 1)];
      dig[r] = valid[r] ? (key[r] >> (8 * p)) & 255u : 0u;
    }
    (void)tile_stable_rank<NT, IT>(dig, valid, 256, 8, cnt, dstart, wsum, lpos);
#pragma unroll
    for (int r = 0; r < IT; ++r) {
      if (valid[r]) {
        key_s[cur ^ 1][lpos[r]] = key[r];
        pos_s[cur ^ 1][lpos[r]] = pos[r];
      }
    }
    cur ^= 1;
    __syncthreads();
  }
  const uint32_t* sk = key_s[cur];
  const int32_t* sp = pos_s[cur];
  // 4. segments: heads, unique indices, ids, starts, offsets of the owner groups
  for (int e = threadIdx.x; e < n; e += NT) hs[e] = (e == 0 || sk[e] != sk[e - 1]) ? 1u : 0u;
  __syncthreads();
  const int U = static_cast<int>(block_exclusive_scan<NT>(hs, n, wsum));
  for (int e = threadIdx.x; e < n; e += NT) {
    if (e > 0 && sk[e] == sk[e - 1]) continue;  // not a head
    const int u = static_cast<int>(hs[e]);
    uniq_ids[u] = static_cast<int32_t>(sk[e] & ks.id_mask);
    seg_offsets[u] = e;
    sstart[u] = e;
    const int o = min(group_of(sk[e], ks), ks.G);  // groups o_prev < q <= o start at this row
    const int o_prev = e == 0 ? -1 : group_of(sk[e - 1], ks);
    for (int q = o_prev + 1; q <= o; ++q) goff[q] = u;
  }
  if (threadIdx.x == 0) {
    seg_offsets[U] = n;
    sstart[U] = n;
    num_unique[0] = U;
    const int o_last = n > 0 ? min(group_of(sk[n - 1], ks), ks.G) : -1;
    for (int q = o_last + 1; q <= ks.G; ++q) goff[q] = U;
  }
  __syncthreads();
  if (group_offsets != nullptr)
    for (int q = threadIdx.x; q <= ks.G; q += NT) {
      group_offsets[q] = goff[q];
      if (q < ks.G) group_counts[q] = goff[q + 1] - goff[q];
    }
  // 5. the sums: L lanes per segment, each segment's rows in sorted order
  using Row = GradRow<BF16, VEC>;
  using Acc = typename Row::Acc;
  const int Dv = D / VEC;
  const int L = 1 << log2L;
  const int rpw = kWave >> log2L;
  const int sub = lane >> log2L;
  const int cl = lane & (L - 1);
  Acc* out = reinterpret_cast<Acc*>(uniq_grad);
  for (int u = w * rpw + sub; u < U; u += NW * rpw) {
    const int S = sstart[u], E = sstart[u + 1];
    for (int cb = 0; cb < Dv; cb += L) {
      const int c = cb + cl;
      if (c >= Dv) continue;
      Acc acc = Acc{};
      int i = S;
      // eight rows in flight, added in order (a hot segment's chain of round trips is the
      // longest part of the kernel: 512 Zipf tokens, 14.2 -> 12.8 us with eight instead of four)
      for (; i + 8 <= E; i += 8) {
        Acc g[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) g[k] = Row::load(grad, static_cast<size_t>(sp[i + k]), Dv, c);
#pragma unroll
        for (int k = 0; k < 8; ++k) acc += g[k];
      }
      for (; i + 4 <= E; i += 4) {  // four rows in flight, added in order
        const Acc g0 = Row::load(grad, static_cast<size_t>(sp[i]), Dv, c);
        const Acc g1 = Row::load(grad, static_cast<size_t>(sp[i + 1]), Dv, c);
        const Acc g2 = Row::load(grad, static_cast<size_t>(sp[i + 2]), Dv, c);
        const Acc g3 = Row::load(grad, static_cast<size_t>(sp[i + 3]), Dv, c);
        acc += g0;
        acc += g1;
        acc += g2;
        acc += g3;
      }
      for (; i < E; ++i) acc += Row::load(grad, static_cast<size_t>(sp[i]), Dv, c);
      out[static_cast<size_t>(u) * Dv + c] = acc;
    }
  }
}

// Lookup requests of the row-wise partition, from the owner-major sorted
// tokens: one thread per sorted token.  A token heads its id when its key
// differs from the previous one; its unique index u is the number of heads up
// to it (earlier workgroups' counts from seg_count, then the workgroup's own)
// minus one.  Heads write req_ids[u] and the owner-group starts; every sorted
// token writes inverse[its position] = u.  Token t = the same thread index
// writes inverse[t] = -1 when it takes no part (those tokens are not in the
// sorted sequence).
__global__ __launch_bounds__(kRedTile) void request_kernel(const uint32_t* __restrict__ skeys,
                                                           const int32_t* __restrict__ spos,
                                                           const uint32_t* __restrict__ n_valid, int T,
                                                           const uint32_t* __restrict__ tile_heads, KeySpec ks,
                                                           const int32_t* __restrict__ ids,
                                                           int32_t* __restrict__ req_ids,
                                                           int32_t* __restrict__ req_offsets,
                                                           int32_t* __restrict__ num_unique,
                                                           int32_t* __restrict__ inverse) {
  constexpr int NW = kRedTile / kWave;
  __shared__ uint32_t wave_heads[NW];
  __shared__ uint32_t red[NW];
  const int tile = blockIdx.x;
  const int w = threadIdx.x / kWave;
  const int lane = static_cast<int>(lane_id());
  const int tv = static_cast<int>(min(*n_valid, static_cast<uint32_t>(T)));
  const int e = tile * kRedTile + static_cast<int>(threadIdx.x);
  const int ec = min(e, T - 1);
  const uint32_t key = skeys[ec];
  const uint32_t key_prev = skeys[max(ec - 1, 0)];
  const int32_t pos = spos[ec];
  const bool valid = e < tv;
  const bool head = valid && (e == 0 || key_prev != key);
  const uint64_t heads = __ballot(head);
  if (lane == 0) wave_heads[w] = static_cast<uint32_t>(__popcll(heads));
  uint32_t before = 0;
  for (int t = static_cast<int>(threadIdx.x); t < tile; t += kRedTile) before += tile_heads[t];
  before = wave_sum(before);
  if (lane == 0) red[w] = before;
  __syncthreads();
  uint32_t ubase = 0;
#pragma unroll
  for (int q = 0; q < NW; ++q) ubase += red[q];
  for (int q = 0; q < w; ++q) ubase += wave_heads[q];
  const uint64_t upto = (lane == kWave - 1) ? ~0ull : ((2ull << lane) - 1ull);
  const int u = static_cast<int>(ubase + __popcll(heads & upto)) - 1;
  if (valid && u >= 0 && u < T) {
    if (pos >= 0 && pos < T) inverse[pos] = u;
    if (head) {
      req_ids[u] = static_cast<int32_t>(key & ks.id_mask);
      const int o = min(group_of(key, ks), ks.G);  // owners o_prev < p <= o start here
      const int o_prev = e == 0 ? -1 : group_of(key_prev, ks);
      for (int p = o_prev + 1; p <= o; ++p) req_offsets[p] = u;
    }
    if (e + 1 == tv) {
      num_unique[0] = u + 1;
      for (int p = min(group_of(key, ks), ks.G) + 1; p <= ks.G; ++p) req_offsets[p] = u + 1;
    }
  }
  if (e == 0 && !valid) {  // no token takes part
    num_unique[0] = 0;
    for (int p = 0; p <= ks.G; ++p) req_offsets[p] = 0;
  }
  if (e < T) {
    const int32_t id = ids[e];
    bool take = id >= 0 && static_cast<uint32_t>(id) < ks.V;
    if (take) take = static_cast<uint32_t>(ks.row_owner[id]) < static_cast<uint32_t>(ks.P);
    if (!take) inverse[e] = -1;
  }
}

// Per-owner request counts from the offsets (one workgroup, P <= 1024); with
// an empty batch it writes the empty result first.
__global__ __launch_bounds__(1024) void request_counts_kernel(int32_t* __restrict__ req_offsets,
                                                              int32_t* __restrict__ req_counts,
                                                              int32_t* __restrict__ num_unique, int P, int empty) {
  for (int p = threadIdx.x; p <= P; p += blockDim.x) {
    if (empty) {
      req_offsets[p] = 0;
      if (p == 0) num_unique[0] = 0;
    }
    if (p < P) req_counts[p] = empty ? 0 : req_offsets[p + 1] - req_offsets[p];
  }
}

__global__ void empty_batch_kernel(int32_t* seg_offsets, int32_t* num_unique, int32_t* owner_counts,
                                   int32_t* owner_offsets, int P) {
  if (threadIdx.x == 0) {
    seg_offsets[0] = 0;
    num_unique[0] = 0;
  }
  if (owner_counts != nullptr) {
    for (int p = threadIdx.x; p <= P; p += blockDim.x) {
      owner_offsets[p] = 0;
      if (p < P) owner_counts[p] = 0;
    }
  }
}

struct CoalesceWs {
  uint32_t *keys_a, *keys_b;
  int32_t *vals_a, *vals_b;
  uint32_t* up_hist;     // [nup][npass][kBins]
  uint32_t* tickets;     // [kMaxPasses]; starts the region that starts at zero
  int32_t* span_count;
  uint32_t* sort_lb;     // [npass][ntiles][kBins]; ends that region (npass of the call)
  uint32_t* n_valid;     // tokens that take part (written by the radix passes)
  uint32_t* starts;      // [kMaxPasses][512]: where each digit of passes 1.. starts (written by pass 0)
  int32_t* span_list;
  uint32_t* tile_heads;  // [nred]
  float* partial;
  uint32_t* next_tab;    // vertical split: set of the next batch's ids [tab_words]
  int tab_words;
  bool tab_bytemap;      // a byte per row of [0, V); else a hash set of 2^(32 - tab_shift) slots
  int tab_shift;
  size_t bytes;
};

int tab_log2_slots(int T_next) {  // at least twice the ids, at least 64 slots
  int lg = 6;
  while ((int64_t{1} << lg) < 2 * static_cast<int64_t>(T_next)) ++lg;
  return lg;
}

// The set of next ids is a byte per row (one load per lookup, one plain store
// per insert) unless the table is so large that clearing V bytes per call
// would cost more than the hash set.
constexpr int64_t kBytemapMaxRows = int64_t{1} << 24;

// The layout does not depend on the number of radix passes (sized for the
// most), so one size serves the plain and the owner-major call; the split
// appends its hash set (T_next < 0: none).
template <class C>
CoalesceWs carve_with(void* base, int T, int D, int T_next, int64_t V) {
  Carver cv{static_cast<char*>(base)};
  const size_t n = static_cast<size_t>(T);
  const size_t ntiles = (n + C::kTile - 1) / C::kTile;
  const size_t nup = (n + C::kUpTile - 1) / C::kUpTile;
  const size_t nred = (n + kRedTile - 1) / kRedTile;
  CoalesceWs w;
  w.keys_a = cv.take<uint32_t>(n);
  w.keys_b = cv.take<uint32_t>(n);
  w.vals_a = cv.take<int32_t>(n);
  w.vals_b = cv.take<int32_t>(n);
  w.up_hist = cv.take<uint32_t>(nup * kHistPerTile);
  w.tickets = cv.take<uint32_t>(kMaxPasses);
  w.span_count = cv.take<int32_t>(1);
  w.sort_lb = cv.take<uint32_t>(static_cast<size_t>(kHistPerTile) * ntiles);
  w.n_valid = cv.take<uint32_t>(1);
  w.starts = cv.take<uint32_t>(static_cast<size_t>(kMaxPasses) * Wide9::kBins);
  w.span_list = cv.take<int32_t>(nred);  // at most one crossing id starts in each reduction workgroup
  w.tile_heads = cv.take<uint32_t>(nred);
  w.partial = cv.take<float>(nred * 2 * static_cast<size_t>(D));
  w.next_tab = nullptr;
  w.tab_words = 0;
  w.tab_bytemap = false;
  w.tab_shift = 32;
  if (T_next >= 0) {
    w.tab_bytemap = V <= kBytemapMaxRows;
    if (w.tab_bytemap) {
      w.tab_words = static_cast<int>((V + 3) / 4);
    } else {
      const int lg = tab_log2_slots(T_next);
      w.tab_words = 1 << lg;
      w.tab_shift = 32 - lg;
    }
    w.next_tab = cv.take<uint32_t>(static_cast<size_t>(w.tab_words));
  }
  w.bytes = cv.size();
  return w;
}

CoalesceWs carve(void* base, int T, int D, int T_next, int64_t V) { return carve_with<Narrow>(base, T, D, T_next, V); }

// The key build with the histograms, then the radix passes over (key, position).
template <class C>
void launch_sort(const int32_t* ids, int T, const KeySpec& ks, const RadixPlan& plan, const CoalesceWs& ws,
                 int32_t* status, hipStream_t stream, const uint32_t** skeys, const int32_t** spos) {
  const int ntiles = (T + C::kTile - 1) / C::kTile;
  const int nup = (T + C::kUpTile - 1) / C::kUpTile;
  uint32_t* zero_begin = ws.tickets;
  const int zero_words =
      static_cast<int>((ws.sort_lb + static_cast<size_t>(plan.npass) * ntiles * C::kBins) - zero_begin);
  hipLaunchKernelGGL(sort_keys_upsweep_kernel<C>, dim3(nup), dim3(C::kNT), 0, stream, ids, T, ks, plan, ws.keys_b,
                     ws.vals_b, ws.up_hist, zero_begin, zero_words, status);
  const uint32_t* kin = ws.keys_b;
  const int32_t* vin = ws.vals_b;
  uint32_t* kout = ws.keys_a;
  int32_t* vout = ws.vals_a;
  for (int p = 0; p < plan.npass; ++p) {
    hipLaunchKernelGGL((p == 0 ? sort_pass_kernel<C, true> : sort_pass_kernel<C, false>), dim3(ntiles), dim3(C::kNT), 0,
                       stream, kin, vin, T, plan, p, ws.up_hist, nup,
                       ws.sort_lb + static_cast<size_t>(p) * ntiles * C::kBins, ws.tickets + p, ntiles, kout, vout,
                       ws.n_valid, ws.starts, status);
    kin = kout;
    vin = vout;
    kout = (kout == ws.keys_a) ? ws.keys_b : ws.keys_a;
    vout = (vout == ws.vals_a) ? ws.vals_b : ws.vals_a;
  }
  *skeys = kin;
  *spos = vin;
}

// Workgroups per chunk group of the reduction: batches with few chunks and wide
// rows split the columns over several workgroups (one or more blocks of kWave
// vectors each), so that the launch holds about kReduceTargetGroups groups.
constexpr int kReduceTargetGroups = 1024;
int reduce_col_split(int nred, int Dv) {
  const int nblocks = (Dv + kWave - 1) / kWave;
  const int want = (kReduceTargetGroups + nred - 1) / nred;
  return max(1, min(nblocks, want));
}

bool is_split(const CoalesceVariant& var) { return var.row_owner != nullptr && var.T_next >= 0; }

RadixPlan plan_for_call(int64_t V, const CoalesceVariant& var) {
  return plan_for(key_bits(V, var.row_owner != nullptr, var.P, is_split(var)));
}

// The keys start in keys_b / vals_b and the passes alternate from keys_a, so
// the sorted keys and positions are in the buffer the last pass wrote.
void sorted_arrays(const CoalesceWs& ws, const RadixPlan& plan, const uint32_t** skeys, const int32_t** spos) {
  const bool odd = plan.npass % 2 == 1;
  *skeys = odd ? ws.keys_a : ws.keys_b;
  *spos = odd ? ws.vals_a : ws.vals_b;
}

}  // namespace

size_t coalesce_workspace_bytes(int T, int D, int T_next, int64_t V) { return carve(nullptr, T, D, T_next, V).bytes; }

bool coalesce_by_owner_supported(int64_t V, int P, bool split) {
  return key_bits(V, true, P, split) <= 8 * kMaxPasses;
}

namespace {

// Batches the one-workgroup kernel coalesces (its groups fit its LDS table).
bool small_batch(int T, const KeySpec& ks) { return T <= kSmallMax && ks.G <= kSmallGroupsMax; }

// full: the radix passes and head counts even for a small batch (the lookup
// requests read the sorted keys).
hipError_t sort_chain(const int32_t* ids, int T, int64_t V, int D, const CoalesceVariant& var, void* workspace,
                      int32_t* status, hipStream_t stream, bool full) {
  if (T == 0) return hipSuccess;
  CoalesceWs ws = carve(workspace, T, D, is_split(var) ? var.T_next : -1, V);
  KeySpec ks = key_spec(V, var.row_owner, var.P, is_split(var));
  ks.count_dev = var.count_dev;
  const RadixPlan plan = plan_for_call(V, var);
  const int nred = (T + kRedTile - 1) / kRedTile;
  // 0. the next batch's ids into a set (vertical split)
  if (is_split(var)) {
    hipLaunchKernelGGL(tab_clear_kernel, dim3(grid_for((ws.tab_words + kThreads - 1) / kThreads, 1024)),
                       dim3(kThreads), 0, stream, ws.next_tab, ws.tab_words);
    if (var.T_next > 0)
      hipLaunchKernelGGL(tab_insert_kernel, dim3((var.T_next + kThreads - 1) / kThreads), dim3(kThreads), 0, stream,
                         var.next_ids, var.T_next, ks.V, ws.next_tab, ws.tab_bytemap, ws.tab_shift);
    ks.next_tab = ws.next_tab;
    ks.next_bytemap = ws.tab_bytemap;
    ks.tab_shift = ws.tab_shift;
  }
  // a small batch is sorted and summed by the one-workgroup kernel of the reduction half
  if (!full && small_batch(T, ks)) return hipGetLastError();
  // 1-3. the key of every token (owner and next-batch lookups once) with the digit
  // histograms of all passes, then the radix passes over (key, position)
  const uint32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  const bool big = T > kBigTileAbove;
  if (plan.digit == 9) {
    if (big)
      launch_sort<Wide9Big>(ids, T, ks, plan, ws, status, stream, &kin, &vin);
    else
      launch_sort<Wide9>(ids, T, ks, plan, ws, status, stream, &kin, &vin);
  } else {
    if (big)
      launch_sort<NarrowBig>(ids, T, ks, plan, ws, status, stream, &kin, &vin);
    else
      launch_sort<Narrow>(ids, T, ks, plan, ws, status, stream, &kin, &vin);
  }
  // 4. heads per reduction workgroup
  hipLaunchKernelGGL(seg_count_kernel, dim3((nred + kWaves - 1) / kWaves), dim3(kThreads), 0, stream, kin, ws.n_valid,
                     ws.tile_heads, nred);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_coalesce_sort(const int32_t* ids, int T, int64_t V, int D, const CoalesceVariant& var,
                                void* workspace, int32_t* status, hipStream_t stream) {
  return sort_chain(ids, T, V, D, var, workspace, status, stream, false);
}

hipError_t launch_coalesce_reduce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                                  const CoalesceVariant& var, int32_t* uniq_ids, int32_t* seg_offsets,
                                  float* uniq_grad, int32_t* num_unique, int32_t* group_counts,
                                  int32_t* group_offsets, void* workspace, int32_t* status, hipStream_t stream,
                                  hipEvent_t done) {
  // group_offsets / group_counts are given exactly for the owner-major variants
  const KeySpec ks = key_spec(V, var.row_owner, var.P, is_split(var));
  if (T == 0) {
    hipExtLaunchKernelGGL(empty_batch_kernel, dim3(1), dim3(kThreads), 0, stream, nullptr, done, 0, seg_offsets,
                          num_unique, group_counts, group_offsets, ks.G);
    return hipGetLastError();
  }
  if (small_batch(T, ks)) {  // sort and sums in one workgroup (the sort half built only the next-id set)
    const CoalesceWs wsn = carve(workspace, T, D, is_split(var) ? var.T_next : -1, V);
    KeySpec kss = ks;
    kss.count_dev = var.count_dev;
    if (is_split(var)) {
      kss.next_tab = wsn.next_tab;
      kss.next_bytemap = wsn.tab_bytemap;
      kss.tab_shift = wsn.tab_shift;
    }
    const int npass = (max(key_bits(V, var.row_owner != nullptr, var.P, is_split(var)), 1) + 7) / 8;
    const bool v4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(grad) % (grad_bf16 ? 8 : 16) == 0) &&
                    (reinterpret_cast<uintptr_t>(uniq_grad) % 16 == 0);
    const int log2L = row_lanes_for(v4 ? D / 4 : D).log2_lanes;
#define EMB_SMALL(BF, VC)                                                                                           \
  hipExtLaunchKernelGGL((small_coalesce_kernel<BF, VC>), dim3(1), dim3(kSmallThreads), 0, stream, nullptr, done, 0, \
                        ids, T, kss, npass, grad, D, log2L, uniq_ids, seg_offsets, num_unique, uniq_grad,  \
                        group_counts, group_offsets, status)
    if (v4) {
      if (grad_bf16)
        EMB_SMALL(true, 4);
      else
        EMB_SMALL(false, 4);
    } else {
      if (grad_bf16)
        EMB_SMALL(true, 1);
      else
        EMB_SMALL(false, 1);
    }
#undef EMB_SMALL
    return hipGetLastError();
  }
  CoalesceWs ws = carve(workspace, T, D, -1, V);  // the next-id set, if any, lies past everything used here
  const RadixPlan plan = plan_for_call(V, var);
  const int nred = (T + kRedTile - 1) / kRedTile;
  const uint32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  sorted_arrays(ws, plan, &kin, &vin);
  // 5. segments and their sums; 6. ids that cross reduction workgroups
  const bool vec4 = (D % 4 == 0) && (reinterpret_cast<uintptr_t>(grad) % (grad_bf16 ? 8 : 16) == 0) &&
                    (reinterpret_cast<uintptr_t>(uniq_grad) % 16 == 0);
  const dim3 cgrid(grid_for(nred, 256), grid_for((D / (vec4 ? 4 : 1) + kWave - 1) / kWave, 8));
#define EMB_REDUCE(BF, VC)                                                                                          \
  hipLaunchKernelGGL((seg_reduce_kernel<BF, VC>), dim3(nred, reduce_col_split(nred, D / (VC))), dim3(kThreads), 0,   \
                     stream, kin, vin, ws.n_valid, T,                                                                \
                     grad, D, ws.tile_heads, ks, uniq_ids, seg_offsets, num_unique, uniq_grad, group_offsets,        \
                     ws.partial, ws.span_list, ws.span_count, nred)
#define EMB_COMBINE(VC)                                                                                             \
  hipExtLaunchKernelGGL(seg_combine_kernel<VC>, cgrid, dim3(kCombineThreads), 0, stream, nullptr, done, 0,         \
                        ws.partial, D,                                                                               \
                        seg_offsets, ws.span_list, ws.span_count, uniq_grad, group_offsets, group_counts, ks.G, T,  \
                        nred)
  if (vec4) {
    if (grad_bf16)
      EMB_REDUCE(true, 4);
    else
      EMB_REDUCE(false, 4);
    EMB_COMBINE(4);
  } else {
    if (grad_bf16)
      EMB_REDUCE(true, 1);
    else
      EMB_REDUCE(false, 1);
    EMB_COMBINE(1);
  }
#undef EMB_REDUCE
#undef EMB_COMBINE
  return hipGetLastError();
}

hipError_t launch_lookup_request(const int32_t* ids, int T, int64_t V, const int32_t* row_owner, int P,
                                 int32_t* req_ids, int32_t* req_counts, int32_t* req_offsets, int32_t* num_unique,
                                 int32_t* inverse, void* workspace, int32_t* status, hipStream_t stream) {
  if (T == 0) {
    hipLaunchKernelGGL(request_counts_kernel, dim3(1), dim3(1024), 0, stream, req_offsets, req_counts, num_unique, P,
                       1);
    return hipGetLastError();
  }
  CoalesceVariant var;
  var.row_owner = row_owner;
  var.P = P;
  const hipError_t e = sort_chain(ids, T, V, 0, var, workspace, status, stream, true);
  if (e != hipSuccess) return e;
  const CoalesceWs ws = carve(workspace, T, 0, -1, V);
  const KeySpec ks = key_spec(V, row_owner, P, false);
  const RadixPlan plan = plan_for_call(V, var);
  const uint32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  sorted_arrays(ws, plan, &kin, &vin);
  const int nred = (T + kRedTile - 1) / kRedTile;
  hipLaunchKernelGGL(request_kernel, dim3(nred), dim3(kRedTile), 0, stream, kin, vin, ws.n_valid, T, ws.tile_heads, ks,
                     ids, req_ids, req_offsets, num_unique, inverse);
  hipLaunchKernelGGL(request_counts_kernel, dim3(1), dim3(1024), 0, stream, req_offsets, req_counts, num_unique, P, 0);
  return hipGetLastError();
}

hipError_t launch_coalesce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                           const CoalesceVariant& var, int32_t* uniq_ids, int32_t* seg_offsets, float* uniq_grad,
                           int32_t* num_unique, int32_t* group_counts, int32_t* group_offsets, void* workspace,
                           int32_t* status, hipStream_t stream) {
  const hipError_t e = launch_coalesce_sort(ids, T, V, D, var, workspace, status, stream);
  if (e != hipSuccess) return e;
  return launch_coalesce_reduce(ids, T, grad, grad_bf16, D, V, var, uniq_ids, seg_offsets, uniq_grad, num_unique,
                                group_counts, group_offsets, workspace, status, stream, nullptr);
}

}  // namespace emb
