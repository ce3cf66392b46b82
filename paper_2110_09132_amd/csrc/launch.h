// Host-side launchers of the kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace emb {

hipError_t launch_gather(const float* table, int64_t V, int D, const int32_t* ids, int T, float* out,
                         int32_t* status, hipStream_t stream);

size_t coalesce_workspace_bytes(int T, int64_t V, int D);
hipError_t launch_coalesce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                           int32_t* uniq_ids, int32_t* seg_offsets, float* uniq_grad, int32_t* num_unique,
                           void* workspace, int32_t* status, hipStream_t stream);

size_t pack_workspace_bytes(int cap_rows, int P);
hipError_t launch_pack(const int32_t* uniq_ids, const float* uniq_grad, const int32_t* num_unique, int cap_rows,
                       int D, const int32_t* row_owner, int64_t V, int P, int32_t* send_ids, float* send_rows,
                       int32_t* send_counts, int32_t* send_offsets, void* workspace, int32_t* status,
                       hipStream_t stream);

struct AdamCoeffs {
  float beta1, one_minus_beta1, beta2, one_minus_beta2;
  float step_size;  // lr / (1 - beta1^t)
  float inv_bc2;    // 1 / (1 - beta2^t)
  float eps;
};

hipError_t launch_adam(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int D, const int32_t* row_ids,
                       const float* rows, const int32_t* offsets, int shard_begin, int shard_end, int cap_rows,
                       const AdamCoeffs& c, int32_t* status, hipStream_t stream);

// Carves aligned regions out of a workspace; with base == nullptr it only measures.
struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~static_cast<size_t>(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t size() const { return (off + 255) & ~static_cast<size_t>(255); }
};

// Grid of at most `cap` blocks for `work` blocks of work (grid-stride kernels).
inline unsigned grid_for(long long work, long long cap) {
  if (work < 1) work = 1;
  return static_cast<unsigned>(work < cap ? work : cap);
}

}  // namespace emb
