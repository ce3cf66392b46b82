// Host-side launchers of the kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace emb {

// done (may be null): an event attached to the kernel's dispatch.
hipError_t launch_gather(const float* table, int64_t V, int D, const int32_t* ids, int T, float* out,
                         int32_t* status, hipStream_t stream, hipEvent_t done = nullptr);

// Which coalesce: plain (ids ascending), owner-major (row_owner given: the
// distinct ids grouped by owner in [0, P)), or owner-major with the vertical
// split (T_next >= 0 as well: the prior rows, whose ids occur in next_ids, in
// groups 0 .. P-1, then the delayed rows in groups P .. 2P-1).
struct CoalesceVariant {
  const int32_t* row_owner = nullptr;
  int P = 1;
  const int32_t* next_ids = nullptr;
  int T_next = -1;
  const int32_t* count_dev = nullptr;  // if given: only the first *count_dev of the T tokens take part
};

// Workspace size (T_next < 0: no split); it does not depend on the other choices.
size_t coalesce_workspace_bytes(int T, int D, int T_next, int64_t V);
bool coalesce_by_owner_supported(int64_t V, int P, bool split);  // the composite keys fit the radix passes
// The two halves of launch_coalesce, for schedules that run them on different
// streams (same ids, workspace and variant; the reduce half must follow the
// sort half).  A batch of at most 2048 tokens is sorted and summed by one
// kernel of the reduce half (the sort half then only builds the next-id set
// of the split).  done (may be null): an event attached to the reduce half's
// last kernel.
hipError_t launch_coalesce_sort(const int32_t* ids, int T, int64_t V, int D, const CoalesceVariant& var,
                                void* workspace, int32_t* status, hipStream_t stream);
hipError_t launch_coalesce_reduce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                                  const CoalesceVariant& var, int32_t* uniq_ids, int32_t* seg_offsets,
                                  float* uniq_grad, int32_t* num_unique, int32_t* group_counts,
                                  int32_t* group_offsets, void* workspace, int32_t* status, hipStream_t stream,
                                  hipEvent_t done);
hipError_t launch_coalesce(const int32_t* ids, int T, const void* grad, bool grad_bf16, int D, int64_t V,
                           const CoalesceVariant& var, int32_t* uniq_ids, int32_t* seg_offsets, float* uniq_grad,
                           int32_t* num_unique, int32_t* group_counts, int32_t* group_offsets, void* workspace,
                           int32_t* status, hipStream_t stream);
// Lookup requests of the row-wise partition: the owner-major sort of the
// coalesce (workspace coalesce_workspace_bytes(T, 0, -1, V)), then the
// distinct ids per owner and every token's index into them.
hipError_t launch_lookup_request(const int32_t* ids, int T, int64_t V, const int32_t* row_owner, int P,
                                 int32_t* req_ids, int32_t* req_counts, int32_t* req_offsets, int32_t* num_unique,
                                 int32_t* inverse, void* workspace, int32_t* status, hipStream_t stream);
// Host-side argument checks of emb_grad_coalesce, emb_grad_coalesce_by_owner and
// emb_grad_coalesce_split (EMB_OK when the call is valid).
int coalesce_args_status(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D, int64_t V,
                         const int32_t* uniq_ids, const int32_t* seg_offsets, const float* uniq_grad,
                         const int32_t* num_unique, const void* workspace, size_t workspace_bytes);
int coalesce_by_owner_args_status(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D,
                                  int64_t V, const int32_t* row_owner, int32_t P, const int32_t* next_ids,
                                  int32_t T_next, const int32_t* send_ids, const int32_t* seg_offsets,
                                  const float* send_rows, const int32_t* send_counts, const int32_t* send_offsets,
                                  const int32_t* num_unique, const void* workspace, size_t workspace_bytes);

// Column-block layout (block p = the [C][w(p)] slice of owner p's columns at
// float offset C * off(p), off(p) = floor(p * D / P)); see column.hip.
hipError_t launch_column_pack(const float* rows, const int32_t* num_rows, int cap, int D, int P, float* blocks,
                              int32_t* send_counts, hipStream_t stream);
hipError_t launch_column_gather(const float* shards, int64_t V, int D, int P, const int32_t* ids, int T,
                                float* blocks, int32_t* status, hipStream_t stream);
hipError_t launch_column_assemble(const float* blocks, int64_t C, int64_t row0, int R, int D, int P, float* rows,
                                  hipStream_t stream);

// The simulated AlltoAll of P workers' send layouts (send_* of worker w at
// w * cap_rows): receiver-major blocks, senders in order inside a receiver.
hipError_t launch_exchange(const int32_t* send_ids, const float* send_rows, const int32_t* send_offsets, int P,
                           int cap, int D, int32_t* recv_ids, float* recv_rows, int32_t* recv_offsets,
                           int32_t* recv_total, hipStream_t stream);

size_t pack_workspace_bytes(int cap_rows, int P);
hipError_t launch_pack(const int32_t* uniq_ids, const float* uniq_grad, const int32_t* num_unique, int cap_rows,
                       int D, const int32_t* row_owner, int64_t V, int P, int32_t* send_ids, float* send_rows,
                       int32_t* send_counts, int32_t* send_offsets, void* workspace, int32_t* status,
                       hipStream_t stream);

// The update's coefficients, in the order emb_adam_coeffs writes them.
struct AdamCoeffs {
  float beta1, one_minus_beta1, beta2, one_minus_beta2;
  float step_size;  // lr / (1 - beta1^t)
  float inv_bc2;    // 1 / (1 - beta2^t)
  float eps;
};
static_assert(sizeof(AdamCoeffs) <= EMB_ADAM_COEFFS_WORDS * sizeof(float), "coefficients fit their words");
// The coefficients of step `step`, formed in fp64 and rounded once to fp32; EMB_ERR_INVALID_ARG for
// hyper-parameters the update refuses.
int adam_coeffs(double lr, double beta1, double beta2, double eps, int64_t step, AdamCoeffs* c);

// start / stop (may be null): timing events around the kernel; stop is
// attached to the kernel's dispatch (no separate marker packet), start is
// recorded just before it.
// coeffs_dev (may be null): device memory holding the coefficients, read by the
// kernel when it runs in place of `c` (steps replayed from a graph).
hipError_t launch_adam(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int D, const int32_t* row_ids,
                       const float* rows, const int32_t* offsets, int shard_begin, int shard_end, int cap_rows,
                       const AdamCoeffs& c, const AdamCoeffs* coeffs_dev, int32_t* status, hipStream_t stream,
                       hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
// emb_sparse_adam_apply with the optional start / stop events of launch_adam and
// coefficients in device memory.
int sparse_adam_call(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int32_t D, const int32_t* row_ids,
                     const float* rows, const int32_t* offsets, int32_t P, int32_t shard_begin, int32_t shard_end,
                     int32_t cap_rows, double lr, double beta1, double beta2, double eps, int64_t step,
                     const void* coeffs_dev, int32_t* dev_status, hipStream_t stream, hipEvent_t start,
                     hipEvent_t stop);

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

// Grid of the bandwidth-bound row kernels (gather, row copy, update): one
// workgroup per few dozen rows rather than a persistent grid.  Kernels of the
// other streams of a step occupy CUs now and then; with small workgroups the
// hardware hands the remaining work to whichever CU frees up, where a
// persistent grid would wait for its late workgroups (measured: ~9 us per
// step less than two persistent workgroups per CU).  The cap only bounds
// huge launches.
constexpr long long kMaxBlocks = 1 << 20;

// Grid of at most `cap` blocks for `work` blocks of work (grid-stride kernels).
inline unsigned grid_for(long long work, long long cap) {
  if (work < 1) work = 1;
  return static_cast<unsigned>(work < cap ? work : cap);
}

}  // namespace emb
