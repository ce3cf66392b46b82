// C ABI entry points: host-side argument checks, workspace checks, and the
// launches of each stage on the caller's stream.  Contract: include/emb.h.
#include <cmath>

#include "common.h"
#include "launch.h"

namespace {

constexpr int64_t kMaxV = (int64_t{1} << 31) - 1;
constexpr int kMaxOwners = 1024;

int launch_status(hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH; }

bool bad_table_dims(int64_t V, int32_t D) { return V < 1 || V > kMaxV || D < 1; }

}  // namespace

namespace emb {

int coalesce_args_status(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D, int64_t V,
                         const int32_t* uniq_ids, const int32_t* seg_offsets, const float* uniq_grad,
                         const int32_t* num_unique, const void* workspace, size_t workspace_bytes) {
  if (T < 0 || T >= (1 << 30) || bad_table_dims(V, D) || (grad_dtype != EMB_F32 && grad_dtype != EMB_BF16))
    return EMB_ERR_INVALID_ARG;
  if (!seg_offsets || !num_unique) return EMB_ERR_INVALID_ARG;
  if (T > 0 && (!ids || !grad || !uniq_ids || !uniq_grad || !workspace)) return EMB_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(grad) % (grad_dtype == EMB_BF16 ? 2 : 4) != 0) return EMB_ERR_INVALID_ARG;
  if (T > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return EMB_ERR_INVALID_ARG;
  if (T > 0 && workspace_bytes < coalesce_workspace_bytes(T, D, -1, V)) return EMB_ERR_WORKSPACE;
  return EMB_OK;
}

// T_next < 0: the owner-major call without the split.
int coalesce_by_owner_args_status(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D,
                                  int64_t V, const int32_t* row_owner, int32_t P, const int32_t* next_ids,
                                  int32_t T_next, const int32_t* send_ids, const int32_t* seg_offsets,
                                  const float* send_rows, const int32_t* send_counts, const int32_t* send_offsets,
                                  const int32_t* num_unique, const void* workspace, size_t workspace_bytes) {
  const bool split = T_next >= 0;
  if (P < 1 || P > kMaxOwners || !send_counts || !send_offsets) return EMB_ERR_INVALID_ARG;
  if (T > 0 && !row_owner) return EMB_ERR_INVALID_ARG;
  if (split && (T_next >= (1 << 30) || (T_next > 0 && !next_ids))) return EMB_ERR_INVALID_ARG;
  if (!bad_table_dims(V, D) && !coalesce_by_owner_supported(V, P, split)) return EMB_ERR_UNSUPPORTED;
  const int st = coalesce_args_status(ids, T, grad, grad_dtype, D, V, send_ids, seg_offsets, send_rows, num_unique,
                                      workspace, workspace_bytes);
  if (st != EMB_OK) return st;
  if (split && T > 0 && workspace_bytes < coalesce_workspace_bytes(T, D, T_next, V)) return EMB_ERR_WORKSPACE;
  return EMB_OK;
}


int adam_coeffs(double lr, double beta1, double beta2, double eps, int64_t step, AdamCoeffs* c) {
  if (step < 1 || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0) ||
      !std::isfinite(lr) || !std::isfinite(eps))
    return EMB_ERR_INVALID_ARG;
  // bias corrections in fp64 on the host, then the fp32 coefficients of the kernel
  const double bc1 = 1.0 - std::pow(beta1, static_cast<double>(step));
  const double bc2 = 1.0 - std::pow(beta2, static_cast<double>(step));
  if (!(bc1 > 0.0) || !(bc2 > 0.0)) return EMB_ERR_INVALID_ARG;  // beta == 0 edge cases stay valid: bc == 1
  c->beta1 = static_cast<float>(beta1);
  c->one_minus_beta1 = static_cast<float>(1.0 - beta1);
  c->beta2 = static_cast<float>(beta2);
  c->one_minus_beta2 = static_cast<float>(1.0 - beta2);
  c->step_size = static_cast<float>(lr / bc1);
  c->inv_bc2 = static_cast<float>(1.0 / bc2);
  c->eps = static_cast<float>(eps);
  return EMB_OK;
}

int sparse_adam_call(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int32_t D, const int32_t* row_ids,
                     const float* rows, const int32_t* offsets, int32_t P, int32_t shard_begin, int32_t shard_end,
                     int32_t cap_rows, double lr, double beta1, double beta2, double eps, int64_t step,
                     const void* coeffs_dev, int32_t* dev_status, hipStream_t stream, hipEvent_t start,
                     hipEvent_t stop) {
  if (bad_table_dims(V, D) || P < 1 || P > kMaxOwners || cap_rows < 0) return EMB_ERR_INVALID_ARG;
  if (shard_begin < 0 || shard_begin > shard_end || shard_end > P) return EMB_ERR_INVALID_ARG;
  AdamCoeffs c;
  const int cst = adam_coeffs(lr, beta1, beta2, eps, step, &c);
  if (cst != EMB_OK) return cst;
  if (coeffs_dev != nullptr && reinterpret_cast<uintptr_t>(coeffs_dev) % 16 != 0) return EMB_ERR_INVALID_ARG;
  if (cap_rows == 0 || shard_begin == shard_end) {  // nothing to launch: the timing pair still brackets this point
    if (start && hipEventRecord(start, stream) != hipSuccess) return EMB_ERR_LAUNCH;
    if (stop && hipEventRecord(stop, stream) != hipSuccess) return EMB_ERR_LAUNCH;
    return EMB_OK;
  }
  if (!table || !exp_avg || !exp_avg_sq || !row_ids || !rows || !offsets) return EMB_ERR_INVALID_ARG;
  return launch_status(launch_adam(table, exp_avg, exp_avg_sq, V, D, row_ids, rows, offsets, shard_begin, shard_end,
                                   cap_rows, c, static_cast<const AdamCoeffs*>(coeffs_dev), dev_status, stream,
                                   start, stop));
}

}  // namespace emb

extern "C" {

int emb_abi_version(void) { return EMB_ABI_VERSION; }

const char* emb_status_string(int status) {
  switch (status) {
    case EMB_OK: return "ok";
    case EMB_ERR_INVALID_ARG: return "invalid argument";
    case EMB_ERR_WORKSPACE: return "workspace too small";
    case EMB_ERR_LAUNCH: return "kernel launch failed";
    case EMB_ERR_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

int emb_gather(const float* table, int64_t V, int32_t D, const int32_t* ids, int32_t T, float* out,
               int32_t* dev_status, void* stream) {
  if (bad_table_dims(V, D) || T < 0) return EMB_ERR_INVALID_ARG;
  if (T == 0) return EMB_OK;
  if (!table || !ids || !out) return EMB_ERR_INVALID_ARG;
  return launch_status(emb::launch_gather(table, V, D, ids, T, out, dev_status, static_cast<hipStream_t>(stream)));
}

size_t emb_grad_coalesce_workspace_bytes(int32_t T, int64_t V, int32_t D, int32_t grad_dtype) {
  if (T < 0 || bad_table_dims(V, D) || (grad_dtype != EMB_F32 && grad_dtype != EMB_BF16)) return 0;
  return emb::coalesce_workspace_bytes(T, D, -1, V);
}

size_t emb_grad_coalesce_split_workspace_bytes(int32_t T, int32_t T_next, int64_t V, int32_t D, int32_t grad_dtype) {
  if (T < 0 || T_next < 0 || bad_table_dims(V, D) || (grad_dtype != EMB_F32 && grad_dtype != EMB_BF16)) return 0;
  return emb::coalesce_workspace_bytes(T, D, T_next, V);
}

int emb_grad_coalesce(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D, int64_t V,
                      int32_t* uniq_ids, int32_t* seg_offsets, float* uniq_grad, int32_t* num_unique,
                      void* workspace, size_t workspace_bytes, int32_t* dev_status, void* stream) {
  const int st = emb::coalesce_args_status(ids, T, grad, grad_dtype, D, V, uniq_ids, seg_offsets, uniq_grad,
                                           num_unique, workspace, workspace_bytes);
  if (st != EMB_OK) return st;
  return launch_status(emb::launch_coalesce(ids, T, grad, grad_dtype == EMB_BF16, D, V, emb::CoalesceVariant{},
                                            uniq_ids, seg_offsets, uniq_grad, num_unique, nullptr, nullptr, workspace,
                                            dev_status, static_cast<hipStream_t>(stream)));
}

int emb_grad_coalesce_by_owner(const int32_t* ids, int32_t T, const void* grad, int32_t grad_dtype, int32_t D,
                               int64_t V, const int32_t* row_owner, int32_t P, int32_t* send_ids,
                               int32_t* seg_offsets, float* send_rows, int32_t* send_counts, int32_t* send_offsets,
                               int32_t* num_unique, void* workspace, size_t workspace_bytes, int32_t* dev_status,
                               void* stream) {
  const int st = emb::coalesce_by_owner_args_status(ids, T, grad, grad_dtype, D, V, row_owner, P, nullptr, -1,
                                                    send_ids, seg_offsets, send_rows, send_counts, send_offsets,
                                                    num_unique, workspace, workspace_bytes);
  if (st != EMB_OK) return st;
  emb::CoalesceVariant var;
  var.row_owner = row_owner;
  var.P = P;
  return launch_status(emb::launch_coalesce(ids, T, grad, grad_dtype == EMB_BF16, D, V, var, send_ids, seg_offsets,
                                            send_rows, num_unique, send_counts, send_offsets, workspace, dev_status,
                                            static_cast<hipStream_t>(stream)));
}

int emb_grad_coalesce_split(const int32_t* ids, int32_t T, const int32_t* next_ids, int32_t T_next, const void* grad,
                            int32_t grad_dtype, int32_t D, int64_t V, const int32_t* row_owner, int32_t P,
                            int32_t* send_ids, int32_t* seg_offsets, float* send_rows, int32_t* send_counts,
                            int32_t* send_offsets, int32_t* num_unique, void* workspace, size_t workspace_bytes,
                            int32_t* dev_status, void* stream) {
  if (T_next < 0) return EMB_ERR_INVALID_ARG;
  const int st = emb::coalesce_by_owner_args_status(ids, T, grad, grad_dtype, D, V, row_owner, P, next_ids, T_next,
                                                    send_ids, seg_offsets, send_rows, send_counts, send_offsets,
                                                    num_unique, workspace, workspace_bytes);
  if (st != EMB_OK) return st;
  emb::CoalesceVariant var;
  var.row_owner = row_owner;
  var.P = P;
  var.next_ids = next_ids;
  var.T_next = T_next;
  return launch_status(emb::launch_coalesce(ids, T, grad, grad_dtype == EMB_BF16, D, V, var, send_ids, seg_offsets,
                                            send_rows, num_unique, send_counts, send_offsets, workspace, dev_status,
                                            static_cast<hipStream_t>(stream)));
}

size_t emb_lookup_request_workspace_bytes(int32_t T, int64_t V) {
  if (T < 0 || bad_table_dims(V, 1)) return 0;
  return emb::coalesce_workspace_bytes(T, 0, -1, V);
}

int emb_lookup_request(const int32_t* ids, int32_t T, int64_t V, const int32_t* row_owner, int32_t P,
                       int32_t* req_ids, int32_t* req_counts, int32_t* req_offsets, int32_t* num_unique,
                       int32_t* inverse, void* workspace, size_t workspace_bytes, int32_t* dev_status,
                       void* stream) {
  if (T < 0 || T >= (1 << 30) || bad_table_dims(V, 1) || P < 1 || P > kMaxOwners) return EMB_ERR_INVALID_ARG;
  if (!req_counts || !req_offsets || !num_unique) return EMB_ERR_INVALID_ARG;
  if (!emb::coalesce_by_owner_supported(V, P, false)) return EMB_ERR_UNSUPPORTED;
  if (T > 0 && (!ids || !row_owner || !req_ids || !inverse || !workspace)) return EMB_ERR_INVALID_ARG;
  if (T > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return EMB_ERR_INVALID_ARG;
  if (T > 0 && workspace_bytes < emb::coalesce_workspace_bytes(T, 0, -1, V)) return EMB_ERR_WORKSPACE;
  return launch_status(emb::launch_lookup_request(ids, T, V, row_owner, P, req_ids, req_counts, req_offsets,
                                                  num_unique, inverse, workspace, dev_status,
                                                  static_cast<hipStream_t>(stream)));
}

int emb_exchange_simulated(const int32_t* send_ids, const float* send_rows, const int32_t* send_offsets, int32_t P,
                           int32_t cap_rows, int32_t D, int32_t* recv_ids, float* recv_rows, int32_t* recv_offsets,
                           int32_t* recv_total, void* stream) {
  if (P < 1 || P > kMaxOwners || cap_rows < 0 || D < 0) return EMB_ERR_INVALID_ARG;
  if (static_cast<int64_t>(P) * cap_rows >= (int64_t{1} << 30)) return EMB_ERR_INVALID_ARG;
  if (!send_offsets || !recv_offsets || !recv_total) return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && (!send_ids || !recv_ids)) return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && D > 0 && (!send_rows || !recv_rows)) return EMB_ERR_INVALID_ARG;
  return launch_status(emb::launch_exchange(send_ids, send_rows, send_offsets, P, cap_rows, D, recv_ids, recv_rows,
                                            recv_offsets, recv_total, static_cast<hipStream_t>(stream)));
}

int emb_receive_merge(const int32_t* recv_ids, const float* recv_rows, const int32_t* recv_total, int32_t cap,
                      int32_t D, int64_t V, const int32_t* row_owner, int32_t P, int32_t* merged_ids,
                      int32_t* seg_offsets, float* merged_rows, int32_t* merged_counts, int32_t* merged_offsets,
                      int32_t* num_unique, void* workspace, size_t workspace_bytes, int32_t* dev_status,
                      void* stream) {
  if (!recv_total) return EMB_ERR_INVALID_ARG;
  const int st = emb::coalesce_by_owner_args_status(recv_ids, cap, recv_rows, EMB_F32, D, V, row_owner, P, nullptr,
                                                    -1, merged_ids, seg_offsets, merged_rows, merged_counts,
                                                    merged_offsets, num_unique, workspace, workspace_bytes);
  if (st != EMB_OK) return st;
  emb::CoalesceVariant var;
  var.row_owner = row_owner;
  var.P = P;
  var.count_dev = recv_total;
  return launch_status(emb::launch_coalesce(recv_ids, cap, recv_rows, false, D, V, var, merged_ids, seg_offsets,
                                            merged_rows, num_unique, merged_counts, merged_offsets, workspace,
                                            dev_status, static_cast<hipStream_t>(stream)));
}

namespace {
bool bad_column_split(int32_t D, int32_t P) {
  return D < 1 || P < 1 || P > D || P > kMaxOwners || static_cast<int64_t>(D) * P >= (int64_t{1} << 31);
}
}  // namespace

int emb_pack_by_column(const float* rows, const int32_t* num_rows, int32_t cap_rows, int32_t D, int32_t P,
                       float* blocks, int32_t* send_counts, void* stream) {
  if (cap_rows < 0 || bad_column_split(D, P)) return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && (!rows || !blocks)) return EMB_ERR_INVALID_ARG;
  return launch_status(
      emb::launch_column_pack(rows, num_rows, cap_rows, D, P, blocks, send_counts, static_cast<hipStream_t>(stream)));
}

int emb_gather_by_column(const float* shards, int64_t V, int32_t D, int32_t P, const int32_t* ids, int32_t T,
                         float* blocks, int32_t* dev_status, void* stream) {
  if (bad_table_dims(V, D) || bad_column_split(D, P) || T < 0) return EMB_ERR_INVALID_ARG;
  if (T > 0 && (!shards || !ids || !blocks)) return EMB_ERR_INVALID_ARG;
  return launch_status(
      emb::launch_column_gather(shards, V, D, P, ids, T, blocks, dev_status, static_cast<hipStream_t>(stream)));
}

int emb_assemble_by_column(const float* blocks, int64_t C, int64_t row0, int32_t R, int32_t D, int32_t P,
                           float* rows, void* stream) {
  if (bad_column_split(D, P) || C < 0 || row0 < 0 || R < 0 || row0 > C - R) return EMB_ERR_INVALID_ARG;
  if (R > 0 && (!blocks || !rows)) return EMB_ERR_INVALID_ARG;
  return launch_status(
      emb::launch_column_assemble(blocks, C, row0, R, D, P, rows, static_cast<hipStream_t>(stream)));
}

int emb_comm_cost(int32_t scheme, int64_t N, int64_t S, double M, double alpha, double B, double beta,
                  double* seconds) {
  if (!seconds || N < 1 || S < 1 || !(M >= 0) || !(alpha >= 0 && alpha <= 1) || !(B > 0) || !(beta >= 0) ||
      !std::isfinite(M) || !std::isfinite(B) || !std::isfinite(beta))
    return EMB_ERR_INVALID_ARG;
  const double n = static_cast<double>(N);
  const double sparse = alpha * M;  // bytes of the sparse gradient
  switch (scheme) {
    case EMB_COMM_ALLTOALL:  // N - 1 peers, 1/N of the sparse gradient each, twice
      *seconds = 2.0 * (n - 1.0) * (sparse / (n * B) + beta);
      return EMB_OK;
    case EMB_COMM_ALLREDUCE:  // ring reduce-scatter then all-gather of dense 1/N chunks
      *seconds = 2.0 * (n - 1.0) * (M / (n * B) + beta);
      return EMB_OK;
    case EMB_COMM_PS:  // pull and push of the sparse rows, 1/S per server, N workers
      *seconds = 2.0 * n * (sparse / (static_cast<double>(S) * B) + beta);
      return EMB_OK;
    case EMB_COMM_ALLGATHER:  // every worker's whole sparse gradient to every other
      *seconds = (n - 1.0) * (sparse / B + beta);
      return EMB_OK;
    default:
      return EMB_ERR_INVALID_ARG;
  }
}

size_t emb_pack_by_owner_workspace_bytes(int32_t cap_rows, int32_t P) {
  if (cap_rows < 0 || P < 1 || P > kMaxOwners) return 0;
  return emb::pack_workspace_bytes(cap_rows, P);
}

int emb_pack_by_owner(const int32_t* uniq_ids, const float* uniq_grad, const int32_t* num_unique, int32_t cap_rows,
                      int32_t D, const int32_t* row_owner, int64_t V, int32_t P, int32_t* send_ids, float* send_rows,
                      int32_t* send_counts, int32_t* send_offsets, void* workspace, size_t workspace_bytes,
                      int32_t* dev_status, void* stream) {
  if (cap_rows < 0 || bad_table_dims(V, D) || P < 1 || P > kMaxOwners) return EMB_ERR_INVALID_ARG;
  if (!send_counts || !send_offsets) return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && (!uniq_ids || !uniq_grad || !num_unique || !row_owner || !send_ids || !send_rows ||
                       !workspace))
    return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return EMB_ERR_INVALID_ARG;
  if (cap_rows > 0 && workspace_bytes < emb::pack_workspace_bytes(cap_rows, P)) return EMB_ERR_WORKSPACE;
  return launch_status(emb::launch_pack(uniq_ids, uniq_grad, num_unique, cap_rows, D, row_owner, V, P, send_ids,
                                        send_rows, send_counts, send_offsets, workspace, dev_status,
                                        static_cast<hipStream_t>(stream)));
}

int emb_sparse_adam_apply(float* table, float* exp_avg, float* exp_avg_sq, int64_t V, int32_t D,
                          const int32_t* row_ids, const float* rows, const int32_t* offsets, int32_t P,
                          int32_t shard_begin, int32_t shard_end, int32_t cap_rows, double lr, double beta1,
                          double beta2, double eps, int64_t step, int32_t* dev_status, void* stream) {
  return emb::sparse_adam_call(table, exp_avg, exp_avg_sq, V, D, row_ids, rows, offsets, P, shard_begin, shard_end,
                               cap_rows, lr, beta1, beta2, eps, step, nullptr, dev_status,
                               static_cast<hipStream_t>(stream), nullptr, nullptr);
}

int emb_adam_coeffs(double lr, double beta1, double beta2, double eps, int64_t step, float* out) {
  if (out == nullptr) return EMB_ERR_INVALID_ARG;
  emb::AdamCoeffs c;
  const int st = emb::adam_coeffs(lr, beta1, beta2, eps, step, &c);
  if (st != EMB_OK) return st;
  const float words[EMB_ADAM_COEFFS_WORDS] = {c.beta1, c.one_minus_beta1, c.beta2, c.one_minus_beta2,
                                              c.step_size, c.inv_bc2, c.eps, 0.0f};
  for (int i = 0; i < EMB_ADAM_COEFFS_WORDS; ++i) out[i] = words[i];
  return EMB_OK;
}

}  // extern "C"
