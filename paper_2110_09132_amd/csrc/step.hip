// Step executor: one host call enqueues a whole training step of one table
// on three streams with the event waits of the schedule in include/emb.h.
#include "common.h"
#include "launch.h"

namespace {

hipStream_t S(void* p) { return static_cast<hipStream_t>(p); }
hipEvent_t E(void* p) { return static_cast<hipEvent_t>(p); }

int record(void* ev, void* stream) {
  if (ev == nullptr) return EMB_OK;
  return hipEventRecord(E(ev), S(stream)) == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
}

int wait(void* stream, void* ev) {
  return hipStreamWaitEvent(S(stream), E(ev), 0) == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
}

}  // namespace

extern "C" {

int emb_event_create(void** event, int32_t timing) {
  if (event == nullptr) return EMB_ERR_INVALID_ARG;
  hipEvent_t e;
  if (hipEventCreateWithFlags(&e, timing ? hipEventDefault : hipEventDisableTiming) != hipSuccess)
    return EMB_ERR_LAUNCH;
  *event = e;
  return EMB_OK;
}

int emb_event_destroy(void* event) {
  if (event == nullptr) return EMB_ERR_INVALID_ARG;
  return hipEventDestroy(E(event)) == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
}

int emb_event_elapsed_ms(void* start, void* end, float* ms) {
  if (start == nullptr || end == nullptr || ms == nullptr) return EMB_ERR_INVALID_ARG;
  return hipEventElapsedTime(ms, E(start), E(end)) == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
}

int emb_train_step(const emb_step_args* a, const emb_step_schedule* s) {
  if (a == nullptr || s == nullptr) return EMB_ERR_INVALID_ARG;
  if (s->coalesced == nullptr || s->updated == nullptr) return EMB_ERR_INVALID_ARG;
  if ((s->by_owner ? s->sorted : s->packed) == nullptr) return EMB_ERR_INVALID_ARG;
  if (a->T < 0 || a->cap_rows < a->T) return EMB_ERR_INVALID_ARG;
  const bool sep_c = s->coalesce != s->lookup_update;
  const bool sep_p = s->pack != s->lookup_update;
  int st = EMB_OK;
  // each step stops the sequence at the first failing call
  auto ok = [&st](int r) { return (st = r) == EMB_OK; };
  if (s->by_owner) {
    // owner-major coalesce in its two halves: the sort on the coalesce stream,
    // the reduction (straight into the send buffers) on the pack stream, the
    // lookup and the update on the main stream
    if (!ok(emb::coalesce_by_owner_args_status(a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->row_owner, a->P,
                                               a->send_ids, a->seg_offsets, a->send_rows, a->send_counts,
                                               a->send_offsets, a->num_unique, a->ws_coalesce, a->ws_coalesce_bytes)))
      return st;
    auto launched = [](hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH; };
    const bool sep_sr = s->coalesce != s->pack;  // sort beside the reduction
    // sort(s): after the reduction of step s-2 has finished with this set's workspace
    if (s->reuse && sep_sr && !ok(wait(s->coalesce, s->coalesced))) return st;
    if (!ok(record(s->timing[2], s->coalesce))) return st;
    if (!ok(launched(emb::launch_coalesce_sort(a->ids, a->T, a->V, a->D, a->row_owner, a->P, a->ws_coalesce,
                                               a->dev_status, S(s->coalesce)))))
      return st;
    if (sep_sr && !ok(record(s->sorted, s->coalesce))) return st;
    // reduction(s): after the sort, and after update(s-2) has read this set's send buffers
    if (sep_sr && !ok(wait(s->pack, s->sorted))) return st;
    if (s->reuse && sep_p && !ok(wait(s->pack, s->updated))) return st;
    if (!ok(launched(emb::launch_coalesce_reduce(a->T, a->grad, a->grad_dtype == EMB_BF16, a->D, a->V, a->row_owner,
                                                 a->P, a->send_ids, a->seg_offsets, a->send_rows, a->num_unique,
                                                 a->send_counts, a->send_offsets, a->ws_coalesce, S(s->pack),
                                                 (sep_sr || sep_p) ? E(s->coalesced) : nullptr))))
      return st;
    if (!ok(record(s->timing[3], s->pack))) return st;
    // lookup(s), then update(s) once the rows are reduced
    if (!ok(record(s->timing[0], s->lookup_update))) return st;
    if (!ok(emb_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status, s->lookup_update))) return st;
    if (!ok(record(s->timing[1], s->lookup_update))) return st;
    if (sep_p && !ok(wait(s->lookup_update, s->coalesced))) return st;
  } else {
    // coalesce(s): after pack(s-2) has read this buffer set's unique rows
    if (s->reuse && s->coalesce != s->pack && !ok(wait(s->coalesce, s->packed))) return st;
    if (!ok(record(s->timing[2], s->coalesce))) return st;
    if (!ok(emb_grad_coalesce(a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->uniq_ids, a->seg_offsets,
                              a->uniq_grad, a->num_unique, a->ws_coalesce, a->ws_coalesce_bytes, a->dev_status,
                              s->coalesce)))
      return st;
    if (!ok(record(s->timing[3], s->coalesce)) || !ok(record(s->coalesced, s->coalesce))) return st;
    // pack(s): after coalesce(s), and after update(s-2) has read this set's send rows
    if (s->pack != s->coalesce && !ok(wait(s->pack, s->coalesced))) return st;
    if (s->reuse && sep_p && !ok(wait(s->pack, s->updated))) return st;
    if (!ok(record(s->timing[4], s->pack))) return st;
    if (!ok(emb_pack_by_owner(a->uniq_ids, a->uniq_grad, a->num_unique, a->cap_rows, a->D, a->row_owner, a->V, a->P,
                              a->send_ids, a->send_rows, a->send_counts, a->send_offsets, a->ws_pack,
                              a->ws_pack_bytes, a->dev_status, s->pack)))
      return st;
    if (!ok(record(s->timing[5], s->pack)) || !ok(record(s->packed, s->pack))) return st;
    // lookup(s) on the main stream, then update(s) once the rows are packed
    if (!ok(record(s->timing[0], s->lookup_update))) return st;
    if (!ok(emb_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status, s->lookup_update))) return st;
    if (!ok(record(s->timing[1], s->lookup_update))) return st;
    if (sep_p && !ok(wait(s->lookup_update, s->packed))) return st;
  }
  // Events after a kernel are attached to its dispatch where possible: that
  // costs less idle time on the stream than a separate marker.
  void* update_end = s->timing[7];
  void* after_update = nullptr;
  if (sep_p) {  // the pack stream's next use of this set waits for it
    if (update_end == nullptr)
      update_end = s->updated;
    else
      after_update = s->updated;
  }
  if (!ok(emb::sparse_adam_call(a->table, a->exp_avg, a->exp_avg_sq, a->V, a->D, a->send_ids, a->send_rows,
                                a->send_offsets, a->P, 0, a->P, a->cap_rows, a->lr, a->beta1, a->beta2, a->eps,
                                a->step, a->dev_status, S(s->lookup_update), E(s->timing[6]), E(update_end))))
    return st;
  if (!ok(record(after_update, s->lookup_update))) return st;
  return EMB_OK;
}

}  // extern "C"
