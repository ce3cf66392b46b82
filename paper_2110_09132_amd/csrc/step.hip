// Step executor: one host call enqueues a whole training step of one table
// on up to four streams with the event waits of the schedule in include/emb.h.
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
  if (a->T < 0 || a->cap_rows < a->T) return EMB_ERR_INVALID_ARG;
  if (s->coalesced == nullptr || s->updated == nullptr) return EMB_ERR_INVALID_ARG;
  if (s->split && (!s->by_owner || s->sorted == nullptr || s->gathered == nullptr || s->delayed_done == nullptr ||
                   a->T_next < 0 || a->T_next > a->cap_rows))  // streams may be NULL: the null stream
    return EMB_ERR_INVALID_ARG;
  if ((s->by_owner ? s->sorted : s->packed) == nullptr) return EMB_ERR_INVALID_ARG;
  const bool sep_p = s->pack != s->lookup_update;
  int st = EMB_OK;
  // each step stops the sequence at the first failing call
  auto ok = [&st](int r) { return (st = r) == EMB_OK; };
  auto launched = [](hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH; };
  auto update = [&](int32_t groups_from, void* stream, void* t0, void* t1, void* end_event) {
    // Adam on the groups [groups_from, groups_from + P) of the send layout; the
    // event after the kernel is attached to its dispatch (less idle time on
    // the stream than a separate marker), a second one is recorded after it
    void* first = t1 != nullptr ? t1 : end_event;
    void* second = t1 != nullptr ? end_event : nullptr;
    return ok(emb::sparse_adam_call(a->table, a->exp_avg, a->exp_avg_sq, a->V, a->D, a->send_ids, a->send_rows,
                                    a->send_offsets + groups_from, a->P, 0, a->P, a->cap_rows, a->lr, a->beta1,
                                    a->beta2, a->eps, a->step, a->dev_status, S(stream), E(t0), E(first))) &&
           ok(record(second, stream));
  };
  if (s->by_owner) {
    // owner-major coalesce in its two halves: the sort on the coalesce stream,
    // the reduction (straight into the send buffers) on the pack stream, the
    // lookup and the update on the main stream; with the split, the delayed
    // rows are updated on the delayed stream
    emb::CoalesceVariant var;
    var.row_owner = a->row_owner;
    var.P = a->P;
    if (s->split) {
      var.next_ids = a->next_ids;
      var.T_next = a->T_next;
    }
    if (!ok(emb::coalesce_by_owner_args_status(a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->row_owner, a->P,
                                               var.next_ids, var.T_next, a->send_ids, a->seg_offsets, a->send_rows,
                                               a->send_counts, a->send_offsets, a->num_unique, a->ws_coalesce,
                                               a->ws_coalesce_bytes)))
      return st;
    const bool sep_sr = s->coalesce != s->pack;  // sort beside the reduction
    // sort(s): after the reduction of step s-2 has finished with this set's workspace
    if (s->reuse && sep_sr && !ok(wait(s->coalesce, s->coalesced))) return st;
    if (!ok(record(s->timing[2], s->coalesce))) return st;
    if (!ok(launched(emb::launch_coalesce_sort(a->ids, a->T, a->V, a->D, var, a->ws_coalesce, a->dev_status,
                                               S(s->coalesce)))))
      return st;
    if (sep_sr && !ok(record(s->sorted, s->coalesce))) return st;
    // reduction(s): after the sort, and after the updates of step s-2 have read this set's send buffers
    if (sep_sr && !ok(wait(s->pack, s->sorted))) return st;
    if (s->reuse && sep_p && !ok(wait(s->pack, s->updated))) return st;
    if (s->reuse && s->split && s->delayed != s->pack && !ok(wait(s->pack, s->delayed_done))) return st;
    if (!ok(launched(emb::launch_coalesce_reduce(a->T, a->grad, a->grad_dtype == EMB_BF16, a->D, a->V, var,
                                                 a->send_ids, a->seg_offsets, a->send_rows, a->num_unique,
                                                 a->send_counts, a->send_offsets, a->ws_coalesce, S(s->pack),
                                                 E(s->coalesced)))))
      return st;
    if (!ok(record(s->timing[3], s->pack))) return st;
    if (s->split) {
      // lookup(s): after the delayed update of step s-2 (its rows may be in this
      // batch; those of step s-1 are not, by construction)
      const bool sep_d = s->delayed != s->lookup_update;
      if (s->reuse && sep_d && !ok(wait(s->lookup_update, s->delayed_done))) return st;
      if (!ok(record(s->timing[0], s->lookup_update))) return st;
      if (!ok(launched(emb::launch_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status,
                                          S(s->lookup_update), E(s->gathered)))))
        return st;
      if (!ok(record(s->timing[1], s->lookup_update))) return st;
      // prior update(s): the rows the next lookup reads, right after this lookup
      if (sep_p && !ok(wait(s->lookup_update, s->coalesced))) return st;
      if (!update(0, s->lookup_update, s->timing[4], s->timing[5], s->updated)) return st;
      // delayed update(s): beside the next lookup (it reads none of these rows),
      // after this step's lookup has read them and the reduction has written them
      if (sep_d && !ok(wait(s->delayed, s->gathered))) return st;
      if (s->delayed != s->pack && !ok(wait(s->delayed, s->coalesced))) return st;
      if (!update(a->P, s->delayed, s->timing[6], s->timing[7], s->delayed_done)) return st;
      return EMB_OK;
    }
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
  // the pack stream's next use of this set waits for `updated`
  if (!update(0, s->lookup_update, s->timing[6], s->timing[7], sep_p ? s->updated : nullptr)) return st;
  return EMB_OK;
}

}  // extern "C"
