// Step executor: one host call enqueues a whole training step of one table
// on up to four streams, with the cross-stream order of the schedule in
// include/emb.h kept either by the caller's events or by step signals.
//
// Step signals are words of HIP signal memory, one per stage (sorted,
// coalesced, packed, updated, gathered, delayed_done).  The end of a stage of
// step n writes n into its word (hipStreamWriteValue32, after the stage's
// kernels on that stream); a stream that must follow the stage of step n - k
// waits for the word to reach n - k (hipStreamWaitValue32, ">=").  The step
// numbers are kept by the handle, so the values only grow.  A wait on an event
// that is still pending costs the host far more than these two operations,
// and with the host running steps ahead of the GPU nearly every wait is.
#include <chrono>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "common.h"
#include "launch.h"

namespace {

hipStream_t S(void* p) { return static_cast<hipStream_t>(p); }
hipEvent_t E(void* p) { return static_cast<hipEvent_t>(p); }

int status_of(hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH; }

int record(void* ev, void* stream) {
  if (ev == nullptr) return EMB_OK;
  return status_of(hipEventRecord(E(ev), S(stream)));
}

int wait(void* stream, void* ev) { return status_of(hipStreamWaitEvent(S(stream), E(ev), 0)); }

enum Stage { kSorted = 0, kCoalesced, kPacked, kUpdated, kGathered, kDelayedDone, kStages };

// Two words per stage, for the steps of even and of odd number: in a schedule
// whose odd and even steps run on two streams, each word then has one writer.
struct StepSignals {
  int device;
  void* word[kStages][2];       // hipMallocSignalMemory allocations
  uint32_t seq;                 // number of the last step enqueued with this handle
  uint32_t written[kStages][2]; // the largest value a write already enqueued puts in each word
  void* writer[kStages][2];     // the stream of that write
};

// Released handles are kept for reuse rather than freed, so that no signal
// memory a queue may still poll is ever returned to the runtime.
std::mutex g_pool_mu;
std::vector<StepSignals*> g_pool;

// The cross-stream order of one step.
struct Order {
  const emb_step_schedule* s;
  StepSignals* sig;  // null: the schedule's events
  uint32_t seq;      // this step's number (signals)
  uint32_t sets;     // buffer sets in rotation: a set's buffers come back after this many steps
  bool capturing;    // the streams are being captured into a graph: no events attached to dispatches

  void* event(Stage k) const {
    switch (k) {
      case kSorted: return s->sorted;
      case kCoalesced: return s->coalesced;
      case kPacked: return s->packed;
      case kUpdated: return s->updated;
      case kGathered: return s->gathered;
      default: return s->delayed_done;
    }
  }
  // The event to attach to the last kernel of stage k (events only, and not under capture, where an
  // event attached to a dispatch would not become a node of the graph).
  hipEvent_t attach(Stage k) const { return (sig != nullptr || capturing) ? nullptr : E(event(k)); }
  // Stage k of this step ends here on `stream`; `attached`: its event was attached to the last kernel.
  int done(Stage k, void* stream, bool attached = false) const {
    if (sig != nullptr) return write(k, stream);
    return attached ? EMB_OK : record(event(k), stream);
  }
  // Writes this step's number into word k on `stream`.  The values written to
  // a word strictly increase (a second write of the same step is dropped), and
  // the writes stay in enqueue order, so the value only grows: a write on
  // another stream than the word's last one first waits for that write.
  int write(Stage k, void* stream) const {
    const int q = seq & 1;
    if (sig->written[k][q] >= seq) return EMB_OK;
    if (sig->written[k][q] != 0 && sig->writer[k][q] != stream &&
        hipStreamWaitValue32(S(stream), sig->word[k][q], sig->written[k][q], hipStreamWaitValueGte,
                             0xFFFFFFFFu) != hipSuccess)
      return EMB_ERR_LAUNCH;
    if (hipStreamWriteValue32(S(stream), sig->word[k][q], seq, 0) != hipSuccess) return EMB_ERR_LAUNCH;
    sig->written[k][q] = seq;
    sig->writer[k][q] = stream;
    return EMB_OK;
  }
  // `stream` waits for stage k of the step `lag` steps back (lag 0: this step).  A wait on a stage
  // that ran on the waiting stream itself is implied by stream order and costs nothing: the runtime
  // skips a wait on an event recorded on the waiting stream, and with signals it is left out below.
  // With events, a lag > 0 means the step that last used this buffer set (the
  // set's own event), so it must equal `sets`.
  // With signals the wait uses the word of that step's parity, and the target
  // never exceeds what an enqueued write will put in the word: a stage that did
  // not run in that step (another mode, a failed call) is waited for at its
  // last run in a step of that parity, or not at all.  Every
  // wait thus refers to a write enqueued before it, so the waits cannot form a
  // cycle.
  int after(void* stream, Stage k, uint32_t lag) const {
    if (sig != nullptr) {
      if (seq <= lag) return EMB_OK;  // no such step
      const uint32_t n = seq - lag;
      const int q = n & 1;
      const uint32_t target = n < sig->written[k][q] ? n : sig->written[k][q];
      if (target == 0) return EMB_OK;  // the stage never ran in a step of that parity
      // The word's last write was enqueued on this stream: every write to the word is ordered before
      // it (a write on another stream than the previous one waits for that one first), so the word
      // holds at least the target by the time this stream gets here.
      if (sig->writer[k][q] == stream) return EMB_OK;
      return status_of(hipStreamWaitValue32(S(stream), sig->word[k][q], target, hipStreamWaitValueGte, 0xFFFFFFFFu));
    }
    if (lag > 0 && !s->reuse) return EMB_OK;  // the buffer set was not used before
    return wait(stream, event(k));
  }
  // After a failure part-way: mark every stage of this step done, so that no
  // later wait is left without the write it needs.
  void release_all() const {
    if (sig == nullptr) return;
    void* const streams[kStages] = {s->coalesce, s->pack, s->pack, s->lookup_update, s->lookup_update, s->delayed};
    for (int k = 0; k < kStages; ++k) (void)write(static_cast<Stage>(k), streams[k]);
  }
};

// Waits on the earlier use of this buffer set (and the split's wait two steps back) are issued
// whatever the streams, since a set's streams may differ from one use to the next; the stage ends
// they refer to are always announced.  Waits inside one step are issued between different streams
// only.
// Adam on the groups [groups_from, groups_from + P) of the send layout.  An
// event after the kernel is attached to its dispatch (less idle time on the
// stream than a separate marker): the timing event if any, else the end event.
int enqueue_update(const emb_step_args* a, const Order& order, int32_t groups_from, void* stream, void* t0, void* t1,
                   Stage end_stage) {
  const hipEvent_t end_ev = order.attach(end_stage);
  const hipEvent_t first = t1 != nullptr ? E(t1) : end_ev;
  const int st = emb::sparse_adam_call(a->table, a->exp_avg, a->exp_avg_sq, a->V, a->D, a->send_ids, a->send_rows,
                                       a->send_offsets + groups_from, a->P, 0, a->P, a->cap_rows, a->lr, a->beta1,
                                       a->beta2, a->eps, a->step, a->adam_coeffs, a->dev_status, S(stream), E(t0),
                                       first);
  if (st != EMB_OK) return st;
  return order.done(end_stage, stream, t1 == nullptr && end_ev != nullptr);
}

// The side half of an owner-major step: the sort on the coalesce stream, the
// reduction (straight into the send buffers) on the pack stream, with their waits.
int enqueue_by_owner_side(const emb_step_args* a, const emb_step_schedule* s, const Order& order) {
  const bool sep_p = s->pack != s->lookup_update;
  int st = EMB_OK;
  auto ok = [&st](int r) { return (st = r) == EMB_OK; };
  auto launched = [](hipError_t e) { return status_of(e); };
  emb::CoalesceVariant var;
  var.row_owner = a->row_owner;
  var.P = a->P;
  if (s->split) {
    var.next_ids = a->next_ids;
    var.T_next = a->T_next;
  }
  const bool sep_sr = s->coalesce != s->pack;  // sort beside the reduction
  // With four or more sets the sort waits for the update of the set's last
  // step (s - sets), which came after that step's reduction: the workspace and
  // the send buffers are then both free once the sort has run, and the
  // reduction needs to wait for the sort alone (one cross-stream wait fewer;
  // with two sets it would hold the sort back by a whole update).
  const bool chained = order.sets >= 4 && !s->split && sep_sr && sep_p;
  // sort(s): after the reduction of the set's last step (s - sets) has finished with its workspace
  if (!ok(order.after(s->coalesce, chained ? kUpdated : kCoalesced, order.sets))) return st;
  if (!ok(record(s->timing[2], s->coalesce))) return st;
  if (!ok(launched(emb::launch_coalesce_sort(a->ids, a->T, a->V, a->D, var, a->ws_coalesce, a->dev_status,
                                             S(s->coalesce)))))
    return st;
  if (sep_sr && !ok(order.done(kSorted, s->coalesce))) return st;
  // reduction(s): after the sort, and after the updates of step s - sets have read this set's send buffers
  if (sep_sr && !ok(order.after(s->pack, kSorted, 0))) return st;
  if (!chained && !ok(order.after(s->pack, kUpdated, order.sets))) return st;
  if (s->split && !ok(order.after(s->pack, kDelayedDone, order.sets))) return st;
  const hipEvent_t coalesced_ev = order.attach(kCoalesced);
  if (!ok(launched(emb::launch_coalesce_reduce(a->ids, a->T, a->grad, a->grad_dtype == EMB_BF16, a->D, a->V, var,
                                               a->send_ids, a->seg_offsets, a->send_rows, a->num_unique,
                                               a->send_counts, a->send_offsets, a->ws_coalesce, a->dev_status,
                                               S(s->pack), coalesced_ev))))
    return st;
  if (!ok(order.done(kCoalesced, s->pack, coalesced_ev != nullptr))) return st;
  return record(s->timing[3], s->pack);
}

// The main half of an owner-major step without the split: the lookup, then the
// update once the rows are reduced, on lookup_update.
int enqueue_by_owner_main(const emb_step_args* a, const emb_step_schedule* s, const Order& order) {
  const bool sep_p = s->pack != s->lookup_update;
  int st = EMB_OK;
  auto ok = [&st](int r) { return (st = r) == EMB_OK; };
  if (!ok(record(s->timing[0], s->lookup_update))) return st;
  if (!ok(emb_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status, s->lookup_update))) return st;
  if (!ok(record(s->timing[1], s->lookup_update))) return st;
  if (sep_p && !ok(order.after(s->lookup_update, kCoalesced, 0))) return st;
  // the next use of this set waits for `updated`
  return enqueue_update(a, order, 0, s->lookup_update, s->timing[6], s->timing[7], kUpdated);
}

int enqueue_step(const emb_step_args* a, const emb_step_schedule* s, const Order& order) {
  const bool sep_p = s->pack != s->lookup_update;
  int st = EMB_OK;
  // each step stops the sequence at the first failing call
  auto ok = [&st](int r) { return (st = r) == EMB_OK; };
  auto launched = [](hipError_t e) { return status_of(e); };
  if (s->by_owner) {
    // owner-major coalesce in its two halves: the sort on the coalesce stream,
    // the reduction (straight into the send buffers) on the pack stream, the
    // lookup and the update on the main stream; with the split, the delayed
    // rows are updated on the delayed stream
    if (!ok(enqueue_by_owner_side(a, s, order))) return st;
    if (!s->split) return enqueue_by_owner_main(a, s, order);
    // lookup(s): after the delayed update of step s-2 (its rows may be in this
    // batch; those of step s-1 are not, by construction)
    const bool sep_d = s->delayed != s->lookup_update;
    if (!ok(order.after(s->lookup_update, kDelayedDone, 2))) return st;
    if (!ok(record(s->timing[0], s->lookup_update))) return st;
    const hipEvent_t gathered_ev = order.attach(kGathered);
    if (!ok(launched(emb::launch_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status,
                                        S(s->lookup_update), gathered_ev))))
      return st;
    if (!ok(order.done(kGathered, s->lookup_update, gathered_ev != nullptr))) return st;
    if (!ok(record(s->timing[1], s->lookup_update))) return st;
    // prior update(s): the rows the next lookup reads, right after this lookup
    if (sep_p && !ok(order.after(s->lookup_update, kCoalesced, 0))) return st;
    if (!ok(enqueue_update(a, order, 0, s->lookup_update, s->timing[4], s->timing[5], kUpdated))) return st;
    // delayed update(s): beside the next lookup (it reads none of these rows),
    // after this step's lookup has read them and the reduction has written them
    if (sep_d && !ok(order.after(s->delayed, kGathered, 0))) return st;
    if (s->delayed != s->pack && !ok(order.after(s->delayed, kCoalesced, 0))) return st;
    return enqueue_update(a, order, a->P, s->delayed, s->timing[6], s->timing[7], kDelayedDone);
  }
  // coalesce(s): after pack(s - sets) has read this buffer set's unique rows
  if (!ok(order.after(s->coalesce, kPacked, order.sets))) return st;
  if (!ok(record(s->timing[2], s->coalesce))) return st;
  if (!ok(emb_grad_coalesce(a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->uniq_ids, a->seg_offsets,
                            a->uniq_grad, a->num_unique, a->ws_coalesce, a->ws_coalesce_bytes, a->dev_status,
                            s->coalesce)))
    return st;
  if (!ok(record(s->timing[3], s->coalesce)) || !ok(order.done(kCoalesced, s->coalesce))) return st;
  // pack(s): after coalesce(s), and after update(s - sets) has read this set's send rows
  if (s->pack != s->coalesce && !ok(order.after(s->pack, kCoalesced, 0))) return st;
  if (!ok(order.after(s->pack, kUpdated, order.sets))) return st;
  if (!ok(record(s->timing[4], s->pack))) return st;
  if (!ok(emb_pack_by_owner(a->uniq_ids, a->uniq_grad, a->num_unique, a->cap_rows, a->D, a->row_owner, a->V, a->P,
                            a->send_ids, a->send_rows, a->send_counts, a->send_offsets, a->ws_pack,
                            a->ws_pack_bytes, a->dev_status, s->pack)))
    return st;
  if (!ok(record(s->timing[5], s->pack)) || !ok(order.done(kPacked, s->pack))) return st;
  // lookup(s) on the main stream, then update(s) once the rows are packed
  if (!ok(record(s->timing[0], s->lookup_update))) return st;
  if (!ok(emb_gather(a->table, a->V, a->D, a->ids, a->T, a->lookup, a->dev_status, s->lookup_update))) return st;
  if (!ok(record(s->timing[1], s->lookup_update))) return st;
  if (sep_p && !ok(order.after(s->lookup_update, kPacked, 0))) return st;
  // the next use of this set waits for `updated`
  return enqueue_update(a, order, 0, s->lookup_update, s->timing[6], s->timing[7], kUpdated);
}

// Two-thread enqueue (emb_step_queue_*).  The caller's thread enqueues the
// side half of each step itself and posts the main half (the lookup, the wait
// for the reduction, the update) to a worker thread, which enqueues the main
// halves in posting order.  Host order: a main half is posted after its side
// half has recorded the event it waits for; a side half that reuses a buffer
// set first waits (on the host) until the worker has enqueued the main half
// of the set's previous use, whose update event it waits for and whose wait
// on the set's coalesced event must precede that event's next record.
struct PostedMain {
  emb_step_args a;
  emb_step_schedule s;
  uint32_t sets;
  int device;
};

struct StepQueue {
  std::mutex mu;
  std::condition_variable work, progress;
  std::deque<PostedMain> posted_q;
  uint64_t posted = 0;  // main halves posted
  uint64_t done = 0;    // main halves the worker has enqueued (or failed)
  int error = EMB_OK;   // the first failure of a main half
  bool stop = false;
  std::thread worker;

  void run() {
    int current = -1;
    for (;;) {
      PostedMain m;
      {
        std::unique_lock<std::mutex> lock(mu);
        work.wait(lock, [this] { return stop || !posted_q.empty(); });
        if (posted_q.empty()) return;  // stopped with nothing left
        m = posted_q.front();
        posted_q.pop_front();
      }
      int st = EMB_OK;
      if (m.device != current) {
        st = hipSetDevice(m.device) == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
        if (st == EMB_OK) current = m.device;
      }
      if (st == EMB_OK) {
        const Order order{&m.s, nullptr, 0, m.sets, false};
        st = enqueue_by_owner_main(&m.a, &m.s, order);
      }
      {
        std::lock_guard<std::mutex> lock(mu);
        if (st != EMB_OK && error == EMB_OK) error = st;
        ++done;
      }
      progress.notify_all();
    }
  }
  // Waits until the worker has enqueued `n` main halves; false after kQueueWaitLimit.
  bool wait_done(std::unique_lock<std::mutex>& lock, uint64_t n) {
    return progress.wait_for(lock, kQueueWaitLimit, [this, n] { return done >= n; });
  }
  static constexpr std::chrono::seconds kQueueWaitLimit{30};
};

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

int emb_step_signals_create(void** signals) {
  if (signals == nullptr) return EMB_ERR_INVALID_ARG;
  int dev = 0, can = 0;
  if (hipGetDevice(&dev) != hipSuccess) return EMB_ERR_LAUNCH;
  if (hipDeviceGetAttribute(&can, hipDeviceAttributeCanUseStreamWaitValue, dev) != hipSuccess) return EMB_ERR_LAUNCH;
  if (!can) return EMB_ERR_UNSUPPORTED;
  {
    std::lock_guard<std::mutex> lock(g_pool_mu);
    for (size_t i = 0; i < g_pool.size(); ++i) {
      if (g_pool[i]->device == dev) {  // values and step number carry on from the last user
        *signals = g_pool[i];
        g_pool.erase(g_pool.begin() + static_cast<std::ptrdiff_t>(i));
        return EMB_OK;
      }
    }
  }
  auto* h = new StepSignals{};
  h->device = dev;
  for (int k = 0; k < kStages; ++k)  // on failure the partial handle is dropped, not freed
    for (int q = 0; q < 2; ++q)
      if (hipExtMallocWithFlags(&h->word[k][q], 8, hipMallocSignalMemory) != hipSuccess ||
          hipStreamWriteValue32(nullptr, h->word[k][q], 0, 0) != hipSuccess)
        return EMB_ERR_LAUNCH;
  if (hipStreamSynchronize(nullptr) != hipSuccess) return EMB_ERR_LAUNCH;
  *signals = h;
  return EMB_OK;
}

int emb_step_signals_destroy(void* signals) {
  if (signals == nullptr) return EMB_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  g_pool.push_back(static_cast<StepSignals*>(signals));
  return EMB_OK;
}

int emb_step_queue_create(void** queue) {
  if (queue == nullptr) return EMB_ERR_INVALID_ARG;
  auto* q = new StepQueue;
  try {
    q->worker = std::thread([q] { q->run(); });
  } catch (...) {
    delete q;
    return EMB_ERR_LAUNCH;
  }
  *queue = q;
  return EMB_OK;
}

int emb_step_queue_flush(void* queue) {
  if (queue == nullptr) return EMB_ERR_INVALID_ARG;
  auto* q = static_cast<StepQueue*>(queue);
  std::unique_lock<std::mutex> lock(q->mu);
  if (!q->wait_done(lock, q->posted)) return EMB_ERR_LAUNCH;
  return q->error;
}

int emb_step_queue_destroy(void* queue) {
  if (queue == nullptr) return EMB_ERR_INVALID_ARG;
  auto* q = static_cast<StepQueue*>(queue);
  {
    std::lock_guard<std::mutex> lock(q->mu);
    q->stop = true;
  }
  q->work.notify_all();
  q->worker.join();  // the worker enqueues what was posted before it stops
  const int st = q->error;
  delete q;
  return st;
}

int emb_train_step(const emb_step_args* a, const emb_step_schedule* s) {
  if (a == nullptr || s == nullptr) return EMB_ERR_INVALID_ARG;
  if (a->T < 0 || a->cap_rows < a->T) return EMB_ERR_INVALID_ARG;
  const bool events = s->signals == nullptr;
  if (events && (s->coalesced == nullptr || s->updated == nullptr)) return EMB_ERR_INVALID_ARG;
  if (s->split && (!s->by_owner || a->T_next < 0 || a->T_next > a->cap_rows))
    return EMB_ERR_INVALID_ARG;  // streams may be NULL: the null stream
  if (events && s->split && (s->sorted == nullptr || s->gathered == nullptr || s->delayed_done == nullptr))
    return EMB_ERR_INVALID_ARG;
  if (events && (s->by_owner ? s->sorted : s->packed) == nullptr) return EMB_ERR_INVALID_ARG;
  const uint32_t sets = s->sets == 0 ? 2u : static_cast<uint32_t>(s->sets);
  // the split's lookup waits for the delayed update two steps back, a data
  // dependency that the set's own events express only with two sets
  if (s->sets < 0 || s->sets > 64 || (events && s->split && sets != 2)) return EMB_ERR_INVALID_ARG;
  // arguments of the calls that fail on the host, checked before anything is enqueued
  if (s->by_owner) {
    const int st = emb::coalesce_by_owner_args_status(
        a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->row_owner, a->P, s->split ? a->next_ids : nullptr,
        s->split ? a->T_next : -1, a->send_ids, a->seg_offsets, a->send_rows, a->send_counts, a->send_offsets,
        a->num_unique, a->ws_coalesce, a->ws_coalesce_bytes);
    if (st != EMB_OK) return st;
  }
  // under stream capture: events only, no timing pairs, no events attached to dispatches
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(S(s->lookup_update), &cap) != hipSuccess) return EMB_ERR_LAUNCH;
  const bool capturing = cap != hipStreamCaptureStatusNone;
  if (capturing) {
    if (!events) return EMB_ERR_UNSUPPORTED;
    for (void* t : s->timing)
      if (t != nullptr) return EMB_ERR_UNSUPPORTED;
  }
  if (a->adam_coeffs != nullptr && reinterpret_cast<uintptr_t>(a->adam_coeffs) % 16 != 0) return EMB_ERR_INVALID_ARG;
  Order order{s, static_cast<StepSignals*>(s->signals), 0, sets, capturing};
  if (order.sig != nullptr) order.seq = ++order.sig->seq;
  const int st = enqueue_step(a, s, order);
  if (st != EMB_OK) order.release_all();
  return st;
}

int emb_train_step_queued(void* queue, const emb_step_args* a, const emb_step_schedule* s) {
  if (queue == nullptr || a == nullptr || s == nullptr) return EMB_ERR_INVALID_ARG;
  // events, owner-major without the split, outside graph capture, and the sort and the reduction
  // on other streams than the lookup and the update (each stream is fed by one host thread)
  if (s->signals != nullptr || !s->by_owner || s->split) return EMB_ERR_UNSUPPORTED;
  if (s->coalesce == s->lookup_update || s->pack == s->lookup_update) return EMB_ERR_UNSUPPORTED;
  if (a->T < 0 || a->cap_rows < a->T) return EMB_ERR_INVALID_ARG;
  if (s->coalesced == nullptr || s->updated == nullptr || s->sorted == nullptr) return EMB_ERR_INVALID_ARG;
  if (s->sets < 0 || s->sets > 64) return EMB_ERR_INVALID_ARG;
  const uint32_t sets = s->sets == 0 ? 2u : static_cast<uint32_t>(s->sets);
  const int ast = emb::coalesce_by_owner_args_status(
      a->ids, a->T, a->grad, a->grad_dtype, a->D, a->V, a->row_owner, a->P, nullptr, -1, a->send_ids, a->seg_offsets,
      a->send_rows, a->send_counts, a->send_offsets, a->num_unique, a->ws_coalesce, a->ws_coalesce_bytes);
  if (ast != EMB_OK) return ast;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(S(s->lookup_update), &cap) != hipSuccess) return EMB_ERR_LAUNCH;
  if (cap != hipStreamCaptureStatusNone) return EMB_ERR_UNSUPPORTED;
  if (a->adam_coeffs != nullptr && reinterpret_cast<uintptr_t>(a->adam_coeffs) % 16 != 0) return EMB_ERR_INVALID_ARG;
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) return EMB_ERR_LAUNCH;
  auto* q = static_cast<StepQueue*>(queue);
  {
    // this step reuses the buffer set of step posted - sets: its main half must be enqueued
    std::unique_lock<std::mutex> lock(q->mu);
    if (q->posted >= sets && !q->wait_done(lock, q->posted - sets + 1)) return EMB_ERR_LAUNCH;
    if (q->error != EMB_OK) return q->error;
  }
  const Order order{s, nullptr, 0, sets, false};
  const int st = enqueue_by_owner_side(a, s, order);
  if (st != EMB_OK) return st;
  {
    std::lock_guard<std::mutex> lock(q->mu);
    q->posted_q.push_back(PostedMain{*a, *s, sets, device});
    ++q->posted;
  }
  q->work.notify_one();
  return EMB_OK;
}

}  // extern "C"
