// Host-only check of the step executor's cross-stream order with step signals.
//
// The executor (step.hip) is linked against stand-ins for the HIP stream
// operations and for the kernel launchers: every launch, event record or
// wait, and signal write or wait is appended to a trace, per stream, instead
// of reaching a GPU.
// The trace is then executed by a model of the device (each stream runs its
// operations in order; a wait proceeds once its word holds at least its
// value; a write stores its value).  The program fails if a wait ever targets
// more than the writes enqueued before it can supply, or if the model stops
// with work left (a deadlock).  Scenarios: handles reused from the pool across
// modes, a call that fails part-way, and a long random mix of modes.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <deque>
#include <map>
#include <string>
#include <vector>

#include "emb.h"
#include "launch.h"

namespace {

enum Kind { kLaunch, kWrite, kWait, kRecord, kWaitEvent };
struct Op {
  Kind kind;
  long word;        // signal word index; for events: the record's number (a wait: the record it waits for, or -1)
  uint32_t value;   // written / waited-for value
  std::string what;
};

std::map<long, std::deque<Op>> g_streams;  // stream id -> operations in enqueue order
std::map<void*, long> g_word_of;           // signal memory -> word index
std::vector<uint32_t> g_enqueued_max;      // per word: largest value of a write enqueued so far
std::vector<uint32_t> g_mem;               // per word: the model's current value
std::map<void*, long> g_last_record;       // event -> number of its latest record enqueued
std::vector<bool> g_record_done;           // record number -> executed
long g_words = 0;
int g_failures = 0;
long g_ops = 0;

long sid(hipStream_t s) { return reinterpret_cast<long>(s); }

void push(hipStream_t s, Op op) {
  g_streams[sid(s)].push_back(op);
  ++g_ops;
}

void fail(const char* msg) {
  std::printf("FAIL: %s\n", msg);
  std::exit(1);
}

// Runs every queued operation through the device model; fails on a deadlock.
void drain() {
  for (;;) {
    bool progress = false, left = false;
    for (auto& kv : g_streams) {
      auto& q = kv.second;
      while (!q.empty()) {
        Op& op = q.front();
        if (op.kind == kWait && g_mem[op.word] < op.value) break;
        if (op.kind == kWaitEvent && op.word >= 0 && !g_record_done[op.word]) break;
        if (op.kind == kRecord) g_record_done[op.word] = true;
        if (op.kind == kWrite) {
          if (op.value < g_mem[op.word]) {
            std::printf("stream %ld word %ld: %u -> %u\n", kv.first, op.word, g_mem[op.word], op.value);
            fail("a signal word went down");
          }
          g_mem[op.word] = op.value;
        }
        q.pop_front();
        progress = true;
      }
      left |= !q.empty();
    }
    if (!left) return;
    if (!progress) {
      for (auto& kv : g_streams)
        if (!kv.second.empty())
          std::printf("stream %ld blocked at wait word %ld >= %u (word holds %u)\n", kv.first, kv.second.front().word,
                      kv.second.front().value, g_mem[kv.second.front().word]);
      fail("deadlock");
    }
  }
}

}  // namespace

// ---- stand-ins for the HIP runtime calls the executor makes
extern "C" {
hipError_t hipStreamWriteValue32(hipStream_t stream, void* ptr, uint32_t value, unsigned int) {
  const long w = g_word_of.at(ptr);
  if (value > g_enqueued_max[w]) g_enqueued_max[w] = value;
  push(stream, Op{kWrite, w, value, "write"});
  return hipSuccess;
}
hipError_t hipStreamWaitValue32(hipStream_t stream, void* ptr, uint32_t value, unsigned int flags, uint32_t mask) {
  if (flags != hipStreamWaitValueGte || mask != 0xFFFFFFFFu) fail("unexpected wait form");
  const long w = g_word_of.at(ptr);
  if (value > g_enqueued_max[w]) fail("a wait targets a value no enqueued write supplies");
  push(stream, Op{kWait, w, value, "wait"});
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t event, hipStream_t stream) {
  const long n = static_cast<long>(g_record_done.size());
  g_record_done.push_back(false);
  g_last_record[event] = n;
  push(stream, Op{kRecord, n, 0, "record"});
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t stream, hipEvent_t event, unsigned int) {
  // HIP semantics: wait for the event's latest record at the time of the call (none: no wait)
  auto it = g_last_record.find(event);
  push(stream, Op{kWaitEvent, it == g_last_record.end() ? -1 : it->second, 0, "wait event"});
  return hipSuccess;
}
hipError_t hipExtMallocWithFlags(void** ptr, size_t, unsigned int flags) {
  if (flags != hipMallocSignalMemory) fail("unexpected allocation");
  *ptr = std::malloc(8);
  g_word_of[*ptr] = g_words++;
  g_enqueued_max.push_back(0);
  g_mem.push_back(0);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) {
  drain();
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 1;
  return hipSuccess;
}
}  // extern "C"

// ---- stand-ins for the launchers and calls the executor enqueues
namespace emb {
hipError_t launch_gather(const float*, int64_t, int, const int32_t*, int, float*, int32_t*, hipStream_t stream,
                         hipEvent_t done) {
  push(stream, Op{kLaunch, 0, 0, "gather"});
  if (done) fail("an attached event with signals");
  return hipSuccess;
}
hipError_t launch_coalesce_sort(const int32_t*, int, int64_t, int, const CoalesceVariant&, void*, int32_t*,
                                hipStream_t stream) {
  push(stream, Op{kLaunch, 0, 0, "sort"});
  return hipSuccess;
}
hipError_t launch_coalesce_reduce(const int32_t*, int, const void*, bool, int, int64_t, const CoalesceVariant&, int32_t*,
                                  int32_t*, float*, int32_t*, int32_t*, int32_t*, void*, int32_t*, hipStream_t stream,
                                  hipEvent_t done) {
  push(stream, Op{kLaunch, 0, 0, "reduce"});
  if (done) fail("an attached event with signals");
  return hipSuccess;
}
int coalesce_by_owner_args_status(const int32_t*, int32_t, const void*, int32_t, int32_t, int64_t, const int32_t*,
                                  int32_t, const int32_t*, int32_t, const int32_t*, const int32_t*, const float*,
                                  const int32_t*, const int32_t*, const int32_t*, const void*, size_t) {
  return EMB_OK;
}
int sparse_adam_call(float*, float*, float*, int64_t, int32_t, const int32_t*, const float*, const int32_t*, int32_t,
                     int32_t, int32_t, int32_t, double, double, double, double, int64_t, int32_t*, hipStream_t stream,
                     hipEvent_t, hipEvent_t stop) {
  push(stream, Op{kLaunch, 0, 0, "adam"});
  if (stop) hipEventRecord(stop, stream);  // an event attached to the dispatch completes with it
  return EMB_OK;
}
}  // namespace emb

extern "C" {
int emb_gather(const float*, int64_t, int32_t, const int32_t*, int32_t, float*, int32_t*, void* stream) {
  push(static_cast<hipStream_t>(stream), Op{kLaunch, 0, 0, "gather"});
  return EMB_OK;
}
int emb_grad_coalesce(const int32_t*, int32_t, const void*, int32_t, int32_t, int64_t, int32_t*, int32_t*, float*,
                      int32_t*, void* workspace, size_t, int32_t*, void* stream) {
  if (workspace == nullptr) return EMB_ERR_INVALID_ARG;
  push(static_cast<hipStream_t>(stream), Op{kLaunch, 0, 0, "coalesce"});
  return EMB_OK;
}
int emb_pack_by_owner(const int32_t*, const float*, const int32_t*, int32_t, int32_t, const int32_t*, int64_t, int32_t,
                      int32_t*, float*, int32_t*, int32_t*, void*, size_t workspace_bytes, int32_t*, void* stream) {
  if (workspace_bytes == 1) return EMB_ERR_WORKSPACE;  // the scenario's failure part-way
  push(static_cast<hipStream_t>(stream), Op{kLaunch, 0, 0, "pack"});
  return EMB_OK;
}
}  // extern "C"

namespace {

hipStream_t fake_stream(long i) { return reinterpret_cast<hipStream_t>(i); }

struct Table {
  void* signals = nullptr;
  emb_step_args args{};
  emb_step_schedule sched{};
};

void new_handle(Table& t) {
  if (emb_step_signals_create(&t.signals) != EMB_OK) fail("create");
  t.sched.signals = t.signals;
}

void drop_handle(Table& t) {
  drain();  // the steps of the handle have completed before it goes back
  if (emb_step_signals_destroy(t.signals) != EMB_OK) fail("destroy");
  t.signals = nullptr;
}

// mode 0: coalesce then pack; 1: owner-major; 2: owner-major with the split
int step(Table& t, int mode, bool fail_pack) {
  t.sched.by_owner = mode >= 1;
  t.sched.split = mode == 2;
  t.args.ws_pack_bytes = fail_pack ? 1 : 1 << 20;
  return emb_train_step(&t.args, &t.sched);
}

}  // namespace

int main() {
  static char dummy[256];
  Table tabs[2];
  for (auto& t : tabs) {
    t.args.T = 100;
    t.args.T_next = 100;
    t.args.cap_rows = 100;
    t.args.ws_coalesce = dummy;
    t.args.ws_pack = dummy;
    t.sched.lookup_update = fake_stream(1);
    t.sched.coalesce = fake_stream(2);
    t.sched.pack = fake_stream(3);
    t.sched.delayed = fake_stream(4);
    t.sched.updated = reinterpret_cast<void*>(&t);  // the update's end goes through this event
    new_handle(t);
  }
  // handles taken back from the pool by pipelines of other modes
  for (int mode : {0, 1, 2, 1, 0, 2, 2, 0}) {
    for (int s = 0; s < 7; ++s)
      for (auto& t : tabs)
        if (step(t, mode, false) != EMB_OK) fail("step");
    for (auto& t : tabs) drop_handle(t);
    for (auto& t : tabs) new_handle(t);
  }
  // a call that fails part-way (coalesce-then-pack: after the coalesce is enqueued)
  for (int s = 0; s < 9; ++s)
    for (auto& t : tabs) {
      const int st = step(t, 0, s == 3);
      if ((st != EMB_OK) != (s == 3)) fail("failure path");
    }
  // a long random mix of modes, failures and single-stream schedules
  unsigned x = 12345;
  auto rnd = [&x](unsigned n) {
    x = x * 1103515245u + 12345u;
    return (x >> 16) % n;
  };
  for (int s = 0; s < 3000; ++s) {
    Table& t = tabs[rnd(2)];
    const int mode = static_cast<int>(rnd(3));
    const bool fail_pack = mode == 0 && rnd(10) == 0;
    const bool one_stream = rnd(8) == 0;
    t.sched.sets = static_cast<int32_t>(rnd(5));  // 0 (two), 1 .. 4
    // sorts of odd steps on another stream, sometimes with their reductions (paired)
    if (rnd(2)) t.sched.coalesce = fake_stream(s % 2 ? 5 : 2);
    if (rnd(3) == 0) t.sched.pack = t.sched.coalesce;
    if (one_stream) t.sched.coalesce = t.sched.pack = t.sched.delayed = fake_stream(1);
    t.sched.reuse = rnd(2);
    t.sched.updated = rnd(4) == 0 ? nullptr : reinterpret_cast<void*>(&t);  // sometimes no event: a signal
    const int st = step(t, mode, fail_pack);
    if ((st != EMB_OK) != fail_pack) fail("random step");
    t.sched.coalesce = fake_stream(2);
    t.sched.pack = fake_stream(3);
    t.sched.delayed = fake_stream(4);
    if (rnd(50) == 0) {
      drop_handle(t);
      new_handle(t);
    }
  }
  drain();
  std::printf("ok: %ld operations, %ld signal words, no wait beyond the enqueued writes, no deadlock\n", g_ops,
              g_words);
  return 0;
}
