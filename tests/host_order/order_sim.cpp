// Host-only check of the step executor's cross-stream order (step.hip), with step signals and with
// events.
//
// The executor is linked against stand-ins for the HIP stream operations and for the kernel
// launchers: every launch, event record or wait, and signal write or wait is appended to a trace,
// per stream, instead of reaching a GPU.  A model of the device then runs the trace: each stream
// runs its operations in order; a signal wait proceeds once its word holds at least its value; an
// event wait once the record it refers to has run.  Checks:
//  - no wait targets more than the writes enqueued before it can supply, no signal word goes down,
//    and the model never stops with work left (a deadlock);
//  - happens-before: the model keeps a vector clock per stream (a wait joins the clock of the write
//    or record it waited for), and every two launches that touch the same buffer (a set's coalesce
//    workspace, unique rows, send rows, pack workspace) or overlapping table rows, one of them
//    writing, must be ordered as the executor enqueued them.  Table rows follow the data of the
//    steps: the lookup of step n reads the rows of batch n, its update writes them; with the split,
//    the prior update writes the rows of batch n that batch n + 1 also holds and the delayed update
//    the others, which no operation on batch n + 1 touches.
// Scenarios: every mode (coalesce then pack, owner-major, owner-major with the split) with events,
// with signals and with events under graph capture (no event attached to a dispatch), two to six
// buffer sets, more steps than sets, and stream choices that include a set's streams
// changing between its uses; signal handles reused from the pool across modes; a call that fails
// part-way; and a long random mix of modes (deadlock freedom only).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <deque>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "emb.h"
#include "launch.h"

namespace {

enum Kind { kLaunch, kWrite, kWait, kRecord, kWaitEvent };
enum RowSet { kNoRows, kAllRows, kPriorRows, kDelayedRows };  // table rows of the op's batch

struct Access {
  const void* buf;  // a buffer, or the table
  bool write;
};

struct Op {
  Kind kind;
  long word;        // signal word index; for events: the record's number (a wait: the record it waits for, or -1)
  uint32_t value;   // written / waited-for value
  std::string what;
  std::vector<Access> acc;  // launches: the buffers they touch
  long step = -1;           // launches: the step of the batch (for table rows)
  RowSet rows = kNoRows;    // launches on the table: which rows of that batch
  const void* table = nullptr;
  long seq = 0;             // launches: enqueue order
};

using Clock = std::map<long, long>;  // stream -> count

struct Executed {
  Op op;
  long stream;
  Clock clock;
};

std::map<long, std::deque<Op>> g_streams;  // stream id -> operations in enqueue order
std::map<void*, long> g_word_of;           // signal memory -> word index
std::vector<uint32_t> g_enqueued_max;      // per word: largest value of a write enqueued so far
std::vector<uint32_t> g_mem;               // per word: the model's current value
std::vector<std::vector<std::pair<uint32_t, Clock>>> g_writes;  // per word: executed writes (value, clock)
std::map<void*, long> g_last_record;       // event -> number of its latest record enqueued
std::vector<bool> g_record_done;           // record number -> executed
std::vector<Clock> g_record_clock;         // record number -> clock when it ran
std::map<long, Clock> g_clock;             // stream -> its clock
std::vector<Executed> g_launches;          // launches in execution order (for the happens-before check)
long g_words = 0;
long g_ops = 0;
long g_seq = 0;
bool g_track = false;  // record launches for the happens-before check

// What the next launches touch (set by the stand-ins from their arguments).
long g_cur_step = 0;                      // step number of the call being enqueued
// Two-thread enqueue: the worker enqueues a step's main half after the caller has moved on, so the
// step of a launch is read from its arguments instead (ids = kIdsBase + 16 * step, Adam step = step + 1).
bool g_step_from_args = false;
constexpr uintptr_t kIdsBase = 0x100000;
std::recursive_mutex g_sim_mu;  // the stand-ins are called from two host threads
long step_of_ids(const int32_t* ids) {
  return g_step_from_args ? static_cast<long>((reinterpret_cast<uintptr_t>(ids) - kIdsBase) / 16) : g_cur_step;
}
std::map<const void*, bool> g_is_table;   // table pointers

long sid(hipStream_t s) { return reinterpret_cast<long>(s); }

void push(hipStream_t s, Op op) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  if (op.kind == kLaunch) op.seq = g_seq++;
  g_streams[sid(s)].push_back(op);
  ++g_ops;
}

void fail(const char* msg) {
  std::printf("FAIL: %s\n", msg);
  std::exit(1);
}

void join(Clock& a, const Clock& b) {
  for (auto& kv : b) a[kv.first] = std::max(a[kv.first], kv.second);
}

// Runs every queued operation through the device model; fails on a deadlock.
void drain() {
  for (;;) {
    bool progress = false, left = false;
    for (auto& kv : g_streams) {
      auto& q = kv.second;
      Clock& clk = g_clock[kv.first];
      while (!q.empty()) {
        Op& op = q.front();
        if (op.kind == kWait && g_mem[op.word] < op.value) break;
        if (op.kind == kWaitEvent && op.word >= 0 && !g_record_done[op.word]) break;
        clk[kv.first] += 1;
        if (op.kind == kWait) {  // ordered after the first write that supplied the value
          for (auto& w : g_writes[op.word])
            if (w.first >= op.value) {
              join(clk, w.second);
              break;
            }
        }
        if (op.kind == kWaitEvent && op.word >= 0) join(clk, g_record_clock[op.word]);
        if (op.kind == kRecord) {
          g_record_done[op.word] = true;
          g_record_clock[op.word] = clk;
        }
        if (op.kind == kWrite) {
          if (op.value < g_mem[op.word]) {
            std::printf("stream %ld word %ld: %u -> %u\n", kv.first, op.word, g_mem[op.word], op.value);
            fail("a signal word went down");
          }
          g_mem[op.word] = op.value;
          g_writes[op.word].push_back({op.value, clk});
        }
        if (op.kind == kLaunch && g_track && (!op.acc.empty() || op.rows != kNoRows))
          g_launches.push_back(Executed{op, kv.first, clk});
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

// The sets of table rows two launches touch can overlap, unless one is the delayed part of batch m
// and the other touches only rows of batch m + 1 (the delayed rows are those batch m + 1 lacks).
bool rows_overlap(const Op& a, const Op& b) {
  if (a.rows == kNoRows || b.rows == kNoRows || a.table != b.table) return false;
  if (a.rows == kDelayedRows && b.step == a.step + 1) return false;
  if (b.rows == kDelayedRows && a.step == b.step + 1) return false;
  if (a.step == b.step && ((a.rows == kDelayedRows && b.rows == kPriorRows) ||
                           (a.rows == kPriorRows && b.rows == kDelayedRows)))
    return false;
  return true;
}

bool table_write(const Op& o) { return o.what == "adam"; }

// Every two conflicting launches must be ordered as they were enqueued.
void check_happens_before(const char* scenario) {
  drain();
  for (size_t i = 0; i < g_launches.size(); ++i)
    for (size_t j = 0; j < g_launches.size(); ++j) {
      const Executed& a = g_launches[i];
      const Executed& b = g_launches[j];
      if (a.op.seq >= b.op.seq) continue;
      bool conflict = false;
      for (auto& x : a.op.acc)
        for (auto& y : b.op.acc)
          if (x.buf == y.buf && (x.write || y.write)) conflict = true;
      if (rows_overlap(a.op, b.op) && (table_write(a.op) || table_write(b.op))) conflict = true;
      if (!conflict) continue;
      auto it = b.clock.find(a.stream);
      const long seen = it == b.clock.end() ? 0 : it->second;
      if (seen < a.clock.at(a.stream)) {
        std::printf("%s: %s of step %ld rows %d (stream %ld) is not ordered before %s of step %ld rows %d (stream %ld)\n", scenario,
                    a.op.what.c_str(), a.op.step, (int)a.op.rows, a.stream, b.op.what.c_str(), b.op.step, (int)b.op.rows, b.stream);
        fail("a conflicting pair runs unordered");
      }
    }
  g_launches.clear();
}

Op launch_op(const char* what, std::vector<Access> acc, RowSet rows = kNoRows, const void* table = nullptr,
             long step = -1) {
  Op o{kLaunch, 0, 0, what, std::move(acc)};
  o.step = step >= 0 ? step : g_cur_step;
  o.rows = rows;
  o.table = table;
  return o;
}

}  // namespace

// ---- stand-ins for the HIP runtime calls the executor makes
extern "C" {
hipError_t hipStreamWriteValue32(hipStream_t stream, void* ptr, uint32_t value, unsigned int) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  const long w = g_word_of.at(ptr);
  if (value > g_enqueued_max[w]) g_enqueued_max[w] = value;
  push(stream, Op{kWrite, w, value, "write"});
  return hipSuccess;
}
hipError_t hipStreamWaitValue32(hipStream_t stream, void* ptr, uint32_t value, unsigned int flags, uint32_t mask) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  if (flags != hipStreamWaitValueGte || mask != 0xFFFFFFFFu) fail("unexpected wait form");
  const long w = g_word_of.at(ptr);
  if (value > g_enqueued_max[w]) fail("a wait targets a value no enqueued write supplies");
  push(stream, Op{kWait, w, value, "wait"});
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t event, hipStream_t stream) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  const long n = static_cast<long>(g_record_done.size());
  g_record_done.push_back(false);
  g_record_clock.push_back(Clock{});
  g_last_record[event] = n;
  push(stream, Op{kRecord, n, 0, "record"});
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t stream, hipEvent_t event, unsigned int) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  if (event == nullptr) fail("a wait on a null event");
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
  g_writes.emplace_back();
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) {
  drain();
  return hipSuccess;
}
bool g_capturing = false;  // the streams are being captured into a graph
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* st) {
  *st = g_capturing ? hipStreamCaptureStatusActive : hipStreamCaptureStatusNone;
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 1;
  return hipSuccess;
}
}  // extern "C"

// ---- stand-ins for the launchers and calls the executor enqueues
namespace emb {
hipError_t launch_gather(const float* table, int64_t, int, const int32_t* ids, int, float*, int32_t*,
                         hipStream_t stream, hipEvent_t done) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  push(stream, launch_op("gather", {}, kAllRows, table, step_of_ids(ids)));
  if (done && g_capturing) fail("an event attached to a dispatch under capture");
  if (done) (void)hipEventRecord(done, stream);  // an event attached to the dispatch completes with it
  return hipSuccess;
}
hipError_t launch_coalesce_sort(const int32_t* ids, int, int64_t, int, const CoalesceVariant&, void* ws, int32_t*,
                                hipStream_t stream) {
  push(stream, launch_op("sort", {{ws, true}}, kNoRows, nullptr, step_of_ids(ids)));
  return hipSuccess;
}
hipError_t launch_coalesce_reduce(const int32_t* ids, int, const void*, bool, int, int64_t, const CoalesceVariant&,
                                  int32_t* send_ids, int32_t*, float*, int32_t*, int32_t*, int32_t*, void* ws,
                                  int32_t*, hipStream_t stream, hipEvent_t done) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  push(stream, launch_op("reduce", {{ws, false}, {send_ids, true}}, kNoRows, nullptr, step_of_ids(ids)));
  if (done && g_capturing) fail("an event attached to a dispatch under capture");
  if (done) (void)hipEventRecord(done, stream);
  return hipSuccess;
}
int coalesce_by_owner_args_status(const int32_t*, int32_t, const void*, int32_t, int32_t, int64_t, const int32_t*,
                                  int32_t, const int32_t*, int32_t, const int32_t*, const int32_t*, const float*,
                                  const int32_t*, const int32_t*, const int32_t*, const void*, size_t) {
  return EMB_OK;
}
int sparse_adam_call(float* table, float*, float*, int64_t, int32_t, const int32_t* send_ids, const float*,
                     const int32_t* offsets, int32_t P, int32_t, int32_t, int32_t, double, double, double, double,
                     int64_t adam_step, const void*, int32_t*, hipStream_t stream, hipEvent_t, hipEvent_t stop) {
  std::lock_guard<std::recursive_mutex> lock(g_sim_mu);
  // the split's two parts: groups [0, P) prior, [P, 2P) delayed (offsets is send_offsets + P)
  extern const int32_t* g_offsets_base;
  RowSet rows = kAllRows;
  if (g_offsets_base != nullptr) rows = offsets == g_offsets_base ? kPriorRows : kDelayedRows;
  push(stream, launch_op("adam", {{send_ids, false}}, rows, table, g_step_from_args ? adam_step - 1 : -1));
  (void)P;
  if (stop && g_capturing) fail("an event attached to a dispatch under capture");
  if (stop) (void)hipEventRecord(stop, stream);
  return EMB_OK;
}
const int32_t* g_offsets_base = nullptr;  // the split's send_offsets while a split step is enqueued
}  // namespace emb

extern "C" {
int emb_gather(const float* table, int64_t, int32_t, const int32_t* ids, int32_t, float*, int32_t*, void* stream) {
  push(static_cast<hipStream_t>(stream), launch_op("gather", {}, kAllRows, table, step_of_ids(ids)));
  return EMB_OK;
}
int emb_grad_coalesce(const int32_t*, int32_t, const void*, int32_t, int32_t, int64_t, int32_t* uniq_ids, int32_t*,
                      float*, int32_t*, void* workspace, size_t, int32_t*, void* stream) {
  if (workspace == nullptr) return EMB_ERR_INVALID_ARG;
  push(static_cast<hipStream_t>(stream), launch_op("coalesce", {{workspace, true}, {uniq_ids, true}}));
  return EMB_OK;
}
int emb_pack_by_owner(const int32_t* uniq_ids, const float*, const int32_t*, int32_t, int32_t, const int32_t*, int64_t,
                      int32_t, int32_t* send_ids, float*, int32_t*, int32_t*, void* ws_pack, size_t workspace_bytes,
                      int32_t*, void* stream) {
  if (workspace_bytes == 1) return EMB_ERR_WORKSPACE;  // the scenario's failure part-way
  push(static_cast<hipStream_t>(stream),
       launch_op("pack", {{uniq_ids, false}, {send_ids, true}, {ws_pack, true}}));
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
  emb::g_offsets_base = mode == 2 ? t.args.send_offsets : nullptr;
  const int st = emb_train_step(&t.args, &t.sched);
  emb::g_offsets_base = nullptr;
  return st;
}

// ---- the happens-before scenarios: per-set buffers and events, fixed modes
struct SetBuffers {
  char ws[256], ws_pack[256];
  int32_t uniq_ids[4], send_ids[4], send_offsets[8];
  char ev[6];  // six distinct event handles (addresses)
};

// Streams of step n (buffer set k = n mod sets) under stream rule r.
void streams_for(int r, long n, int k, unsigned& rnd_state, emb_step_schedule& s) {
  auto rnd = [&rnd_state](unsigned m) {
    rnd_state = rnd_state * 1103515245u + 12345u;
    return (rnd_state >> 16) % m;
  };
  s.lookup_update = fake_stream(1);  // the lookup of a step follows the previous update on this stream
  s.coalesce = fake_stream(2);
  s.pack = fake_stream(3);
  s.delayed = fake_stream(4);
  switch (r) {
    case 0: break;                                                  // one stream per role
    case 1: s.coalesce = fake_stream(k % 2 ? 5 : 2); break;         // two sort streams, by set
    case 2: s.coalesce = s.pack = fake_stream(k % 2 ? 5 : 2); break;  // paired, by set
    case 3: s.coalesce = s.pack = fake_stream(n % 2 ? 5 : 2); break;  // paired, by step parity (odd sets: a
                                                                    // set's streams change between uses)
    case 4: s.coalesce = s.pack = s.delayed = fake_stream(1); break;  // one stream
    case 5: s.pack = fake_stream(1); break;                         // reduction beside the update
    default:                                                        // anything, per step
      s.coalesce = fake_stream(1 + static_cast<long>(rnd(5)));
      s.pack = fake_stream(1 + static_cast<long>(rnd(5)));
      s.delayed = fake_stream(1 + static_cast<long>(rnd(5)));
      break;
  }
}

void happens_before_scenarios() {
  static char table_mem[64];
  int scenarios = 0;
  // order 0: events; 1: step signals; 2: events under graph capture (no event attached to a dispatch:
  // every stage's end is an event record of its own)
  for (int order = 0; order < 3; ++order)
    for (int mode = 0; mode < 3; ++mode)
      for (int sets = 2; sets <= 6; ++sets) {
        const bool signals = order == 1;
        if (!signals && mode == 2 && sets != 2) continue;  // with events the split takes two sets
        g_capturing = order == 2;
        for (int r = 0; r < 7; ++r) {
          drain();
          g_clock.clear();
          g_launches.clear();
          g_track = true;
          std::vector<SetBuffers> bufs(sets);
          Table t;
          t.args.T = 100;
          t.args.T_next = 100;
          t.args.cap_rows = 100;
          t.args.table = reinterpret_cast<float*>(table_mem);
          t.args.P = 4;
          t.sched.sets = sets;
          if (signals) new_handle(t);
          unsigned rs = 777u + static_cast<unsigned>(r * 31 + sets);
          for (long n = 0; n < 16; ++n) {
            const int k = static_cast<int>(n % sets);
            SetBuffers& b = bufs[k];
            t.args.ws_coalesce = b.ws;
            t.args.ws_coalesce_bytes = sizeof b.ws;
            t.args.ws_pack = b.ws_pack;
            t.args.uniq_ids = b.uniq_ids;
            t.args.send_ids = b.send_ids;
            t.args.send_offsets = b.send_offsets;
            if (!signals) {
              t.sched.signals = nullptr;
              t.sched.sorted = &b.ev[0];
              t.sched.coalesced = &b.ev[1];
              t.sched.packed = &b.ev[2];
              t.sched.updated = &b.ev[3];
              t.sched.gathered = &b.ev[4];
              t.sched.delayed_done = &b.ev[5];
              t.sched.reuse = n >= sets;
            }
            streams_for(r, n, k, rs, t.sched);
            g_cur_step = n;
            if (step(t, mode, false) != EMB_OK) fail("happens-before step");
          }
          char name[96];
          std::snprintf(name, sizeof name, "%s, mode %d, %d sets, streams rule %d",
                        order == 0 ? "events" : order == 1 ? "signals" : "events under capture", mode, sets, r);
          check_happens_before(name);
          g_track = false;
          if (signals) drop_handle(t);
          ++scenarios;
        }
        g_capturing = false;
      }
  std::printf("happens-before: %d scenarios ordered\n", scenarios);
}

// The two-thread enqueue (emb_train_step_queued): the worker thread enqueues each step's lookup and
// update while this thread goes on with the next steps' sorts and reductions.  Each scenario runs
// several times, so that the two threads meet in different interleavings.
void queued_scenarios() {
  static char table_mem[64];
  int scenarios = 0;
  g_step_from_args = true;
  for (int sets = 2; sets <= 6; ++sets)
    for (int r = 0; r < 4; ++r)  // stream rules with the sort and the reduction off the main stream
      for (int rep = 0; rep < 5; ++rep) {
        drain();
        g_clock.clear();
        g_launches.clear();
        g_track = true;
        std::vector<SetBuffers> bufs(sets);
        Table t;
        t.args.T = 100;
        t.args.cap_rows = 100;
        t.args.table = reinterpret_cast<float*>(table_mem);
        t.args.P = 4;
        t.sched.sets = sets;
        t.sched.by_owner = 1;
        t.sched.split = 0;
        t.sched.signals = nullptr;
        void* q = nullptr;
        if (emb_step_queue_create(&q) != EMB_OK) fail("queue create");
        unsigned rs = 901u + static_cast<unsigned>(r * 31 + sets);
        for (long n = 0; n < 24; ++n) {
          const int k = static_cast<int>(n % sets);
          SetBuffers& b = bufs[k];
          t.args.ws_coalesce = b.ws;
          t.args.ws_coalesce_bytes = sizeof b.ws;
          t.args.send_ids = b.send_ids;
          t.args.send_offsets = b.send_offsets;
          t.args.ids = reinterpret_cast<const int32_t*>(kIdsBase + 16 * static_cast<uintptr_t>(n));
          t.args.step = n + 1;
          t.sched.sorted = &b.ev[0];
          t.sched.coalesced = &b.ev[1];
          t.sched.updated = &b.ev[3];
          t.sched.reuse = n >= sets;
          streams_for(r, n, k, rs, t.sched);
          if (emb_train_step_queued(q, &t.args, &t.sched) != EMB_OK) fail("queued step");
        }
        if (emb_step_queue_flush(q) != EMB_OK) fail("queue flush");
        if (emb_step_queue_destroy(q) != EMB_OK) fail("queue destroy");
        char name[96];
        std::snprintf(name, sizeof name, "queued, %d sets, streams rule %d, run %d", sets, r, rep);
        check_happens_before(name);
        g_track = false;
        ++scenarios;
      }
  // a schedule with the reduction on the main stream is refused
  {
    void* q = nullptr;
    if (emb_step_queue_create(&q) != EMB_OK) fail("queue create");
    Table t;
    static char ws[256];
    static int32_t ids_dummy[4], offs_dummy[8];
    static char ev[6];
    t.args.T = 4;
    t.args.cap_rows = 4;
    t.args.ws_coalesce = ws;
    t.args.send_ids = ids_dummy;
    t.args.send_offsets = offs_dummy;
    t.sched.by_owner = 1;
    t.sched.sorted = &ev[0];
    t.sched.coalesced = &ev[1];
    t.sched.updated = &ev[3];
    t.sched.lookup_update = fake_stream(1);
    t.sched.coalesce = fake_stream(2);
    t.sched.pack = fake_stream(1);
    if (emb_train_step_queued(q, &t.args, &t.sched) != EMB_ERR_UNSUPPORTED) fail("queued step on the main stream");
    if (emb_step_queue_destroy(q) != EMB_OK) fail("queue destroy");
  }
  g_step_from_args = false;
  std::printf("queued: %d scenarios ordered\n", scenarios);
}

}  // namespace

int main() {
  happens_before_scenarios();
  queued_scenarios();
  static char dummy[256];
  static int32_t ids_dummy[4], offs_dummy[8];
  Table tabs[2];
  for (auto& t : tabs) {
    t.args.T = 100;
    t.args.T_next = 100;
    t.args.cap_rows = 100;
    t.args.ws_coalesce = dummy;
    t.args.ws_pack = dummy;
    t.args.send_ids = ids_dummy;
    t.args.send_offsets = offs_dummy;
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
