// Native consumer of the C ABI (include/emb.h), no Python and no torch: two
// training steps of one table on one stream, checked against the CPU oracle
// (oracle/oracle.h; test infrastructure, linked by tests only).
//   step 1: emb_gather, emb_grad_coalesce_by_owner, emb_sparse_adam_apply
//           (5000 tokens: the multi-kernel coalesce);
//   step 2: emb_train_step, owner-major, every stage on the one stream
//           (1500 tokens: the one-workgroup coalesce).
// Checks per step: the lookup bit-exact against the oracle's gather of the
// table as it was before the step; send ids, counts and offsets bit-exact
// against the oracle's coalesce and pack; each sent row within 1e-5 of the
// sum of magnitudes of its tokens' gradients (the fp32 summation bound);
// the update against the oracle's Adam on the same inputs (the GPU's send
// layout and pre-step state): W, m, v within 1e-5 of each row's max-norm, the
// change of W within 1e-5 of the row's largest change plus one unit in the
// last place, and rows not sent bit-identical.  Exit status 0 when all hold.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "emb.h"
#include "oracle.h"

namespace {

constexpr int64_t kV = 50000;
constexpr int32_t kD = 64;
constexpr int32_t kP = 4;
constexpr int32_t kT1 = 5000, kT2 = 1500, kCap = 5000;
constexpr double kLr = 1e-3, kB1 = 0.9, kB2 = 0.999, kEps = 1e-8;

int g_fail = 0;
#define CHECK(cond, ...)                 \
  do {                                   \
    if (!(cond)) {                       \
      std::printf("FAIL: " __VA_ARGS__); \
      std::printf("\n");                 \
      g_fail = 1;                        \
      return false;                      \
    }                                    \
  } while (0)
#define HIP_OK(call)                                                          \
  do {                                                                        \
    hipError_t e_ = (call);                                                   \
    if (e_ != hipSuccess) {                                                   \
      std::printf("FAIL: %s: %s\n", #call, hipGetErrorString(e_));            \
      std::exit(2);                                                           \
    }                                                                         \
  } while (0)
#define EMB_OK_(call)                                                         \
  do {                                                                        \
    int s_ = (call);                                                          \
    if (s_ != EMB_OK) {                                                       \
      std::printf("FAIL: %s: %s\n", #call, emb_status_string(s_));            \
      std::exit(3);                                                           \
    }                                                                         \
  } while (0)

// Seeded synthetic inputs (a counter-based hash; no part of the method).
uint64_t mix(uint64_t z) {
  z += 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
double unit(uint64_t key, uint64_t i) { return static_cast<double>(mix(key * 0x100000001b3ull + i) >> 11) * 0x1p-53; }
std::vector<int32_t> make_ids(uint64_t key, int32_t T) {  // skewed: id = V u^3
  std::vector<int32_t> ids(T);
  for (int32_t t = 0; t < T; ++t) {
    const double u = unit(key, t);
    ids[t] = std::min<int32_t>(static_cast<int32_t>(kV * u * u * u), kV - 1);
  }
  return ids;
}
std::vector<float> make_vals(uint64_t key, size_t n, double scale) {
  std::vector<float> v(n);
  for (size_t i = 0; i < n; ++i) v[i] = static_cast<float>(scale * (2.0 * unit(key, i) - 1.0));
  return v;
}

template <class T>
T* dev_alloc(size_t n) {
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, std::max<size_t>(n, 1) * sizeof(T)));
  return static_cast<T*>(p);
}
template <class T>
void to_dev(T* d, const std::vector<T>& h) {
  HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
}
template <class T>
std::vector<T> to_host(const T* d, size_t n) {
  std::vector<T> h(n);
  HIP_OK(hipMemcpy(h.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
  return h;
}

struct Dev {
  float *W, *M, *S, *grad, *lookup, *uniq_grad, *send_rows;
  int32_t *ids, *owner, *uniq_ids, *seg, *nu, *send_ids, *counts, *offs, *status;
  void *ws, *ws_pack;
  size_t ws_bytes, ws_pack_bytes;
};

struct State {  // host copies of the table and moments
  std::vector<float> W, M, S;
};
State read_state(const Dev& d) {
  const size_t n = static_cast<size_t>(kV) * kD;
  return State{to_host(d.W, n), to_host(d.M, n), to_host(d.S, n)};
}

float ulp(float x) {
  const float a = std::fabs(x);
  return std::nextafter(a, INFINITY) - a;
}

bool check_step(int step, const std::vector<int32_t>& ids, const std::vector<float>& G, const State& before,
                const Dev& d, const std::vector<int32_t>& owner) {
  const int32_t T = static_cast<int32_t>(ids.size());
  HIP_OK(hipDeviceSynchronize());
  CHECK(to_host(d.status, 1)[0] == 0, "step %d: device status %d", step, to_host(d.status, 1)[0]);
  // lookup
  std::vector<float> want(static_cast<size_t>(T) * kD);
  orc_gather(before.W.data(), kV, kD, ids.data(), T, want.data());
  const std::vector<float> got = to_host(d.lookup, want.size());
  CHECK(std::memcmp(got.data(), want.data(), want.size() * sizeof(float)) == 0, "step %d: lookup differs", step);
  // coalesce + pack
  std::vector<int32_t> uid(T), seg(T + 1);
  std::vector<float> ug(static_cast<size_t>(T) * kD);
  std::vector<double> sum(ug.size()), absum(ug.size());
  const int64_t U = orc_coalesce(ids.data(), T, G.data(), 0, kD, kV, uid.data(), seg.data(), ug.data(), sum.data(),
                                 absum.data(), nullptr);
  std::vector<int32_t> sid(U), cnt(kP), off(kP + 1);
  std::vector<float> srows(static_cast<size_t>(U) * kD);
  orc_pack_by_owner(uid.data(), ug.data(), U, kD, owner.data(), kV, kP, sid.data(), srows.data(), cnt.data(),
                    off.data());
  CHECK(to_host(d.nu, 1)[0] == U, "step %d: %d distinct ids, the oracle has %lld", step, to_host(d.nu, 1)[0],
        static_cast<long long>(U));
  const std::vector<int32_t> g_sid = to_host(d.send_ids, U), g_cnt = to_host(d.counts, kP),
                             g_off = to_host(d.offs, kP + 1);
  CHECK(g_sid == sid && g_cnt == cnt && g_off == off, "step %d: send ids, counts or offsets differ", step);
  const std::vector<float> g_rows = to_host(d.send_rows, static_cast<size_t>(U) * kD);
  for (int64_t r = 0; r < U; ++r) {
    const int64_t k = std::lower_bound(uid.begin(), uid.begin() + U, sid[r]) - uid.begin();
    for (int32_t j = 0; j < kD; ++j) {
      const double err = std::fabs(static_cast<double>(g_rows[r * kD + j]) - sum[k * kD + j]);
      CHECK(err <= 1e-5 * absum[k * kD + j], "step %d: row %lld col %d: error %.3e, bound %.3e", step,
            static_cast<long long>(r), j, err, 1e-5 * absum[k * kD + j]);
    }
  }
  // update, on the GPU's own send layout and pre-step state
  State orc = before;
  orc_sparse_adam(orc.W.data(), orc.M.data(), orc.S.data(), kV, kD, g_sid.data(), g_rows.data(), g_off.data(), 0, kP,
                  kLr, kB1, kB2, kEps, step);
  const State after = read_state(d);
  std::vector<char> sent(kV, 0);
  for (int32_t id : g_sid) sent[id] = 1;
  for (int64_t v = 0; v < kV; ++v) {
    const size_t o = static_cast<size_t>(v) * kD;
    if (!sent[v]) {
      CHECK(std::memcmp(&after.W[o], &before.W[o], kD * sizeof(float)) == 0 &&
                std::memcmp(&after.M[o], &before.M[o], kD * sizeof(float)) == 0 &&
                std::memcmp(&after.S[o], &before.S[o], kD * sizeof(float)) == 0,
            "step %d: row %lld was not sent but changed", step, static_cast<long long>(v));
      continue;
    }
    const std::vector<float>* gpu[3] = {&after.W, &after.M, &after.S};
    const std::vector<float>* ref[3] = {&orc.W, &orc.M, &orc.S};
    for (int a = 0; a < 3; ++a) {
      double num = 0, den = 0;
      for (int32_t j = 0; j < kD; ++j) {
        num = std::max(num, std::fabs(static_cast<double>((*gpu[a])[o + j]) - (*ref[a])[o + j]));
        den = std::max(den, std::fabs(static_cast<double>((*ref[a])[o + j])));
      }
      CHECK(num <= 1e-5 * den, "step %d: row %lld array %d: %.3e > 1e-5 * %.3e", step, static_cast<long long>(v), a,
            num, den);
    }
    double dmax = 0;
    for (int32_t j = 0; j < kD; ++j) dmax = std::max(dmax, std::fabs(static_cast<double>(orc.W[o + j]) - before.W[o + j]));
    for (int32_t j = 0; j < kD; ++j) {
      const double err = std::fabs(static_cast<double>(after.W[o + j]) - orc.W[o + j]);
      CHECK(err <= 1e-5 * dmax + ulp(orc.W[o + j]), "step %d: row %lld col %d: update error %.3e (row change %.3e)",
            step, static_cast<long long>(v), j, err, dmax);
    }
  }
  std::printf("step %d: %d tokens, %lld distinct ids: ok\n", step, T, static_cast<long long>(U));
  return true;
}

}  // namespace

int main() {
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
    std::printf("FAIL: no GPU\n");
    return 2;
  }
  HIP_OK(hipSetDevice(0));
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  const size_t nW = static_cast<size_t>(kV) * kD;
  std::vector<int32_t> owner(kV);
  for (int64_t v = 0; v < kV; ++v) owner[v] = static_cast<int32_t>(v % kP);
  Dev d{};
  d.W = dev_alloc<float>(nW);
  d.M = dev_alloc<float>(nW);
  d.S = dev_alloc<float>(nW);
  d.grad = dev_alloc<float>(static_cast<size_t>(kCap) * kD);
  d.lookup = dev_alloc<float>(static_cast<size_t>(kCap) * kD);
  d.uniq_grad = dev_alloc<float>(static_cast<size_t>(kCap) * kD);
  d.send_rows = dev_alloc<float>(static_cast<size_t>(kCap) * kD);
  d.ids = dev_alloc<int32_t>(kCap);
  d.owner = dev_alloc<int32_t>(kV);
  d.uniq_ids = dev_alloc<int32_t>(kCap);
  d.seg = dev_alloc<int32_t>(kCap + 1);
  d.nu = dev_alloc<int32_t>(1);
  d.send_ids = dev_alloc<int32_t>(kCap);
  d.counts = dev_alloc<int32_t>(kP);
  d.offs = dev_alloc<int32_t>(kP + 1);
  d.status = dev_alloc<int32_t>(1);
  d.ws_bytes = emb_grad_coalesce_workspace_bytes(kCap, kV, kD, EMB_F32);
  d.ws_pack_bytes = emb_pack_by_owner_workspace_bytes(kCap, kP);
  if (d.ws_bytes == 0 || d.ws_pack_bytes == 0) {
    std::printf("FAIL: workspace query\n");
    return 3;
  }
  d.ws = dev_alloc<unsigned char>(d.ws_bytes);
  d.ws_pack = dev_alloc<unsigned char>(d.ws_pack_bytes);
  to_dev(d.W, make_vals(11, nW, 1.0));
  HIP_OK(hipMemset(d.M, 0, nW * sizeof(float)));
  HIP_OK(hipMemset(d.S, 0, nW * sizeof(float)));
  HIP_OK(hipMemset(d.status, 0, sizeof(int32_t)));
  to_dev(d.owner, owner);

  // step 1: the calls one by one
  {
    const std::vector<int32_t> ids = make_ids(21, kT1);
    const std::vector<float> G = make_vals(31, static_cast<size_t>(kT1) * kD, 0.01);
    to_dev(d.ids, ids);
    to_dev(d.grad, G);
    const State before = read_state(d);
    EMB_OK_(emb_gather(d.W, kV, kD, d.ids, kT1, d.lookup, d.status, stream));
    EMB_OK_(emb_grad_coalesce_by_owner(d.ids, kT1, d.grad, EMB_F32, kD, kV, d.owner, kP, d.send_ids, d.seg,
                                       d.send_rows, d.counts, d.offs, d.nu, d.ws, d.ws_bytes, d.status, stream));
    EMB_OK_(emb_sparse_adam_apply(d.W, d.M, d.S, kV, kD, d.send_ids, d.send_rows, d.offs, kP, 0, kP, kCap, kLr, kB1,
                                  kB2, kEps, 1, d.status, stream));
    if (!check_step(1, ids, G, before, d, owner)) return 1;
  }
  // step 2: the step executor, owner-major, every stage on the one stream
  {
    const std::vector<int32_t> ids = make_ids(22, kT2);
    const std::vector<float> G = make_vals(32, static_cast<size_t>(kT2) * kD, 0.01);
    to_dev(d.ids, ids);
    to_dev(d.grad, G);
    const State before = read_state(d);
    void* ev[4] = {};
    for (auto& e : ev) EMB_OK_(emb_event_create(&e, 0));
    emb_step_schedule s{};
    s.lookup_update = s.coalesce = s.pack = s.delayed = stream;
    s.sorted = ev[0];
    s.coalesced = ev[1];
    s.packed = ev[2];
    s.updated = ev[3];
    s.by_owner = 1;
    s.sets = 2;
    emb_step_args a{};
    a.table = d.W;
    a.exp_avg = d.M;
    a.exp_avg_sq = d.S;
    a.V = kV;
    a.D = kD;
    a.row_owner = d.owner;
    a.P = kP;
    a.ids = d.ids;
    a.T = kT2;
    a.T_next = 0;
    a.grad = d.grad;
    a.grad_dtype = EMB_F32;
    a.cap_rows = kCap;
    a.lookup = d.lookup;
    a.uniq_ids = d.uniq_ids;
    a.seg_offsets = d.seg;
    a.num_unique = d.nu;
    a.uniq_grad = d.uniq_grad;
    a.send_ids = d.send_ids;
    a.send_counts = d.counts;
    a.send_offsets = d.offs;
    a.send_rows = d.send_rows;
    a.ws_coalesce = d.ws;
    a.ws_coalesce_bytes = d.ws_bytes;
    a.ws_pack = d.ws_pack;
    a.ws_pack_bytes = d.ws_pack_bytes;
    a.lr = kLr;
    a.beta1 = kB1;
    a.beta2 = kB2;
    a.eps = kEps;
    a.step = 2;
    a.dev_status = d.status;
    EMB_OK_(emb_train_step(&a, &s));
    const bool ok = check_step(2, ids, G, before, d, owner);
    for (auto& e : ev) EMB_OK_(emb_event_destroy(e));
    if (!ok) return 1;
  }
  HIP_OK(hipStreamDestroy(stream));
  std::printf("native driver: ok\n");
  return g_fail;
}
