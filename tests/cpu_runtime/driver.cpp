// Scenarios for the CPU build of the runtime (host stand-ins for HIP and the kernels),
// run under AddressSanitizer and under ThreadSanitizer by tests/test_runtime_sanitizers.py:
//   1. the session state machine of Sec. 3.6 and Alg. 1 (budget skip, pre-position,
//      every mutation invalidating the handle, restore);
//   2. Alg. 2's gate while the pre-position's device work is still pending (falls through
//      as INVALID, never blocks), then served once it has finished;
//   3. the idle-window pass of Sec. 3.1 yielding to a flag set by another thread;
//   4. gates of several sessions from several threads while another thread pre-positions,
//      mutates and destroys sessions (the registry keeps a gated session alive);
//   5. the batched pre-position and gate, and the gate entry point that allocates nothing.
// Prints "OK" and exits 0 when every check holds.
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include <hip/hip_runtime.h>

#include "spp.h"

namespace {

int g_fail = 0;
#define CHECK(c)                                                                  \
  do {                                                                            \
    if (!(c)) {                                                                   \
      std::fprintf(stderr, "%s:%d: check failed: %s (%s)\n", __FILE__, __LINE__, #c, \
                   spp_last_error());                                             \
      ++g_fail;                                                                   \
    }                                                                             \
  } while (0)

constexpr int kLayers = 4, kD = 256, kNq = 4, kNkv = 2, kDh = 64, kF = 512, kV = 2048;

struct Weights {
  std::vector<void*> bufs;
  std::vector<const void*> per[9];
  spp_weights w{};
  void* dev(size_t n) {
    void* p = nullptr;
    hipMalloc(&p, n);
    bufs.push_back(p);
    return p;
  }
  Weights() {
    w.embed = dev((size_t)kV * kD * 2);
    w.final_norm = dev(kD * 2);
    w.lm_head = dev((size_t)kV * kD * 2);
    w.lm_bias = nullptr;
    const size_t sz[9] = {(size_t)kD * 2,           (size_t)kNq * kDh * kD * 2,
                          (size_t)kNkv * kDh * kD * 2, (size_t)kNkv * kDh * kD * 2,
                          (size_t)kD * kNq * kDh * 2, (size_t)kD * 2,
                          (size_t)kF * kD * 2,         (size_t)kF * kD * 2,
                          (size_t)kD * kF * 2};
    for (int k = 0; k < 9; ++k)
      for (int l = 0; l < kLayers; ++l) per[k].push_back(dev(sz[k]));
    w.attn_norm = per[0].data();
    w.wq = per[1].data();
    w.wk = per[2].data();
    w.wv = per[3].data();
    w.wo = per[4].data();
    w.mlp_norm = per[5].data();
    w.w_gate = per[6].data();
    w.w_up = per[7].data();
    w.w_down = per[8].data();
  }
  ~Weights() {
    for (void* p : bufs) hipFree(p);
  }
};

spp_model_config config(int max_sessions) {
  spp_model_config c{};
  c.n_layers = kLayers;
  c.d_model = kD;
  c.n_q_heads = kNq;
  c.n_kv_heads = kNkv;
  c.head_dim = kDh;
  c.ffn_dim = kF;
  c.vocab = kV;
  c.rms_eps = 1e-5f;
  c.rope_base = 1e4;
  c.dtype = SPP_DTYPE_BF16;
  c.max_tokens = 64;
  c.max_sessions = max_sessions;
  c.weights_packed = 1;
  c.weight_format = SPP_WFMT_DTYPE;
  return c;
}

struct Sess {
  spp_session_t h = nullptr;
  void* kv = nullptr;
  float* dist = nullptr;
  Sess(spp_model_t m, int capacity, int budget) {
    spp_session_config sc{capacity, budget};
    const size_t kvb = spp_session_kv_bytes(m, capacity);
    hipMalloc(&kv, kvb);
    hipMalloc((void**)&dist, kV * 4);
    CHECK(spp_session_create(m, &sc, kv, kvb, &h) == SPP_OK);
  }
  void destroy() {
    if (h) CHECK(spp_session_destroy(h) == SPP_OK);
    h = nullptr;
  }
  ~Sess() {
    destroy();
    hipFree(kv);
    hipFree(dist);
  }
};

std::vector<int32_t> tokens(int n, int seed) {
  std::vector<int32_t> t(n);
  for (int i = 0; i < n; ++i) t[i] = (seed * 131 + i * 17) % kV;
  return t;
}

// a device bitmap holding the given tokens
uint32_t* bitmap(std::vector<void*>& keep, std::initializer_list<int> ids) {
  std::vector<uint32_t> h((kV + 31) / 32, 0u);
  for (int t : ids) h[t >> 5] |= 1u << (t & 31);
  void* d = nullptr;
  hipMalloc(&d, h.size() * 4);
  hipMemcpy(d, h.data(), h.size() * 4, hipMemcpyHostToDevice);
  keep.push_back(d);
  return static_cast<uint32_t*>(d);
}

// blocks until the pre-position behind r has finished (the gate itself never waits for it)
void finished(spp_ready_t r) {
  spp_summary sum{};
  CHECK(spp_ready_summary(r, &sum) == SPP_OK);
}

spp_gate_outcome gate(spp_ready_t r, const uint32_t* set, const std::vector<int32_t>* realized,
                      int32_t* tok, hipStream_t st = nullptr) {
  spp_gate_outcome o = SPP_FALL_INVALID;
  CHECK(spp_gate(r, 2.f, set, realized ? realized->data() : nullptr,
                 realized ? (int32_t)realized->size() : 0, st, tok, &o, nullptr) == SPP_OK);
  return o;
}

void state_machine(spp_model_t m, const uint32_t* set) {
  Sess s(m, 256, 64);
  const auto delta = tokens(40, 1);
  CHECK(spp_kv_append_delta(s.h, delta.data(), 40, nullptr) == SPP_OK);
  // Alg. 1's budget: B = 64 - 40 = 24 cells
  spp_ready_t r{};
  const auto big = tokens(25, 2), entry = tokens(24, 3);
  CHECK(spp_preposition(s.h, big.data(), 25, s.dist, set, nullptr, &r) == SPP_SKIPPED_BUDGET);
  CHECK(spp_preposition(s.h, entry.data(), 24, s.dist, set, nullptr, &r) == SPP_OK);
  spp_summary sum{};
  CHECK(spp_ready_summary(r, &sum) == SPP_OK);
  CHECK(sum.argmax == 7 && sum.gap > 9.f && sum.position == 64 && (sum.flags & 2u));
  int32_t tok = -1;
  CHECK(gate(r, set, &entry, &tok) == SPP_SERVED && tok == 7);
  const auto other = tokens(24, 4);
  CHECK(gate(r, set, &other, &tok) == SPP_FALL_INELIGIBLE && tok == -1);
  CHECK(gate(r, nullptr, nullptr, &tok) == SPP_FALL_NOT_IN_SET);
  // every mutation invalidates the handle (Sec. 3.6)
  for (int kind : {SPP_MUT_UPDATE, SPP_MUT_ROLLBACK, SPP_MUT_SHIFT}) {
    CHECK(spp_preposition(s.h, entry.data(), 24, s.dist, set, nullptr, &r) == SPP_OK);
    finished(r);
    CHECK(gate(r, set, nullptr, &tok) == SPP_SERVED);
    CHECK(spp_invalidate_on_mutation(s.h, (spp_mutation)kind, 40) == SPP_OK);
    CHECK(gate(r, set, nullptr, &tok) == SPP_FALL_INVALID && tok == -1);
    spp_summary dummy{};
    CHECK(spp_ready_summary(r, &dummy) == SPP_E_STATE);
  }
  CHECK(spp_preposition(s.h, entry.data(), 24, s.dist, set, nullptr, &r) == SPP_OK);
  CHECK(spp_shift(s.h, 8, nullptr) == SPP_OK);
  CHECK(gate(r, set, nullptr, &tok) == SPP_FALL_INVALID);
  spp_session_info_t info{};
  CHECK(spp_session_info(s.h, &info) == SPP_OK);
  CHECK(info.n_committed == 32 && info.valid == 0 && info.entry_len == 0);
  // fall-through resume: a new ready state at the new end
  CHECK(spp_preposition(s.h, entry.data(), 16, s.dist, set, nullptr, &r) == SPP_OK);
  const auto d2 = tokens(3, 5);
  spp_ready_t r2{};
  CHECK(spp_resume(s.h, d2.data(), 3, s.dist, set, nullptr, &r2) == SPP_OK);
  CHECK(gate(r, set, nullptr, &tok) == SPP_FALL_INVALID);
  finished(r2);
  CHECK(gate(r2, set, nullptr, &tok) == SPP_SERVED && tok == 7);
  CHECK(spp_session_info(s.h, &info) == SPP_OK);
  CHECK(info.n_committed == 32 + 16 + 3 && info.position == 51);
  CHECK(spp_session_restore(s.h, 10) == SPP_OK);
  CHECK(gate(r2, set, nullptr, &tok) == SPP_FALL_INVALID);
}

void pending_gate(spp_model_t m, const uint32_t* set) {
  Sess s(m, 256, 0);
  const auto delta = tokens(20, 6), entry = tokens(12, 7);
  CHECK(spp_kv_append_delta(s.h, delta.data(), 20, nullptr) == SPP_OK);
  hipDeviceSynchronize();
  stub::hold(true);  // the device starts nothing: the pre-position stays pending
  spp_ready_t r{};
  CHECK(spp_preposition(s.h, entry.data(), 12, s.dist, set, nullptr, &r) == SPP_OK);
  int32_t tok = -1;
  for (int i = 0; i < 3; ++i) CHECK(gate(r, set, &entry, &tok) == SPP_FALL_INVALID && tok == -1);
  spp_session_info_t info{};
  CHECK(spp_session_info(s.h, &info) == SPP_OK && info.valid == 1 && info.decoded == 0);
  // a gate from another thread while the device is released
  std::atomic<int> served{0};
  std::thread t([&] {
    int32_t tk = -1;
    const auto until = std::chrono::steady_clock::now() + std::chrono::seconds(20);
    while (!served.load() && std::chrono::steady_clock::now() < until) {
      if (gate(r, set, &entry, &tk) == SPP_SERVED) served = 1;
      else std::this_thread::yield();
    }
  });
  std::this_thread::sleep_for(std::chrono::milliseconds(5));
  stub::hold(false);
  t.join();
  CHECK(served.load() == 1);
  CHECK(spp_session_info(s.h, &info) == SPP_OK && info.decoded == 1);
}

void idle_yield(spp_model_t m, const uint32_t* set) {
  Sess s(m, 256, 0);
  const auto delta = tokens(20, 8), entry = tokens(12, 9);
  CHECK(spp_kv_append_delta(s.h, delta.data(), 20, nullptr) == SPP_OK);
  spp_ready_t r{};
  uint32_t flag = 1;  // a request already waiting: nothing is enqueued
  CHECK(spp_preposition_idle(s.h, entry.data(), 12, s.dist, set, &flag, 1, nullptr, &r) ==
        SPP_YIELDED);
  // the flag raised by a serving thread while the pass waits on the device
  __atomic_store_n(&flag, 0u, __ATOMIC_RELEASE);
  hipDeviceSynchronize();
  stub::hold(true);
  std::thread server([&] {
    std::this_thread::sleep_for(std::chrono::milliseconds(5));
    __atomic_store_n(&flag, 1u, __ATOMIC_RELEASE);
    std::this_thread::sleep_for(std::chrono::milliseconds(2));
    stub::hold(false);
  });
  const spp_status rc =
      spp_preposition_idle(s.h, entry.data(), 12, s.dist, set, &flag, 1, nullptr, &r);
  server.join();
  CHECK(rc == SPP_YIELDED);
  spp_session_info_t info{};
  CHECK(spp_session_info(s.h, &info) == SPP_OK && info.valid == 0 && info.n_committed == 20);
  int32_t tok = -1;
  CHECK(gate(r, set, nullptr, &tok) == SPP_FALL_INVALID);
  // with the flag clear the pass completes and serves
  __atomic_store_n(&flag, 0u, __ATOMIC_RELEASE);
  CHECK(spp_preposition_idle(s.h, entry.data(), 12, s.dist, set, &flag, 1, nullptr, &r) == SPP_OK);
  CHECK(gate(r, set, &entry, &tok) == SPP_SERVED && tok == 7);
}

void concurrent(spp_model_t m, const uint32_t* set) {
  constexpr int kS = 4;
  std::vector<Sess*> ss;
  std::vector<spp_ready_t> handles(kS);
  const auto entry = tokens(8, 10);
  for (int i = 0; i < kS; ++i) {
    ss.push_back(new Sess(m, 512, 0));
    const auto d = tokens(16 + i, 11 + i);
    CHECK(spp_kv_append_delta(ss[i]->h, d.data(), (int)d.size(), nullptr) == SPP_OK);
    CHECK(spp_preposition(ss[i]->h, entry.data(), 8, ss[i]->dist, set, nullptr, &handles[i]) ==
          SPP_OK);
  }
  std::atomic<bool> stop{false};
  std::atomic<long> gates{0}, bad{0};
  std::vector<std::thread> gaters;
  for (int g = 0; g < 3; ++g)
    gaters.emplace_back([&, g] {
      hipStream_t st = nullptr;
      hipStreamCreate(&st);
      long k = 0;
      while (!stop.load()) {
        const spp_ready_t r = handles[(g + k++) % kS];  // possibly stale: that is the point
        int32_t tok = -1;
        spp_gate_outcome o = SPP_FALL_INVALID;
        if (spp_gate(r, 2.f, set, nullptr, 0, st, &tok, &o, nullptr) != SPP_OK) ++bad;
        if (o == SPP_SERVED && tok != 7) ++bad;
        if (o != SPP_SERVED && o != SPP_FALL_INVALID) ++bad;
        ++gates;
      }
      hipStreamDestroy(st);
    });
  // the mutating thread: pre-position, shift, roll back and destroy while gates run
  for (int round = 0; round < 40; ++round) {
    const int i = round % kS;
    spp_ready_t r{};
    CHECK(spp_preposition(ss[i]->h, entry.data(), 8, ss[i]->dist, set, nullptr, &r) == SPP_OK);
    if (round % 3 == 0) CHECK(spp_invalidate_on_mutation(ss[i]->h, SPP_MUT_ROLLBACK, 16) == SPP_OK);
    if (round % 5 == 0) {
      spp_session_info_t info{};
      CHECK(spp_session_info(ss[i]->h, &info) == SPP_OK);
      if (info.n_committed > 1) CHECK(spp_shift(ss[i]->h, 1, nullptr) == SPP_OK);
    }
  }
  // destroy two sessions while their (now stale) handles are still gated
  ss[0]->destroy();
  ss[1]->destroy();
  std::this_thread::sleep_for(std::chrono::milliseconds(20));
  stop = true;
  for (auto& t : gaters) t.join();
  CHECK(bad.load() == 0);
  CHECK(gates.load() > 0);
  for (Sess* s : ss) delete s;
}

void batched(spp_model_t m, const uint32_t* set) {
  constexpr int kS = 6;
  std::vector<Sess*> ss;
  std::vector<spp_session_t> hs;
  std::vector<std::vector<int32_t>> entries;
  std::vector<const int32_t*> eptr;
  std::vector<int32_t> lens;
  std::vector<float*> dists;
  for (int i = 0; i < kS; ++i) {
    ss.push_back(new Sess(m, 256, 0));
    const auto d = tokens(10 + 3 * i, 20 + i);
    CHECK(spp_kv_append_delta(ss[i]->h, d.data(), (int)d.size(), nullptr) == SPP_OK);
    hs.push_back(ss[i]->h);
    entries.push_back(tokens(4 + i, 30 + i));
    lens.push_back(4 + i);
    dists.push_back(ss[i]->dist);
  }
  for (auto& e : entries) eptr.push_back(e.data());
  std::vector<spp_ready_t> ready(kS);
  std::vector<spp_status> st(kS);
  CHECK(spp_preposition_batch(kS, hs.data(), eptr.data(), lens.data(), dists.data(), nullptr,
                              ready.data(), st.data()) == SPP_OK);
  for (int i = 0; i < kS; ++i) CHECK(st[i] == SPP_OK);
  hipDeviceSynchronize();
  std::vector<float> taus(kS, 2.f);
  std::vector<const uint32_t*> bms(kS, set);
  std::vector<int32_t> tok(kS, -1), tok2(kS, -1);
  std::vector<spp_gate_outcome> out(kS), out2(kS);
  CHECK(spp_gate_batch(kS, ready.data(), taus.data(), bms.data(), nullptr, tok.data(),
                       out.data()) == SPP_OK);
  CHECK(spp_gate_batch_noalloc(kS, ready.data(), taus.data(), bms.data(), nullptr, tok2.data(),
                               out2.data()) == SPP_OK);
  for (int i = 0; i < kS; ++i) {
    // the batched LM head planted token 7 + i; the set holds 7..10
    const bool in_set = 7 + i <= 10;
    CHECK(out[i] == (in_set ? SPP_SERVED : SPP_FALL_NOT_IN_SET));
    CHECK(out2[i] == out[i] && tok2[i] == tok[i]);
    if (in_set) CHECK(tok[i] == 7 + i);
  }
  // two threads on the allocation-free entry point (calls on one device serialize)
  std::thread a([&] {
    std::vector<int32_t> t(kS);
    std::vector<spp_gate_outcome> o(kS);
    for (int k = 0; k < 50; ++k)
      CHECK(spp_gate_batch_noalloc(kS, ready.data(), taus.data(), bms.data(), nullptr, t.data(),
                                   o.data()) == SPP_OK &&
            o[0] == SPP_SERVED && t[0] == 7);
  });
  std::vector<int32_t> t(3);
  std::vector<spp_gate_outcome> o(3);
  for (int k = 0; k < 50; ++k)
    CHECK(spp_gate_batch_noalloc(3, ready.data() + 1, taus.data(), bms.data(), nullptr, t.data(),
                                 o.data()) == SPP_OK &&
          o[0] == SPP_SERVED && t[0] == 8);
  a.join();
  {
    std::vector<spp_ready_t> r65(65, ready[0]);
    std::vector<float> t65(65, 2.f);
    std::vector<const uint32_t*> b65(65, set);
    std::vector<int32_t> k65(65);
    std::vector<spp_gate_outcome> o65(65);
    CHECK(spp_gate_batch_noalloc(65, r65.data(), t65.data(), b65.data(), nullptr, k65.data(),
                                 o65.data()) == SPP_E_INVALID_ARG);
  }
  for (Sess* s : ss) delete s;
}

}  // namespace

int main() {
  const long base = stub::live_allocations();
  {
    Weights w;
    spp_model_config c = config(8);
    spp_model_t m = nullptr;
    CHECK(spp_model_create(&c, &w.w, &m) == SPP_OK);
    std::vector<void*> keep;
    const uint32_t* set = bitmap(keep, {7, 8, 9, 10});
    state_machine(m, set);
    pending_gate(m, set);
    idle_yield(m, set);
    concurrent(m, set);
    batched(m, set);
    hipDeviceSynchronize();
    CHECK(spp_model_destroy(m) == SPP_OK);
    for (void* p : keep) hipFree(p);
  }
  // every device and pinned allocation of the models and sessions is returned
  CHECK(stub::live_allocations() == base);
  stub::shutdown();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("OK\n");
  return 0;
}
