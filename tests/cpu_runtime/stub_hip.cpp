// Host-only implementation of the HIP stand-in declared in hip/hip_runtime.h (test
// infrastructure for the CPU build of the runtime under the sanitizers).
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <mutex>
#include <set>
#include <thread>
#include <vector>

struct StubEvent {
  std::mutex mu;
  std::condition_variable cv;
  uint64_t recorded = 0;   // records issued
  uint64_t completed = 0;  // records their stream has reached
  std::chrono::steady_clock::time_point at;
};

struct StubStream {
  std::mutex mu;
  std::condition_variable cv;       // work arrived / stop
  std::condition_variable idle_cv;  // queue drained
  std::deque<std::function<void()>> q;
  bool busy = false, stop = false;
  std::thread worker;
};

namespace {

std::atomic<bool> g_hold{false};
std::mutex g_streams_mu;
std::vector<StubStream*> g_streams;
StubStream* g_default = nullptr;

std::mutex g_alloc_mu;
std::set<void*> g_allocs;

void run(StubStream* s) {
  for (;;) {
    std::function<void()> fn;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv.wait(lk, [&] { return s->stop || !s->q.empty(); });
      if (s->q.empty()) return;  // stopped and drained
    }
    // a held device starts nothing new
    while (g_hold.load(std::memory_order_acquire))
      std::this_thread::sleep_for(std::chrono::microseconds(100));
    {
      std::lock_guard<std::mutex> lk(s->mu);
      fn = std::move(s->q.front());
      s->q.pop_front();
      s->busy = true;
    }
    fn();
    {
      std::lock_guard<std::mutex> lk(s->mu);
      s->busy = false;
      if (s->q.empty()) s->idle_cv.notify_all();
    }
  }
}

StubStream* make_stream() {
  StubStream* s = new StubStream;
  s->worker = std::thread(run, s);
  std::lock_guard<std::mutex> lk(g_streams_mu);
  g_streams.push_back(s);
  return s;
}

StubStream* resolve(hipStream_t st) {
  if (st) return st;
  std::lock_guard<std::mutex> lk(g_streams_mu);
  if (!g_default) {
    g_default = new StubStream;
    g_default->worker = std::thread(run, g_default);
    g_streams.push_back(g_default);
  }
  return g_default;
}

void sync_stream(StubStream* s) {
  std::unique_lock<std::mutex> lk(s->mu);
  s->idle_cv.wait(lk, [&] { return s->q.empty() && !s->busy; });
}

void* alloc(size_t n) {
  const size_t b = (n + 255) / 256 * 256 + 256;
  void* p = std::aligned_alloc(256, b);
  if (!p) return nullptr;
  std::memset(p, 0, b);
  std::lock_guard<std::mutex> lk(g_alloc_mu);
  g_allocs.insert(p);
  return p;
}

hipError_t release(void* p) {
  if (!p) return hipSuccess;
  {
    std::lock_guard<std::mutex> lk(g_alloc_mu);
    if (!g_allocs.erase(p)) return hipErrorInvalidValue;
  }
  std::free(p);
  return hipSuccess;
}

}  // namespace

namespace stub {
void enqueue(hipStream_t st, std::function<void()> fn) {
  StubStream* s = resolve(st);
  std::lock_guard<std::mutex> lk(s->mu);
  s->q.push_back(std::move(fn));
  s->cv.notify_one();
}
void hold(bool on) { g_hold.store(on, std::memory_order_release); }
long live_allocations() {
  std::lock_guard<std::mutex> lk(g_alloc_mu);
  return (long)g_allocs.size();
}
void shutdown() {
  std::vector<StubStream*> all;
  {
    std::lock_guard<std::mutex> lk(g_streams_mu);
    all.swap(g_streams);
    g_default = nullptr;
  }
  for (StubStream* s : all) {
    {
      std::lock_guard<std::mutex> lk(s->mu);
      s->stop = true;
      s->cv.notify_one();
    }
    s->worker.join();
    delete s;
  }
}
}  // namespace stub

hipError_t hipMalloc(void** p, size_t n) {
  if (!p) return hipErrorInvalidValue;
  *p = alloc(n);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void* p) { return release(p); }
hipError_t hipHostMalloc(void** p, size_t n, unsigned) { return hipMalloc(p, n); }
hipError_t hipHostFree(void* p) { return release(p); }
hipError_t hipHostGetDevicePointer(void** dev, void* host, unsigned) {
  *dev = host;
  return hipSuccess;
}

hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  hipDeviceSynchronize();
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t st) {
  stub::enqueue(st, [dst, src, n] { std::memcpy(dst, src, n); });
  return hipSuccess;
}

hipError_t hipEventCreate(hipEvent_t* e) {
  *e = new StubEvent;
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  if (!e) return hipErrorInvalidResourceHandle;
  {
    // a record still pending on a stream would touch the event after this: wait for it
    std::unique_lock<std::mutex> lk(e->mu);
    e->cv.wait(lk, [&] { return e->completed >= e->recorded; });
  }
  delete e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t st) {
  if (!e) return hipErrorInvalidResourceHandle;
  uint64_t gen;
  {
    std::lock_guard<std::mutex> lk(e->mu);
    gen = ++e->recorded;
  }
  stub::enqueue(st, [e, gen] {
    std::lock_guard<std::mutex> lk(e->mu);
    if (gen > e->completed) {
      e->completed = gen;
      e->at = std::chrono::steady_clock::now();
    }
    e->cv.notify_all();
  });
  return hipSuccess;
}
hipError_t hipEventQuery(hipEvent_t e) {
  std::lock_guard<std::mutex> lk(e->mu);
  return e->completed >= e->recorded ? hipSuccess : hipErrorNotReady;
}
hipError_t hipEventSynchronize(hipEvent_t e) {
  std::unique_lock<std::mutex> lk(e->mu);
  const uint64_t want = e->recorded;
  e->cv.wait(lk, [&] { return e->completed >= want; });
  return hipSuccess;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  std::scoped_lock lk(a->mu, b->mu);
  if (a->completed < a->recorded || b->completed < b->recorded || !a->recorded || !b->recorded)
    return hipErrorNotReady;
  *ms = std::chrono::duration<float, std::milli>(b->at - a->at).count();
  return hipSuccess;
}

hipError_t hipStreamCreate(hipStream_t* st) {
  *st = make_stream();
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t st) {
  if (!st) return hipErrorInvalidResourceHandle;
  sync_stream(st);
  {
    std::lock_guard<std::mutex> lk(g_streams_mu);
    for (auto it = g_streams.begin(); it != g_streams.end(); ++it)
      if (*it == st) {
        g_streams.erase(it);
        break;
      }
  }
  {
    std::lock_guard<std::mutex> lk(st->mu);
    st->stop = true;
    st->cv.notify_one();
  }
  st->worker.join();
  delete st;
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t st, hipEvent_t e, unsigned) {
  uint64_t want;
  {
    std::lock_guard<std::mutex> lk(e->mu);
    want = e->recorded;
  }
  stub::enqueue(st, [e, want] {
    std::unique_lock<std::mutex> lk(e->mu);
    e->cv.wait(lk, [&] { return e->completed >= want; });
  });
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t st) {
  sync_stream(resolve(st));
  return hipSuccess;
}
hipError_t hipStreamQuery(hipStream_t st) {
  StubStream* s = resolve(st);
  std::lock_guard<std::mutex> lk(s->mu);
  return s->q.empty() && !s->busy ? hipSuccess : hipErrorNotReady;
}
hipError_t hipDeviceSynchronize() {
  std::vector<StubStream*> all;
  {
    std::lock_guard<std::mutex> lk(g_streams_mu);
    all = g_streams;
  }
  for (StubStream* s : all) sync_stream(s);
  return hipSuccess;
}
hipError_t hipSetDevice(int dev) { return dev == 0 ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t, int) {
  *value = 256;
  return hipSuccess;
}
hipError_t hipGetSymbolAddress(void** p, const void* symbol) {
  *p = const_cast<void*>(symbol);
  return hipSuccess;
}
hipError_t hipGetLastError() { return hipSuccess; }
const char* hipGetErrorString(hipError_t e) {
  switch (e) {
    case hipSuccess: return "hipSuccess";
    case hipErrorNotReady: return "hipErrorNotReady";
    case hipErrorOutOfMemory: return "hipErrorOutOfMemory";
    case hipErrorInvalidValue: return "hipErrorInvalidValue";
    default: return "hipError (stub)";
  }
}
