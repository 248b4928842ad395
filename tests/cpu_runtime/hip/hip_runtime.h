// Host-only stand-in for the part of the HIP runtime API that the library's runtime
// (runtime.cpp) uses, so that the runtime builds with g++ and runs under AddressSanitizer
// and ThreadSanitizer with no GPU.  Test infrastructure: never linked into libspp.so.
//
// "Device" memory is zeroed host memory.  Every stream is a worker thread that runs its
// queue in order, so device work really is asynchronous to the calling thread; events
// complete when their stream's worker reaches them.  stub::hold() stops every worker
// from starting new work, which makes "the device has not finished yet" reproducible.
#pragma once

#include <cstddef>
#include <cstdint>
#include <functional>

typedef int hipError_t;
enum {
  hipSuccess = 0,
  hipErrorInvalidValue = 1,
  hipErrorOutOfMemory = 2,
  hipErrorInvalidResourceHandle = 400,
  hipErrorNotReady = 600,
};

struct StubStream;
struct StubEvent;
typedef StubStream* hipStream_t;
typedef StubEvent* hipEvent_t;

enum hipMemcpyKind {
  hipMemcpyHostToHost = 0,
  hipMemcpyHostToDevice = 1,
  hipMemcpyDeviceToHost = 2,
  hipMemcpyDeviceToDevice = 3,
  hipMemcpyDefault = 4,
};
enum hipDeviceAttribute_t { hipDeviceAttributeMultiprocessorCount = 1 };

#define hipEventDefault 0u
#define hipEventDisableTiming 2u
#define hipHostMallocDefault 0u
#define hipHostMallocMapped 2u
#define hipHostMallocCoherent 0x40000000u

#define __device__
#define __host__
#define __align__(n) __attribute__((aligned(n)))
#define HIP_SYMBOL(x) (reinterpret_cast<const void*>(&(x)))

struct float2 {
  float x, y;
};

hipError_t hipMalloc(void** p, size_t n);
hipError_t hipFree(void* p);
hipError_t hipHostMalloc(void** p, size_t n, unsigned flags);
hipError_t hipHostFree(void* p);
hipError_t hipHostGetDevicePointer(void** dev, void* host, unsigned flags);
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind kind);
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind kind,
                          hipStream_t st);
hipError_t hipEventCreate(hipEvent_t* e);
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned flags);
hipError_t hipEventDestroy(hipEvent_t e);
hipError_t hipEventRecord(hipEvent_t e, hipStream_t st);
hipError_t hipEventQuery(hipEvent_t e);
hipError_t hipEventSynchronize(hipEvent_t e);
hipError_t hipEventElapsedTime(float* ms, hipEvent_t start, hipEvent_t stop);
hipError_t hipStreamCreate(hipStream_t* st);
hipError_t hipStreamDestroy(hipStream_t st);
hipError_t hipStreamWaitEvent(hipStream_t st, hipEvent_t e, unsigned flags);
hipError_t hipStreamSynchronize(hipStream_t st);
hipError_t hipStreamQuery(hipStream_t st);
hipError_t hipDeviceSynchronize();
hipError_t hipSetDevice(int dev);
hipError_t hipGetDevice(int* dev);
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int dev);
hipError_t hipGetSymbolAddress(void** p, const void* symbol);
hipError_t hipGetLastError();
const char* hipGetErrorString(hipError_t e);

namespace stub {
// Runs fn on the stream's worker after everything enqueued before it (the kernels'
// stand-ins enqueue their work this way).
void enqueue(hipStream_t st, std::function<void()> fn);
// While on, no worker starts new work (work already running finishes).
void hold(bool on);
// Device and pinned allocations not yet freed.
long live_allocations();
// Stops every worker thread (end of the program).
void shutdown();
}  // namespace stub
