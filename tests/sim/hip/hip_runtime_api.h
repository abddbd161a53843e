// Host stand-in for the HIP runtime calls the transfer engine makes, used only
// by the executor tests.  Streams, events and copies become a queue simulator
// (hip_sim.cpp): operations run when something synchronises, in a random order
// among the streams whose next operation is ready, so every ordering the
// engine's waits allow can occur.  Device memory is host memory.
#pragma once

#include <cstddef>
#include <cstdint>

enum hipError_t { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorOutOfMemory = 2, hipErrorNotInitialized = 3, hipErrorUnknown = 999 };
enum hipMemcpyKind {
  hipMemcpyHostToHost = 0, hipMemcpyHostToDevice = 1, hipMemcpyDeviceToHost = 2, hipMemcpyDeviceToDevice = 3
};
enum hipDeviceAttribute_t { hipDeviceAttributeMultiprocessorCount = 63 };

constexpr unsigned hipEventDefault = 0, hipEventDisableTiming = 2, hipEventDisableSystemFence = 0x20000000;
constexpr unsigned hipHostMallocDefault = 0;

struct SimStream;
struct SimEvent;
typedef SimStream* hipStream_t;
typedef SimEvent* hipEvent_t;

const char* hipGetErrorString(hipError_t e);
hipError_t hipSetDevice(int device);
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int device);
hipError_t hipExtStreamCreateWithCUMask(hipStream_t* s, uint32_t n, const uint32_t* mask);
hipError_t hipStreamDestroy(hipStream_t s);
hipError_t hipStreamSynchronize(hipStream_t s);
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned flags);
hipError_t hipEventCreate(hipEvent_t* e);
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned flags);
hipError_t hipEventDestroy(hipEvent_t e);
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s);
hipError_t hipEventSynchronize(hipEvent_t e);
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b);
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind kind, hipStream_t s);
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind kind);
hipError_t hipMalloc(void** p, size_t n);
hipError_t hipFree(void* p);
hipError_t hipHostMalloc(void** p, size_t n, unsigned flags);
hipError_t hipHostFree(void* p);
