/* Host-only stand-in for the few HIP runtime declarations the library's
 * host code uses, so that kvq_api.cpp can be compiled by the system C++
 * compiler with AddressSanitizer and UBSan and run without a GPU.
 * Test infrastructure only: "device" memory is host memory here, copies are
 * memcpy, and kernel launches do nothing (tests/sanitize/hip_stub.cpp). */
#pragma once
#include <stddef.h>

typedef int hipError_t;
enum { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNoDevice = 100 };
typedef void* hipStream_t;
typedef enum {
  hipMemcpyHostToHost = 0,
  hipMemcpyHostToDevice = 1,
  hipMemcpyDeviceToHost = 2,
  hipMemcpyDeviceToDevice = 3,
  hipMemcpyDefault = 4
} hipMemcpyKind;
typedef enum { hipDeviceAttributeMultiprocessorCount = 63 } hipDeviceAttribute_t;

hipError_t hipGetDevice(int* dev);
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int dev);
const char* hipGetErrorString(hipError_t e);
hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind);
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t s);
hipError_t hipStreamSynchronize(hipStream_t s);
