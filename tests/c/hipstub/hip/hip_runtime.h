/* Host-only test double of the few HIP runtime declarations the C-ABI layer
 * (kf_api.cpp) uses, so that the layer can be compiled with g++ under
 * AddressSanitizer and UndefinedBehaviorSanitizer without a GPU.  The
 * definitions, and those of the kernel launchers, live in
 * tests/c/api_stress.cpp, which checks every launch it receives. */
#pragma once

#include <stddef.h>
#include <stdint.h>

typedef enum { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNoDevice = 100 } hipError_t;
typedef struct ihipStream_t* hipStream_t;
typedef enum { hipDeviceAttributeMultiprocessorCount = 63 } hipDeviceAttribute_t;

hipError_t hipGetDevice(int* device);
hipError_t hipGetLastError(void);
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int device);
