// Candidate keys shared by the kernels: a candidate (logit or score, id) is
// the 64-bit key (ord(value) << 32) | ~id, where ord() maps fp32 to an
// unsigned integer of the same order.  A larger key is a better candidate:
// larger value first, smaller id first on equal values.  That is the
// (dist, id) order of the search with dist = -value.  No candidate has key 0
// (the id half of a key is never zero), so 0 serves as "none".
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace vie {

__device__ __forceinline__ uint32_t f2ord(float f)
{
    const uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);  // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float ord2f(uint32_t o)
{
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

__device__ __forceinline__ uint64_t make_key(float v, int32_t id)
{
    return ((uint64_t)f2ord(v) << 32) | (uint64_t)(~(uint32_t)id);
}

__device__ __forceinline__ int32_t key_id(uint64_t k) { return (int32_t)(~(uint32_t)k); }
__device__ __forceinline__ float key_logit(uint64_t k) { return ord2f((uint32_t)(k >> 32)); }

}  // namespace vie
