// ql_exchange.h -- values passed between the workgroups of one persistent
// launch, and the bounded waits that go with them.
//
// Two protocols.  Tagged words: a value is published as a 64-bit word
// (step tag << 32 | fp32 bits) with a device-coherent store, and a consumer
// re-reads the words it needs until every tag matches.  Arrival counters:
// producers store fp32 values with device-coherent stores, then (after their
// stores have completed and the workgroup has met at a barrier) one thread
// adds 1 to a counter; a consumer waits until the counter reaches the number
// of producer arrivals it needs, then reads with device-coherent loads.
// Every wait is bounded: on expiry a flag in the workspace header is raised,
// and every workgroup leaves at its next wait, so the grid always drains.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ql {

constexpr long kSpinLimit = 1l << 22;
constexpr int kHeaderBytes = 256;  // timeout flag at byte 64
constexpr int kHdrFlag = 16;       // 32-bit word index of the timeout flag
constexpr int kMaxSlices = 256;    // arrival counters per kind and parity
constexpr int kCounterBytes = 2 * 2 * kMaxSlices * 64;  // one 64-byte line per counter


// ---------------------------------------------------------------------------
// Exchange primitives
// ---------------------------------------------------------------------------
__device__ __forceinline__ void publish(uint64_t *p, uint32_t tag, float v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
// The same for consumers on the producer's own XCD only: a plain store, which
// lands in that XCD's L2 without being written through to memory.  Their
// device-coherent loads see it there sooner (a ping-pong between two
// workgroups of one XCD: 0.52-0.68 us a round trip against 0.83-0.95 us);
// a consumer on another XCD might not see it before the end of the launch.
__device__ __forceinline__ void publish_local(uint64_t *p, uint32_t tag, float v) {
  const uint64_t w = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v);
  // one 8-byte store without cache-policy bits (a workgroup-scope atomic
  // store would carry sc0)
  asm volatile("global_store_dwordx2 %0, %1, off" ::"v"(p), "v"(w) : "memory");
}
__device__ __forceinline__ uint64_t ld_tagged(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coherent(const float *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent64(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_coherent64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent_i(int32_t *p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_coherent_i(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Re-reads counted at the start of every wait of this code object's kernels:
// 0, or kSpinLimit - n to bound each wait to n re-reads.  A test hook sets it
// from the host (set_wait_bound_here); every source file that includes this
// header has its own copy.  Constant memory: read with scalar loads.
static __constant__ long g_wait_it0 = 0;

// Bounded-wait bookkeeping: true when the wait must be abandoned.  Called
// once per failed poll with `it` zero before the first.
__device__ __forceinline__ bool wait_expired(int *flag, long &it) {
  if (it == 0) it = g_wait_it0;
  if ((++it & 63) == 0 && __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
    return true;
  if (it > kSpinLimit) {
    __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
  }
  return false;  // no sleep: every re-read is a memory round trip already
}

// Counter protocol (batched tiles): after its coherent stores of step t have
// completed (every wave waits for its own memory operations, then the
// workgroup barrier), thread 0 adds 1 to the arrival counter of the batch
// slice the values belong to; a consumer's thread 0 waits until the counter
// of the slot holds uses * producers.  The stores precede the increment in
// time, and the consumer's loads follow its observation of the count.
__device__ __forceinline__ void arrive(unsigned *cnt) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Thread 0 waits for *cnt >= target; returns false (for thread 0) on expiry.
__device__ __forceinline__ bool wait_count(const unsigned *cnt, unsigned target, int *flag) {
  if (threadIdx.x != 0) return true;
  long it = 0;
  while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target)
    if (wait_expired(flag, it)) return false;
  return true;
}

// Host side: this source file's bound, on the current device (polls = 0:
// the default).
static inline hipError_t set_wait_bound_here(int polls) {
  const long v = polls > 0 && polls < kSpinLimit ? kSpinLimit - polls : 0;
  return hipMemcpyToSymbol(HIP_SYMBOL(g_wait_it0), &v, sizeof v);
}

}  // namespace ql
