// ql_xcd.h -- exchange primitives of the kernels that keep every hand-off
// of a step inside one XCD: 64-bit tagged words (step tag << 32 | payload)
// written with plain stores, which stay in the XCD's L2, and read with
// device-coherent loads, which find them there; bounded polls of such words;
// lane-group reductions.
#pragma once
#include "ql_device.h"
#include "ql_exchange.h"

namespace ql {

// n rounded up to 16 bytes (LDS layouts fixed at compile time)
constexpr size_t xal16(size_t n) { return (n + 15) / 16 * 16; }

// Quantizer params of a row as the encoder needs them.
struct XParam {
  double q;
  int32_t z;
  float inv_q;
};

// A 64-bit exchange word with a plain store (no cache-policy bits): it stays
// in the L2 of the producer's XCD, where the consumers' device-coherent loads
// find it.  A wavefront-scope atomic store is exactly that instruction, and
// the compiler counts it among the outstanding memory operations.
__device__ __forceinline__ void put_word(uint64_t *p, uint32_t tag, uint32_t v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | (uint64_t)v, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_WAVEFRONT);
}

typedef __attribute__((address_space(3))) void *lds_ptr;

// Waits until every vector memory operation of the wave has completed (gfx9
// encoding: only the vector-memory count limited).
__device__ __forceinline__ void wait_vmcnt0() {
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
}

// Re-reads the words addr(i), i < N, whose bit is set in `need` until each
// carries `tag`; the payloads go to v.  A word is read again only while its
// tag has not matched.  False if the wait expired.
template <int N, class AddrFn>
__device__ __forceinline__ bool poll_words(uint32_t need, uint32_t tag, uint32_t (&v)[N],
                                           AddrFn addr, int *flag) {
  static_assert(N < 32, "one bit per word");
  uint32_t got = ~need & ((1u << N) - 1);
  long it = 0;
  for (;;) {
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (!((got >> i) & 1u)) {
        const uint64_t w = ld_tagged(addr(i));
        if ((uint32_t)(w >> 32) == tag) {
          got |= 1u << i;
          v[i] = (uint32_t)w;
        }
      }
    if (!__any(got != (1u << N) - 1)) return true;
    if (wait_expired(flag, it)) return false;
  }
}

// The same for wider sets of words whose payloads go to LDS: each payload is
// stored at dst(i, th) as soon as its tag matches, so no word is held in
// registers between rounds.  Source and destination addresses are recomputed
// every round from an opaque thread id th (nothing per word stays live).  The
// loads of a round are all issued before any of them is examined.
template <int N, class SrcFn, class DstFn>
__device__ __forceinline__ bool poll_to_lds(uint32_t need, uint32_t tag, SrcFn src, DstFn dst,
                                            int *flag) {
  static_assert(N < 32, "one bit per word");
  constexpr uint32_t all = (1u << N) - 1;
  uint32_t got = ~need & all;
  long it = 0;
  for (;;) {
    int th = (int)threadIdx.x;
    asm volatile("" : "+v"(th));
    uint64_t w[N];
#pragma unroll
    for (int i = 0; i < N; ++i) w[i] = ((got >> i) & 1u) ? 0 : ld_tagged(src(i, th));
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (!((got >> i) & 1u) && (uint32_t)(w[i] >> 32) == tag) {
        got |= 1u << i;
        *dst(i, th) = (uint32_t)w[i];
      }
    if (!__any(got != all)) return true;
    if (wait_expired(flag, it)) return false;
  }
}

// The first round of poll_to_lds issued ahead of other work: the words
// whose bit is set in `need` are loaded into w; poll_to_lds_finish examines
// them later (and polls on for those whose tag had not matched).
template <int N, class SrcFn>
__device__ __forceinline__ void poll_to_lds_issue(uint32_t need, SrcFn src, uint64_t (&w)[N]) {
  int th = (int)threadIdx.x;
  asm volatile("" : "+v"(th));
#pragma unroll
  for (int i = 0; i < N; ++i) w[i] = ((need >> i) & 1u) ? ld_tagged(src(i, th)) : 0;
}
template <int N, class SrcFn, class DstFn>
__device__ __forceinline__ bool poll_to_lds_finish(uint32_t need, uint32_t tag, const uint64_t (&w)[N],
                                                   SrcFn src, DstFn dst, int *flag) {
  // every load of the round has landed, on every path (they are the wave's
  // youngest memory operations, so this waits for nothing more)
  wait_vmcnt0();
  int th = (int)threadIdx.x;
  asm volatile("" : "+v"(th));
#pragma unroll
  for (int i = 0; i < N; ++i)
    if (((need >> i) & 1u) && (uint32_t)(w[i] >> 32) == tag) {
      need &= ~(1u << i);
      *dst(i, th) = (uint32_t)w[i];
    }
  if (!__any(need != 0)) return true;
  return poll_to_lds<N>(need, tag, src, dst, flag);
}

// Reductions over aligned groups of 8 or 16 lanes (DPP): every lane of the
// group ends with the group's result.
template <class Op>
__device__ __forceinline__ int red8(int v, Op op) {
  v = op(v, __builtin_amdgcn_mov_dpp(v, 0xb1, 0xf, 0xf, false));   // quad_perm [1,0,3,2]
  v = op(v, __builtin_amdgcn_mov_dpp(v, 0x4e, 0xf, 0xf, false));   // quad_perm [2,3,0,1]
  return op(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, false));  // row_half_mirror
}
template <class Op>
__device__ __forceinline__ int red16(int v, Op op) {
  v = red8(v, op);
  return op(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, false));  // row_mirror
}
// Over aligned groups of W = 16, 32 or 64 lanes.
template <class Op>
__device__ __forceinline__ int red_w(int v, int W, Op op) {
  v = red16(v, op);
  if (W == 16) return v;
  const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
  const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
  if (W == 64) return op(op(r0, r1), op(r2, r3));
  return (threadIdx.x & 32) ? op(r2, r3) : op(r0, r1);
}
struct MinI {
  __device__ int operator()(int a, int b) const { return min(a, b); }
};
struct AddI {
  __device__ int operator()(int a, int b) const { return a + b; }
};

}  // namespace ql
