// HBM page cache shared by all waves of the paged search (GORIO Sec. 3.2:
// GPU page cache, per-slot ready table, lock-free request descriptors): the
// slot state machine (slot_state.hpp) and the coherent buffer operations that
// move page bytes into and out of the cache's slots.
#pragma once

#include "common.hpp"
#include "slot_state.hpp"

namespace gorio {

// ---------------------------------------------------------------------------
// Page bytes in the cache are read and written with device-scope coherent
// buffer operations (cache policy sc1): a slot is refilled with another page
// while other XCDs may still hold lines of the old page in their L2, and sc1
// accesses are coherent across XCDs by the memory model's definition.  The
// buffer descriptor also bounds every offset to the cache (an offset past it
// reads zero instead of faulting).
// ---------------------------------------------------------------------------
constexpr int kCoherentAgent = 16;  // cache policy bits: sc1

__device__ __forceinline__ __amdgpu_buffer_rsrc_t cache_rsrc(const CacheView &c) {
  const uint32_t bytes = (uint32_t)min((uint64_t)c.slots * c.page_bytes, (uint64_t)0x7FFFFFF0u);
  return __builtin_amdgcn_make_buffer_rsrc(c.data, (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint32_t coherent_load_u32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, kCoherentAgent);
}

__device__ __forceinline__ uint4 coherent_load_u128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kCoherentAgent);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Every page-byte store of this wave has been performed at device scope
// (sc1 stores complete once coherent); also a compiler barrier.  Orders the
// copy of a page before the atomic that marks it READY without the L2
// write-back an agent-scope release would do.
__device__ __forceinline__ void wait_stores_performed() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The READY state was read before any page byte is: the state load has
// completed and no later load is hoisted above this point.  Page bytes are
// read with sc1 loads, so no cache invalidation is needed.
__device__ __forceinline__ void order_after_ready() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void coherent_store_u128(__amdgpu_buffer_rsrc_t r, uint32_t off, uint4 x) {
  __attribute__((ext_vector_type(4))) unsigned int v = {x.x, x.y, x.z, x.w};
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, kCoherentAgent);
}

}  // namespace gorio
