// Messages between the CUs of the persistent multi-CU kernels (gfx950): 64-bit words that carry an
// fp32 value in the low half and the step they belong to (step + 1) in the high half, written and
// read with relaxed atomics.  A reader re-reads a word until the tag it expects appears, so it needs
// no fence: each word validates itself.  Also the launch-time grid meeting in which every block
// learns which XCD each block of the launch runs on.
#pragma once
#include <hip/hip_runtime.h>

#include "wn.h"
#include "wn_internal.h"

namespace wnk {

typedef unsigned long long u64;

__device__ __forceinline__ u64 pack(float v, unsigned tag) {
  return ((u64)tag << 32) | (u64)__float_as_uint(v);
}
__device__ __forceinline__ float wval(u64 w) { return __uint_as_float((unsigned)w); }
__device__ __forceinline__ unsigned wtag(u64 w) { return (unsigned)(w >> 32); }
__device__ __forceinline__ u64 ldw(const u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void stw(u64* p, u64 w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// A post whose reader runs on the same XCD: the store only has to reach that XCD's L2, which the
// reader's agent-scope loads read through, so it is issued at workgroup scope (it is not written
// through to memory; measured: 0.64 against 0.86 us per round trip between two CUs of one XCD).
__device__ __forceinline__ void stw(u64* p, u64 w, bool local) {
  if (local) __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  else __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Which posts of a block go to a reader on its own XCD: bit k of m for destination k, or, with ALL,
// every post (every role of the block's replica runs on its XCD in this launch).  ALL is a
// compile-time constant, so that build of a role posts with no branch on the scope (a branch per
// post measured 0.7 us per step at l = 20, r = 64, one stream: ~3 posts per layer).
template <bool ALL>
struct Local {
  unsigned m;
  __device__ __forceinline__ bool operator()(int k) const { return ALL || ((m >> k) & 1u); }
};
__device__ __forceinline__ int ld_status(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls of pairs of tagged words (16 bytes) through a buffer resource over the workspace's tagged
// region (histories and mailboxes): 128-bit loads at agent scope (cache policy sc1: past the CU's
// L1, from the L2), about three times the rate of 64-bit atomic loads per CU (measured: 123 against
// 38 GB/s), and bounds-checked by the hardware (a read past the region returns zeros; the host keeps
// the region under 2 GiB, the buffer's 32-bit byte offsets).  Each 64-bit word is written whole by
// one store, so a word read in a pair is never torn; the two words of a pair carry their own tags.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t wrsrc;
__device__ __forceinline__ wrsrc region_rsrc(const u64* base, size_t words) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)(words * 8), 0x00020000);
}
// words `word`, `word` + 1 of the region (word even)
__device__ __forceinline__ u32x4 ld_pair(wrsrc rs, unsigned word) {
  return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(word * 8u), 0, 16 /* sc1 */);
}

// Block-uniform abort flag kept in LDS.
struct Sync {
  int* flag;
  __device__ bool failed() const { return *flag != 0; }
};

// The grid's meeting at the start of a launch of a multi-CU kernel.  Thread 0 of every active block
// stores the block's XCC_ID at xmap[blockIdx.x], then the n_active blocks meet once (an arrival count
// and a generation word after the map; a cooperative launch keeps every block resident, and the wait
// is bounded).  Returns the block's XCD, or -1 when the grid never met (WN_ETIMEOUT is then in the
// status word).  Every thread of the block gets the result.
__device__ __forceinline__ int grid_meet(u64* xmap, int n_active, int spin_limit, int* status, int* s_me) {
  if (threadIdx.x == 0) {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    *s_me = (int)(v & 0xf);
    __hip_atomic_store(xmap + blockIdx.x, (u64)(v & 0xf), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    u64* cnt = xmap + WN_CHAIN_GRID;
    u64* gen = cnt + 1;
    const u64 g0 = __hip_atomic_load(gen, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
    if (__hip_atomic_fetch_add(cnt, 1ull, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) == (u64)(n_active - 1)) {
      __hip_atomic_store(cnt, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_add(gen, 1ull, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      int spins = 0;
      while (__hip_atomic_load(gen, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == g0) {
        if (++spins > spin_limit) {
          atomicCAS(status, 0, (int)WN_ETIMEOUT);
          *s_me = -1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  __syncthreads();
  return *s_me;
}

}  // namespace wnk
