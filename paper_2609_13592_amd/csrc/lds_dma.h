// Direct-to-LDS buffer loads (buffer_load ... lds) and the waits on them,
// shared by the kernels that stream operands through LDS rings.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace bst {

// s_waitcnt immediate that waits until at most n vector-memory loads of this
// wavefront are outstanding (other counters untouched)
template <int n>
constexpr int vmcnt_imm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);
}

// 16 bytes per lane from buffer resource r at byte offset off into LDS at
// lds_block + 16 lane (lds_block uniform over the wavefront).  M0 is set here
// and declared clobbered; nothing else in these kernels uses M0 (clang warns
// that a reserved register is clobbered, which is the intent).  One wait
// state separates the M0 write from the load that reads it, as the compiler
// leaves between its own M0 writes and direct-to-LDS loads.  The compiler
// does not see these loads: waits on them are explicit (vmcnt, in issue
// order).  A lane whose offset lies outside the resource writes zeros.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load16_lds(__amdgpu_buffer_rsrc_t r, uint32_t off,
                                           const char* lds_block) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;  // LDS byte address
  const uint32_t la = __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr)lds_block)));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(la), "v"(off), "s"(r)
               : "memory", "m0");
}
#pragma clang diagnostic pop

}  // namespace bst
