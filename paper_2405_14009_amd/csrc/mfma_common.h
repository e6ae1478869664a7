// CDNA4 building blocks shared by the MFMA kernels: fragment types, buffer
// descriptors, buffer-load-to-LDS copies, LDS addresses, stage barriers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

namespace {

constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that is always out of range -> zeros

// Buffer descriptor (4 dwords: base, stride 0, size in bytes, format) over
// [base, base + bytes).  Base and size are workgroup uniform and made provably
// so (readfirstlane), so the descriptor lives in scalar registers.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, long bytes) {
  const long cap = 0x7fffffffL;
  const uint64_t a = (uint64_t)base;
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane((uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) & 0xffff;
  r.z = __builtin_amdgcn_readfirstlane((int)(bytes < cap ? bytes : cap));
  r.w = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer offset `off` into LDS at lds_base + 16 * lane
// (zeros when off is out of range).  Issued as inline assembly so that the
// compiler does not order later LDS reads of the other stage behind it; the
// kernel waits for it explicitly (vmcnt) before the barrier that publishes
// the stage.  M0 carries the LDS base and is not otherwise used by these
// kernels.
__device__ __forceinline__ void dma16(const i32x4& r, uint32_t lds_base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_base), "v"(off), "s"(r)
               : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// vmcnt(0): this thread's copies have landed; the barrier then makes every
// wave's copies visible and frees the stage just read for the next copy.
// The scheduling fences keep the wait after every MFMA of the stage just
// computed (the scheduler would otherwise hoist it above MFMAs, which touch
// no memory, and shrink the time the next stage's copy has to land).
__device__ __forceinline__ void stage_sync() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  __builtin_amdgcn_sched_barrier(0);
}

}  // namespace
