// Device helpers shared by the gfx950 MFMA convolution kernels: fragment
// types, MFMA wrappers, LDS DMA and its waits, and the XCD-aware block
// order.  Internal linkage: each kernel translation unit gets its own copy.
#pragma once
#include <hip/hip_runtime.h>

namespace tgpk {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
// 16-byte chunk as a native vector (HIP's uint4 wraps a union that keeps
// arrays of it out of registers)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// D = A B + C on 32 x 32 x 16 bf16 (A: lane l holds row l % 32, k 8 (l / 32)
// .. + 7; B: column l % 32, same k; D: element v of lane l is row
// 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32).
__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D = A B + C on 16 x 16 x 32 bf16 (A: lane l holds row l % 16, k 8 (l / 16)
// .. + 7; B: column l % 16, same k; D: element v of lane l is row
// 4 (l / 16) + v, column l % 16).
__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

#define TGP_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// s_waitcnt with only the vector-memory counter limited to N (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// Waits until at most `ahead` stages of LPS loads each are still in flight.
template <int NS, int LPS>
__device__ __forceinline__ void wait_stages(int ahead) {
  static_assert(NS >= 2 && NS <= 8 && (NS - 2) * LPS < 64, "vmcnt range");
  if constexpr (NS >= 8) {
    if (ahead >= 6) { wait_vmcnt<6 * LPS>(); return; }
  }
  if constexpr (NS >= 7) {
    if (ahead >= 5) { wait_vmcnt<5 * LPS>(); return; }
  }
  if constexpr (NS >= 6) {
    if (ahead >= 4) { wait_vmcnt<4 * LPS>(); return; }
  }
  if constexpr (NS >= 5) {
    if (ahead >= 3) { wait_vmcnt<3 * LPS>(); return; }
  }
  if constexpr (NS >= 4) {
    if (ahead >= 2) { wait_vmcnt<2 * LPS>(); return; }
  }
  if constexpr (NS >= 3) {
    if (ahead >= 1) { wait_vmcnt<LPS>(); return; }
  }
  wait_vmcnt<0>();
}

// The dispatcher deals workgroups round-robin over the 8 XCDs (each with its
// own L2); this maps dispatch index bid of nb to a logical index so that each
// XCD runs one contiguous range of logical indices.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  const int per = nb / 8, rem = nb % 8;
  const int x = bid % 8, i = bid / 8;
  return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

// Buffer resource descriptor for raw (unswizzled, stride 0) loads of `bytes`
// bytes at p: base address, record count, and the data-format word.
__device__ __forceinline__ u32x4 make_rsrc(const void* p, int bytes) {
  const unsigned long a = (unsigned long)p;
  return u32x4{(unsigned)a, (unsigned)(a >> 32) & 0xffffu, (unsigned)bytes, 0x00020000u};
}

// 16 bytes per lane from a buffer into LDS (lane l -> dst + 16 l).  A byte
// offset voff + soff at or past the buffer's size (negative voff included,
// read as unsigned) yields zeros; soff must be wave-uniform.  Issued from inline assembly so that the
// compiler does not see an LDS write: it cannot tell the ring slots apart
// and would otherwise wait for every load in flight before the next LDS
// read, which serialises the ring.  The kernels order their rings
// themselves (wait_vmcnt / wait_stages, then ring_barrier).  M0 holds the
// LDS destination only while the load issues and is restored after it; the
// wait state the hardware needs between writing M0 and a load that reads it
// is in the block, since the compiler's hazard checks do not look inside.
__device__ __forceinline__ void dma16(u32x4 rsrc, __attribute__((address_space(3))) void* dst,
                                      int voff, int soff) {
  const unsigned m = __builtin_amdgcn_readfirstlane((unsigned)(unsigned long)dst);
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"          // the load reads M0: one wait state after writing it
      "buffer_load_dwordx4 %2, %3, %4 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(m), "v"(voff), "s"(rsrc), "s"(__builtin_amdgcn_readfirstlane(soff))
      : "memory");
}

// Workgroup barrier of a DMA ring: s_barrier, plus a compiler fence so that
// no LDS read of the stage just waited for is moved above it.
__device__ __forceinline__ void ring_barrier() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace
}  // namespace tgpk
