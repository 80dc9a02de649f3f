// Building blocks of the MFMA contraction kernels: direct global->LDS loads,
// pipeline waits and barriers, compile-time loops, and the two ways an MFMA
// operand fragment is read from LDS.
#pragma once

#include <type_traits>

#include "pfc_device.h"

namespace pfc {

typedef __attribute__((address_space(3))) void* lds_void_t;
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t* lds_v4i16_t;

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds_base + 16 * l (the base must be wave-uniform).
__device__ __forceinline__ void dma16(const void* g, void* lds_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void_t)lds_base, 16, 0, 0);
}

// s_waitcnt vmcnt(N), N < 64; LDS / scalar (lgkm) and export counters not waited on.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without a memory fence: each wave has already waited for
// its own loads into the stage about to be read; the compiler barrier keeps
// LDS accesses from being moved across it.
__device__ __forceinline__ void stage_barrier() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// vmcnt(N) and lgkmcnt(0) in one wait: the wave's direct-to-LDS loads older
// than the last N and all of its LDS writes are complete (needed before a
// barrier after which other waves read what this wave wrote to LDS).
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// s_waitcnt lgkmcnt(0): this wave's LDS reads and writes are complete (vector
// memory counter not waited on).
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// 32-bit LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// LDS accesses issued as inline assembly.  Inside the pipelined loops every
// LDS access goes through these: the compiler would otherwise hoist plain
// LDS loads above the stage barrier, and make each plain LDS access wait for
// every pending direct-to-LDS load (it cannot tell the stages apart).  It
// neither orders these against pending direct-to-LDS loads (the pipeline's
// own waits do) nor waits for their results: lgkm_wait() below must separate
// a read from the first use of its destination.
template <int OFF>
__device__ __forceinline__ void ds_read_tr_b64(u32x2_t& dst, uint32_t addr) {
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(OFF));
}
template <int OFF>
__device__ __forceinline__ void ds_read_128(u32x4_t& dst, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(OFF));
}

template <int OFF>
__device__ __forceinline__ void ds_read_32(uint32_t& dst, uint32_t addr) {
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(OFF));
}
template <int OFF>
__device__ __forceinline__ void ds_write_128(uint32_t addr, const u32x4_t& v) {
  asm volatile("ds_write_b128 %0, %1 offset:%2" ::"v"(addr), "v"(v), "i"(OFF) : "memory");
}

template <typename T>
__device__ __forceinline__ void pin_reg(T& r) {
  asm volatile("" : "+v"(r));
}
template <typename T, int N>
__device__ __forceinline__ void pin_reg(T (&r)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) pin_reg(r[i]);
}

// s_waitcnt lgkmcnt(N) that also redefines the fragment registers it is
// given, so no use of them can be scheduled before the wait.
template <int N, typename... T>
__device__ __forceinline__ void lgkm_wait(T&... regs) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N));
  (pin_reg(regs), ...);
}


template <int C, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (C < N) {
    f(std::integral_constant<int, C>{});
    static_for<C + 1, N>(f);
  }
}

// Operand fragment of v_mfma_f32_32x32x16 (lane l: 8 consecutive k at
// row / column mn = mn0 + l % 32, k = k0 + 8 (l / 32) + 0..7) from an LDS tile
// stored MN-major: element (k, mn) at base[k * LD + mn].  Two transposing
// reads (ds_read_b64_tr_b16): within each 16-lane group, lane i's element e
// is element i % 4 of the 8 bytes addressed by lane 4 e + i / 4, so lane
// 4 e + q points at row (k + e), columns 4 q .. 4 q + 3 of its 16-column half.
// With LD * 2 bytes = 32 mod 128, the four rows of a group hit distinct banks.
template <int LD>
__device__ __forceinline__ uint4 frag_mn_major(const uint16_t* base, int k0, int mn0, int lane) {
  const int g = lane >> 4, src = lane & 15;
  const int krow = k0 + 8 * (g >> 1) + (src >> 2);
  const int col = mn0 + 16 * (g & 1) + 4 * (src & 3);
  const uint16_t* p = base + krow * LD + col;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t)p);
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t)(p + 4 * LD));
  uint4 r;
  __builtin_memcpy(&r.x, &lo, 8);
  __builtin_memcpy(&r.z, &hi, 8);
  return r;
}

// Operand fragment from an LDS tile stored K-major in rows of 32 elements
// (64 B): element (mn, k) at base[mn * 32 + (((k / 8) ^ ((mn >> 2) & 3)) * 8) + k % 8].
// The XOR spreads sixteen consecutive rows of one 16-byte read over all 64
// banks.
__device__ __forceinline__ uint4 frag_k_major32(const uint16_t* base, int kk, int mn0, int lane) {
  const int mn = mn0 + (lane & 31);
  const int pos = ((2 * kk + (lane >> 5)) ^ ((lane >> 2) & 3)) * 8;
  return *reinterpret_cast<const uint4*>(base + mn * 32 + pos);
}

// Element offset of 16-byte chunk `chunk` (0..3) of row `row` in a K-major
// 32-element-row tile (the layout frag_k_major32 reads).
__device__ __forceinline__ int k_major32_offset(int row, int chunk) {
  return row * 32 + ((chunk ^ ((row >> 2) & 3)) * 8);
}

}  // namespace pfc
