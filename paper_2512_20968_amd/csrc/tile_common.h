// Device helpers shared by the tile kernels (gfx950, wave64).
//
// MFMA conventions (v_mfma_f32_32x32x16_bf16): lane l of a wave holds, for
// the A operand, row l % 32 and the 8 k-values of group l / 32; for B,
// column l % 32 and the same k group; the 16 accumulator registers of lane l
// hold column l % 32 and rows 8*(r/4) + 4*(l/32) + r%4.
//
// Tiles staged in LDS are 64 rows of one head.  A row-major tile is
// [64][D] bf16 with its 16-byte chunks XOR-swizzled by row; a transposed
// tile is [D][64] bf16 with chunks swizzled by dim.  Both swizzles make the
// MFMA operand reads (16 lanes reading 16 consecutive rows at one logical
// chunk) hit distinct banks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mesh_attn {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // four waves
constexpr int kTileRows = 64;  // rows of a staged tile

// Item slot of this workgroup in an item order of n_items (XCD lane x at
// slots j * 8 + x): slot blockIdx.x below queued_static_slots(n_items), else
// the next remaining item of this workgroup's XCD lane, else of another lane;
// -1 if every lane is taken.  A plain read of a lane's counter skips a taken
// lane without an atomic.  s_slot is one int of LDS; every thread of the
// workgroup must call this (it ends at a barrier when it takes the queue).
__device__ __forceinline__ int queued_slot(int n_items, int32_t* queue,
                                           int* s_slot) {
  constexpr int kLanes = kNumXcd;
  const int n_static = static_cast<int>(queued_static_slots(n_items));
  const int slot = static_cast<int>(blockIdx.x);
  if (slot < n_static) return slot;
  if (threadIdx.x == 0) {
    const int x = static_cast<int>(blockIdx.x % kLanes);
    const int j0 = n_static / kLanes;  // positions taken statically
    int got = -1;
    for (int t = 0; t < kLanes && got < 0; ++t) {
      const int y = (x + t) % kLanes;
      const int len = (n_items - y + kLanes - 1) / kLanes - j0;
      if (__hip_atomic_load(&queue[y], __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_AGENT) >= len)
        continue;
      const int c = atomicAdd(&queue[y], 1);
      if (c < len) got = (j0 + c) * kLanes + y;
    }
    *s_slot = got;
  }
  __syncthreads();
  return __builtin_amdgcn_readfirstlane(*s_slot);
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b,
                                         const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_fast(float x) {
  return __builtin_amdgcn_exp2f(x);
}

// Read-only kernel data (work lists) through the constant address space: the
// compiler may then always use scalar loads for uniform addresses, whatever
// else the kernel does.
template <typename T>
__device__ __forceinline__ T load_const(const T* p, int64_t i) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef const __attribute__((address_space(4))) T* cptr;
  T v;
  __builtin_memcpy(&v, (cptr)(p) + i, sizeof(T));
  return v;
#else
  return p[i];
#endif
}

// Workgroup barrier for LDS-only hand-offs: waits for this wave's own LDS
// (and scalar) accesses, then s_barrier.  Unlike __syncthreads() it does not
// drain outstanding global loads, so loads streaming into LDS may stay in
// flight across it; the code that issued them waits (vmcnt) before the
// barrier that publishes their buffer.  The empty asm statements keep the
// compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Make the compiler wait here for the loads that produced `v` (an empty asm
// that reads the registers).  Used before a loop so the wait analysis at the
// loop header sees these registers as complete; unlike an s_waitcnt
// intrinsic it has no memory effect, so uniform loads stay scalar.
template <typename T>
__device__ __forceinline__ void wait_for(const T& v) {
  asm volatile("" ::"v"(v));
}

// max(x, x of the lane 32 apart): v_permlane32_swap exchanges the two
// half-waves of a register pair in the VALU, without an LDS round trip.
__device__ __forceinline__ float max_with_other_half(float x) {
  const unsigned u = __float_as_uint(x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}

__device__ __forceinline__ void zero(f32x16& a) {
#pragma unroll
  for (int i = 0; i < 16; ++i) a[i] = 0.f;
}

// Order in which the 32 rows of an operand tile are fed to the MFMA: bits 2
// and 3 of the row index swapped.  With it, accumulator register r of lane
// half h holds row 16*(r/8) + 8*h + r%8, i.e. every lane half owns runs of 8
// consecutive rows -- the k-contiguous layout the next MFMA's operand needs.
__device__ __forceinline__ int mfma_row_perm(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Row of the permuted 32-row tile held by accumulator register r, lane half h.
__device__ __forceinline__ int acc_row(int r, int h) {
  return (r >> 3) * 16 + h * 8 + (r & 7);
}

// Operand fragments of 32 rows held in registers for a whole workgroup
// item: lane (l % 32, half h) holds row l % 32, dims 16*kk + 8*h .. +7.
template <int D>
__device__ __forceinline__ void load_frags(bf16x8 (&f)[D / 16],
                                           const uint16_t* __restrict__ g,
                                           int64_t row, int heads, int head,
                                           int h) {
  const uint16_t* p = g + (row * heads + head) * D + h * 8;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk)
    f[kk] = *reinterpret_cast<const bf16x8*>(p + kk * 16);
}

// ---------------------------------------------------------------------------
// Raw buffer loads: the 128-bit descriptor holds a scalar base address and a
// byte range; the per-lane offset is a 32-bit VGPR and the per-load offset a
// scalar, so loads of a tile need no per-load vector address arithmetic, and
// reads past the range return zero instead of touching memory.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // Word 3 = 0x00020000: 32-bit data format, the gfx9-family setting.
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           static_cast<int>(bytes), 0x00020000);
}

// Direct global -> LDS load of 16 bytes per lane (buffer_load_dwordx4 ... lds):
// lane i of the wave writes LDS bytes [lds + 16 i, lds + 16 i + 16) with the
// 16 bytes at buffer offset voff + soff.  `lds` must be wave-uniform.  The
// load is counted by vmcnt; the data is in LDS once vmcnt has drained.
__device__ __forceinline__ void buffer_load16_lds(rsrc_t r, void* lds,
                                                  uint32_t voff,
                                                  uint32_t soff) {
  typedef __attribute__((address_space(3))) void lds_void;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(lds), 16,
                                           static_cast<int>(voff),
                                           static_cast<int>(soff), 0, 0);
}

// s_waitcnt vmcnt(0): this wave's vector-memory loads (including those
// written straight into LDS) have completed.
__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

// ---------------------------------------------------------------------------
// LDS transpose read (gfx950 ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane s supplies the address of 4 consecutive bf16 values x[s][0..3];
// lane l receives x[4e + l/4][l%4] as its element e.  With lane s pointing at
// row (r0 + s/4), columns (c0 + 4*(s%4)) .. +3 of a row-major tile, lane l
// receives column c0 + l of rows r0 .. r0+3: a transposed 4x16 block.
// ---------------------------------------------------------------------------
typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ s16x4 lds_read_tr16(const void* lds_addr) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)(lds_addr));
}

__device__ __forceinline__ bf16x8 join_bf16(const s16x4& lo, const s16x4& hi) {
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

}  // namespace dev
}  // namespace mesh_attn
