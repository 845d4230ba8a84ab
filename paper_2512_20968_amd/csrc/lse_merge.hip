// Online-softmax reducer over k partial results (Section 2.2; the reducer of
// the reduce-scatter in Algorithm 2), gfx950.
//
// A pure streaming kernel: every partial O element is read once and every
// output element written once, so it is bound by HBM bandwidth.  Each
// (row, head) item of head_dim values is handled by head_dim/8 lanes, each
// owning one 8-element slice (a 16-byte load for bf16 partials, two for
// float32).  Consecutive lanes cover consecutive addresses and consecutive
// items are consecutive heads of a row, so loads and stores are fully
// coalesced.  Each lane first folds the item's k LSE values (max, then
// sum of exp) in registers, then streams the k slices with loads issued
// several parts ahead of their use.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mesh_attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;
constexpr int UNROLL = 8;  // partial slices in flight per lane

template <bool IN_F32>
__device__ __forceinline__ f32x8 load8(const void* base, int64_t off) {
  f32x8 r;
  if constexpr (IN_F32) {
    const f32x4* p = reinterpret_cast<const f32x4*>(
        static_cast<const float*>(base) + off);
    const f32x4 a = __builtin_nontemporal_load(p);
    const f32x4 b = __builtin_nontemporal_load(p + 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r[i] = a[i];
      r[4 + i] = b[i];
    }
  } else {
    const bf16x8 a = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(
        static_cast<const __bf16*>(base) + off));
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = static_cast<float>(a[i]);
  }
  return r;
}

template <bool IN_F32, bool OUT_F32>
__global__ __launch_bounds__(NT) void lse_merge_kernel(MergeParams p) {
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr float kLn2 = 0.69314718055994531f;
  const int lpi = p.head_dim / 8;  // lanes per (row, head) item
  const int64_t n_items = p.rows * p.heads;
  const int64_t stride = int64_t{gridDim.x} * NT;
  for (int64_t gid = int64_t{blockIdx.x} * NT + threadIdx.x;
       gid < n_items * lpi; gid += stride) {
    const int64_t item = gid / lpi;
    const int sub = static_cast<int>(gid - item * lpi);
    const int64_t row = item / p.heads;
    const int h = static_cast<int>(item - row * p.heads);

    // lse_parts[kp][h][row]
    const float* lp = p.lse_parts + int64_t{h} * p.rows + row;
    const int64_t lstride = int64_t{p.heads} * p.rows;
    float mx = -INFINITY;
    for (int kp = 0; kp < p.k_parts; ++kp) mx = fmaxf(mx, lp[kp * lstride]);

    f32x8 acc;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    float lse = -INFINITY;
    if (mx != -INFINITY) {
      float s = 0.f;
      for (int kp = 0; kp < p.k_parts; ++kp)
        s += __builtin_amdgcn_exp2f((lp[kp * lstride] - mx) * kLog2e);
      lse = mx + __builtin_amdgcn_logf(s) * kLn2;
      // o_parts[kp][row][h][d]
      const int64_t ostride = p.rows * p.heads * p.head_dim;
      const int64_t off0 = item * p.head_dim + sub * 8;
      int kp = 0;
      for (; kp + UNROLL <= p.k_parts; kp += UNROLL) {
        f32x8 x[UNROLL];
        float w[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          x[u] = load8<IN_F32>(p.o_parts, (kp + u) * ostride + off0);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          w[u] = __builtin_amdgcn_exp2f((lp[(kp + u) * lstride] - lse) * kLog2e);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] = fmaf(w[u], x[u][i], acc[i]);
      }
      for (; kp < p.k_parts; ++kp) {
        const f32x8 x = load8<IN_F32>(p.o_parts, kp * ostride + off0);
        const float w =
            __builtin_amdgcn_exp2f((lp[kp * lstride] - lse) * kLog2e);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(w, x[i], acc[i]);
      }
    }
    const int64_t oo = item * p.head_dim + sub * 8;
    if constexpr (OUT_F32) {
      f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(p.o_out) + oo);
      f32x4 a, b;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = acc[i];
        b[i] = acc[4 + i];
      }
      __builtin_nontemporal_store(a, dst);
      __builtin_nontemporal_store(b, dst + 1);
    } else {
      bf16x8 o;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = static_cast<__bf16>(acc[i]);
      __builtin_nontemporal_store(
          o, reinterpret_cast<bf16x8*>(static_cast<__bf16*>(p.o_out) + oo));
    }
    if (sub == 0) p.lse_out[int64_t{h} * p.rows + row] = lse;
  }
}

template <bool IF, bool OF>
hipError_t launch(const MergeParams& p, hipStream_t stream) {
  const int64_t threads = p.rows * p.heads * (p.head_dim / 8);
  int64_t blocks = (threads + NT - 1) / NT;
  // Enough workgroups to fill 256 CUs several times over; the kernel loops.
  const int64_t cap = 256 * 64;
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL((lse_merge_kernel<IF, OF>), dim3(static_cast<int>(blocks)),
                     dim3(NT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lse_merge(const MergeParams& p, bool in_f32, bool out_f32,
                            hipStream_t stream) {
  if (in_f32) return out_f32 ? launch<true, true>(p, stream)
                             : launch<true, false>(p, stream);
  return out_f32 ? launch<false, true>(p, stream)
                 : launch<false, false>(p, stream);
}

}  // namespace mesh_attn
