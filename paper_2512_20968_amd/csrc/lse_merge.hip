// Online-softmax reducer over k partial results (Section 2.2; the reducer of
// the reduce-scatter in Algorithm 2), gfx950.
//
// A pure streaming kernel: every partial O element is read once and every
// output element written once, so it is bound by HBM bandwidth.  Each
// (row, head) item of head_dim values is handled by head_dim/8 lanes, each
// owning one 8-element slice (a 16-byte load for bf16 partials, two for
// float32).  Consecutive lanes cover consecutive addresses and consecutive
// items are consecutive heads of a row, so loads and stores are fully
// coalesced.  Each lane loads the slices and LSE values of a batch of
// partials at once (one round trip to memory per batch; a whole merge of up
// to 16 bf16 partials is one batch) and folds them into a running
// (max, sum of exp, weighted sum) reducer.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mesh_attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;

// 8 values of one partial slice, as loaded (16 bytes of bf16 or 32 bytes of
// float32), converted to float32 only when used.
template <bool IN_F32>
struct Slice;
template <>
struct Slice<false> {
  bf16x8 v;
  __device__ void load(const void* base, int64_t off) {
    v = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(
        static_cast<const __bf16*>(base) + off));
  }
  __device__ float at(int i) const { return static_cast<float>(v[i]); }
};
template <>
struct Slice<true> {
  f32x4 a, b;
  __device__ void load(const void* base, int64_t off) {
    const f32x4* p = reinterpret_cast<const f32x4*>(
        static_cast<const float*>(base) + off);
    a = __builtin_nontemporal_load(p);
    b = __builtin_nontemporal_load(p + 1);
  }
  __device__ float at(int i) const { return i < 4 ? a[i] : b[i - 4]; }
};

// B partials per batch: the slices and LSE values of a batch are loaded
// together (all loads issued before any is used), so a lane waits for one
// round trip to memory per batch.  The host picks the smallest B that covers
// k_parts (at most 16 for bf16 partials, 8 for float32).
template <bool IN_F32, bool OUT_F32, int B>
__global__ __launch_bounds__(NT) void lse_merge_kernel(MergeParams p) {
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr float kLn2 = 0.69314718055994531f;
  const int lpi = p.head_dim / 8;  // lanes per (row, head) item
  const int64_t n_items = p.rows * p.heads;
  const int64_t stride = int64_t{gridDim.x} * NT;
  const int64_t lstride = int64_t{p.heads} * p.rows;
  const int64_t ostride = p.rows * p.heads * p.head_dim;
  for (int64_t gid = int64_t{blockIdx.x} * NT + threadIdx.x;
       gid < n_items * lpi; gid += stride) {
    const int64_t item = gid / lpi;
    const int sub = static_cast<int>(gid - item * lpi);
    const int64_t row = item / p.heads;
    const int h = static_cast<int>(item - row * p.heads);
    // lse_parts[kp][h][row], o_parts[kp][row][h][d]
    const float* lp = p.lse_parts + int64_t{h} * p.rows + row;
    const int64_t off0 = item * p.head_dim + sub * 8;

    // Running reducer over the batches: M the largest LSE so far, S the sum
    // of exp(lse_k - M), acc the sum of exp(lse_k - M) O_k; at the end
    // lse = M + ln S and O = acc / S (Section 2.2's merge, two parts at a
    // time across batches).
    float M = -INFINITY, S = 0.f;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    for (int kb = 0; kb < p.k_parts; kb += B) {
      Slice<IN_F32> x[B];
      float lv[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int kp = min(kb + u, p.k_parts - 1);
        x[u].load(p.o_parts, kp * ostride + off0);
        lv[u] = lp[kp * lstride];
      }
      // Keep every load of the batch ahead of the first use (the scheduler
      // would otherwise sink each load to its use, one round trip each).
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (kb + u >= p.k_parts) lv[u] = -INFINITY;
      float mb = -INFINITY;
#pragma unroll
      for (int u = 0; u < B; ++u) mb = fmaxf(mb, lv[u]);
      const float mn = fmaxf(M, mb);
      const float mu = mn == -INFINITY ? 0.f : mn;  // no exp(-inf - -inf)
      const float r = __builtin_amdgcn_exp2f((M - mu) * kLog2e);
      S *= r;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] *= r;
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const float w = __builtin_amdgcn_exp2f((lv[u] - mu) * kLog2e);
        S += w;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(w, x[u].at(i), acc[i]);
      }
      M = mn;
    }
    const float lse =
        M == -INFINITY ? -INFINITY : M + __builtin_amdgcn_logf(S) * kLn2;
    const float inv = S > 0.f ? 1.f / S : 0.f;
    const int64_t oo = item * p.head_dim + sub * 8;
    if constexpr (OUT_F32) {
      f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(p.o_out) + oo);
      f32x4 a, b;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = acc[i] * inv;
        b[i] = acc[4 + i] * inv;
      }
      __builtin_nontemporal_store(a, dst);
      __builtin_nontemporal_store(b, dst + 1);
    } else {
      bf16x8 o;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = static_cast<__bf16>(acc[i] * inv);
      __builtin_nontemporal_store(
          o, reinterpret_cast<bf16x8*>(static_cast<__bf16*>(p.o_out) + oo));
    }
    if (sub == 0) p.lse_out[int64_t{h} * p.rows + row] = lse;
  }
}

template <bool IF, bool OF, int B>
hipError_t launch_b(const MergeParams& p, hipStream_t stream) {
  const int64_t threads = p.rows * p.heads * (p.head_dim / 8);
  int64_t blocks = (threads + NT - 1) / NT;
  // Enough workgroups to fill 256 CUs several times over; the kernel loops.
  const int64_t cap = 256 * 64;
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL((lse_merge_kernel<IF, OF, B>),
                     dim3(static_cast<int>(blocks)), dim3(NT), 0, stream, p);
  return hipGetLastError();
}

template <bool IF, bool OF>
hipError_t launch(const MergeParams& p, hipStream_t stream) {
  if (p.k_parts <= 2) return launch_b<IF, OF, 2>(p, stream);
  if (p.k_parts <= 4) return launch_b<IF, OF, 4>(p, stream);
  if (IF || p.k_parts <= 8) return launch_b<IF, OF, 8>(p, stream);
  return launch_b<IF, OF, 16>(p, stream);
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
