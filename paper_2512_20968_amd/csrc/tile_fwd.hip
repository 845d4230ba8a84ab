// Tile attention forward for gfx950 (MI355X).
//
// One workgroup computes one (Q block, query head) item: BM = 128 query rows,
// four waves of 32 rows each.  It walks the Q block's runs of KV blocks
// (BN = 64 keys each) from the work list, so EMPTY blocks are never touched
// and only PARTIAL runs evaluate the causal mask (a wave-uniform branch).  For
// every KV block it forms scores, updates the online softmax of each row and
// accumulates P V -- the per-pair computation of Algorithm 2 with the
// online-softmax reducer applied inside the kernel (Section 2.2).
//
// Layout choices (all for 64-wide wavefronts and the 32x32x16 bf16 MFMA):
//  * Scores are computed transposed, S^T = K Q^T (A = K rows from LDS,
//    B = Q columns held in registers for the whole item), so each lane owns
//    one query row (lane % 32) and the row max / row sum are in-lane
//    reductions plus one exchange between the two half-waves.
//  * The K rows of a 32-key tile are fed to the MFMA in an order that swaps
//    bits 2 and 3 of the row index.  The S^T accumulator then holds, for lane
//    half h, keys 8h..8h+7 (+16) in consecutive registers -- exactly the
//    k-contiguous B operand that O^T += V^T P^T needs, so P goes from the
//    score accumulator into the PV MFMA with a convert and no shuffles.
//  * V is staged into LDS transposed ([dim][key]) through a 4x8 register
//    transpose, so the V^T A operand is one 16-byte LDS read per MFMA.
//  * K and V^T tiles are double buffered in LDS with XOR-swizzled 16-byte
//    chunks (conflict-free reads); the next block's global loads (coalesced
//    16-byte) are issued before the current block's MFMAs.
//  * Softmax runs in the log2 domain with the scale folded into one FMA
//    before v_exp_f32.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mesh_attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = kFwdBM;  // 128
constexpr int BN = kFwdBN;  // 64
constexpr int NT = 256;     // 4 waves

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b,
                                         const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

// Row order of a 32-key tile as fed to the MFMA: swap bits 2 and 3.
__device__ __forceinline__ int key_perm(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// 16-byte chunk swizzles.  K tile: rows of D bf16; V^T tile: rows of BN bf16.
template <int D>
__device__ __forceinline__ int k_chunk(int row, int chunk) {
  return chunk ^ (D == 128 ? (row & 15) : (row & 7));
}
__device__ __forceinline__ int vt_chunk(int dim, int chunk) {
  return chunk ^ ((dim ^ (dim >> 3)) & 7);
}

__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {
  return (a & 0xffffu) | (b << 16);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {
  return (a >> 16) | (b & 0xffff0000u);
}

template <int D>
struct Stage {
  static constexpr int CPR = D / 8;        // 16-byte chunks per K row
  static constexpr int RSTEP = NT / CPR;   // K rows covered per load pass
  static constexpr int NLD = BN / RSTEP;   // loads per thread per tensor
  u32x4 k[NLD];
  u32x4 v[NLD];

  // Global -> registers for KV block `blk` (rows blk*BN ..) of KV head hk.
  __device__ __forceinline__ void load(const uint16_t* __restrict__ kg,
                                       const uint16_t* __restrict__ vg,
                                       int64_t blk, int hkv, int hk, int tid) {
    const int c = tid % CPR;
    const int r0 = tid / CPR;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int64_t row = blk * BN + r0 + i * RSTEP;
      k[i] = *reinterpret_cast<const u32x4*>(kg + (row * hkv + hk) * D + c * 8);
    }
    // V: this thread takes NLD consecutive keys of one 8-dim slice.
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int64_t row = blk * BN + r0 * NLD + j;
      v[j] = *reinterpret_cast<const u32x4*>(vg + (row * hkv + hk) * D + c * 8);
    }
  }

  // Registers -> LDS: K as [key][dim], V transposed as [dim][key].
  __device__ __forceinline__ void store(uint16_t* sk, uint16_t* svt, int tid) {
    const int c = tid % CPR;
    const int r0 = tid / CPR;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int row = r0 + i * RSTEP;
      *reinterpret_cast<u32x4*>(sk + row * D + k_chunk<D>(row, c) * 8) = k[i];
    }
    const int key0 = r0 * NLD;  // first of this thread's NLD keys
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int dim = c * 8 + e;
      const int w = e >> 1;
      uint16_t* rowp = svt + dim * BN;
      if constexpr (NLD == 4) {
        u32x2 val;
        if (e & 1) {
          val[0] = pack_hi(v[0][w], v[1][w]);
          val[1] = pack_hi(v[2][w], v[3][w]);
        } else {
          val[0] = pack_lo(v[0][w], v[1][w]);
          val[1] = pack_lo(v[2][w], v[3][w]);
        }
        const int chunk = key0 >> 3, sub = key0 & 7;
        *reinterpret_cast<u32x2*>(rowp + vt_chunk(dim, chunk) * 8 + sub) = val;
      } else {
        static_assert(NLD == 2, "unsupported head_dim");
        const uint32_t val = (e & 1) ? pack_hi(v[0][w], v[1][w])
                                     : pack_lo(v[0][w], v[1][w]);
        const int chunk = key0 >> 3, sub = key0 & 7;
        *reinterpret_cast<uint32_t*>(rowp + vt_chunk(dim, chunk) * 8 + sub) =
            val;
      }
    }
  }
};

template <int D, bool OUT_F32>
__global__ __launch_bounds__(NT, 2) void tile_fwd_kernel(FwdParams p) {
  extern __shared__ __align__(16) uint16_t smem[];
  uint16_t* s_k = smem;                 // [2][BN * D]
  uint16_t* s_vt = smem + 2 * BN * D;   // [2][D * BN]

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  const int2 item = p.order[blockIdx.x];
  if (item.x < 0) return;
  const int qblk = item.x;
  const int h = item.y;
  const int hk = h / p.group;
  const int run_b = p.qblk_ptr[qblk];
  const int run_e = p.qblk_ptr[qblk + 1];

  const int64_t q_row = int64_t{qblk} * BM + wave * 32 + li;
  const int q_in_blk = wave * 32 + li;

  // Q columns for the B operand: lane half lh holds dims 16kk + 8lh .. +7.
  bf16x8 qf[D / 16];
  {
    const uint16_t* qp = p.q + (q_row * p.hq + h) * D + lh * 8;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      qf[kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 16);
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[cc][r] = 0.f;
  float m = -INFINITY;  // running max of scaled scores (log2 units)
  float l = 0.f;        // this lane's share of the running row sum

  if (run_b < run_e) {
    Stage<D> st;
    int r = run_b, off = 0;
    DevRun cur = p.runs[r];
    st.load(p.k, p.v, cur.blk0, p.hkv, hk, tid);
    st.store(s_k, s_vt, tid);
    __syncthreads();
    int stage = 0;
    while (true) {
      // Next block of the flattened run list.
      int nr = r, noff = off + 1;
      if (noff == cur.nblk) {
        nr = r + 1;
        noff = 0;
      }
      const bool has_next = nr < run_e;
      DevRun nxt = cur;
      if (has_next) {
        nxt = p.runs[nr];
        st.load(p.k, p.v, int64_t{nxt.blk0} + noff, p.hkv, hk, tid);
      }

      const uint16_t* sk = s_k + stage * BN * D;
      const uint16_t* svt = s_vt + stage * D * BN;

      // S^T = K Q^T for two 32-key tiles.
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s[kt][i] = 0.f;
        const int row = kt * 32 + key_perm(li);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(
              sk + row * D + k_chunk<D>(row, 2 * kk + lh) * 8);
          s[kt] = mfma32(a, qf[kk], s[kt]);
        }
      }

      // Causal mask on PARTIAL runs: key j of the run is hidden from query i
      // of the block iff j - i > delta.
      if (cur.cls == 1) {
        const int lim = cur.delta - off * BN + q_in_blk;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = kt * 32 + (i >> 3) * 16 + lh * 8 + (i & 7);
            if (key > lim) s[kt][i] = -INFINITY;
          }
      }

      // Online softmax (log2 domain).
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kt][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m, mx * p.scale_log2);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = fast_exp2(m - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float e = fast_exp2(fmaf(s[kt][i], p.scale_log2, -m_use));
          s[kt][i] = e;
          rs += e;
        }
      l = l * alpha + rs;
      m = m_new;
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[cc][i] *= alpha;

      // P^T as B operand: key step ss covers keys 16ss + 8lh + 0..7.
      bf16x8 pb[4];
#pragma unroll
      for (int ss = 0; ss < 4; ++ss)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pb[ss][e] = static_cast<__bf16>(s[ss >> 1][(ss & 1) * 8 + e]);

      // O^T += V^T P^T.
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const int dim = cc * 32 + li;
#pragma unroll
        for (int ss = 0; ss < 4; ++ss) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(
              svt + dim * BN + vt_chunk(dim, 2 * ss + lh) * 8);
          oacc[cc] = mfma32(a, pb[ss], oacc[cc]);
        }
      }

      if (!has_next) break;
      st.store(s_k + (stage ^ 1) * BN * D, s_vt + (stage ^ 1) * D * BN, tid);
      __syncthreads();
      stage ^= 1;
      r = nr;
      off = noff;
      cur = nxt;
    }
  }

  // Epilogue: O = acc / l, LSE = ln(sum) = (m + log2 l) * ln 2.
  const float lt = l + __shfl_xor(l, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (lh == 0) {
    const float lse = lt > 0.f ? (m + __builtin_amdgcn_logf(lt)) *
                                     0.69314718055994531f
                               : -INFINITY;
    p.lse[int64_t{h} * p.rows_q + q_row] = lse;
  }
  // O^T accumulator: register 4g+t of chunk cc holds dim 32cc + 8g + 4lh + t.
  const int64_t obase = (q_row * p.hq + h) * D;
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int dim = cc * 32 + g * 8 + lh * 4;
      const float x0 = oacc[cc][4 * g + 0] * inv;
      const float x1 = oacc[cc][4 * g + 1] * inv;
      const float x2 = oacc[cc][4 * g + 2] * inv;
      const float x3 = oacc[cc][4 * g + 3] * inv;
      if constexpr (OUT_F32) {
        float4 val = make_float4(x0, x1, x2, x3);
        *reinterpret_cast<float4*>(static_cast<float*>(p.o) + obase + dim) =
            val;
      } else {
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        bf16x4 val;
        val[0] = static_cast<__bf16>(x0);
        val[1] = static_cast<__bf16>(x1);
        val[2] = static_cast<__bf16>(x2);
        val[3] = static_cast<__bf16>(x3);
        *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(p.o) + obase + dim) =
            val;
      }
    }
}

template <int D, bool F32>
hipError_t launch(const FwdParams& p, int grid, hipStream_t stream) {
  const size_t smem = 2 * (2 * BN * D) * sizeof(uint16_t);
  auto kern = tile_fwd_kernel<D, F32>;
  static bool attr_done = false;  // benign race: idempotent attribute set
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(kern),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    if (e != hipSuccess) return e;
    attr_done = true;
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(NT), smem, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tile_fwd(const FwdParams& p, int head_dim, bool out_f32,
                           int grid, hipStream_t stream) {
  if (head_dim == 128)
    return out_f32 ? launch<128, true>(p, grid, stream)
                   : launch<128, false>(p, grid, stream);
  if (head_dim == 64)
    return out_f32 ? launch<64, true>(p, grid, stream)
                   : launch<64, false>(p, grid, stream);
  return hipErrorInvalidValue;
}

}  // namespace mesh_attn
