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
// Layout choices (64-wide wavefronts, v_mfma_f32_32x32x16_bf16):
//  * Scores are computed transposed, S^T = K Q^T (A = K rows from LDS,
//    B = Q columns held in registers for the whole item), so each lane owns
//    one query row and the row max / row sum are in-lane reductions plus one
//    exchange between the two half-waves.
//  * K rows are fed to the MFMA in an order that swaps bits 2 and 3 of the
//    row index, which leaves P^T in the accumulators already laid out as the
//    k-contiguous B operand of O^T += V^T P^T.
//  * K and V tiles are stored row-major in LDS with padded rows (272 B and
//    320 B for d = 128), conflict-free for the reads below and affine in the
//    loop indices, so every LDS read is one base register plus an immediate.
//  * The V^T operand comes straight from the row-major V tile through the
//    LDS transpose read (ds_read_b64_tr_b16), two per MFMA.
//  * Global loads are raw buffer loads: scalar base per KV block, one
//    per-lane offset register, scalar per-load offsets.  The next block's
//    loads are issued before the current block's MFMAs; K/V tiles are double
//    buffered in LDS with one barrier per block.
//  * Softmax runs in the log2 domain with the scale folded into one FMA
//    before v_exp_f32.  The running max is exact (the largest probability of
//    a row is exactly 1, which keeps its bf16 rounding error-free), but the
//    O rescale is skipped when no row of the wave has a new max -- a
//    wave-uniform branch taken on a small fraction of blocks once the max has
//    settled.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "tile_common.h"

namespace mesh_attn {
namespace {

using namespace dev;

constexpr int BM = kFwdBM;  // 128
constexpr int BN = kFwdBN;  // 64
constexpr int NT = kThreads;

template <int D>
struct FwdLayout {
  static constexpr int KSTR = 2 * D + 16;   // K tile row stride, bytes
  static constexpr int VSTR = 2 * D + 64;   // V tile row stride, bytes
  static constexpr int KBYTES = BN * KSTR;
  static constexpr int VBYTES = BN * VSTR;
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int SMEM = 2 * STAGE;
  static constexpr int CPR = D / 8;         // 16-byte chunks per row
  static constexpr int RSTEP = NT / CPR;    // rows per load pass
  static constexpr int NLD = BN / RSTEP;    // loads per thread per tensor
};

// Row order of a 32-key tile as fed to the MFMA: swap bits 2 and 3.
__device__ __forceinline__ int key_perm(int r) { return mfma_row_perm(r); }

template <int D, bool OUT_F32>
__global__ __launch_bounds__(NT, 2) void tile_fwd_kernel(FwdParams p) {
  using L = FwdLayout<D>;
  extern __shared__ __align__(16) char smem[];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  const int2 item = load_const(p.order, blockIdx.x);
  if (item.x < 0) return;
  const int qblk = item.x;
  const int h = item.y;
  const int hk = h / p.group;
  const int run_b = load_const(p.qblk_ptr, qblk);
  const int run_e = load_const(p.qblk_ptr, qblk + 1);

  const int64_t q_row = int64_t{qblk} * BM + wave * 32 + li;
  const int q_in_blk = wave * 32 + li;

  // Q columns for the B operand: lane half lh holds dims 16kk + 8lh .. +7.
  bf16x8 qf[D / 16];
  load_frags<D>(qf, p.q, q_row, p.hq, h, lh);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc) zero(oacc[cc]);
  float m = -INFINITY;  // reference max of scaled scores (log2 units)
  float l = 0.f;        // this lane's share of the row sum

  if (run_b < run_e) {
    // Per-thread byte offsets that stay fixed for the whole item.
    const int c = tid % L::CPR;
    const int r0 = tid / L::CPR;
    const int64_t row_elems = int64_t{p.hkv} * D;  // elements per KV row
    const uint32_t g_voff = static_cast<uint32_t>((r0 * row_elems + c * 8) * 2);
    const uint32_t g_step = static_cast<uint32_t>(L::RSTEP * row_elems * 2);
    const uint32_t blk_bytes = static_cast<uint32_t>(BN * row_elems * 2);
    const int k_w = r0 * L::KSTR + c * 16;
    const int v_w = L::KBYTES + r0 * L::VSTR + c * 16;
    // K operand read: row kt*32 + perm(li), 16 bytes at dims 16kk + 8lh.
    const int k_r = key_perm(li) * L::KSTR + lh * 16;
    // V^T operand read (transpose): 16-lane group g, lane s: row
    // 8*(g>>1) + s/4 (+16ss, +4 for the second half), dims
    // 16*(g&1) + 4*(s%4) (+32cc).
    const int grp = lane >> 4, s16 = lane & 15;
    const int v_r = L::KBYTES + (8 * (grp >> 1) + (s16 >> 2)) * L::VSTR +
                    (16 * (grp & 1) + 4 * (s16 & 3)) * 2;

    u32x4 kreg[L::NLD], vreg[L::NLD];
    auto gload = [&](int64_t blk) {
      const int64_t e0 = (blk * BN * p.hkv + hk) * D;
      const rsrc_t rk = make_rsrc(p.k + e0, blk_bytes);
      const rsrc_t rv = make_rsrc(p.v + e0, blk_bytes);
#pragma unroll
      for (int i = 0; i < L::NLD; ++i) {
        kreg[i] = buffer_load16(rk, g_voff, i * g_step);
        vreg[i] = buffer_load16(rv, g_voff, i * g_step);
      }
    };
    auto lstore = [&](int stage) {
      char* base = smem + stage * L::STAGE;
#pragma unroll
      for (int i = 0; i < L::NLD; ++i) {
        *reinterpret_cast<u32x4*>(base + k_w + i * L::RSTEP * L::KSTR) =
            kreg[i];
        *reinterpret_cast<u32x4*>(base + v_w + i * L::RSTEP * L::VSTR) =
            vreg[i];
      }
    };

    int r = run_b, off = 0;
    DevRun cur = load_const(p.runs, r);
    gload(cur.blk0);
    lstore(0);
    // Complete the Q fragment loads here, so the loop never waits on them
    // behind the next block's prefetch.
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) wait_for(qf[kk]);
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
        nxt = load_const(p.runs, nr);
        gload(int64_t{nxt.blk0} + noff);
      }

      const char* sb = smem + stage * L::STAGE;

      // S^T = K Q^T for two 32-key tiles.
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        zero(s[kt]);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(
              sb + k_r + kt * 32 * L::KSTR + kk * 32);
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
          for (int i = 0; i < 16; ++i)
            if (kt * 32 + acc_row(i, lh) > lim) s[kt][i] = -INFINITY;
      }

      // Online softmax (log2 domain), rescaling only on a large max jump.
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kt][i]);
      mx = max_with_other_half(mx) * p.scale_log2;
      const bool need = mx > m;
      if (__builtin_amdgcn_ballot_w64(need)) {
        const float m_new = need ? mx : m;
        const float alpha = exp2_fast(m - m_new);  // 1 if unchanged, 0 from -inf
        l *= alpha;
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[cc][i] *= alpha;
        m = m_new;
      }
      const float m_use = (m == -INFINITY) ? 0.f : m;
      bf16x8 pb[4];
      float rs[4];
#pragma unroll
      for (int ss = 0; ss < 4; ++ss) {
        float e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          e8[e] = exp2_fast(
              fmaf(s[ss >> 1][(ss & 1) * 8 + e], p.scale_log2, -m_use));
          pb[ss][e] = static_cast<__bf16>(e8[e]);
        }
        rs[ss] = ((e8[0] + e8[1]) + (e8[2] + e8[3])) +
                 ((e8[4] + e8[5]) + (e8[6] + e8[7]));
      }
      l += (rs[0] + rs[1]) + (rs[2] + rs[3]);

      // O^T += V^T P^T; key step ss covers keys 16ss + 8lh + 0..7.
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
#pragma unroll
        for (int ss = 0; ss < 4; ++ss) {
          const char* a0 = sb + v_r + ss * 16 * L::VSTR + cc * 64;
          const bf16x8 a =
              join_bf16(lds_read_tr16(a0), lds_read_tr16(a0 + 4 * L::VSTR));
          oacc[cc] = mfma32(a, pb[ss], oacc[cc]);
        }
      }

      if (!has_next) break;
      lstore(stage ^ 1);
      __syncthreads();
      stage ^= 1;
      r = nr;
      off = noff;
      cur = nxt;
    }
  }

  // Epilogue: O = acc / l, LSE = (m + log2 l) * ln 2.
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
      f32x4 x;
#pragma unroll
      for (int t = 0; t < 4; ++t) x[t] = oacc[cc][4 * g + t] * inv;
      if constexpr (OUT_F32) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(p.o) + obase + dim) = x;
      } else {
        bf16x4 val;
#pragma unroll
        for (int t = 0; t < 4; ++t) val[t] = static_cast<__bf16>(x[t]);
        *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(p.o) + obase + dim) =
            val;
      }
    }
}

template <int D, bool F32>
hipError_t launch(const FwdParams& p, int grid, hipStream_t stream) {
  const size_t smem = FwdLayout<D>::SMEM;
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
