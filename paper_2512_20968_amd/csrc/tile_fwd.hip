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
  static constexpr int ROWB = 2 * D;         // bytes per K/V row
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;       // rows per 1 KB wave load
  static constexpr int RPW = BN / 4;         // rows each wave loads
  static constexpr int NLI = RPW / RPI;      // wave loads per tile
  static constexpr int TILE = BN * ROWB;     // bytes per K or V tile
  static constexpr int SMEM = 4 * TILE;      // K0, K1, V0, V1
  // XOR swizzles of the 16-byte chunk index, chosen so that the MFMA operand
  // reads below hit distinct LDS banks.
  __device__ static int kswz(int row) {
    return D == 128 ? (row & 15) : ((row >> 1) & 7);
  }
  __device__ static int vswz(int row) {
    return D == 128 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
  }
};

// Position in the flattened list of KV blocks of one Q block's runs.
struct Cursor {
  DevRun run;
  int r, off;
  bool valid;
  __device__ int64_t blk() const { return int64_t{run.blk0} + off; }
};

__device__ __forceinline__ Cursor first_block(const FwdParams& p, int r) {
  Cursor c;
  c.run = load_const(p.runs, r);
  c.r = r;
  c.off = 0;
  c.valid = true;
  return c;
}

__device__ __forceinline__ Cursor next_block(const FwdParams& p, Cursor c,
                                             int run_e) {
  if (!c.valid) return c;
  if (++c.off == c.run.nblk) {
    c.off = 0;
    if (++c.r < run_e)
      c.run = load_const(p.runs, c.r);
    else
      c.valid = false;
  }
  return c;
}

// Row order of a 32-key tile as fed to the MFMA: swap bits 2 and 3.
__device__ __forceinline__ int key_perm(int r) { return mfma_row_perm(r); }

template <int D, bool OUT_F32>
__global__ __launch_bounds__(NT, 2) void tile_fwd_kernel(FwdParams p) {
  using L = FwdLayout<D>;
  extern __shared__ __align__(16) char smem[];

  const int tid = threadIdx.x;
  // Wave index as a scalar (the compiler cannot infer that tid >> 6 is
  // uniform across the wave).
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
    // Direct global -> LDS staging.  Wave `wave` fills rows
    // wave*RPW .. +RPW of a tile with NLI loads of 1 KB; lane i of load j
    // takes row wave*RPW + j*RPI + i/CPR and writes physical chunk i%CPR,
    // i.e. the logical chunk (i%CPR) ^ swizzle(row).
    const int64_t row_elems = int64_t{p.hkv} * D;  // elements per KV row
    const uint32_t row_bytes_g = static_cast<uint32_t>(row_elems * 2);
    const uint32_t blk_bytes = static_cast<uint32_t>(BN * row_elems * 2);
    uint32_t kvo[L::NLI], vvo[L::NLI];
#pragma unroll
    for (int j = 0; j < L::NLI; ++j) {
      const int row = wave * L::RPW + j * L::RPI + lane / L::CPR;
      const int phys = lane % L::CPR;
      kvo[j] = (lane / L::CPR) * row_bytes_g + ((phys ^ L::kswz(row)) * 16);
      vvo[j] = (lane / L::CPR) * row_bytes_g + ((phys ^ L::vswz(row)) * 16);
    }
    auto rsrc_of = [&](const uint16_t* base, int64_t blk) {
      return make_rsrc(base + (blk * BN * p.hkv + hk) * D, blk_bytes);
    };
    // LDS: K buffers 0, 1 then V buffers 0, 1.
    auto load_k = [&](int64_t blk, int buf) {
      const rsrc_t rk = rsrc_of(p.k, blk);
#pragma unroll
      for (int j = 0; j < L::NLI; ++j) {
        const int row0 = wave * L::RPW + j * L::RPI;
        buffer_load16_lds(rk, smem + buf * L::TILE + row0 * L::ROWB, kvo[j],
                          row0 * row_bytes_g);
      }
    };
    auto load_v = [&](int64_t blk, int buf) {
      const rsrc_t rv = rsrc_of(p.v, blk);
#pragma unroll
      for (int j = 0; j < L::NLI; ++j) {
        const int row0 = wave * L::RPW + j * L::RPI;
        buffer_load16_lds(rv, smem + (2 + buf) * L::TILE + row0 * L::ROWB,
                          vvo[j], row0 * row_bytes_g);
      }
    };
    // K operand read: row kt*32 + perm(li), dims 16kk + 8lh (logical chunk
    // 2kk + lh); the swizzle of such a row does not depend on kt.
    int kra[D / 16];
    {
      const int prow = key_perm(li);
      const int ks = L::kswz(prow);
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
        kra[kk] = prow * L::ROWB + (((2 * kk + lh) ^ ks) * 16);
    }
    // V^T operand read (transpose): 16-lane group g, lane s reads row
    // 8*(g>>1) + s/4 (+16ss, +4 for the second half) at dims
    // 32cc + 16*(g&1) + 4*(s%4) .. +3; the swizzle of those rows depends on
    // s only.
    int vra[D / 32];
    {
      const int grp = lane >> 4, s16 = lane & 15;
      const int vrow = 8 * (grp >> 1) + (s16 >> 2);
      const int vs = L::vswz(vrow);
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const int c16 = 4 * cc + 2 * (grp & 1) + ((s16 & 3) >> 1);
        vra[cc] = 2 * L::TILE + vrow * L::ROWB + ((c16 ^ vs) * 16) +
                  8 * (s16 & 1);
      }
    }

    // S^T = K Q^T of one 64-key block from K buffer `buf`.
    auto scores = [&](f32x16 (&sc)[2], int buf) {
      const char* kb = smem + buf * L::TILE;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        zero(sc[kt]);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
          sc[kt] = mfma32(*reinterpret_cast<const bf16x8*>(
                              kb + kra[kk] + kt * 32 * L::ROWB),
                          qf[kk], sc[kt]);
      }
    };
    // Causal mask of a PARTIAL block: key j of the run is hidden from query
    // i of the Q block iff j - i > delta.
    auto apply_mask = [&](f32x16 (&sc)[2], const Cursor& cu) {
      const int lim = cu.run.delta - cu.off * BN + q_in_blk;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (kt * 32 + acc_row(i, lh) > lim) sc[kt][i] = -INFINITY;
    };
    // Scaled row max (both half-waves hold the same query row).
    auto row_max = [&](const f32x16 (&sc)[2]) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[kt][i]);
      return max_with_other_half(mx) * p.scale_log2;
    };

    // Pipeline: iteration n computes P of block n and O += V(n)^T P(n)^T,
    // and meanwhile the scores of block n+1.  K runs one block ahead of V:
    // during iteration n, K buffer (n+1)&1 holds K(n+1) and V buffer n&1
    // holds V(n); K(n+2) and V(n+1) stream straight into the other buffers.
    Cursor cur = first_block(p, run_b);   // block n
    Cursor nx = next_block(p, cur, run_e);  // block n+1
    Cursor nn = next_block(p, nx, run_e);   // block n+2
    load_k(cur.blk(), 0);
    load_v(cur.blk(), 0);
    if (nx.valid) load_k(nx.blk(), 1);
    // Complete the Q fragment loads and the first tiles here, so the loop
    // never waits on them behind the next block's prefetch.
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) wait_for(qf[kk]);
    wait_vmem();
    __syncthreads();

    f32x16 s_cur[2];
    scores(s_cur, 0);
    if (cur.run.cls == 1) apply_mask(s_cur, cur);
    m = row_max(s_cur);  // first block: nothing to rescale yet
    // Every wave has read K(0) before iteration 0 refills K buffer 0.
    __syncthreads();
    int ph = 0;  // n & 1
    while (true) {
      // K(n+2) -> K buffer n&1 (K(n) was consumed last iteration) and
      // V(n+1) -> V buffer (n+1)&1 (V(n-1) likewise), straight into LDS.
      if (nn.valid) load_k(nn.blk(), ph);
      if (nx.valid) load_v(nx.blk(), ph ^ 1);

      // --- one scheduling region: no branches until the row max ---------
      // P(n) = exp2(s S(n) - m), row sums, bf16 B operand ...
      const float m_use = (m == -INFINITY) ? 0.f : m;
      bf16x8 pb[4];
      float rs[4];
#pragma unroll
      for (int ss = 0; ss < 4; ++ss) {
        float e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          e8[e] = exp2_fast(
              fmaf(s_cur[ss >> 1][(ss & 1) * 8 + e], p.scale_log2, -m_use));
          pb[ss][e] = static_cast<__bf16>(e8[e]);
        }
        rs[ss] = ((e8[0] + e8[1]) + (e8[2] + e8[3])) +
                 ((e8[4] + e8[5]) + (e8[6] + e8[7]));
      }
      l += (rs[0] + rs[1]) + (rs[2] + rs[3]);
      // ... the scores of block n+1 (independent of the exponentials; after
      // the last block they read a stale buffer and are discarded) ...
      f32x16 s_nxt[2];
      scores(s_nxt, ph ^ 1);
      // ... then O^T += V(n)^T P(n)^T (key step ss: keys 16ss + 8lh + 0..7)
      const char* vb = smem + ph * L::TILE;
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
#pragma unroll
        for (int ss = 0; ss < 4; ++ss) {
          const char* a0 = vb + vra[cc] + ss * 16 * L::ROWB;
          const bf16x8 a =
              join_bf16(lds_read_tr16(a0), lds_read_tr16(a0 + 4 * L::ROWB));
          oacc[cc] = mfma32(a, pb[ss], oacc[cc]);
        }
      }
      // ... with the unmasked row max of block n+1 alongside.
      float mx = row_max(s_nxt);
      // --------------------------------------------------------------------
      if (!nx.valid) break;
      if (nx.run.cls == 1) {
        apply_mask(s_nxt, nx);
        mx = row_max(s_nxt);
      }

      // Running max with block n+1; rescale O and l only if some row of the
      // wave has a new max (exact max: a row's largest probability stays 1).
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

      wait_vmem();
      __syncthreads();
      s_cur[0] = s_nxt[0];
      s_cur[1] = s_nxt[1];
      cur = nx;
      nx = nn;
      nn = next_block(p, nn, run_e);
      ph ^= 1;
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
