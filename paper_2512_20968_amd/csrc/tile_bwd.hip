// Tile attention backward for gfx950 (MI355X): the per-pair gradient loop of
// Algorithm 3, summed over the tile.  Deterministic: every output element is
// owned by exactly one thread, no atomics.
//
// Three launches on the caller's stream:
//  1. delta:  D_i = <dO_i, O_i> for every (row, query head), float32.
//  2. dK/dV:  one workgroup per (KV block of 128 keys, KV head), 4 waves x 32
//     keys.  It walks the KV block's runs of Q blocks (KV-major work list) for
//     every query head of the GQA group, in 64-row stages, and keeps dK, dV
//     in registers:  S = Q K^T,  P = exp(s S - LSE),  dP = dO V^T,
//     dS = P (dP - D),  dV += P^T dO,  dK += s dS^T Q.
//  3. dQ:     one workgroup per (Q block of 128 rows, query head), 4 waves x
//     32 rows, walking the Q-major runs of KV blocks in 64-key stages:
//     S^T = K Q^T,  dP^T = V dO^T,  dS^T = P^T (dP^T - D),  dQ^T += s K^T dS^T.
//
// As in the forward, the operand that feeds a score tile is read in the
// bit-2/3-swapped row order, so the probability / dS accumulators are already
// k-contiguous operands of the next MFMA.  Tiles needed with k along rows
// (Q, dO in dK/dV; K in dQ) are also stored transposed in LDS.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "tile_common.h"

namespace mesh_attn {
namespace {

using namespace dev;

constexpr int NT = kThreads;
constexpr int BQ = kBwdBM;    // 128
constexpr int BK = kBwdBN;    // 128
constexpr int SUB = kTileRows;  // 64 rows per LDS stage
constexpr float kLog2e = 1.4426950408889634f;

static_assert(BQ == 2 * SUB && BK == 2 * SUB, "two stages per block");

// ---------------------------------------------------------------------------
// 1. delta
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(NT) void bwd_delta_kernel(BwdParams p) {
  constexpr int LPI = D / 8;  // lanes per (row, head)
  const int64_t gid = int64_t{blockIdx.x} * NT + threadIdx.x;
  const int64_t item = gid / LPI;  // row * hq + h
  const int sub = static_cast<int>(gid % LPI);
  const bool valid = item < p.rows_q * p.hq;
  float s = 0.f;
  if (valid) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(p.o + item * D + sub * 8);
    const bf16x8 b =
        *reinterpret_cast<const bf16x8*>(p.d_o + item * D + sub * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      s = fmaf(static_cast<float>(a[i]), static_cast<float>(b[i]), s);
  }
#pragma unroll
  for (int off = LPI / 2; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (valid && sub == 0) {
    const int64_t row = item / p.hq;
    const int h = static_cast<int>(item - row * p.hq);
    p.delta[int64_t{h} * p.rows_q + row] = s;
  }
}

// Log2-domain LSE used to form P; a row without any visible key (LSE = -inf)
// maps to +inf so that its probabilities are exp2(-inf) = 0.
__device__ __forceinline__ float lse_log2(float lse) {
  return lse == -INFINITY ? INFINITY : lse * kLog2e;
}

// ---------------------------------------------------------------------------
// 2. dK / dV
// ---------------------------------------------------------------------------
template <int D>
struct DkdvStage {
  static constexpr int TILE = SUB * D;          // bf16 elements per tile
  static constexpr int FLOATS = 2 * SUB;        // lse2 + delta
  static constexpr int ELEMS = 4 * TILE + 2 * FLOATS;  // in uint16 units
};

template <int D>
__global__ __launch_bounds__(NT, 1) void bwd_dkdv_kernel(BwdParams p) {
  extern __shared__ __align__(16) uint16_t smem[];
  using S = DkdvStage<D>;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  const int2 item = p.kvorder[blockIdx.x];
  if (item.x < 0) return;
  const int kvblk = item.x;
  const int hk = item.y;
  const int run_b = p.kvblk_ptr[kvblk];
  const int run_e = p.kvblk_ptr[kvblk + 1];
  const int k_in_blk = wave * 32 + li;
  const int64_t kv_row = int64_t{kvblk} * BK + k_in_blk;

  bf16x8 kf[D / 16], vf[D / 16];
  load_frags<D>(kf, p.k, kv_row, p.hkv, hk, lh);
  load_frags<D>(vf, p.v, kv_row, p.hkv, hk, lh);

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc) {
    zero(dk[cc]);
    zero(dv[cc]);
  }

  if (run_b < run_e) {
    RowTile<D> tq, tdo;
    float lse_v = 0.f, dlt_v = 0.f;
    // Cursor over (query head of the group, run, block in run, stage).
    int g = 0, r = run_b, off = 0, s = 0;
    DevRun cur = p.kvruns[r];

    auto load = [&](const DevRun& rn, int gg, int of, int st) {
      const int h = hk * p.group + gg;
      const int64_t row0 = int64_t{rn.blk0 + of} * BQ + st * SUB;
      tq.load(p.q, row0, p.hq, h, tid);
      tdo.load(p.d_o, row0, p.hq, h, tid);
      if (tid < SUB) {
        lse_v = lse_log2(p.lse[int64_t{h} * p.rows_q + row0 + tid]);
        dlt_v = p.delta[int64_t{h} * p.rows_q + row0 + tid];
      }
    };
    auto store = [&](int stage) {
      uint16_t* base = smem + stage * S::ELEMS;
      tq.store_rows(base, tid);
      tq.store_cols(base + S::TILE, tid);
      tdo.store_rows(base + 2 * S::TILE, tid);
      tdo.store_cols(base + 3 * S::TILE, tid);
      if (tid < SUB) {
        float* f = reinterpret_cast<float*>(base + 4 * S::TILE);
        f[tid] = lse_v;
        f[SUB + tid] = dlt_v;
      }
    };

    load(cur, g, off, s);
    store(0);
    __syncthreads();
    int stage = 0;
    while (true) {
      int ng = g, nr = r, noff = off, ns = s + 1;
      if (ns == 2) {
        ns = 0;
        if (++noff == cur.nblk) {
          noff = 0;
          if (++nr == run_e) {
            nr = run_b;
            ++ng;
          }
        }
      }
      const bool has_next = ng < p.group;
      DevRun nxt = cur;
      if (has_next) {
        nxt = p.kvruns[nr];
        load(nxt, ng, noff, ns);
      }

      const uint16_t* base = smem + stage * S::ELEMS;
      const uint16_t* sq = base;
      const uint16_t* sqt = base + S::TILE;
      const uint16_t* sdo = base + 2 * S::TILE;
      const uint16_t* sdot = base + 3 * S::TILE;
      const float* slse = reinterpret_cast<const float*>(base + 4 * S::TILE);
      const float* sdlt = slse + SUB;

      // S = Q K^T and dP = dO V^T for two 32-row query tiles; lane li owns
      // key k_in_blk, register i owns query 32*qt + acc_row(i, lh).
      f32x16 sc[2], dp[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        zero(sc[qt]);
        zero(dp[qt]);
        const int row = qt * 32 + mfma_row_perm(li);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          sc[qt] = mfma32(read_rows<D>(sq, row, kk, lh), kf[kk], sc[qt]);
          dp[qt] = mfma32(read_rows<D>(sdo, row, kk, lh), vf[kk], dp[qt]);
        }
      }
      if (cur.cls == 1) {
        // key k of the block is hidden from query q of the run iff
        // k - q > delta + (offset of this stage in the run).
        const int lim = k_in_blk - cur.delta - off * BQ - s * SUB;
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (qt * 32 + acc_row(i, lh) < lim) sc[qt][i] = -INFINITY;
      }
      bf16x8 pb[4], dsb[4];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int q0 = qt * 32 + hh * 16 + lh * 8;
          const f32x4 l0 = *reinterpret_cast<const f32x4*>(slse + q0);
          const f32x4 l1 = *reinterpret_cast<const f32x4*>(slse + q0 + 4);
          const f32x4 d0 = *reinterpret_cast<const f32x4*>(sdlt + q0);
          const f32x4 d1 = *reinterpret_cast<const f32x4*>(sdlt + q0 + 4);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int i = hh * 8 + e;
            const float lq = e < 4 ? l0[e] : l1[e - 4];
            const float dq = e < 4 ? d0[e] : d1[e - 4];
            const float pv = exp2_fast(fmaf(sc[qt][i], p.scale_log2, -lq));
            pb[qt * 2 + hh][e] = static_cast<__bf16>(pv);
            dsb[qt * 2 + hh][e] = static_cast<__bf16>(pv * (dp[qt][i] - dq));
          }
        }
      // dV += P^T dO,  dK += dS^T Q   (scale applied at the end)
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const int dim = cc * 32 + li;
#pragma unroll
        for (int ss = 0; ss < 4; ++ss) {
          dv[cc] = mfma32(pb[ss], read_cols(sdot, dim, ss, lh), dv[cc]);
          dk[cc] = mfma32(dsb[ss], read_cols(sqt, dim, ss, lh), dk[cc]);
        }
      }

      if (!has_next) break;
      store(stage ^ 1);
      __syncthreads();
      stage ^= 1;
      g = ng;
      r = nr;
      off = noff;
      s = ns;
      cur = nxt;
    }
  }

  // Accumulator register i of chunk cc: key row 8*(i/4) + 4*lh + i%4 of the
  // wave, dim 32*cc + li.
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t row =
          int64_t{kvblk} * BK + wave * 32 + 8 * (i >> 2) + 4 * lh + (i & 3);
      const int64_t idx = (row * p.hkv + hk) * D + cc * 32 + li;
      float kv = dk[cc][i] * p.scale;
      float vv = dv[cc][i];
      if (p.accumulate) {
        kv += p.dk[idx];
        vv += p.dv[idx];
      }
      p.dk[idx] = kv;
      p.dv[idx] = vv;
    }
}

// ---------------------------------------------------------------------------
// 3. dQ
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(NT, 1) void bwd_dq_kernel(BwdParams p) {
  extern __shared__ __align__(16) uint16_t smem[];
  constexpr int TILE = SUB * D;
  constexpr int ELEMS = 3 * TILE;  // K rows, K cols, V rows
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  const int2 item = p.qorder[blockIdx.x];
  if (item.x < 0) return;
  const int qblk = item.x;
  const int h = item.y;
  const int hk = h / p.group;
  const int run_b = p.qblk_ptr[qblk];
  const int run_e = p.qblk_ptr[qblk + 1];
  const int q_in_blk = wave * 32 + li;
  const int64_t q_row = int64_t{qblk} * BQ + q_in_blk;

  bf16x8 qf[D / 16], dof[D / 16];
  load_frags<D>(qf, p.q, q_row, p.hq, h, lh);
  load_frags<D>(dof, p.d_o, q_row, p.hq, h, lh);
  const float lse2 = lse_log2(p.lse[int64_t{h} * p.rows_q + q_row]);
  const float dlt = p.delta[int64_t{h} * p.rows_q + q_row];

  f32x16 acc[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc) zero(acc[cc]);

  if (run_b < run_e) {
    RowTile<D> tk, tv;
    int r = run_b, off = 0, s = 0;
    DevRun cur = p.qruns[r];
    auto load = [&](const DevRun& rn, int of, int st) {
      const int64_t row0 = int64_t{rn.blk0 + of} * BK + st * SUB;
      tk.load(p.k, row0, p.hkv, hk, tid);
      tv.load(p.v, row0, p.hkv, hk, tid);
    };
    auto store = [&](int stage) {
      uint16_t* base = smem + stage * ELEMS;
      tk.store_rows(base, tid);
      tk.store_cols(base + TILE, tid);
      tv.store_rows(base + 2 * TILE, tid);
    };
    load(cur, off, s);
    store(0);
    __syncthreads();
    int stage = 0;
    while (true) {
      int nr = r, noff = off, ns = s + 1;
      if (ns == 2) {
        ns = 0;
        if (++noff == cur.nblk) {
          noff = 0;
          ++nr;
        }
      }
      const bool has_next = nr < run_e;
      DevRun nxt = cur;
      if (has_next) {
        nxt = p.qruns[nr];
        load(nxt, noff, ns);
      }

      const uint16_t* base = smem + stage * ELEMS;
      const uint16_t* sk = base;
      const uint16_t* skt = base + TILE;
      const uint16_t* sv = base + 2 * TILE;

      // S^T = K Q^T, dP^T = V dO^T: lane li owns query q_in_blk, register i
      // owns key 32*kt + acc_row(i, lh) of the stage.
      f32x16 sc[2], dp[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        zero(sc[kt]);
        zero(dp[kt]);
        const int row = kt * 32 + mfma_row_perm(li);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          sc[kt] = mfma32(read_rows<D>(sk, row, kk, lh), qf[kk], sc[kt]);
          dp[kt] = mfma32(read_rows<D>(sv, row, kk, lh), dof[kk], dp[kt]);
        }
      }
      if (cur.cls == 1) {
        const int lim = cur.delta - off * BK - s * SUB + q_in_blk;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (kt * 32 + acc_row(i, lh) > lim) sc[kt][i] = -INFINITY;
      }
      bf16x8 dsb[4];
#pragma unroll
      for (int ss = 0; ss < 4; ++ss)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int kt = ss >> 1, i = (ss & 1) * 8 + e;
          const float pv = exp2_fast(fmaf(sc[kt][i], p.scale_log2, -lse2));
          dsb[ss][e] = static_cast<__bf16>(pv * (dp[kt][i] - dlt));
        }
      // dQ^T += K^T dS^T
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const int dim = cc * 32 + li;
#pragma unroll
        for (int ss = 0; ss < 4; ++ss)
          acc[cc] = mfma32(read_cols(skt, dim, ss, lh), dsb[ss], acc[cc]);
      }

      if (!has_next) break;
      store(stage ^ 1);
      __syncthreads();
      stage ^= 1;
      r = nr;
      off = noff;
      s = ns;
      cur = nxt;
    }
  }

  // Register 4g+t of chunk cc holds dim 32cc + 8g + 4lh + t of query q_row.
  float* dst = p.dq + (q_row * p.hq + h) * D;
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int dim = cc * 32 + g * 8 + lh * 4;
      f32x4 val;
#pragma unroll
      for (int t = 0; t < 4; ++t) val[t] = acc[cc][4 * g + t] * p.scale;
      f32x4* out = reinterpret_cast<f32x4*>(dst + dim);
      if (p.accumulate) val += *out;
      *out = val;
    }
}

template <typename K>
hipError_t set_smem(K kern, size_t bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             static_cast<int>(bytes));
}

template <int D>
hipError_t launch(const BwdParams& p, int grid_q, int grid_kv,
                  hipStream_t stream) {
  const size_t smem_kv = 2 * DkdvStage<D>::ELEMS * sizeof(uint16_t);
  const size_t smem_q = 2 * 3 * SUB * D * sizeof(uint16_t);
  static bool attr_done = false;  // benign race: idempotent attribute set
  if (!attr_done) {
    hipError_t e = set_smem(bwd_dkdv_kernel<D>, smem_kv);
    if (e == hipSuccess) e = set_smem(bwd_dq_kernel<D>, smem_q);
    if (e != hipSuccess) return e;
    attr_done = true;
  }
  const int64_t delta_threads = p.rows_q * p.hq * (D / 8);
  const int delta_grid = static_cast<int>((delta_threads + NT - 1) / NT);
  hipLaunchKernelGGL(bwd_delta_kernel<D>, dim3(delta_grid), dim3(NT), 0,
                     stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (grid_kv > 0) {
    hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3(grid_kv), dim3(NT), smem_kv,
                       stream, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (grid_q > 0) {
    hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3(grid_q), dim3(NT), smem_q,
                       stream, p);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t launch_tile_bwd(const BwdParams& p, int head_dim, int grid_q,
                           int grid_kv, hipStream_t stream) {
  if (head_dim == 128) return launch<128>(p, grid_q, grid_kv, stream);
  if (head_dim == 64) return launch<64>(p, grid_q, grid_kv, stream);
  return hipErrorInvalidValue;
}

}  // namespace mesh_attn
