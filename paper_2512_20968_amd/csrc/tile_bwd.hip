// Tile attention backward for gfx950 (MI355X): the per-pair gradient loop of
// Algorithm 3, summed over the tile.  Deterministic: every output element is
// owned by exactly one thread, no atomics.
//
// Three launches on the caller's stream:
//  1. prep:   D_i = <dO_i, O_i> and LSE_i * log2(e) for every (row, query
//     head), float32 (a row without a visible key gets +inf, so that its
//     probabilities exp2(s S - LSE) are 0).
//  2. dK/dV:  one workgroup per (KV block of 128 keys, KV head), eight waves
//     in two roles over four 32-key groups.  It walks the KV block's runs of
//     Q blocks (KV-major work list) for every query head of the GQA group, in
//     64-row stages, and keeps dK, dV in registers.  The dV role computes
//     S = Q K^T,  P = exp(s S - LSE),  dV += P^T dO  and leaves P in LDS; the
//     dK role, one stage behind, computes  dP = dO V^T,  dS = P (dP - D),
//     dK += s dS^T Q.
//  3. dQ:     one workgroup per (Q block of 128 rows, query head), 4 waves x
//     32 rows (two workgroups per CU), walking the Q-major runs of KV blocks
//     in 64-key stages:
//     S^T = K Q^T,  dP^T = V dO^T,  dS^T = P^T (dP^T - D),  dQ^T += s K^T dS^T.
//
// The stage tiles (Q and dO, or K and V: 64 rows x d) stream from HBM
// straight into LDS (buffer loads with the LDS-destination form), one barrier
// per stage; dQ keeps two stages, dK/dV three (the dK role reads the stage
// before the one the dV role reads).  Each tile is stored once, row-major, and
// read two ways: as rows (the A operand of the score MFMAs, 16-byte reads) and
// transposed (the B operand of dV / dK, the A operand of dQ) through the
// gfx950 LDS transpose read ds_read_b64_tr_b16.  One XOR swizzle of the
// 16-byte chunks serves both access patterns without bank conflicts.  As in
// the forward, the operand that feeds a score tile is read in the
// bit-2/3-swapped row order, so the probability and dS accumulators are
// already the k-contiguous operands of the next MFMA.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "tile_common.h"

namespace mesh_attn {
namespace {

using namespace dev;

constexpr int NT = kThreads;    // 256: four waves
constexpr int BQ = kBwdBM;      // 128
constexpr int BK = kBwdBN;      // 128
constexpr int SUB = kTileRows;  // 64 rows per LDS stage
constexpr float kLog2e = 1.4426950408889634f;

static_assert(BQ == 2 * SUB && BK == 2 * SUB, "two stages per block");

// ---------------------------------------------------------------------------
// 1. prep: delta and the log2-domain LSE
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(NT) void bwd_prep_kernel(BwdParams p) {
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
    const int64_t idx = int64_t{h} * p.rows_q + row;
    p.delta[idx] = s;
    const float lse = p.lse[idx];
    p.lse2[idx] = lse == -INFINITY ? INFINITY : lse * kLog2e;
  }
}

// ---------------------------------------------------------------------------
// Stage tiles: 64 rows x D bf16, row-major, 16-byte chunks XOR-swizzled.
// ---------------------------------------------------------------------------
template <int D>
struct StageTile {
  static constexpr int ROWB = 2 * D;        // bytes per row
  static constexpr int CPR = D / 8;         // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;      // rows per 1 KB wave load
  static constexpr int BYTES = SUB * ROWB;
  // Physical chunk of logical chunk c in row r is c ^ swz(r).  Row reads (16
  // lanes: 16 distinct rows, one chunk) need swz to be one-to-one on the 16
  // rows of a group; transpose reads (32 lanes: 4 rows x 4 chunks, or for
  // d = 64 two row pairs sharing the banks) need the rows of a quad to land
  // in different 4-chunk groups.  Both hold for these maps.
  __device__ static int swz(int r) {
    return D == 128 ? 4 * (r & 3) + ((r >> 2) & 3)
                    : 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
  }
};

// Per-lane byte offsets into a stage tile.
template <int D>
struct TileAddr {
  using T = StageTile<D>;
  uint32_t load;   // load j: lane's global offset within the rows of load j
  int row;         // row reads: row perm(li) (+32 t), chunk 2kk + lh
  int tr0, tr1;    // transpose reads, first and second half (+4 rows)

  __device__ void init(int lane, int wg, uint32_t row_bytes_g) {
    const int li = lane & 31, lh = lane >> 5;
    {
      const int r = mfma_row_perm(li);
      row = r * T::ROWB + ((lh ^ T::swz(r)) * 16);
    }
    {
      // ds_read_b64_tr_b16: in 16-lane group g, lane s supplies row
      // 8*(g>>1) + s/4 (+4 for the second half, +16 per key step) at columns
      // 16*(g&1) + 4*(s%4) .. +3 of a 32-column chunk; lane l then holds
      // column l%32 of 8 consecutive rows (4 per half).
      const int g16 = lane >> 4, s16 = lane & 15;
      const int c16 = 2 * (g16 & 1) + ((s16 & 3) >> 1);
      const int r0 = 8 * (g16 >> 1) + (s16 >> 2);
      tr0 = r0 * T::ROWB + ((c16 ^ T::swz(r0)) * 16) + 8 * (s16 & 1);
      const int r1 = r0 + 4;
      tr1 = r1 * T::ROWB + ((c16 ^ T::swz(r1)) * 16) + 8 * (s16 & 1);
    }
    (void)wg;
    (void)row_bytes_g;
  }
};

// Rows [row0, row0 + 64) of one head of a [rows][heads][D] bf16 tensor into a
// stage tile, shared by NW waves: wave wg loads rows wg*64/NW .. +64/NW with
// 1 KB loads.  Lane i of load j fills row wg*64/NW + j*RPI + i/CPR, physical
// chunk i%CPR, i.e. logical chunk (i%CPR) ^ swz(row).
template <int D, int NW = 4>
__device__ __forceinline__ void load_stage_tile(const uint16_t* base,
                                                int64_t row0, int heads,
                                                int head, char* tile, int wg,
                                                int lane) {
  using T = StageTile<D>;
  constexpr int RPW = SUB / NW;
  static_assert(RPW % T::RPI == 0, "whole loads per wave");
  const uint32_t row_bytes_g = static_cast<uint32_t>(heads) * D * 2;
  const rsrc_t r = make_rsrc(base + (row0 * heads + head) * D,
                             static_cast<uint32_t>(SUB) * row_bytes_g);
  const int lrow = lane / T::CPR, lchunk = lane % T::CPR;
#pragma unroll
  for (int j = 0; j < RPW / T::RPI; ++j) {
    const int tr = wg * RPW + j * T::RPI;  // first row of this load
    const uint32_t voff =
        lrow * row_bytes_g + ((lchunk ^ T::swz(tr + lrow)) * 16);
    buffer_load16_lds(r, tile + tr * T::ROWB, voff, tr * row_bytes_g);
  }
}

// 64 floats (one stage's rows of one head) into LDS, by one wave.
__device__ __forceinline__ void load_stage_floats(const float* src,
                                                  float* dst, int lane) {
  typedef __attribute__((address_space(3))) void lds_void;
  const rsrc_t r = make_rsrc(src, SUB * 4);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst), 4, lane * 4,
                                           0, 0, 0);
}

// A operand: rows perm(li) + 32*t of a tile, dims 16*kk + 8*lh .. +7.
template <int D>
__device__ __forceinline__ bf16x8 read_row_op(const char* tile, int addr,
                                              int t, int kk) {
  return *reinterpret_cast<const bf16x8*>(
      tile + (addr ^ (32 * kk)) + t * 32 * StageTile<D>::ROWB);
}

// Transposed operand: column 32*cc + l%32 of rows 16*ss + 8*lh .. +7.
template <int D>
__device__ __forceinline__ bf16x8 read_tr_op(const char* tile,
                                             const TileAddr<D>& a, int cc,
                                             int ss) {
  const char* b = tile + ss * 16 * StageTile<D>::ROWB;
  return join_bf16(lds_read_tr16(b + (a.tr0 ^ (64 * cc))),
                   lds_read_tr16(b + (a.tr1 ^ (64 * cc))));
}

// ---------------------------------------------------------------------------
// 2. dK / dV
// ---------------------------------------------------------------------------
template <int D>
struct DkdvLayout {
  static constexpr int TILE = StageTile<D>::BYTES;
  static constexpr int STAGE = 2 * TILE + 2 * SUB * 4;  // Q, dO, lse2, delta
  static constexpr int NSTAGE = 3;
  // P of one stage, bf16, in the dV waves' register layout: [key wave 4]
  // [query tile 2][half 2][lane 64] x 16 bytes.
  static constexpr int PBUF = 4 * 2 * 2 * 64 * 16;
  static constexpr int SMEM = NSTAGE * STAGE + 2 * PBUF;
};

constexpr int NT_KV = 512;  // dK/dV: eight waves

// Eight waves in two roles over the same 128 keys (wave w: keys 32*(w%4) ..
// +32).  Waves 0-3 (dV role) compute S = Q K^T, P = exp(s S - LSE) and
// dV += P^T dO for stage t, and leave P (bf16) in LDS; waves 4-7 (dK role)
// follow one stage behind: dP = dO V^T, dS = P (dP - D) with the P of stage
// t-1 from LDS, dK += dS^T Q.  Four products per (key block, query stage)
// as in the algorithm, split evenly between the roles, and each wave needs
// one accumulator and its operand fragments, so it fits 256 registers and
// two waves share each SIMD.  Stage tiles are kept three deep (the dK role
// reads stage t-1 while the dV role reads t and loads t+1).
template <int D, int ROLE>
__device__ __forceinline__ void dkdv_role(const BwdParams& p, char* smem,
                                          int kvblk, int hk, int run_b,
                                          int run_e, int wave, int lane) {
  using L = DkdvLayout<D>;
  const int li = lane & 31;
  const int lh = lane >> 5;
  const int kw = wave & 3;
  const int k_in_blk = kw * 32 + li;
  const int64_t kv_row = int64_t{kvblk} * BK + k_in_blk;

  // dV role: K fragments (B operand of S); dK role: V fragments (of dP).
  bf16x8 frag[D / 16];
  load_frags<D>(frag, ROLE == 0 ? p.k : p.v, kv_row, p.hkv, hk, lh);

  f32x16 acc[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc) zero(acc[cc]);

  if (run_b < run_e) {
    TileAddr<D> ta;
    ta.init(lane, wave, 0);
    bf16x8* pbuf = reinterpret_cast<bf16x8*>(smem + L::NSTAGE * L::STAGE);
    // Stage cursor over (query head of the group, run, block in run, half).
    struct Cur {
      int g, r, off, s;
      DevRun run;
      bool valid;
    };
    auto advance = [&](Cur c) {
      if (!c.valid) return c;
      if (++c.s == 2) {
        c.s = 0;
        if (++c.off == c.run.nblk) {
          c.off = 0;
          if (++c.r == run_e) {
            c.r = run_b;
            ++c.g;
          }
          c.run = load_const(p.kvruns, c.r);
        }
      }
      c.valid = c.g < p.group;
      return c;
    };
    auto issue = [&](const Cur& c, int buf) {
      char* base = smem + buf * L::STAGE;
      const int h = hk * p.group + c.g;
      const int64_t row0 = int64_t{c.run.blk0 + c.off} * BQ + c.s * SUB;
      // Only the dV waves load: a wave that issues direct-to-LDS loads is
      // held up for a few hundred cycles per stage, and the dK role is the
      // longer of the two (its products read P from LDS after the dV role
      // wrote it), so the loads go where there is slack (measured: dK/dV
      // 4-5 % faster than eight loading waves).
      if constexpr (ROLE == 0) {
        load_stage_tile<D, 4>(p.q, row0, p.hq, h, base, kw, lane);
        load_stage_tile<D, 4>(p.d_o, row0, p.hq, h, base + L::TILE, kw, lane);
        float* f = reinterpret_cast<float*>(base + 2 * L::TILE);
        if (kw == 0) load_stage_floats(p.lse2 + int64_t{h} * p.rows_q + row0,
                                       f, lane);
        if (kw == 1) load_stage_floats(p.delta + int64_t{h} * p.rows_q + row0,
                                       f + SUB, lane);
      }
    };

    // Stages: every query head of the group x every block of the runs x 2.
    int nstage = 0;
    for (int r = run_b; r < run_e; ++r) nstage += load_const(p.kvruns, r).nblk;
    nstage *= 2 * p.group;
    // Iterations t = 0 .. nstage: loads of stage t+1; the dV role computes
    // stage t (t < nstage), the dK role stage t-1 (t >= 1).  Every iteration
    // but the last ends with a barrier, the same count in both roles.  Stage
    // j lives in buffer j % 3 (its previous occupant, stage j-3, was last
    // read by the dK role in iteration j-2) and its P in P buffer j % 2.
    Cur lc{0, run_b, 0, 0, load_const(p.kvruns, run_b), true};  // next load
    Cur cc_ = lc;  // stage this wave computes next
    issue(lc, 0);
    lc = advance(lc);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) wait_for(frag[kk]);
    wait_vmem();
    __syncthreads();
    int lbuf = 1;   // buffer of the stage loaded next
    int cbuf = 0;   // buffer of the stage computed next
    int pb_i = 0;   // P buffer of that stage
    for (int t = 0; t <= nstage; ++t) {
      if (t + 1 < nstage) {
        issue(lc, lbuf);
        lc = advance(lc);
        lbuf = lbuf == L::NSTAGE - 1 ? 0 : lbuf + 1;
      }
      const bool work = ROLE == 0 ? t < nstage : t >= 1;
      if (work) {
        const char* base = smem + cbuf * L::STAGE;
        const char* sq = base;
        const char* sdo = base + L::TILE;
        const float* slse =
            reinterpret_cast<const float*>(base + 2 * L::TILE);
        const float* sdlt = slse + SUB;
        const int lim =
            k_in_blk - cc_.run.delta - cc_.off * BQ - cc_.s * SUB;
        bf16x8* pst = pbuf + pb_i * (L::PBUF / 16) + kw * 256;
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          __builtin_amdgcn_sched_barrier(0);
          // dV role: S = Q K^T; dK role: dP = dO V^T.  Lane li owns key
          // k_in_blk, register i owns query 32*qt + acc_row(i, lh).
          f32x16 x;
          zero(x);
          const char* at = ROLE == 0 ? sq : sdo;
#pragma unroll
          for (int kk = 0; kk < D / 16; ++kk)
            x = mfma32(read_row_op<D>(at, ta.row, qt, kk), frag[kk], x);
          {
            constexpr int NM = D / 16;
            __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
            for (int i = 0; i < NM - 3; ++i) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
          }
          bf16x8 op[2];  // P (dV role) or dS (dK role), k-contiguous
          if constexpr (ROLE == 0) {
            if (cc_.run.cls == 1) {
              // key k of the block is hidden from query q of the run iff
              // k - q > delta + (offset of this stage in the run).
#pragma unroll
              for (int i = 0; i < 16; ++i)
                if (qt * 32 + acc_row(i, lh) < lim) x[i] = -INFINITY;
            }
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int q0 = qt * 32 + hh * 16 + lh * 8;
              const f32x4 l0 = *reinterpret_cast<const f32x4*>(slse + q0);
              const f32x4 l1 = *reinterpret_cast<const f32x4*>(slse + q0 + 4);
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float lq = e < 4 ? l0[e] : l1[e - 4];
                op[hh][e] = static_cast<__bf16>(
                    exp2_fast(fmaf(x[hh * 8 + e], p.scale_log2, -lq)));
              }
              pst[(qt * 2 + hh) * 64 + lane] = op[hh];
            }
          } else {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int q0 = qt * 32 + hh * 16 + lh * 8;
              const f32x4 d0 = *reinterpret_cast<const f32x4*>(sdlt + q0);
              const f32x4 d1 = *reinterpret_cast<const f32x4*>(sdlt + q0 + 4);
              const bf16x8 pv = pst[(qt * 2 + hh) * 64 + lane];
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float dq = e < 4 ? d0[e] : d1[e - 4];
                op[hh][e] = static_cast<__bf16>(static_cast<float>(pv[e]) *
                                                (x[hh * 8 + e] - dq));
              }
            }
          }
          // dV += P^T dO or dK += dS^T Q (scale at the end); the B operand
          // is read transposed from the dO or Q row tile.
          __builtin_amdgcn_sched_barrier(0);
          const char* bt = ROLE == 0 ? sdo : sq;
#pragma unroll
          for (int c = 0; c < D / 32; ++c)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
              acc[c] = mfma32(op[hh], read_tr_op<D>(bt, ta, c, 2 * qt + hh),
                              acc[c]);
          {
            constexpr int NM = D / 16;  // two transpose reads per MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
            for (int i = 0; i < NM - 3; ++i) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
          }
        }
      }
      if (work) {
        cc_ = advance(cc_);
        cbuf = cbuf == L::NSTAGE - 1 ? 0 : cbuf + 1;
        pb_i ^= 1;
      }
      if (t < nstage) {
        wait_vmem();
        lds_barrier();
      }
    }
  }

  // Accumulator register i of chunk c: key row 8*(i/4) + 4*lh + i%4 of the
  // wave's 32 keys, dim 32*c + li.
  // With accumulate, every old value is read before the first store, so the
  // loads are issued back to back instead of one read-modify-write at a time.
  float* out = ROLE == 0 ? p.dv : p.dk;
  const float sc_out = ROLE == 0 ? 1.f : p.scale;
  auto index = [&](int c, int i) {
    const int64_t row =
        int64_t{kvblk} * BK + kw * 32 + 8 * (i >> 2) + 4 * lh + (i & 3);
    return (row * p.hkv + hk) * D + c * 32 + li;
  };
  f32x16 prev[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) zero(prev[c]);
  if (p.accumulate) {
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) prev[c][i] = out[index(c, i)];
  }
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      out[index(c, i)] = fmaf(acc[c][i], sc_out, prev[c][i]);
}

template <int D>
__global__ __launch_bounds__(NT_KV, 1) void bwd_dkdv_kernel(BwdParams p) {
  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int slot = queued_slot(p.kv_items, p.kvqueue,
                               reinterpret_cast<int*>(smem + DkdvLayout<D>::SMEM));
  if (slot < 0) return;
  const int2 item = load_const(p.kvorder, slot);
  const int kvblk = item.x;
  const int hk = item.y;
  const int run_b = load_const(p.kvblk_ptr, kvblk);
  const int run_e = load_const(p.kvblk_ptr, kvblk + 1);
  if (wave < 4)
    dkdv_role<D, 0>(p, smem, kvblk, hk, run_b, run_e, wave, lane);
  else
    dkdv_role<D, 1>(p, smem, kvblk, hk, run_b, run_e, wave, lane);
}

// ---------------------------------------------------------------------------
// 3. dQ
// ---------------------------------------------------------------------------
template <int D>
struct DqLayout {
  static constexpr int TILE = StageTile<D>::BYTES;
  static constexpr int STAGE = 2 * TILE;  // K, V
  static constexpr int SMEM = 2 * STAGE;
};

template <int D>
__global__ __launch_bounds__(NT, 1) void bwd_dq_kernel(BwdParams p) {
  extern __shared__ __align__(16) char smem[];
  using L = DqLayout<D>;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  const int slot = queued_slot(p.q_items, p.qqueue,
                               reinterpret_cast<int*>(smem + L::SMEM));
  if (slot < 0) return;
  const int2 item = load_const(p.qorder, slot);
  const int qblk = item.x;
  const int h = item.y;
  const int hk = h / p.group;
  const int run_b = load_const(p.qblk_ptr, qblk);
  const int run_e = load_const(p.qblk_ptr, qblk + 1);
  const int q_in_blk = wave * 32 + li;
  const int64_t q_row = int64_t{qblk} * BQ + q_in_blk;

  bf16x8 qf[D / 16], dof[D / 16];
  load_frags<D>(qf, p.q, q_row, p.hq, h, lh);
  load_frags<D>(dof, p.d_o, q_row, p.hq, h, lh);
  const float lse2 = p.lse2[int64_t{h} * p.rows_q + q_row];
  const float dlt = p.delta[int64_t{h} * p.rows_q + q_row];

  f32x16 acc[D / 32];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc) zero(acc[cc]);

  if (run_b < run_e) {
    TileAddr<D> ta;
    ta.init(lane, wave, 0);
    struct Cur {
      int r, off, s;
      DevRun run;
    };
    auto advance = [&](Cur c, bool* valid) {
      *valid = true;
      if (++c.s == 2) {
        c.s = 0;
        if (++c.off == c.run.nblk) {
          c.off = 0;
          if (++c.r == run_e)
            *valid = false;
          else
            c.run = load_const(p.qruns, c.r);
        }
      }
      return c;
    };
    auto issue = [&](const Cur& c, int buf) {
      char* base = smem + buf * L::STAGE;
      const int64_t row0 = int64_t{c.run.blk0 + c.off} * BK + c.s * SUB;
      load_stage_tile<D>(p.k, row0, p.hkv, hk, base, wave, lane);
      load_stage_tile<D>(p.v, row0, p.hkv, hk, base + L::TILE, wave, lane);
    };

    Cur cur{run_b, 0, 0, load_const(p.qruns, run_b)};
    issue(cur, 0);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      wait_for(qf[kk]);
      wait_for(dof[kk]);
    }
    wait_vmem();
    __syncthreads();
    int buf = 0;
    while (true) {
      bool has_next;
      const Cur nxt = advance(cur, &has_next);
      if (has_next) issue(nxt, buf ^ 1);

      const char* base = smem + buf * L::STAGE;
      const char* sk = base;
      const char* sv = base + L::TILE;

      // S^T = K Q^T, dP^T = V dO^T: lane li owns query q_in_blk, register i
      // owns key 32*kt + acc_row(i, lh) of the stage.
      f32x16 sc[2], dp[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        zero(sc[kt]);
        zero(dp[kt]);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          sc[kt] = mfma32(read_row_op<D>(sk, ta.row, kt, kk), qf[kk], sc[kt]);
          dp[kt] = mfma32(read_row_op<D>(sv, ta.row, kt, kk), dof[kk], dp[kt]);
        }
      }
      {
        constexpr int NM = D / 4;  // one operand read per MFMA, 3 in flight
        __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
        for (int i = 0; i < NM - 3; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
      }
      if (cur.run.cls == 1) {
        const int lim = cur.run.delta - cur.off * BK - cur.s * SUB + q_in_blk;
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
      // dQ^T += K^T dS^T: the A operand K^T is read transposed from the K
      // row tile.
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
        for (int ss = 0; ss < 4; ++ss)
          acc[cc] = mfma32(read_tr_op<D>(sk, ta, cc, ss), dsb[ss], acc[cc]);
      {
        constexpr int NM = D / 8;  // two transpose reads per MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
        for (int i = 0; i < NM - 3; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
      }

      if (!has_next) break;
      wait_vmem();
      lds_barrier();  // stage buf^1 landed; every wave is done with buf
      buf ^= 1;
      cur = nxt;
    }
  }

  // Register 4g+t of chunk cc holds dim 32cc + 8g + 4lh + t of query q_row.
  // With accumulate, all old values are read before the first store.
  float* dst = p.dq + (q_row * p.hq + h) * D;
  f32x4 prev[D / 32][4];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int g = 0; g < 4; ++g) prev[cc][g] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (p.accumulate) {
#pragma unroll
    for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        prev[cc][g] = *reinterpret_cast<const f32x4*>(
            dst + cc * 32 + g * 8 + lh * 4);
  }
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      f32x4 val;
#pragma unroll
      for (int t = 0; t < 4; ++t)
        val[t] = fmaf(acc[cc][4 * g + t], p.scale, prev[cc][g][t]);
      *reinterpret_cast<f32x4*>(dst + cc * 32 + g * 8 + lh * 4) = val;
    }
}

template <int D>
hipError_t launch(const BwdParams& p, int grid_q, int grid_kv,
                  hipStream_t stream) {
  // + one int for the item slot of a queued workgroup
  const size_t smem_kv = DkdvLayout<D>::SMEM + 16;
  const size_t smem_q = DqLayout<D>::SMEM + 16;
  {
    hipError_t e = ensure_dynamic_lds<bwd_dkdv_kernel<D>>(smem_kv);
    if (e == hipSuccess) e = ensure_dynamic_lds<bwd_dq_kernel<D>>(smem_q);
    if (e != hipSuccess) return e;
  }
  const int64_t prep_threads = p.rows_q * p.hq * (D / 8);
  const int prep_grid = static_cast<int>((prep_threads + NT - 1) / NT);
  hipLaunchKernelGGL(bwd_prep_kernel<D>, dim3(prep_grid), dim3(NT), 0, stream,
                     p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (grid_kv > 0) {
    hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3(grid_kv), dim3(NT_KV), smem_kv,
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
