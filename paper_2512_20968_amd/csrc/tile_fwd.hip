// Tile attention forward for gfx950 (MI355X).
//
// One workgroup computes one (Q block, query head) item: BM = 256 query rows,
// eight waves of 32 rows each.  It walks the Q block's runs of KV blocks
// (BN = 64 keys each) from the work list, so EMPTY blocks are never touched
// and only PARTIAL runs evaluate the causal mask (a wave-uniform branch).  For
// every KV block it forms scores, updates the online softmax of each row and
// accumulates P V -- the per-pair computation of Algorithm 2 with the
// online-softmax reducer applied inside the kernel (Section 2.2).
//
// Schedule: two-group ping-pong.  Waves 0-3 (group A) and 4-7 (group B)
// share the four SIMDs pairwise (wave w and w+4 on SIMD w % 4).  Per KV block
// each wave runs an MFMA phase X(n) -- the scores of block n+1 and
// O += V(n)^T P(n)^T -- and a VALU phase Y(n) -- mask, running max, rescale
// and the exponentials that make P(n+1).  Group B runs one phase behind
// group A and every phase ends at a workgroup barrier, so on each SIMD one
// wave's MFMAs always overlap the other wave's softmax.  Group B also issues
// the K/V loads, which makes both of its phases the longer ones of their
// slots, so its waves run at raised issue priority.  On launches with many
// items, the last items of each XCD's share are taken from per-XCD counters
// (queued_slot), so that faster XCDs take more of them.
//
// Layout choices (64-wide wavefronts, v_mfma_f32_32x32x16_bf16):
//  * Scores are computed transposed, S^T = K Q^T (A = K rows from LDS,
//    B = Q columns held in registers for the whole item), so each lane owns
//    one query row and the row max / row sum are in-lane reductions plus one
//    exchange between the two half-waves.
//  * K rows are fed to the MFMA in an order that swaps bits 2 and 3 of the
//    row index, which leaves P^T in the accumulators already laid out as the
//    k-contiguous B operand of O^T += V^T P^T.
//  * K and V tiles stream from HBM straight into LDS (buffer loads with the
//    LDS-destination form, no staging registers), double buffered, rows
//    XOR-swizzled so every MFMA operand read is bank-conflict free.
//  * The V^T operand comes from the row-major V tile through the LDS
//    transpose read (ds_read_b64_tr_b16), two per MFMA.
//  * Softmax runs in the log2 domain with the scale folded into one FMA
//    before v_exp_f32.  The running max is exact, so a row's largest
//    probability is exactly 1 and its bf16 rounding is error-free.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "tile_common.h"

namespace mesh_attn {
namespace {

using namespace dev;

constexpr int BM = kFwdBM;  // 256
constexpr int BN = kFwdBN;  // 64
constexpr int NW = 8;       // waves per workgroup
constexpr int NT = NW * 64;
static_assert(BM == NW * 32, "one 32-row tile per wave");

template <int D>
struct FwdLayout {
  static constexpr int ROWB = 2 * D;         // bytes per K/V row
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;       // rows per 1 KB wave load
  static constexpr int RPW = BN / 4;         // rows each loading wave loads
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

__device__ __forceinline__ Cursor first_block(const FwdParams& p, int r,
                                              int run_e) {
  Cursor c;
  c.r = r;
  c.off = 0;
  c.valid = r < run_e;
  if (c.valid) c.run = load_const(p.runs, r);
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
__global__ __launch_bounds__(NT, 1) void tile_fwd_kernel(FwdParams p) {
  using L = FwdLayout<D>;
  extern __shared__ __align__(16) char smem[];

  const int tid = threadIdx.x;
  // Wave index as a scalar (the compiler cannot infer that tid >> 6 is
  // uniform across the wave).
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;   // 0: group A, 1: group B
  const int wg = wave & 3;     // wave within its group
  const int lane = tid & 63;
  const int li = lane & 31;
  const int lh = lane >> 5;

  // Item (order slot; see queued_static_slots).
  const int slot = queued_slot(p.n_items, p.queue,
                               reinterpret_cast<int*>(smem + L::SMEM));
  if (slot < 0) return;
  const int2 item = load_const(p.order, slot);
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

  // Number of KV blocks of this Q block.
  int nblocks = 0;
  for (int r = run_b; r < run_e; ++r) nblocks += load_const(p.runs, r).nblk;

  if (nblocks > 0) {
    // Direct global -> LDS staging, done by the four waves of group B.
    // Wave wg of the group fills rows wg*RPW .. +RPW of a tile with NLI
    // loads of 1 KB; lane i of load j takes row wg*RPW + j*RPI + i/CPR and
    // writes physical chunk i%CPR, i.e. the logical chunk
    // (i%CPR) ^ swizzle(row).
    const int64_t row_elems = int64_t{p.hkv} * D;  // elements per KV row
    const uint32_t row_bytes_g = static_cast<uint32_t>(row_elems * 2);
    const uint32_t blk_bytes = static_cast<uint32_t>(BN * row_elems * 2);
    // Every swizzled offset below has the form base ^ (stride * index): the
    // swizzle XORs a lane-dependent value into the chunk bits, and the loop
    // index only flips higher chunk bits that the row part leaves zero.  So
    // one base register per stream plus a v_xor per access replaces a
    // register per access.
    // Loads: lane i of load j reads logical chunk (i%CPR) ^ swizzle(row) of
    // row wg*RPW + j*RPI + i/CPR; for K that is kvo0 ^ (64 j), for V the
    // swizzle does not depend on j.
    const int lrow = lane / L::CPR;
    const uint32_t kvo0 =
        lrow * row_bytes_g + (((lane % L::CPR) ^ L::kswz(wg * L::RPW + lrow)) * 16);
    const uint32_t vvo0 =
        lrow * row_bytes_g + (((lane % L::CPR) ^ L::vswz(wg * L::RPW + lrow)) * 16);
    auto rsrc_of = [&](const uint16_t* base, int64_t blk) {
      return make_rsrc(base + (blk * BN * p.hkv + hk) * D, blk_bytes);
    };
    // LDS: K buffers 0, 1 then V buffers 0, 1; block j uses buffers j & 1.
    // One load round (the K tile of one block and the V tile of another) as
    // 2 NLI single loads, so that they can be spread over a phase.  A block
    // past the end gets an empty buffer range: its loads fetch nothing and
    // write zeros into a buffer that is free and never read.
    struct Round {
      rsrc_t rk, rv;
      char* kdst;
      char* vdst;
    };
    auto make_round = [&](const Cursor& ck, const Cursor& cv, int n) {
      Round rd;
      rd.rk = ck.valid ? rsrc_of(p.k, ck.blk()) : make_rsrc(p.k, 0);
      rd.rv = cv.valid ? rsrc_of(p.v, cv.blk()) : make_rsrc(p.v, 0);
      rd.kdst = smem + (n & 1) * L::TILE;
      rd.vdst = smem + (2 + ((n + 1) & 1)) * L::TILE;
      return rd;
    };
    auto load_part = [&](const Round& rd, int t) {  // t in [0, 2 NLI)
      const int j = t % L::NLI;
      const int row0 = wg * L::RPW + j * L::RPI;
      if (t < L::NLI)
        buffer_load16_lds(rd.rk, rd.kdst + row0 * L::ROWB, kvo0 ^ (64u * j),
                          row0 * row_bytes_g);
      else
        buffer_load16_lds(rd.rv, rd.vdst + row0 * L::ROWB, vvo0,
                          row0 * row_bytes_g);
    };
    auto load_k = [&](int64_t blk, int buf) {
      const rsrc_t rk = rsrc_of(p.k, blk);
#pragma unroll
      for (int j = 0; j < L::NLI; ++j) {
        const int row0 = wg * L::RPW + j * L::RPI;
        buffer_load16_lds(rk, smem + buf * L::TILE + row0 * L::ROWB,
                          kvo0 ^ (64u * j), row0 * row_bytes_g);
      }
    };
    auto load_v = [&](int64_t blk, int buf) {
      const rsrc_t rv = rsrc_of(p.v, blk);
#pragma unroll
      for (int j = 0; j < L::NLI; ++j) {
        const int row0 = wg * L::RPW + j * L::RPI;
        buffer_load16_lds(rv, smem + (2 + buf) * L::TILE + row0 * L::ROWB,
                          vvo0, row0 * row_bytes_g);
      }
    };
    // K operand read: row kt*32 + perm(li), dims 16kk + 8lh (logical chunk
    // 2kk + lh); the swizzle of such a row does not depend on kt, and the
    // byte offset is kra0 ^ (32 kk).
    int kra0;
    {
      const int prow = key_perm(li);
      kra0 = prow * L::ROWB + ((lh ^ L::kswz(prow)) * 16);
    }
    // V^T operand read (transpose): 16-lane group g, lane s reads row
    // 8*(g>>1) + s/4 (+16ss, +4 for the second half) at dims
    // 32cc + 16*(g&1) + 4*(s%4) .. +3; the swizzle of those rows depends on
    // s only, and the byte offset is vra0 ^ (64 cc).
    int vra0;
    {
      const int g16 = lane >> 4, s16 = lane & 15;
      const int vrow = 8 * (g16 >> 1) + (s16 >> 2);
      const int c16 = 2 * (g16 & 1) + ((s16 & 3) >> 1);
      vra0 = vrow * L::ROWB + ((c16 ^ L::vswz(vrow)) * 16) + 8 * (s16 & 1);
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
                              kb + (kra0 ^ (32 * kk)) + kt * 32 * L::ROWB),
                          qf[kk], sc[kt]);
      }
      // Keep three operand reads in flight ahead of the MFMAs instead of
      // hoisting all of them (which would cost ~64 registers).
      constexpr int NM = D / 8;  // MFMAs in this block
      __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
      for (int i = 0; i < NM - 3; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
    };
    // O^T += V^T P^T from V buffer `buf`; key step ss covers keys
    // 16ss + 8lh + 0..7.
    auto pv = [&](const bf16x8 (&pb)[4], int buf) {
      const char* vb = smem + (2 + buf) * L::TILE;
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
#pragma unroll
        for (int ss = 0; ss < 4; ++ss) {
          const char* a0 = vb + (vra0 ^ (64 * cc)) + ss * 16 * L::ROWB;
          const bf16x8 a =
              join_bf16(lds_read_tr16(a0), lds_read_tr16(a0 + 4 * L::ROWB));
          oacc[cc] = mfma32(a, pb[ss], oacc[cc]);
        }
      }
      // Two transpose reads per MFMA, three MFMAs' worth in flight.
      constexpr int NM = D / 8;
      __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
      for (int i = 0; i < NM - 3; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
    };
    // Softmax of one block's scores: causal mask (PARTIAL blocks: key j of
    // the run is hidden from query i of the Q block iff j - i > delta),
    // running max, rescale of O and l if some row of the wave has a new max,
    // then P = exp2(s S - m) into the bf16 B operand and the row sums.
    auto softmax = [&](f32x16 (&sc)[2], const Cursor& cu, bf16x8 (&pb)[4],
                       auto&& hook) {
      if (cu.run.cls == 1) {
        const int lim = cu.run.delta - cu.off * BN + q_in_blk;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (kt * 32 + acc_row(i, lh) > lim) sc[kt][i] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[kt][i]);
      mx = max_with_other_half(mx) * p.scale_log2;
      // Rescale O and l only when some row of the wave has a new maximum
      // (a wave-uniform branch).  Past the first few blocks of a row that is
      // rare, and the 4 * D / 2 multiplies would otherwise be the largest
      // VALU item of this phase after the exponentials.  A row whose maximum
      // is still -inf takes alpha = exp2(-inf) = 0 on 0-valued sums.
      const float m_new = fmaxf(m, mx);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      if (__builtin_amdgcn_ballot_w64(m_new != m)) {
        const float alpha = exp2_fast(m - m_use);
        l *= alpha;
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[cc][i] *= alpha;
        m = m_new;
      }
      float rs[4];
#pragma unroll
      for (int ss = 0; ss < 4; ++ss) {
        hook(ss);
        float e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          e8[e] = exp2_fast(
              fmaf(sc[ss >> 1][(ss & 1) * 8 + e], p.scale_log2, -m_use));
          pb[ss][e] = static_cast<__bf16>(e8[e]);
        }
        rs[ss] = ((e8[0] + e8[1]) + (e8[2] + e8[3])) +
                 ((e8[4] + e8[5]) + (e8[6] + e8[7]));
      }
      l += (rs[0] + rs[1]) + (rs[2] + rs[3]);
    };

    // Prologue (all waves): K(0), V(0) and K(1) into LDS (group B loads),
    // then the scores and probabilities of block 0.
    Cursor c0 = first_block(p, run_b, run_e);
    Cursor c1 = next_block(p, c0, run_e);
    if (grp == 1) {
      load_k(c0.blk(), 0);
      load_v(c0.blk(), 0);
      if (c1.valid) load_k(c1.blk(), 1);
    }
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) wait_for(qf[kk]);
    wait_vmem();
    __syncthreads();
    bf16x8 pb[4];
    {
      f32x16 s0[2];
      scores(s0, 0);
      softmax(s0, c0, pb, [](int) {});
    }
    // Every wave has read K(0) before group B refills K buffer 0.
    __syncthreads();

    // Phase loops.  There are 2N slots (N = nblocks), each ending at a
    // workgroup barrier (an LDS-only barrier: group B's loads stay in flight
    // across the barrier of the slot that issues them).  Group A runs X(0) Y(0) X(1) ... X(N-1) and idles in
    // the last slot; group B idles in the first slot and then runs the same
    // sequence, one slot behind.  Group B issues the loads of K(n+2) and
    // V(n+1) in slot 2n and drains them at the end of slot 2n+1, so they are
    // in LDS by slot 2n+2, when A's X(n+1) first reads them; the buffers they
    // overwrite were last read in slots 2n-2 and 2n-1.
    f32x16 snx[2];
    Cursor cs = c1;  // block whose scores X(n) computes (block n+1)
    if (grp == 0) {
      for (int n = 0; n < nblocks; ++n) {
        if (cs.valid) scores(snx, (n + 1) & 1);
        pv(pb, n & 1);
        lds_barrier();
        if (cs.valid) {
          softmax(snx, cs, pb, [](int) {});
          cs = next_block(p, cs, run_e);
        }
        lds_barrier();
      }
    } else {
      Cursor ck = next_block(p, c1, run_e);  // K block to load next
      Cursor cv = c1;                        // V block to load next
      // Round n: K(n+2) and V(n+1), issued in slot 2n.  Issued as one burst
      // at the end of the softmax phase, the 2 NLI loads per wave held the
      // issuing waves up for several hundred cycles (measured: that phase
      // grew by about half); spread over the four exponential groups they
      // overlap the VALU work instead (about 5% faster overall).
      auto advance = [&]() {
        ck = next_block(p, ck, run_e);
        cv = next_block(p, cv, run_e);
      };
      {
        const Round rd = make_round(ck, cv, 0);
#pragma unroll
        for (int t = 0; t < 2 * L::NLI; ++t) load_part(rd, t);
        advance();
      }
      lds_barrier();
      // Group B's slots are the longer ones: its softmax phase also issues
      // the loads, and its MFMA phase runs beside group A's shorter softmax.
      // So its waves take issue priority over their group-A partners for the
      // whole loop (2-3 % faster than equal priority; raising it only for
      // the softmax phase gave half of that).
      __builtin_amdgcn_s_setprio(1);
      constexpr int PER = (2 * L::NLI) / 4;  // loads per exponential group
      static_assert(PER * 4 == 2 * L::NLI, "loads split evenly over 4 groups");
      for (int n = 0; n < nblocks; ++n) {
        if (cs.valid) scores(snx, (n + 1) & 1);
        pv(pb, n & 1);
        wait_vmem();
        lds_barrier();
        // Block n+1 exists iff n + 1 < N; the last slot belongs to X(N-1)
        // and has no round after it.
        if (cs.valid) {
          // Cursor updates (scalar code with branches) go first, so that the
          // compiler does not sink the exponentials below them, away from
          // the loads they are meant to hide.
          const Round rd = make_round(ck, cv, n + 1);
          const Cursor cur = cs;
          cs = next_block(p, cs, run_e);
          advance();
          softmax(snx, cur, pb, [&](int ss) {
            // Keep the compiler from hoisting all loads to the phase start.
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int t = 0; t < PER; ++t) load_part(rd, ss * PER + t);
          });
          lds_barrier();
        }
      }
      __builtin_amdgcn_s_setprio(0);
    }
  }

  // Epilogue: O = acc / l, LSE = (m + log2 l) * ln 2.
  const float lt = l + __shfl_xor(l, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  const float lse2 = lt > 0.f ? m + __builtin_amdgcn_logf(lt) : -INFINITY;
  const int64_t lidx = int64_t{h} * p.rows_q + q_row;
  // Running accumulation (float32 partials only): fold (O, LSE) of this
  // call into the stored pair with the two-part online-softmax reducer,
  // lse = M + ln(e^(lse_old - M) + e^(lse_new - M)) with M the larger, and
  // O = w_old O_old + w_new O_new with w = e^(lse_part - lse).  Both lane
  // halves of a row read the stored LSE before the first half rewrites it
  // (same wave, program order).
  float w_old = 0.f, w_new = 1.f, lse_out = lse2;  // log2 units
  if constexpr (OUT_F32) {
    if (p.accumulate) {
      const float old2 = p.lse[lidx] * 1.4426950408889634f;
      const float mx = fmaxf(old2, lse2);
      if (mx == -INFINITY) {
        w_old = 1.f;  // neither part sees a key: keep the stored O = 0
        w_new = 0.f;
      } else {
        const float a = exp2_fast(old2 - mx), b = exp2_fast(lse2 - mx);
        const float sum = a + b;
        lse_out = mx + __builtin_amdgcn_logf(sum);
        w_old = a / sum;
        w_new = b / sum;
      }
    }
  }
  if (lh == 0)
    p.lse[lidx] =
        lse_out == -INFINITY ? -INFINITY : lse_out * 0.69314718055994531f;
  // O^T accumulator: register 4g+t of chunk cc holds dim 32cc + 8g + 4lh + t.
  const int64_t obase = (q_row * p.hq + h) * D;
  const float sc_new = inv * w_new;
  // Accumulating: every stored value is read before the first store, so the
  // loads are issued back to back.
  f32x4 prev[OUT_F32 ? D / 32 : 1][4];
  if constexpr (OUT_F32) {
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
              static_cast<const float*>(p.o) + obase + cc * 32 + g * 8 +
              lh * 4);
    }
  }
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int dim = cc * 32 + g * 8 + lh * 4;
      f32x4 x;
#pragma unroll
      for (int t = 0; t < 4; ++t) x[t] = oacc[cc][4 * g + t] * sc_new;
      if constexpr (OUT_F32) {
        f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(p.o) + obase +
                                              dim);
#pragma unroll
        for (int t = 0; t < 4; ++t) x[t] = fmaf(w_old, prev[cc][g][t], x[t]);
        *dst = x;
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
  const size_t smem = FwdLayout<D>::SMEM + 16;  // + the item slot
  const hipError_t e = ensure_dynamic_lds<tile_fwd_kernel<D, F32>>(smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((tile_fwd_kernel<D, F32>), dim3(grid), dim3(NT), smem,
                     stream, p);
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
