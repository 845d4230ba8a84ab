// The allocation-free forward: the tile's work list is built on the device,
// into a fixed scratch array that every call on a GPU shares, instead of
// being built on the host and uploaded from pinned memory into a
// caller-provided workspace.  Everything a launch needs travels in kernel
// arguments (the index lists included), so the call allocates nothing, host
// or device, and never waits.
//
// The builder reproduces the host's canonical work list (Section 3.7 rule per
// block pair; runs in KV-list order, FULL before PARTIAL, EMPTY dropped) and
// its workgroup order (longest Q block first, the items of one KV head on one
// XCD when the KV head count allows it) with one workgroup of 1024 threads.
// Along one KV partition a Q block's classes only fall (positions grow with
// the row under both layouts), so each (Q block, KV partition) pair has a
// FULL prefix and a PARTIAL middle whose lengths are found by binary search.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "internal.h"
#include "mesh_attn.h"

namespace mesh_attn {
namespace {

// The scratch array of the allocation-free forward: kNoAllocScratchBytes on
// every GPU the library runs on, held until the process ends.  Host code
// must never pass its name to a kernel (the name is a host-side stand-in):
// noalloc_scratch() gives the device address.
__device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kBuildThreads = 1024;

__device__ int64_t tok_pos(const PlanBuildParams& p, int part, int64_t row) {
  return p.layout == 1 ? row * p.n + part : int64_t{part} * p.P + row;
}

// Length of the prefix of [0, p.nkbp) on which `pred` holds (pred holds on a
// prefix).
template <class F>
__device__ int prefix_len(int nkbp, F pred) {
  int lo = 0, hi = nkbp;  // pred(lo - 1) holds, pred(hi) fails
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (pred(mid))
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

struct PairRuns {
  int nfull, nvis;        // FULL blocks [0, nfull), PARTIAL [nfull, nvis)
  int32_t qp, kp;
  int64_t q_row0;
};

__device__ PairRuns pair_runs(const PlanBuildParams& p, int qb, int b) {
  const int qpb = p.P / p.bm;
  PairRuns r;
  r.qp = p.q_idx[qb / qpb];
  r.kp = p.kv_idx[b];
  r.q_row0 = int64_t{qb % qpb} * p.bm;
  if (!p.causal) {
    r.nfull = r.nvis = p.nkbp;
    return r;
  }
  const int64_t qf = tok_pos(p, r.qp, r.q_row0);
  const int64_t ql = tok_pos(p, r.qp, r.q_row0 + p.bm - 1);
  const int kp = r.kp;
  // FULL: every key of the block at or before every query of the Q block.
  r.nfull = prefix_len(p.nkbp, [&](int kb) {
    return tok_pos(p, kp, int64_t{kb} * p.bn + p.bn - 1) <= qf;
  });
  // Not EMPTY: some key of the block at or before some query.
  r.nvis = prefix_len(p.nkbp, [&](int kb) {
    return tok_pos(p, kp, int64_t{kb} * p.bn) <= ql;
  });
  return r;
}

// Mask offset of a run starting at KV block kb0 (see DevRun).
__device__ int32_t run_delta(const PlanBuildParams& p, const PairRuns& r,
                             int kb0) {
  const int64_t k_row0 = int64_t{kb0} * p.bn;
  if (p.layout == 1)
    return static_cast<int32_t>((r.q_row0 - k_row0) + (r.qp >= r.kp ? 0 : -1));
  return static_cast<int32_t>(tok_pos(p, r.qp, r.q_row0) -
                              tok_pos(p, r.kp, k_row0));
}

__global__ __launch_bounds__(kBuildThreads) void fwd_plan_build_kernel(
    PlanBuildParams p) {
  __shared__ int s_work[kNoAllocMaxQBlocks];
  __shared__ int s_scan[kBuildThreads];
  const int t = threadIdx.x;
  // Thread t owns a contiguous segment of Q blocks for the run list.
  const int seg = (p.nqb + kBuildThreads - 1) / kBuildThreads;
  const int lo = min(t * seg, p.nqb);
  const int hi = min(lo + seg, p.nqb);
  int cnt = 0;
  for (int qb = lo; qb < hi; ++qb) {
    int work = 0;
    for (int b = 0; b < p.nkv; ++b) {
      const PairRuns r = pair_runs(p, qb, b);
      cnt += (r.nfull > 0) + (r.nvis > r.nfull);
      work += r.nvis;
    }
    s_work[qb] = work;
  }
  s_scan[t] = cnt;
  __syncthreads();
  // Inclusive scan of the segment counts (Hillis-Steele).
  for (int off = 1; off < kBuildThreads; off <<= 1) {
    const int add = t >= off ? s_scan[t - off] : 0;
    __syncthreads();
    s_scan[t] += add;
    __syncthreads();
  }
  int at = s_scan[t] - cnt;
  for (int qb = lo; qb < hi; ++qb) {
    p.qblk_ptr[qb] = at;
    for (int b = 0; b < p.nkv; ++b) {
      const PairRuns r = pair_runs(p, qb, b);
      if (r.nfull > 0)
        p.runs[at++] = DevRun{b * p.nkbp, r.nfull, MA_CLS_FULL,
                              run_delta(p, r, 0)};
      if (r.nvis > r.nfull)
        p.runs[at++] = DevRun{b * p.nkbp + r.nfull, r.nvis - r.nfull,
                              MA_CLS_PARTIAL, run_delta(p, r, r.nfull)};
    }
  }
  if (t == kBuildThreads - 1) p.qblk_ptr[p.nqb] = s_scan[t];

  // Workgroup order.  Items (Q block, head) sorted by (work descending, head,
  // Q block); with the KV heads a multiple of the XCD count, the items of KV
  // head x go to XCD x % 8 (slot j * 8 + x), else item i takes slot i.
  const bool by_kv = p.hkv % kNumXcd == 0;
  for (int qb = t; qb < p.nqb; qb += kBuildThreads) {
    const int w = s_work[qb];
    int gt = 0, eq = 0, eq_before = 0;
    for (int b2 = 0; b2 < p.nqb; ++b2) {
      const int w2 = s_work[b2];
      gt += w2 > w;
      eq += w2 == w;
      eq_before += (w2 == w) & (b2 < qb);
    }
    for (int h = 0; h < p.hq; ++h) {
      int slot;
      if (by_kv) {
        const int kvh = h / p.group;
        const int lane_heads = p.hq / kNumXcd;
        const int heads_before = (kvh / kNumXcd) * p.group + h % p.group;
        slot = (gt * lane_heads + eq * heads_before + eq_before) * kNumXcd +
               kvh % kNumXcd;
      } else {
        slot = gt * p.hq + h * eq + eq_before;
      }
      p.order[slot] = make_int2(qb, h);
    }
  }
  for (int slot = p.nqb * p.hq + t; slot < p.grid; slot += kBuildThreads)
    p.order[slot] = make_int2(-1, -1);
  if (t < kNumXcd) p.queue[t] = 0;
}

// Device address of the scratch array, per device (each GPU holds its own
// copy at its own address).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    // Once per device, with that device current.
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_fwd_plan_build(const PlanBuildParams& p,
                                 hipStream_t stream) {
  hipLaunchKernelGGL(fwd_plan_build_kernel, dim3(1), dim3(kBuildThreads), 0,
                     stream, p);
  return hipGetLastError();
}

}  // namespace mesh_attn
