// Internal interface between the host library (host.cpp) and the HIP kernel
// translation units.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace mesh_attn {

// gfx950 (MI355X) has 8 XCDs; consecutive workgroup ids are dispatched to
// XCDs round robin, so id i runs on XCD i % 8.
constexpr int kNumXcd = 8;

// Forward block shape: 8 waves x 32 query rows, 64 keys per LDS stage.
constexpr int kFwdBM = 256;
constexpr int kFwdBN = 64;

// Backward block shapes.
constexpr int kBwdBM = 128;  // Q rows per dQ workgroup (4 waves x 32)
constexpr int kBwdBN = 128;  // KV rows per dK/dV workgroup (4 waves x 32)

// One run of consecutive KV blocks of one KV list entry, as the kernels read
// it: x = first KV block (index into the tile's KV buffer, in blocks of the
// pass's KV block size), y = number of blocks, z = class (MA_CLS_*),
// w = position of the Q block's first row minus position of the run's first
// key (the causal mask of a PARTIAL run: key j of the run is hidden from
// query i of the block iff j - i > w).
struct DevRun {
  int32_t blk0, nblk, cls, delta;
};

struct FwdParams {
  const uint16_t* q;   // bf16 [rows_q][hq][d]
  const uint16_t* k;   // bf16 [rows_kv][hkv][d]
  const uint16_t* v;
  void* o;             // bf16 or f32 [rows_q][hq][d]
  float* lse;          // [hq][rows_q]
  const int32_t* qblk_ptr;   // [n_qblk + 1]
  const DevRun* runs;
  const int2* order;         // (qblk, q head); XCD lane x at slots j*8 + x
  int32_t* queue;            // [8] items taken from each lane; 0 at launch
  int32_t n_items;           // items (Q block, q head) in the order
  int64_t rows_q;
  int32_t hq, hkv, group;
  float scale_log2;    // softmax scale * log2(e)
  int32_t accumulate;  // 1: fold into the float32 (O, LSE) already stored
};

// Workgroup items of the forward and of both backward kernels.  The XCDs of
// the part run at different speeds (a few per cent apart under load) while
// the dispatcher gives each an eighth of the workgroups, so on launches with
// many items per compute unit the last quarter of every XCD lane of the item
// order is taken from per-lane counters: the first queued_static_slots(n)
// workgroups take slot blockIdx.x, the others the next remaining item of
// their XCD's lane or else of another lane, and about one in eight more of
// them are launched than remaining items, so an XCD that runs faster takes
// more of the last items.  Below kQueuedMinItems (16 items per compute unit
// of the 256-CU part) every whole row of eight slots is static.
constexpr int64_t kQueuedMinItems = 4096;
__host__ __device__ inline int64_t queued_static_slots(int64_t n_items) {
  return n_items >= kQueuedMinItems ? (n_items / 8) * 3 / 4 * 8
                                    : (n_items / 8) * 8;
}
__host__ __device__ inline int64_t queued_launch_grid(int64_t n_items) {
  const int64_t fixed = queued_static_slots(n_items);
  const int64_t dyn = n_items - fixed;
  const int64_t extra = n_items >= kQueuedMinItems ? dyn / 8 + 8 : 0;
  return fixed + (dyn + extra + 7) / 8 * 8;
}

hipError_t launch_tile_fwd(const FwdParams& p, int head_dim, bool out_f32,
                           int grid, hipStream_t stream);

struct MergeParams {
  const void* o_parts;
  const float* lse_parts;
  void* o_out;
  float* lse_out;
  int64_t rows;
  int32_t k_parts, heads, head_dim;
};

hipError_t launch_lse_merge(const MergeParams& p, bool in_f32, bool out_f32,
                            hipStream_t stream);

struct BwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* d_o;
  const float* lse;
  float* dq;
  float* dk;
  float* dv;
  float* delta;        // workspace [hq][rows_q]: rowsum(dO * O)
  float* lse2;         // workspace [hq][rows_q]: LSE * log2(e), -inf -> +inf
  // Q-major runs (dQ kernel): Q blocks of kBwdBM rows, KV blocks of kBwdBN.
  const int32_t* qblk_ptr;
  const DevRun* qruns;
  const int2* qorder;
  // KV-major runs (dK/dV kernel): Q blocks of kBwdBM rows per KV block of
  // kBwdBN; the delta field is q-first minus kv-first, as in the Q-major runs.
  const int32_t* kvblk_ptr;
  const DevRun* kvruns;
  const int2* kvorder;   // (kvblk, kv head)
  // Per-XCD-lane item counters of the two orders, 0 at launch, and their
  // item counts (see queued_static_slots).
  int32_t* qqueue;
  int32_t* kvqueue;
  int32_t q_items, kv_items;
  int64_t rows_q, rows_kv;
  int32_t hq, hkv, group;
  float scale, scale_log2;
  int32_t accumulate;
};

hipError_t launch_tile_bwd(const BwdParams& p, int head_dim, int grid_q,
                           int grid_kv, hipStream_t stream);

// ---------------------------------------------------------------------------
// Allocation-free forward (noalloc.hip): the work list is built on the device
// into a fixed scratch array instead of a caller workspace.
// ---------------------------------------------------------------------------

constexpr size_t kNoAllocScratchBytes = size_t{8} << 20;  // per GPU
constexpr int kNoAllocMaxList = 256;      // partitions per index list
constexpr int kNoAllocMaxQBlocks = 4096;  // forward Q blocks of the tile

struct PlanBuildParams {
  int32_t P, n, layout, causal;   // problem (partition length, partitions)
  int32_t nq, nkv, hq, hkv, group;
  int32_t bm, bn;                 // forward block shape
  int32_t nqb, nkbp;              // Q blocks of the tile, KV blocks per part
  int32_t grid;                   // workgroup slots of the order
  int32_t* qblk_ptr;              // [nqb + 1] in the scratch array
  DevRun* runs;                   // [<= 2 nqb nkv]
  int2* order;                    // [grid]
  int32_t* queue;                 // [8] lane counters, zeroed by the build
  int32_t q_idx[kNoAllocMaxList];
  int32_t kv_idx[kNoAllocMaxList];
};

// Device address of the scratch array on the current device (looked up with
// hipGetSymbolAddress on the first call per device, then cached).
hipError_t noalloc_scratch(void** ptr);

// Builds the forward work list and workgroup order of `p` (one workgroup).
hipError_t launch_fwd_plan_build(const PlanBuildParams& p, hipStream_t stream);

// Kernels with more than 64 KB of dynamic LDS need the limit raised once per
// kernel and device; this does it on the first launch on each device (ids
// below 64; higher ids set it on every launch).  Safe to call from several
// threads: the attribute set is idempotent and the flags are atomic.
template <auto Kern>
hipError_t ensure_dynamic_lds(size_t bytes) {
  static std::atomic<uint64_t> done{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev >= 0 && dev < 64 ? uint64_t{1} << dev : 0;
  if (bit != 0 && (done.load(std::memory_order_acquire) & bit) != 0)
    return hipSuccess;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(Kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize,
                          static_cast<int>(bytes));
  if (e == hipSuccess && bit != 0)
    done.fetch_or(bit, std::memory_order_release);
  return e;
}

}  // namespace mesh_attn
