// Host side of the mesh_attn C ABI: argument validation, error text, the
// canonical block work list, workgroup ordering and kernel launches.
//
// The work list follows the causal rule of Section 3.7 (a key is visible to a
// query iff its global position is not larger) applied per (Q block, KV block)
// pair; see include/mesh_attn.h for the exact layout.

#include "mesh_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "host_error.h"
#include "internal.h"

using namespace mesh_attn;

static_assert(MA_NOALLOC_SCRATCH_BYTES == kNoAllocScratchBytes &&
                  MA_NOALLOC_MAX_LIST == kNoAllocMaxList &&
                  MA_NOALLOC_MAX_QBLOCKS == kNoAllocMaxQBlocks,
              "public limits of the allocation-free forward");

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace mesh_attn {
namespace host {

ma_status_t fail(ma_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ma_status_t ok() {
  g_last_error.clear();
  return MA_OK;
}

}  // namespace host
}  // namespace mesh_attn

namespace {

using mesh_attn::host::fail;
using mesh_attn::host::ok;

ma_status_t hip_fail(hipError_t e, const char* what) {
  return fail(MA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

ma_status_t check_list(const char* name, const int32_t* idx, int32_t n,
                       int32_t num_partitions) {
  if (n < 1) return fail(MA_ERR_INVALID_ARG, "%s: length %d < 1", name, n);
  if (!idx) return fail(MA_ERR_INVALID_ARG, "%s is NULL", name);
  std::vector<char> seen(static_cast<size_t>(num_partitions), 0);
  for (int32_t i = 0; i < n; ++i) {
    if (idx[i] < 0 || idx[i] >= num_partitions)
      return fail(MA_ERR_INVALID_ARG, "%s[%d] = %d outside [0, %d)", name, i,
                  idx[i], num_partitions);
    if (seen[idx[i]])
      return fail(MA_ERR_INVALID_ARG, "%s[%d] = %d is a duplicate", name, i,
                  idx[i]);
    seen[idx[i]] = 1;
  }
  return MA_OK;
}

ma_status_t check_problem(const ma_problem_t* p) {
  if (!p) return fail(MA_ERR_INVALID_ARG, "problem is NULL");
  if (p->num_partitions < 1)
    return fail(MA_ERR_INVALID_ARG, "num_partitions %d < 1", p->num_partitions);
  if (p->partition_len < 1)
    return fail(MA_ERR_INVALID_ARG, "partition_len %d < 1", p->partition_len);
  if (static_cast<int64_t>(p->num_partitions) * p->partition_len >
      (int64_t{1} << 30))
    return fail(MA_ERR_INVALID_ARG,
                "sequence of %lld tokens exceeds 2^30",
                static_cast<long long>(p->num_partitions) * p->partition_len);
  if (p->num_q_heads < 1 || p->num_kv_heads < 1)
    return fail(MA_ERR_INVALID_ARG, "head counts must be >= 1 (Hq %d, Hkv %d)",
                p->num_q_heads, p->num_kv_heads);
  if (p->num_q_heads % p->num_kv_heads != 0)
    return fail(MA_ERR_INVALID_ARG, "num_q_heads %d not a multiple of "
                "num_kv_heads %d", p->num_q_heads, p->num_kv_heads);
  if (p->causal != 0 && p->causal != 1)
    return fail(MA_ERR_INVALID_ARG, "causal must be 0 or 1, got %d", p->causal);
  if (p->layout != MA_LAYOUT_CONTIGUOUS && p->layout != MA_LAYOUT_STRIPED)
    return fail(MA_ERR_INVALID_ARG, "layout must be %d or %d, got %d",
                MA_LAYOUT_CONTIGUOUS, MA_LAYOUT_STRIPED, p->layout);
  if (!(p->softmax_scale > 0.f) || !std::isfinite(p->softmax_scale))
    return fail(MA_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  if (p->head_dim < 1)
    return fail(MA_ERR_INVALID_ARG, "head_dim %d < 1", p->head_dim);
  return MA_OK;
}

ma_status_t check_blocks(const ma_problem_t* p, int32_t bm, int32_t bn) {
  if (bm < 1 || bn < 1)
    return fail(MA_ERR_INVALID_ARG, "block sizes must be >= 1 (%d, %d)", bm, bn);
  if (p->partition_len % bm != 0 || p->partition_len % bn != 0)
    return fail(MA_ERR_INVALID_ARG,
                "partition_len %d must be a multiple of the block sizes "
                "(%d, %d)", p->partition_len, bm, bn);
  return MA_OK;
}

ma_status_t check_tile(const ma_problem_t* p, const int32_t* q_idx, int32_t nq,
                       const int32_t* kv_idx, int32_t nkv) {
  ma_status_t st = check_problem(p);
  if (st != MA_OK) return st;
  st = check_list("q_idx", q_idx, nq, p->num_partitions);
  if (st != MA_OK) return st;
  return check_list("kv_idx", kv_idx, nkv, p->num_partitions);
}

// Global position of token `row` of partition `part` (Section 3.7 layouts).
// Within a partition positions grow with the row under both layouts, so a
// block's first and last rows hold its extreme positions.
inline int64_t token_pos(const ma_problem_t* p, int32_t part, int64_t row) {
  return p->layout == MA_LAYOUT_STRIPED
             ? row * p->num_partitions + part
             : int64_t{part} * p->partition_len + row;
}

// Mask offset of a (query block, key run) pair in rows: key row k0 + j is
// hidden from query row q0 + i iff j - i > offset.  Contiguous: the position
// difference q0 - k0 across partitions.  Striped: position (row * n + part),
// so key after query iff (j - i) * n > (q0 - k0) * n + (qp - kp), i.e. iff
// j - i > (q0 - k0) + floor((qp - kp) / n), and |qp - kp| < n.
inline int64_t mask_offset(const ma_problem_t* p, int32_t qp, int64_t q0,
                           int32_t kp, int64_t k0) {
  if (p->layout == MA_LAYOUT_STRIPED) return (q0 - k0) + (qp >= kp ? 0 : -1);
  return token_pos(p, qp, q0) - token_pos(p, kp, k0);
}

// Class of one block pair from its extreme token positions.
inline int block_class(int64_t q_first, int64_t q_last, int64_t k_first,
                       int64_t k_last, bool causal) {
  if (!causal) return MA_CLS_FULL;
  if (k_first > q_last) return MA_CLS_EMPTY;   // every key after every query
  if (k_last <= q_first) return MA_CLS_FULL;   // every key at/before every query
  return MA_CLS_PARTIAL;
}

struct Run {
  int32_t row, list, begin, end, cls;
};

// The rows of each partition a buffer holds: `len` consecutive local rows
// starting at local row `off` (the whole partition, or one GOO chunk of it).
struct Slice {
  int64_t len, off;
};

// Runs of one orientation.  "Rows" are the blocks of side A (bm_a rows each,
// lists a_idx), walked in buffer order; for each row, every list entry of side
// B (blocks of bm_b) yields maximal equal-class runs, EMPTY dropped.  When
// a_is_q, side A is the query side.  Each side's buffer holds slice sa / sb of
// each of its partitions.
void build_runs(const ma_problem_t* p, const int32_t* a_idx, int32_t na,
                int32_t bm_a, Slice sa, const int32_t* b_idx, int32_t nb,
                int32_t bm_b, Slice sb, bool a_is_q, std::vector<int32_t>* ptr,
                std::vector<Run>* runs) {
  const int32_t nab = static_cast<int32_t>(sa.len / bm_a);
  const int32_t nbb = static_cast<int32_t>(sb.len / bm_b);
  const bool causal = p->causal != 0;
  ptr->assign(static_cast<size_t>(na) * nab + 1, 0);
  runs->clear();
  for (int32_t a = 0; a < na; ++a) {
    for (int32_t ab = 0; ab < nab; ++ab) {
      const int32_t row = a * nab + ab;
      (*ptr)[row] = static_cast<int32_t>(runs->size());
      const int64_t a_row = sa.off + int64_t{ab} * bm_a;
      const int64_t a_first = token_pos(p, a_idx[a], a_row);
      const int64_t a_last = token_pos(p, a_idx[a], a_row + bm_a - 1);
      for (int32_t b = 0; b < nb; ++b) {
        int32_t kb = 0, cur = -1, start = 0;
        for (; kb <= nbb; ++kb) {
          int c = -2;
          if (kb < nbb) {
            const int64_t b_row = sb.off + int64_t{kb} * bm_b;
            const int64_t b_first = token_pos(p, b_idx[b], b_row);
            const int64_t b_last = token_pos(p, b_idx[b], b_row + bm_b - 1);
            c = a_is_q ? block_class(a_first, a_last, b_first, b_last, causal)
                       : block_class(b_first, b_last, a_first, a_last, causal);
          }
          if (c != cur) {
            if (cur > MA_CLS_EMPTY) runs->push_back({row, b, start, kb, cur});
            cur = c;
            start = kb;
          }
        }
      }
    }
  }
  (*ptr)[static_cast<size_t>(na) * nab] = static_cast<int32_t>(runs->size());
}

ma_status_t export_runs(const std::vector<int32_t>& ptr,
                        const std::vector<Run>& runs, int32_t* out_ptr,
                        ma_run_t* out_runs, int64_t cap, int64_t* n_runs) {
  if (n_runs) *n_runs = static_cast<int64_t>(runs.size());
  if (out_ptr) std::memcpy(out_ptr, ptr.data(), ptr.size() * sizeof(int32_t));
  if (static_cast<int64_t>(runs.size()) > cap || (!out_runs && !runs.empty()))
    return fail(MA_ERR_CAPACITY, "run list needs %zu entries, capacity %lld",
                runs.size(), static_cast<long long>(cap));
  for (size_t i = 0; i < runs.size(); ++i)
    out_runs[i] = ma_run_t{runs[i].row, runs[i].list, runs[i].begin,
                           runs[i].end, runs[i].cls};
  return ok();
}

// ---------------------------------------------------------------------------
// Device plans: the run list in the kernels' form plus the workgroup order,
// packed into one pinned host buffer that is copied to the caller's
// workspace on the caller's stream.
//
// Plans are cached per tile (at most kMaxPlans, least recently used evicted).
// A pinned source must outlive every asynchronous copy from it, and freeing
// pinned memory would wait for the device, so buffers are never freed while
// the library is in use: every upload records an event on the caller's
// stream, an evicted plan's buffer joins a spare list, and a spare buffer is
// reused for a new plan only once all events recorded after copies from it
// have completed (hipEventQuery, which does not wait).  No call synchronizes.
// ---------------------------------------------------------------------------

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Side {
  size_t off_ptr = 0, off_runs = 0, off_order = 0, off_queue = 0;
  int32_t grid = 0;
  int32_t n_items = 0;  // non-idle slots of the order
};

// An event recorded after a copy, with the device it belongs to (an event
// can only be recorded on a stream of the device it was created on).
struct PendingEvent {
  hipEvent_t ev;
  int dev;
};

struct PinnedBuf {
  void* host = nullptr;
  size_t cap = 0;
  std::vector<PendingEvent> pending;  // recorded after copies from this buffer
};

struct Plan {
  PinnedBuf* buf = nullptr;
  size_t bytes = 0;
  Side a, b;             // fwd uses a; bwd uses a (Q-major) and b (KV-major)
  uint64_t last_use = 0;
};

// What a kernel launch needs from a plan once it is uploaded.
struct PlanView {
  size_t bytes = 0;
  Side a, b;
};

std::mutex g_plan_mu;
std::map<std::string, Plan> g_plans;
std::vector<PinnedBuf*> g_spare;       // buffers of evicted plans
std::map<int, std::vector<hipEvent_t>> g_free_events;  // per device, completed
uint64_t g_plan_clock = 0;
constexpr size_t kMaxPlans = 1024;

// Drops the completed events of `b` (to the free list); true if none remain.
bool retire_completed(PinnedBuf* b) {
  size_t keep = 0;
  for (const PendingEvent& pe : b->pending) {
    if (hipEventQuery(pe.ev) == hipSuccess)
      g_free_events[pe.dev].push_back(pe.ev);
    else
      b->pending[keep++] = pe;
  }
  b->pending.resize(keep);
  return keep == 0;
}

// A pinned buffer of at least `bytes`: an idle spare if one is large enough
// (the smallest such), else a new allocation.
ma_status_t take_buffer(size_t bytes, PinnedBuf** out) {
  size_t best = g_spare.size();
  for (size_t i = 0; i < g_spare.size(); ++i) {
    PinnedBuf* b = g_spare[i];
    if (b->cap < bytes || !retire_completed(b)) continue;
    if (best == g_spare.size() || b->cap < g_spare[best]->cap) best = i;
  }
  if (best != g_spare.size()) {
    *out = g_spare[best];
    g_spare.erase(g_spare.begin() + best);
    return MA_OK;
  }
  auto* b = new PinnedBuf;
  b->cap = std::max(bytes, kAlign);
  hipError_t e = hipHostMalloc(&b->host, b->cap, hipHostMallocDefault);
  if (e != hipSuccess) {
    delete b;
    return hip_fail(e, "hipHostMalloc(work list)");
  }
  *out = b;
  return MA_OK;
}

std::string plan_key(int pass, const ma_problem_t* p, const int32_t* q_idx,
                     int32_t nq, const int32_t* kv_idx, int32_t nkv,
                     const ma_chunk_t& ch) {
  std::string k;
  auto put = [&k](const void* d, size_t n) {
    k.append(static_cast<const char*>(d), n);
  };
  put(&pass, sizeof pass);
  put(&ch, sizeof ch);
  put(&p->num_partitions, sizeof(int32_t));
  put(&p->partition_len, sizeof(int32_t));
  put(&p->num_q_heads, sizeof(int32_t));
  put(&p->num_kv_heads, sizeof(int32_t));
  put(&p->causal, sizeof(int32_t));
  put(&p->layout, sizeof(int32_t));
  put(&nq, sizeof nq);
  put(q_idx, sizeof(int32_t) * nq);
  put(&nkv, sizeof nkv);
  put(kv_idx, sizeof(int32_t) * nkv);
  return k;
}

// Kernel-side runs of one orientation.  Side A blocks (bm_a rows) own the
// workgroups; side B blocks (bm_b rows) are iterated.  delta = mask offset of
// the query block/run against the key block/run (mask_offset).
void device_runs(const ma_problem_t* p, const int32_t* a_idx, int32_t na,
                 int32_t bm_a, Slice sa, const int32_t* b_idx, int32_t nb,
                 int32_t bm_b, Slice sb, bool a_is_q, std::vector<int32_t>* ptr,
                 std::vector<DevRun>* out, std::vector<int64_t>* work) {
  std::vector<Run> runs;
  build_runs(p, a_idx, na, bm_a, sa, b_idx, nb, bm_b, sb, a_is_q, ptr, &runs);
  const int32_t nab = static_cast<int32_t>(sa.len / bm_a);
  const int32_t nbb = static_cast<int32_t>(sb.len / bm_b);
  out->resize(runs.size());
  work->assign(ptr->size() - 1, 0);
  for (size_t i = 0; i < runs.size(); ++i) {
    const Run& r = runs[i];
    const int32_t a_part = a_idx[r.row / nab];
    const int64_t a_row0 = sa.off + int64_t{r.row % nab} * bm_a;
    const int32_t b_part = b_idx[r.list];
    const int64_t b_row0 = sb.off + int64_t{r.begin} * bm_b;
    const int64_t delta = a_is_q ? mask_offset(p, a_part, a_row0, b_part, b_row0)
                                 : mask_offset(p, b_part, b_row0, a_part, a_row0);
    (*out)[i] = DevRun{r.list * nbb + r.begin, r.end - r.begin, r.cls,
                       static_cast<int32_t>(delta)};
    (*work)[r.row] += r.end - r.begin;
  }
}

// Workgroup order: items (block, head) sorted longest first, grouped so that
// the items of one KV head land on one XCD when the KV head count allows it
// (their workgroups then stream the same K/V through that XCD's L2).  Slot i
// of the grid runs on XCD i % kNumXcd.
std::vector<int2> workgroup_order(const std::vector<int64_t>& work,
                                  int32_t heads, int32_t group_to_kv,
                                  int32_t num_kv_heads) {
  struct Item {
    int64_t work;
    int32_t blk, head, kvh;
  };
  std::vector<Item> items;
  items.reserve(work.size() * heads);
  // Blocks without runs are kept: their workgroup still writes the output
  // (O = 0 and LSE = -inf, or zero gradients).
  for (int32_t h = 0; h < heads; ++h)
    for (size_t b = 0; b < work.size(); ++b)
      items.push_back({work[b], static_cast<int32_t>(b), h, h / group_to_kv});
  std::stable_sort(items.begin(), items.end(),
                   [](const Item& x, const Item& y) {
                     if (x.work != y.work) return x.work > y.work;
                     if (x.kvh != y.kvh) return x.kvh < y.kvh;
                     if (x.head != y.head) return x.head < y.head;
                     return x.blk < y.blk;
                   });
  std::vector<std::vector<int2>> lanes(kNumXcd);
  if (num_kv_heads % kNumXcd == 0) {
    for (const Item& it : items)
      lanes[it.kvh % kNumXcd].push_back(make_int2(it.blk, it.head));
  } else {
    for (size_t i = 0; i < items.size(); ++i)
      lanes[i % kNumXcd].push_back(make_int2(items[i].blk, items[i].head));
  }
  size_t depth = 0;
  for (auto& l : lanes) depth = std::max(depth, l.size());
  std::vector<int2> order(depth * kNumXcd, make_int2(-1, -1));
  for (int x = 0; x < kNumXcd; ++x)
    for (size_t j = 0; j < lanes[x].size(); ++j)
      order[j * kNumXcd + x] = lanes[x][j];
  return order;
}

struct SideData {
  std::vector<int32_t> ptr;
  std::vector<DevRun> runs;
  std::vector<int2> order;
};

size_t side_bytes(const SideData& s) {
  return align_up(s.ptr.size() * 4) + align_up(s.runs.size() * sizeof(DevRun)) +
         align_up(s.order.size() * sizeof(int2)) + align_up(kNumXcd * 4);
}

void side_pack(const SideData& s, char* base, size_t off, Side* out) {
  out->off_ptr = off;
  std::memcpy(base + off, s.ptr.data(), s.ptr.size() * 4);
  off += align_up(s.ptr.size() * 4);
  out->off_runs = off;
  if (!s.runs.empty())
    std::memcpy(base + off, s.runs.data(), s.runs.size() * sizeof(DevRun));
  off += align_up(s.runs.size() * sizeof(DevRun));
  out->off_order = off;
  if (!s.order.empty())
    std::memcpy(base + off, s.order.data(), s.order.size() * sizeof(int2));
  off += align_up(s.order.size() * sizeof(int2));
  // The item counters of this side's order, one per XCD lane (see
  // queued_static_slots), uploaded as zeros with every call.
  out->off_queue = off;
  std::memset(base + off, 0, kNumXcd * 4);
  out->grid = static_cast<int32_t>(s.order.size());
  out->n_items = 0;
  for (const int2& it : s.order) out->n_items += it.x >= 0;
}

// Upper bound of one side's packed bytes from sizes alone (at most two
// non-empty runs per (block, list entry): along a partition visibility only
// drops, FULL blocks first, then PARTIAL, then EMPTY).
size_t side_bound(int64_t n_blocks, int64_t n_list, int64_t heads) {
  return align_up((n_blocks + 1) * 4) +
         align_up(n_blocks * n_list * 2 * sizeof(DevRun)) +
         align_up((n_blocks * heads + kNumXcd) * sizeof(int2)) +
         align_up(kNumXcd * 4);
}

constexpr ma_chunk_t kWholeTile{0, 1, 0, 1};

// Builds (or finds) the plan of a tile, copies it to `ws` on `stream` and
// records the copy's completion event, all under the cache lock, so that no
// other thread can recycle the source buffer in between.
ma_status_t upload_plan(int pass, const ma_problem_t* p, const int32_t* q_idx,
                        int32_t nq, const int32_t* kv_idx, int32_t nkv,
                        const ma_chunk_t& ch, void* ws, hipStream_t stream,
                        PlanView* view) {
  const std::string key = plan_key(pass, p, q_idx, nq, kv_idx, nkv, ch);
  const int64_t P = p->partition_len;
  const Slice sq{P / ch.num_q_chunks, ch.q_chunk * (P / ch.num_q_chunks)};
  const Slice skv{P / ch.num_kv_chunks, ch.kv_chunk * (P / ch.num_kv_chunks)};
  std::lock_guard<std::mutex> lock(g_plan_mu);
  auto it = g_plans.find(key);
  if (it == g_plans.end()) {
    const int32_t g = p->num_q_heads / p->num_kv_heads;
    SideData sa, sb;
    std::vector<int64_t> work;
    if (pass == 0) {
      device_runs(p, q_idx, nq, kFwdBM, sq, kv_idx, nkv, kFwdBN, skv, true,
                  &sa.ptr, &sa.runs, &work);
      sa.order = workgroup_order(work, p->num_q_heads, g, p->num_kv_heads);
    } else {
      device_runs(p, q_idx, nq, kBwdBM, sq, kv_idx, nkv, kBwdBN, skv, true,
                  &sa.ptr, &sa.runs, &work);
      sa.order = workgroup_order(work, p->num_q_heads, g, p->num_kv_heads);
      device_runs(p, kv_idx, nkv, kBwdBN, skv, q_idx, nq, kBwdBM, sq, false,
                  &sb.ptr, &sb.runs, &work);
      sb.order = workgroup_order(work, p->num_kv_heads, 1, p->num_kv_heads);
    }
    if (g_plans.size() >= kMaxPlans) {
      auto lru = g_plans.begin();
      for (auto i = g_plans.begin(); i != g_plans.end(); ++i)
        if (i->second.last_use < lru->second.last_use) lru = i;
      g_spare.push_back(lru->second.buf);
      g_plans.erase(lru);
    }
    Plan plan;
    plan.bytes = side_bytes(sa) + (pass == 0 ? 0 : side_bytes(sb));
    ma_status_t st = take_buffer(plan.bytes, &plan.buf);
    if (st != MA_OK) return st;
    char* base = static_cast<char*>(plan.buf->host);
    side_pack(sa, base, 0, &plan.a);
    if (pass != 0) side_pack(sb, base, side_bytes(sa), &plan.b);
    it = g_plans.emplace(key, plan).first;
  }
  Plan& plan = it->second;
  plan.last_use = ++g_plan_clock;
  retire_completed(plan.buf);  // keeps the list as short as the copies in flight
  hipError_t e = hipMemcpyAsync(ws, plan.buf->host, plan.bytes,
                                hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(work list)");
  int dev = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::vector<hipEvent_t>& pool = g_free_events[dev];
  hipEvent_t ev;
  if (!pool.empty()) {
    ev = pool.back();
    pool.pop_back();
  } else {
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
  }
  e = hipEventRecord(ev, stream);
  if (e != hipSuccess) {
    pool.push_back(ev);
    return hip_fail(e, "hipEventRecord(work list)");
  }
  plan.buf->pending.push_back(PendingEvent{ev, dev});
  view->bytes = plan.bytes;
  view->a = plan.a;
  view->b = plan.b;
  return MA_OK;
}

size_t fwd_ws_bound(const ma_problem_t* p, int32_t nq, int32_t nkv) {
  const int64_t nqb = int64_t{nq} * p->partition_len / kFwdBM;
  return side_bound(nqb, nkv, p->num_q_heads);
}

size_t bwd_ws_bound(const ma_problem_t* p, int32_t nq, int32_t nkv) {
  const int64_t nqb = int64_t{nq} * p->partition_len / kBwdBM;
  const int64_t nkb = int64_t{nkv} * p->partition_len / kBwdBN;
  const int64_t rows_q = int64_t{nq} * p->partition_len;
  return side_bound(nqb, nkv, p->num_q_heads) +
         side_bound(nkb, nq, p->num_kv_heads) +
         2 * align_up(static_cast<size_t>(rows_q) * p->num_q_heads * 4);
}

ma_status_t check_head_dim(const ma_problem_t* p) {
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(MA_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)",
                p->head_dim);
  return MA_OK;
}

constexpr float kLog2e = 1.4426950408889634f;

ma_status_t check_chunk(const ma_problem_t* p, const ma_chunk_t& c, int32_t bm,
                        int32_t bn) {
  if (c.num_q_chunks < 1 || c.num_kv_chunks < 1)
    return fail(MA_ERR_INVALID_ARG, "chunk counts must be >= 1 (%d, %d)",
                c.num_q_chunks, c.num_kv_chunks);
  if (c.q_chunk < 0 || c.q_chunk >= c.num_q_chunks || c.kv_chunk < 0 ||
      c.kv_chunk >= c.num_kv_chunks)
    return fail(MA_ERR_INVALID_ARG, "chunk (%d of %d, %d of %d) out of range",
                c.q_chunk, c.num_q_chunks, c.kv_chunk, c.num_kv_chunks);
  const int64_t P = p->partition_len;
  if (P % c.num_q_chunks != 0 || (P / c.num_q_chunks) % bm != 0 ||
      P % c.num_kv_chunks != 0 || (P / c.num_kv_chunks) % bn != 0)
    return fail(MA_ERR_INVALID_ARG,
                "partition_len %lld must split into %d Q chunks of whole "
                "%d-row blocks and %d KV chunks of whole %d-row blocks",
                static_cast<long long>(P), c.num_q_chunks, bm,
                c.num_kv_chunks, bn);
  return MA_OK;
}

// Forward of one chunk pair of a tile (the whole tile: one chunk each).
ma_status_t fwd_impl(const ma_problem_t* prob, const int32_t* q_idx,
                     int32_t nq, const int32_t* kv_idx, int32_t nkv,
                     const ma_chunk_t& ch, const void* q, const void* k,
                     const void* v, void* o, bool o_f32, float* lse,
                     int32_t accumulate, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_head_dim(prob);
  if (st == MA_OK) st = check_blocks(prob, kFwdBM, kFwdBN);
  if (st == MA_OK) st = check_chunk(prob, ch, kFwdBM, kFwdBN);
  if (st != MA_OK) return st;
  const void* ptrs[] = {q, k, v, o, lse, ws};
  const char* names[] = {"q", "k", "v", "o", "lse", "ws"};
  for (int i = 0; i < 6; ++i) {
    if (!ptrs[i]) return fail(MA_ERR_INVALID_ARG, "%s is NULL", names[i]);
    if (!aligned16(ptrs[i]))
      return fail(MA_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  }
  const size_t need = fwd_ws_bound(prob, nq, nkv);
  if (ws_bytes < need)
    return fail(MA_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes < %zu",
                ws_bytes, need);
  PlanView plan;
  st = upload_plan(0, prob, q_idx, nq, kv_idx, nkv, ch, ws, stream, &plan);
  if (st != MA_OK) return st;
  char* wsb = static_cast<char*>(ws);
  FwdParams fp{};
  fp.q = static_cast<const uint16_t*>(q);
  fp.k = static_cast<const uint16_t*>(k);
  fp.v = static_cast<const uint16_t*>(v);
  fp.o = o;
  fp.lse = lse;
  fp.qblk_ptr = reinterpret_cast<const int32_t*>(wsb + plan.a.off_ptr);
  fp.runs = reinterpret_cast<const DevRun*>(wsb + plan.a.off_runs);
  fp.order = reinterpret_cast<const int2*>(wsb + plan.a.off_order);
  fp.queue = reinterpret_cast<int32_t*>(wsb + plan.a.off_queue);
  fp.n_items = plan.a.n_items;
  fp.rows_q = int64_t{nq} * (prob->partition_len / ch.num_q_chunks);
  fp.hq = prob->num_q_heads;
  fp.hkv = prob->num_kv_heads;
  fp.group = prob->num_q_heads / prob->num_kv_heads;
  fp.scale_log2 = prob->softmax_scale * kLog2e;
  fp.accumulate = accumulate;
  if (plan.a.grid == 0) return ok();  // cannot happen: every block is listed
  hipError_t e = launch_tile_fwd(
      fp, prob->head_dim, o_f32,
      static_cast<int>(queued_launch_grid(plan.a.n_items)), stream);
  if (e != hipSuccess) return hip_fail(e, "tile_fwd launch");
  return ok();
}

// Backward of one chunk pair of a tile (the whole tile: one chunk each).
ma_status_t bwd_impl(const ma_problem_t* prob, const int32_t* q_idx,
                     int32_t nq, const int32_t* kv_idx, int32_t nkv,
                     const ma_chunk_t& ch, const void* q, const void* k,
                     const void* v, const void* o, const void* d_o,
                     const float* lse, float* dq, float* dk, float* dv,
                     int32_t accumulate, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_head_dim(prob);
  if (st == MA_OK) st = check_blocks(prob, kBwdBM, kBwdBN);
  if (st == MA_OK) st = check_chunk(prob, ch, kBwdBM, kBwdBN);
  if (st != MA_OK) return st;
  if (accumulate != 0 && accumulate != 1)
    return fail(MA_ERR_INVALID_ARG, "accumulate must be 0 or 1, got %d",
                accumulate);
  const void* ptrs[] = {q, k, v, o, d_o, lse, dq, dk, dv, ws};
  const char* names[] = {"q", "k", "v", "o", "d_o", "lse", "dq", "dk", "dv",
                         "ws"};
  for (int i = 0; i < 10; ++i) {
    if (!ptrs[i]) return fail(MA_ERR_INVALID_ARG, "%s is NULL", names[i]);
    if (!aligned16(ptrs[i]))
      return fail(MA_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  }
  const size_t need = bwd_ws_bound(prob, nq, nkv);
  if (ws_bytes < need)
    return fail(MA_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes < %zu",
                ws_bytes, need);
  PlanView plan;
  st = upload_plan(1, prob, q_idx, nq, kv_idx, nkv, ch, ws, stream, &plan);
  if (st != MA_OK) return st;
  char* wsb = static_cast<char*>(ws);
  BwdParams bp{};
  bp.q = static_cast<const uint16_t*>(q);
  bp.k = static_cast<const uint16_t*>(k);
  bp.v = static_cast<const uint16_t*>(v);
  bp.o = static_cast<const uint16_t*>(o);
  bp.d_o = static_cast<const uint16_t*>(d_o);
  bp.lse = lse;
  bp.dq = dq;
  bp.dk = dk;
  bp.dv = dv;
  bp.delta = reinterpret_cast<float*>(wsb + align_up(plan.bytes));
  bp.lse2 = reinterpret_cast<float*>(
      wsb + align_up(plan.bytes) +
      align_up(static_cast<size_t>(nq) * prob->partition_len *
               prob->num_q_heads * 4));
  bp.qblk_ptr = reinterpret_cast<const int32_t*>(wsb + plan.a.off_ptr);
  bp.qruns = reinterpret_cast<const DevRun*>(wsb + plan.a.off_runs);
  bp.qorder = reinterpret_cast<const int2*>(wsb + plan.a.off_order);
  bp.kvblk_ptr = reinterpret_cast<const int32_t*>(wsb + plan.b.off_ptr);
  bp.kvruns = reinterpret_cast<const DevRun*>(wsb + plan.b.off_runs);
  bp.kvorder = reinterpret_cast<const int2*>(wsb + plan.b.off_order);
  bp.qqueue = reinterpret_cast<int32_t*>(wsb + plan.a.off_queue);
  bp.kvqueue = reinterpret_cast<int32_t*>(wsb + plan.b.off_queue);
  bp.q_items = plan.a.n_items;
  bp.kv_items = plan.b.n_items;
  bp.rows_q = int64_t{nq} * (prob->partition_len / ch.num_q_chunks);
  bp.rows_kv = int64_t{nkv} * (prob->partition_len / ch.num_kv_chunks);
  bp.hq = prob->num_q_heads;
  bp.hkv = prob->num_kv_heads;
  bp.group = prob->num_q_heads / prob->num_kv_heads;
  bp.scale = prob->softmax_scale;
  bp.scale_log2 = prob->softmax_scale * kLog2e;
  bp.accumulate = accumulate;
  hipError_t e = launch_tile_bwd(
      bp, prob->head_dim,
      plan.a.n_items > 0 ? static_cast<int>(queued_launch_grid(plan.a.n_items)) : 0,
      plan.b.n_items > 0 ? static_cast<int>(queued_launch_grid(plan.b.n_items)) : 0,
      stream);
  if (e != hipSuccess) return hip_fail(e, "tile_bwd launch");
  return ok();
}


}  // namespace

extern "C" {

const char* mesh_attn_last_error(void) { return g_last_error.c_str(); }

void mesh_attn_block_shape(int32_t head_dim, int32_t pass, int32_t* bm,
                           int32_t* bn) {
  int32_t m = 0, n = 0;
  if (head_dim == 64 || head_dim == 128) {
    if (pass == 0) {
      m = kFwdBM;
      n = kFwdBN;
    } else if (pass == 1) {
      m = kBwdBM;
      n = kBwdBN;
    }
  }
  if (bm) *bm = m;
  if (bn) *bn = n;
}

ma_status_t mesh_attn_classify(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               int32_t bm, int32_t bn, uint8_t* cls) {
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_blocks(prob, bm, bn);
  if (st != MA_OK) return st;
  if (!cls) return fail(MA_ERR_INVALID_ARG, "cls is NULL");
  const int64_t P = prob->partition_len;
  const int64_t nqb = nq * P / bm, nkb = nkv * P / bn;
  const int64_t qpb = P / bm, kpb = P / bn;
  for (int64_t qb = 0; qb < nqb; ++qb) {
    const int32_t qp = q_idx[qb / qpb];
    const int64_t q_row = (qb % qpb) * bm;
    const int64_t q_first = token_pos(prob, qp, q_row);
    const int64_t q_last = token_pos(prob, qp, q_row + bm - 1);
    for (int64_t kb = 0; kb < nkb; ++kb) {
      const int32_t kp = kv_idx[kb / kpb];
      const int64_t k_row = (kb % kpb) * bn;
      cls[qb * nkb + kb] = static_cast<uint8_t>(block_class(
          q_first, q_last, token_pos(prob, kp, k_row),
          token_pos(prob, kp, k_row + bn - 1), prob->causal != 0));
    }
  }
  return ok();
}

ma_status_t mesh_attn_worklist(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               int32_t bm, int32_t bn, int32_t* qblk_ptr,
                               ma_run_t* runs, int64_t cap, int64_t* n_runs) {
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_blocks(prob, bm, bn);
  if (st != MA_OK) return st;
  std::vector<int32_t> ptr;
  std::vector<Run> rl;
  const Slice whole{prob->partition_len, 0};
  build_runs(prob, q_idx, nq, bm, whole, kv_idx, nkv, bn, whole, true, &ptr,
             &rl);
  return export_runs(ptr, rl, qblk_ptr, runs, cap, n_runs);
}

ma_status_t mesh_attn_worklist_kv_major(const ma_problem_t* prob,
                                        const int32_t* q_idx, int32_t nq,
                                        const int32_t* kv_idx, int32_t nkv,
                                        int32_t bm, int32_t bn,
                                        int32_t* kvblk_ptr, ma_run_t* runs,
                                        int64_t cap, int64_t* n_runs) {
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_blocks(prob, bm, bn);
  if (st != MA_OK) return st;
  std::vector<int32_t> ptr;
  std::vector<Run> rl;
  const Slice whole{prob->partition_len, 0};
  build_runs(prob, kv_idx, nkv, bn, whole, q_idx, nq, bm, whole, false, &ptr,
             &rl);
  return export_runs(ptr, rl, kvblk_ptr, runs, cap, n_runs);
}

size_t mesh_attn_fwd_workspace_size(const ma_problem_t* prob, int32_t nq,
                                    int32_t nkv) {
  if (check_problem(prob) != MA_OK || nq < 1 || nkv < 1) return 0;
  return fwd_ws_bound(prob, nq, nkv);
}

size_t mesh_attn_bwd_workspace_size(const ma_problem_t* prob, int32_t nq,
                                    int32_t nkv) {
  if (check_problem(prob) != MA_OK || nq < 1 || nkv < 1) return 0;
  return bwd_ws_bound(prob, nq, nkv);
}

ma_status_t mesh_attn_tile_fwd(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               const void* q, const void* k, const void* v,
                               void* o, ma_dtype_t o_dtype, float* lse,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  if (o_dtype != MA_BF16 && o_dtype != MA_FP32)
    return fail(MA_ERR_INVALID_ARG, "o_dtype %d invalid", (int)o_dtype);
  return fwd_impl(prob, q_idx, nq, kv_idx, nkv, kWholeTile, q, k, v, o,
                  o_dtype == MA_FP32, lse, 0, ws, ws_bytes, stream);
}

size_t mesh_attn_chunk_fwd_workspace_size(const ma_problem_t* prob,
                                          int32_t nq, int32_t nkv) {
  // A chunk's work list is never longer than the whole tile's.
  return mesh_attn_fwd_workspace_size(prob, nq, nkv);
}

ma_status_t mesh_attn_chunk_fwd(const ma_problem_t* prob, const int32_t* q_idx,
                                int32_t nq, const int32_t* kv_idx, int32_t nkv,
                                const ma_chunk_t* chunk, const void* q,
                                const void* k, const void* v, float* o,
                                float* lse, int32_t accumulate, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
  if (!chunk) return fail(MA_ERR_INVALID_ARG, "chunk is NULL");
  if (accumulate != 0 && accumulate != 1)
    return fail(MA_ERR_INVALID_ARG, "accumulate must be 0 or 1, got %d",
                accumulate);
  return fwd_impl(prob, q_idx, nq, kv_idx, nkv, *chunk, q, k, v, o, true, lse,
                  accumulate, ws, ws_bytes, stream);
}

ma_status_t mesh_attn_tile_fwd_noalloc(const ma_problem_t* prob,
                                       const int32_t* q_idx, int32_t nq,
                                       const int32_t* kv_idx, int32_t nkv,
                                       const void* q, const void* k,
                                       const void* v, void* o,
                                       ma_dtype_t o_dtype, float* lse,
                                       hipStream_t stream) {
  if (o_dtype != MA_BF16 && o_dtype != MA_FP32)
    return fail(MA_ERR_INVALID_ARG, "o_dtype %d invalid", (int)o_dtype);
  ma_status_t st = check_tile(prob, q_idx, nq, kv_idx, nkv);
  if (st == MA_OK) st = check_head_dim(prob);
  if (st == MA_OK) st = check_blocks(prob, kFwdBM, kFwdBN);
  if (st != MA_OK) return st;
  const void* ptrs[] = {q, k, v, o, lse};
  const char* names[] = {"q", "k", "v", "o", "lse"};
  for (int i = 0; i < 5; ++i) {
    if (!ptrs[i]) return fail(MA_ERR_INVALID_ARG, "%s is NULL", names[i]);
    if (!aligned16(ptrs[i]))
      return fail(MA_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  }
  if (nq > kNoAllocMaxList || nkv > kNoAllocMaxList)
    return fail(MA_ERR_UNSUPPORTED,
                "noalloc forward: index lists of %d and %d partitions exceed "
                "the maximum of %d", nq, nkv, kNoAllocMaxList);
  const int64_t nqb = int64_t{nq} * prob->partition_len / kFwdBM;
  const size_t need = fwd_ws_bound(prob, nq, nkv);
  if (nqb > kNoAllocMaxQBlocks || need > kNoAllocScratchBytes)
    return fail(MA_ERR_UNSUPPORTED,
                "noalloc forward: the tile's work list (%lld Q blocks, %zu "
                "bytes) exceeds the scratch maximum (%d Q blocks, %zu bytes)",
                static_cast<long long>(nqb), need, kNoAllocMaxQBlocks,
                kNoAllocScratchBytes);
  void* scratch = nullptr;
  hipError_t e = noalloc_scratch(&scratch);
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
  // Same regions as the uploaded plan: Q-block pointers, runs, order.
  char* base = static_cast<char*>(scratch);
  const size_t off_runs = align_up(static_cast<size_t>(nqb + 1) * 4);
  const size_t off_order =
      off_runs + align_up(static_cast<size_t>(nqb) * nkv * 2 * sizeof(DevRun));
  const int64_t items = nqb * prob->num_q_heads;
  const bool by_kv = prob->num_kv_heads % kNumXcd == 0;
  const int64_t grid = by_kv ? items : (items + kNumXcd - 1) / kNumXcd * kNumXcd;
  if (grid > INT32_MAX)
    return fail(MA_ERR_UNSUPPORTED, "noalloc forward: %lld workgroups",
                static_cast<long long>(grid));
  PlanBuildParams bp{};
  bp.P = prob->partition_len;
  bp.n = prob->num_partitions;
  bp.layout = prob->layout;
  bp.causal = prob->causal;
  bp.nq = nq;
  bp.nkv = nkv;
  bp.hq = prob->num_q_heads;
  bp.hkv = prob->num_kv_heads;
  bp.group = prob->num_q_heads / prob->num_kv_heads;
  bp.bm = kFwdBM;
  bp.bn = kFwdBN;
  bp.nqb = static_cast<int32_t>(nqb);
  bp.nkbp = prob->partition_len / kFwdBN;
  bp.grid = static_cast<int32_t>(grid);
  bp.qblk_ptr = reinterpret_cast<int32_t*>(base);
  bp.runs = reinterpret_cast<DevRun*>(base + off_runs);
  bp.order = reinterpret_cast<int2*>(base + off_order);
  bp.queue = reinterpret_cast<int32_t*>(
      base + off_order + align_up(static_cast<size_t>(grid) * sizeof(int2)));
  for (int32_t i = 0; i < nq; ++i) bp.q_idx[i] = q_idx[i];
  for (int32_t i = 0; i < nkv; ++i) bp.kv_idx[i] = kv_idx[i];
  e = launch_fwd_plan_build(bp, stream);
  if (e != hipSuccess) return hip_fail(e, "noalloc work-list build launch");
  FwdParams fp{};
  fp.q = static_cast<const uint16_t*>(q);
  fp.k = static_cast<const uint16_t*>(k);
  fp.v = static_cast<const uint16_t*>(v);
  fp.o = o;
  fp.lse = lse;
  fp.qblk_ptr = bp.qblk_ptr;
  fp.runs = bp.runs;
  fp.order = bp.order;
  fp.queue = bp.queue;
  fp.n_items = static_cast<int32_t>(items);
  fp.rows_q = int64_t{nq} * prob->partition_len;
  fp.hq = prob->num_q_heads;
  fp.hkv = prob->num_kv_heads;
  fp.group = bp.group;
  fp.scale_log2 = prob->softmax_scale * kLog2e;
  fp.accumulate = 0;
  e = launch_tile_fwd(fp, prob->head_dim, o_dtype == MA_FP32,
                      static_cast<int>(queued_launch_grid(items)), stream);
  if (e != hipSuccess) return hip_fail(e, "tile_fwd launch");
  return ok();
}

ma_status_t mesh_attn_lse_merge(int32_t k_parts, int64_t rows, int32_t heads,
                                int32_t head_dim, const void* o_parts,
                                ma_dtype_t in_dtype, const float* lse_parts,
                                void* o_out, ma_dtype_t out_dtype,
                                float* lse_out, hipStream_t stream) {
  if (k_parts < 1 || k_parts > 4096)
    return fail(MA_ERR_INVALID_ARG, "k_parts %d outside [1, 4096]", k_parts);
  if (rows < 0) return fail(MA_ERR_INVALID_ARG, "rows %lld < 0", (long long)rows);
  if (heads < 1) return fail(MA_ERR_INVALID_ARG, "heads %d < 1", heads);
  if (head_dim < 8 || head_dim > 256 || head_dim % 8 != 0)
    return fail(MA_ERR_UNSUPPORTED, "head_dim %d: need a multiple of 8 in "
                "[8, 256]", head_dim);
  if ((in_dtype != MA_BF16 && in_dtype != MA_FP32) ||
      (out_dtype != MA_BF16 && out_dtype != MA_FP32))
    return fail(MA_ERR_INVALID_ARG, "dtype invalid (in %d, out %d)",
                (int)in_dtype, (int)out_dtype);
  if (rows == 0) return ok();
  const void* ptrs[] = {o_parts, lse_parts, o_out, lse_out};
  const char* names[] = {"o_parts", "lse_parts", "o_out", "lse_out"};
  for (int i = 0; i < 4; ++i) {
    if (!ptrs[i]) return fail(MA_ERR_INVALID_ARG, "%s is NULL", names[i]);
    if (!aligned16(ptrs[i]))
      return fail(MA_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  }
  if (rows * heads > (int64_t{1} << 40))
    return fail(MA_ERR_INVALID_ARG, "rows * heads too large");
  MergeParams mp{o_parts, lse_parts, o_out, lse_out, rows, k_parts, heads,
                 head_dim};
  hipError_t e = launch_lse_merge(mp, in_dtype == MA_FP32,
                                  out_dtype == MA_FP32, stream);
  if (e != hipSuccess) return hip_fail(e, "lse_merge launch");
  return ok();
}

ma_status_t mesh_attn_tile_bwd(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               const void* q, const void* k, const void* v,
                               const void* o, const void* d_o,
                               const float* lse, float* dq, float* dk,
                               float* dv, int32_t accumulate, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  return bwd_impl(prob, q_idx, nq, kv_idx, nkv, kWholeTile, q, k, v, o, d_o,
                  lse, dq, dk, dv, accumulate, ws, ws_bytes, stream);
}

size_t mesh_attn_chunk_bwd_workspace_size(const ma_problem_t* prob,
                                          int32_t nq, int32_t nkv) {
  // A chunk's work lists and row buffers never exceed the whole tile's.
  return mesh_attn_bwd_workspace_size(prob, nq, nkv);
}

ma_status_t mesh_attn_chunk_bwd(const ma_problem_t* prob, const int32_t* q_idx,
                                int32_t nq, const int32_t* kv_idx, int32_t nkv,
                                const ma_chunk_t* chunk, const void* q,
                                const void* k, const void* v, const void* o,
                                const void* d_o, const float* lse, float* dq,
                                float* dk, float* dv, int32_t accumulate,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!chunk) return fail(MA_ERR_INVALID_ARG, "chunk is NULL");
  return bwd_impl(prob, q_idx, nq, kv_idx, nkv, *chunk, q, k, v, o, d_o, lse,
                  dq, dk, dv, accumulate, ws, ws_bytes, stream);
}

}  // extern "C"
