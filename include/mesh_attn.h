/*
 * mesh_attn.h -- C ABI of the single-GPU tile compute of Mesh-Attention
 * (arXiv 2512.20968) for AMD Instinct MI355X (gfx950).
 *
 * In Mesh-Attention every GPU owns a 2-D tile of the Q-KV interaction matrix:
 * a list of Q partitions times a list of KV partitions (the footprints
 * I_g^Q, I_g^KV of Section 3.1).  After the all-gathers of Algorithm 2 the GPU
 * computes attention for every (Q_u, KV_v) pair of its tile and merges the
 * partial results with the online-softmax reducer; after those of Algorithm 3
 * it computes the partial gradients of every pair.  This library is that
 * per-GPU compute.  The collectives around it are not part of it.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - The sequence of num_partitions (n) * partition_len (P) tokens is split
 *    into n partitions of P tokens.  The problem's layout fixes the global
 *    position of token r of partition p: p * P + r (MA_LAYOUT_CONTIGUOUS) or
 *    r * n + p (MA_LAYOUT_STRIPED).  The causal rule (Section 3.7) lets a
 *    query see a key iff key position <= query position.
 *  - A tile buffer stacks its partitions in the order of its index list: row
 *    a * P + r of the Q buffer is token r of partition q_idx[a] (the order an
 *    all-gather over the Q group delivers).  The same holds for the KV side.
 *  - Q, O, dO, dQ are [nq * P][num_q_heads][head_dim]; K, V, dK, dV are
 *    [nkv * P][num_kv_heads][head_dim]; LSE is [num_q_heads][rows], float32,
 *    natural log.  All dense, row-major, no padding.
 *  - GQA (Section 4.8): query head h reads KV head h / (num_q_heads /
 *    num_kv_heads).
 *  - Device pointers must be 16-byte aligned.  Outputs must not alias inputs.
 *  - A call writes its device workspace on `stream` (the work list and the
 *    counters its workgroups take items from) and reads it back in its
 *    kernels, so a workspace serves one call at a time: calls that may
 *    overlap need workspaces of their own.  The work list is copied from a
 *    cached pinned host buffer that the library may reuse for another tile
 *    after the copy has completed, so calls that take a workspace must not
 *    be recorded into a graph (stream capture) and replayed;
 *    mesh_attn_tile_fwd_noalloc is the forward for that case.
 *  - The caller owns every buffer, host and device.  The library never
 *    allocates or frees device memory and never synchronizes a stream or the
 *    device; its only state is a bounded cache of pinned host copies of work
 *    lists (guarded by a mutex).  A cached copy is released only after the
 *    device has finished every upload from it (an event recorded after each
 *    upload, polled without waiting).
 *  - Arguments are validated on the host before anything is enqueued.  On a
 *    non-OK status nothing was launched and mesh_attn_last_error() describes
 *    the problem.  Device work runs asynchronously on `stream`, which must
 *    belong to the current device (the work-list copy and its event are
 *    made there); a launch failure returns MA_ERR_HIP.
 */
#ifndef MESH_ATTN_H
#define MESH_ATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MA_OK = 0,
  MA_ERR_INVALID_ARG = 1,         /* bad size, index, flag or pointer */
  MA_ERR_UNSUPPORTED = 2,         /* valid request the library does not serve */
  MA_ERR_WORKSPACE_TOO_SMALL = 3, /* ws_bytes below the *_workspace_size() */
  MA_ERR_HIP = 4,                 /* HIP runtime error, text in last_error */
  MA_ERR_CAPACITY = 5             /* caller-provided output array too small */
} ma_status_t;

typedef enum { MA_BF16 = 0, MA_FP32 = 1 } ma_dtype_t;

/* Block classes of a (Q block, KV block) pair under the causal rule. */
enum { MA_CLS_EMPTY = 0, MA_CLS_PARTIAL = 1, MA_CLS_FULL = 2 };

/* Sequence layout: which global position token r of partition p holds (it
 * matters only for causal problems, Section 3.7).
 *   MA_LAYOUT_CONTIGUOUS: position p * P + r (the even split of Section 2.2).
 *   MA_LAYOUT_STRIPED:    position r * n + p (positions dealt round robin over
 *                         the n partitions, the striped layout Section 3.7
 *                         adopts to balance causal work across tiles). */
typedef enum { MA_LAYOUT_CONTIGUOUS = 0, MA_LAYOUT_STRIPED = 1 } ma_layout_t;

typedef struct {
  int32_t num_partitions; /* n: partitions of the whole sequence, >= 1        */
  int32_t partition_len;  /* P: tokens per partition, multiple of the blocks  */
  int32_t num_q_heads;    /* Hq >= 1                                         */
  int32_t num_kv_heads;   /* Hkv >= 1, divides Hq                            */
  int32_t head_dim;       /* d: 64 or 128                                    */
  int32_t causal;         /* 0 or 1; a key is visible to a query iff its
                             position is not larger (causal problems)        */
  int32_t layout;         /* an ma_layout_t value                            */
  float softmax_scale;    /* s > 0, finite; usually 1/sqrt(d)                */
} ma_problem_t;

/* ---------------------------------------------------------------------------
 * Work list (host only, deterministic).
 *
 * The tile's Q buffer is cut into Q blocks of bm rows, its KV buffer into KV
 * blocks of bn rows (both divide P, so no block straddles partitions).  Q
 * block a*(P/bm)+qb is block qb of list entry a.  A (Q block, KV block) pair is
 * EMPTY if no (query, key) pair in it is visible under the causal rule
 * (Section 3.7), FULL if every pair is (always, without a mask), PARTIAL
 * otherwise.  Fully masked pairs are skipped by the kernels; PARTIAL pairs are
 * the only ones that evaluate the per-element mask.
 * ------------------------------------------------------------------------- */

/* Block shape (rows per Q block, rows per KV block) the kernels of `pass`
 * (0 = forward, 1 = backward) use for `head_dim`; both are 0 for an
 * unsupported head_dim or pass. */
void mesh_attn_block_shape(int32_t head_dim, int32_t pass, int32_t* bm,
                           int32_t* bn);

/* Class of every block pair into cls[(nq*P/bm) * (nkv*P/bn)] (row-major, Q
 * block major), values MA_CLS_*.  q_idx, kv_idx are host arrays of distinct
 * partition indices in [0, num_partitions). */
ma_status_t mesh_attn_classify(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               int32_t bm, int32_t bn, uint8_t* cls);

/* One run of the work list: the KV blocks [kb_begin, kb_end) of KV list
 * entry kv_list_pos (blocks counted within that partition) against Q block
 * qblk (counted in the tile's Q buffer), all of class cls (MA_CLS_PARTIAL or
 * MA_CLS_FULL).  In the KV-major list the roles of the sides swap (see
 * mesh_attn_worklist_kv_major). */
typedef struct {
  int32_t qblk, kv_list_pos, kb_begin, kb_end, cls;
} ma_run_t;

/* Canonical Q-major run list.  For every Q block in buffer order, for every
 * KV list entry b in list order, the maximal runs of consecutive KV blocks kb
 * (ascending) of equal class, EMPTY runs dropped, as ma_run_t
 * {qblk, b, kb_begin, kb_end exclusive, cls}.  qblk_ptr[q] (nq*P/bm + 1
 * entries) is the first run of Q block q and its last entry the run count.
 * cap is the capacity of runs in ma_run_t entries; if it is too small,
 * *n_runs gets the required count and MA_ERR_CAPACITY is returned.  A NULL
 * runs with cap 0 queries the count. */
ma_status_t mesh_attn_worklist(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               int32_t bm, int32_t bn, int32_t* qblk_ptr,
                               ma_run_t* runs, int64_t cap, int64_t* n_runs);

/* KV-major mirror: the same rule with the sides swapped.  For every KV block
 * in buffer order, for every Q list entry a, runs of Q blocks; each ma_run_t
 * then holds {KV block, a, qb_begin, qb_end, cls} in the fields
 * {qblk, kv_list_pos, kb_begin, kb_end, cls}.  kvblk_ptr has nkv*P/bn + 1
 * entries. */
ma_status_t mesh_attn_worklist_kv_major(const ma_problem_t* prob,
                                        const int32_t* q_idx, int32_t nq,
                                        const int32_t* kv_idx, int32_t nkv,
                                        int32_t bm, int32_t bn,
                                        int32_t* kvblk_ptr, ma_run_t* runs,
                                        int64_t cap, int64_t* n_runs);

/* ---------------------------------------------------------------------------
 * Forward (Algorithm 2, the per-pair loop; attention as defined in Section
 * 2.1, partial (O, lse) as in Section 2.2, merged over the tile's KV footprint
 * with the online-softmax reducer inside the kernel).
 * ------------------------------------------------------------------------- */

/* Device workspace bytes mesh_attn_tile_fwd needs for this tile. */
size_t mesh_attn_fwd_workspace_size(const ma_problem_t* prob, int32_t nq,
                                    int32_t nkv);

/* O and LSE of every Q row of the tile over every key of the tile.
 *   q       [nq*P][Hq][d] bf16 device;  k, v [nkv*P][Hkv][d] bf16 device.
 *   o       [nq*P][Hq][d] device, bf16 (o_dtype MA_BF16, the final output) or
 *           float32 (MA_FP32, a partial to be merged exactly later).
 *   lse     [Hq][nq*P] float32 device; -inf for a row that sees no key, whose
 *           O row is then 0.
 *   ws      device workspace of ws_bytes >= mesh_attn_fwd_workspace_size().
 * O = sum_j exp(x_j - LSE) v_j with x_j = s <q, k_j> over the visible keys;
 * LSE = ln sum_j exp(x_j).  bf16 MFMA products, float32 accumulation and
 * softmax. */
ma_status_t mesh_attn_tile_fwd(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               const void* q, const void* k, const void* v,
                               void* o, ma_dtype_t o_dtype, float* lse,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* Maximum size of the scratch array of mesh_attn_tile_fwd_noalloc, per GPU. */
#define MA_NOALLOC_SCRATCH_BYTES (8u << 20)
/* Longest index list, and most forward Q blocks (nq * P / 256), it serves. */
#define MA_NOALLOC_MAX_LIST 256
#define MA_NOALLOC_MAX_QBLOCKS 4096

/* mesh_attn_tile_fwd for callers that cannot allocate memory: code under
 * stream (graph) capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments and results as mesh_attn_tile_fwd without the
 * workspace: the work list is built on the device (from the index lists,
 * passed by value as kernel arguments) into a scratch array of
 * MA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends.  The call allocates nothing (no hipMalloc, no
 * pinned host memory, no host heap), copies nothing from the host and never
 * synchronizes.
 * Limits: nq, nkv <= MA_NOALLOC_MAX_LIST; nq * P / 256 <= MA_NOALLOC_MAX_QBLOCKS;
 * the tile's work list (mesh_attn_fwd_workspace_size bytes) must fit the
 * scratch array.  Larger tiles return MA_ERR_UNSUPPORTED with the sizes in
 * mesh_attn_last_error(), before anything is launched.
 * Every call on one GPU shares that GPU's scratch array (each call rewrites
 * it before reading it): calls on one stream are ordered, but calls that
 * overlap on one GPU (different streams without ordering between them) race
 * and give undefined results. */
ma_status_t mesh_attn_tile_fwd_noalloc(const ma_problem_t* prob,
                                       const int32_t* q_idx, int32_t nq,
                                       const int32_t* kv_idx, int32_t nkv,
                                       const void* q, const void* k,
                                       const void* v, void* o,
                                       ma_dtype_t o_dtype, float* lse,
                                       hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Greedy Overlapping Optimization (GOO, Section 3.4): chunk compute tasks and
 * the step planner.  Each Q partition of the tile is cut into k_Q chunks of
 * P / k_Q rows and each KV partition into k_KV chunks of P / k_KV rows along
 * the sequence; the chunk collectives AG-Q-i, AG-KV-j and RS-Q-i replace the
 * whole-tile all-gathers and reduce-scatter, and compute task C-i-j attends
 * Q chunk i of every Q partition to KV chunk j of every KV partition.
 * ------------------------------------------------------------------------- */

typedef struct {
  int32_t q_chunk;       /* i in [0, num_q_chunks)                           */
  int32_t num_q_chunks;  /* k_Q >= 1; P / k_Q a multiple of the Q block rows */
  int32_t kv_chunk;      /* j in [0, num_kv_chunks)                          */
  int32_t num_kv_chunks; /* k_KV >= 1; P / k_KV a multiple of the KV block
                            rows (see mesh_attn_block_shape, pass 0)         */
} ma_chunk_t;

/* Device workspace bytes mesh_attn_chunk_fwd needs (any chunk of the tile). */
size_t mesh_attn_chunk_fwd_workspace_size(const ma_problem_t* prob,
                                          int32_t nq, int32_t nkv);

/* Compute task C-i-j of the tile, as a running partial.
 *   q     [nq*P/k_Q][Hq][d] bf16 device: chunk i of every Q partition in q_idx
 *         order (the buffer AG-Q-i produces; row a*P/k_Q + r is local row
 *         i*P/k_Q + r of partition q_idx[a]).
 *   k, v  [nkv*P/k_KV][Hkv][d] bf16 device: chunk j of every KV partition in
 *         kv_idx order (the buffer AG-KV-j produces).
 *   o     [nq*P/k_Q][Hq][d] float32 device;  lse [Hq][nq*P/k_Q] float32.
 *   accumulate  0: write the (O, LSE) of this chunk pair (O = 0, LSE = -inf
 *               for a row that sees no key of it);
 *               1: fold it into the (O, LSE) already in o, lse with the
 *               online-softmax reducer (running accumulation over j), so
 *               that after C-i-0 .. C-i-(k_KV-1) they hold Q chunk i's result
 *               over the tile's whole KV footprint, ready for RS-Q-i.
 * Positions, the causal rule and the layout are those of the whole problem:
 * the result is exactly the tile's on these rows and keys.  Errors: as
 * mesh_attn_tile_fwd, and MA_ERR_INVALID_ARG for a chunk outside its count or
 * counts that do not divide P into whole blocks. */
ma_status_t mesh_attn_chunk_fwd(const ma_problem_t* prob, const int32_t* q_idx,
                                int32_t nq, const int32_t* kv_idx, int32_t nkv,
                                const ma_chunk_t* chunk, const void* q,
                                const void* k, const void* v, float* o,
                                float* lse, int32_t accumulate, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/* Device workspace bytes mesh_attn_chunk_bwd needs (any chunk of the tile). */
size_t mesh_attn_chunk_bwd_workspace_size(const ma_problem_t* prob,
                                          int32_t nq, int32_t nkv);

/* Backward of compute task C-i-j (the per-pair loop of Algorithm 3 over one
 * chunk pair).  Buffers as in mesh_attn_chunk_fwd: q, o, d_o
 * [nq*P/k_Q][Hq][d] bf16 (chunk i of every Q partition), lse [Hq][nq*P/k_Q]
 * (the FINAL LSE of those rows, over the whole key set, with the final O);
 * k, v [nkv*P/k_KV][Hkv][d] bf16 (chunk j of every KV partition); dq like q,
 * dk and dv like k, float32.  accumulate 0 overwrites, 1 adds: the tile's dQ
 * on Q chunk i is the sum of C-i-j over j and its dK, dV on KV chunk j the sum
 * over i, so a caller zeroes the gradients and accumulates, or orders the
 * tasks so that each buffer's first task overwrites.  Errors as
 * mesh_attn_tile_bwd, plus those of the chunk (mesh_attn_chunk_fwd; the
 * block rows are those of pass 1). */
ma_status_t mesh_attn_chunk_bwd(const ma_problem_t* prob, const int32_t* q_idx,
                                int32_t nq, const int32_t* kv_idx, int32_t nkv,
                                const ma_chunk_t* chunk, const void* q,
                                const void* k, const void* v, const void* o,
                                const void* d_o, const float* lse, float* dq,
                                float* dk, float* dv, int32_t accumulate,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/* Kinds of the collective a GOO step runs. */
enum { MA_GOO_NONE = 0, MA_GOO_AG_Q = 1, MA_GOO_AG_KV = 2, MA_GOO_RS_Q = 3 };

typedef struct {
  int32_t comm_kind;   /* MA_GOO_*; MA_GOO_NONE for a compute-only step     */
  int32_t comm_chunk;  /* chunk index of the collective (-1 if none)        */
  int32_t first_task;  /* this step's tasks are tasks[first_task ..         */
  int32_t num_tasks;   /*   first_task + num_tasks) of the task list        */
} ma_goo_step_t;

/* Step-based greedy schedule of one tile's chunk tasks (host only,
 * deterministic: every GPU of a mesh that calls it with the same shared costs
 * gets the same collective order).  Each step runs one collective and the
 * compute tasks listed for it, all ready when the step starts:
 *   - its collective is, among every chunk collective that can run (each
 *     AG-Q-i and AG-KV-j not yet run, each RS-Q-i not yet run whose C-i-j
 *     are all done), the one with the largest (time of the compute it makes
 *     ready) / (its time); ties go to the one that makes more compute ready,
 *     then to AG-KV, AG-Q, RS-Q in that order, then to the lower chunk index;
 *   - its compute tasks are the ready ones in (i, j) order until their time
 *     reaches gamma times the collective's time;
 *   - when no collective can run, a compute-only step runs one ready task.
 *   t_ag_q, t_ag_kv, t_rs_q  time of one chunk collective of each kind, > 0.
 *   t_c         host [k_q][k_kv] float64, time of each C-i-j, >= 0.
 *   steps       host array of max_steps entries (2 k_q + k_kv + k_q k_kv
 *               always suffice); *num_steps receives the count.
 *   tasks       host int32 [k_q * k_kv][2]: (i, j) in execution order.
 * Errors: MA_ERR_INVALID_ARG for counts < 1 or k_q * k_kv > 4096, times that
 * are not finite or not positive, NULL pointers; MA_ERR_CAPACITY if max_steps
 * is too small. */
ma_status_t mesh_attn_goo_plan(int32_t k_q, int32_t k_kv, double t_ag_q,
                               double t_ag_kv, double t_rs_q,
                               const double* t_c, double gamma,
                               ma_goo_step_t* steps, int32_t max_steps,
                               int32_t* tasks, int32_t* num_steps);

/* ---------------------------------------------------------------------------
 * Online-softmax reducer (Section 2.2; the reducer of Algorithm 2's
 * reduce-scatter).  Folds k_parts partial results of the same rows over
 * disjoint key sets:  M = max_k lse_k,  lse = M + ln sum_k exp(lse_k - M),
 * O = sum_k exp(lse_k - lse) O_k.  Parts with lse = -inf weigh 0; a row whose
 * parts are all -inf gets O = 0, lse = -inf.
 *   o_parts   [k_parts][rows][heads][head_dim] device, in_dtype.
 *   lse_parts [k_parts][heads][rows] float32 device.
 *   o_out     [rows][heads][head_dim] device, out_dtype.
 *   lse_out   [heads][rows] float32 device.
 * head_dim must be a multiple of 8 (16-byte vectors) and at most 256;
 * rows >= 0 (0 launches nothing), 1 <= k_parts <= 4096.
 * ------------------------------------------------------------------------- */
ma_status_t mesh_attn_lse_merge(int32_t k_parts, int64_t rows, int32_t heads,
                                int32_t head_dim, const void* o_parts,
                                ma_dtype_t in_dtype, const float* lse_parts,
                                void* o_out, ma_dtype_t out_dtype,
                                float* lse_out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Backward (Algorithm 3, the per-pair loop, summed over the tile).
 * ------------------------------------------------------------------------- */

/* Device workspace bytes mesh_attn_tile_bwd needs for this tile. */
size_t mesh_attn_bwd_workspace_size(const ma_problem_t* prob, int32_t nq,
                                    int32_t nkv);

/* Gradients of <dO, O> for the tile, given the FINAL O and LSE of its Q rows
 * (those of the full key set, as gathered in Algorithm 3).
 *   q, o, d_o  [nq*P][Hq][d] bf16 device;  k, v [nkv*P][Hkv][d] bf16 device.
 *   lse        [Hq][nq*P] float32 device.
 *   dq         [nq*P][Hq][d] float32 device;  dk, dv [nkv*P][Hkv][d] float32.
 *   accumulate 0: overwrite dq, dk, dv;  1: add into them.
 * With P_ij = exp(s <q_i,k_j> - LSE_i) over visible pairs, D_i = <dO_i, O_i>:
 * dV_j = sum_i P_ij dO_i;  dS_ij = P_ij (<dO_i, v_j> - D_i);
 * dQ_i = s sum_j dS_ij k_j;  dK_j = s sum_i dS_ij q_i.  Under GQA dK, dV of a
 * KV head sum over its query heads.  Deterministic (no atomics). */
ma_status_t mesh_attn_tile_bwd(const ma_problem_t* prob, const int32_t* q_idx,
                               int32_t nq, const int32_t* kv_idx, int32_t nkv,
                               const void* q, const void* k, const void* v,
                               const void* o, const void* d_o,
                               const float* lse, float* dq, float* dk,
                               float* dv, int32_t accumulate, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/* Text of the last non-OK status returned on the calling thread ("" if none).
 * The pointer stays valid until the next library call on that thread. */
const char* mesh_attn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MESH_ATTN_H */
