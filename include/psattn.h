/*
 * psattn.h -- prefix-shared causal attention, forward and backward, on one
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (psRL, arXiv 2608.25683):
 *   A batch of training samples forms a prefix forest: every node is one
 *   shared token segment whose K/V is stored once, and every sample is a
 *   root-to-node path (Sec. 2.3 sampling modes; Sec. 5.2, each tree node is a
 *   KV block and common prefixes merge).  Attention masking (Sec. 2.5): a
 *   token at position a of node n attends to every token of n's strict
 *   ancestors and to tokens 0..a of n, so the shared result equals
 *   independent causal attention over each sample.  K/V are located through
 *   per-block metadata {base, size, position, reference count} (Sec. 6,
 *   "Adaptive KV cache manager" and "Prefix-sharing training runtime"), with
 *   block sizes that follow the shared spans (Sec. 5.1, adaptive block
 *   allocation).  The backward pass takes the accumulated adjoint of every
 *   consumer of a shared token and runs once (Sec. 6, training runtime).
 *
 * Layouts (row-major, all device pointers 16-byte aligned):
 *   Q, O, dO        [Ns][Hq][d]      Ns = sum of internal segment lengths, rows of node
 *                                    i at row_off[i] .. row_off[i]+seg_len[i]-1
 *   dQ              [Ns][Hq][d]      fp32
 *   K, V            [pool_slots][Hkv][d]   token t of a block at slot base+t
 *   dK, dV          [pool_slots][Hkv][d]   fp32; written for the tokens of
 *                                    internal nodes, added to for the tokens of
 *                                    external nodes (the accumulators of cached
 *                                    blocks, complete once the block's last
 *                                    consuming call has run: Sec. 5.2), zero on
 *                                    the unused slots of internal nodes' blocks;
 *                                    every other slot is left untouched
 *   LSE             [Hq][Ns]         fp32, natural log of the softmax
 *                                    denominator (scale included)
 *   dtype PSATTN_BF16: Q/K/V/O/dO bf16; LSE/dQ/dK/dV fp32.
 *   dtype PSATTN_FP32: every tensor fp32.
 *   Query head h reads key/value head h / (Hq/Hkv).
 *
 * Ownership: the caller owns every device buffer (inputs, outputs, the plan
 * buffer given to psattn_tree_upload, and the workspaces).  The library owns
 * only the host-side psattn_tree.  psattn_fwd / psattn_bwd allocate nothing,
 * never synchronise, and enqueue their kernels on the given stream (a
 * hipStream_t passed as void*, NULL = the null stream); a device fault inside
 * a kernel surfaces at the caller's next synchronisation.  A tree is
 * immutable after creation; calls on different streams are safe with
 * distinct workspaces and outputs.
 *
 * Errors: every call returns a psattn_status; on failure nothing is
 * enqueued, no output of *out is set, and psattn_last_error() (thread-local)
 * holds a message naming the offending field.  No C++ exception crosses this
 * interface.
 */
#ifndef PSATTN_H
#define PSATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PSATTN_OK = 0,
  PSATTN_E_INVALID_ARG = -1,     /* null pointer, bad count or option */
  PSATTN_E_INVALID_TREE = -2,    /* parent order, empty segment, row layout, sample, refcount */
  PSATTN_E_BLOCK_RANGE = -3,     /* block outside the pool, or len > capacity */
  PSATTN_E_BLOCK_OVERLAP = -4,   /* two blocks share a pool slot */
  PSATTN_E_BLOCK_COVERAGE = -5,  /* blocks do not cover a node's tokens exactly, or pos mismatch */
  PSATTN_E_UNSUPPORTED = -6,     /* head_dim, dtype or size outside what the kernels handle */
  PSATTN_E_WORKSPACE = -7,       /* workspace or plan buffer too small */
  PSATTN_E_ALIGNMENT = -8,       /* device pointer not 16-byte aligned */
  PSATTN_E_HIP = -9,             /* a HIP runtime call failed (message has the HIP error) */
  PSATTN_E_NOT_UPLOADED = -10,   /* psattn_fwd/bwd called before psattn_tree_upload */
  PSATTN_E_INTERNAL = -11        /* plan consistency check failed (builds with PSATTN_PLAN_CHECKS) */
} psattn_status;

typedef enum { PSATTN_BF16 = 0, PSATTN_FP32 = 1 } psattn_dtype;

/* One page-table entry: the per-block metadata of Sec. 6 (base address,
 * block size, position of the token segment in the full sequence, reference
 * count).  A node's blocks are listed in token order. */
typedef struct {
  int64_t base;      /* first pool slot of the block */
  int32_t capacity;  /* slots reserved for the block (its size) */
  int32_t len;       /* tokens held, 1..capacity, in slots base..base+len-1 */
  int32_t pos;       /* sequence position of the block's first token (sum of
                        ancestor lengths + tokens of earlier blocks of the node) */
  int32_t refcount;  /* 0 = not given; otherwise must equal the number of
                        samples whose path holds the block (Sec. 5.2) */
} psattn_block;

typedef struct {
  int32_t num_nodes;
  const int32_t* parent;      /* [num_nodes]; parent[i] < i, or -1 for a root (forests allowed) */
  const int32_t* seg_len;     /* [num_nodes]; >= 1 */
  const int64_t* row_off;     /* [num_nodes]; the row ranges of the internal nodes must tile
                                 [0, Ns) exactly.  row_off[i] = -1 marks an external node:
                                 one an earlier call computed (Sec. 4.1.1 inter-batch sharing,
                                 Sec. 4.1.2 self-sequence sharing).  Its K/V are read from its
                                 blocks, it has no query rows here, its parent (if any) must be
                                 external too, no sample may end at it, and the backward adds
                                 this call's share of its dK/dV to what dK/dV already hold. */
  const int32_t* blk_ptr;     /* [num_nodes+1]; node i owns blocks[blk_ptr[i] .. blk_ptr[i+1]) */
  const psattn_block* blocks;
  int64_t pool_slots;         /* slots in the K/V pool (< 2^31) */
  int32_t num_samples;
  const int32_t* sample_end;  /* [num_samples]; endpoint node of each sample's path */
  int32_t hq, hkv, head_dim;  /* Hq % Hkv == 0; head_dim 64 or 128 */
  float softmax_scale;        /* > 0, finite; usually 1/sqrt(head_dim) */
  psattn_dtype dtype;
} psattn_tree_desc;

/* Planner knobs.  Zero-initialise for the defaults. */
typedef struct {
  int32_t fwd_kv_split;   /* 0 auto; > 0 max keys per forward work item (rounded up to 64); < 0 never split */
  int32_t bwd_q_chunk;    /* 0 auto; > 0 max query rows per dK/dV work item (rounded up to 32); < 0 never split */
  int32_t num_cus;        /* compute units to balance for; 0 = 256 */
  int32_t reserved[5];    /* must be 0 */
} psattn_plan_opts;

/* Opaque handle: a validated tree, its page-table view and its work plan. */
typedef struct psattn_tree psattn_tree;

/* Summary of a planned tree (host-side figures). */
typedef struct {
  int64_t num_rows;         /* Ns */
  int64_t unshared_tokens;  /* Nu = sum over samples of path length */
  int64_t visible_pairs;    /* sum over rows of visible keys (per query head) */
  int64_t fwd_items, fwd_merges, bkv_items, bkv_reduces, pad_slots;
  int64_t fwd_partial_rows, bkv_partial_tiles;
  int64_t plan_bytes;       /* == psattn_tree_device_bytes */
  int32_t q_tile_rows, kv_tile_keys, bkv_tile_keys, head_chunk;
} psattn_tree_info;

/* Validate a descriptor, build the page-table view and the work plan (host
 * only; no GPU call).  Sec. 5.2 (reference counts from the prefix tree),
 * Sec. 4.2 Eq. "single_sequence" and greedy placement (cost model and
 * longest-first ordering of work items).  opts may be NULL. */
psattn_status psattn_tree_create(const psattn_tree_desc* desc, const psattn_plan_opts* opts,
                                 psattn_tree** out);
void psattn_tree_destroy(psattn_tree* tree);

/* Bytes of device memory the plan needs (caller allocates, >= 256-byte aligned). */
psattn_status psattn_tree_device_bytes(const psattn_tree* tree, size_t* bytes);

/* Copy the plan into dev_buf on stream and wait for the copy.  Must precede
 * psattn_fwd/psattn_bwd; dev_buf must outlive every later call on the tree. */
psattn_status psattn_tree_upload(psattn_tree* tree, void* dev_buf, size_t bytes, void* stream);

/* Workspace bytes for pass 0 (psattn_fwd) or 1 (psattn_bwd); may be 0. */
psattn_status psattn_workspace_size(const psattn_tree* tree, int pass, size_t* bytes);

/* Forward (Sec. 2.5 attention masking over the shared layout):
 *   O[r][h]   = sum_j P_rj V[slot(j)][h/G],  P_r = softmax_j(scale * Q[r][h] . K[slot(j)][h/G])
 *   LSE[h][r] = log sum_j exp(scale * Q[r][h] . K[slot(j)][h/G])
 * over the keys j visible to row r.  Long key ranges may be split across
 * work items and merged by log-sum-exp.  ws may be NULL when its size is 0.
 * O_lo (bf16 trees only, else NULL; optional, [Ns][Hq][d] like O, caller-owned):
 * when given, it receives the rounding residual bf16(O_fp32 - O) of the fp32
 * result, so that O + O_lo carries O to about 2^-16 relative.  psattn_bwd uses
 * it for Delta (see there). */
psattn_status psattn_fwd(const psattn_tree* tree, const void* Q, const void* K, const void* V,
                         void* O, float* LSE, void* O_lo, void* ws, size_t ws_bytes, void* stream);

/* Backward (Sec. 6: one backward pass over the accumulated adjoints).  dO is
 * the total adjoint of each shared token.  With P as above,
 * Delta_r = dO_r . O_r and dS = P * (dO V^T - Delta):
 * (bf16: Delta_r = dO_r . (O_r + O_lo_r) when O_lo, the forward's residual, is
 * given, else from the bf16 O alone.  Its error times sum_j P_rj K_j enters dQ,
 * which matters on rows whose softmax sits on one large key; dK/dV use the
 * exact sum_j P dP either way.)
 *   dQ = scale * dS K;  dK = scale * dS^T Q;  dV = P^T dO
 * where prefix dK/dV sum over every consuming branch and query head of the
 * group.  Partial sums are reduced in a fixed order (no floating-point
 * atomics): results are bitwise reproducible for a given tree and plan. */
psattn_status psattn_bwd(const psattn_tree* tree, const void* Q, const void* K, const void* V,
                         const void* O, const float* LSE, const void* O_lo, const void* dO,
                         float* dQ, float* dK, float* dV, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): psattn_bwd with its workspace taken from a file-scope
 * device array of PSATTN_NOALLOC_SCRATCH_MIB MiB, one copy per GPU, held until the process ends.
 * It calls no hipMalloc/hipFree and allocates nothing else.  Arguments and results as for
 * psattn_bwd, without ws / ws_bytes.  A tree whose backward workspace (psattn_workspace_size,
 * pass 1) exceeds the array is rejected with PSATTN_E_WORKSPACE before anything is enqueued.
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU (other streams,
 * other host threads) race and must be serialised by the caller.  The array needs no clearing:
 * each call writes every workspace byte it reads. */
#define PSATTN_NOALLOC_SCRATCH_MIB 128
psattn_status psattn_bwd_noalloc(const psattn_tree* tree, const void* Q, const void* K, const void* V,
                                 const void* O, const float* LSE, const void* O_lo, const void* dO,
                                 float* dQ, float* dK, float* dV, void* stream);

/* ---- Adaptive KV cache manager (Sec. 5.1 adaptive block allocation, Sec. 5.2 dynamic block
 * caching; Sec. 6 "Adaptive KV cache manager").  Host-only planning over a schedule of calls
 * (micro-batches) on one pool of capacity_slots slots: which nodes each call computes (internal)
 * and which it reads from the cache (external, psattn_tree_desc.row_off = -1), where each node's
 * blocks lie, and the events the caller acts on.
 *   - A node is stored when first needed: one block of exactly seg_len slots (block_size 0), or
 *     ceil(seg_len / block_size) fixed pages.
 *   - Reference count = samples that read the node.  After a call's backward it drops by the
 *     call's samples that read it; with dbc at 0 the node is freed (PSATTN_KVM_FREE: its dK/dV
 *     accumulators are complete).  Without dbc every block stays to the end of the schedule.
 *   - When a block does not fit, cached nodes the call does not read are evicted, farthest next
 *     use first (PSATTN_KVM_EVICT: flush the partial dK/dV accumulated so far, then the slots are
 *     reused).  A later call that reads an evicted node gets it back in a new block
 *     (PSATTN_KVM_REFILL: write its K/V there again and zero its dK/dV) as an external node.
 *   - PSATTN_E_WORKSPACE when one call's own blocks do not fit in the pool. */
typedef struct psattn_kvm psattn_kvm;
typedef enum {
  PSATTN_KVM_ALLOC = 0,   /* before the call: new block of a node the call computes */
  PSATTN_KVM_REFILL = 1,  /* before the call: new block of an evicted node the call reads */
  PSATTN_KVM_EVICT = 2,   /* before the call: block released while still to be read */
  PSATTN_KVM_FREE = 3     /* after the call's backward: reference count 0, block released */
} psattn_kvm_event_kind;
typedef struct {
  int32_t kind;        /* psattn_kvm_event_kind */
  int32_t node;        /* forest node */
  int32_t num_blocks;  /* blocks of the node (1, or its fixed pages) */
  int32_t capacity;    /* slots of its first block */
  int64_t base;        /* first slot of its first block */
} psattn_kvm_event;
typedef struct {
  int64_t capacity_slots;  /* pool slots the manager allocates from (>= 1) */
  int32_t block_size;      /* 0: adaptive, one block of exactly seg_len slots per node; > 0: fixed pages */
  int32_t dbc;             /* 1: free a block at reference count 0; 0: keep every block to the end */
  int32_t reserved[4];     /* must be 0 */
} psattn_kvm_opts;
typedef struct {
  int64_t peak_slots;        /* most slots in use during any call */
  int64_t final_slots;       /* slots still in use after the last call */
  int64_t evictions;         /* blocks evicted before their last use */
  int64_t refilled_tokens;   /* tokens written again after an eviction */
  int64_t allocated_tokens;  /* tokens stored, first stores and refills */
  int32_t num_calls;
  int32_t pad_;
} psattn_kvm_stats;

/* Plan a schedule: the forest (parent / seg_len as in psattn_tree_desc) and, for each sample, its
 * endpoint and the call that processes it (calls run in increasing index order; every index up
 * to the largest holds a sample). */
psattn_status psattn_kvm_plan(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                              int32_t num_samples, const int32_t* sample_end, const int32_t* call_of_sample,
                              const psattn_kvm_opts* opts, psattn_kvm** out);
void psattn_kvm_destroy(psattn_kvm* kvm);
/* The descriptor of one call: fills num_nodes, parent, seg_len, row_off (-1 for external nodes,
 * internal rows packed in node order), blk_ptr, blocks, pool_slots and the samples; the caller
 * sets hq, hkv, head_dim, softmax_scale, dtype.  node_ids (optional) maps the call's nodes to
 * forest nodes.  Arrays stay valid until psattn_kvm_destroy. */
psattn_status psattn_kvm_call_desc(const psattn_kvm* kvm, int32_t call, psattn_tree_desc* desc,
                                   const int32_t** node_ids);
/* The events of a call: phase 0 before it runs, 1 after its backward. */
psattn_status psattn_kvm_events(const psattn_kvm* kvm, int32_t call, int32_t phase,
                                const psattn_kvm_event** events, int32_t* count);
/* Statistics; used_per_call (optional, num_calls entries) receives the slots in use during each
 * call. */
psattn_status psattn_kvm_get_stats(const psattn_kvm* kvm, psattn_kvm_stats* stats, int64_t* used_per_call);

/* ---- Host scheduling (Sec. 4.2 workload model and greedy placement, Sec. 4.3 token-wise
 * micro-batching).  The workload of a sequence of length l whose first h tokens are cached is
 * Eq. "single_sequence": T = a1 * l_suf * l + a2 * l_suf + a3, l_suf = l - h (attention, the
 * per-token layers, a fixed overhead); alpha = (a1, a2, a3) from profiling. */

/* Least-squares fit of alpha to n >= 3 measured runs (l_suf[i], l[i]) -> t[i]. */
psattn_status psattn_sched_fit(int32_t n, const double* l_suf, const double* l, const double* t, double alpha[3]);
/* Workload of each semantic group: the sum of T over its samples (in sample order), each counting
 * as cached the nodes its group's earlier samples hold.  group_cost has num_groups entries. */
psattn_status psattn_sched_group_costs(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                                       int32_t num_samples, const int32_t* sample_end,
                                       const int32_t* group_of_sample, int32_t num_groups,
                                       const double alpha[3], double* group_cost);
/* Greedy placement: groups in descending workload (ties by index), each whole onto the worker
 * with the least load so far (ties: lowest index).  worker_load (optional) gets the loads. */
psattn_status psattn_sched_place(int32_t num_groups, const double* group_cost, int32_t num_workers,
                                 int32_t* worker_of_group, double* worker_load);
/* Token-wise micro-batching of one worker's samples, in their order: budget = total workload /
 * num_micro_batches; a sequence that would overflow the current micro-batch is cut at the token
 * where it fills it, and its remaining tokens go on in the next micro-batch with the part done as
 * cached prefix (the last micro-batch takes whatever remains).  The result is a refined forest in
 * which every cut is a node boundary, and one chunk (a sample of the refined forest) per
 * (sample, micro-batch) piece: ready for psattn_kvm_plan with call = micro-batch. */
typedef struct psattn_sched_mb psattn_sched_mb;
typedef struct {
  int32_t num_nodes;                /* refined forest */
  const int32_t* parent;
  const int32_t* seg_len;
  const int32_t* src_node;          /* original node of each refined node */
  const int32_t* src_offset;        /* its first token within that node */
  int32_t num_chunks;
  const int32_t* chunk_end;         /* refined endpoint node of each chunk */
  const int32_t* chunk_micro_batch; /* micro-batch of each chunk (0 .. num_micro_batches-1) */
  const int32_t* chunk_sample;      /* original sample of each chunk */
  int32_t num_micro_batches;        /* micro-batches that received work */
  const double* micro_batch_cost;   /* estimated workload of each */
} psattn_sched_mb_view;
psattn_status psattn_sched_microbatch(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                                      int32_t num_samples, const int32_t* sample_end, const double alpha[3],
                                      int32_t num_micro_batches, psattn_sched_mb** out);
/* Arrays stay valid until psattn_sched_mb_destroy. */
psattn_status psattn_sched_mb_get(const psattn_sched_mb* mb, psattn_sched_mb_view* view);
void psattn_sched_mb_destroy(psattn_sched_mb* mb);

/* ---- The rest of a layer in the shared layout (Sec. 6, prefix-sharing training runtime): the
 * tree-dependent steps around the attention.  Each shared token has one sequence position (its
 * block's pos), so every step below touches each shared row once. */

/* Rotary position embedding in place: X [Ns][heads][d] of the given dtype (queries and keys in
 * the tree's dtype, their fp32 gradients), row r at sequence position p(r): the pair
 * (x_i, x_{i+d/2}), i < d/2, turns by p * theta^(-2i/d) (inverse != 0: by minus that, the
 * transposed rotation for the backward).  theta > 1 (e.g. 10000). */
psattn_status psattn_rope(const psattn_tree* tree, void* X, psattn_dtype dtype, int32_t heads, float theta,
                          int32_t inverse, void* stream);
/* K/V rows [Ns][Hkv][d] (the tree's dtype) written into their pool slots of K, V
 * [pool_slots][Hkv][d]. */
psattn_status psattn_kv_scatter(const psattn_tree* tree, const void* K_rows, const void* V_rows, void* K, void* V,
                                void* stream);
/* dK/dV of each row's pool slot, fp32 [pool_slots][Hkv][d] -> rows [Ns][Hkv][d]. */
psattn_status psattn_kv_gather(const psattn_tree* tree, const float* dK, const float* dV, float* dK_rows,
                               float* dV_rows, void* stream);

/* Reference count of every node: the number of samples whose path holds it
 * (Sec. 5.2).  node_refcount has num_nodes entries. */
psattn_status psattn_tree_refcounts(const psattn_tree* tree, int32_t* node_refcount);

psattn_status psattn_tree_get_info(const psattn_tree* tree, psattn_tree_info* info);

/* Read-only view of a host plan array, for inspection and tests.  which:
 *   0 row_pos [Ns]            sequence position of each packed row
 *   1 q_list                  packed row indices referenced by work items
 *   2 kv_list                 pool slots referenced by work items
 *   3 fwd_items [n][8]        q_off nq kv_off nkv kv_pos0 head0 part nfull
 *   4 fwd_merges [n][4]       q_off nq part0 nparts
 *   5 bkv_items [n][10]       kv_off nk kv_pos0 q_off nq hk part mask_lo mask_hi acc
 *   6 bkv_reduces [n][8]      kv_off nk hk part0 nparts acc 0 0
 *   7 pad_slots [n]           pool slots that hold no token
 *   8 row_slot [Ns]           pool slot of each packed row's K/V
 *   9 q_pos                   sequence position of each q_list entry
 * *data stays valid until psattn_tree_destroy. */
psattn_status psattn_tree_plan_array(const psattn_tree* tree, int which, const int32_t** data,
                                     int64_t* count, int32_t* width);

/* Kernel timing for measurement: when enabled, every kernel launch made by
 * psattn_fwd/psattn_bwd is bracketed by HIP events recorded on its stream.
 * psattn_profile_read waits for the recorded events and reports, per kernel
 * name, the launch count and the summed duration in milliseconds since the
 * last reset.  Not thread-safe; meant for single-threaded benchmarking. */
psattn_status psattn_profile_enable(int enable);
psattn_status psattn_profile_reset(void);
psattn_status psattn_profile_read(int32_t max_entries, int32_t* num_entries, const char** names,
                                  int64_t* launches, double* total_ms);

const char* psattn_status_string(psattn_status status);
const char* psattn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PSATTN_H */
