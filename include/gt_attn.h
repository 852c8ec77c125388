/*
 * gt_attn.h - topology-biased graph attention on AMD Instinct MI355X (gfx950).
 *
 * C ABI of libgtattn.so. Plain pointers and sizes only; every tensor pointer
 * is a DEVICE pointer owned by the caller, dense and row-major in the layout
 * stated for it. The library never allocates, frees or retains caller memory
 * and keeps no mutable global state.
 *
 * The operation (MegaGraph, Section II-A, Eq. (1)): for every head h,
 *
 *     O_h = softmax( scale * Q_h K_h^T + B_h ) V_h,
 *     B_h[i, j] = table[h, spd[i, j]]   (0 when spd[i, j] >= n_buckets),
 *
 * i.e. the structural-encoding bias of the paper realised as one learned
 * scalar per (head, shortest-path-distance bucket). spd is a uint8 index
 * matrix shared by all heads. The scale multiplies Q K^T only; the bias is
 * added unscaled. LSE is the natural-log log-sum-exp of each score row.
 *
 * Conventions shared by every entry point
 *   - dtype GT_BF16: Q, K, V, O, dO, dQ, dK, dV are bfloat16; the products
 *     run on bf16 matrix cores with fp32 accumulation, and P and dS are
 *     rounded to bf16 before their products. d = 8 and 16 (the 8 heads over
 *     a 64-wide model of Section IV-A give d = 8) run on the same kernels
 *     with 32-wide tiles whose extra features are zero.
 *     GT_F32: all of those tensors are fp32 and computed in fp32. table,
 *     dtable, LSE, partial O and partial LSE are always fp32.
 *     The bf16 rounding of dS bounds dQ's error per element by about
 *     2 scale 2^-9 sum_j |dS_ij| |K_jc|: rows whose dQ sums nearly
 *     cancelling terms over large-norm keys lose relative accuracy (about
 *     15 % relative L2 on a head whose scores reach ~170 along keys of norm
 *     ~230), while scores of order one give about 2e-3.
 *   - d (head dim) must be 8, 16, 32 or 64; 1 <= n_buckets <= 256;
 *     N <= 2^25 - 16 (GT_ERR_UNSUPPORTED otherwise: spd offsets are
 *     32-bit).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream) and stream-ordered; results are valid once the stream has
 *     synchronised. Calls on different streams do not interfere except
 *     through memory the caller shares between them.
 *   - Errors: arguments are validated on the host BEFORE anything is
 *     launched; on any error no output is touched. A failed launch returns
 *     GT_ERR_LAUNCH.
 *   - Not checked (preconditions): device pointers really are device memory
 *     of the stated size; outputs do not alias inputs; table entries are
 *     finite or -inf. A row whose every score is -inf gets O = 0, LSE = -inf
 *     and zero gradient.
 */
#ifndef GT_ATTN_H
#define GT_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { GT_F32 = 0, GT_BF16 = 1 } gt_dtype_t;

typedef enum {
  GT_OK = 0,
  GT_ERR_INVALID = 1,     /* null pointer, bad size, bad offset, bad scale   */
  GT_ERR_UNSUPPORTED = 2, /* head dim, dtype or spd stride with no kernel    */
  GT_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required      */
  GT_ERR_LAUNCH = 4       /* the HIP runtime rejected a kernel launch        */
} gt_status_t;

/* Forward over all N nodes (Eq. (1)).
 *   q, k, v  [H, N, d] dtype          spd    [N, N] uint8, element (i,j) at i*N + j
 *   table    [H, n_buckets] fp32      o      [H, N, d] dtype (written)
 *   lse      [H, N] fp32 (written)    scale  > 0 and finite (1/sqrt(d) usual)
 * Deterministic: the same inputs give bitwise identical O and LSE. */
gt_status_t gt_attn_fwd(const void* q, const void* k, const void* v,
                        const uint8_t* spd, const float* table, int32_t n_buckets,
                        void* o, float* lse,
                        int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                        float scale, void* stream);

/* A batch of B graphs (sequences) of N nodes each, H heads per graph, every
 * graph with its own spd and all sharing one table (a training batch of b
 * sampled sequences, as in the memory model of Section III-B, Eqs. (6)-(7),
 * and the batch sizes of Section IV-A; Eq. (1) per graph):
 *   q, k, v  [B, H, N, d] dtype          o [B, H, N, d] dtype (written)
 *   spd      graph b's [N, N] uint8 matrix at spd + b * spd_bstride
 *            (spd_bstride = N * N for a dense [B, N, N] array; 0 lets every
 *            graph share one spd); the caller keeps every graph's N * N bytes
 *            inside its allocation
 *   table    [H, n_buckets] fp32, shared by the batch
 *   lse      [B, H, N] fp32 (written)
 * B >= 1, spd_bstride >= 0; otherwise as gt_attn_fwd, which is this call
 * with B = 1. Deterministic. Performance: in bf16 with d <= 32, graphs of at
 * most 256 nodes (N a multiple of 4 for the forward, spd rows 4-byte aligned)
 * run on persistent whole-sequence kernels that also pack 2, 4 or 8 graphs
 * of at most 128, 64 or 32 nodes to a workgroup; the backward of such graphs
 * is one fused kernel. */
gt_status_t gt_attn_fwd_batch(const void* q, const void* k, const void* v,
                              const uint8_t* spd, int64_t spd_bstride,
                              const float* table, int32_t n_buckets,
                              void* o, float* lse,
                              int32_t B, int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                              float scale, void* stream);

/* Bytes of device workspace gt_attn_bwd needs for these sizes. */
size_t gt_attn_bwd_workspace_size(int32_t H, int64_t N, int32_t d, gt_dtype_t dtype);

/* Backward of L = sum(O * dO) (the chain rule through Eq. (1); the paper's
 * training step needs it but does not write it out):
 *   dV = P^T dO,  dS = P * (dO V^T - rowsum(dO * O)),
 *   dQ = scale dS K,  dK = scale dS^T Q,
 *   dtable[h, b] = sum of dS[h, i, j] over pairs with spd[i, j] == b.
 *   spd_t    OPTIONAL [N, N] uint8 transpose of spd (spd_t[j*N + i] ==
 *            spd[i*N + j]), caller-owned device memory, read only. The
 *            key-stationary stage reads spd by columns; with spd_t it reads
 *            rows instead. The shortest-path matrix of an undirected graph is
 *            symmetric: pass spd itself. A directed graph's spd is fixed per
 *            graph, so its transpose can be built once. NULL, or a spd_t
 *            that is not 16-byte aligned or with N not a multiple of 16, is
 *            ignored (columns of spd are gathered). A spd_t that is not the
 *            transpose of spd gives wrong dK, dV and dtable.
 *   o, lse   the forward outputs for the same inputs
 *   d_o      [H, N, d] dtype
 *   dq,dk,dv [H, N, d] dtype, OVERWRITTEN
 *   dtable   [H, n_buckets] fp32, OVERWRITTEN (not accumulated)
 *   workspace at least gt_attn_bwd_workspace_size(H, N, d, dtype) bytes of
 *            device memory, 256-byte aligned; contents on entry are ignored.
 * dtable is reduced with floating-point atomics: its last bits may differ
 * from run to run. No gradient flows to spd. */
gt_status_t gt_attn_bwd(const void* q, const void* k, const void* v,
                        const uint8_t* spd, const uint8_t* spd_t,
                        const float* table, int32_t n_buckets,
                        const void* o, const float* lse, const void* d_o,
                        void* dq, void* dk, void* dv, float* dtable,
                        void* workspace, size_t workspace_bytes,
                        int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                        float scale, void* stream);

/* gt_attn_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). The scratch that gt_attn_bwd takes as
 * its workspace is a fixed device array inside the library instead, of
 * gt_attn_bwd_noalloc_max_bytes() = 16 MiB on each GPU the library runs on,
 * held until the process ends. The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the array's device address is
 * looked up once per device, on the first call with that device current.
 *   Arguments, results and validation as gt_attn_bwd. Sizes whose
 *   gt_attn_bwd_workspace_size(H, N, d, dtype) exceeds the array (H * N
 *   above about 2.09 million rows) give GT_ERR_WORKSPACE and touch nothing;
 *   a failed address lookup gives GT_ERR_LAUNCH.
 *   Every call on one GPU shares that GPU's array: calls that overlap in time
 *   on one GPU (different streams, or host threads without ordering) race
 *   and give wrong results. Calls ordered on one stream are safe; each call
 *   rewrites every part of the array it reads, so nothing needs clearing. */
size_t gt_attn_bwd_noalloc_max_bytes(void);
gt_status_t gt_attn_bwd_noalloc(const void* q, const void* k, const void* v,
                                const uint8_t* spd, const uint8_t* spd_t,
                                const float* table, int32_t n_buckets,
                                const void* o, const float* lse, const void* d_o,
                                void* dq, void* dk, void* dv, float* dtable,
                                int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                                float scale, void* stream);

/* Backward of gt_attn_fwd_batch: dq, dk, dv [B, H, N, d] dtype (overwritten);
 * dtable [H, n_buckets] fp32 (overwritten) sums the gradient over every graph
 * of the batch, since they share the table. spd_t (optional) holds graph b's
 * transpose at spd_t + b * spd_bstride. workspace: at least
 * gt_attn_bwd_workspace_size(B * H, N, d, dtype) bytes. Otherwise as
 * gt_attn_bwd, which is this call with B = 1. */
gt_status_t gt_attn_bwd_batch(const void* q, const void* k, const void* v,
                              const uint8_t* spd, const uint8_t* spd_t, int64_t spd_bstride,
                              const float* table, int32_t n_buckets,
                              const void* o, const float* lse, const void* d_o,
                              void* dq, void* dk, void* dv, float* dtable,
                              void* workspace, size_t workspace_bytes,
                              int32_t B, int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                              float scale, void* stream);

/* The backward split into its three stages, for callers that schedule them
 * (e.g. the two independent stages on two streams) or time them:
 *   phase 0  prepare: rowsum(dO * O) and LSE * log2(e) into the workspace;
 *            dtable = 0
 *   phase 1  dK and dV, and dtable for bf16 (needs phase 0)
 *   phase 2  dQ, and dtable for fp32
 *            (needs phase 0; independent of phase 1)
 * Arguments and results are exactly those of gt_attn_bwd; running phases
 * 0, 1, 2 on one stream is gt_attn_bwd. Outputs a phase does not produce
 * are not touched. phase outside 0..2 gives GT_ERR_INVALID. */
gt_status_t gt_attn_bwd_phase(int32_t phase,
                              const void* q, const void* k, const void* v,
                              const uint8_t* spd, const uint8_t* spd_t,
                              const float* table, int32_t n_buckets,
                              const void* o, const float* lse, const void* d_o,
                              void* dq, void* dk, void* dv, float* dtable,
                              void* workspace, size_t workspace_bytes,
                              int32_t H, int64_t N, int32_t d, gt_dtype_t dtype,
                              float scale, void* stream);

/* Calling convention of a rank's whole ring (Section III-A-1 parts 1-3), for
 * the entry points below. P ranks split the N' regular nodes into P
 * contiguous blocks [b_r, b_{r+1}); the batch may also hold N_s super nodes
 * (global nodes, ids N' .. N' + N_s - 1) that every rank replicates.
 *   - Rank r's query shard is its regular rows [b_r, b_{r+1}) followed by
 *     every super-node row, and it holds only those rows of spd (its bias
 *     shard, [b_{r+1} - b_r + N_s, N' + N_s]); row_off indexes that shard.
 *   - At step t = 0 .. P-1 the rank holds regular KV block (r - t) mod P and
 *     calls a ring step with col_off = that block's first node id. With
 *     N_s > 0 it then makes ONE more step over the super-node KV block,
 *     col_off = N'. The paper places the super nodes in every KV block; read
 *     literally, every super-node key would then enter each row's softmax P
 *     times, so the super block is visited once instead and every key counts
 *     exactly once (the merged result equals the unsharded attention over
 *     all N' + N_s nodes).
 *   - The forward merges the P (+1) partials: gt_attn_ring_step for the
 *     first step, gt_attn_ring_step_acc for the others (or partials and
 *     gt_attn_merge). Every rank computes the same super-node rows.
 *   - The backward visits the same blocks in the same order with
 *     gt_attn_bwd_ring_step, using the merged O and LSE. The replicated
 *     super-node rows' loss must count once: rank 0 passes their dO and
 *     every other rank passes zeros for those rows. dK/dV of a block
 *     accumulate over every rank's step on it (the accumulators travel with
 *     the block); dQ of a super-node row is the sum of its rows' dq_acc over
 *     the ranks (only rank 0's is nonzero); dtable is summed over the ranks.
 * The Python binding's paper_2609_34420_amd.ring module returns these
 * shards and step lists. */

/* One step of graph-aware context parallelism (Section III-A-1: ring-based
 * KV rotation, query-dimension bias sharding, Eq. (2)). A rank holding the
 * query shard q_shard and, at this step, one KV block computes the block's
 * biased attention with the bias columns sliced to match that block:
 *
 *   S[i, j] = scale * q_shard[i] . k_shard[j] + table[h, spd[(row_off+i)*ld_spd + col_off + j]]
 *
 * and returns the block-normalised partial O_p = softmax_j(S) v_shard with
 * its log-sum-exp LSE_p (natural log). Combine partials with gt_attn_merge.
 *   q_shard  [H, Sq, d] dtype         k_shard, v_shard [H, Sk, d] dtype
 *   spd      the rank's bias shard; element (r, c) at spd[r*ld_spd + c],
 *            r = row_off + i, c = col_off + j (typically row_off = 0 and
 *            col_off = the KV block's first global node id)
 *   o_part   [H, Sq, d] fp32 (written)  lse_part [H, Sq] fp32 (written)
 * Sq >= 1, Sk >= 0, row_off >= 0, col_off >= 0, ld_spd >= col_off + Sk;
 * ld_spd <= 2^25 - 16 (GT_ERR_UNSUPPORTED otherwise: spd offsets are
 * 32-bit). Sk = 0 gives o_part = 0 and lse_part = -inf (k_shard, v_shard,
 * spd may then be NULL). Deterministic. */
gt_status_t gt_attn_ring_step(const void* q_shard, int64_t Sq,
                              const void* k_shard, const void* v_shard, int64_t Sk,
                              const uint8_t* spd, int64_t ld_spd,
                              int64_t row_off, int64_t col_off,
                              const float* table, int32_t n_buckets,
                              float* o_part, float* lse_part,
                              int32_t H, int32_t d, gt_dtype_t dtype,
                              float scale, void* stream);

/* One context-parallel step merged in place into a running result (the
 * running max/sum update of Section III-A-1 part 3, applied per KV block):
 * the step of gt_attn_ring_step, whose partial (O_p, LSE_p) is combined with
 * the state (o_acc, lse_acc) in the same kernel,
 *   LSE = log(exp(lse_acc) + exp(LSE_p)),
 *   O   = exp(lse_acc - LSE) o_acc + exp(LSE_p - LSE) O_p,
 * and written back. After the last step (o_acc, lse_acc) is the merged O
 * (normalised, fp32) and LSE of the shard's rows over every block seen, so no
 * per-step partial buffer and no separate merge pass are needed (cast O with
 * gt_attn_merge, n_parts = 1, if the dtype is wanted).
 *   o_acc    [H, Sq, d] fp32, read and written; lse_acc [H, Sq] fp32, read and
 *            written. Start from the first step's gt_attn_ring_step output
 *            (o_part, lse_part), or from o_acc = 0, lse_acc = -inf (no block).
 *            Rows whose running LSE and step LSE are both -inf stay O = 0,
 *            LSE = -inf.
 * Other arguments, validation and errors as gt_attn_ring_step (Sk = 0 leaves
 * the state unchanged). Steps on one state must be ordered (one stream);
 * the result depends on the order only through fp32 rounding. */
gt_status_t gt_attn_ring_step_acc(const void* q_shard, int64_t Sq,
                                  const void* k_shard, const void* v_shard, int64_t Sk,
                                  const uint8_t* spd, int64_t ld_spd,
                                  int64_t row_off, int64_t col_off,
                                  const float* table, int32_t n_buckets,
                                  float* o_acc, float* lse_acc,
                                  int32_t H, int32_t d, gt_dtype_t dtype,
                                  float scale, void* stream);

/* Combine n_parts block partials into the attention over all of their keys
 * (Section III-A-1 part 3: every partial's softmax statistics already hold
 * its bias slice, so the combination is exact):
 *   LSE = log sum_p exp(LSE_p),  O = sum_p exp(LSE_p - LSE) O_p.
 * Parts with LSE_p = -inf contribute nothing; if every part is -inf the row
 * gets O = 0, LSE = -inf.
 *   o_parts  [n_parts, H, S, d] fp32   lse_parts [n_parts, H, S] fp32
 *   o        [H, S, d] dtype (written) lse       [H, S] fp32 (written)
 * n_parts >= 1; n_parts = 1 is a copy/cast. Deterministic. */
gt_status_t gt_attn_merge(const float* o_parts, const float* lse_parts, int32_t n_parts,
                          void* o, float* lse,
                          int32_t H, int64_t S, int32_t d, gt_dtype_t dtype,
                          void* stream);

/* Bytes of device workspace gt_attn_bwd_ring_step needs for these sizes. */
size_t gt_attn_bwd_ring_workspace_size(int32_t H, int64_t Sq, int64_t Sk, int32_t d,
                                       gt_dtype_t dtype);

/* Backward of one ring step (Section III-A-1, Eq. (2); the chain rule through
 * the block's share of Eq. (1)). The probabilities of the pairs (query shard
 * row i, KV block key j) are recomputed with the merged statistics of the
 * whole row, P[i, j] = exp(S[i, j] - LSE[i]) with S as in gt_attn_ring_step,
 * so summing this step over every KV block of the ring is exactly the
 * unsharded backward. The step ADDS its contributions:
 *   dq_acc     += scale dS k_blk            dS = P * (d_o V^T - rowsum(d_o * o))
 *   dk_acc     += scale dS^T q_shard        dv_acc += P^T d_o
 *   dtable_acc[h, b] += sum of dS[h, i, j] over pairs whose spd byte is b
 *   q_shard, d_o_shard  [H, Sq, d] dtype
 *   o_shard    [H, Sq, d] dtype: the MERGED output of the shard's rows (the
 *              result of gt_attn_merge over all blocks), not a partial
 *   lse_shard  [H, Sq] fp32: the merged log-sum-exp of the same rows
 *   k_blk, v_blk [H, Sk, d] dtype
 *   spd, ld_spd, row_off, col_off  as in gt_attn_ring_step
 *   dq_acc     [H, Sq, d] fp32, dk_acc, dv_acc [H, Sk, d] fp32,
 *   dtable_acc [H, n_buckets] fp32: read and updated in place (zero them
 *              before the first step of a ring)
 *   workspace  at least gt_attn_bwd_ring_workspace_size(H, Sq, Sk, d, dtype)
 *              bytes of device memory, 256-byte aligned, contents ignored.
 * Sq >= 1, Sk >= 0, row_off >= 0, col_off >= 0, col_off + Sk <= ld_spd <=
 * 2^25 - 16; the spd buffer must hold rows row_off .. row_off + Sq - 1.
 * Sk = 0 touches nothing (k_blk, v_blk, spd, dk_acc, dv_acc may then be
 * NULL). Steps on one stream are ordered; steps that update the same
 * accumulators must not run concurrently. dtable_acc is updated with
 * floating-point atomics. */
gt_status_t gt_attn_bwd_ring_step(const void* q_shard, const void* o_shard,
                                  const float* lse_shard, const void* d_o_shard, int64_t Sq,
                                  const void* k_blk, const void* v_blk, int64_t Sk,
                                  const uint8_t* spd, int64_t ld_spd,
                                  int64_t row_off, int64_t col_off,
                                  const float* table, int32_t n_buckets,
                                  float* dq_acc, float* dk_acc, float* dv_acc,
                                  float* dtable_acc,
                                  void* workspace, size_t workspace_bytes,
                                  int32_t H, int32_t d, gt_dtype_t dtype,
                                  float scale, void* stream);

/* Static, human-readable name of a status code. */
const char* gt_status_string(gt_status_t s);

/* Library version as major*10000 + minor*100 + patch. */
int32_t gt_attn_version(void);

#ifdef __cplusplus
}
#endif
#endif /* GT_ATTN_H */
