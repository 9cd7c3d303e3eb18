/*
 * augtree.h — C ABI of the shared-prompt group attention library (libaugtree.so)
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation is one attention layer of a batch of replay trees
 * T = (P, {R_i}_{i=1..G}) (paper §2.1, §3.1): a shared prompt P and G response
 * branches. A response token of branch i attends to every prompt key and to
 * its own prefix, never to a sibling branch (§2.2; Eq. 1:
 * KV(R_{i,t}) = KV_P ∪ KV(R_{i,<t})). Attention is
 * O = softmax(s Q K^T + M) V with s = softmax_scale (§2.2).
 *
 * The library splits it the way the method does (§3.2, §3.3):
 *   prefill_fwd   causal attention over the prompt, run once per tree;
 *   replay_fwd    every branch against the prompt KV (read in place, never
 *                 copied) plus its own causal KV, two partial softmax states
 *                 merged by log-sum-exp;
 *   lse_merge     the merge of partial states on its own;
 *   replay_bwd    gradients of the replay, with each branch's prompt-KV
 *                 gradient ("seed") accumulated on the prompt KV (Eq. 2);
 *   prefill_bwd   gradients of the prefill (the prompt's own contribution);
 *   prompt_grad_reduce  the Eq. 2 sum of the prefill contribution and the
 *                 seeds, in a fixed order, without atomics;
 *   tree_fwd / tree_bwd  the same step in two calls with fewer launches (the
 *                 prefill and replay tiles share launches, and the Eq. 2 sum
 *                 is formed in registers).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout (packed varlen, head_dim innermost, row-major):
 *   Q_P [T_P, Hq, d]   K_P, V_P [T_P, Hkv, d]   (T_P = total prompt rows)
 *   Q_R [T_R, Hq, d]   K_R, V_R [T_R, Hkv, d]   (T_R = total response rows)
 *   O, dO, dQ like Q; dK, dV like K.   LSE [Hq, T] fp32 (head-major).
 *   bf16 tensors are passed as uint16_t bit patterns.
 * GQA: KV head k serves query heads k*g .. k*g+g-1, g = Hq / Hkv.
 * LSE is the natural log of sum_j exp(s q.k_j) over the visible keys.
 * Pointers: every tensor pointer is a DEVICE pointer of the current HIP
 *   device and must be 16-byte aligned; the descriptor's offset arrays are
 *   HOST pointers. `stream` is a hipStream_t (NULL = the null stream).
 * Ownership: the caller allocates and owns every buffer, workspace included.
 *   The library never allocates or frees memory and never synchronises the
 *   device; all work is enqueued on `stream`. Prompt tensors must stay alive
 *   from prefill_fwd until prefill_bwd.
 * Outputs are overwritten, never accumulated into.
 * Workspace: `ws` must hold augtree_workspace_size(...) bytes (256-byte
 *   aligned). A launch of more than a few dozen tiles reads its tile schedule
 *   from the workspace, written there with an asynchronous host-to-device copy
 *   on `stream` (the host staging happens before the call returns); smaller
 *   schedules travel in the kernel arguments. The backward also keeps
 *   D = rowsum(dO * O) of every row there (written by its dQ kernel, read by
 *   its dK/dV kernel).
 * Errors: every call returns an augtree_status. Arguments are validated on
 *   the host before any work is enqueued; on error nothing is launched and
 *   augtree_last_error() gives a detail string (thread-local). No C++
 *   exception crosses the ABI. Asynchronous kernel faults surface at the
 *   caller's next synchronisation, as in HIP.
 * Determinism: every output is bitwise reproducible run to run (no atomics),
 *   and a tree's outputs do not depend on the other trees of the batch (each
 *   output element is computed by one workgroup in a fixed order, whatever
 *   order the tiles are scheduled in).
 * Thread safety: calls are reentrant; calls on different streams that share a
 *   workspace race.
 */
#ifndef AUGTREE_H
#define AUGTREE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum augtree_status {
  AUGTREE_OK = 0,
  AUGTREE_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad count, bad offsets */
  AUGTREE_ERR_UNSUPPORTED = 2,      /* head_dim not in {64,128}, Hq % Hkv != 0 */
  AUGTREE_ERR_MISALIGNED = 3,       /* a tensor pointer not 16-byte aligned */
  AUGTREE_ERR_WORKSPACE = 4,        /* workspace missing or too small */
  AUGTREE_ERR_DEVICE = 5,           /* current device is not gfx950 */
  AUGTREE_ERR_HIP = 6               /* a HIP launch or copy reported an error */
} augtree_status;

typedef enum augtree_replay_mode {
  AUGTREE_REPLAY_FUSED = 0, /* prompt sweep then own-branch sweep, merged in registers */
  AUGTREE_REPLAY_SPLIT = 1, /* two partial states written out, then lse_merge */
  AUGTREE_REPLAY_AUTO = 2   /* per group, FUSED or SPLIT by a cost rule (augtree_replay_split_groups) */
} augtree_replay_mode;

typedef enum augtree_op {
  AUGTREE_OP_PREFILL_FWD = 0,
  AUGTREE_OP_REPLAY_FWD = 1, /* workspace arg: replay mode */
  AUGTREE_OP_PREFILL_BWD = 2,
  AUGTREE_OP_REPLAY_BWD = 3, /* workspace arg: n_seed */
  AUGTREE_OP_TREE_FWD = 4,   /* workspace arg: replay mode */
  AUGTREE_OP_TREE_BWD = 5    /* workspace arg ignored */
} augtree_op;

/*
 * A batch of replay trees (§3.1: T = (P, {R_i})). Offsets are HOST arrays.
 *   cu_prompt [num_groups+1]  group g's prompt rows are cu_prompt[g] .. cu_prompt[g+1]-1
 *   cu_branch [num_groups+1]  group g owns branches cu_branch[g] .. cu_branch[g+1]-1
 *   cu_resp   [num_branches+1] branch b's response rows are cu_resp[b] .. cu_resp[b+1]-1
 * Requirements: cu_*[0] == 0, every prompt and branch length >= 1, every
 * group has >= 1 branch, cu_branch[num_groups] == num_branches, branches of a
 * group are consecutive, offsets fit int32. softmax_scale > 0 (normally
 * 1/sqrt(head_dim)).
 */
typedef struct augtree_groups {
  int32_t num_groups;
  int32_t num_branches;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  float softmax_scale;
  const int32_t* cu_prompt;
  const int32_t* cu_branch;
  const int32_t* cu_resp;
} augtree_groups;

/* Bytes of workspace an entry point needs for this batch. `arg` is the replay
 * mode for AUGTREE_OP_REPLAY_FWD / AUGTREE_OP_TREE_FWD, n_seed for
 * AUGTREE_OP_REPLAY_BWD, ignored otherwise. Returns 0 on invalid arguments
 * (see augtree_last_error). */
size_t augtree_workspace_size(const augtree_groups* grp, int op, int arg);

/*
 * Prompt prefill forward (§3.2, shared prompt prefill pass; attention of §2.2
 * with the causal mask). For every group and query head h:
 *   O_P[r] = sum_{j<=r} exp(s q_r.k_j - LSE_r) v_j,  LSE_r = ln sum_{j<=r} exp(s q_r.k_j)
 * over the group's prompt rows, KV head h / g.
 * In:  q_p [T_P,Hq,d], k_p, v_p [T_P,Hkv,d] bf16.
 * Out: o_p [T_P,Hq,d] bf16, lse_p [Hq,T_P] fp32.
 * Reads num_groups, cu_prompt and the head shape only: cu_branch / cu_resp may
 * be NULL and num_branches is ignored (a batch of plain causal sequences).
 */
int augtree_prefill_fwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p,
                        const uint16_t* v_p, uint16_t* o_p, float* lse_p, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * Response replay forward (§3.2 response replay; Eq. 1; §3.3 merge of partial
 * states). Every response row of branch b (group g) attends to all prompt keys
 * of g (partial A, no mask) and to rows 0..t of branch b (partial B, causal);
 * the two partial states are merged by log-sum-exp:
 *   LSE = ln(exp(LSE_A) + exp(LSE_B)),  O = exp(LSE_A-LSE) O_A + exp(LSE_B-LSE) O_B.
 * FUSED: one sweep over both key sets, merged in registers.
 * SPLIT: partial A and partial B are written to o_part [2][T_R,Hq,d] fp32 and
 *   lse_part [2][Hq,T_R] fp32 (part 0 = prompt, part 1 = own branch), then
 *   merged by the lse_merge kernel into o_r / lse_r. The prompt partial's
 *   query tiles pack the rows of all branches of a group (they all see the
 *   same prompt keys), so short branches do not leave tiles mostly empty.
 * AUTO: each group runs FUSED or SPLIT as augtree_replay_split_groups reports;
 *   o_part / lse_part are required (only the split groups' rows are written
 *   there). In FUSED mode o_part and lse_part may be NULL.
 * In:  q_r [T_R,Hq,d], k_r, v_r [T_R,Hkv,d], k_p, v_p [T_P,Hkv,d] bf16.
 * Out: o_r [T_R,Hq,d] bf16, lse_r [Hq,T_R] fp32.
 */
int augtree_replay_fwd(const augtree_groups* grp, int mode, const uint16_t* q_r, const uint16_t* k_r,
                       const uint16_t* v_r, const uint16_t* k_p, const uint16_t* v_p, uint16_t* o_r,
                       float* lse_r, float* o_part, float* lse_part, void* ws, size_t ws_bytes,
                       void* stream);

/*
 * The replay-forward mode AUGTREE_REPLAY_AUTO gives each group (the choice of
 * a way to run one step of §3.2 per group, like the per-tree primitive choice
 * of §3.4, made here from the kernels' own costs). Writes split[g] = 1 when
 * group g runs SPLIT, 0 when FUSED. The rule: a mode costs the number of
 * (query tile, 64-key block) steps its forward tiles execute at a measured
 * time per step, plus, for SPLIT, the merge's HBM bytes at a measured
 * bandwidth; SPLIT is taken when it costs less. Short branches favour SPLIT
 * (a fused tile of a 16-row branch sweeps every prompt block for 16 rows),
 * long ones FUSED (same steps, no merge).
 * In:  grp (host offsets). Out: split [num_groups] int32, host memory.
 * Errors: INVALID_ARGUMENT for a bad descriptor or a NULL split.
 */
int augtree_replay_split_groups(const augtree_groups* grp, int32_t* split);

/*
 * Merge of n partial softmax states of the same rows (§3.3, the associative
 * merge applied to full states). For every row r and head h, in part order:
 *   M = max_k lse_k;  LSE = M + ln sum_k exp(lse_k - M);  O = sum_k exp(lse_k - LSE) o_k.
 * Parts with lse = -inf carry weight 0; if all parts are -inf the row gets
 * O = 0 and LSE = -inf.
 * In:  o_parts [n_parts][rows,heads,head_dim] fp32, lse_parts [n_parts][heads,rows] fp32.
 * Out: o [rows,heads,head_dim] bf16 (nullable), o_f32 same shape fp32 (nullable,
 *      at least one of o / o_f32), lse [heads,rows] fp32 (nullable).
 * head_dim must be a multiple of 8 and <= 256; n_parts >= 1; rows >= 0.
 */
int augtree_lse_merge(int64_t rows, int32_t heads, int32_t head_dim, int32_t n_parts,
                      const float* o_parts, const float* lse_parts, uint16_t* o, float* o_f32,
                      float* lse, void* stream);

/*
 * Response replay backward (§3.2 exact many-to-one backward; Eq. 2). With the
 * merged O and LSE of replay_fwd and D_r = sum_c dO_rc O_rc, for each branch
 * row and both partials: P = exp(s q.k - LSE), dP = dO.v, dS = P (dP - D);
 *   dQ_R = s (dS_A K_P + dS_B K_R),  dK_R = s dS_B^T Q_R,  dV_R = P_B^T dO_R,
 *   seeds  dK_P += s dS_A^T Q_R,  dV_P += P_A^T dO_R  (summed over the g query
 *   heads of each KV head and over the group's branches).
 * The group's response rows are cut into n_seed contiguous chunks of about
 * equal size; chunk c's prompt-key gradient is written to slab c of
 * dkv_p_seed [n_seed][2][T_P,Hkv,d] fp32 (index 0 = dK, 1 = dV). n_seed = 1
 * sums every branch in-kernel; n_seed > 1 trades a larger Eq. 2 reduction for
 * more parallelism. Slabs are overwritten.
 * In:  q_r, k_r, v_r, k_p, v_p, o_r (bf16), lse_r (fp32), do_r (bf16).
 * Out: dq_r [T_R,Hq,d], dk_r, dv_r [T_R,Hkv,d] bf16; dkv_p_seed fp32.
 * 1 <= n_seed <= 64.
 * dQ: with dS rounded to bf16 for the dQ product, the kernel subtracts c times
 * the row sum of the rounded dS, c = the group's first prompt key (exact in
 * arithmetic since every row of dS sums to zero over its keys); this keeps a
 * component shared by all keys from amplifying the rounding of dS.
 */
int augtree_replay_bwd(const augtree_groups* grp, const uint16_t* q_r, const uint16_t* k_r,
                       const uint16_t* v_r, const uint16_t* k_p, const uint16_t* v_p,
                       const uint16_t* o_r, const float* lse_r, const uint16_t* do_r, uint16_t* dq_r,
                       uint16_t* dk_r, uint16_t* dv_r, int32_t n_seed, float* dkv_p_seed, void* ws,
                       size_t ws_bytes, void* stream);

/*
 * Prompt prefill backward: the prompt queries' own contribution to every
 * gradient, i.e. the backward of the causal prefill attention itself (§3.2;
 * Eq. 2's first term for the prompt keys), causal over P.
 * In:  q_p, k_p, v_p, o_p (bf16), lse_p (fp32), do_p (bf16).
 * Out: dq_p [T_P,Hq,d] bf16 (nullable) and/or dq_p_f32 same shape fp32
 *      (nullable; at least one), dkv_p_self [2][T_P,Hkv,d] fp32 (0 = dK, 1 = dV).
 * Like prefill_fwd, reads only num_groups, cu_prompt and the head shape.
 */
int augtree_prefill_bwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p,
                        const uint16_t* v_p, const uint16_t* o_p, const float* lse_p,
                        const uint16_t* do_p, uint16_t* dq_p, float* dq_p_f32, float* dkv_p_self,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * One tree step's forward in one call (§3.2: prefill once, then replay every
 * branch against the prompt KV read in place; Eq. 1; §3.3). Computes exactly what
 * augtree_prefill_fwd followed by augtree_replay_fwd compute (bit for bit:
 * the same kernels and per-row arithmetic), but the prefill tiles and the
 * fused replay tiles run in ONE kernel launch (fewer launches and one launch
 * tail; the replay tiles read the prompt KV the prefill reads).
 * mode: as for augtree_replay_fwd (SPLIT / AUTO groups add the fp32 partial
 *   launch and the merge; o_part / lse_part are then required).
 * In:  q_p [T_P,Hq,d], k_p, v_p [T_P,Hkv,d], q_r [T_R,Hq,d], k_r, v_r [T_R,Hkv,d] bf16.
 * Out: o_p [T_P,Hq,d] bf16, lse_p [Hq,T_P], o_r [T_R,Hq,d] bf16, lse_r [Hq,T_R] fp32.
 * Workspace: augtree_workspace_size(grp, AUGTREE_OP_TREE_FWD, mode).
 */
int augtree_tree_fwd(const augtree_groups* grp, int mode, const uint16_t* q_p, const uint16_t* k_p,
                     const uint16_t* v_p, const uint16_t* q_r, const uint16_t* k_r, const uint16_t* v_r,
                     uint16_t* o_p, float* lse_p, uint16_t* o_r, float* lse_r, float* o_part,
                     float* lse_part, void* ws, size_t ws_bytes, void* stream);

/*
 * One tree step's backward in one call (§3.2 exact many-to-one backward;
 * Eq. 2). The same gradients as augtree_replay_bwd + augtree_prefill_bwd +
 * augtree_prompt_grad_reduce, in two kernel launches:
 *   dQ launch: every prompt row (causal over the prompt) and every response
 *     row (prompt keys, then its own causal keys); also forms
 *     D = rowsum(dO * O) of every row into the workspace;
 *   dK/dV launch: each prompt-key tile sweeps every response row of its group
 *     (all branches, every prompt key visible) and then the prompt rows at or
 *     after its first key (causal), so the whole Eq. 2 sum (branch seeds and
 *     the prompt queries' own contribution) is accumulated in registers, in
 *     that fixed order, and rounded once; each branch-key tile sweeps its
 *     branch's rows (causal).
 * A group whose branch rows exceed augtree_tree_chunk_blocks() query blocks
 * (64 rows of one query head) per prompt-key tile has that sweep cut into
 * chunks (at most 64) of consecutive branch rows, the first chunk also taking
 * the prompt rows; the chunks write fp32 partial sums to the workspace and a
 * third launch adds them per row in chunk order and rounds once (role
 * "reduce_tree"). Long sweeps otherwise lose the L2 sharing of the query rows.
 * The prompt gradient is the same sum as the three-call path up to fp32
 * rounding order (that path adds two fp32 partial sums); it is bitwise
 * reproducible for a given chunk setting. dQ carries the same common-mode
 * correction as augtree_replay_bwd.
 * In:  q_p, k_p, v_p, o_p (bf16), lse_p (fp32), do_p (bf16) [prompt rows];
 *      q_r, k_r, v_r, o_r (bf16), lse_r (fp32), do_r (bf16) [response rows].
 * Out: dq_p [T_P,Hq,d], dk_p, dv_p [T_P,Hkv,d], dq_r [T_R,Hq,d], dk_r, dv_r
 *      [T_R,Hkv,d] bf16; dkv_p_f32 [2][T_P,Hkv,d] fp32 (nullable: the prompt
 *      gradient before its bf16 rounding, 0 = dK, 1 = dV).
 * Workspace: augtree_workspace_size(grp, AUGTREE_OP_TREE_BWD, 0) (with chunks:
 * the fp32 partials, 2 x (sum over chunked groups of chunks x P) x Hkv x d x 4
 * bytes, and a row map of chunks x T_P int32).
 */
int augtree_tree_bwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p,
                     const uint16_t* v_p, const uint16_t* o_p, const float* lse_p,
                     const uint16_t* do_p, const uint16_t* q_r, const uint16_t* k_r,
                     const uint16_t* v_r, const uint16_t* o_r, const float* lse_r,
                     const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p, uint16_t* dv_p,
                     float* dkv_p_f32, uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r, void* ws,
                     size_t ws_bytes, void* stream);

/*
 * augtree_tree_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation). Same inputs, outputs and results as
 * augtree_tree_bwd (bit for bit: same kernels and schedule, except that a
 * batch whose chunked schedule does not fit the array runs one sweep per
 * prompt-key tile: the same prompt gradient up to fp32 summation order). Its
 * workspace is
 * a fixed 64 MiB device array of the library (augtree_noalloc_scratch_bytes()),
 * one copy per GPU, held from the first call on that GPU until the process
 * ends; the call performs no allocation. A batch whose unchunked workspace
 * exceeds it is rejected with AUGTREE_ERR_WORKSPACE before anything is
 * enqueued. Calls that overlap on
 * one GPU (several streams or threads) share the array and race; serialise
 * them. Stream capture: a launch whose tile schedule has more than 32 tiles
 * (and a chunked batch's row map) receives it by a host-to-device copy from
 * a host buffer the call frees on return, so a graph captured around such a
 * call must not be replayed; batches of at most 32 tiles per launch and no
 * chunks enqueue kernels only (schedules in the kernel arguments).
 */
int augtree_tree_bwd_noalloc(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p,
                             const uint16_t* v_p, const uint16_t* o_p, const float* lse_p,
                             const uint16_t* do_p, const uint16_t* q_r, const uint16_t* k_r,
                             const uint16_t* v_r, const uint16_t* o_r, const float* lse_r,
                             const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p, uint16_t* dv_p,
                             float* dkv_p_f32, uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r,
                             void* stream);

/* Bytes of the device array augtree_tree_bwd_noalloc works in (its limit). */
size_t augtree_noalloc_scratch_bytes(void);

/*
 * Eq. 2 reduction: the prompt-KV gradient is the prefill's own contribution
 * plus the sum of the branch seeds. Elementwise, in a fixed order (self first,
 * then terms in index order), fp32 sum and one rounding to bf16:
 *   out[t][r] = self[t][r] + sum_{k<n_parts} parts[k*part_stride + (t*part_rows + src(k,r))*E]
 * for tensor t < n_tensors (t = 0 dK, 1 dV), row r < rows, E = heads*head_dim
 * elements per row (a row is contiguous).
 *   self:  [n_tensors][rows][heads][head_dim] fp32, or NULL (treated as 0).
 *   parts: fp32; term k starts at parts + k*part_stride (elements) and holds
 *          [n_tensors][part_rows][heads][head_dim]. Dense seed slabs use
 *          part_stride = n_tensors*part_rows*E; part_stride = 0 lets every
 *          term read one slab through row_map.
 *   row_map: NULL means src(k,r) = r (then part_rows must equal rows);
 *            otherwise a DEVICE int32 array [n_parts][rows] of source rows in
 *            [0, part_rows), -1 meaning "term k has no row for r" (used to sum
 *            the prompt copies of a flattened batch).
 *   out: [n_tensors][rows][heads][head_dim] bf16 (nullable); out_f32 same
 *        shape fp32 (nullable); at least one.
 * n_tensors in {1,2}; 0 <= n_parts <= 4096; E a multiple of 4; part_stride
 * a multiple of 4 and >= 0. Source rows outside [0, part_rows) are the
 * caller's error (not checked on the device).
 */
int augtree_prompt_grad_reduce(int32_t n_tensors, int64_t rows, int32_t heads, int32_t head_dim,
                               const float* self, int32_t n_parts, int64_t part_rows,
                               int64_t part_stride, const float* parts, const int32_t* row_map,
                               uint16_t* out, float* out_f32, void* stream);

/*
 * Launch hook (instrumentation; not part of the method). When set, `hook` is
 * called on the calling thread immediately before (phase 0) and after
 * (phase 1) every kernel launch the library enqueues from that thread, with a
 * static role name ("fwd_prefill", "fwd_replay", "fwd_tree", "fwd_replay_split",
 * "lse_merge", "dq_prefill", "dkv_prefill", "dq_replay", "dkv_replay", "dq_tree",
 * "dkv_tree", "grad_reduce", "reduce_tree") and the stream the
 * kernel is enqueued on, so that a caller can record HIP events around single
 * kernels. The hook must not call back into the library. NULL removes it.
 * Per thread; the library keeps no other state.
 */
typedef void (*augtree_launch_hook)(const char* role, int phase, void* stream, void* user);
void augtree_set_launch_hook(augtree_launch_hook hook, void* user);

/*
 * Tuning of augtree_tree_bwd (process-wide; schedules and workspace sizes
 * computed after the call use it): the most query blocks (64 rows x one
 * query head) one prompt-key tile sweeps over a group's branch rows before
 * the sweep is cut into chunks. blocks >= 1 sets it, 0 restores the default
 * (1024); negative: AUGTREE_ERR_INVALID_ARGUMENT.
 */
int augtree_set_tree_chunk_blocks(int32_t blocks);
int32_t augtree_tree_chunk_blocks(void);

/* Static text of a status code. */
const char* augtree_status_string(int status);

/* Detail of the last error on the calling thread ("" if none). */
const char* augtree_last_error(void);

/* AUGTREE_OK if the current HIP device is gfx950, AUGTREE_ERR_DEVICE otherwise. */
int augtree_check_device(void);

/* Library version string. */
const char* augtree_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AUGTREE_H */
