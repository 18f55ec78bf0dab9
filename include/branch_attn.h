/*
 * branch_attn.h -- C ABI of the MI355X (gfx950) branch-attention library.
 *
 * Draft branch attention under context parallelism (Sec. 3.2 of "Online Draft
 * Co-Training for Speculative Decoding in Large-Scale, Long-Context RL
 * Post-Training"): every branch query attends (a) a causal prefix of its main
 * sequence, which is sharded over CP ranks with the packed zigzag ring, and
 * (b) its own branch's keys, which never leave the rank holding the anchor
 * token.  Both parts are attended separately and combined by log-sum-exp
 * rescaling (Eq. lse-merge).  For gradients the ring is walked a second time
 * and every rank sums its contributions in place (Sec. 3.2).
 *
 * This library evaluates ONE rank's share on one GPU.  The KV blocks that a
 * real ring would deliver step by step (one per rank) are all resident in
 * device memory and are passed as an array of pointers.
 *
 * Conventions shared by every entry point
 *   - Status: BA_OK (0) on success, a negative BA_E_* code otherwise; no C++
 *     exception crosses the ABI.  branch_attn_last_error() describes the last
 *     failure of the calling thread.  Nothing is launched when validation
 *     fails.  Kernel faults surface asynchronously at the caller's next
 *     synchronisation of the stream.
 *   - Streams are hipStream_t values passed as void* (NULL = default stream).
 *     Every device entry point is asynchronous with respect to the host.
 *   - Device tensors are dense, row-major "token, head, dim" (THD) arrays of
 *     bf16 (raw 16-bit storage) unless stated otherwise.  LSE arrays are fp32
 *     [heads, rows] and hold natural logarithms.
 *   - Grouped-query attention: query head h reads key/value head
 *     h / (hq / hkv).
 *   - The library never allocates device memory: scratch space is the
 *     caller-provided workspace.
 */
#ifndef BRANCH_ATTN_H
#define BRANCH_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ codes */
#define BA_OK 0
#define BA_E_INVAL (-1)        /* malformed arguments / descriptors        */
#define BA_E_UNSUPPORTED (-2)  /* valid but not implemented (head_dim, GPU)*/
#define BA_E_HIP (-3)          /* a HIP runtime call or launch failed       */
#define BA_E_WORKSPACE (-4)    /* workspace missing or too small            */

/* Branch structures of the three draft families (Sec. 3.2). */
#define BA_KIND_EAGLE_CHAIN 0  /* EAGLE-3 train-time test: member i sees members 0..i   */
#define BA_KIND_DFLASH_BLOCK 1 /* DFlash / DSpark block: every member sees every member */

#define BA_DTYPE_BF16 0
#define BA_DTYPE_F32 1

/* How the main-sequence ring is executed.
 * BA_MODE_PER_STEP: one launch per ring step, each merging its partial result
 *   into a running fp32 (O, LSE) pair with Eq. lse-merge; the branch-local
 *   part is then merged by a final launch.  This is the schedule a real
 *   C-rank ring runs.
 * BA_MODE_FUSED: one launch walks every ring step's KV block for a query
 *   tile, carrying the running (O, LSE) in registers (the online-softmax
 *   rescale is Eq. lse-merge applied between steps), then merges the
 *   branch-local part with Eq. lse-merge and writes the result; the
 *   backward's dQ likewise.
 * In both, the backward's dK/dV (of each ring step's KV block) is launched
 * once per ring step. */
#define BA_MODE_PER_STEP 0
#define BA_MODE_FUSED 1
/* BA_MODE_AUTO: the plan picks one of the two; today the fused schedule for
 * every plan, measured the faster one on one GPU for every share (the
 * per-step schedule pays a running-sum pass per ring step and finalize
 * passes; both launch dK/dV per ring step).  branch_attn_plan_mode reports
 * the choice.  Accepted wherever a mode is. */
#define BA_MODE_AUTO 2

#define BA_MAX_GROUP_LEN 64    /* members per branch group                 */
#define BA_HEAD_DIM 128        /* the only head_dim with kernels            */

/* Branch-anchor descriptor: one branch (an EAGLE-3 chain at one position, or
 * one DFlash block).  Its members live in the rank-local branch arrays at rows
 * row0 + i * row_stride, i = 0..len-1.  The branch's causal main prefix is the
 * main keys of sequence `seq` at positions 0..anchor (inclusive).  A group
 * must be anchored in a chunk owned by the evaluated rank (Sec. 3.2: branch
 * keys stay with the rank that holds the anchor token). */
typedef struct ba_group {
  int32_t seq;
  int32_t anchor;
  int32_t kind;        /* BA_KIND_* */
  int32_t len;         /* 1..BA_MAX_GROUP_LEN */
  int32_t row0;
  int32_t row_stride;  /* >= 1 */
} ba_group;

/* One rank's share of a packed varlen problem (all arrays on the HOST and
 * only read during branch_attn_plan_create / zigzag_partition).
 *   cu_seqlens  [num_seqs+1] global packed offsets, non-decreasing, starting
 *               at 0; every length must be a multiple of 2*cp_size (zigzag).
 *   has_main    [num_seqs] 1 if the sequence's main tokens are queries too
 *               (EAGLE-3 trains depth 0), 0 if only its branches are
 *               (DFlash); NULL means all 1.
 *   The rank-local main arrays hold the rank's tokens of every sequence
 *   (chunk r then chunk 2C-1-r, see zigzag_partition), n_local =
 *   cu_seqlens[num_seqs] / cp_size rows. */
typedef struct ba_problem {
  int32_t num_seqs;
  const int32_t* cu_seqlens;
  const uint8_t* has_main;
  int32_t cp_size;
  int32_t cp_rank;
  int32_t hq;
  int32_t hkv;
  int32_t head_dim;
  float softmax_scale;
  int32_t num_groups;
  const ba_group* groups;
  int32_t num_branch_rows;
} ba_problem;

/* Device pointers of one forward call.  k_step / v_step are HOST arrays of
 * cp_size device pointers: entry j is rank j's local main K (V), [n_local,
 * hkv, d], in rank j's zigzag-local order (what the ring delivers at the step
 * that brings rank j's block).  Branch arrays are [num_branch_rows, h, d].
 * Outputs: o_main [n_local, hq, d] bf16 (rows of sequences without main
 * queries are left untouched), o_br [num_branch_rows, hq, d] bf16, lse_main
 * [hq, n_local], lse_br [hq, num_branch_rows] fp32 (natural log).  Rows of
 * the branch arrays not covered by any group are neither read nor written.
 * Pointers may be NULL when the corresponding row count is 0.
 * ring_begin / ring_end: optional hipEvent_t (NULL = none), recorded on the
 * call's stream right before the first and right after the last launch of the
 * main-sequence (ring) kernels, so a caller can time that part alone. */
typedef struct ba_fwd_io {
  const void* q_main;
  const void* q_br;
  const void* k_br;
  const void* v_br;
  const void* const* k_step;
  const void* const* v_step;
  void* o_main;
  void* o_br;
  float* lse_main;
  float* lse_br;
  void* ring_begin;
  void* ring_end;
} ba_fwd_io;

/* Device pointers of one backward call.  Inputs as in ba_fwd_io plus the
 * forward outputs (o_*, lse_*) and the output gradients do_main / do_br
 * (bf16, same shapes as o_*).  Outputs (dtype grad_dtype, overwritten, not
 * accumulated): dq_main / dq_br like q_*, dk_step[j] / dv_step[j] like
 * k_step[j] (the gradient contributed by THIS rank's queries to rank j's
 * block; a real ring returns it to rank j), dk_br / dv_br like k_br.  The
 * LSE outputs receive no gradient.  ring_begin / ring_end as in ba_fwd_io;
 * kv_end (optional hipEvent_t) is recorded between the dK/dV launches and
 * the dQ launches of the ring part (in BA_MODE_PER_STEP all C dK/dV steps
 * are launched before the C dQ steps). */
typedef struct ba_bwd_io {
  const void* q_main;
  const void* q_br;
  const void* k_br;
  const void* v_br;
  const void* const* k_step;
  const void* const* v_step;
  const void* o_main;
  const void* o_br;
  const float* lse_main;
  const float* lse_br;
  const void* do_main;
  const void* do_br;
  void* dq_main;
  void* dq_br;
  void* const* dk_step;
  void* const* dv_step;
  void* dk_br;
  void* dv_br;
  int32_t grad_dtype;  /* BA_DTYPE_BF16 or BA_DTYPE_F32 */
  void* ring_begin;
  void* ring_end;
  void* kv_end;
} ba_bwd_io;

typedef struct ba_plan ba_plan; /* opaque, host-side */

/* ------------------------------------------------------------ host calls */

/* Zigzag partition of a packed batch (Sec. 3.2, packed zigzag ring; each
 * sequence is cut into 2*cp_size equal chunks and rank r owns chunks r and
 * 2*cp_size-1-r).  HOST arrays, all caller-allocated:
 *   local_cu_seqlens [num_seqs+1]  rank-local offsets (L_s / cp_size each)
 *   local_to_global  [n_local]     global packed index of each local token
 *   local_pos        [n_local]     position of each local token in its sequence
 * Local order per sequence is chunk r followed by chunk 2C-1-r.
 * BA_E_INVAL if num_seqs < 1, cp_size < 1, cp_rank outside [0, cp_size),
 * cu_seqlens[0] != 0, a length is negative or not a multiple of 2*cp_size. */
int zigzag_partition(const int32_t* cu_seqlens, int32_t num_seqs, int32_t cp_size,
                     int32_t cp_rank, int32_t* local_cu_seqlens, int32_t* local_to_global,
                     int32_t* local_pos);

/* Validate a problem and build its execution plan on the host (query token
 * list ordered by causal limit, query tiles, KV tiles and their ring-step
 * classes).  The problem's arrays are copied; the caller may free them.
 * BA_E_INVAL on malformed descriptors (group anchored on another rank,
 * member rows out of range or overlapping, hq % hkv != 0, ...),
 * BA_E_UNSUPPORTED if head_dim != 128.  *out is NULL on failure. */
int branch_attn_plan_create(const ba_problem* prob, ba_plan** out);
void branch_attn_plan_destroy(ba_plan* plan);

/* Rotary position embedding in front of the attention: the step before the
 * op inside a draft layer, whose queries and keys are rotated by their
 * positions.  The paper gives no positional scheme for branch tokens; this
 * library's reading: a main token at position p of its sequence has
 * position p, member i (0-based) of a branch group anchored at a has
 * position a + 1 + i (an EAGLE-3 member of depth i + 1, or block position
 * i + 1 of a DFlash block, after its anchor).  Dims j and j + 64 (j < 64)
 * turn together by the angle pos * theta^(-j/64) (x_j' = x_j cos - x_{j+64}
 * sin, x_{j+64}' = x_{j+64} cos + x_j sin); the rotated queries and keys are
 * evaluated in double (angle, sine, cosine, products) and rounded once to
 * bf16 (RNE) before attending, values are not rotated.
 * With theta > 0 every later branch_attn_fwd / branch_attn_bwd call on the
 * plan attends the rotated queries and keys, and the backward returns dQ and
 * dK with respect to the unrotated inputs (the transposed rotation of the
 * gradients of the rotated ones).  theta = 0 turns the rotation off.  The
 * plan's workspace sizes grow (query them again): rotated copies of Q and K,
 * and fp32 staging of the gradients.  Host only.  BA_E_INVAL for a negative
 * or non-finite theta, BA_E_UNSUPPORTED if a position reaches 2^24. */
int branch_attn_plan_set_rope(ba_plan* plan, float theta);

/* Positions of the plan's rows, host arrays filled by the call:
 * main_pos[u] (n_local entries) is the position in its sequence of local
 * main row u, br_pos[b] (num_branch_rows entries) is a + 1 + i for member i
 * of a group anchored at a, -1 for a row of no group.  The positions the
 * rotary embedding of branch_attn_plan_set_rope uses, and the ones to pass to
 * branch_attn_qkv_fwd / _bwd.  Either pointer may be NULL (skipped). */
int branch_attn_plan_positions(const ba_plan* plan, int32_t* main_pos, int32_t* br_pos);

/* The schedule `mode` stands for with this plan (BA_MODE_AUTO resolved;
 * the other modes map to themselves).  Host only.  BA_E_INVAL for an unknown
 * mode. */
int branch_attn_plan_mode(const ba_plan* plan, int32_t mode, int32_t* resolved);

/* Workspace bytes needed by branch_attn_fwd / branch_attn_bwd in `mode`. */
int branch_attn_workspace_size(const ba_plan* plan, int32_t mode, size_t* fwd_bytes,
                               size_t* bwd_bytes);

/* Rank-local row counts of a plan: n_local main rows, number of query
 * tokens (main + branch rows that are queries). */
int branch_attn_plan_info(const ba_plan* plan, int64_t* n_local, int64_t* n_query_tokens);

/* Useful FLOPs of one forward / backward call: allowed (query, key) pairs
 * summed over query heads, times 4*head_dim (QK^T and PV) forward and
 * 10*head_dim (QK^T recompute, dP, dV, dK, dQ) backward.  Work spent on
 * masked-out pairs inside partial tiles is not counted. */
int branch_attn_useful_flops(const ba_plan* plan, double* fwd_flops, double* bwd_flops);

/* Allowed (query, key) pairs per query head, split into the causal
 * main-sequence prefix (computed by the ring kernels) and the branch-local
 * keys. */
int branch_attn_pair_counts(const ba_plan* plan, double* main_pairs, double* local_pairs);

/* Message for the last non-OK status returned on this thread. */
const char* branch_attn_last_error(void);

/* ---------------------------------------------------------- device calls */

/* Forward (Sec. 3.2): writes O and LSE of every query of the rank share.
 * `workspace` is device memory of at least the fwd_bytes reported by
 * branch_attn_workspace_size for the same mode, 256-byte aligned; its
 * content on entry is irrelevant and it is clobbered.  Concurrent calls
 * must use distinct workspaces. */
int branch_attn_fwd(void* stream, const ba_plan* plan, int32_t mode, const ba_fwd_io* io,
                    void* workspace, size_t workspace_bytes);

/* branch_attn_fwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The scratch is a static device array of
 * 64 MiB per GPU, held until the process ends; it covers the fused forward of
 * every workload up to the 256K-token share (4 MiB of plan tables there),
 * and the per-step schedule of small shares.  Allocates nothing: no
 * hipMalloc, hipFree or allocating library call.  BA_E_WORKSPACE if the plan
 * and mode need more scratch than that (per-step running sums of large
 * shares, rotary-embedding copies); other errors as branch_attn_fwd.  Every
 * call on one GPU shares that GPU's scratch: calls that overlap on one GPU
 * (several streams or threads) race and must be serialised by the caller.
 * Results are identical to branch_attn_fwd with the same plan and mode. */
int branch_attn_fwd_noalloc(void* stream, const ba_plan* plan, int32_t mode, const ba_fwd_io* io);

/* Backward (Sec. 3.2: the ring is replayed and gradients accumulate
 * locally): gradients of sum <dO, O> with respect to every input of the
 * rank share.  Workspace rules as for branch_attn_fwd (bwd_bytes). */
int branch_attn_bwd(void* stream, const ba_plan* plan, int32_t mode, const ba_bwd_io* io,
                    void* workspace, size_t workspace_bytes);

/* In-place merge of a partial attention result into a running one
 * (Eq. lse-merge): l = log(e^l_acc + e^l_part),
 * o_acc = e^(l_acc - l) o_acc + e^(l_part - l) o_part.
 *   o_acc    fp32 [rows, heads, head_dim], device
 *   lse_acc  fp32 [heads, rows], natural log, device
 *   o_part   [rows, heads, head_dim] of dtype o_part_dtype (BA_DTYPE_BF16 or
 *            BA_DTYPE_F32), normalised partial output, device
 *   lse_part fp32 [heads, rows], device
 * A partial with LSE = -inf has zero weight; when both are -inf the result
 * is O = 0, LSE = -inf.  head_dim must be a multiple of 4.  Asynchronous on
 * `stream`; rows == 0 is a no-op. */
int lse_merge(void* stream, int64_t rows, int32_t heads, int32_t head_dim, float* o_acc,
              float* lse_acc, const void* o_part, int32_t o_part_dtype, const float* lse_part);

/* ------------------------------------------- QKV projection (draft layer)
 *
 * The step in front of the op inside a draft layer (the paper gives no
 * projection detail; this library reads the draft layer as a Llama-style
 * decoder layer, its own reading): grouped-query projection
 * of hidden states to q-, k- and v-heads, with the rotary embedding of
 * branch_attn_plan_set_rope applied to the queries and keys.  Plan-free: the
 * caller projects the main rows and the branch rows in separate calls, with
 * the positions of branch_attn_plan_positions, and hands the results to
 * branch_attn_fwd with the plan's own rotation off (theta 0).
 *
 *   x    bf16 [rows, hidden], hidden a positive multiple of 128
 *   w    bf16 [(hq + 2 hkv) * 128, hidden]: the fused q/k/v weight of a
 *        linear layer (output-major, like torch.nn.Linear.weight), rows
 *        0 .. hq*128-1 the q-heads, then hkv k-heads, then hkv v-heads
 *   pos  int32 [rows], device; a row with a negative position is not
 *        rotated; read only when theta > 0 (positions below 2^24 keep the
 *        angle error near 1e-7 rad)
 *   theta  rotary base (> 0), or 0 for no rotation
 * All device pointers 16-byte aligned; hq % hkv == 0.  BA_E_INVAL for
 * malformed arguments, BA_E_UNSUPPORTED for a hidden size that is not a
 * multiple of 128.  rows == 0 is a no-op (the backward still clears dw
 * unless accumulate_dw).  Asynchronous on `stream`. */

/* q = R(pos) (x W_q^T), k = R(pos) (x W_k^T), v = x W_v^T, fp32 accumulation,
 * each rounded once to bf16 (RNE): q [rows, hq, 128], k and v
 * [rows, hkv, 128]. */
int branch_attn_qkv_fwd(void* stream, int64_t rows, int32_t hidden, int32_t hq, int32_t hkv, const void* x,
                        const void* w, const int32_t* pos, float theta, void* q, void* k, void* v);

/* Backward of branch_attn_qkv_fwd for the loss gradients dq, dk, dv (dtype
 * grad_dtype, the layouts of q, k, v; the gradients of the rotated queries
 * and keys, as branch_attn_bwd returns them for a plan without rotation):
 * dY = [R^T dq, R^T dk, dv] rounded to bf16 into the workspace, then
 *   dx [rows, hidden] (dtype dx_dtype) = dY W,
 *   dw [(hq + 2 hkv) * 128, hidden] fp32 = dY^T x, or dw += dY^T x when
 *   accumulate_dw is non-zero (main and branch rows share the weight).
 * The workspace (device, 256-byte aligned) holds at least the bytes of
 * branch_attn_qkv_workspace_size; BA_E_WORKSPACE otherwise. */
int branch_attn_qkv_bwd(void* stream, int64_t rows, int32_t hidden, int32_t hq, int32_t hkv, const void* x,
                        const void* w, const int32_t* pos, float theta, const void* dq, const void* dk,
                        const void* dv, int32_t grad_dtype, void* dx, int32_t dx_dtype, float* dw,
                        int32_t accumulate_dw, void* workspace, size_t workspace_bytes);

/* Workspace bytes of branch_attn_qkv_bwd: rows * (hq + 2 hkv) * 128 * 2. */
int branch_attn_qkv_workspace_size(int64_t rows, int32_t hq, int32_t hkv, size_t* bytes);

#ifdef __cplusplus
}
#endif

#endif /* BRANCH_ATTN_H */
