/*
 * pg_attn.h -- grouped (shared-prefix) causal attention for AMD MI355X (gfx950).
 *
 * The operation is the Grouped Attention of Prefix Grouper (Section 2.1,
 * Eq. (4) and Algorithm 1): for every group, the shared prefix runs causal
 * self-attention once, and each of the group's G responses ("suffixes") runs
 * concat-attention whose queries see the whole prefix plus their own
 * response up to themselves. By Lemma 1 (Section 2.2) the outputs equal
 * standard causal attention over every [prefix; response_i] sequence
 * (Repeated-Prefix Forward, Eq. (1) and (3)), and the gradient of the shared
 * prefix is the sum of the gradients its G copies would receive there.
 *
 * Layout (all tensors contiguous, row-major, token-major "packed varlen"):
 *   q_pre, o_pre, do_pre, dq_pre : [total_prefix, h_q,  head_dim]
 *   k_pre, v_pre, dk_pre, dv_pre : [total_prefix, h_kv, head_dim]
 *   q_suf, o_suf, do_suf, dq_suf : [total_suffix, h_q,  head_dim]
 *   k_suf, v_suf, dk_suf, dv_suf : [total_suffix, h_kv, head_dim]
 *   lse_pre : float [h_q, total_prefix],  lse_suf : float [h_q, total_suffix]
 * Element type: bfloat16 (PG_BF16) or float (PG_FP32) for every tensor
 * except the log-sum-exp, which is always float (natural log).
 *
 * Grouping (device int32 arrays):
 *   cu_prefix_lens [n_groups+1]  : group g owns prefix rows
 *                                  [cu_prefix_lens[g], cu_prefix_lens[g+1]);
 *                                  [0] = 0, nondecreasing, [n_groups] = total_prefix.
 *   cu_suffix_lens [n_suffixes+1]: member m owns suffix rows
 *                                  [cu_suffix_lens[m], cu_suffix_lens[m+1]);
 *                                  [0] = 0, nondecreasing, [n_suffixes] = total_suffix.
 *   group_sizes    [n_groups]    : members per group, >= 0, summing to n_suffixes;
 *                                  members of group g follow those of group g-1.
 * Empty prefixes, empty responses and groups without members are legal.
 * GQA: query head h reads key/value head h / (h_q / h_kv); h_q % h_kv == 0.
 * head_dim must be 64 or 128 and h_q * head_dim at most 65536 (else
 * PG_EUNSUPPORTED); (total_prefix + total_suffix) * h_q must fit in 31 bits.
 * softmax_scale multiplies q.k before the softmax
 * (q and k arrive already rotary-encoded, as Algorithm 1 requires).
 *
 * Ownership and execution: every pointer except those of the size queries is
 * DEVICE memory owned by the caller. The library allocates nothing and keeps
 * no pointer after a call returns. Calls are asynchronous and ordered on the
 * given HIP stream (a hipStream_t passed as void*, NULL = the null stream).
 * Outputs are overwritten, never accumulated. Results are bitwise
 * deterministic for identical inputs (no floating-point atomics).
 *
 * Errors: each call returns a pg_status. Host-side argument checks run before
 * anything is launched, and on error no output is touched. The consistency of
 * the device grouping arrays is checked on the device: if they are
 * inconsistent no attention work is done (outputs are left as they were);
 * pg_plan_status() reports that afterwards, and with the environment variable
 * PG_DEBUG_VALIDATE=1 (which makes every call synchronise) the call itself
 * returns PG_EINVAL. HIP failures return PG_EHIP.
 * pg_last_error() gives a message for the calling thread's last failure.
 *
 * Planning: each attention call first plans its tiles on the device, in one
 * launch when every tile list fits one workgroup and in a short sequence of
 * launches otherwise; both give the same plan. PG_PLAN_MULTI=1 in the
 * environment forces the sequence (for testing).
 */
#ifndef PG_ATTN_H
#define PG_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PG_BF16 = 0, PG_FP32 = 1 } pg_dtype;

typedef enum {
  PG_OK = 0,
  PG_EINVAL = 1,       /* bad argument (sizes, null pointers, scale, grouping arrays) */
  PG_EUNSUPPORTED = 2, /* valid but unsupported (head_dim, dtype, size limits)         */
  PG_EWORKSPACE = 3,   /* workspace missing or smaller than the size query returns     */
  PG_EHIP = 4          /* HIP runtime failure (no device, launch error, ...)           */
} pg_status;

/* Workspace bytes pg_attn_fwd needs for these sizes (host call, no GPU use; 0 for negative sizes). */
size_t pg_attn_fwd_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                  int h_kv, int head_dim);

/* Workspace bytes pg_attn_bwd needs for these sizes (host call, no GPU use; 0 for negative sizes). It holds
 * the tile plan, rowsum(dO*O) and, when the walks of long prefix key tiles are split over several workgroups,
 * their fp32 dK/dV partial sums. */
size_t pg_attn_bwd_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                  int h_kv, int head_dim);

/*
 * Forward pass: Eq. (4). Writes o_pre, o_suf and the natural-log
 * log-sum-exp of every query row, lse = ln sum_s exp(softmax_scale * q.k_s)
 * over the keys the row sees (prefix row t of a group: prefix keys 0..t;
 * response row j of member i: the whole prefix and response keys 0..j of
 * member i). The log-sum-exp is what pg_attn_bwd consumes.
 */
int pg_attn_fwd(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                int h_q, int h_kv, int head_dim, float softmax_scale,
                const void* q_pre, const void* k_pre, const void* v_pre,
                const void* q_suf, const void* k_suf, const void* v_suf,
                void* o_pre, void* o_suf, float* lse_pre, float* lse_suf,
                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Forward pass without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation and the same kernels as
 * pg_attn_fwd, bitwise the same results, with the tile plan kept in a scratch
 * array of PG_NOALLOC_SCRATCH_BYTES that the library holds in each device's
 * memory until the process ends. The call allocates nothing (no hipMalloc,
 * no library allocation); on a device's first call it looks up that device's
 * copy of the array. Problems whose plan needs more than
 * pg_attn_fwd_workspace_size() <= PG_NOALLOC_SCRATCH_BYTES bytes are rejected
 * with PG_EUNSUPPORTED before anything is launched (16 MiB holds the plan of
 * about four million response rows). Every call on one device shares that
 * device's array: calls that overlap in time on one device (other streams,
 * other threads) race and must not be issued. Arguments, layout, ownership
 * and the other errors are those of pg_attn_fwd.
 */
#define PG_NOALLOC_SCRATCH_BYTES (16u << 20)
int pg_attn_fwd_noalloc(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                        const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                        int h_q, int h_kv, int head_dim, float softmax_scale,
                        const void* q_pre, const void* k_pre, const void* v_pre,
                        const void* q_suf, const void* k_suf, const void* v_suf,
                        void* o_pre, void* o_suf, float* lse_pre, float* lse_suf, void* stream);

/*
 * Backward pass: the vector-Jacobian product of the forward with upstream
 * gradients do_pre, do_suf (Lemma 1 and its proof, Appendix A.1). dq/dk/dv of
 * the suffix rows are those of each member's own rows; dq_pre, dk_pre, dv_pre
 * are the full gradients of the shared prefix, i.e. summed over all G members
 * (and, for dk/dv, over the query heads sharing a key/value head), reduced in
 * a fixed order. o_* and lse_* must be the forward's outputs for the same
 * inputs.
 */
int pg_attn_bwd(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                int h_q, int h_kv, int head_dim, float softmax_scale,
                const void* q_pre, const void* k_pre, const void* v_pre,
                const void* q_suf, const void* k_suf, const void* v_suf,
                const void* o_pre, const void* o_suf, const float* lse_pre, const float* lse_suf,
                const void* do_pre, const void* do_suf,
                void* dq_pre, void* dk_pre, void* dv_pre,
                void* dq_suf, void* dk_suf, void* dv_suf,
                void* workspace, size_t workspace_bytes, void* stream);

/*
 * The same two calls on the single-buffer layout of Eq. (2): every tensor is one
 * buffer whose rows are, group after group, the group's prefix rows followed by
 * the response rows of its members in member order ([P; R_1; ...; R_G]), so
 * q, k, v, o, do, dq, dk, dv are [total_prefix + total_suffix, h, head_dim] and
 * lse is [h_q, total_prefix + total_suffix] fp32 in the same row order. This is
 * the layout the paper feeds (X_ours); splitting it into prefix and response
 * parts ("ungroup") and putting the outputs back ("group") cost nothing. The
 * grouping arrays, sizes, numerics, workspace sizes (same queries), determinism
 * and error behaviour are those of pg_attn_fwd / pg_attn_bwd; results are
 * bitwise identical to theirs on the same rows.
 */
int pg_attn_fwd_xours(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                      const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                      int h_q, int h_kv, int head_dim, float softmax_scale,
                      const void* q, const void* k, const void* v, void* o, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream);

int pg_attn_bwd_xours(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                      const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                      int h_q, int h_kv, int head_dim, float softmax_scale,
                      const void* q, const void* k, const void* v, const void* o, const float* lse,
                      const void* d_o, void* dq, void* dk, void* dv,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Forward of the final token of every member only (Section 2, "Further
 * discussion": multi-QA judging, where a long response is the shared prefix,
 * each short question a member, and predictions come from the hidden state at
 * each question's final token). For member i the query is the last row of the
 * sequence [P; R_i] (its last response row, or the group's last prefix row when
 * the response is empty); it attends to the whole prefix and to all of R_i, as
 * in pg_attn_fwd. Outputs: o_last [n_suffixes, h_q, head_dim] (dtype of the
 * inputs) and lse_last [h_q, n_suffixes] fp32 (natural log). A member whose
 * sequence is empty (no prefix, no response) gets zeros and lse = -inf.
 * Inputs, grouping arrays, sizes and errors as for pg_attn_fwd; additionally
 * h_q / h_kv <= 128. Workspace: pg_attn_fwd_last_workspace_size(...) bytes
 * (it holds per-chunk fp32 partial results). Deterministic.
 */
size_t pg_attn_fwd_last_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                       int h_kv, int head_dim);

int pg_attn_fwd_last(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                     const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                     int h_q, int h_kv, int head_dim, float softmax_scale,
                     const void* q_pre, const void* k_pre, const void* v_pre,
                     const void* q_suf, const void* k_suf, const void* v_suf,
                     void* o_last, float* lse_last, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Rotary position embedding with grouped position ids, the step before the
 * attention calls (Algorithm 1 takes q and k already rotary-encoded). Each
 * token gets the position it has in the Repeated-Prefix Forward (Section 2,
 * "Algorithm implementation", after Eq. (4)): prefix row t of a group is at
 * position t, row j of any member's response at P + j, P being the group's
 * prefix length. Positions are derived from the grouping arrays (same
 * meaning as for pg_attn_fwd); no position tensor is needed.
 *
 * The first rotary_dim dimensions of every head vector form rotary_dim / 2
 * pairs; pair i turns by the angle pos * base^(-2 i / rotary_dim) (computed in
 * double precision), the other dimensions are copied unchanged. Pair layout:
 * half-split (pair i = dims i and i + rotary_dim/2) by default,
 * PG_ROPE_INTERLEAVED for dims 2i and 2i+1. PG_ROPE_INVERSE turns by the
 * negative angle: applied to the gradients of the rotated q and k it gives the
 * gradients of the unrotated ones (the rotation is orthogonal).
 *
 * Tensors: q_* [rows, h_q, head_dim], k_* [rows, h_kv, head_dim], dtype as for
 * the attention calls, contiguous, 16-byte aligned device pointers; *_out may
 * equal the input (in place). h_q or h_kv may be 0 to rotate only the other
 * tensor (its pointers may then be NULL). head_dim is 64 or 128, rotary_dim a
 * multiple of 16 in [16, head_dim], (h_q + h_kv) * head_dim <= 65536, base
 * finite and > 0. Workspace: pg_rope_workspace_size(n_groups) bytes of device
 * memory. Errors as for the attention calls (host checks before any launch;
 * inconsistent grouping arrays leave the outputs untouched, reported only
 * under PG_DEBUG_VALIDATE=1).
 */
typedef enum { PG_ROPE_INVERSE = 1, PG_ROPE_INTERLEAVED = 2 } pg_rope_flags;

size_t pg_rope_workspace_size(int n_groups);

int pg_rope(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
            const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
            int h_q, int h_kv, int head_dim, int rotary_dim, double base, int flags,
            const void* q_pre, const void* q_suf, const void* k_pre, const void* k_suf,
            void* q_pre_out, void* q_suf_out, void* k_pre_out, void* k_suf_out,
            void* workspace, size_t workspace_bytes, void* stream);

/*
 * The grouped position ids themselves: pos_pre [total_prefix] and pos_suf
 * [total_suffix] int32 device arrays, by the rule of pg_rope (for callers that
 * apply their own positional encoding). Workspace as for pg_rope.
 */
int pg_grouped_positions(int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                         const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                         int32_t* pos_pre, int32_t* pos_suf, void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * Kernel timing for benchmarks. Between pg_timing_start() and pg_timing_stop()
 * every call brackets each of its kernel launches with a pair of HIP events
 * recorded on the call's stream (at most 16384 launches are recorded per start;
 * later ones are not). pg_timing_get() waits for the recorded events and
 * returns, for one kernel kind, how many launches were recorded and their
 * summed duration in milliseconds. pg_timing_start() discards earlier records.
 * Not meant to be used while other threads issue calls.
 */
typedef enum {
  PG_K_PLAN = 0,     /* the planner kernels of one call, as one interval      */
  PG_K_FWD = 1,      /* forward attention kernel                              */
                     /* 2: unused (rowsum(dO * O) is formed inside the dQ kernel) */
  PG_K_DKDV = 3,     /* backward: dK, dV (key-stationary, G-way prefix sum)   */
  PG_K_DQ = 4,       /* backward: dQ and rowsum(dO * O) (query-stationary)    */
  PG_K_ROPE = 5,     /* rotary embedding kernel of pg_rope                    */
  PG_K_LAST = 6,     /* pg_attn_fwd_last: chunk kernel and merge, one interval */
  PG_K_KV_REDUCE = 7 /* backward: fixed-order sum of the prefix dK/dV partials  */
} pg_kernel;

int pg_timing_start(void);
int pg_timing_stop(void);
int pg_timing_get(int kernel, int* launches, double* total_ms);

/*
 * Verdict of the device-side check of the grouping arrays in the last call
 * that used this workspace (pg_attn_fwd, pg_attn_bwd, their _xours forms,
 * pg_attn_fwd_last, pg_rope, pg_grouped_positions), or with workspace == NULL
 * the last pg_attn_fwd_noalloc on the current device: PG_OK when they were
 * consistent, PG_EINVAL when they were not (that call did no work). It waits
 * for the stream (the one that call used) to finish. PG_EWORKSPACE when the
 * workspace is smaller than a plan header (256 bytes).
 */
int pg_plan_status(const void* workspace, size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* pg_status_string(int status);

/* Message for the calling thread's most recent failing call ("" if none). */
const char* pg_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PG_ATTN_H */
