/*
 * treewy.h - C ABI of libtreewy.so: tree-structured WY verification of the
 * gated delta rule on AMD Instinct MI355X (gfx950).
 *
 * Notation (paper: Background, eq. 1; Method, eq. 2 and eq. 3).  For every
 * sequence b and value head h ("unit") there is a committed recurrent state
 * S0 in R^{d_v x d_k}.  A draft tree of N nodes is given by parent pointers
 * with parent[t] in [-1, t-1] (-1 = the node hangs directly off S0), so that
 * every ancestor of t has a smaller index.  Node t carries q_t, k_t in R^{d_k},
 * v_t in R^{d_v}, a decay gate alpha_t and a write strength beta_t.  The gated
 * delta rule S_t = alpha_t S_p (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
 * o_t = S_t q_t (eq. 1) applied along every root-to-node path defines what
 * these calls compute.
 *
 * Conventions shared by every call:
 *  - All tensor pointers are DEVICE pointers to row-major, contiguous arrays
 *    whose base address is 16-byte aligned.  The caller allocates and owns
 *    every buffer; the library allocates nothing and keeps no state between
 *    calls, so calls are re-entrant and may come from several host threads.
 *  - Sizes supported: d_k == d_v == 128, 0 <= N <= 256 (N = 0 is an empty
 *    draft), 0 <= L_max <= 256, B * H < 2^31; the fused call and the
 *    snapshot baseline take N, N_prev, L_max <= 64.  Other sizes return
 *    TREEWY_ERR_UNSUPPORTED, negative sizes TREEWY_ERR_INVALID_ARG.  B == 0 or
 *    H == 0 launches nothing and returns TREEWY_OK; so does N == 0 for the
 *    verify calls (commit with N == 0 still copies S0 to S_new).
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream) and returns after the launch.  The returned status covers only
 *    what the host can check without reading device memory; a failed launch
 *    returns TREEWY_ERR_HIP.
 *  - Malformed trees or paths are found on the device: when `err` (device
 *    int32 [B], nullable) is given, the kernels OR a TREEWY_FLAG_* bit into
 *    err[b] and never read or write out of bounds.  The caller zeroes err.
 *  - All heads of a sequence share its tree (parent[b]) and its path.
 *  - alpha must lie in (0, 1] and beta in [0, 1] (the paper's gates lie in
 *    (0, 1)); other values are not checked.
 */
#ifndef TREEWY_H
#define TREEWY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum treewy_status {
    TREEWY_OK = 0,
    TREEWY_ERR_INVALID_ARG = 1,  /* null or misaligned pointer, negative size, bad dtype */
    TREEWY_ERR_UNSUPPORTED = 2,  /* d_k or d_v != 128, N or L_max too large, too many units */
    TREEWY_ERR_HIP = 3           /* the HIP runtime refused the launch */
} treewy_status;

typedef enum treewy_dtype {
    TREEWY_F32 = 0,              /* float32 */
    TREEWY_BF16 = 1              /* bfloat16 */
} treewy_dtype;
/* in_dtype / k_dtype name the type of q, k, v and o.  state_dtype names the
 * type of S0 / S_new: float32, or bfloat16 (the state storage the paper's
 * vLLM accounting assumes, Section "The memory problem") with bfloat16 inputs
 * only.  A bfloat16 state is read exactly, all arithmetic stays float32, and
 * S_new is rounded to nearest even once when written.  U, alpha and beta are
 * always float32. */

#define TREEWY_FLAG_BAD_PARENT 1 /* some parent[b][t] outside [-1, t-1]; treated as -1 */
#define TREEWY_FLAG_BAD_PATH 2   /* path[b] is not a root-to-node path; state left unchanged */

/*
 * treewy_verify - one triangular solve for the whole draft (Method, eq. 2).
 *
 * Forms, per unit, the ancestor-masked, decay-weighted system
 *   (I + diag(beta) G) U = R,  G[t,i] = (g_t/g_i) (k_t . k_i) [i strict ancestor of t],
 *   R[t] = beta_t v_t - beta_t g_t (S0 k_t),
 * where g_t is the product of alpha over t and its ancestors, solves it for the
 * pseudo-values U (the paper's V-tilde, N x d_v), and reads every node's output
 *   o_t = g_t S0 q_t + sum over i ancestor-or-self of t of (g_t/g_i) (k_i . q_t) U[i]
 * out of the same solve (equal to S_t q_t of eq. 1).
 *
 *   S0     [B, H, d_v, d_k] state_dtype    committed states (read only)
 *   q, k   [B, H, N, d_k]   in_dtype
 *   v      [B, H, N, d_v]   in_dtype
 *   alpha, beta [B, H, N]   float32
 *   parent [B, N]           int32          parent[b][t] in [-1, t-1]
 *   o      [B, H, N, d_v]   in_dtype       written: every node's output
 *   U      [B, H, N, d_v]   float32        written: pseudo-values, read by treewy_commit
 *   err    [B] int32 or NULL               TREEWY_FLAG_BAD_PARENT
 *
 * Up to 64 nodes a unit is one pass.  Larger trees (65 to 256 nodes) are
 * walked in chunks of 64 nodes in index order; the system is block lower
 * triangular, so each chunk first adds the terms of its ancestors in earlier
 * chunks (G and the output weights against the U rows already written for
 * them) and then solves its own diagonal block.  The result is the same
 * system solved whole.
 */
treewy_status treewy_verify(const void *S0, const void *q, const void *k, const void *v,
                            const float *alpha, const float *beta, const int32_t *parent, int N,
                            int B, int H, int d_k, int d_v, treewy_dtype in_dtype, treewy_dtype state_dtype,
                            void *o, float *U, int32_t *err, void *stream);

/*
 * treewy_commit - reconstruct only the accepted node's state (Method, eq. 3):
 *   S_a = g_a S0 + sum over i on the root-to-a path of (g_a/g_i) U[i] k_i^T,
 * which becomes the next round's S0.  Replaces full-state snapshotting.
 *
 *   S0       [B, H, d_v, d_k] state_dtype  committed states
 *   U        [B, H, N, d_v]   float32      pseudo-values from treewy_verify
 *   k        [B, H, N, d_k]   k_dtype      the keys given to treewy_verify
 *   alpha    [B, H, N]        float32
 *   path     [B, L_max]       int32        root -> accepted node; entries past path_len ignored
 *   path_len [B]              int32        0 = nothing accepted: S_new = S0 bit for bit
 *   parent   [B, N] int32 or NULL          when given, each path is checked against the tree
 *   S_new    [B, H, d_v, d_k] state_dtype  written; may be the same buffer as S0 (in place)
 *   err      [B] int32 or NULL             TREEWY_FLAG_BAD_PATH (that sequence keeps S0)
 * Without `parent` a path is only checked to be strictly increasing and in [0, N).
 */
treewy_status treewy_commit(const void *S0, const float *U, const void *k, const float *alpha,
                            const int32_t *path, const int32_t *path_len, int L_max,
                            const int32_t *parent, int N, int B, int H, int d_k, int d_v,
                            treewy_dtype k_dtype, treewy_dtype state_dtype, void *S_new, int32_t *err,
                            void *stream);

/*
 * treewy_commit_verify - the previous round's commit fused into this round's
 * verify (deferred state write).  The paper's chain kernel verifies and
 * commits in one fused kernel (Implementation), and its Conclusion and the
 * ReplaySSM comparison (appendix) name deferring the state write as the next
 * lever.  Per unit this computes exactly
 *   S_new = treewy_commit(S_old, U_prev, k_prev, alpha_prev, path)   (eq. 3)
 *   (o, U) = treewy_verify(S_new, q, k, v, alpha, beta, parent)      (eq. 2)
 * but reads the state once: S_new is formed in registers, written, and used
 * as this round's S0 without a second read.
 *
 *   S_old      [B, H, d_v, d_k] state_dtype committed state before the previous round
 *   U_prev     [B, H, N_prev, d_v] float32 the previous round's pseudo-values
 *   k_prev     [B, H, N_prev, d_k] in_dtype its keys
 *   alpha_prev [B, H, N_prev] float32      its decay gates
 *   path, path_len, L_max                  its accepted paths, as for treewy_commit
 *   parent_prev [B, N_prev] int32 or NULL  its tree, to check the paths
 *   q, k, v, alpha, beta, parent, N        this round's draft, as for treewy_verify
 *   S_new      [B, H, d_v, d_k] state_dtype written (a bf16 state: rounded, and this round verifies
 *                                          from the rounded value, as the separate calls do);
 *                                          may be the same buffer as S_old
 *   o, U                                    written, as for treewy_verify
 *   err        [B] int32 or NULL           BAD_PATH (that sequence's S_new = S_old) | BAD_PARENT
 * 0 <= N_prev <= 64.  U may be the same buffer as U_prev only when N == N_prev;
 * no other output may overlap an input.  N == 0 still commits (S_new is
 * written, o and U are empty).
 */
treewy_status treewy_commit_verify(const void *S_old, const float *U_prev, const void *k_prev,
                                   const float *alpha_prev, const int32_t *path,
                                   const int32_t *path_len, int L_max, const int32_t *parent_prev,
                                   int N_prev, const void *q, const void *k, const void *v,
                                   const float *alpha, const float *beta, const int32_t *parent,
                                   int N, int B, int H, int d_k, int d_v, treewy_dtype in_dtype,
                                   treewy_dtype state_dtype, void *S_new, void *o, float *U, int32_t *err,
                                   void *stream);

/*
 * treewy_chain_prefill - run the gated delta rule (Background, eq. 1) over a
 * chain of T tokens per unit and return every token's output and the final
 * state.  This is the chain WY form that the tree method generalises
 * (Related work and Method: DeltaNet's chain transform): in chunks of 32
 * tokens (64 with fp32 tokens), each chunk is one chain verify (eq. 2) from
 * the current state, and
 * the state after its last token is rebuilt with eq. 3 and becomes the next
 * chunk's S0.  One launch on `stream`; the state stays on chip between
 * chunks, so it is read and written once per unit.
 *   S0     [B, H, d_v, d_k] state_dtype   initial state (read only unless S_T == S0)
 *   q, k   [B, H, T, d_k]   in_dtype
 *   v      [B, H, T, d_v]   in_dtype
 *   alpha, beta [B, H, T]   float32
 *   S_T    [B, H, d_v, d_k] state_dtype   written: the state after token T - 1; may be S0
 *   o      [B, H, T, d_v]   in_dtype      written: o_t = S_t q_t for every token
 *   err    [B] int32 or NULL
 * T >= 0 with T * B * H < 2^31; T == 0 copies S0 to S_T.  A bf16 state is
 * rounded once per chunk, as chunk-by-chunk commits would round it.
 */
treewy_status treewy_chain_prefill(const void *S0, const void *q, const void *k, const void *v,
                                   const float *alpha, const float *beta, int T, int B, int H, int d_k, int d_v,
                                   treewy_dtype in_dtype, treewy_dtype state_dtype, void *S_T, void *o,
                                   int32_t *err, void *stream);

/*
 * treewy_snapshot_verify - full-state-snapshotting baseline (Section "The
 * memory problem", approach (i)): runs eq. 1 node by node and writes every
 * node's full state, so that commit is a copy of one snapshot.  Same inputs
 * and outputs as treewy_verify with a float32 state (no state_dtype), except:
 *   snapshots [B, H, N, d_v, d_k] float32  written: S_t of every node
 * The speculative memory is N full states per unit instead of U.
 */
treewy_status treewy_snapshot_verify(const float *S0, const void *q, const void *k, const void *v,
                                     const float *alpha, const float *beta, const int32_t *parent,
                                     int N, int B, int H, int d_k, int d_v, treewy_dtype in_dtype,
                                     void *o, float *snapshots, int32_t *err, void *stream);

/*
 * treewy_snapshot_commit - rollback by indexing (approach (i)):
 *   S_new[b,h] = snapshots[b,h,accepted[b]], or S0[b,h] when accepted[b] == -1.
 *   accepted [B] int32 in [-1, N-1]; other values set TREEWY_FLAG_BAD_PATH and keep S0.
 *   S_new may be the same buffer as S0.
 */
treewy_status treewy_snapshot_commit(const float *S0, const float *snapshots, const int32_t *accepted,
                                     int N, int B, int H, int d_k, int d_v, float *S_new,
                                     int32_t *err, void *stream);

/*
 * treewy_path_from_node - the root-to-node path of each sequence's accepted
 * node, in the layout treewy_commit reads (Method: the accepted node's
 * ancestors and itself).  Bit exact.
 *   parent   [B, N] int32
 *   accepted [B] int32 in [-1, N-1] (-1 = nothing accepted -> path_len 0)
 *   path     [B, L_max] int32 written (root first; entries past the length set to -1)
 *   path_len [B] int32 written
 * A path longer than L_max, an out-of-range node or a malformed tree sets
 * TREEWY_FLAG_BAD_PATH and path_len[b] = 0.
 */
treewy_status treewy_path_from_node(const int32_t *parent, const int32_t *accepted, int N, int B,
                                    int L_max, int32_t *path, int32_t *path_len, int32_t *err,
                                    void *stream);

/*
 * treewy_accept_greedy - greedy acceptance of the draft tree, on the device
 * (Background: the target keeps the longest run of draft tokens it would have
 * generated itself; the paper verifies greedily, Implementation).  From the
 * committed prefix, move to the child whose draft token equals the target's
 * prediction at the current position (the lowest index among equal siblings)
 * until no child matches.  The accepted path comes out in the layout
 * treewy_commit and treewy_commit_verify read, with no host round trip.
 * Bit exact.
 *   parent       [B, N] int32
 *   draft_token  [B, N] int32              token proposed at node t
 *   target_token [B, N] int32              the target's greedy next token after node t
 *   root_token   [B] int32                 the target's greedy next token after the committed prefix
 *   path         [B, L_max] int32 written  accepted nodes, root first, then -1
 *   path_len     [B] int32 written
 *   bonus        [B] int32 or NULL         written: the target's token after the last accepted node
 *                                          (root_token when nothing is accepted)
 *   err          [B] int32 or NULL         BAD_PARENT (that parent counts as -1); BAD_PATH when the
 *                                          accepted path is longer than L_max (then path_len = 0;
 *                                          bonus is still the end of the full walk)
 */
treewy_status treewy_accept_greedy(const int32_t *parent, const int32_t *draft_token,
                                   const int32_t *target_token, const int32_t *root_token, int N, int B,
                                   int L_max, int32_t *path, int32_t *path_len, int32_t *bonus,
                                   int32_t *err, void *stream);

/* Static description of a status code; never NULL. */
const char *treewy_status_string(treewy_status status);

#ifdef __cplusplus
}
#endif

#endif /* TREEWY_H */
