/*
 * tsubame.h - C ABI of the MI355X (gfx950) tree-replay library.
 *
 * One decoding round of Tsubame (Tree Replay for Diffusion-Based Speculative
 * Decoding) for R independent requests, over vocabulary-wide logits:
 *
 *   tsb_plan    first pass: row normalisers, planning candidates and a frozen
 *               topology by best-first expansion of draft path scores under a
 *               node budget B (Section 3.1; Appendix B.3; Figure 1).
 *   tsb_plan_ep the same first pass by expand-then-prune with a frontier
 *               width (Section 3.1; Appendix B.3).
 *   tsb_replay  second pass: refill every node of the frozen topology with
 *               fresh samples drawn without replacement from the draft
 *               distribution of its depth (Section 3.2, eq. (2); Appendix A).
 *   tsb_verify  recursive rejection sampling without replacement over the
 *               replayed tree against the target, accepted path plus one bonus
 *               token (Section 2.3, eq. (1); Appendix A; Section 3.3,
 *               Proposition 1: the probabilities used are those of the
 *               replayed candidates).
 *   tsb_step    plan -> replay -> verify with target logits supplied up front.
 *   tsb_verify_traversal, tsb_step_traversal
 *               the same round verified by traversal verification, the
 *               sequence-level verifier for trees drawn without replacement
 *               (Appendix A; Table 2).
 *
 * and the deterministic baseline of Section 3.1 with target-sample matching
 * (Table 2, Naive): tsb_first_tokens, tsb_verify_naive, tsb_step_first;
 * and the same round over sparse candidate pools with a drafter whose
 * distribution depends on the replayed prefix (Section 3.1; Section 3.2,
 * eq. (2); Section 3.3): tsb_pool_plan, tsb_pool_replay, tsb_pool_verify,
 * tsb_pool_step.
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer owned by the caller, row-major,
 *     vocabulary index fastest. The library never allocates, frees or
 *     synchronises; all work is enqueued on `stream` and returns immediately.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     non-zero status means nothing was enqueued (except TSB_E_HIP, where a
 *     launch failed part-way; tsb_last_error() has the detail).
 *   - Scratch memory comes from the caller's `workspace` of at least
 *     tsb_workspace_bytes(cfg) bytes, 256-byte aligned. Its content before a
 *     call does not matter (it need not be initialised) and nothing in it is
 *     kept between calls: the entry points are stateless. One workspace may
 *     be reused by successive calls on one stream; calls that overlap in time
 *     need separate workspaces.
 *   - Topologies and node tokens passed in by the caller are checked on the
 *     device before any entry becomes an address. A node with m > 0
 *     children is well formed when m <= TSB_MAX_K, its children occupy
 *     [first_child, first_child + m) with node < first_child and
 *     first_child + m <= n_nodes, and its depth is in [0, D); n_nodes must
 *     lie in [1, B + 1]; node tokens must lie in [0, V). Violations never
 *     fault: verification flags the request (TSB_REQ_BAD_TREE, n_acc =
 *     bonus = -1; a token outside [0, V): TSB_REQ_BAD_TOKEN, with the outputs
 *     each verifier states) and replay skips the parent (its child slots are
 *     not written). Candidate tokens given to tsb_replay that are outside
 *     [0, V) or repeated switch the pruning of their parents off.
 *   - Results are a deterministic function of (inputs, cfg.seed, step): the
 *     randomness is Philox4x32-10 (Salmon et al., SC'11) keyed by
 *     (seed, step, request, node, draw), independent of launch shapes.
 *   - Problems found on the device are reported per request in `req_status`
 *     (TSB_REQ_* bits); the outputs of such a request are defined (n_acc =
 *     -1, bonus = -1 on NONFINITE) but carry no meaning.
 *
 * Numeric contract (the paper states no precision):
 *   invT = fl32(1/T); a = fl32(x * invT) for every logit x (fp32 or bf16).
 *   draft_lse[r,d] = binary64 log-sum-exp of row a_{r,d}; its binary32
 *   rounding lse32 is canonical: topk_lp = fl32(a(tok) - lse32).
 *   Path scores are binary64 sums of topk_lp from the root.
 */
#ifndef TSUBAME_H
#define TSUBAME_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TSB_MAX_D 64   /* draft block depth */
#define TSB_MAX_K 32   /* planning candidates per position */
#define TSB_MAX_B 1023 /* non-root nodes per tree */
#define TSB_TRACE_MAX 256 /* acceptance tests recorded per request in the optional trace */

typedef enum tsb_status {
    TSB_OK = 0,
    TSB_E_NULL = 1,        /* a required pointer is NULL */
    TSB_E_SHAPE = 2,       /* R, D, V, B or K out of range, or flags that exclude each other */
    TSB_E_DTYPE = 3,       /* unknown logit dtype */
    TSB_E_TEMPERATURE = 4, /* temperature not finite or not > 0 */
    TSB_E_WORKSPACE = 5,   /* workspace too small or not 256-byte aligned */
    TSB_E_HIP = 6,         /* a HIP runtime call failed (see tsb_last_error) */
    TSB_E_DEVICE = 7       /* no usable device */
} tsb_status;

typedef enum tsb_dtype { TSB_F32 = 0, TSB_BF16 = 1 } tsb_dtype;

/* Bits of req_status[r]. */
enum {
    TSB_REQ_NONFINITE = 1,           /* NaN/+inf logit, or a row with no finite logit */
    TSB_REQ_DEGENERATE_RESIDUAL = 2, /* empty residual after a rejection: bonus drawn from p at that node */
    TSB_REQ_BUDGET_SHORT = 4,        /* fewer than B nodes exist: n_nodes < B + 1 */
    TSB_REQ_WALK_TIMEOUT = 8,        /* a cross-workgroup wait in verification hit its spin limit */
    TSB_REQ_BAD_TOKEN = 16,          /* a visited node token is outside [0, V) (tsb_pool_verify: outside its
                                        position's pool) */
    TSB_REQ_BAD_TREE = 32            /* a visited node's topology entries are out of range (see the conventions
                                        above), or n_nodes is outside [1, B + 1] */
};

/* cfg.flags */
enum {
    TSB_FLAG_NO_PRUNE = 1,   /* replay scores every token (no early rejection by the Gumbel bound) */
    TSB_FLAG_READ_ROWS = 2,  /* the WoR-RRS walk reads each target row when it enters the row's node (the
                                default when the target holds more than 128 MiB) */
    TSB_FLAG_STREAM_ROWS = 4 /* the WoR-RRS walk takes the row normalisers from a stream of every target row
                                before it (the default up to 128 MiB); not with TSB_FLAG_READ_ROWS. Results do
                                not depend on the choice, except for rounding in trace values */
};

typedef struct tsb_config {
    int32_t R;           /* requests in the batch, >= 1 */
    int32_t D;           /* draft positions (maximum tree depth), 1..TSB_MAX_D */
    int32_t V;           /* vocabulary size, K..2^30 */
    int32_t B;           /* node budget excluding the root, 0..TSB_MAX_B */
    int32_t K;           /* planning candidates per position, 1..min(TSB_MAX_K, V) */
    float temperature;   /* T > 0 */
    uint32_t dtype;      /* tsb_dtype of draft and target logits */
    uint32_t flags;      /* TSB_FLAG_* */
    uint64_t seed;       /* Philox key */
} tsb_config;

/* Frozen topology, BFS order (depth, then parent, then rank); node 0 is the
 * root; parent[i] < i; the children of a node are contiguous, in rank order.
 * Arrays are [R, B+1] except n_nodes and plan_margin ([R]). Entries at
 * i >= n_nodes[r] are filled with -1 (score: 0). */
typedef struct tsb_tree {
    int32_t* parent;      /* -1 at the root */
    int32_t* depth;       /* 0 at the root */
    int32_t* rank;        /* child slot among siblings, -1 at the root */
    int32_t* n_children;
    int32_t* first_child; /* -1 if none */
    double* score;        /* binary64 draft path log-probability, 0 at the root */
    int32_t* n_nodes;     /* 1 + committed nodes */
    double* plan_margin;  /* score(last committed) - score(best uncommitted); +inf if none left */
} tsb_tree;

/* Outputs of verification. n_acc, bonus and req_status are [R]; acc_node and
 * acc_tok are [R, D] (entries >= n_acc[r] set to -1). req_status is OR-ed
 * into (tsb_plan clears it). target_lse ([R, B+1], binary64 log-sum-exp of
 * the scaled target rows, NaN for an unusable row and beyond n_nodes) and
 * trace are optional (NULL to skip; asking for target_lse makes the WoR-RRS
 * entry points stream every row of the tree). trace is [R, TSB_TRACE_MAX, 4]
 * doubles per acceptance test, in walk order: (child node, uniform U, ratio,
 * residual mass after rejection or -1), unused entries -1. */
typedef struct tsb_verdict {
    int32_t* n_acc;
    int32_t* acc_node;
    int32_t* acc_tok;
    int32_t* bonus;
    int32_t* req_status;
    double* target_lse;
    double* trace;
} tsb_verdict;

/* Bytes of workspace every entry point needs for this configuration (0 if
 * the configuration is invalid). */
size_t tsb_workspace_bytes(const tsb_config* cfg);

/* First pass (Section 3.1). draft: [R, D, V] logits of dtype cfg.dtype.
 * Writes draft_lse [R, D] (binary64), topk_tok [R, D, K] (token ids by logit
 * desc, id asc), topk_lp [R, D, K] (binary32), the tree, and clears and sets
 * req_status [R] (NONFINITE, BUDGET_SHORT). A request with a non-finite
 * draft row gets a root-only tree. */
tsb_status tsb_plan(const tsb_config* cfg, const void* draft, double* draft_lse, int32_t* topk_tok,
                    float* topk_lp, const tsb_tree* tree, int32_t* req_status, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* First pass by expand-then-prune (Section 3.1; Appendix B.3: the EAGLE-2
 * style planner the paper uses for drafters that correct per prefix, with a
 * frontier of 10). Same inputs and outputs as tsb_plan. Layer 1 is the
 * root's K candidates; the frontier of each layer is its `frontier` best
 * nodes (score desc, rank path lexicographic asc); the next layer holds every
 * child of every frontier node; the tree is the first B generated nodes
 * under tsb_plan's order (score desc, depth asc, rank path asc), in BFS
 * order. plan_margin = score of the last chosen node - score of the first
 * generated node left out (+inf if none). With frontier >= B the tree equals
 * tsb_plan's. TSB_E_SHAPE if frontier is outside [1, 64] or the generated
 * nodes, K + sum over depths of min(layer, frontier) * K, exceed 6144. */
tsb_status tsb_plan_ep(const tsb_config* cfg, int32_t frontier, const void* draft, double* draft_lse,
                       int32_t* topk_tok, float* topk_lp, const tsb_tree* tree, int32_t* req_status,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Second pass (Section 3.2, eq. (2)). For every node u with m children at
 * depth d the children receive, in rank order, the m largest keys of
 * a_{d,v} + G(seed, step, request, u, v) over all v (Gumbel-top-k sampling
 * without replacement; equal keys to the smaller id). topk_tok is the output
 * of tsb_plan. Writes node_tok [R, B+1] (-1 at the root and beyond n_nodes). */
tsb_status tsb_replay(const tsb_config* cfg, const void* draft, const int32_t* topk_tok,
                      const tsb_tree* tree, uint32_t step, int32_t* node_tok, void* workspace,
                      size_t workspace_bytes, hipStream_t stream);

/* Verification (eq. (1); Appendix A). target: [R, B+1, V] logits, row i is
 * the target's next-token logits at tree node i (rows >= n_nodes unread).
 * draft_lse as written by tsb_plan. A visited node token outside [0, V)
 * stops the walk with TSB_REQ_BAD_TOKEN and n_acc = bonus = -1. Only the
 * target rows of the nodes the walk enters decide the request: one of them
 * with a NaN or +inf logit, or with no finite logit, ends it with
 * TSB_REQ_NONFINITE and n_acc = bonus = -1; other rows are not checked. The
 * walk reads those rows as it enters their nodes (TSB_FLAG_READ_ROWS, the
 * default above 128 MiB of target; rows 0 and 1 of every request, the root
 * and its first child, are streamed before the walk, in a round beside the
 * planner), or takes their normalisers from a stream of every row launched
 * before it (TSB_FLAG_STREAM_ROWS, the default up to 128 MiB, and whenever
 * out->target_lse is asked for). */
tsb_status tsb_verify(const tsb_config* cfg, const void* draft, const double* draft_lse,
                      const void* target, const tsb_tree* tree, const int32_t* node_tok,
                      uint32_t step, const tsb_verdict* out, void* workspace,
                      size_t workspace_bytes, hipStream_t stream);

/* plan -> replay -> verify back to back on one stream (target supplied up
 * front). When every target row is streamed (see tsb_verify), the replay
 * scan's grid carries that stream (one launch for both); otherwise it clears
 * the walk's exchange slots and the walk reads the rows of the nodes it
 * enters. Results as tsb_plan, tsb_replay and tsb_verify in turn. */
tsb_status tsb_step(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                    double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                    int32_t* node_tok, const tsb_verdict* out, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* tsb_step without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that must not
 * call hipMalloc, harnesses that forbid it). The scratch is a file-scope
 * device array of TSB_NOALLOC_SCRATCH_BYTES inside the library, one per GPU,
 * held until the process ends; its address is taken once per device on the
 * first call there. The call itself allocates and frees nothing. Every call
 * on one GPU shares that GPU's array: calls that overlap in time on one GPU
 * (other streams, other host threads) race and must be serialised by the
 * caller. Nothing in the array is carried from one call to the next (the
 * stages rewrite or clear what they read). TSB_E_WORKSPACE if
 * tsb_workspace_bytes(cfg) exceeds TSB_NOALLOC_SCRATCH_BYTES (the batched
 * workload, R = 16, V = 151936, B = 128, needs about 20 MiB). */
#define TSB_NOALLOC_SCRATCH_BYTES (32u << 20)
tsb_status tsb_step_noalloc(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                            double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                            int32_t* node_tok, const tsb_verdict* out, hipStream_t stream);

/* Traversal verification (Appendix A; Table 2: the sequence-level verifier
 * paired with sampling without replacement; compared with layer-wise RRS on
 * replayed trees in Section 4.2). Same arguments and outputs as tsb_verify,
 * except that every target row of the tree is streamed and must be usable
 * (else TSB_REQ_NONFINITE). The replayed tree is traversed in post-order (the
 * first remaining child first, down to a node with no children left); the
 * node reached is accepted, with the path from the root, with probability
 * alpha, where alpha_root = 1 and a child c with token y of node u gets
 * alpha_c = min(1, alpha_u Mb_u(y) / Ms_u(y)); Mb_u starts as p_u and Ms_u as
 * u's draft distribution. When c is rejected, u updates with the
 * distributions c was drawn from: T = sum_v max(alpha_u Mb_u - Ms_u, 0),
 * Mb_u <- max(alpha_u Mb_u - Ms_u, 0) / T, alpha_u <- T / (T + 1 - alpha_u),
 * y leaves Ms_u (renormalised). The root is accepted once its children are
 * all rejected. The bonus token is a Gumbel-max sample of Mb at the accepted
 * node (BONUS stream of that node); U of a tested node comes from its
 * ACCEPT stream. An empty residual (T <= 0 with alpha_u = 1, or an
 * exhausted Ms_u with children left) ends the round at u with a bonus from
 * p_u and TSB_REQ_DEGENERATE_RESIDUAL. trace rows are (tested node, U,
 * alpha, T after its rejection or -1). */
tsb_status tsb_verify_traversal(const tsb_config* cfg, const void* draft, const double* draft_lse,
                                const void* target, const tsb_tree* tree, const int32_t* node_tok, uint32_t step,
                                const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* plan -> replay -> traversal verification on one stream (target supplied up front). */
tsb_status tsb_step_traversal(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                              double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                              int32_t* node_tok, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* Planning tokens as node tokens: the first-pass tree verified directly is
 * the deterministic baseline First (Section 3.1; Tables 3 and 4, TopK).
 * Writes node_tok[r, i] = topk_tok[r, depth[i] - 1, rank[i]] for
 * 0 < i < n_nodes[r]; -1 at the root, beyond n_nodes, and where depth or
 * rank is out of range. topk_tok and tree as written by tsb_plan. Needs no
 * workspace. */
tsb_status tsb_first_tokens(const tsb_config* cfg, const int32_t* topk_tok, const tsb_tree* tree,
                            int32_t* node_tok, hipStream_t stream);

/* Target-sample matching (Table 2, Naive; Section 2.3): from the root, draw
 * y ~ p_u as argmax_v a_v + G(seed, step, request, u, v) over the scaled
 * target row a = fl32(target[r, u, :] * invT) (Gumbel-max, BONUS stream of
 * node u; equal keys to the smaller id); the first child of u (in rank
 * order) whose node_tok is y is accepted and the walk continues there,
 * otherwise y is the bonus token. Lossless for any tree and node tokens
 * (replayed or First). Only visited target rows are read; no normaliser is
 * computed. Writes n_acc, acc_node, acc_tok, bonus and ORs into req_status
 * (NONFINITE if a visited row holds NaN or +inf or no finite logit, or if
 * req_status already holds NONFINITE from tsb_plan: then n_acc = bonus = -1;
 * WALK_TIMEOUT as in tsb_verify). out->target_lse and out->trace are not
 * written. The walk stops accepting at depth D. */
tsb_status tsb_verify_naive(const tsb_config* cfg, const void* target, const tsb_tree* tree,
                            const int32_t* node_tok, uint32_t step, const tsb_verdict* out,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* plan -> first tokens -> naive verification on one stream: one round of the
 * First + Naive baseline (target supplied up front, one row per tree node). */
tsb_status tsb_step_first(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                          double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                          int32_t* node_tok, const tsb_verdict* out, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- pools
 * Sparse candidate pools with a drafter conditioned on the replayed prefix
 * (Section 3.1: the draft vocabulary of each position is restricted to a
 * pool of the backbone's P top-scoring tokens, the drafter's correction is
 * computed inside the pool and the corrected logits are normalised over the
 * pool; drafters that look their conditionals up in a table of transition
 * scores are planned by max-heap expansion. Section 3.2, eq. (2): replay
 * recomputes q_u under the replayed prefix with the same pools. Section 3.3:
 * verification uses these pool-normalised probabilities; the target stays
 * vocabulary-wide). The paper's pools hold 16 or 64 tokens.
 *
 *   pool_tok [R, D, P]   pool d: the P best tokens of draft row d by (logit
 *                        desc, id asc), in that order (pool slot j).
 *   trans [R, D-1, P, P] binary32 transition scores: trans[r, d-1, i, j]
 *                        corrects slot j of pool d after a token in slot i of
 *                        pool d - 1 (NULL allowed when D = 1). Every entry
 *                        must be finite, else the request is NONFINITE.
 *   For a node u at depth d >= 1 whose token holds slot s of pool d - 1:
 *     z_u(j) = fl32(a_{d,j} + fl32(trans[r, d-1, s, j] * invT)),
 *     a_{d,j} = fl32(draft[r, d, pool_tok[r, d, j]] * invT); z_root = a_0.
 *     q_u(j) = exp(z_u(j) - L_u), L_u the binary64 log-sum-exp of z_u;
 *     lp_u(j) = fl32(z_u(j) - fl32(L_u)); u's candidates are the slots by
 *     (lp desc, slot asc) with lp > -inf, at most K; child rank k of u is
 *     its k-th candidate.
 *   P must satisfy K <= P <= min(64, V). Workspaces of these entry points are
 *   tsb_pool_workspace_bytes(cfg, P) bytes (stateless, as above).
 */
size_t tsb_pool_workspace_bytes(const tsb_config* cfg, int32_t P);

/* First pass over the pools. Writes pool_tok, the tree (the first B rank
 * paths under the order of tsb_plan: score desc, depth asc, rank path asc,
 * with score the binary64 sum of lp_u along the path; plan_margin as in
 * tsb_plan) and, if plan_tok is not NULL, the planning token of every node
 * ([R, B+1], -1 at the root and beyond n_nodes: the First tree of Section
 * 3.1 over the pools). Clears and sets req_status (NONFINITE: a non-finite
 * draft row or transition score; BUDGET_SHORT). */
tsb_status tsb_pool_plan(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                         int32_t* pool_tok, const tsb_tree* tree, int32_t* plan_tok, int32_t* req_status,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Second pass over the pools, layer by layer: the m children of u receive,
 * in rank order, the pool tokens with the m largest keys
 * z_u(j) + G(seed, step, request, u, pool_tok[r, d, j]) in binary64 (G from
 * the REPLAY stream, draw = token id; equal keys to the smaller id), with
 * z_u built from the slot of u's replayed token. Writes node_tok [R, B+1]
 * (-1 at the root and beyond n_nodes). Needs no workspace. */
tsb_status tsb_pool_replay(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                           const int32_t* pool_tok, const tsb_tree* tree, uint32_t step, int32_t* node_tok,
                           hipStream_t stream);

/* Verification as tsb_verify with q_u of the pools (zero outside pool d):
 * acceptance U < max(p(y) - C q_u(y), 0) / (W q_u(y)), residual
 * max(p - C q_u, 0), bonus by Gumbel-max of the residual or of p. Node
 * tokens are looked up in their position's pool; one that is not there is
 * tested with q = 0 (accepted iff p(y) > 0), its children are built from slot
 * 0, and the request gets TSB_REQ_BAD_TOKEN. out->target_lse and out->trace
 * as in tsb_verify. */
tsb_status tsb_pool_verify(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                           const int32_t* pool_tok, const void* target, const tsb_tree* tree,
                           const int32_t* node_tok, uint32_t step, const tsb_verdict* out, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* pool plan -> pool replay -> pool verify back to back on one stream. */
tsb_status tsb_pool_step(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                         const void* target, uint32_t step, int32_t* pool_tok, const tsb_tree* tree,
                         int32_t* node_tok, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* Instrumentation (for benchmarks). On the calling thread, every later
 * launch of kernel `kernel_id` (a TSB_KERNEL_* value) is bracketed by
 * hipEventRecord(start) / hipEventRecord(stop) on the launch stream, so
 * hipEventElapsedTime(start, stop) is that kernel's duration. kernel_id < 0
 * clears the hook. The events stay owned by the caller. */
enum {
    TSB_KERNEL_DRAFT_PARTIALS = 0, /* draft row statistics + candidates (streams the draft) */
    TSB_KERNEL_PLAN_TREE = 1,      /* row merge + topology planning */
    TSB_KERNEL_REPLAY_SCAN = 2,    /* replay scan of tsb_replay (after its threshold kernel) */
    TSB_KERNEL_REPLAY_MERGE = 3,
    TSB_KERNEL_TARGET_PARTIALS = 4, /* target row statistics (streams the target; verification entry points) */
    TSB_KERNEL_VERIFY_WALK = 5,
    TSB_KERNEL_VERIFY_NAIVE = 6,    /* target-sample matching walk */
    TSB_KERNEL_POOL_PARTIALS = 7,   /* pool selection (streams the draft) */
    TSB_KERNEL_POOL_LISTS = 8,      /* pools and candidate lists of every context */
    TSB_KERNEL_POOL_PLAN = 9,       /* best-first topology over per-node candidate lists */
    TSB_KERNEL_POOL_REPLAY = 10,
    TSB_KERNEL_POOL_WALK = 11,      /* verification with pool-restricted q_u */
    TSB_KERNEL_TRAVERSAL_WALK = 12, /* traversal verification */
    TSB_KERNEL_SCAN_TARGET = 13,    /* replay scan + target row statistics in one grid (whole rounds) */
    TSB_KERNEL_COUNT = 14
};
tsb_status tsb_profile_kernel(int32_t kernel_id, hipEvent_t start, hipEvent_t stop);

/* Work counters (for benchmarks). While counting is enabled on the calling
 * thread, the replay scan, the WoR-RRS walk and the max-heap planner of
 * every later call on the current device add what they did to a counter
 * block held on that device (a file-scope array, one per device, kept until
 * the process ends; calls that overlap on one device add into the same
 * block). Counting costs a few atomic additions per wave and per request.
 * tsb_stats_read copies the block of the current device to *out after the
 * device has finished its work (a synchronous copy: not for use under stream
 * capture) and zeroes it when reset != 0. Ticks are of the 100 MHz
 * real-time counter, summed over requests. */
typedef struct tsb_stats {
    uint64_t replay_items;        /* (parent, vocabulary tile) items scanned */
    uint64_t replay_tokens;       /* tokens of the scanned tiles */
    uint64_t replay_groups_live;  /* groups of four tokens whose largest key bound reaches the parent's threshold */
    uint64_t replay_groups_keyed; /* of those, groups whose largest uniform word passes the word floor */
    uint64_t walk_requests;       /* requests walked */
    uint64_t walk_nodes;          /* nodes entered (children tested, or the bonus drawn there) */
    uint64_t walk_tests;          /* acceptance tests */
    uint64_t walk_exchanges;      /* cross-workgroup exchange rounds */
    uint64_t plan_requests;       /* requests planned */
    uint64_t plan_merge_ticks;    /* merge of the draft row partials */
    uint64_t plan_search_ticks;   /* threshold search */
    uint64_t plan_emit_ticks;     /* emission of the topology */
    uint64_t plan_rounds;         /* threshold counting rounds */
    uint64_t reserved[3];
} tsb_stats;
tsb_status tsb_stats_enable(int32_t on);
tsb_status tsb_stats_read(tsb_stats* out, int32_t reset);

const char* tsb_status_string(tsb_status status);
/* Detail of the last failure on the calling thread ("" if none). */
const char* tsb_last_error(void);
/* Library ABI version (major * 10000 + minor * 100 + patch). */
int32_t tsb_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TSUBAME_H */
