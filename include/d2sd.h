/*
 * d2sd.h - C ABI of libd2sd: the verification hot path of dual diffusion-draft
 * speculative decoding (D^2SD, arXiv 2606.04446) on AMD Instinct MI355X (gfx950).
 *
 * One verify step of the target model over the confidence-guided prefix tree:
 *
 *   d2sd_tree_plan        host    validate (B, p_k), node counts, mask width
 *   d2sd_tree_build       device  canonical tree arrays + ancestor-or-self masks
 *   d2sd_cascade_verify_attention
 *                         device  shared-prefix (context) attention, each context
 *                                 slab read once per (split, workgroup of up to
 *                                 384 query rows) and shared by the tree nodes
 *                                 and GQA heads it holds, plus tree-suffix
 *                                 attention under the
 *                                 ancestor mask, states merged by log-sum-exp
 *   d2sd_merge_state      device  the log-sum-exp merge of two attention states
 *   d2sd_accept_path      device  greedy longest-accepted-path selection + bonus
 *   d2sd_sample_targets   device  target token per node from logits: draw at
 *                                 T > 0 (one per distinct context), argmax at T = 0
 *   d2sd_tree_from_parents device general trees (third-level cascade, resampling)
 *   d2sd_select_reanchor  device  re-anchor positions from drafter confidences (Eq. 4-5)
 *   d2sd_tree_indptr      device  node offsets of the candidate trees
 *   d2sd_commit_accepted_kv device accepted path's K/V appended to the paged cache
 *   d2sd_noncascade_verify_attention
 *                         device  same attention, context re-read per tree node
 *                                 (comparison baseline)
 *
 * Conventions (every entry point):
 *  - Ownership: the caller owns every buffer. Device pointers are device memory
 *    allocated by the caller; host pointers are ordinary host memory read only
 *    during the call. The library never frees or retains caller memory and
 *    allocates no device memory (the attention workspace is caller-provided).
 *  - Streams: device entry points enqueue kernels on `stream` (0 = the null
 *    stream) and return without synchronising. Host entry points
 *    (d2sd_tree_plan, d2sd_cascade_workspace_size, d2sd_status_string,
 *    d2sd_last_error) make no HIP call.
 *  - Errors: arguments are validated on the host before any launch. On error
 *    nothing is launched, outputs are untouched, and d2sd_last_error() returns
 *    a thread-local message. A failed launch returns D2SD_ERR_HIP. Device
 *    arrays whose contents disagree with the host-side sizes (node_indptr,
 *    ctx_len, page ids) are clamped inside the kernels so that no access leaves
 *    the buffers the host-side sizes describe; the results are then undefined.
 *  - Layouts are row-major, innermost dimension last; no padding between rows.
 *
 * Notation: B is the draft block length gamma including the anchor at block
 * position 0 (sec. 2 "DFlash", sec. 3.3 (i)); K is the number of second-draft
 * branches (Eq. 5); branch k re-anchors at block position p_k = i_k + 1 where
 * i_k in {0..B-2} is the selected prefix length (sec. 3.2), keeps the anchor and
 * the first p_k - 1 first-draft tokens, and owns tree nodes for positions
 * p_k..B-1. N_b = B + sum_k (B - p_k) is the number of tree nodes of request b.
 */
#ifndef D2SD_H_
#define D2SD_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status -- */
#define D2SD_OK 0
#define D2SD_ERR_INVALID_ARG 1          /* null pointer, bad size or value    */
#define D2SD_ERR_UNSUPPORTED 2          /* valid but not implemented shape     */
#define D2SD_ERR_WORKSPACE_TOO_SMALL 3  /* ws_bytes below the required size    */
#define D2SD_ERR_HIP 4                  /* a HIP runtime call or launch failed */

typedef int d2sd_status;

/* Element type of q, k/v cache, k/v tree and out. Accumulation is fp32. */
#define D2SD_F32 0
#define D2SD_BF16 1

/* Which key set d2sd_cascade_verify_attention attends to (field `stage`). */
#define D2SD_STAGE_CASCADE 0 /* context keys + tree ancestors (the verify pass) */
#define D2SD_STAGE_PREFIX 1  /* context keys only: the shared-prefix state      */
#define D2SD_STAGE_TREE 2    /* tree ancestors only: the tree-suffix state      */

/* Limits of this implementation. */
#define D2SD_MAX_B 64        /* block length; a request's mask row fits 2080 nodes */
#define D2SD_HEAD_DIM 128
#define D2SD_PAGE_SIZE 16
#define D2SD_MAX_VOCAB 1048576 /* logits per row for d2sd_sample_targets */

/* Static string for a status code; never NULL. */
const char* d2sd_status_string(d2sd_status s);

/* Detail of the last error raised on the calling thread ("" if none). The
 * pointer stays valid until the next d2sd_* call on the same thread. */
const char* d2sd_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int d2sd_version(void);

/* ------------------------------------------------------------ tree build -- */

/* Number of 32-bit words in one ancestor-mask row for block length B:
 * ceil((B + B(B-1)/2) / 32), the largest node count any p set can produce
 * (K = B-1, p = {1..B-1}). Returns 0 if B is outside [2, D2SD_MAX_B]. */
int d2sd_mask_words(int B);

/*
 * Host. Validates the branch sets of a batch and sizes the tree (sec. 3.2,
 * branch construction after Eq. 5; sec. 3.3 (ii)-(iii)).
 *  batch          >= 1 requests.
 *  B              block length, 2 <= B <= D2SD_MAX_B.
 *  K_host[b]      branch count of request b, 0 <= K_host[b] <= min(Kmax, B-1).
 *  p_host         [batch, Kmax]; row b holds K_host[b] distinct re-anchor
 *                 positions in [1, B-1], any order; the rest of the row is ignored.
 *  Kmax           row stride of p_host, >= 0.
 *  node_indptr_host [batch+1] out: node_indptr[0] = 0,
 *                 node_indptr[b+1] = node_indptr[b] + B + sum_k (B - p_k).
 *  mask_words_out out (nullable): d2sd_mask_words(B).
 * Errors: INVALID_ARG (node_indptr_host untouched).
 */
d2sd_status d2sd_tree_plan(int batch, int B, const int* K_host, const int* p_host, int Kmax,
                           int* node_indptr_host, int* mask_words_out);

/*
 * Device. Builds the canonical candidate tree of every request (sec. 3.2: each
 * branch keeps the anchor and the first p_k - 1 first-draft tokens and
 * re-drafts positions p_k..B-1; Fig. 1(b) step 4: the K+1 candidates share
 * their prefixes). Canonical node order of request b (indices local to b):
 *   nodes 0..B-1        main (first-draft) chain, node j = block position j,
 *                       parent j-1, root (the anchor) has parent -1;
 *   then one run per branch in ascending p_k: branch k (1-based rank) owns
 *                       B - p_k nodes for positions p_k..B-1; its first node's
 *                       parent is main node p_k - 1, later nodes chain.
 * Outputs (device, caller-allocated; global node index = node_indptr[b] + local):
 *   parent[ΣN]    local parent index (-1 for the root)
 *   depth[ΣN]     block position (0 for the root)
 *   path_id[ΣN]   0 on the main chain, k on branch k
 *   anc_mask[ΣN, mask_words]  ancestor-or-self set of the node over local node
 *                 indices, bit m of the row = word m/32, bit m%32 (LSB first)
 *   path_leaf[batch, Kmax+1]  local index of the last node of path k
 *                 (path 0 = main chain, leaf B-1); -1 for k > K[b]
 * Inputs: K[batch], p[batch, Kmax] (device, validated by d2sd_tree_plan; p in
 * any order), node_indptr[batch+1] (device, from d2sd_tree_plan).
 * total_nodes = node_indptr[batch] (host value) bounds every write.
 * mask_words must equal d2sd_mask_words(B).
 */
d2sd_status d2sd_tree_build(int batch, int B, int Kmax, const int* K, const int* p,
                            const int* node_indptr, int total_nodes, int mask_words,
                            int* parent, int* depth, int* path_id, uint32_t* anc_mask,
                            int* path_leaf, hipStream_t stream);

/*
 * Device. Trees given as parent arrays, for candidate sets that are not the
 * canonical chain-plus-branches tree: the third-level cascade (sec. 4.3:
 * every branch gets a sub-branch re-anchored inside its tail, up to 2K+1
 * candidates sharing prefixes) and independent resampling (K+1 chains under
 * the anchor). Request b's nodes are node_indptr[b] .. node_indptr[b+1]-1,
 * in topological order: local node 0 is the anchor (parent -1) and every
 * other node's parent precedes it; a parent outside [0, n) makes node n a
 * root of its own. Outputs (device, caller-allocated), same meaning as for
 * d2sd_tree_build:
 *   depth[ΣN]     edges to the root
 *   path_id[ΣN]   number of path-starting nodes m in 1..n (m starts a path
 *                 when its parent is not m - 1); equals the branch number on
 *                 a canonical tree
 *   anc_mask[ΣN, mask_words] ancestor-or-self bits over local indices
 * The outputs feed d2sd_cascade_verify_attention and d2sd_accept_path
 * unchanged (the accept path needs depths <= B - 1). 1 <= max_nodes <= 2080
 * bounds every request's node count; mask_words * 32 >= max_nodes.
 */
d2sd_status d2sd_tree_from_parents(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                   int mask_words, const int* parent, int* depth, int* path_id,
                                   uint32_t* anc_mask, hipStream_t stream);

/*
 * Device. Re-anchor selection from the first drafter's confidences (sec. 3.1
 * Eq. 3-4, sec. 3.2 Eq. 5, sec. 3.3 (ii)). For every request b:
 *   r(i) = (c_1 c_2 ... c_i) (1 - c_{i+1}),  i = 0 .. B-2,
 * the probability that exactly i drafts are accepted, evaluated in float64 in
 * that order (product from c_1 upward, then the factor 1 - c_{i+1}, no fused
 * operations), so the result is reproducible bit for bit. The min(K[b], Kmax,
 * B-1) largest r(i) are kept, equal values going to the smaller i; prefix
 * length i gives the re-anchor position p = i + 1.
 *  conf[batch, B-1]  float32, conf[b, k-1] = c_k in [0, 1] (not checked; a
 *                    NaN r(i) ranks below every number, so exactly
 *                    min(K[b], Kmax, B-1) positions are written whatever
 *                    the values).
 *  K[batch]          int32 branch counts (clamped to [0, min(Kmax, B-1)]).
 *  p_out[batch, Kmax] int32 out: the kept positions in ascending order, then
 *                    -1 up to Kmax. Feeds d2sd_tree_indptr / d2sd_tree_build.
 *  r_out[batch, B-1] float64 out (nullable): r(0 .. B-2).
 * All pointers are device pointers. Errors: INVALID_ARG (nothing launched).
 */
d2sd_status d2sd_select_reanchor(int batch, int B, int Kmax, const float* conf, const int* K, int* p_out,
                                 double* r_out, hipStream_t stream);

/*
 * Device. Node offsets of the candidate trees (same sizes as d2sd_tree_plan,
 * computed on the device): node_indptr[0] = 0, node_indptr[b+1] =
 * node_indptr[b] + B + sum_{k < K[b]} (B - p[b, k]), with K and p clamped the
 * way d2sd_tree_build clamps them (K to [0, min(Kmax, B-1)], p to [1, B-1]).
 * Unlike d2sd_tree_plan it does not validate p (distinctness is the caller's
 * contract, as for d2sd_tree_build). node_indptr: device int32 [batch+1].
 * Callers that size buffers on the host use the bound
 * batch * (B + Kmax (B-1) - Kmax (Kmax-1) / 2) for node_indptr[batch].
 */
d2sd_status d2sd_tree_indptr(int batch, int B, int Kmax, const int* K, const int* p, int* node_indptr,
                             hipStream_t stream);

/* ----------------------------------------------- cascade verify attention -- */

/*
 * Arguments of the verify attention (sec. 3.3 (iv): the target verifies the
 * K+1 candidates in one pass with shared-prefix cascade attention; sec. 1,
 * contribution 2: the shared context KV is reused rather than replicated per
 * candidate). For request b, KV head h and tree node n, query head
 * hq = h*G + g (G = num_qo_heads / num_kv_heads) attends to
 *   context keys 0..ctx_len[b]-1 of KV head h (through the page table), and
 *   the tree keys of the ancestors-or-self of n (bit set in anc_mask row n),
 * with softmax scale sm_scale. Context and tree states are combined exactly
 * by the log-sum-exp merge; the result equals one softmax over the union.
 *
 * Layouts (element type `dtype`):
 *   q        [total_nodes, num_qo_heads, head_dim]   (pre-rotated queries)
 *   k_cache, v_cache [num_pages, num_kv_heads, page_size, head_dim]
 *   page_table [batch, max_pages] int32 physical page of logical page i
 *   ctx_len  [batch] int32 (device), 0 <= ctx_len[b] <= max_ctx_len
 *   k_tree, v_tree [total_nodes, num_kv_heads, head_dim] keys/values computed
 *            for the tree nodes in this pass (the anchor is node 0)
 *   node_indptr [batch+1] int32 (device)
 *   anc_mask [total_nodes, mask_words] uint32 (from d2sd_tree_build)
 *   out      [total_nodes, num_qo_heads, head_dim]
 *   lse      [total_nodes, num_qo_heads] fp32, natural log; nullable
 * q, k_cache, v_cache, k_tree, v_tree and out must be 16-byte aligned (the
 * kernels move them in 16-byte chunks); INVALID_ARG otherwise.
 * STAGE_PREFIX writes the normalised context-only state (rows of a request
 * with ctx_len 0 get out = 0, lse = -inf); STAGE_TREE the tree-only state.
 */
typedef struct d2sd_attn_args {
  int batch;
  int num_qo_heads;
  int num_kv_heads;
  int head_dim;      /* must be D2SD_HEAD_DIM */
  int page_size;     /* must be D2SD_PAGE_SIZE */
  int dtype;         /* D2SD_F32 or D2SD_BF16 */
  int stage;         /* D2SD_STAGE_* */
  float sm_scale;    /* <= 0 selects 1/sqrt(head_dim) */
  int total_nodes;   /* host copy of node_indptr[batch] */
  int max_nodes;     /* host upper bound of node_indptr[b+1]-node_indptr[b] */
  int max_ctx_len;   /* host upper bound of ctx_len[b], <= max_pages*page_size */
  int num_pages;     /* rows of k_cache / v_cache */
  int max_pages;     /* row stride of page_table */
  int mask_words;    /* row stride of anc_mask; >= ceil(max_nodes/32) */
  int kv_split;      /* context tokens per split, multiple of 64; 0 = automatic */
  int row_group;     /* bf16 query rows per workgroup: 0 = automatic, 128 (4 waves,
                        three workgroups per CU) or 384 (12 waves sharing one K/V
                        ring, one workgroup per CU); fp32 always takes 128 */
  int packed;        /* 384-row workgroups: 0 = automatic, 1 = one stream (request,
                        KV head, split) per workgroup, 2 = workgroups over the
                        sequence of all streams' query tiles (several streams per
                        workgroup, no idle waves) when node_indptr_host is given,
                        every stream has >= 6 tiles of 32 rows, batch <= 2048 and
                        the split is <= 16384 tokens; else as 1 */
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int* page_table;
  const int* ctx_len;
  const void* k_tree;
  const void* v_tree;
  const int* node_indptr;
  const uint32_t* anc_mask;
  void* out;
  float* lse;
  const int* node_indptr_host; /* nullable: host copy of node_indptr; when given
                                  (and valid: starts at 0, ends at total_nodes,
                                  every request within max_nodes) the automatic
                                  split counts the work items exactly */
} d2sd_attn_args;

/*
 * Host. Device workspace bytes d2sd_cascade_verify_attention needs for `args`
 * (partial states of the context splits). Writes *bytes (0 when no split is
 * needed). Errors: INVALID_ARG / UNSUPPORTED as the attention call would.
 */
d2sd_status d2sd_cascade_workspace_size(const d2sd_attn_args* args, size_t* bytes);

/*
 * Host. The context split length (tokens, multiple of 64) the attention call
 * will use for `args` (args->kv_split if nonzero, else the automatic choice).
 */
d2sd_status d2sd_cascade_kv_split(const d2sd_attn_args* args, int* kv_split);

/*
 * Host. The query rows per workgroup (128 or 384) the attention call will use
 * for `args` (args->row_group if nonzero, else the automatic choice), and in
 * *packed (nullable) 1 when the 384-row workgroups run over the sequence of
 * all streams' tiles (args->packed), else 0.
 */
d2sd_status d2sd_cascade_row_group(const d2sd_attn_args* args, int* rows, int* packed);

/*
 * Device. Verify attention (see d2sd_attn_args). The M = N_b * G query rows
 * of a (request, KV head) are cut into row groups of 128 or 384 (bf16,
 * d2sd_cascade_row_group), or, in the packed shape, into the 32-row tiles of
 * the sequence of all (request, KV head, split) streams, twelve consecutive
 * tiles per workgroup; every context page slab is streamed once per
 * (context split, workgroup) and reused by all rows the workgroup holds of
 * that stream, i.e. by all G query heads of their tree nodes. The
 * workgroups of one stream run as neighbours on one XCD, so that later
 * readers of a slab can hit its L2.
 * ws: device workspace of ws_bytes >= d2sd_cascade_workspace_size(args) (may
 * be NULL when that size is 0). Concurrent calls must not share a workspace.
 */
d2sd_status d2sd_cascade_verify_attention(const d2sd_attn_args* args, void* ws, size_t ws_bytes,
                                          hipStream_t stream);

/*
 * Device. The same verify attention as d2sd_cascade_verify_attention, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): it takes no
 * workspace and allocates nothing. The split partial states live in a static
 * device scratch of the library, 64 MiB (67,108,864 bytes) per GPU, held on
 * every GPU the library runs on until the process ends. With an explicit
 * kv_split whose partial states exceed 64 MiB it returns
 * D2SD_ERR_WORKSPACE_TOO_SMALL; with the automatic split (kv_split = 0) it
 * takes the automatic plan, or, when that does not fit, the fewest-split
 * longer splits that do (the results then differ from the workspace entry
 * point's by summation order only), and returns D2SD_ERR_WORKSPACE_TOO_SMALL
 * if even ceil(max_ctx_len / 32768) splits do not fit. The scratch holds
 * nothing that must start at zero; every call on one GPU shares it and
 * leaves its last contents there, so calls that overlap on one GPU (two
 * streams, two host threads) race. Arguments, errors and outputs otherwise
 * as for d2sd_cascade_verify_attention.
 */
d2sd_status d2sd_cascade_verify_attention_noalloc(const d2sd_attn_args* args, hipStream_t stream);

/*
 * Device. Log-sum-exp merge of two attention states over disjoint key sets
 * (the cascade merge): with m = max(lse_a, lse_b), wa = exp(lse_a - m),
 * wb = exp(lse_b - m): o = (wa*o_a + wb*o_b)/(wa+wb), lse = m + ln(wa+wb).
 * A state with lse = -inf has weight 0; both -inf gives o = 0, lse = -inf.
 *  o_a, o_b, o_out [rows, head_dim] fp32; lse_a, lse_b, lse_out [rows] fp32.
 *  o_out/lse_out may alias o_a/lse_a. head_dim in [1, 1024].
 */
d2sd_status d2sd_merge_state(int rows, int head_dim, const float* o_a, const float* lse_a,
                             const float* o_b, const float* lse_b, float* o_out,
                             float* lse_out, hipStream_t stream);

/*
 * Device. The same attention as STAGE_CASCADE computed without sharing the
 * context: one workgroup per (tree node, KV head) streams the whole context
 * of its request, so the context is read N_b times per KV head. Comparison
 * baseline for the cascade kernel. args->stage must be STAGE_CASCADE;
 * kv_split is ignored. No workspace.
 */
d2sd_status d2sd_noncascade_verify_attention(const d2sd_attn_args* args, hipStream_t stream);

/* ----------------------------------------------------------- accept path -- */

/*
 * Device. Greedy longest-accepted-prefix search across the candidate tree and
 * the bonus token (sec. 2 "DFlash": accept up to, not including, the first
 * mismatch; sec. 3.3 (iv): commit the longest accepted prefix across branches,
 * the target's prediction at the rejection point is the next anchor).
 * Node c (not the root) matches iff draft_tokens[c] == target_argmax[parent(c)];
 * c is accepted iff it and all its non-root ancestors match. L is the largest
 * depth of an accepted node (0 if none); the chosen node is the accepted node
 * of depth L with the lowest canonical index (main chain first, then branches
 * by ascending p_k).
 * Inputs (device): node_indptr[batch+1]; parent, depth[ΣN] (from
 * d2sd_tree_build); path_id[ΣN]; draft_tokens[ΣN] (the root's entry is the
 * anchor and is not compared); target_argmax[ΣN] (target prediction after
 * each node).
 * Outputs (device, caller-allocated):
 *   accept_len[batch]   L, accepted draft tokens, 0 <= L <= B-1
 *   best_path[batch]    path_id of the chosen node
 *   accept_node[batch]  local index of the chosen node
 *   path_nodes[batch, B] local nodes of depths 0..L on the chosen path, -1 after
 *   out_tokens[batch, B] committed tokens: drafts at depths 1..L then the bonus
 *                       target_argmax[chosen]; L+1 valid entries, -1 after
 * total_nodes = node_indptr[batch] (host value) bounds every read.
 */
d2sd_status d2sd_accept_path(int batch, int B, const int* node_indptr, int total_nodes,
                             const int* parent, const int* depth, const int* path_id,
                             const int* draft_tokens, const int* target_argmax, int* accept_len,
                             int* best_path, int* accept_node, int* path_nodes, int* out_tokens,
                             hipStream_t stream);

/* --------------------------------------------------- sampling verification -- */

/*
 * Device. Target tokens at every tree node for verification at temperature T
 * (Tables 3-4 report T = 1 next to greedy decoding; the paper states no tree
 * rule for T > 0, so this is the rule taken here). Feed the result to
 * d2sd_accept_path as target_argmax: the longest-accepted-path selection and
 * the bonus token are then those of the sampling rule.
 *  - T > 0: node n's token is drawn from softmax(logits[r] / T) by inversion
 *    with uniform[r]: the smallest token index j with
 *      sum_{i <= j} w_i > uniform[r] * sum_i w_i,  w_i = exp((l_i - max l) / T),
 *    sums in vocabulary order (fp32 weights, fp32 sums). If rounding leaves no
 *    such j, the last token of positive weight is taken.
 *  - T = 0: the argmax of logits[r], the lowest index on ties.
 *  - r is n's representative: the lowest-index node of the same request whose
 *    root path has the same length and the same draft tokens (the same
 *    context). Nodes with one context thus share one draw, which keeps the
 *    emitted tokens distributed as the target's when branches repeat a
 *    context; a child is then accepted with probability p(its token), the
 *    rejection-sampling rule for drafted tokens taken as point masses.
 * A row with no finite logit gives -1. Logits must be finite or -inf (NaN and
 * +inf give an unspecified token in [-1, vocab)).
 * Inputs (device): node_indptr[batch+1]; parent[ΣN] (local indices, parents
 * before children, -1 for the root, as from d2sd_tree_build or
 * d2sd_tree_from_parents); draft_tokens[ΣN] (the root's entry is not
 * compared); logits[ΣN, vocab] row-major, dtype D2SD_F32 or D2SD_BF16, the
 * target's next-token logits after each node, 16-byte aligned; uniform[ΣN]
 * float32 in [0, 1) (read only for representatives; may be NULL when
 * temperature == 0).
 * Outputs (device, caller-allocated): target_tokens[ΣN] int32;
 * context_rep[ΣN] int32 local representative index (nullable).
 * 1 <= max_nodes <= 2080 must bound every request's node count; batch *
 * max_nodes < 2^31; 1 <= vocab <= D2SD_MAX_VOCAB; temperature is 0 or in
 * [1e-6, 1e6]. total_nodes = node_indptr[batch] (host value) bounds every read.
 * Root paths longer than 64 nodes leave a node as its own representative.
 */
d2sd_status d2sd_sample_targets(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                const int* parent, const int* draft_tokens, int vocab, int dtype,
                                const void* logits, float temperature, const float* uniform,
                                int* context_rep, int* target_tokens, hipStream_t stream);

/* -------------------------------------------------------- commit (cache) -- */

/*
 * Device. Commits every request's accepted path into the paged KV cache
 * (sec. 3.3: a decoding cycle consumes the verified cache and the previous
 * bonus token; the longest accepted prefix is committed and the target's
 * prediction at the rejection point becomes the next anchor). For request b
 * with context length C = ctx_len[b] and L = accept_len[b], the K and V rows
 * of the tree nodes path_nodes[b, 0..L] (the anchor, then the L accepted
 * drafts) are copied to positions C..C+L of the request's pages, position q
 * living in page page_table[b, q / page_size] at row q % page_size, and
 * ctx_len[b] becomes C + L + 1. The bonus token (out_tokens[b, L] of
 * d2sd_accept_path) is not written: it is the next cycle's anchor and its
 * K/V is computed as the root of the next tree. Nothing else in the cache
 * changes.
 *  node_indptr[batch+1], path_nodes[batch, B], accept_len[batch]: as
 *      produced by d2sd_tree_plan / d2sd_tree_indptr and d2sd_accept_path.
 *  k_tree, v_tree [total_nodes, num_kv_heads, head_dim] (dtype): this pass's
 *      tree-node K/V.
 *  page_table[batch, max_pages]: must already hold pages for every position
 *      below ctx_len[b] + B (the caller allocates them); ids are clamped to
 *      [0, num_pages).
 *  ctx_len[batch]: in/out (device). Values are clamped to [0, max_ctx_len].
 *  k_cache, v_cache [num_pages, num_kv_heads, page_size, head_dim]: out.
 * head_dim = D2SD_HEAD_DIM, page_size = D2SD_PAGE_SIZE, dtype D2SD_F32 or
 * D2SD_BF16; max_ctx_len + B <= max_pages * page_size;
 * B * num_kv_heads * head_dim * sizeof(dtype) / 16 <= 2^31 - 1. Entries of
 * path_nodes outside [0, total_nodes - node_indptr[b]) are skipped. Must not
 * run concurrently with an attention call reading the same cache or ctx_len.
 * Errors: INVALID_ARG / UNSUPPORTED before any launch.
 */
d2sd_status d2sd_commit_accepted_kv(int batch, int B, int num_kv_heads, int head_dim, int page_size, int dtype,
                                    int num_pages, int max_pages, int max_ctx_len, const int* node_indptr,
                                    int total_nodes, const int* path_nodes, const int* accept_len,
                                    const void* k_tree, const void* v_tree, const int* page_table, int* ctx_len,
                                    void* k_cache, void* v_cache, hipStream_t stream);

/* ------------------------------------------------------------ profiling -- */

/*
 * Host. When enabled (nonzero), d2sd_cascade_verify_attention and
 * d2sd_noncascade_verify_attention record HIP events on their stream before
 * their main (context-streaming) kernel, after it, and after the split merge
 * that follows it when the context is split. d2sd_kernel_timing_collect
 * waits for the recorded events, returns the call count and the summed
 * duration of the whole attention operation (main kernel + split merge) in
 * milliseconds, and clears the record. Thread-safe.
 */
d2sd_status d2sd_kernel_timing_enable(int enable);
d2sd_status d2sd_kernel_timing_collect(int* launches, double* total_ms);

/*
 * Host. As d2sd_kernel_timing_collect, but writes the duration of each
 * recorded call (main kernel + split merge, milliseconds, call order) to
 * ms_each[0 .. min(n, capacity)) (host memory, caller-owned) and the call
 * count n to *launches; durations past capacity are dropped. Clears the record.
 */
d2sd_status d2sd_kernel_timing_collect_each(int capacity, float* ms_each, int* launches);

/*
 * Host. As d2sd_kernel_timing_collect_each, with the two parts of each call
 * apart: kernel_ms[i] the main kernel, merge_ms[i] the split merge (0 when
 * the call had none). Clears the record.
 */
d2sd_status d2sd_kernel_timing_collect_parts(int capacity, float* kernel_ms, float* merge_ms, int* launches);

#ifdef __cplusplus
}
#endif

#endif /* D2SD_H_ */
