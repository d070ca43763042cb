/*
 * tss.h -- C ABI of the sparse-depth target verification step (TSS) on MI355X.
 *
 * The library verifies a chain or tree of drafted tokens with one forward pass
 * of a LLaMA-shaped decoder in which the blocks named by a skip mask are
 * bypassed, then takes the greedy accept decision.  Sources in the paper
 * (arXiv 2609.26100, "TSS: Target-Side Sparsification for Speculative
 * Decoding in Domain-Specific Large Language Models"):
 *   - Method / Problem Formulation: the sparse verifier T_S is the target with
 *     the blocks in S bypassed; S = {} is the dense verifier; the target
 *     verifies the draft's candidate tokens in parallel.
 *   - Method / Domain-Aware Skip Controller: the skip set is fixed for a whole
 *     request (unknown domains fall back to the dense path), and before each
 *     block the forward checks the layer index against it: a skipped block
 *     passes its input hidden state through, with no attention and no
 *     feed-forward work.
 *   - Experiments / Models and speculative decoding methods, and Appendix /
 *     Evaluation Protocol: greedy decoding (temperature 0) with the underlying
 *     method's accept/reject logic unchanged.
 *   - Appendix / Models: LLaMA targets (pre-norm RMSNorm blocks, rotary
 *     embedding, multi-head attention, SwiGLU MLP, untied lm_head).
 *
 * Conventions shared by every call:
 *   - Every function returning int returns TSS_OK (0) or a negative
 *     tss_status; no C++ exception crosses the ABI.  A message for the last
 *     failure of a context is available from tss_last_error().
 *   - Layers are numbered from 0.  A skip mask is n_layers bytes, 1 = skip the
 *     block, 0 = run it; a NULL mask means the sequence's mask (verify) and a
 *     mask of all zeros is the dense verifier.
 *   - The library never allocates device memory.  Packed weights, the
 *     workspace and the KV pool are device buffers owned by the caller, who
 *     keeps them alive for the context's lifetime.  Host arrays passed in are
 *     only read during the call.
 *   - All device work is enqueued on the HIP stream given to tss_create.
 *     tss_verify and tss_prefill return after that work has finished.
 *   - Validation finishes before any device work is enqueued and sequence
 *     state changes only when a call succeeds.  A HIP error poisons the
 *     context: every later call that touches the device returns TSS_ESTATE.
 *   - A context is not thread-safe.
 */
#ifndef TSS_H
#define TSS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tss_ctx tss_ctx;

enum tss_status {
  TSS_OK = 0,
  TSS_EINVAL = -1,     /* bad argument: shape, pointer, token, tree, mask */
  TSS_ENOSPACE = -2,   /* a caller buffer is smaller than the size query says */
  TSS_ECAPACITY = -3,  /* the sequence's KV capacity would be exceeded */
  TSS_ESTATE = -4,     /* wrong call order, stale KV for an active layer, or a poisoned context */
  TSS_EHIP = -5        /* the HIP runtime reported an error (the context is poisoned) */
};

enum tss_dtype { TSS_F32 = 0, TSS_BF16 = 1 };

/* tss_verify flags */
enum tss_flags {
  TSS_COMMIT = 1u      /* keep the K/V of the root and the accepted path; n_kv += accept_len + 1 */
};

/* How tss_verify issues its kernels (tss_set_launch_mode). */
enum tss_launch_mode {
  TSS_LAUNCH_DIRECT = 0, /* one launch per kernel */
  TSS_LAUNCH_GRAPH = 1   /* default: the step's launches are captured once per step shape
                            (sequences, skip masks, node counts, tree-path compaction;
                            not context lengths) into a HIP graph and replayed; results
                            are bit-identical to direct launches */
};

/* Kernel kinds for tss_profile_kernel. */
enum tss_kernel {
  TSS_K_EMBED = 0,
  TSS_K_QKV = 1,       /* RMSNorm + Q/K/V projection + rotary + KV append */
  TSS_K_ATTN = 2,      /* tree-masked attention over the paged KV cache */
  TSS_K_OPROJ = 3,     /* output projection + residual */
  TSS_K_GATEUP = 4,    /* RMSNorm + gate/up projection + SwiGLU */
  TSS_K_DOWN = 5,      /* down projection + residual */
  TSS_K_LMHEAD = 6,    /* final RMSNorm + lm_head + per-tile argmax */
  TSS_K_ACCEPT = 7,    /* argmax reduction + accept scan */
  TSS_K_COMPACT = 8    /* moves the accepted tree path's K/V next to the context */
};

/* Model shape.  Constraints (checked by tss_cfg_check):
 *   d_model == n_heads * head_dim; head_dim in {64, 128};
 *   d_model and ffn_dim multiples of 32; vocab a multiple of 32;
 *   1 <= max_nodes <= 64 (nodes of one sequence in one verify, root included);
 *   1 <= max_batch <= 8 (sequences of one tss_verify_batch);
 *   d_model <= 8192 (<= 4096 for TSS_F32);
 * One step carries at most min(max_nodes * max_batch, 128) rows (64 for
 * TSS_F32): the nodes of all its sequences.
 *   dtype TSS_BF16 (bf16 weights, held as fp16: exact for magnitudes
 *   2^-17 .. 65504, smaller ones within 2^-25, larger ones refused by
 *   tss_load_weights with TSS_EINVAL; fp16 KV cache, attention operands and
 *   projection inputs, i.e. fp16 MFMAs as in the paper's fp16 runs; fp32
 *   accumulation, residual stream, softmax and logits) or TSS_F32
 *   (everything fp32).
 * The KV page size is fixed at 16 tokens. */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t head_dim;
  int32_t ffn_dim;
  int32_t vocab;
  float rope_base;     /* rotary base, 10000 for LLaMA */
  float rms_eps;       /* RMSNorm epsilon, 1e-6 */
  int32_t dtype;       /* enum tss_dtype */
  int32_t max_nodes;   /* most nodes of one sequence in a verify */
  int32_t max_batch;   /* most sequences of one tss_verify_batch (1 for single-sequence use) */
} tss_model_cfg;

/* Checks the constraints above.  Pure host function.  TSS_OK or TSS_EINVAL.
 * Paper: Appendix / Models (the LLaMA target shapes the step serves). */
int tss_cfg_check(const tss_model_cfg* cfg);

/* Size queries (bytes); 0 when cfg is invalid.  The caller allocates these
 * device buffers (the library allocates none).  Paper: Appendix / Models
 * (weights), Problem Formulation (the workspace of one parallel verification
 * pass), Experiments / Models (the KV cache the underlying method keeps). */
size_t tss_weights_bytes(const tss_model_cfg* cfg);
size_t tss_workspace_bytes(const tss_model_cfg* cfg);
size_t tss_kv_bytes(const tss_model_cfg* cfg, int32_t n_seqs, int32_t max_tokens_per_seq);

/* The conversion tss_load_weights applies to TSS_BF16 weights, on the host:
 * src[n] bf16 bit patterns to dst[n] fp16 bit patterns of the same value,
 * round to nearest even (exact for magnitudes 2^-14 .. 65280; below that the
 * nearest multiple of 2^-24; infinities and NaNs map across, NaNs quiet).
 * Returns the number of finite values of magnitude >= 65536, which become
 * infinities here and make tss_load_weights refuse the tensor; -1 for n < 0
 * or a NULL buffer with n > 0.  Host memory only; no GPU call.  Paper:
 * Appendix, Experimental Setup / Models and Hardware and Software (the
 * target's weights are held in float16). */
int64_t tss_bf16_to_f16(const uint16_t* src, uint16_t* dst, int64_t n);

/* Creates a context bound to hip_stream (a hipStream_t; NULL = the null
 * stream), a packed-weight buffer of tss_weights_bytes() and a workspace of
 * tss_workspace_bytes(), both device memory owned by the caller, who keeps
 * them alive until tss_destroy.  *out receives the context (NULL on failure).
 * TSS_EINVAL (bad cfg, NULL buffer), TSS_ENOSPACE (buffer too small),
 * TSS_EHIP.  Paper: Method / Domain-Aware Skip Controller (one loaded target
 * serves every domain; all parameters stay loaded). */
int tss_create(const tss_model_cfg* cfg, void* hip_stream, void* dev_weights, size_t weights_bytes,
               void* dev_workspace, size_t workspace_bytes, tss_ctx** out);

/* Loads host tensors first .. first+count-1 of the fixed tensor order into the
 * packed device buffer (may be called several times, e.g. one tensor at a time
 * to stream a large model).  Order, all row-major [out][in] in the cfg dtype
 * (fp32, or bf16 bit patterns as uint16):
 *   0: embed [vocab][d_model]
 *   1 + 9*l + {0..8} for layer l: attn_norm [d], wq [d][d], wk [d][d],
 *       wv [d][d], wo [d][d], mlp_norm [d], w_gate [ffn][d], w_up [ffn][d],
 *       w_down [d][ffn]
 *   1 + 9*n_layers: final_norm [d];   2 + 9*n_layers: lm_head [vocab][d]
 * Returns when the copies are complete. */
/* Paper: Appendix / Models (LLaMA blocks: attention and SwiGLU MLP
 * weights, RMSNorm gains, untied lm_head).  TSS_EINVAL for a range outside
 * the list or a NULL tensor; TSS_EHIP poisons the context. */
int tss_load_weights(tss_ctx* ctx, int32_t first, int32_t count, const void* const* host_tensors);

/* Binds a KV pool of tss_kv_bytes(cfg, n_seqs, max_tokens_per_seq) bytes of
 * device memory and resets every sequence to length 0 (masks to dense).
 * page_order, if not NULL, lists a permutation of the pool's
 * n_seqs * ceil(max_tokens/16) pages; sequence s owns the s-th run of pages
 * in that order (NULL = identity); TSS_EINVAL if it is not a permutation.
 * Rebinding (the same or another pool) is allowed at any time: steps
 * captured for the previous binding are discarded.  The caller owns the
 * pool.  Paper: Problem Formulation (the drafts are verified against the
 * committed prefix, whose keys and values the underlying method caches). */
int tss_kv_alloc(tss_ctx* ctx, int32_t n_seqs, int32_t max_tokens_per_seq, void* dev_pool, size_t pool_bytes,
                 const int32_t* page_order);

/* Sets the skip mask of a sequence (n_layers bytes of 0/1; NULL = dense).
 * The mask is the sequence's default for prefill and verify.  TSS_EINVAL for
 * an unknown sequence or a byte other than 0/1.  Paper: Method /
 * Domain-Aware Skip Controller (the skip set of the request's domain, fixed
 * for the whole request; the empty set for unsupported domains). */
int tss_set_skip_mask(tss_ctx* ctx, int32_t seq, const uint8_t* mask);

/* Appends n context tokens to sequence seq under its skip mask: their K/V are
 * computed and kept for every layer the mask runs.  The tokens go through the
 * decoder in chunks of min(64, rows of one step).  TSS_ECAPACITY past the
 * sequence's capacity, TSS_ESTATE if an active layer lacks K/V for the
 * committed context.  Paper: Method / Domain-Aware Skip Controller (the same
 * block rule in the target's forward for every token of the request). */
int tss_prefill(tss_ctx* ctx, int32_t seq, const int32_t* tokens, int32_t n);

/* One verification step.  Paper: Method / Problem Formulation (the target
 * verifies the drafted tokens in one parallel pass; T_S bypasses the blocks
 * of S), Method / Domain-Aware Skip Controller (the per-block membership
 * check: a skipped block passes its hidden state through, with no attention
 * or feed-forward work), Experiments / Models and speculative decoding
 * methods and Appendix / Evaluation Protocol (greedy acceptance, temperature
 * 0, the underlying method's accept rule unchanged).
 *   draft_tokens[n_nodes]: node 0 is the root (the last committed token,
 *     whose K/V are not cached yet); nodes 1.. are drafted tokens.
 *   tree_parent[n_nodes]: parent[0] = -1 and 0 <= parent[i] < i; NULL = chain.
 *   skip_mask: n_layers bytes or NULL for the sequence's mask.  Every layer the
 *     mask runs must hold K/V for the whole committed context (TSS_ESTATE
 *     otherwise).
 * Node i sits at position n_kv + depth(i) and attends to the cached context and
 * to itself and its ancestors.  Outputs: accept_len = depth of the deepest node
 * whose root path matches the greedy (argmax, lowest index on ties) tokens,
 * lowest node index among equal depths; next_token = the greedy token at that
 * node (the bonus token).  With TSS_COMMIT the root and accepted path are kept
 * for the layers that ran and n_kv grows by accept_len + 1. */
int tss_verify(tss_ctx* ctx, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent, int32_t n_nodes,
               const uint8_t* skip_mask, uint32_t flags, int32_t* accept_len, int32_t* next_token);

/* For callers that cannot allocate device memory (serving loops and
 * harnesses that forbid allocation, which cannot provide tss_create's
 * workspace for a second context, for example): tss_verify, with the same
 * arguments, results and errors, but with the step's workspace (activations,
 * attention partial states, merge counters, K-split partial products,
 * logits, argmax partials, per-step results) in a static device array of
 * TSS_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends, instead of the workspace given to tss_create.  It
 * calls no allocating routine: its launches are direct (never captured into
 * a graph) and results come back through the context's pinned buffer.
 *   TSS_ENOSPACE, with a message, when tss_static_workspace_bytes(cfg)
 *   exceeds TSS_STATIC_SCRATCH_BYTES (larger models use tss_verify).
 * Every call on a GPU shares that GPU's scratch, which keeps the last call's
 * contents: calls that overlap on one GPU (from several host threads, or on
 * streams that run at the same time) race, and the caller must serialise
 * them.  The merge counters are cleared at the start of every step.
 * tss_get_logits, tss_get_logits_device, tss_get_greedy and
 * tss_get_attn_split read the last step's workspace, so after a static call
 * they are valid only until the next call on that GPU reuses the scratch. */
#define TSS_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
size_t tss_static_workspace_bytes(const tss_model_cfg* cfg);
int tss_verify_static(tss_ctx* ctx, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent,
                      int32_t n_nodes, const uint8_t* skip_mask, uint32_t flags, int32_t* accept_len,
                      int32_t* next_token);

/* Paper: as tss_verify, for several requests, each with its own domain's
 * skip set (Domain-Aware Skip Controller).
 * Verifies several sequences in one step (the same forward as tss_verify, on
 * the rows of every sequence at once, so each active block's weights are read
 * once for the whole batch).
 *   seq_ids[n_seqs]: distinct sequences.
 *   node_offsets[n_seqs + 1]: node_offsets[0] = 0, increasing; sequence i's
 *     nodes are draft_tokens[node_offsets[i] .. node_offsets[i + 1]), its root
 *     first, numbered locally from 0.
 *   tree_parents: per node the local parent index (-1 for each root), laid
 *     out like draft_tokens; NULL = every sequence is a chain.
 *   skip_masks: n_seqs * n_layers bytes (sequence i's mask at i * n_layers),
 *     or NULL for each sequence's own mask.
 * A block skipped by every sequence is not launched; inside a launched block
 * the rows of a sequence that skips it are left untouched (no attention, no
 * KV, residual unchanged), so each sequence's result equals its own
 * tss_verify up to floating-point summation order.  accept_len[i] and
 * next_token[i] are sequence i's decision; TSS_COMMIT commits every
 * sequence.  The logits / greedy rows of tss_get_logits and tss_get_greedy
 * follow the batch's node order. */
int tss_verify_batch(tss_ctx* ctx, int32_t n_seqs, const int32_t* seq_ids, const int32_t* node_offsets,
                     const int32_t* draft_tokens, const int32_t* tree_parents, const uint8_t* skip_masks,
                     uint32_t flags, int32_t* accept_len, int32_t* next_token);

/* Verifies one draft tree of one sequence under n_masks skip masks, without
 * committing: the candidate evaluations of the offline skip-set search
 * (Acceptance- and Metric-Aware Breadth Search, Algorithm 1, which evaluates
 * the dense baseline, every single-layer skip and every subset of the
 * candidate pool at each search depth on the same calibration input).
 * Results equal n_masks calls of tss_verify(seq, draft, parent, n_nodes,
 * mask_k, 0, ...) up to floating-point summation order.
 *   skip_masks: n_masks * n_layers bytes, mask k at k * n_layers.  Every layer
 *     any mask runs must hold K/V for the committed context (TSS_ESTATE
 *     otherwise; prefill the sequence dense for a sweep).
 *   accept_len[n_masks], next_token[n_masks]: mask k's decision.
 *   greedy: n_masks * n_nodes greedy tokens (mask k's at k * n_nodes), or NULL.
 *   dev_prefix, prefix_bytes: NULL / 0, or a device buffer of at least
 *     tss_sweep_prefix_bytes(cfg, n_nodes) bytes (TSS_ENOSPACE otherwise)
 *     that the call may overwrite: with it the masks are ordered by their
 *     first skipped layer and, when that saves more blocks than it costs, one
 *     dense pass stores every node's residual before every layer; each step
 *     then starts at the earliest first-skipped layer of its masks from the
 *     stored residual (a mask runs every layer before its first skipped one
 *     exactly as the dense verifier does), and the dense pass answers the
 *     masks that skip nothing.
 * Masks are verified together as segments of one step (at most 32, at most
 * min(max_nodes * max_batch, 128) rows, and only as many as the sequence's
 * free KV slots hold: each segment writes its draft K/V to its own slots
 * after the context).  Such a step launches each block that any of its masks
 * runs once, reading its weights and each context page once for all of
 * them; without a prefix buffer consecutive masks share steps, so callers
 * should order masks that share skipped layers next to each other.  The
 * sequence's length and committed K/V are unchanged; tss_get_logits /
 * tss_get_greedy / tss_get_path then describe the last step's segments. */
int tss_verify_sweep(tss_ctx* ctx, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent,
                     int32_t n_nodes, int32_t n_masks, const uint8_t* skip_masks, int32_t* accept_len,
                     int32_t* next_token, int32_t* greedy, void* dev_prefix, size_t prefix_bytes);

/* Paper: Algorithm 1 (the evaluations of the search).
 * Bytes of the prefix buffer of tss_verify_sweep for trees of n_nodes nodes:
 * n_layers * n_nodes * d_model fp32 values (0 when cfg or n_nodes is
 * invalid). */
size_t tss_sweep_prefix_bytes(const tss_model_cfg* cfg, int32_t n_nodes);

/* Copies the last verify's fp32 logits [n_nodes][vocab] / greedy tokens
 * [n_nodes] to host memory (rows in the step's node order); returns when the
 * copy is done.  n_nodes must not exceed the last verify's node count (all
 * sequences of a batch; TSS_EINVAL otherwise).  Paper: Experiments / Models
 * and speculative decoding methods (the greedy tokens the accept rule
 * compares the drafts with). */
int tss_get_logits(tss_ctx* ctx, float* host_dst, int32_t n_nodes);
int tss_get_greedy(tss_ctx* ctx, int32_t* host_dst, int32_t n_nodes);

/* Enqueues on the context's stream a copy of the last verify's fp32 logits
 * [n_nodes][vocab] into dev_dst, device memory of at least n_nodes * vocab
 * floats owned by the caller, and returns without waiting (the copy is
 * ordered before any later work on that stream).  TSS_EINVAL as for
 * tss_get_logits.  Paper: as tss_get_logits. */
int tss_get_logits_device(tss_ctx* ctx, float* dev_dst, int32_t n_nodes);

/* Paper: Experiments / Models and speculative decoding methods (the accepted
 * draft path that the underlying method commits).
 * Accepted path of result i of the last verify (i = the sequence's index in
 * the batch, 0 for tss_verify; for tss_verify_sweep, the mask's index in the
 * last step): path_nodes[0 .. *path_len) = local node ids from the root to
 * the deepest accepted node, *path_len = accept_len + 1.  With TSS_COMMIT
 * these nodes' tokens (after the root) are the committed draft tokens.
 * path_nodes must hold max_nodes entries. */
int tss_get_path(tss_ctx* ctx, int32_t index, int32_t* path_nodes, int32_t* path_len);

/* Committed length of a sequence, and rewinding it (n_kv <= current length;
 * TSS_EINVAL otherwise).  Paper: Problem Formulation (the committed prefix). */
int tss_seq_length(tss_ctx* ctx, int32_t seq, int32_t* n_kv);
int tss_seq_truncate(tss_ctx* ctx, int32_t seq, int32_t n_kv);

/* Pure host checks, the same code the calls above run.  Paper: Problem
 * Formulation (draft trees: each node's parent precedes it; the skip set is
 * a subset of the blocks). */
int tss_validate_tree(const int32_t* parent, int32_t n_nodes, int32_t max_nodes);
int tss_validate_mask(const uint8_t* mask, int32_t n_layers);
/* depth[i] and anc[i] (bit j set iff node j is i or an ancestor of i). */
int tss_tree_meta(const int32_t* parent, int32_t n_nodes, int32_t* depth, uint64_t* anc);

/* Selects the launch mode of tss_verify (enum tss_launch_mode).  At most 32
 * captured step shapes are kept per context (least recently used dropped).
 * Runtime plumbing; no passage of the paper. */
int tss_set_launch_mode(tss_ctx* ctx, int32_t mode);

/* Times one kernel launch per verify: the launch of kind `kernel` (enum
 * tss_kernel) for layer `layer` (ignored for kinds outside the layer loop);
 * kernel = -1 switches timing off.  Two HIP events are bound to that launch's
 * own dispatch (hipExtLaunchKernel), so they hold the start and end of the
 * kernel's execution, the figure a kernel-trace profiler reports, with no
 * event-record overhead between them.  While timing is on, verify steps use
 * direct launches (a captured graph cannot carry the events).
 * tss_profile_read returns the summed milliseconds and the launch count
 * (reset != 0 clears them). */
int tss_profile_kernel(tss_ctx* ctx, int32_t kernel, int32_t layer);
int tss_profile_read(tss_ctx* ctx, double* total_ms, int64_t* count, int32_t reset);

/* How the last step (verify, sweep step or prefill chunk) divided the
 * attention of its last launched block: *n_items attention items (runs of at
 * most 64 consecutive rows of one KV sequence), and for item i the number of
 * workgroups per head its context pages were split among (groups[i]; 1 = no
 * cross-workgroup merge) and its rows (rows[i]).  groups and rows must hold
 * 16 entries.  *n_items = 0 when the step launched no block.  Waits for the
 * context's stream.  Inspection only (tests assert with it which attention
 * path a launch took); no passage of the paper. */
int tss_get_attn_split(tss_ctx* ctx, int32_t* n_items, int32_t* groups, int32_t* rows);

/* Consistency check of the KV binding, a debugging aid (it waits for the
 * context's stream and copies the page table back): the page table is a
 * permutation of the pool's pages (every entry inside the pool, none owned
 * twice), the device copy equals the host's, and every sequence's committed
 * length and per-layer K/V lengths stay within its capacity.  TSS_OK,
 * TSS_ESTATE naming the first inconsistency (tss_last_error), or TSS_EHIP.
 * No passage of the paper. */
int tss_check_kv(tss_ctx* ctx);

/* Message of the context's last failure; with ctx = NULL, of the calling
 * thread's last failed tss_create. */
const char* tss_last_error(const tss_ctx* ctx);
const char* tss_status_string(int status);
void tss_destroy(tss_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* TSS_H */
