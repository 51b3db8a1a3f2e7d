/*
 * msd.h -- C ABI of the MI355X (gfx950) multimodal speculative decoding
 * (MSD) decode path.
 *
 * One decode cycle of MSD (arXiv 2505.14260) at temperature 0:
 *   msd_draft_tree      the one-layer draft head builds a token tree from the
 *                       decoupled draft input (Sec. 4.1, Eq. decouple) with
 *                       tree-structured drafting (Sec. 3.2);
 *   msd_verify          the target runs one tree-masked forward over the tree
 *                       (Sec. 3.2, verification phase);
 *   msd_accept_compact  greedy longest-path acceptance plus the bonus token
 *                       (Sec. 3.2 acceptance rule with a one-hot target) and
 *                       in-place compaction of the target KV cache;
 *   msd_accept_sample   the same at temperature > 0 (speculative sampling).
 * msd_prefill processes the interleaved visual + text prompt (Sec. 3.1).
 *
 * Conventions
 *  - Every pointer named *_d is device memory owned by the caller.  The
 *    library allocates device memory of its own only for the draft-training
 *    state (msd_train_*); the rocBLAS handle of the prompt GEMMs works in
 *    workspace carved from the caller's buffer.  *_h pointers are host.
 *  - Weights are bfloat16 (raw 16-bit patterns), row-major [out][in], no
 *    biases.  Norm gains are bfloat16 [d].
 *  - All device work is enqueued on the stream given to msd_create, in order.
 *    Only msd_prefill and the two acceptance calls wait for the stream (to
 *    return host outputs).  A context serves one stream and is not thread-safe.
 *  - Return value: MSD_OK (0) or a negative MSD_ERR_*; msd_last_error()
 *    returns a message for the last failure on that context (or of
 *    msd_create when ctx is NULL).
 */
#ifndef MSD_H
#define MSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  MSD_OK = 0,
  MSD_ERR_INVALID_ARG = -1, /* null pointer, shape beyond limits, bad tree  */
  MSD_ERR_CAPACITY = -2,    /* the KV cache cannot hold the request          */
  MSD_ERR_STATE = -3,       /* call out of order (e.g. verify before prefill)*/
  MSD_ERR_HIP = -4          /* a HIP runtime call failed                     */
};

/* Llama-style decoder shape (the target; the draft layer uses the same). */
typedef struct msd_model_desc {
  int32_t n_layers;
  int32_t d_model;     /* multiple of 8, at most 8192 */
  int32_t n_heads;     /* query heads */
  int32_t n_kv_heads;  /* key/value heads (n_heads % n_kv_heads == 0) */
  int32_t head_dim;    /* must be 128 or 64 */
  int32_t ffn_dim;
  int32_t vocab;       /* 16 .. 262144 */
  float rope_theta;
  float norm_eps;
} msd_model_desc;
/* Every weight matrix (q, k and v stacked, o, gate, up, down, f_down, the LM
 * head) must stay under 2 GiB in the library's padded layout (64-row x
 * 128-column blocks of bf16). */

typedef struct msd_limits {
  int32_t max_batch;   /* sequences decoded together (<= 8) */
  int32_t max_seq;     /* KV slots per sequence: prompt + generated + tree */
  int32_t max_tree;    /* nodes per tree including the root (<= 64) */
  int32_t max_prompt;  /* rows of one prefill */
} msd_limits;

typedef struct msd_layer_weights {
  const void *wq, *wk, *wv, *wo;   /* [H*hd][d], [KV*hd][d] x2, [d][H*hd] */
  const void *w_gate, *w_up;       /* [F][d] */
  const void *w_down;              /* [d][F] */
  const void *attn_norm, *ffn_norm;/* [d] */
} msd_layer_weights;

typedef struct msd_target_weights {
  const void* embed;                 /* [V][d] token embedding E_t */
  const msd_layer_weights* layers;   /* host array of n_layers entries */
  const void* final_norm;            /* [d] */
  const void* lm_head;               /* [V][d] projection head */
} msd_target_weights;

/* One-layer draft head: f_down [d][2d] acting on Concat(h, e) (h first),
 * one decoder layer, then the target's LM head. */
typedef struct msd_draft_weights {
  const void* fc;
  msd_layer_weights layer;
} msd_draft_weights;

/*
 * Caller-owned device buffers (sizes from msd_buffer_sizes).
 *  target_k: per layer, per sequence, per kv head: [max_seq][head_dim] bf16
 *            i.e. index ((layer*B + b)*KV + g)*max_seq*hd + slot*hd + e
 *  target_v: same blocks, transposed: [head_dim][max_seq] bf16
 *            i.e. index ((layer*B + b)*KV + g)*hd*max_seq + e*max_seq + slot
 *  draft_k / draft_v: the same layouts with one layer.
 *  workspace: scratch, contents undefined between calls except the library's
 *            own per-sequence state that it keeps there.
 *  packed_weights: msd_create writes a copy of every matrix the decode path
 *            multiplies by (target q, k, v, o, gate, up, down per layer, the
 *            draft layer's, f_down and the LM head) in the streaming layout
 *            of the library's GEMM (64-row x 128-column blocks, zero-padded).
 */
typedef struct msd_buffers {
  void *target_k, *target_v, *draft_k, *draft_v, *workspace, *packed_weights;
} msd_buffers;

/* Draft-tree shape for one decode cycle.
 *  STATIC: n_nodes drafted nodes (root excluded) given in canonical order
 *          (depth ascending); node i (1-based) has parent parent[i-1]
 *          (0 = root) and is the rank[i-1]-th best token of its parent's
 *          draft distribution.  Siblings have distinct ranks.
 *  DYNAMIC: depth levels, topk children per expanded node, topk frontier
 *          nodes per depth ranked by cumulative draft log-probability,
 *          n_nodes best candidates of the pool kept (Sec. 3.2 tree drafting,
 *          breadth-wise expansion).  Ties: score descending, then creation
 *          order.  Requires topk*(depth-1) <= 64 and n_nodes + 1 <= max_tree. */
enum { MSD_TREE_STATIC = 0, MSD_TREE_DYNAMIC = 1 };
typedef struct msd_tree_spec {
  int32_t kind;
  int32_t n_nodes;
  int32_t depth;
  int32_t topk;            /* DYNAMIC only */
  const int32_t* parent;   /* STATIC only, host, [n_nodes] */
  const int32_t* rank;     /* STATIC only, host, [n_nodes] */
} msd_tree_spec;

/* Device-resident token tree of one sequence.  Node 0 is the root (the last
 * emitted token, not yet in the cache); nodes are in canonical order so
 * parent[i] < i.  anc[i] has bit j set iff node j is node i or an ancestor. */
#define MSD_MAX_TREE 64
typedef struct msd_tree {
  int32_t n_nodes;                 /* including the root */
  int32_t token[MSD_MAX_TREE];
  int32_t parent[MSD_MAX_TREE];    /* -1 for the root */
  int32_t depth[MSD_MAX_TREE];
  float score[MSD_MAX_TREE];       /* cumulative draft log-prob (DYNAMIC) */
  uint64_t anc[MSD_MAX_TREE];
} msd_tree;

typedef struct msd_ctx msd_ctx;

/* Byte sizes of the caller-owned buffers for this shape and these limits
 * (any output pointer may be NULL).  Errors: MSD_ERR_INVALID_ARG for a shape
 * or limit outside the documented ranges. */
int msd_buffer_sizes(const msd_model_desc* m, const msd_limits* lim,
                     size_t* target_kv_bytes /* each of K and V */,
                     size_t* draft_kv_bytes /* each of K and V */,
                     size_t* workspace_bytes, size_t* weight_bytes /* packed_weights */);

/* The workspace size alone (the workspace_bytes of msd_buffer_sizes). */
int msd_workspace_size(const msd_model_desc* m, const msd_limits* lim, size_t* bytes);

/* Creates a context over caller-owned weights and buffers.  stream: a
 * hipStream_t (NULL = the null stream).  Packs the matrices into
 * bufs->packed_weights, initialises the workspace and zeroes the four KV
 * caches (enqueued on the stream, waited for before returning).  After it
 * returns, the library reads the embedding table, the norm gains and the
 * packed copies only: the row-major matrices may be released; every other
 * pointer must stay valid until msd_destroy.
 * When the limits allow passes over more than 256 rows (a prompt of
 * max_prompt rows, or max_batch trees of max_tree nodes), the GEMMs of such
 * passes run on rocBLAS (bf16 inputs, float32 results) in launches of up to
 * 1024 rows (a last launch of 64 rows or fewer takes the library's own
 * kernels), against a row-major copy of one weight at a time that the
 * library unpacks into the workspace: msd_create then also creates a rocBLAS
 * handle on the stream, gives it a 32 MB workspace carved from
 * bufs->workspace, and runs the prompt GEMM shapes once so that rocBLAS
 * loads their kernels here rather than in the first msd_prefill.
 * MSD_ERR_HIP if the handle cannot be set up. */
int msd_create(const msd_model_desc* m, const msd_limits* lim,
               const msd_target_weights* tw, const msd_draft_weights* dw,
               const msd_buffers* bufs, void* stream, msd_ctx** out);
/* Waits for the context's stream and frees the host-side context (NULL: no
 * effect).  The caller's device buffers are untouched.  Returns MSD_ERR_HIP
 * if that wait or the release of the pinned staging buffer failed (the
 * context is freed either way; msd_last_error(NULL) has the message). */
int msd_destroy(msd_ctx* ctx);
const char* msd_last_error(const msd_ctx* ctx);

/*
 * Prompt processing for sequence `seq` (Sec. 3.1): n rows, row i is the text
 * token tokens_h[i] (embedded with E_t) when is_visual_h[i] == 0, otherwise
 * the next unused row of visual_d ([n_visual][d] bf16, in prompt order).
 * The prompt must end in a text token (the draft's text rows need the next
 * token's embedding).  Runs the target over the prompt (causal), fills the
 * target KV slots [0, n), stores the features of every row as pending draft
 * inputs and returns the first generated token (greedy) in *first_token_h.
 * Waits for the stream.  Resets the sequence.
 */
int msd_prefill(msd_ctx* ctx, int seq, int n, const int32_t* tokens_h,
                const uint8_t* is_visual_h, const void* visual_d,
                int32_t* first_token_h);

/*
 * Draft input of the visual prompt rows (the input-decoupling ablation,
 * Sec. 5.3, Table decouple_input).  MSD_DRAFT_VISUAL_EMBEDDING (the default,
 * the method's Eq. decouple): a visual row enters the draft as its own
 * embedding e_v.  MSD_DRAFT_VISUAL_FEATURE: it enters as the target's feature
 * h_v of that row (the final-norm output the text rows concatenate), again
 * without f_down.  Text rows are f_down(Concat(h_i, e_{i+1})) either way.
 * Applies to the msd_prefill calls that follow on this context (only prompt
 * rows are visual).  MSD_ERR_INVALID_ARG for another value.
 */
enum { MSD_DRAFT_VISUAL_EMBEDDING = 0, MSD_DRAFT_VISUAL_FEATURE = 1 };
int msd_set_draft_input(msd_ctx* ctx, int visual_input);

/*
 * Where msd_prefill's many-row products find the target's weights (the
 * prompt forward of Sec. 3.1; msd_train_accumulate's target forward takes
 * the same path).  enable != 0: the rocBLAS products (see msd_create)
 * read the row-major matrices given to msd_create (wo, w_gate, w_up and
 * w_down of every target layer) in place, instead of first unpacking each
 * packed copy into a workspace slot (a 640-row
 * LLaVA-1.5-7B-shaped prefill: 29.3 -> 25.1 ms).  Those matrices must then
 * stay valid and unchanged until msd_destroy or a call with enable = 0.
 * The q|k|v product keeps its unpacked, stacked copy (one product over all
 * three fills the GPU better than three), and so do the draft layer and
 * f_down (draft training rewrites their packed copies).  Results equal the
 * default path's bit for bit: the same rocBLAS products of the same
 * shapes on the same values.  Takes effect at the next prompt; enqueues no
 * device work.  Default: disabled.  Errors: MSD_ERR_INVALID_ARG for a NULL
 * ctx.
 */
int msd_use_caller_weights(msd_ctx* ctx, int enable);

/*
 * Draft phase for sequences seqs_h[0..n_seq): runs the pending rows through
 * the draft head (text: f_down(Concat(h_i, e_{i+1})); visual: e_i, or h_i
 * after msd_set_draft_input(MSD_DRAFT_VISUAL_FEATURE)), then
 * builds the tree of `spec` depth by depth.  Writes one msd_tree per
 * sequence to trees_d[0..n_seq).  All sequences use the same spec.
 */
int msd_draft_tree(msd_ctx* ctx, int n_seq, const int32_t* seqs_h,
                   const msd_tree_spec* spec, msd_tree* trees_d);

/*
 * Verification (Sec. 3.2, verification phase): the target runs over the
 * n_nodes tree tokens of each sequence (node i at position L + depth[i],
 * cache slot L + i) with the ancestor mask, L being the sequence's committed
 * length.  Writes the greedy token of every node to argmax_d
 * [n_seq][n_nodes] (lowest id on ties) and, when logits_d is not NULL, the
 * logits to logits_d [n_seq][n_nodes][V] float32.  The tree rows' KV stay in
 * slots [L, L+n_nodes) until msd_accept_compact.
 * Trees are read on the device, so their check travels with the stream: a
 * tree whose n_nodes differs, whose parent does not precede its child, whose
 * depth or ancestor mask disagrees with its parents, whose token id is out of
 * range or which repeats a token among siblings is computed with clamped ids
 * (no access leaves its buffers), and the acceptance call that follows
 * returns MSD_ERR_INVALID_ARG and accepts nothing for any sequence of it.
 * Errors here: MSD_ERR_INVALID_ARG (null pointer, n_nodes outside
 * [1, max_tree], bad sequence list), MSD_ERR_STATE (sequence without a
 * prompt), MSD_ERR_CAPACITY (L + n_nodes > max_seq).
 */
int msd_verify(msd_ctx* ctx, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
               int n_nodes, int32_t* argmax_d, float* logits_d);

/*
 * msd_verify for callers that cannot allocate device memory or must not make
 * the library use its workspace for per-call scratch (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments, results and errors as msd_verify, and the same kernels; the
 * call's scratch (GEMM split-K partials, attention partials, top-k scratch)
 * lives in a static device array of MSD_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends.  Nothing is
 * allocated.  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (other contexts or streams) race and must be ordered by
 * the caller.  MSD_ERR_INVALID_ARG when n_seq * n_nodes > 256 or when the
 * call's scratch exceeds MSD_NOALLOC_SCRATCH_BYTES (the message gives the
 * size needed).
 */
#define MSD_NOALLOC_SCRATCH_BYTES (64u << 20)
int msd_verify_noalloc(msd_ctx* ctx, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
                       int n_nodes, int32_t* argmax_d, float* logits_d);

/*
 * Acceptance and compaction: for each sequence, the deepest node whose every
 * token on the root path equals its parent's argmax is accepted; emitted
 * tokens are the accepted drafted tokens followed by the bonus token (the
 * argmax of the deepest accepted node).  KV rows L+path[j] move to L+j for
 * every layer (all reads before any write); slot_map_d [n_seq][MSD_MAX_TREE]
 * receives L+path[j] (-1 past the path).  The accepted nodes' target
 * features become the next pending draft rows and L grows by len(path).
 * emitted_h [n_seq][MSD_MAX_TREE] and n_emitted_h [n_seq] are host outputs;
 * waits for the stream.
 * Errors: MSD_ERR_STATE unless the call follows msd_verify of the same
 * sequence list (same order) and n_nodes, with no msd_prefill,
 * msd_draft_tree, msd_set_state or other acceptance in between;
 * MSD_ERR_INVALID_ARG for a malformed tree found by that verify (then
 * nothing is accepted: caches, lengths and pending rows are unchanged and
 * n_emitted_h is all zero).
 */
int msd_accept_compact(msd_ctx* ctx, int n_seq, const int32_t* seqs_h,
                       const msd_tree* trees_d, int n_nodes, const int32_t* argmax_d,
                       int32_t* emitted_h, int32_t* n_emitted_h, int32_t* slot_map_d);

/*
 * Acceptance by speculative sampling at temperature > 0 (Sec. 3.2,
 * verification phase: acceptance probability min(1, p/q) and the adjusted
 * distribution norm(max(0, p - q)) after a rejection; the extra draw from p
 * when every drafted token is accepted).  The tree's children are the
 * draft's top-ranked tokens, so each child's proposal q is the point mass on
 * its token: walking down from the root, the children of the current node
 * are tried in node order, a child with token x being accepted with
 * probability p(x) / (1 - target mass of the children already rejected
 * there), where p = softmax(logits / temperature) at the current node; a
 * rejection removes x from p.  When no child is accepted, the bonus token is
 * drawn from p without the rejected tokens.  The emitted tokens follow the
 * target's own sampling distribution.
 *
 * logits_d [n_seq][n_nodes][V] float32: the logits msd_verify wrote for these
 * trees (its logits_d output).  temperature: positive and finite.  Draw j of
 * sequence slot b in the cycle starting at committed length L (L < 2^24) is
 * output n = b*2^40 + L*2^8 + j of the SplitMix64 generator (Steele, Lea and
 * Flood, 2014) started at `seed`, its top 24 bits scaled by 2^-24.
 * Everything else (outputs, compaction, pending rows, the wait) is as for
 * msd_accept_compact, which remains the temperature-0 rule.
 */
int msd_accept_sample(msd_ctx* ctx, int n_seq, const int32_t* seqs_h,
                      const msd_tree* trees_d, int n_nodes, const float* logits_d,
                      float temperature, uint64_t seed, int32_t* emitted_h,
                      int32_t* n_emitted_h, int32_t* slot_map_d);

/* Committed KV length of a sequence (host-side bookkeeping), or < 0. */
int msd_seq_len(const msd_ctx* ctx, int seq);

/*
 * Sets a sequence's committed length without running the prompt, for callers
 * that filled the target KV cache slots [0, L) themselves (cache import).
 * The pending draft rows become the single text row (h_d [d] bf16, the
 * target feature of position L-1; next_token = the token at position L, which
 * is also the next tree root).  The draft cache is not touched: the caller
 * fills draft slots [0, L-1) as well, or accepts whatever they hold.
 */
int msd_set_state(msd_ctx* ctx, int seq, int L, const void* h_d, int32_t next_token);

/*
 * Optional timing trace of the weight-streaming GEMM launches and the
 * tree-attention passes (for measurement tools).  msd_trace_enable(ctx,
 * capacity, kinds) starts timing the next `capacity` launches whose kind has
 * its bit set in `kinds`, with events carried by the launches themselves
 * (capacity <= 0 stops and clears); msd_trace_read waits for the stream and
 * returns up to max_recs records (return value: count, or < 0 on error).
 * kind: 0 = q/k/v projection, 1 = output projection, 2 = down projection,
 * 3 = gate+up (SwiGLU) pair, 4 = draft f_down, 5 = LM head (for these m is
 * the number of input rows and the weight is n x k bf16, twice that for
 * kind 3); 6 = a tree-attention pass with its chunk combine (m = query rows,
 * n = key slots of the longest sequence including the tree, k = key chunks).
 */
/*
 * Draft-head training (Sec. 4.2: the one-layer draft learns from the frozen
 * target; the data schedule is Eq. progressive_data).  The paper leaves the
 * loss and optimiser to the feature-level draft it builds on; this library
 * reads them as follows.  On a training sequence of n positions (tokens,
 * visual flags and visual rows as for msd_prefill) the target's features
 * h_0..h_{n-1} (final-norm outputs) are computed; the draft's input rows
 * i = 0..n-2 follow the decoupled rule (Eq. decouple: text rows
 * f_down(Concat(h_i, e_{i+1})), visual rows e_i, or h_i after
 * msd_set_draft_input(..., MSD_DRAFT_VISUAL_FEATURE)) and the draft layer runs
 * causally over them at positions i; its output d_i is trained toward
 * h_{i+1}:
 *   loss_i = mean_k SmoothL1(d_i - h_{i+1})_k
 *            + 0.1 CE(softmax(W_lm h_{i+1}), softmax(W_lm d_i)),
 * with SmoothL1's beta = 1 and the cross-entropy against the target's full
 * next-token distribution.  A batch's loss is the mean of loss_i over all
 * rows of its sequences.  Trained: f_down, the draft layer's seven matrices
 * and two norm gains (float32 master copies); the embedding table and the
 * LM head stay frozen.  Arithmetic in float32 (the contractions on rocBLAS).
 *
 * msd_train_accumulate adds one sequence's gradient sums and writes its
 * loss sums to loss_h[3] (total, regression part, token part, each summed
 * over its n - 1 rows).  It runs the target over the sequence in slot `seq`
 * (2 <= n <= max_prompt): the slot's cache is overwritten and the slot must
 * be prefilled again before decoding.  The first training call allocates
 * the training state (device memory of its own, freed by msd_destroy).
 * msd_train_apply performs one AdamW step (beta1 0.9, beta2 0.999, eps 1e-8,
 * no weight decay) with the mean gradient over the accumulated rows and
 * learning rate lr, refreshes the draft the decoder uses (its packed
 * weights, and from the first training call on the draft's norm gains are
 * read from the library's copy), and clears the sums; MSD_ERR_INVALID_ARG
 * when nothing was accumulated.  msd_train_read copies the float32 gradient
 * sums (what = 0) or master parameters (what = 1), concatenated row-major in
 * the order f_down [d][2d], wq [H hd][d], wk [KV hd][d], wv [KV hd][d],
 * wo [d][H hd], w_gate [F][d], w_up [F][d], w_down [d][F], attn_norm [d],
 * ffn_norm [d], to the device buffer out_d of exactly that many floats.
 * msd_train_lr gives the cosine schedule lr_max (1 + cos(pi step / total)) / 2
 * (0 <= step <= total); msd_train_mix gives the text-only and visual sample
 * counts of epoch t of T in stage 2 (Eq. progressive_data: a visual share of
 * t / T of n_per_epoch, rounded to the nearest integer, ties to even).
 * Errors: MSD_ERR_INVALID_ARG (arguments), MSD_ERR_HIP (device or rocBLAS).
 */
int msd_train_accumulate(msd_ctx* ctx, int seq, int n, const int32_t* tokens_h,
                         const uint8_t* is_visual_h, const void* visual_d, double* loss_h);
int msd_train_apply(msd_ctx* ctx, double lr);
int msd_train_read(msd_ctx* ctx, int what, float* out_d, size_t n_floats);
int msd_train_lr(int step, int total_steps, double lr_max, double* lr_out);
int msd_train_mix(int epoch, int n_epochs, int n_per_epoch, int* n_text_out, int* n_visual_out);

/*
 * Diagnostic for measurement tools: one kernel that reads `bytes` of the
 * device buffer buf_d (16-byte aligned, zero-filled, bytes a multiple of
 * 64 KiB) with the access pattern of the library's weight stream (every wave
 * load 1 KB contiguous, nontemporal), spread over `workgroups` workgroups; it
 * computes nothing the decode uses.  sink_d: `workgroups` 32-bit words the
 * kernel may write.  Enqueued on `stream` (a hipStream_t); no context needed.
 * This is the achievable streaming rate the GEMMs are compared against.
 */
int msd_stream_read(const void* buf_d, size_t bytes, int workgroups, void* sink_d,
                    void* stream);

typedef struct msd_trace_rec {
  int32_t kind, m, n, k;
  float ms;
} msd_trace_rec;
int msd_trace_enable(msd_ctx* ctx, int capacity, int kinds);
int msd_trace_read(msd_ctx* ctx, int max_recs, msd_trace_rec* out);

#ifdef __cplusplus
}
#endif
#endif /* MSD_H */
