/*
 * seed.h -- C ABI of the SEED draft-verify decoding library for AMD Instinct MI355X (gfx950).
 *
 * SEED (Self-Speculative Encoder-Decoder) views a decoder-only transformer with l layers as an
 * encoder f_enc = f_{1:l'} followed by a thin decoder f_dec = f_{l'+1:l} (Sec. 3.1, Eq. 3-4).
 * Decoding alternates two passes (Algorithm 2, fixed draft length d):
 *   - draft : the decoder alone runs d autoregressive steps. Step i feeds the raw embedding
 *             W_in X_draft[i-1] (Eq. 5) and attends to the decoder layers' cache, i.e. the deep
 *             keys/values left by the last verification plus the drafts' own entries.
 *   - verify: the full model runs once over X_draft[0..d] (pending token + d drafts), writing
 *             deep keys/values in every layer; the longest prefix of drafts that equals the
 *             verifier's greedy argmax is accepted, plus one bonus token.
 * The output equals plain greedy decoding of the same model (d = 0 is plain greedy decoding).
 *
 * Conventions for every call:
 *   - Every function returns a seed_status; nothing throws, aborts or exits. On failure
 *     seed_last_error() describes the cause and the decoding state is left unchanged.
 *   - Token ids are int32 in [0, vocab). Logits are float32.
 *   - "host" pointers are ordinary CPU memory, read or written synchronously before the call
 *     returns. "device" pointers are GPU memory; device outputs are written in stream order on
 *     the context's HIP stream (synchronise that stream before reading them).
 *   - The library never allocates device memory after seed_create: the caller supplies the
 *     weight arena, the KV pool and the workspace (sizes from seed_arena_bytes), each at least
 *     256-byte aligned, and keeps them alive until seed_destroy.
 *   - Positions are 0-based. After a commit, sequence b holds t_b committed tokens; the last
 *     one (the pending token, position t_b - 1) has no cache entry yet.
 *   - A context is not thread-safe; use one context per stream.
 */
#ifndef SEED_H
#define SEED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* the library is built with hidden host symbols: only the functions declared here are exported */
#if defined(__GNUC__)
#pragma GCC visibility push(default)
#endif

typedef struct seed_ctx seed_ctx;

typedef enum seed_status {
  SEED_OK = 0,
  SEED_ERR_ARG = -1,         /* NULL pointer, bad size, shape, dtype or tensor name, k out of range */
  SEED_ERR_STATE = -2,       /* call out of order: draft/verify before prefill, weights missing */
  SEED_ERR_CAPACITY = -3,    /* a sequence would pass max_ctx, or batch > max_batch */
  SEED_ERR_HIP = -4,         /* a HIP runtime call failed; the message names it */
  SEED_ERR_UNSUPPORTED = -5  /* a shape the kernels do not handle (see seed_config) */
} seed_status;

typedef enum seed_dtype {
  SEED_F32 = 0,   /* fp32 weights and KV cache */
  SEED_BF16 = 1   /* bf16 weights and KV cache; all arithmetic and the residual stream stay fp32 */
} seed_dtype;

/*
 * Model shape and capacities (Preliminaries; Appendix E gives the model sizes).
 * Supported: hidden, ffn, n_heads*head_dim, n_kv_heads*head_dim multiples of 32; vocab a
 * multiple of 16; head_dim in {64, 128}; n_heads a multiple of n_kv_heads with
 * (n_heads/n_kv_heads) <= 32; 0 <= n_dec_layers <= n_layers; kv_block == 16;
 * 1 <= max_batch <= 64; 0 <= max_draft <= 15; 2 <= max_ctx <= 2^20.
 */
typedef struct seed_config {
  int32_t n_layers;       /* l */
  int32_t n_dec_layers;   /* l - l': the last n_dec_layers layers form the drafter (paper: 2) */
  int32_t hidden;
  int32_t n_heads;        /* query heads */
  int32_t n_kv_heads;     /* key/value heads (grouped-query attention) */
  int32_t head_dim;
  int32_t ffn;            /* SwiGLU inner width */
  int32_t vocab;          /* the embedding is tied to the LM head */
  float rope_base;        /* rotary base; rotate-half pairing (i, i + head_dim/2) */
  float rms_eps;          /* RMSNorm epsilon */
  int32_t dtype;          /* seed_dtype of the weights and the KV cache */
  int32_t max_batch;      /* sequences decoded together */
  int32_t max_ctx;        /* positions per sequence: prompt + generated + max_draft + 1 */
  int32_t max_draft;      /* largest draft length d accepted by draft/verify/generate */
  int32_t kv_block;       /* positions per paged KV block; must be 16 */
} seed_config;

/*
 * One named weight tensor. Names and shapes ([out, in] row-major, as nn.Linear):
 *   "embed"                    [vocab, hidden]    (also the LM head: W_out = W_in)
 *   "final_norm"               [hidden]
 *   "layers.<i>.attn_norm"     [hidden]
 *   "layers.<i>.wq"            [n_heads*head_dim, hidden]
 *   "layers.<i>.wk", ".wv"     [n_kv_heads*head_dim, hidden]
 *   "layers.<i>.wo"            [hidden, n_heads*head_dim]
 *   "layers.<i>.mlp_norm"      [hidden]
 *   "layers.<i>.w_gate", ".w_up" [ffn, hidden]
 *   "layers.<i>.w_down"        [hidden, ffn]
 * dtype must equal the config's dtype (bf16 data is raw bf16 bit patterns).
 */
typedef struct seed_tensor {
  const char* name;
  const void* data;     /* host or device pointer, see on_device */
  int32_t dtype;        /* seed_dtype */
  int32_t on_device;    /* 1: data is device memory; 0: host memory */
  int32_t ndim;         /* 1 or 2 */
  int64_t shape[2];
} seed_tensor;

/* Options of seed_generate. */
typedef struct seed_gen_opts {
  int32_t k;             /* draft length d (0 = plain greedy decoding), 0 <= k <= max_draft */
  int32_t max_new;       /* tokens to generate per sequence (the last round may overshoot; the
                            output is cut to max_new, Algorithm 2 returns X_{1:T}) */
  int32_t eos_id;        /* -1: off. Otherwise a sequence stops right after emitting it */
  int32_t sim_accept;    /* -1: real drafts. 0..k: benchmark mode that replaces the drafts after
                            the draft pass with forced_trace so that exactly sim_accept drafts
                            are accepted per round (the draft pass still runs in full) */
  const int32_t* forced_trace; /* host [B * max_new]: the plain greedy continuation of each
                            prompt; required iff sim_accept >= 0 */
  int32_t use_graph;     /* 1: capture one round into a HIP graph and replay it */
} seed_gen_opts;

/* Statistics filled by seed_generate (nullable). */
typedef struct seed_stats {
  int64_t rounds;            /* draft-verify rounds run */
  int64_t drafted;           /* sum over rounds and live sequences of k */
  int64_t accepted;          /* sum over rounds and live sequences of n_accept */
  double prefill_ms;         /* prefill time (HIP events) */
  double decode_ms;          /* first round start to last round end (HIP events) */
  int32_t* n_accept_log;     /* nullable host [n_accept_log_cap * B]: n_accept per round per
                                sequence, -1 once a sequence has finished */
  int64_t n_accept_log_cap;  /* rows available in n_accept_log */
  /* Step latencies, medians over the rounds of the call, from the device's constant-rate clock
   * stamped by the kernels that open and close each phase inside the (graph-replayed) rounds:
   * verify_ms = one verification (row setup to acceptance and commit); draft_ms = one drafting
   * step of seed_generate (the k-step drafting phase / k; 0 when k = 0) or, for
   * seed_generate_tree, one round's whole drafting phase (its step count varies). */
  double verify_ms;
  double draft_ms;
} seed_stats;

/* Kernel ids for seed_kernel_timing: phase * 16 + op. SEED_OP_ATTN times the attention partial
 * kernel, SEED_OP_COMBINE the merge of its group partials (launched when the context capacity
 * spans more than one attention group of 64, 128 or 256 positions). */
enum {
  SEED_PHASE_VERIFY = 0, SEED_PHASE_DRAFT = 1, SEED_PHASE_PREFILL = 2, SEED_PHASE_SPEC = 3,
  SEED_OP_SETUP = 0, SEED_OP_QKV = 1, SEED_OP_ATTN = 2, SEED_OP_COMBINE = 3, SEED_OP_O = 4,
  SEED_OP_GATEUP = 5, SEED_OP_DOWN = 6, SEED_OP_HEAD = 7, SEED_OP_ACCEPT = 8,
  SEED_OP_HEAD_ARGMAX = 9, SEED_OP_TOPK = 10
};

/* Bytes the caller must provide for the weight arena, the KV pool and the workspace. */
seed_status seed_arena_bytes(const seed_config* cfg, size_t* weight_bytes, size_t* kv_bytes,
                             size_t* workspace_bytes);

/*
 * Create a context on the current HIP device. hip_stream is a hipStream_t (NULL = the null
 * stream) on which every kernel of this context runs. The three buffers are device memory of at
 * least the sizes from seed_arena_bytes; the context borrows them until seed_destroy. The KV
 * pool is cleared here.
 */
seed_status seed_create(const seed_config* cfg, void* hip_stream, void* weight_arena,
                        void* kv_pool, void* workspace, seed_ctx** out);

/*
 * Copy the model weights into the arena, re-laid out for the kernels (MFMA tiles, fused QKV and
 * gate/up). Tensors may be loaded over several calls, each name at most once per call; a later
 * load of the same name replaces it. The sources may be freed after the call returns. Unknown,
 * duplicated, mis-shaped or mis-typed tensors give SEED_ERR_ARG naming the tensor. Until every
 * tensor listed at seed_tensor has been loaded, prefill/draft/verify/generate return
 * SEED_ERR_STATE naming the first missing one.
 */
seed_status seed_load_weights(seed_ctx* ctx, const seed_tensor* tensors, int32_t n);

/*
 * Initialisation of Algorithm 2: run the full model over each prompt X_{1:t} and keep the cache
 * of positions 0..t-2 in every layer; X_t becomes the pending token (no token is emitted).
 * tokens: host, the B prompts packed back to back; lens: host [B], each >= 1 and
 * lens[b] + max_draft + 1 <= max_ctx. Resets all decoding state of the context.
 */
seed_status seed_prefill(seed_ctx* ctx, int32_t B, const int32_t* tokens, const int32_t* lens);

/*
 * Drafting phase of Algorithm 2: k steps of the decoder only, from the pending token. Writes
 * the decoder layers' cache at positions p..p+k-1 (p = t_b - 1) and leaves the committed state
 * unchanged, so repeated calls give the same drafts.
 * drafts: nullable host [B * k], draft tokens X_draft[1..k] per sequence.
 * logits: nullable device [B * k * vocab], q_1..q_k per sequence.
 * Errors: SEED_ERR_STATE before seed_prefill; SEED_ERR_ARG if k < 1 or k > max_draft;
 * SEED_ERR_CAPACITY if some t_b + k + 1 > max_ctx.
 */
seed_status seed_draft(seed_ctx* ctx, int32_t k, int32_t* drafts, float* logits);

/*
 * Verification phase of Algorithm 2 plus acceptance and commit: truncate to t_b - 1 cached
 * positions, run the full model over X_draft[0..k] (row r at position p + r attends to
 * positions 0..p+r), accept the longest prefix with argmax p_i == X_draft[i], append the
 * accepted drafts and the bonus token argmax p_{n_accept+1}, keep the deep cache of positions
 * < t_b + n_accept. k = 0 is one step of plain greedy decoding.
 * drafts: nullable host [B * k]; NULL uses the drafts of the preceding seed_draft with the same
 *         k (SEED_ERR_STATE if there was none since the last commit).
 * n_accept, bonus: nullable host [B].
 * logits: nullable device [B * (k+1) * vocab], p_1..p_{k+1} per sequence.
 * Argmax ties go to the lowest token id.
 */
seed_status seed_verify(seed_ctx* ctx, int32_t k, const int32_t* drafts, int32_t* n_accept,
                        int32_t* bonus, float* logits);

/*
 * Run n_rounds draft-verify rounds (Algorithm 2's loop body) on every sequence without host
 * synchronisation; returns once the work is queued on the stream. use_graph = 1 captures one
 * round into a HIP graph (once per batch size and k) and replays it. Errors as seed_draft, with
 * capacity checked for the worst case t_b + n_rounds*(k+1) + k + 1 <= max_ctx (the committed
 * lengths are re-read first when that bound does not fit).
 */
seed_status seed_rounds(seed_ctx* ctx, int32_t k, int32_t n_rounds, int32_t use_graph);

/*
 * Algorithm 2 end to end: prefill, then rounds until every sequence has max_new new tokens (or
 * emitted eos_id). out: host [B * max_new] (positions past counts[b] are -1); counts: host [B].
 */
seed_status seed_generate(seed_ctx* ctx, int32_t B, const int32_t* tokens, const int32_t* lens,
                          const seed_gen_opts* opts, int32_t* out, int32_t* counts,
                          seed_stats* stats);

/*
 * Tree-based verification (Method, Adaptive Drafting with Tree-Based Verification; appendix
 * "Tree-Based Verification", Fig. 3 right) of one packed draft tree of the context's single
 * sequence (B = 1), with acceptance and commit. Node 0 is the pending token X[p] (p = t - 1, the
 * root); nodes 1..D are the top-1 chain (parent of node i is i-1, depth i); every later node is a
 * leaf whose parent is the root or a chain node of depth < D, at depth parent + 1. One full-model
 * pass runs over the nodes: node i at rotary position p + depth(i) attends to the committed prefix
 * and to its ancestors (and itself). From the root, the path follows the child whose token equals
 * the verifier's argmax at the current node; the accepted tokens and the bonus token (the argmax
 * at the last node reached) are appended; the cache keeps the root's and the accepted nodes'
 * keys/values at positions p, p+1, ...
 * tokens, parents: host [n], 1 <= n <= 64. path: nullable host [D], the accepted nodes;
 * path_len, bonus: nullable host. logits: nullable device [n * vocab], one row per node.
 * Errors: SEED_ERR_STATE before seed_prefill; SEED_ERR_UNSUPPORTED if B != 1; SEED_ERR_ARG for a
 * malformed tree or token; SEED_ERR_CAPACITY if t + n + 1 > max_ctx.
 */
seed_status seed_verify_tree(seed_ctx* ctx, int32_t n, const int32_t* tokens, const int32_t* parents,
                             int32_t* path, int32_t* path_len, int32_t* bonus, float* logits);

/*
 * Options of confidence-aware dynamic drafting (Method, Adaptive Drafting with Tree-Based
 * Verification; appendix "Confidence-Aware Dynamic Drafting"). Each drafting step runs the
 * decoder-only step of Algorithm 2 on the current chain token; p0 is the softmax probability of
 * its top-1 token. The step's candidates are its k highest-logit tokens (equal logits: lower id
 * first), k = k[j] for the first level j with p0 > thr[j], else k_rest, cut to the node budget
 * max_nodes. The top-1 candidate extends the chain, the others become leaves. Drafting stops
 * after a step with p0 < tau, after max_depth steps, or when the tree holds max_nodes nodes.
 * p0 and the decisions are taken in fp32.
 */
typedef struct seed_tree_opts {
  float tau;             /* confidence threshold (the paper uses 0.7, or 0.5 for summarisation) */
  int32_t max_depth;     /* drafting steps per round, 1 <= max_depth <= max_draft */
  int32_t n_levels;      /* levels of the top-p table, 0..4 */
  float thr[4];          /* strictly decreasing thresholds */
  int32_t k[4];          /* fan-out of each level, 1..16 */
  int32_t k_rest;        /* fan-out below every threshold, 1..16 */
  int32_t max_nodes;     /* node budget of a tree (root included), max_depth + 1 .. 64 */
} seed_tree_opts;

/* The paper's table (p0 > 0.95: 1, > 0.8: 3, > 0.5: 5, else 10), tau = 0.7, 64 nodes. */
void seed_tree_defaults(seed_tree_opts* opts, int32_t max_depth);

/*
 * One round's dynamic drafting for the context's single sequence (B = 1, after seed_prefill or
 * seed_verify_tree), returning the packed tree that seed_verify_tree takes: node 0 the pending
 * token, nodes 1..D the top-1 chain, then every step's other candidates by step and rank.
 * tokens, parents: host [64]; n_nodes: host. p0: nullable host [max_depth], the top-1
 * probability of each step run. logits: nullable device [max_depth * vocab], row i-1 = step i's
 * drafter logits. Each step waits for the previous one on the host; seed_generate_tree runs the
 * same kernels without waiting.
 * Errors: SEED_ERR_STATE before seed_prefill; SEED_ERR_UNSUPPORTED if B != 1 or the vocabulary is
 * outside 16..262144; SEED_ERR_ARG for invalid options; SEED_ERR_CAPACITY if t + max_nodes + 1 >
 * max_ctx.
 */
seed_status seed_draft_tree(seed_ctx* ctx, const seed_tree_opts* opts, int32_t* tokens, int32_t* parents,
                            int32_t* n_nodes, float* p0, float* logits);

/*
 * Dynamic drafting with tree-based verification end to end for one prompt (the decoding mode of
 * the paper's main experiments): prefill, then rounds of seed_draft_tree + seed_verify_tree until
 * opts->max_new tokens (or opts->eos_id) are committed. Lossless: every committed token is the
 * verifier's greedy choice. opts: as for seed_generate, except that k is not used and
 * sim_accept (0..max_depth) replaces chain nodes 1..sim_accept of every drafted tree with the
 * forced trace and the next chain node with another token (a benchmark of acceptance lengths
 * that random weights do not reach); use_graph replays each drafting step and each tree size's
 * verification from captured HIP graphs. out: host [max_new] (-1 past count); count: host.
 * stats: nullable; drafted counts tree nodes other than the root, n_accept_log the accepted path
 * length per round. Errors as seed_generate and seed_draft_tree; the prompt needs
 * len + max_new + 2 (max_nodes + 1) <= max_ctx.
 */
seed_status seed_generate_tree(seed_ctx* ctx, const int32_t* tokens, int32_t len, const seed_tree_opts* topts,
                               const seed_gen_opts* opts, int32_t* out, int32_t* count, seed_stats* stats);

/*
 * Forward pass of the speculative drafting objective L_spec (Algorithm 1, Sec. 3.2, Fig. 2 right)
 * on one sequence X[0..n-1] with training block size `block`: the full model runs over the
 * sequence (as seed_prefill, which this call replaces: afterwards the decode state is that of
 * seed_prefill(ctx, 1, tokens, &n)), then the decoder layers run once, in parallel for every
 * block, over the raw embeddings H^0 of X[0..n-2]: the row of position q (block start
 * s = floor(q / block) * block) attends causally to the rows s..q of its own block and to the
 * deep decoder keys/values of positions < s, and predicts X[q+1]. Forward only.
 * shallow_kv: device, at least seed_spec_kv_bytes bytes, 256-byte aligned, caller-owned: the
 *             decoder layers' keys/values of this pass (scratch: the call clears it first, so
 *             its prior contents never matter).
 * logits: device [(n-1) * vocab], the drafter's logits of every row (required).
 * row_nll: nullable device [n-1]: -log softmax(logits[q])[X[q+1]].
 * loss: nullable host: L_spec = the sum of row_nll (accumulated in double on the host).
 * Errors: SEED_ERR_ARG if n < 2, block < 1, a token is out of range or a required pointer is
 * NULL; SEED_ERR_CAPACITY if n + 1 > max_ctx.
 */
seed_status seed_spec_kv_bytes(const seed_config* cfg, size_t* bytes);
seed_status seed_spec_forward(seed_ctx* ctx, int32_t n, const int32_t* tokens, int32_t block,
                              void* shallow_kv, float* logits, float* row_nll, double* loss);

/*
 * seed_spec_forward for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same pass, the same kernels and the
 * same results, with the pass's own keys/values in a fixed array inside the library instead of a
 * caller buffer. The array holds 16 MiB per GPU (one copy on each GPU the library runs on, kept
 * until the process ends; its address is taken once per device by seed_create); a sequence needs
 * 2 * n_kv_heads * head_dim * element-size bytes per position and decoder layer, positions
 * rounded up to a multiple of 16 (the 4B-scale model: 8 KiB per
 * position, n <= 2048). The call allocates nothing: no hipMalloc/hipFree, no events (kernel
 * timing is suspended for its duration). Every call on one GPU shares the array and the pass
 * clears what it uses first, so calls that overlap on one GPU (several contexts or streams) race:
 * the caller serialises them. Arguments, outputs and errors as seed_spec_forward, plus
 * SEED_ERR_CAPACITY when the sequence needs more than the array holds.
 */
seed_status seed_spec_forward_noalloc(seed_ctx* ctx, int32_t n, const int32_t* tokens, int32_t block,
                                      float* logits, float* row_nll, double* loss);

/* Committed tokens of sequence b (prompt included): out host [cap]; *len receives t_b. */
seed_status seed_get_tokens(seed_ctx* ctx, int32_t b, int32_t* out, int32_t cap, int32_t* len);

/*
 * Read back the cached keys/values KV^layer of sequence b at positions pos0 .. pos0+n-1 (the
 * per-layer cache of the Inference Algorithm; inspection and testing, not on the decode path).
 * k_out, v_out: host [n][n_kv_heads][head_dim], caller-owned, in the cache's element type
 * (bf16 bit patterns as uint16 for SEED_BF16, float for SEED_F32). Synchronises the context's
 * stream first, so every queued pass has written its entries. Positions below t_b - 1 hold the
 * committed deep keys/values; later positions hold whatever the last pass wrote there (draft
 * entries in the decoder layers, keys/values of rejected verification rows).
 * Errors: SEED_ERR_STATE before seed_prefill; SEED_ERR_ARG if b or layer is out of range, an
 * output pointer is NULL, or a position lies outside the cache blocks the sequence holds.
 */
seed_status seed_read_kv(seed_ctx* ctx, int32_t b, int32_t layer, int32_t pos0, int32_t n, void* k_out,
                         void* v_out);

/*
 * Kernel timing for benchmarks: while enabled, every launch of kernel_id (phase * 16 + op) is
 * bracketed by HIP events on the context's stream. seed_kernel_timing_read synchronises the
 * stream and returns the number of timed launches and their summed duration since enabling.
 * Rounds launched through a HIP graph are not timed.
 */
seed_status seed_kernel_timing(seed_ctx* ctx, int32_t kernel_id, int32_t enable);
seed_status seed_kernel_timing_read(seed_ctx* ctx, int64_t* launches, double* total_ms);

/* Text of the last error on the calling thread; valid until the next call on that thread. */
const char* seed_last_error(void);

/* Release the context (not the caller's buffers). NULL is ignored. */
void seed_destroy(seed_ctx* ctx);

#if defined(__GNUC__)
#pragma GCC visibility pop
#endif

#ifdef __cplusplus
}
#endif

#endif /* SEED_H */
