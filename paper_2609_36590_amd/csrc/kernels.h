// Internal interface between the host runtime and the gfx950 kernels of the SEED decode path.
// Nothing here is part of the public C ABI (include/seed.h).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace seedk {

// ---------------------------------------------------------------------------------------------
// Weight layout ("MFMA tile" packing). A linear weight W [N, K] (nn.Linear [out, in]) is stored
// as N/16 x K/32 tiles of 16 rows x 32 columns, tile (nt, kt) at element offset
// (nt * (K/32) + kt) * 512. Inside a tile, lane l (0..63) owns 8 consecutive elements
//   W[nt*16 + (l & 15)][kt*32 + (l >> 4)*8 + j],  j = 0..7,  at offset l*8 + j,
// which is exactly the A-operand fragment of a 16x16x32 MFMA (and 8 16x16x4 fp32 MFMAs), so a
// wave streams one tile as one fully coalesced 1 KB (bf16) / 2 KB (fp32) load.
//
// Fused matrices (row permutations applied when packing):
//  * QKV: rows [Wq; Wk; Wv]. Within each head, tile j (j < head_dim/16) holds dims
//    8j..8j+7 followed by their rotary partners head_dim/2+8j..+7, so RoPE is tile-local.
//  * gate/up: tile t holds gate rows 8t..8t+7 followed by up rows 8t..8t+7.
// ---------------------------------------------------------------------------------------------

enum Prologue { PRO_NORM = 0, PRO_PLAIN = 1 };
enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_HEAD = 3 };

// Arguments of the weight-streaming linear kernels (MFMA skinny GEMM and VALU GEMV).
struct LinArgs {
  const void* W;          // packed weights
  int N, K;               // output features, input features
  int M;                  // activation rows in this pass
  int NT, KS;             // n-tiles per workgroup pass, K-splits per n-tile
  int S;                  // the KS partial sums are added in S consecutive groups of KS/S, group
                          // by group in order (k_linear_lds: S == 1)
  int NJ;                 // LDS kernel: passes per workgroup (n-group blockIdx.x + j*gridDim.x)
  // input
  const float* X;         // [M][ldx] fp32 activations; PRO_NORM: x*g formed by the producer
  int ldx;
  const float* ssq;       // PRO_NORM: [M][nssq] partial sums of squares of x (per 16 features)
  int nssq;
  float eps;
  // EPI_RESID: h[m][n] += y, xg[m][n] = h[m][n] * gain_next[n] (input of the next RMSNorm
  // consumer), ssq_out[m][n/16] = sum of squares of the 16 updated values
  float* h;
  float* xg;
  const float* gain_next;
  float* ssq_out;
  // EPI_SWIGLU: act[m][f] = silu(gate) * up, f = nt*8 + c
  float* act;
  // EPI_QKV
  float* q;               // [M][n_heads*head_dim] rotated queries (fp32)
  void* kv;               // KV pool
  const int* row_pos;     // [M] absolute position of each row
  const int* row_slot;     // [M] cache position each row's keys/values are written to (= row_pos except for tree rows)
  const int* row_blk;     // [M] KV-pool block holding that position (same block in every layer)
  const float* row_rope;  // [M][head_dim]: cos(pos*theta_i) for i < head_dim/2, then sin(pos*theta_i)
  int layer, n_blocks, n_heads, n_kv, head_dim;
  // EPI_HEAD
  float* logits;          // nullable: logits[m * ld_logits + n]
  long long ld_logits;
  float* amax_val;        // per-workgroup argmax partials [M][amax_stride]
  int* amax_idx;
  int amax_stride;
  float* part;            // LIN_SPLITK: k-range partials [KS][M][N]
  float* part_rs;         // LIN_SPLITK with the RMSNorm prologue: row scales [M]
};

// Arguments of the split-KV paged attention kernel and its combine kernel.
struct AttnArgs {
  const float* q;         // [M][n_heads*head_dim]
  const void* kv;
  int layer, n_blocks;
  const int* bt;
  int bt_stride;
  const int* row_pos;     // [M]; rows m = b*R + r, consecutive positions within a sequence
  const int* row_slot;    // [M] cache slot of each row's keys/values (tree rows: p + node index;
                          // elsewhere equal to row_pos); the tree variant masks with it
  int B, R;               // sequences, rows per sequence
  int n_heads, n_kv, head_dim, G;  // G = n_heads / n_kv
  int RB, n_rb;           // rows per row-block (G*RB <= 32), row-blocks per sequence
  // block-causal pass of the speculative drafting objective (s_block > 0): row q (position q)
  // attends to the deep cache (kv, bt) at positions < s = floor(q / s_block) * s_block and to
  // the shallow cache skv (this pass's keys/values, block id = position / 16) at s..q
  const void* skv;
  int s_layer, s_n_blocks, s_block;
  int tree;               // 1: packed draft tree rows (mask by row_pos and row_slot)
  // one-launch pass attention (launch_attention_prefill): positions split over pf_split workgroups
  // per row-block, whose partials [pf_split][R][n_heads] (o: head_dim floats, then m and l) are
  // merged by a second kernel when pf_split > 1
  int pf_split;
  float* pf_o;
  float* pf_ml;
  int span;               // positions per workgroup group: 64, 128 or 256 (attention_span)
  int nq_alloc;           // set by the launcher: query vectors per row-block the LDS is sized for
  int n_groups_max;       // grid extent over groups; n_groups_max * span == bt_stride * 16
  float scale_log2;       // log2(e) / sqrt(head_dim)
  float* part;            // group partials [B][n_kv][n_rb][n_groups_max][32][head_dim + 4]
  float* out;             // [M][n_heads*head_dim]
};

// bytes of a prefill attention workgroup's staged block table (16-byte aligned)
__host__ __device__ inline int prefill_bt_bytes(int bt_stride) { return (bt_stride * 4 + 15) / 16 * 16; }

// Per-pass row setup + embedding gather.
enum SetupMode { SETUP_PREFILL = 0, SETUP_DRAFT = 1, SETUP_VERIFY = 2, SETUP_SPEC = 3, SETUP_TREE = 4 };

struct SetupArgs {
  int mode;
  int M, R;               // rows, rows per sequence
  const int* t;           // [B] committed lengths
  int* drafts;            // [B][dstride]; drafts[b][0] is the pending token
  int dstride;
  int step;               // SETUP_DRAFT: draft step i (>= 1)
  const int* tokens;      // committed tokens [B][tstride]
  int tstride;
  int pf_seq, pf_pos0;    // SETUP_PREFILL, SETUP_SPEC (rows at positions pf_pos0..)
  int sim_accept;         // SETUP_VERIFY / SETUP_TREE: -1 or forced acceptance length
  const int* trace;       // [B][tstride] greedy trace by absolute position
  int vocab;
  const void* E;          // packed embedding
  int H;
  int* row_seq;
  int* row_pos;
  int* row_slot;          // [M] cache slot of the row's keys/values
  int* tree_tok;          // SETUP_TREE: node tokens [M] (node 0 = the pending token)
  const int* tree_depth;  // SETUP_TREE: node depths [M] (rotary position t-1 + depth)
  // per-row KV block and RoPE row for the pass's QKV epilogues
  const int* bt;          // block tables [B][bt_stride]
  int bt_stride;
  const float* rope_cos;  // [max_ctx][head_dim/2]
  const float* rope_sin;
  int head_dim;
  int* row_blk;           // [M]
  float* row_rope;        // [M][head_dim]
  float* h;               // [M][H]
  float* xg;              // [M][H] h * gain (input of the pass's first RMSNorm consumer)
  const float* gain;      // [H]
  float* ssq;             // [M][H/16]
  // phase clock (nullable): block 0 writes the constant-rate clock to stamp[round * 3 + stamp_col]
  // when the kernel starts (round = *rounds, only while round < stamp_cap)
  long long* stamp;
  int stamp_col, stamp_cap;
  const int* rounds;
};

// Device-resident decoding state.
struct DevState {
  int* t;                 // [B] committed length
  int* len;               // [B] prompt length
  int* limit;             // [B] stop committing once t >= limit
  int* active;            // [B]
  int* nacc;              // [B] last n_accept
  int* bonus;             // [B] last bonus token
  int* rounds;            // [1] rounds run since prefill
  long long* counters;    // [2] drafted, accepted
  int* drafts;            // [B][dstride]
  int dstride;
  int* tokens;            // [B][tstride]
  int tstride;
  int* nacc_log;          // [log_cap][B]
  int log_cap;
  const int* vtok;        // [B*R] verifier argmax per row
  int eos;
  long long* stamp;       // nullable [stamp_cap][3]: the acceptance kernels write column 2 when done
  int stamp_cap;
};

// Kernel choice for a linear launch: weights streamed with the activation rows staged in LDS as
// MFMA fragments (M <= 16 and the rows fit), split-K across workgroups for up to 64 rows, the
// compute-bound tiled GEMM (LIN_WIDE) for wider passes, else activation fragments from global memory.
enum LinearKind { LIN_LDS = 0, LIN_GLOBAL = 1, LIN_SPLITK = 2, LIN_WIDE = 3 };
constexpr int LDS_MAX_PASSES = 8;   // n-tile passes (NJ) of one k_linear_lds workgroup
constexpr int HEAD_WIDE_NT = 16;    // n-tiles (waves) per workgroup of the LM head for 17..64 rows
constexpr int PF_SPLIT_MAX = 4;    // position splits of the one-launch pass attention
constexpr int WIDE_SPLIT_MAX = 4;   // k-ranges of a split wide pass (its partials: WIDE_SPLIT_MAX x rows x N floats)

// Optional timing events stamped by the launches themselves (hipExtLaunchKernel): `start` at the
// start of the first kernel of the operation, `stop` at the end of its last kernel.
struct LaunchEvents {
  hipEvent_t start, stop;
};

template <typename T>
void launch_linear(const LinArgs& a, int prologue, int epilogue, int kind, hipStream_t s,
                   const LaunchEvents* ev = nullptr);
// Attention partials per group of span positions (the final output when the rows see one group).
template <typename T>
void launch_attention(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev = nullptr);
// Causal attention of a single-sequence pass of more than 64 rows (the prompt's prefill), written
// directly (no partials): 64 query vectors per workgroup, every visible tile streamed in order.
bool attention_prefill_supported(const AttnArgs& a);
template <typename T>
void launch_attention_prefill(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev = nullptr);
// Merge of the group partials; needed when the context capacity spans more than one group.
bool attention_needs_combine(const AttnArgs& a);
// Positions per attention group for a context capacity and batch capacity (fixed per decoder, so
// that a query's merge tree depends only on absolute positions).
int attention_span(int max_ctx, int max_batch);
void launch_attn_combine(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev = nullptr);
template <typename T>
void launch_setup(const SetupArgs& a, hipStream_t s);
void launch_accept(const DevState& st, int B, int k, hipStream_t s);
// Tree acceptance for one sequence (packed tree of n nodes: tokens, parents, depths; the verifier
// argmax per node in st.vtok) and the move of an accepted leaf's keys/values in every layer to the
// cache position of its depth. out[0] = accepted path length, out[1] = bonus, out[2..] = path.
void launch_accept_tree(const DevState& st, int n, const int* tree_tok, const int* tree_par, const int* tree_depth,
                        int* out, void* kv, int n_layers, int n_blocks, int n_kv, int head_dim, int esize,
                        const int* bt, int* hstat, hipStream_t s);
// Confidence-aware dynamic drafting (Method, Adaptive Drafting with Tree-Based Verification;
// appendix "Confidence-Aware Dynamic Drafting"): after each drafting step, the top-1 probability
// p0 of the step's logits and its ranked top candidates; the top-p table gives the fan-out, the
// threshold tau the stop, and the tree is packed when drafting stops.
constexpr int TOPK_MAX = 16;        // largest fan-out a table may ask for
constexpr int TREE_MAX_STEPS = 16;  // drafting steps of one round (max_draft <= 15)
constexpr int TOPK_PARTS = 256;     // first-stage waves (each covers a contiguous logit chunk)

struct TreeDraftArgs {
  const float* logits;   // [V] the step's drafter logits
  int V, chunk;          // chunk: logits per first-stage wave (multiple of 64)
  int step;              // drafting step i >= 1 (X_draft[i] is being chosen)
  float* pval;           // first stage: [TOPK_PARTS][TOPK_MAX] candidate logits
  int* pidx;             //   and token ids (-1 = none)
  float* pmax;           //   [TOPK_PARTS] chunk maximum
  float* psum;           //   [TOPK_PARTS] sum of exp(z - chunk maximum)
  // fan-out rule: k = kk[j] for the first j with p0 > thr[j], else k_rest
  float tau;
  int n_levels;
  float thr[4];
  int kk[4];
  int k_rest, k_max;     // k_max: the table's largest fan-out (candidates kept per wave)
  int max_depth, max_nodes;
  // the round's drafting state
  int* cand;             // [TREE_MAX_STEPS][TOPK_MAX] ranked candidates of step i
  int* kcnt;             // [TREE_MAX_STEPS] fan-out used at step i
  float* p0;             // [TREE_MAX_STEPS] top-1 probability of step i
  int* dstate;           // [0] drafting stopped, [1] nodes so far (root included)
  int* drafts;           // sequence 0's drafts row: [0] the root X[p], [i] the chain token of step i
  int* tree;             // packed tree: token [64], parent [64], depth [64]; tree[192] = node count
  const int* rounds;     // rounds run so far: tags the status written when drafting stops
  int* hstat;            // nullable host-visible status: [0] round tag, [1] nodes, [2] depth
};
void launch_tree_topk(const TreeDraftArgs& a, hipStream_t s);
int tree_topk_chunk(int V);

// nll[r] = logsumexp(logits[r]) - logits[r][target[r]] for r < rows (row stride V)
void launch_row_nll(const float* logits, int rows, int V, const int* target, float* nll, hipStream_t s);
// Reduce the head's per-workgroup argmax partials of M rows; row m's token goes to
// tok_out[m * tok_stride] (lowest token id among equal maxima).
void launch_argmax_finalize(const float* val, const int* idx, int stride, int n_parts, int M, int* tok_out,
                            int tok_stride, hipStream_t s);
template <typename T>
void launch_pack(const void* src, void* dst, const int* dst_row, int rows, int K, hipStream_t s);
void launch_to_f32(const void* src, int src_is_bf16, float* dst, long long n, hipStream_t s);
void launch_fill_u32(void* dst, unsigned value, long long n_words, hipStream_t s);

// allow the linear kernels to use more than 64 KB of LDS (once per process and dtype)
hipError_t configure_kernels(int bf16);
// dynamic LDS bytes one linear workgroup may use (valid after configure_kernels)
size_t linear_lds_limit();

// dynamic LDS bytes needed by launch_linear for a given shape
size_t linear_lds_bytes(int M, int K, int NT, int KS, int S, int NJ, int kind);

}  // namespace seedk
