// Host runtime of the SEED decode library: the C ABI declared in include/seed.h.
//
// It plans the three caller-owned buffers (weight arena, paged KV pool, workspace), repacks the
// weights into MFMA tiles, keeps the per-sequence block tables, and enqueues the passes of
// Algorithm 2 (prefill, draft steps, verification + acceptance) on the caller's HIP stream. All
// per-round state (committed lengths, pending token, drafts, acceptance) lives on the device,
// so rounds can be queued back to back, or replayed from a captured HIP graph, with no host
// synchronisation.
#include "seed.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "kernels.h"

using namespace seedk;

// Scratch of seed_spec_forward_noalloc (the drafting-objective pass's own keys/values): one copy
// per GPU, held by the loaded library until the process ends. Every call on a GPU shares it.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)16 << 20;
static __device__ __align__(256) char scratch[NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

// Device address of `scratch` on each GPU (the host-side name is not a device address): taken
// once per device, with that device current, at context creation.
std::mutex g_scratch_mu;
std::map<int, char*> g_scratch_addr;

seed_status fail(seed_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIPCHK(expr)                                                                         \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(SEED_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr int PREFILL_ROWS = 1024; // rows per prefill / drafting-objective pass (tiled MFMA GEMMs)
constexpr int PF_SPLIT_LONG = 3;   // position splits of a pass's attention beyond its first PREFILL_ROWS
static_assert(PF_SPLIT_LONG <= seedk::PF_SPLIT_MAX, "split partials fit the workspace");
constexpr int MAX_ROWS = 64;       // rows per decode pass: max_batch * (max_draft + 1)
constexpr int ATT_ROWS = 256;      // rows per attention launch of a wider single-sequence pass

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int cdiv(int a, int b) { return (a + b - 1) / b; }

struct Plan {
  seed_config cfg;
  int esize = 2;
  int H, NQ, NKV, HD, F, V, L, LD, QD, KVD, G;
  int RB, n_rb_max, max_rows, bt_stride, blocks_per_seq, n_blocks, span, n_groups_max;
  int dstride, tstride, log_cap;
  // weight arena
  size_t w_embed, w_final_norm, w_rope_cos, w_rope_sin, w_total;
  std::vector<size_t> w_attn_norm, w_mlp_norm, w_qkv, w_o, w_gu, w_down;
  size_t kv_total;
  // workspace
  size_t o_pf_o, o_pf_ml, o_wide_part, o_h, o_xg, o_ssq, o_q, o_attn, o_act, o_part, o_row_seq, o_row_pos, o_row_slot, o_row_blk, o_row_rope, o_amax_val,
      o_amax_idx, o_vtok;
  size_t o_t, o_len, o_limit, o_active, o_nacc, o_bonus, o_rounds, o_counters, o_drafts, o_tokens,
      o_trace, o_log, o_bt, o_nll, o_splitk, o_splitk_rs, o_tree, o_tree_out, o_scratch, o_stamp, ws_total;
  // dynamic drafting: top-k partials, the round's drafting state, one step's drafter logits
  size_t o_topk, o_tdraft, o_dlog;
};

seed_status validate(const seed_config* c) {
  if (!c) return fail(SEED_ERR_ARG, "config is NULL");
  if (c->dtype != SEED_F32 && c->dtype != SEED_BF16) return fail(SEED_ERR_ARG, "dtype must be SEED_F32 or SEED_BF16");
  if (c->n_layers < 1 || c->n_dec_layers < 0 || c->n_dec_layers > c->n_layers)
    return fail(SEED_ERR_ARG, "need n_layers >= 1 and 0 <= n_dec_layers <= n_layers");
  if (c->hidden <= 0 || c->ffn <= 0 || c->vocab <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0)
    return fail(SEED_ERR_ARG, "model sizes must be positive");
  if (c->hidden % 32 || c->ffn % 32 || (c->n_heads * c->head_dim) % 32 || (c->n_kv_heads * c->head_dim) % 32)
    return fail(SEED_ERR_UNSUPPORTED, "hidden, ffn, n_heads*head_dim and n_kv_heads*head_dim must be multiples of 32");
  if (c->vocab % 16) return fail(SEED_ERR_UNSUPPORTED, "vocab must be a multiple of 16");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(SEED_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->n_heads % c->n_kv_heads || c->n_heads / c->n_kv_heads > 32)
    return fail(SEED_ERR_UNSUPPORTED, "n_heads must be a multiple of n_kv_heads with a group of at most 32");
  if (c->kv_block != 16) return fail(SEED_ERR_UNSUPPORTED, "kv_block must be 16");
  if (c->max_batch < 1 || c->max_batch > 64) return fail(SEED_ERR_UNSUPPORTED, "max_batch must be in [1, 64]");
  if (c->max_draft < 0 || c->max_draft > 15) return fail(SEED_ERR_UNSUPPORTED, "max_draft must be in [0, 15]");
  if (c->max_batch * (c->max_draft + 1) > MAX_ROWS)
    return fail(SEED_ERR_UNSUPPORTED, "max_batch * (max_draft + 1) must be at most 64");
  if (c->max_ctx < 2) return fail(SEED_ERR_ARG, "max_ctx must be at least 2");
  if (c->max_ctx > (1 << 20)) return fail(SEED_ERR_UNSUPPORTED, "max_ctx must be at most 2^20");
  if (!(c->rope_base > 0.f) || !(c->rms_eps >= 0.f)) return fail(SEED_ERR_ARG, "rope_base must be > 0 and rms_eps >= 0");
  return SEED_OK;
}

void tile_policy(int N, int K, bool head, int& NT, int& KS, int& S, int& NJ);

Plan make_plan(const seed_config& c) {
  Plan p;
  p.cfg = c;
  p.esize = c.dtype == SEED_BF16 ? 2 : 4;
  p.H = c.hidden; p.NQ = c.n_heads; p.NKV = c.n_kv_heads; p.HD = c.head_dim; p.F = c.ffn; p.V = c.vocab;
  p.L = c.n_layers; p.LD = c.n_layers - c.n_dec_layers;
  p.QD = p.NQ * p.HD; p.KVD = p.NKV * p.HD; p.G = p.NQ / p.NKV;
  p.RB = std::max(1, 32 / p.G);
  // attention row-blocks of one launch: a decode pass (<= MAX_ROWS rows over max_batch sequences)
  // or ATT_ROWS rows of one sequence's prefill / drafting-objective pass
  p.n_rb_max = cdiv(MAX_ROWS, p.RB);
  p.max_rows = std::max(MAX_ROWS, PREFILL_ROWS);   // decode passes (B (d+1) <= 64), draft trees of <= 64
                                                  // nodes, prefill and drafting-objective passes
  p.blocks_per_seq = cdiv(c.max_ctx, 16);
  p.span = seedk::attention_span(c.max_ctx, c.max_batch);
  p.bt_stride = cdiv(p.blocks_per_seq, p.span / 16) * (p.span / 16);   // whole groups, padded with block 0
  p.n_blocks = c.max_batch * p.blocks_per_seq + 1;                  // block 0 = permanent zero block

  p.n_groups_max = p.bt_stride * 16 / p.span;
  p.dstride = c.max_draft + 1;
  p.tstride = c.max_ctx;
  p.log_cap = c.max_ctx;

  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align256(o + bytes); return r; };
  const size_t es = p.esize;
  p.w_embed = take((size_t)p.V * p.H * es);
  p.w_final_norm = take((size_t)p.H * 4);
  p.w_rope_cos = take((size_t)c.max_ctx * (p.HD / 2) * 4);
  p.w_rope_sin = take((size_t)c.max_ctx * (p.HD / 2) * 4);
  for (int l = 0; l < p.L; ++l) {
    p.w_attn_norm.push_back(take((size_t)p.H * 4));
    p.w_mlp_norm.push_back(take((size_t)p.H * 4));
    p.w_qkv.push_back(take((size_t)(p.QD + 2 * p.KVD) * p.H * es));
    p.w_o.push_back(take((size_t)p.H * p.QD * es));
    p.w_gu.push_back(take((size_t)2 * p.F * p.H * es));
    p.w_down.push_back(take((size_t)p.H * p.F * es));
  }
  p.w_total = o;

  p.kv_total = align256((size_t)p.L * p.n_blocks * 2 * p.NKV * 16 * p.HD * es);

  o = 0;
  const size_t R = p.max_rows, B = c.max_batch;
  p.o_h = take(R * p.H * 4);
  p.o_xg = take(R * p.H * 4);
  p.o_ssq = take(R * (p.H / 16) * 4);
  p.o_q = take(R * p.QD * 4);
  p.o_attn = take(R * p.QD * 4);
  p.o_act = take(R * p.F * 4);
  p.o_part = take(std::max(B * p.n_rb_max, (size_t)cdiv(ATT_ROWS, p.RB)) * p.NKV * (size_t)p.n_groups_max * 32 *
                  (p.HD + 4) * 4);
  p.o_row_seq = take(R * 4);
  p.o_row_pos = take(R * 4);
  p.o_row_slot = take(R * 4);
  p.o_row_blk = take(R * 4);
  p.o_row_rope = take(R * p.HD * 4);
  p.o_amax_val = take(R * (size_t)(p.V / 16) * 4);
  p.o_amax_idx = take(R * (size_t)(p.V / 16) * 4);
  p.o_vtok = take(R * 4);
  p.o_t = take(B * 4);
  p.o_len = take(B * 4);
  p.o_limit = take(B * 4);
  p.o_active = take(B * 4);
  p.o_nacc = take(B * 4);
  p.o_bonus = take(B * 4);
  p.o_rounds = take(4);
  p.o_counters = take(16);
  p.o_drafts = take(B * p.dstride * 4);
  p.o_tokens = take(B * (size_t)p.tstride * 4);
  p.o_trace = take(B * (size_t)p.tstride * 4);
  p.o_log = take((size_t)p.log_cap * B * 4);
  p.o_stamp = take((size_t)p.log_cap * 3 * 8);   // per round: drafting start, verification start, end
  p.o_bt = take(B * (size_t)p.bt_stride * 4);
  p.o_nll = take((size_t)c.max_ctx * 4);
  p.o_tree = take((3 * MAX_ROWS + 1) * 4);
  p.o_tree_out = take((2 + MAX_ROWS + 2) * 4);
  {
    // k-range partials of the split-K path (passes of more than 16 rows): KS x rows x N floats
    size_t ksn = 0;
    const int shapes[4][2] = {{p.QD + 2 * p.KVD, p.H}, {p.H, p.QD}, {2 * p.F, p.H}, {p.H, p.F}};
    for (const auto& sh : shapes) {
      int NT, KS, S, NJ;
      tile_policy(sh[0], sh[1], false, NT, KS, S, NJ);
      ksn = std::max(ksn, (size_t)KS * sh[0]);
    }
    p.o_splitk = take(ksn * MAX_ROWS * 4);   // only passes of at most MAX_ROWS rows split K
    p.o_splitk_rs = take((size_t)MAX_ROWS * 4);
  }
  p.o_pf_o = take((size_t)PF_SPLIT_LONG * p.max_rows * p.QD * 4);   // split pass attention partials
  p.o_pf_ml = take((size_t)PF_SPLIT_LONG * p.max_rows * p.NQ * 2 * 4);
  p.o_wide_part = take((size_t)seedk::WIDE_SPLIT_MAX * p.max_rows * p.H * 4);   // split wide passes (N = H)
  p.o_topk = take((size_t)TOPK_PARTS * (2 * TOPK_MAX + 2) * 4);
  p.o_tdraft = take((size_t)TREE_MAX_STEPS * (TOPK_MAX + 2) * 4 + 16);
  p.o_dlog = take((size_t)p.V * 4);
  p.o_scratch = take((size_t)std::max({p.V, p.QD + 2 * p.KVD, 2 * p.F, p.H}) * 4);
  p.ws_total = o;
  return p;
}

// Timing events of one call, destroyed on every return path.
struct CallEvents {
  hipEvent_t e[3] = {nullptr, nullptr, nullptr};
  hipError_t create() {
    for (auto& x : e) {
      const hipError_t r = hipEventCreate(&x);
      if (r != hipSuccess) return r;
    }
    return hipSuccess;
  }
  ~CallEvents() {
    for (auto& x : e)
      if (x) hipEventDestroy(x);
  }
};

struct TimedLaunch {
  hipEvent_t a, b;
};

}  // namespace

struct seed_ctx {
  Plan p;
  hipStream_t s = nullptr;
  char* W = nullptr;
  char* KV = nullptr;
  char* WS = nullptr;
  std::vector<bool> loaded;
  bool weights_ok = false;
  // decoding state mirrored on the host
  int B = 0;
  bool prefilled = false;
  std::vector<int> lens, t_upper;
  int drafts_k = -1;
  int sim_accept = -1;
  int eos = -1;
  // paged KV allocator
  std::vector<int> free_blocks;
  std::vector<std::vector<int>> seq_blocks;
  std::vector<int> bt_host;
  // kernel timing
  int timed_id = -1;
  std::vector<TimedLaunch> pending;
  std::vector<TimedLaunch> pool;
  int64_t timed_launches = 0;
  double timed_ms = 0.0;
  // graphs: (B, k, sim_accept, eos) -> exec (the eos id is a kernel argument of the acceptance)
  std::map<std::tuple<int, int, int, int>, hipGraphExec_t> graphs;
  // dynamic drafting: step graphs (for the options in tree_key), verification graphs by node
  // count, and a pinned status the drafting/acceptance kernels write for the host loop
  std::map<int, hipGraphExec_t> tree_step_graphs;
  std::map<std::tuple<int, int, int>, hipGraphExec_t> tree_verify_graphs;   // (nodes, eos, sim_accept)
  seed_tree_opts tree_key{};
  int* hstat = nullptr;       // host pointer
  int* hstat_dev = nullptr;   // its device address
  char* scratch_dev = nullptr;   // this device's copy of `scratch` (nullptr if unavailable)

  template <typename X>
  X* ws(size_t off) { return reinterpret_cast<X*>(WS + off); }
  float* wf(size_t off) { return reinterpret_cast<float*>(W + off); }
};

namespace {

// ---------------------------------------------------------------------------------------------
// kernel timing
// ---------------------------------------------------------------------------------------------
hipError_t drain_timing(seed_ctx* c) {
  if (c->pending.empty()) return hipSuccess;
  hipError_t e = hipStreamSynchronize(c->s);
  if (e != hipSuccess) return e;
  for (auto& t : c->pending) {
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, t.a, t.b);
    if (e != hipSuccess) return e;
    c->timed_ms += ms;
    c->timed_launches += 1;
    c->pool.push_back(t);
  }
  c->pending.clear();
  return hipSuccess;
}

// Linear and attention launches stamp timing events from the kernels themselves
// (hipExtLaunchKernel); the small kernels are bracketed by event records on the stream.
bool stamps_events(int op) {
  return op == SEED_OP_QKV || op == SEED_OP_ATTN || op == SEED_OP_COMBINE || op == SEED_OP_O ||
         op == SEED_OP_GATEUP || op == SEED_OP_DOWN || op == SEED_OP_HEAD;
}

// Runs fn(events): events is non-null only when this (phase, op) is being timed, the stream is
// not being captured and the op's launches stamp the events themselves.
template <typename F>
void timed(seed_ctx* c, int phase, int op, bool capturing, F&& fn) {
  if (!capturing && c->timed_id == phase * 16 + op) {
    if (c->pending.size() >= 512) drain_timing(c);
    TimedLaunch t;
    if (!c->pool.empty()) { t = c->pool.back(); c->pool.pop_back(); }
    else { hipEventCreate(&t.a); hipEventCreate(&t.b); }
    LaunchEvents ev{t.a, t.b};
    if (!stamps_events(op)) hipEventRecord(t.a, c->s);
    fn(stamps_events(op) ? &ev : nullptr);
    if (!stamps_events(op)) hipEventRecord(t.b, c->s);
    c->pending.push_back(t);
  } else {
    fn(nullptr);
  }
}

// ---------------------------------------------------------------------------------------------
// launch helpers
// ---------------------------------------------------------------------------------------------
// Waves per workgroup and how they split the work; a function of the weight shape only, so a
// row's reduction order never depends on how many rows share the pass (measured on MI355X):
//   head (N = vocab): one n-tile per wave over the full K, 8 n-tiles per workgroup.
//   N >= 4096 (QKV, gate/up): 8 K-splits, 2 n-tiles per workgroup pass, and as many passes per
//     workgroup as keep the grid near 200 workgroups (the LDS kernel stages the activations once
//     per workgroup).
//   smaller N (O, down): one n-tile per workgroup, K split in ranges of about 16 k-tiles (<= 16).
void tile_policy(int N, int K, bool head, int& NT, int& KS, int& S, int& NJ) {
  const int KT = K / 32, n_tiles = N / 16;
  S = 1;
  NJ = 1;
  if (head) {
    KS = 1;
    NT = 8;
    return;
  }
  if (n_tiles >= 256) {
    KS = std::min(8, KT);
    NT = 2;
    NJ = std::min(LDS_MAX_PASSES, std::max(1, (cdiv(n_tiles, NT) + 100) / 200));
    return;
  }
  KS = std::min(16, std::max(1, KT / 16));
  NT = 1;
}

DevState dev_state(seed_ctx* c) {
  const Plan& p = c->p;
  DevState st;
  st.t = c->ws<int>(p.o_t);
  st.len = c->ws<int>(p.o_len);
  st.limit = c->ws<int>(p.o_limit);
  st.active = c->ws<int>(p.o_active);
  st.nacc = c->ws<int>(p.o_nacc);
  st.bonus = c->ws<int>(p.o_bonus);
  st.rounds = c->ws<int>(p.o_rounds);
  st.counters = c->ws<long long>(p.o_counters);
  st.drafts = c->ws<int>(p.o_drafts);
  st.dstride = p.dstride;
  st.tokens = c->ws<int>(p.o_tokens);
  st.tstride = p.tstride;
  st.nacc_log = c->ws<int>(p.o_log);
  st.log_cap = p.log_cap;
  st.vtok = c->ws<int>(p.o_vtok);
  st.eos = c->eos;
  st.stamp = c->ws<long long>(p.o_stamp);
  st.stamp_cap = p.log_cap;
  return st;
}

LinArgs lin_base(seed_ctx* c, int M) {
  const Plan& p = c->p;
  LinArgs a;
  std::memset(&a, 0, sizeof(a));
  a.M = M;
  a.ssq = c->ws<float>(p.o_ssq);
  a.nssq = p.H / 16;
  a.eps = p.cfg.rms_eps;
  a.h = c->ws<float>(p.o_h);
  a.xg = c->ws<float>(p.o_xg);
  a.ssq_out = c->ws<float>(p.o_ssq);
  a.act = c->ws<float>(p.o_act);
  a.q = c->ws<float>(p.o_q);
  a.kv = c->KV;
  a.row_pos = c->ws<int>(p.o_row_pos);
  a.row_slot = c->ws<int>(p.o_row_slot);
  a.row_blk = c->ws<int>(p.o_row_blk);
  a.row_rope = c->ws<float>(p.o_row_rope);
  a.n_blocks = p.n_blocks;
  a.n_heads = p.NQ;
  a.n_kv = p.NKV;
  a.head_dim = p.HD;
  a.amax_val = c->ws<float>(p.o_amax_val);
  a.amax_idx = c->ws<int>(p.o_amax_idx);
  a.amax_stride = p.V / 16;
  a.part = c->ws<float>(p.o_splitk);
  a.part_rs = c->ws<float>(p.o_splitk_rs);
  return a;
}

// Kernel for one linear launch: activation rows staged in LDS when they fit (M <= 16); passes of
// more rows split K across workgroups (each stages its k-range only) and add the range partials
// in a second kernel; otherwise activation fragments are read from global memory.
// Measured on MI355X (4B-scale shapes, M = 1..16): staging the rows in LDS wins while a workgroup
// stages at most 9 x 4096 activations; beyond that the split-K kernel (each workgroup stages one
// k-range) is faster than both the LDS kernel and the global-fragment kernel.
int linear_kind(const LinArgs& a, bool head) {
  if (a.M > MAX_ROWS) return LIN_WIDE;   // prefill / drafting-objective passes: compute-bound tiles
  if (a.M <= 16 && (head || (long long)a.M * a.K <= 9 * 4096) &&
      linear_lds_bytes(a.M, a.K, a.NT, a.KS, a.S, a.NJ, LIN_LDS) <= linear_lds_limit())
    return LIN_LDS;
  if (!head && linear_lds_bytes(a.M, a.K, a.NT, a.KS, a.S, a.NJ, LIN_SPLITK) <= linear_lds_limit())
    return LIN_SPLITK;
  return LIN_GLOBAL;
}

// n-tiles per workgroup of the LM head: 8, or HEAD_WIDE_NT for the 17..64-row passes (the chunked
// kernel), where each workgroup stages every row; the argmax partials are per such group
int head_nt(int M) { return (M > 16 && M <= MAX_ROWS) ? HEAD_WIDE_NT : 8; }

template <typename T>
void linear(seed_ctx* c, LinArgs a, int pro, int epi, int phase, int op, bool cap) {
  tile_policy(a.N, a.K, epi == EPI_HEAD, a.NT, a.KS, a.S, a.NJ);
  if (epi == EPI_HEAD) a.NT = head_nt(a.M);
  const int kind = linear_kind(a, epi == EPI_HEAD);
  if (kind == LIN_WIDE) a.part = c->ws<float>(c->p.o_wide_part);
  timed(c, phase, op, cap, [&](const LaunchEvents* ev) { launch_linear<T>(a, pro, epi, kind, c->s, ev); });
}

// The block-causal decoder pass of the speculative drafting objective: its keys/values go to a
// cache of their own (decoder layers only, indexed by position), the deep cache is only read.
struct SpecPass {
  void* kv;
  int n_blocks;   // blocks per layer of kv
  int block;      // block size b of the objective
};

// Layers [l0, l1) over M rows (B sequences x R rows each, consecutive positions per sequence).
template <typename T>
void run_layers(seed_ctx* c, int M, int B, int R, int l0, int l1, int phase,
                const int* bt_override, bool cap, const SpecPass* spec = nullptr, bool tree = false,
                int pass_pos0 = 0) {
  const Plan& p = c->p;
  float* h = c->ws<float>(p.o_h);
  for (int li = l0; li < l1; ++li) {
    LinArgs a = lin_base(c, M);
    a.layer = li;
    if (spec) {
      a.kv = spec->kv;
      a.layer = li - p.LD;
      a.n_blocks = spec->n_blocks;
    }
    // QKV + RoPE + KV write
    a.W = c->W + p.w_qkv[li]; a.N = p.QD + 2 * p.KVD; a.K = p.H;
    a.X = c->ws<float>(p.o_xg); a.ldx = p.H;
    linear<T>(c, a, PRO_NORM, EPI_QKV, phase, SEED_OP_QKV, cap);
    // attention
    AttnArgs at;
    std::memset(&at, 0, sizeof(at));
    at.q = c->ws<float>(p.o_q);
    at.kv = c->KV;
    at.layer = li;
    at.n_blocks = p.n_blocks;
    at.bt = bt_override ? bt_override : c->ws<int>(p.o_bt);
    at.bt_stride = p.bt_stride;
    at.row_pos = c->ws<int>(p.o_row_pos);
    at.row_slot = c->ws<int>(p.o_row_slot);
    at.tree = tree ? 1 : 0;
    at.B = B; at.R = R;
    at.n_heads = p.NQ; at.n_kv = p.NKV; at.head_dim = p.HD; at.G = p.G;
    at.RB = p.RB; at.n_rb = cdiv(R, p.RB);
    at.span = p.span;
    at.n_groups_max = p.n_groups_max;
    if (spec) {
      at.skv = spec->kv;
      at.s_layer = li - p.LD;
      at.s_n_blocks = spec->n_blocks;
      at.s_block = spec->block;
    }
    at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)p.HD));
    at.part = c->ws<float>(p.o_part);
    at.out = c->ws<float>(p.o_attn);
    at.pf_o = c->ws<float>(p.o_pf_o);
    at.pf_ml = c->ws<float>(p.o_pf_ml);
    // a one-launch pass over a long cache splits each row-block's positions over PF_SPLIT_LONG
    // workgroups (4B 16k prefill 651 / 634 / 607 / 610 ms with 1 / 2 / 3 / 4); a pass from position 0
    // stays whole (its 1024-token prefill 23.9 / 24.0 / 24.2 / 24.4 ms: the merge costs more than the
    // shorter chains save)
    at.pf_split = pass_pos0 >= PREFILL_ROWS ? PF_SPLIT_LONG : 1;
    // the prompt's prefill (one sequence, more than 64 rows): one launch over all of the pass's
    // rows, written directly. Otherwise group partials and their merge; a pass wider than the
    // partial buffer (the drafting objective's) runs its rows ATT_ROWS at a time, every row
    // attending to its own positions either way
    const bool whole_pass = B == 1 && R > MAX_ROWS && attention_prefill_supported(at);
    if (whole_pass)
      timed(c, phase, SEED_OP_ATTN, cap, [&](const LaunchEvents* ev) { launch_attention_prefill<T>(at, c->s, ev); });
    const int r_step = (B == 1 && R > MAX_ROWS) ? ATT_ROWS : R;
    for (int r0 = 0; r0 < R && !whole_pass; r0 += r_step) {
      AttnArgs as = at;
      as.R = std::min(r_step, R - r0);
      as.n_rb = cdiv(as.R, p.RB);
      as.q = at.q + (size_t)r0 * p.QD;
      as.out = at.out + (size_t)r0 * p.QD;
      as.row_pos = at.row_pos + r0;
      as.row_slot = at.row_slot + r0;
      timed(c, phase, SEED_OP_ATTN, cap, [&](const LaunchEvents* ev) { launch_attention<T>(as, c->s, ev); });
      if (attention_needs_combine(as))
        timed(c, phase, SEED_OP_COMBINE, cap, [&](const LaunchEvents* ev) { launch_attn_combine(as, c->s, ev); });
    }
    // O + residual
    a = lin_base(c, M);
    a.W = c->W + p.w_o[li]; a.N = p.H; a.K = p.QD;
    a.X = c->ws<float>(p.o_attn); a.ldx = p.QD; a.gain_next = c->wf(p.w_mlp_norm[li]);
    linear<T>(c, a, PRO_PLAIN, EPI_RESID, phase, SEED_OP_O, cap);
    // gate/up + SwiGLU
    a = lin_base(c, M);
    a.W = c->W + p.w_gu[li]; a.N = 2 * p.F; a.K = p.H;
    a.X = c->ws<float>(p.o_xg); a.ldx = p.H;
    linear<T>(c, a, PRO_NORM, EPI_SWIGLU, phase, SEED_OP_GATEUP, cap);
    // down + residual
    a = lin_base(c, M);
    a.W = c->W + p.w_down[li]; a.N = p.H; a.K = p.F;
    a.X = c->ws<float>(p.o_act); a.ldx = p.F;
    a.gain_next = c->wf(li + 1 < p.L ? p.w_attn_norm[li + 1] : p.w_final_norm);
    linear<T>(c, a, PRO_PLAIN, EPI_RESID, phase, SEED_OP_DOWN, cap);
  }
}

template <typename T>
void run_head(seed_ctx* c, int M, int* tok_out, int tok_stride, float* logits, long long ld,
              int phase, bool cap) {
  const Plan& p = c->p;
  LinArgs a = lin_base(c, M);
  a.W = c->W + p.w_embed; a.N = p.V; a.K = p.H;
  a.X = c->ws<float>(p.o_xg); a.ldx = p.H;
  a.logits = logits; a.ld_logits = ld;
  if (!tok_out) a.amax_val = nullptr, a.amax_idx = nullptr;   // logits only: no argmax partials
  linear<T>(c, a, PRO_NORM, EPI_HEAD, phase, SEED_OP_HEAD, cap);
  const int parts = cdiv(p.V / 16, head_nt(M));   // one argmax partial per n-group
  if (!tok_out) return;   // the caller ranks the logits itself (dynamic drafting)
  timed(c, phase, SEED_OP_HEAD_ARGMAX, cap, [&](const LaunchEvents*) {
    launch_argmax_finalize(a.amax_val, a.amax_idx, a.amax_stride, parts, M, tok_out, tok_stride, c->s);
  });
}

// Setup for a pass whose first layer is l0 (its RMSNorm gain forms x*g; the head's gain when the
// pass has no layers).
SetupArgs setup_base(seed_ctx* c, int l0) {
  const Plan& p = c->p;
  SetupArgs s;
  std::memset(&s, 0, sizeof(s));
  s.t = c->ws<int>(p.o_t);
  s.drafts = c->ws<int>(p.o_drafts);
  s.dstride = p.dstride;
  s.tokens = c->ws<int>(p.o_tokens);
  s.tstride = p.tstride;
  s.sim_accept = -1;
  s.trace = c->ws<int>(p.o_trace);
  s.vocab = p.V;
  s.E = c->W + p.w_embed;
  s.H = p.H;
  s.row_seq = c->ws<int>(p.o_row_seq);
  s.row_pos = c->ws<int>(p.o_row_pos);
  s.row_slot = c->ws<int>(p.o_row_slot);
  s.bt = c->ws<int>(p.o_bt);
  s.bt_stride = p.bt_stride;
  s.rope_cos = c->wf(p.w_rope_cos);
  s.rope_sin = c->wf(p.w_rope_sin);
  s.head_dim = p.HD;
  s.row_blk = c->ws<int>(p.o_row_blk);
  s.row_rope = c->ws<float>(p.o_row_rope);
  s.h = c->ws<float>(p.o_h);
  s.xg = c->ws<float>(p.o_xg);
  s.gain = c->wf(l0 < p.L ? p.w_attn_norm[l0] : p.w_final_norm);
  s.ssq = c->ws<float>(p.o_ssq);
  s.rounds = c->ws<int>(p.o_rounds);
  s.stamp_cap = p.log_cap;
  return s;
}

// The setup kernel that opens a phase of a round stamps the device clock (column 0: drafting,
// 1: verification; the acceptance kernel writes column 2 when the round is done).
void stamp_phase(seed_ctx* c, SetupArgs& s, int col) {
  s.stamp = c->ws<long long>(c->p.o_stamp);
  s.stamp_col = col;
}

// Drafting phase: k decoder-only steps for every sequence.
template <typename T>
void enqueue_draft(seed_ctx* c, int k, float* logits, bool cap) {
  const Plan& p = c->p;
  const int B = c->B;
  for (int i = 1; i <= k; ++i) {
    SetupArgs s = setup_base(c, p.LD);
    s.mode = SETUP_DRAFT; s.M = B; s.R = 1; s.step = i;
    if (i == 1) stamp_phase(c, s, 0);
    timed(c, SEED_PHASE_DRAFT, SEED_OP_SETUP, cap, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
    run_layers<T>(c, B, B, 1, p.LD, p.L, SEED_PHASE_DRAFT, nullptr, cap);
    run_head<T>(c, B, c->ws<int>(p.o_drafts) + i, p.dstride,
                logits ? logits + (size_t)(i - 1) * p.V : nullptr, (long long)k * p.V, SEED_PHASE_DRAFT, cap);
  }
}

// Verification phase + acceptance/commit.
template <typename T>
void enqueue_verify(seed_ctx* c, int k, int sim_accept, float* logits, bool cap) {
  const Plan& p = c->p;
  const int B = c->B, R = k + 1, M = B * R;
  SetupArgs s = setup_base(c, 0);
  s.mode = SETUP_VERIFY; s.M = M; s.R = R; s.sim_accept = sim_accept;
  stamp_phase(c, s, 1);
  timed(c, SEED_PHASE_VERIFY, SEED_OP_SETUP, cap, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
  run_layers<T>(c, M, B, R, 0, p.L, SEED_PHASE_VERIFY, nullptr, cap);
  run_head<T>(c, M, c->ws<int>(p.o_vtok), 1, logits, (long long)p.V, SEED_PHASE_VERIFY, cap);
  DevState st = dev_state(c);
  timed(c, SEED_PHASE_VERIFY, SEED_OP_ACCEPT, cap, [&](const LaunchEvents*) { launch_accept(st, B, k, c->s); });
}

template <typename T>
void enqueue_round(seed_ctx* c, int k, int sim_accept, bool cap) {
  enqueue_draft<T>(c, k, nullptr, cap);
  enqueue_verify<T>(c, k, sim_accept, nullptr, cap);
}

// ---------------------------------------------------------------------------------------------
// block tables
// ---------------------------------------------------------------------------------------------
seed_status ensure_blocks(seed_ctx* c, int b, int positions) {
  const Plan& p = c->p;
  positions = std::min(positions, p.cfg.max_ctx);
  const int need = cdiv(positions, 16);
  auto& v = c->seq_blocks[b];
  if ((int)v.size() >= need) return SEED_OK;
  const int first = (int)v.size();
  while ((int)v.size() < need) {
    if (c->free_blocks.empty()) return fail(SEED_ERR_CAPACITY, "KV pool exhausted");
    v.push_back(c->free_blocks.back());
    c->free_blocks.pop_back();
    c->bt_host[(size_t)b * p.bt_stride + v.size() - 1] = v.back();
  }
  int* dst = c->ws<int>(p.o_bt) + (size_t)b * p.bt_stride + first;
  HIPCHK(hipMemcpyAsync(dst, c->bt_host.data() + (size_t)b * p.bt_stride + first, (need - first) * sizeof(int),
                        hipMemcpyHostToDevice, c->s));
  return SEED_OK;
}

void reset_blocks(seed_ctx* c) {
  const Plan& p = c->p;
  c->free_blocks.clear();
  // hand out low block ids first; sequences interleave as they grow
  for (int i = p.n_blocks - 1; i >= 1; --i) c->free_blocks.push_back(i);
  c->seq_blocks.assign(p.cfg.max_batch, {});
  std::fill(c->bt_host.begin(), c->bt_host.end(), 0);
}

seed_status read_t(seed_ctx* c) {
  std::vector<int> t(c->B);
  HIPCHK(hipMemcpyAsync(t.data(), c->ws<int>(c->p.o_t), c->B * sizeof(int), hipMemcpyDeviceToHost, c->s));
  HIPCHK(hipStreamSynchronize(c->s));
  c->t_upper = t;
  return SEED_OK;
}

// ---------------------------------------------------------------------------------------------
// weight packing
// ---------------------------------------------------------------------------------------------
struct TensorSpec {
  std::string name;
  int ndim;
  int64_t d0, d1;
};

std::vector<TensorSpec> tensor_specs(const Plan& p) {
  std::vector<TensorSpec> v;
  v.push_back({"embed", 2, p.V, p.H});
  v.push_back({"final_norm", 1, p.H, 0});
  for (int l = 0; l < p.L; ++l) {
    const std::string pre = "layers." + std::to_string(l) + ".";
    v.push_back({pre + "attn_norm", 1, p.H, 0});
    v.push_back({pre + "wq", 2, p.QD, p.H});
    v.push_back({pre + "wk", 2, p.KVD, p.H});
    v.push_back({pre + "wv", 2, p.KVD, p.H});
    v.push_back({pre + "wo", 2, p.H, p.QD});
    v.push_back({pre + "mlp_norm", 1, p.H, 0});
    v.push_back({pre + "w_gate", 2, p.F, p.H});
    v.push_back({pre + "w_up", 2, p.F, p.H});
    v.push_back({pre + "w_down", 2, p.H, p.F});
  }
  return v;
}

// packed row of source row r of a head-structured projection (RoPE partners share a tile)
int qkv_row(int r, int HD) {
  const int head = r / HD, d = r % HD, half = HD / 2;
  const int hi = d >= half, i = d % half;
  return head * HD + (i / 8) * 16 + (i % 8) + 8 * hi;
}

template <typename T>
void host_pack(const T* src, T* dst, const std::vector<int>& rows, int K) {
  const int KT = K / 32;
  for (size_t r = 0; r < rows.size(); ++r) {
    const int n = rows[r], nt = n >> 4, rr = n & 15;
    for (int k = 0; k < K; k += 8) {
      const int kt = k >> 5, kg = (k >> 3) & 3;
      std::memcpy(dst + ((size_t)nt * KT + kt) * 512 + (rr + 16 * kg) * 8, src + r * (size_t)K + k, 8 * sizeof(T));
    }
  }
}

template <typename T>
seed_status pack_into(seed_ctx* c, const seed_tensor& t, size_t dst_off, int Ntot, const std::vector<int>& rows, int K) {
  T* dst = reinterpret_cast<T*>(c->W + dst_off);
  if (t.on_device) {
    int* map = c->ws<int>(c->p.o_scratch);
    HIPCHK(hipMemcpyAsync(map, rows.data(), rows.size() * sizeof(int), hipMemcpyHostToDevice, c->s));
    launch_pack<T>(t.data, dst, map, (int)rows.size(), K, c->s);
    HIPCHK(hipGetLastError());
    HIPCHK(hipStreamSynchronize(c->s));   // the row map is reused by the next tensor
  } else {
    std::vector<T> tmp((size_t)Ntot * K);
    // keep rows of other sources that share this matrix: read back, then overwrite our rows
    HIPCHK(hipMemcpyAsync(tmp.data(), dst, tmp.size() * sizeof(T), hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    host_pack<T>(reinterpret_cast<const T*>(t.data), tmp.data(), rows, K);
    HIPCHK(hipMemcpyAsync(dst, tmp.data(), tmp.size() * sizeof(T), hipMemcpyHostToDevice, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
  }
  return SEED_OK;
}

seed_status load_one(seed_ctx* c, const seed_tensor& t, const std::string& name) {
  const Plan& p = c->p;
  const bool bf = p.cfg.dtype == SEED_BF16;
  if (name == "final_norm" || name.find("_norm") != std::string::npos) {
    size_t off;
    if (name == "final_norm") off = p.w_final_norm;
    else {
      const int l = std::atoi(name.c_str() + 7);
      off = name.find("attn_norm") != std::string::npos ? p.w_attn_norm[l] : p.w_mlp_norm[l];
    }
    float* dst = c->wf(off);
    if (t.on_device) {
      launch_to_f32(t.data, bf, dst, p.H, c->s);
      HIPCHK(hipGetLastError());
    } else {
      std::vector<float> tmp(p.H);
      for (int i = 0; i < p.H; ++i) {
        if (bf) {
          const uint32_t u = (uint32_t)reinterpret_cast<const uint16_t*>(t.data)[i] << 16;
          std::memcpy(&tmp[i], &u, 4);
        } else {
          tmp[i] = reinterpret_cast<const float*>(t.data)[i];
        }
      }
      HIPCHK(hipMemcpyAsync(dst, tmp.data(), p.H * 4, hipMemcpyHostToDevice, c->s));
    }
    HIPCHK(hipStreamSynchronize(c->s));
    return SEED_OK;
  }
  std::vector<int> rows;
  size_t off;
  int Ntot, K;
  if (name == "embed") {
    off = p.w_embed; Ntot = p.V; K = p.H;
    rows.resize(p.V);
    for (int r = 0; r < p.V; ++r) rows[r] = r;
  } else {
    const int l = std::atoi(name.c_str() + 7);
    const std::string leaf = name.substr(name.rfind('.') + 1);
    if (leaf == "wq" || leaf == "wk" || leaf == "wv") {
      off = p.w_qkv[l]; Ntot = p.QD + 2 * p.KVD; K = p.H;
      const int base = leaf == "wq" ? 0 : (leaf == "wk" ? p.QD : p.QD + p.KVD);
      const int n = leaf == "wq" ? p.QD : p.KVD;
      rows.resize(n);
      for (int r = 0; r < n; ++r) rows[r] = base + qkv_row(r, p.HD);
    } else if (leaf == "wo") {
      off = p.w_o[l]; Ntot = p.H; K = p.QD;
      rows.resize(p.H);
      for (int r = 0; r < p.H; ++r) rows[r] = r;
    } else if (leaf == "w_gate" || leaf == "w_up") {
      off = p.w_gu[l]; Ntot = 2 * p.F; K = p.H;
      rows.resize(p.F);
      const int up = leaf == "w_up";
      for (int r = 0; r < p.F; ++r) rows[r] = (r / 8) * 16 + (r % 8) + 8 * up;
    } else {
      off = p.w_down[l]; Ntot = p.H; K = p.F;
      rows.resize(p.H);
      for (int r = 0; r < p.H; ++r) rows[r] = r;
    }
  }
  return bf ? pack_into<uint16_t>(c, t, off, Ntot, rows, K) : pack_into<float>(c, t, off, Ntot, rows, K);
}

template <typename T>
seed_status do_prefill(seed_ctx* c, const std::vector<int>& tokens_packed) {
  const Plan& p = c->p;
  const int B = c->B;
  // committed tokens + state
  std::vector<int> tok_rows((size_t)B * p.tstride, 0);
  std::vector<int> t(B), len(B), limit(B), active(B, 1), drafts((size_t)B * p.dstride, 0);
  size_t o = 0;
  for (int b = 0; b < B; ++b) {
    std::copy(tokens_packed.begin() + o, tokens_packed.begin() + o + c->lens[b], tok_rows.begin() + (size_t)b * p.tstride);
    o += c->lens[b];
    t[b] = len[b] = c->lens[b];
    limit[b] = p.cfg.max_ctx;
    drafts[(size_t)b * p.dstride] = tok_rows[(size_t)b * p.tstride + c->lens[b] - 1];
  }
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_tokens), tok_rows.data(), tok_rows.size() * 4, hipMemcpyHostToDevice, c->s));
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_t), t.data(), B * 4, hipMemcpyHostToDevice, c->s));
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_len), len.data(), B * 4, hipMemcpyHostToDevice, c->s));
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_limit), limit.data(), B * 4, hipMemcpyHostToDevice, c->s));
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_active), active.data(), B * 4, hipMemcpyHostToDevice, c->s));
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_drafts), drafts.data(), drafts.size() * 4, hipMemcpyHostToDevice, c->s));
  launch_fill_u32(c->ws<int>(p.o_rounds), 0, 1, c->s);
  launch_fill_u32(c->ws<int>(p.o_stamp), 0, (long long)p.log_cap * 6, c->s);
  launch_fill_u32(c->ws<long long>(p.o_counters), 0, 4, c->s);
  HIPCHK(hipGetLastError());
  // run the full model over X[0..t-2]; X[t-1] stays pending (its cache entry would be dropped
  // by the first truncation anyway, and causality makes the kept entries identical)
  for (int b = 0; b < B; ++b) {
    const int n = c->lens[b] - 1;
    for (int s0 = 0; s0 < n; s0 += PREFILL_ROWS) {
      const int M = std::min(PREFILL_ROWS, n - s0);
      SetupArgs s = setup_base(c, 0);
      s.mode = SETUP_PREFILL; s.M = M; s.R = M; s.pf_seq = b; s.pf_pos0 = s0;
      timed(c, SEED_PHASE_PREFILL, SEED_OP_SETUP, false, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
      run_layers<T>(c, M, 1, M, 0, p.L, SEED_PHASE_PREFILL,
                    c->ws<int>(p.o_bt) + (size_t)b * p.bt_stride, false, nullptr, false, s0);
    }
  }
  HIPCHK(hipGetLastError());
  return SEED_OK;
}

// Bytes of the block-causal pass's own cache: the decoder layers' keys/values by position.
// Bytes of the drafting-objective pass's own cache (decoder layers, `blocks` 16-position blocks
// per layer, indexed by position).
size_t spec_cache_bytes(const Plan& p, int blocks) {
  return align256((size_t)std::max(1, p.L - p.LD) * blocks * 2 * p.NKV * 16 * p.HD * p.esize);
}
size_t spec_kv_bytes(const Plan& p) { return spec_cache_bytes(p, p.blocks_per_seq); }

// Decoder rows of the speculative drafting objective (Algorithm 1) over positions 0..n-2, in
// passes of PREFILL_ROWS rows; the deep cache holds the prefill of the same sequence.
template <typename T>
seed_status do_spec(seed_ctx* c, int n, int block, void* skv, int skv_blocks, float* logits) {
  const Plan& p = c->p;
  const SpecPass sp{skv, skv_blocks, block};
  const int rows = n - 1;
  // the pass's own cache starts as zeros: a 16-position tile of it that holds a visible position
  // is contracted whole, and the positions this pass has not written yet (probability 0) must be
  // finite, which the caller's buffer need not be
  launch_fill_u32(skv, 0, (long long)(spec_cache_bytes(p, skv_blocks) / 4), c->s);
  for (int s0 = 0; s0 < rows; s0 += PREFILL_ROWS) {
    const int M = std::min(PREFILL_ROWS, rows - s0);
    SetupArgs s = setup_base(c, p.LD);
    s.mode = SETUP_SPEC; s.M = M; s.R = M; s.pf_seq = 0; s.pf_pos0 = s0;
    timed(c, SEED_PHASE_SPEC, SEED_OP_SETUP, false, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
    run_layers<T>(c, M, 1, M, p.LD, p.L, SEED_PHASE_SPEC, c->ws<int>(p.o_bt), false, &sp, false, s0);
    run_head<T>(c, M, nullptr, 1, logits + (size_t)s0 * p.V, (long long)p.V, SEED_PHASE_SPEC, false);
  }
  HIPCHK(hipGetLastError());
  return SEED_OK;
}

// Medians over rounds [0, rounds) of the stamped phase times (ms): verification (column 1 to 2)
// and drafting (column 0 to 1, divided by steps; 0 when the rounds draft nothing). Rounds whose
// stamps are missing or out of order (a phase not run) are skipped.
seed_status phase_medians(seed_ctx* c, int64_t rounds, int steps, double* verify_ms, double* draft_ms) {
  *verify_ms = 0.0;
  *draft_ms = 0.0;
  const int64_t n = std::min<int64_t>(rounds, c->p.log_cap);
  if (n <= 0) return SEED_OK;
  int dev = 0, khz = 0;
  HIPCHK(hipGetDevice(&dev));
  HIPCHK(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
  if (khz <= 0) return fail(SEED_ERR_HIP, "device reports no constant clock rate");
  std::vector<long long> t((size_t)n * 3);
  HIPCHK(hipMemcpy(t.data(), c->ws<long long>(c->p.o_stamp), t.size() * 8, hipMemcpyDeviceToHost));
  std::vector<double> v, d;
  for (int64_t r = 0; r < n; ++r) {
    const long long a = t[r * 3], b = t[r * 3 + 1], e = t[r * 3 + 2];
    if (e > b && b > 0) v.push_back((double)(e - b) / khz);
    if (steps > 0 && b > a && a > 0) d.push_back((double)(b - a) / khz / steps);
  }
  auto median = [](std::vector<double>& x) {
    if (x.empty()) return 0.0;
    std::sort(x.begin(), x.end());
    const size_t m = x.size() / 2;
    return x.size() % 2 ? x[m] : 0.5 * (x[m - 1] + x[m]);
  };
  *verify_ms = median(v);
  *draft_ms = median(d);
  return SEED_OK;
}

seed_status check_ready(seed_ctx* c) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  if (!c->weights_ok) {
    const auto specs = tensor_specs(c->p);
    for (size_t i = 0; i < specs.size(); ++i)
      if (!c->loaded[i]) return fail(SEED_ERR_STATE, "weights not loaded: missing tensor '" + specs[i].name + "'");
  }
  return SEED_OK;
}

seed_status check_prompts(seed_ctx* c, int32_t B, const int32_t* tokens, const int32_t* lens, int extra,
                          std::vector<int>& packed) {
  const Plan& p = c->p;
  if (B < 1 || B > p.cfg.max_batch) return fail(SEED_ERR_CAPACITY, "batch must be in [1, max_batch]");
  if (!tokens || !lens) return fail(SEED_ERR_ARG, "tokens and lens must not be NULL");
  size_t total = 0;
  for (int b = 0; b < B; ++b) {
    if (lens[b] < 1) return fail(SEED_ERR_ARG, "every prompt needs at least one token");
    if ((int64_t)lens[b] + extra > p.cfg.max_ctx)
      return fail(SEED_ERR_CAPACITY, "prompt " + std::to_string(b) + " does not fit max_ctx");
    total += lens[b];
  }
  packed.assign(tokens, tokens + total);
  for (size_t i = 0; i < total; ++i)
    if (packed[i] < 0 || packed[i] >= p.V) return fail(SEED_ERR_ARG, "token id out of range at " + std::to_string(i));
  return SEED_OK;
}

seed_status start_sequences(seed_ctx* c, int32_t B, const int32_t* lens, int extra) {
  c->B = B;
  c->lens.assign(lens, lens + B);
  c->t_upper = c->lens;
  c->drafts_k = -1;
  c->prefilled = false;
  reset_blocks(c);
  for (int b = 0; b < B; ++b) {
    seed_status st = ensure_blocks(c, b, lens[b] + extra);
    if (st != SEED_OK) return st;
  }
  return SEED_OK;
}

// Captures the launches fn() enqueues on the context's stream into an executable graph.
template <typename F>
seed_status capture_graph(seed_ctx* c, F&& fn, hipGraphExec_t* ex) {
  hipGraph_t g = nullptr;
  HIPCHK(hipStreamBeginCapture(c->s, hipStreamCaptureModeThreadLocal));
  fn();
  HIPCHK(hipStreamEndCapture(c->s, &g));
  const hipError_t e = hipGraphInstantiate(ex, g, nullptr, nullptr, 0);
  hipGraphDestroy(g);
  if (e != hipSuccess) return fail(SEED_ERR_HIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(e));
  return SEED_OK;
}

template <typename T>
seed_status run_rounds(seed_ctx* c, int k, int n, bool use_graph) {
  if (!use_graph) {
    for (int r = 0; r < n; ++r) enqueue_round<T>(c, k, c->sim_accept, false);
    HIPCHK(hipGetLastError());
    return SEED_OK;
  }
  const auto key = std::make_tuple(c->B, k, c->sim_accept, c->eos);
  auto it = c->graphs.find(key);
  if (it == c->graphs.end()) {
    hipGraphExec_t ex;
    seed_status st = capture_graph(c, [&] { enqueue_round<T>(c, k, c->sim_accept, true); }, &ex);
    if (st != SEED_OK) return st;
    it = c->graphs.emplace(key, ex).first;
  }
  for (int r = 0; r < n; ++r) HIPCHK(hipGraphLaunch(it->second, c->s));
  return SEED_OK;
}

// Tree-based verification of one sequence's packed draft tree (the tree arrays in the workspace):
// node rows through every layer with the tree attention mask, the LM head (logits optional),
// then tree acceptance, commit and the move of an accepted leaf's cache entries.
template <typename T>
void enqueue_verify_tree(seed_ctx* c, int n, float* logits, bool cap) {
  const Plan& p = c->p;
  SetupArgs s = setup_base(c, 0);
  s.mode = SETUP_TREE; s.M = n; s.R = n; s.sim_accept = c->sim_accept;
  s.tree_tok = c->ws<int>(p.o_tree);
  s.tree_depth = c->ws<int>(p.o_tree) + 2 * MAX_ROWS;
  stamp_phase(c, s, 1);
  timed(c, SEED_PHASE_VERIFY, SEED_OP_SETUP, cap, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
  run_layers<T>(c, n, 1, n, 0, p.L, SEED_PHASE_VERIFY, nullptr, cap, nullptr, true);
  run_head<T>(c, n, c->ws<int>(p.o_vtok), 1, logits, (long long)p.V, SEED_PHASE_VERIFY, cap);
  DevState st = dev_state(c);
  timed(c, SEED_PHASE_VERIFY, SEED_OP_ACCEPT, cap, [&](const LaunchEvents*) {
    launch_accept_tree(st, n, c->ws<int>(p.o_tree), c->ws<int>(p.o_tree) + MAX_ROWS, c->ws<int>(p.o_tree) + 2 * MAX_ROWS,
                       c->ws<int>(p.o_tree_out), c->KV, p.L, p.n_blocks, p.NKV, p.HD, p.esize, c->ws<int>(p.o_bt),
                       c->hstat_dev, c->s);
  });
}

// B: the number of sequences the call runs (the current state's for seed_draft_tree and
// seed_verify_tree, 1 for seed_generate_tree, which starts a new state)
seed_status check_tree_opts(const seed_ctx* c, const seed_tree_opts* o, int B) {
  const Plan& p = c->p;
  if (!o) return fail(SEED_ERR_ARG, "tree options must not be NULL");
  if (o->max_depth < 1 || o->max_depth > p.cfg.max_draft)
    return fail(SEED_ERR_ARG, "max_depth must be in [1, max_draft]");
  if (o->max_nodes < o->max_depth + 1 || o->max_nodes > MAX_ROWS)
    return fail(SEED_ERR_ARG, "max_nodes must be in [max_depth + 1, 64]");
  if (o->n_levels < 0 || o->n_levels > 4) return fail(SEED_ERR_ARG, "n_levels must be in [0, 4]");
  for (int j = 0; j < o->n_levels; ++j) {
    if (o->k[j] < 1 || o->k[j] > TOPK_MAX) return fail(SEED_ERR_ARG, "every fan-out must be in [1, 16]");
    if (j > 0 && !(o->thr[j] < o->thr[j - 1])) return fail(SEED_ERR_ARG, "thresholds must decrease");
  }
  if (o->k_rest < 1 || o->k_rest > TOPK_MAX) return fail(SEED_ERR_ARG, "k_rest must be in [1, 16]");
  if (!(o->tau >= 0.f && o->tau <= 1.f)) return fail(SEED_ERR_ARG, "tau must be in [0, 1]");
  if (B != 1) return fail(SEED_ERR_UNSUPPORTED, "dynamic drafting runs one sequence (B = 1)");
  if (p.V < TOPK_MAX || p.V > TOPK_PARTS * 64 * 16)
    return fail(SEED_ERR_UNSUPPORTED, "dynamic drafting needs 16 <= vocab <= 262144");
  return SEED_OK;
}

TreeDraftArgs tree_args(seed_ctx* c, const seed_tree_opts& o, int step, const float* logits) {
  const Plan& p = c->p;
  TreeDraftArgs a;
  std::memset(&a, 0, sizeof(a));
  a.logits = logits;
  a.V = p.V;
  a.chunk = tree_topk_chunk(p.V);
  a.step = step;
  float* tk = c->ws<float>(p.o_topk);
  a.pval = tk;
  a.pidx = reinterpret_cast<int*>(tk + TOPK_PARTS * TOPK_MAX);
  a.pmax = tk + 2 * TOPK_PARTS * TOPK_MAX;
  a.psum = a.pmax + TOPK_PARTS;
  a.tau = o.tau;
  a.n_levels = o.n_levels;
  a.k_rest = a.k_max = o.k_rest;
  for (int j = 0; j < o.n_levels; ++j) {
    a.thr[j] = o.thr[j];
    a.kk[j] = o.k[j];
    a.k_max = std::max(a.k_max, o.k[j]);
  }
  a.max_depth = o.max_depth;
  a.max_nodes = o.max_nodes;
  int* td = c->ws<int>(p.o_tdraft);
  a.cand = td;
  a.kcnt = td + TREE_MAX_STEPS * TOPK_MAX;
  a.p0 = reinterpret_cast<float*>(a.kcnt + TREE_MAX_STEPS);
  a.dstate = a.kcnt + 2 * TREE_MAX_STEPS;
  a.drafts = c->ws<int>(p.o_drafts);
  a.tree = c->ws<int>(p.o_tree);
  a.rounds = c->ws<int>(p.o_rounds);
  a.hstat = c->hstat_dev;
  return a;
}

// Drafting step i of dynamic drafting: the decoder-only step of Algorithm 2 (Eq. 5) from the
// chain token X_draft[i-1], its logits, then the top-1 probability, fan-out, candidates and stop.
template <typename T>
void enqueue_tree_step(seed_ctx* c, const seed_tree_opts& o, int step, float* logits, bool cap) {
  const Plan& p = c->p;
  SetupArgs s = setup_base(c, p.LD);
  s.mode = SETUP_DRAFT; s.M = 1; s.R = 1; s.step = step;
  if (step == 1) stamp_phase(c, s, 0);
  timed(c, SEED_PHASE_DRAFT, SEED_OP_SETUP, cap, [&](const LaunchEvents*) { launch_setup<T>(s, c->s); });
  run_layers<T>(c, 1, 1, 1, p.LD, p.L, SEED_PHASE_DRAFT, nullptr, cap);
  run_head<T>(c, 1, nullptr, p.dstride, logits, (long long)p.V, SEED_PHASE_DRAFT, cap);
  const TreeDraftArgs a = tree_args(c, o, step, logits);
  timed(c, SEED_PHASE_DRAFT, SEED_OP_TOPK, cap, [&](const LaunchEvents*) { launch_tree_topk(a, c->s); });
}

template <typename T>
seed_status launch_tree_step(seed_ctx* c, const seed_tree_opts& o, int step, bool use_graph) {
  float* lg = c->ws<float>(c->p.o_dlog);
  if (!use_graph) {
    enqueue_tree_step<T>(c, o, step, lg, false);
    HIPCHK(hipGetLastError());
    return SEED_OK;
  }
  if (std::memcmp(&c->tree_key, &o, sizeof(o)) != 0) {
    for (auto& kv : c->tree_step_graphs) HIPCHK(hipGraphExecDestroy(kv.second));
    c->tree_step_graphs.clear();
    c->tree_key = o;
  }
  auto it = c->tree_step_graphs.find(step);
  if (it == c->tree_step_graphs.end()) {
    hipGraphExec_t ex;
    seed_status st = capture_graph(c, [&] { enqueue_tree_step<T>(c, o, step, lg, true); }, &ex);
    if (st != SEED_OK) return st;
    it = c->tree_step_graphs.emplace(step, ex).first;
  }
  HIPCHK(hipGraphLaunch(it->second, c->s));
  return SEED_OK;
}

template <typename T>
seed_status launch_tree_verify(seed_ctx* c, int n, bool use_graph) {
  if (!use_graph) {
    enqueue_verify_tree<T>(c, n, nullptr, false);
    HIPCHK(hipGetLastError());
    return SEED_OK;
  }
  const auto key = std::make_tuple(n, c->eos, c->sim_accept);
  auto it = c->tree_verify_graphs.find(key);
  if (it == c->tree_verify_graphs.end()) {
    hipGraphExec_t ex;
    seed_status st = capture_graph(c, [&] { enqueue_verify_tree<T>(c, n, nullptr, true); }, &ex);
    if (st != SEED_OK) return st;
    it = c->tree_verify_graphs.emplace(key, ex).first;
  }
  HIPCHK(hipGraphLaunch(it->second, c->s));
  return SEED_OK;
}

// Busy-wait for an event (the host reacts within microseconds; the stream keeps running the
// work queued behind it).
seed_status spin_event(hipEvent_t e) {
  for (;;) {
    const hipError_t r = hipEventQuery(e);
    if (r == hipSuccess) return SEED_OK;
    if (r != hipErrorNotReady) return fail(SEED_ERR_HIP, std::string("hipEventQuery: ") + hipGetErrorString(r));
  }
}

int read_host_int(const int* p) { return __atomic_load_n(p, __ATOMIC_ACQUIRE); }

// Dynamic drafting + tree verification rounds of the single sequence until it is no longer live.
// Pipelined: drafting step i+1 is queued before the host learns whether step i stopped (a stopped
// round turns it into a no-op after its decoder pass), and the next round's first step before the
// host learns whether this round finished the sequence; the host reads the kernels' pinned status
// after each event, so the GPU never waits for it.
template <typename T>
seed_status tree_rounds(seed_ctx* c, const seed_tree_opts& o, bool use_graph, int round0, int* rounds_run) {
  std::vector<hipEvent_t> ev(TREE_MAX_STEPS + 2, nullptr);
  seed_status st = SEED_OK;
  for (auto& e : ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) st = fail(SEED_ERR_HIP, "hipEventCreate failed");
  auto done = [&](seed_status r) {
    for (auto& e : ev)
      if (e) hipEventDestroy(e);
    return r;
  };
  if (st != SEED_OK) return done(st);
  const int D = o.max_depth;
  hipEvent_t ev_v = ev[TREE_MAX_STEPS + 1];
  int r = round0;
  c->hstat[0] = c->hstat[4] = -1;
  st = launch_tree_step<T>(c, o, 1, use_graph);
  if (st != SEED_OK) return done(st);
  if (hipEventRecord(ev[1], c->s) != hipSuccess) return done(fail(SEED_ERR_HIP, "hipEventRecord failed"));
  for (;;) {
    int n = -1;
    for (int i = 1;; ++i) {
      if (i < D) {
        st = launch_tree_step<T>(c, o, i + 1, use_graph);
        if (st != SEED_OK) return done(st);
        if (hipEventRecord(ev[i + 1], c->s) != hipSuccess) return done(fail(SEED_ERR_HIP, "hipEventRecord failed"));
      }
      st = spin_event(ev[i]);
      if (st != SEED_OK) return done(st);
      if (read_host_int(c->hstat) == r) {
        n = read_host_int(c->hstat + 1);
        break;
      }
      if (i >= D) return done(fail(SEED_ERR_HIP, "drafting did not stop at max_depth"));
    }
    if (n < 1 || n > o.max_nodes) return done(fail(SEED_ERR_HIP, "drafted tree size out of range"));
    st = launch_tree_verify<T>(c, n, use_graph);
    if (st != SEED_OK) return done(st);
    if (hipEventRecord(ev_v, c->s) != hipSuccess) return done(fail(SEED_ERR_HIP, "hipEventRecord failed"));
    st = launch_tree_step<T>(c, o, 1, use_graph);   // the next round's first step
    if (st != SEED_OK) return done(st);
    if (hipEventRecord(ev[1], c->s) != hipSuccess) return done(fail(SEED_ERR_HIP, "hipEventRecord failed"));
    st = spin_event(ev_v);
    if (st != SEED_OK) return done(st);
    ++r;
    if (read_host_int(c->hstat + 4) != r) return done(fail(SEED_ERR_HIP, "tree acceptance status missing"));
    if (!read_host_int(c->hstat + 6)) break;
  }
  // let the speculative first step of the round that will not run finish
  if (hipStreamSynchronize(c->s) != hipSuccess) return done(fail(SEED_ERR_HIP, "hipStreamSynchronize failed"));
  *rounds_run = r - round0;
  return done(SEED_OK);
}

}  // namespace

// =============================================================================================
// C ABI
// =============================================================================================
extern "C" {

const char* seed_last_error(void) { return g_err.c_str(); }

seed_status seed_arena_bytes(const seed_config* cfg, size_t* weight_bytes, size_t* kv_bytes, size_t* workspace_bytes) {
  seed_status st = validate(cfg);
  if (st != SEED_OK) return st;
  if (!weight_bytes || !kv_bytes || !workspace_bytes) return fail(SEED_ERR_ARG, "output pointers must not be NULL");
  const Plan p = make_plan(*cfg);
  *weight_bytes = p.w_total;
  *kv_bytes = p.kv_total;
  *workspace_bytes = p.ws_total;
  return SEED_OK;
}

seed_status seed_create(const seed_config* cfg, void* hip_stream, void* weight_arena, void* kv_pool, void* workspace,
                        seed_ctx** out) {
  seed_status st = validate(cfg);
  if (st != SEED_OK) return st;
  if (!out) return fail(SEED_ERR_ARG, "out must not be NULL");
  *out = nullptr;
  if (!weight_arena || !kv_pool || !workspace) return fail(SEED_ERR_ARG, "buffers must not be NULL");
  if (((uintptr_t)weight_arena | (uintptr_t)kv_pool | (uintptr_t)workspace) & 255)
    return fail(SEED_ERR_ARG, "buffers must be 256-byte aligned");
  HIPCHK(configure_kernels(cfg->dtype == SEED_BF16));
  seed_ctx* c = new seed_ctx();
  c->p = make_plan(*cfg);
  c->s = reinterpret_cast<hipStream_t>(hip_stream);
  c->W = reinterpret_cast<char*>(weight_arena);
  c->KV = reinterpret_cast<char*>(kv_pool);
  c->WS = reinterpret_cast<char*>(workspace);
  const Plan& p = c->p;
  c->loaded.assign(tensor_specs(p).size(), false);
  c->bt_host.assign((size_t)cfg->max_batch * p.bt_stride, 0);
  reset_blocks(c);
  // clear the KV pool (finite values everywhere, block 0 stays zero) and the workspace
  launch_fill_u32(c->KV, 0, (long long)(p.kv_total / 4), c->s);
  launch_fill_u32(c->WS, 0, (long long)(p.ws_total / 4), c->s);
  // rotary tables, angles in double precision
  const int half = p.HD / 2;
  std::vector<float> cs((size_t)cfg->max_ctx * half), sn((size_t)cfg->max_ctx * half);
  for (int pos = 0; pos < cfg->max_ctx; ++pos)
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)cfg->rope_base, -2.0 * i / p.HD);
      const double ang = (double)pos * inv;
      cs[(size_t)pos * half + i] = (float)std::cos(ang);
      sn[(size_t)pos * half + i] = (float)std::sin(ang);
    }
  hipError_t e = hipMemcpyAsync(c->wf(p.w_rope_cos), cs.data(), cs.size() * 4, hipMemcpyHostToDevice, c->s);
  if (e == hipSuccess) e = hipMemcpyAsync(c->wf(p.w_rope_sin), sn.data(), sn.size() * 4, hipMemcpyHostToDevice, c->s);
  if (e == hipSuccess) e = hipStreamSynchronize(c->s);
  if (e == hipSuccess) e = hipHostMalloc((void**)&c->hstat, 256, hipHostMallocCoherent);
  if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&c->hstat_dev, c->hstat, 0);
  if (e == hipSuccess) {
    // once per device, with the device current: the address of this GPU's `scratch`
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) {
      std::lock_guard<std::mutex> lock(g_scratch_mu);
      auto it = g_scratch_addr.find(dev);
      if (it == g_scratch_addr.end()) {
        char* ptr = nullptr;
        e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
        if (e == hipSuccess && ptr) it = g_scratch_addr.emplace(dev, ptr).first;
      }
      if (e == hipSuccess && it != g_scratch_addr.end()) c->scratch_dev = it->second;
    }
  }
  if (e != hipSuccess) {
    if (c->hstat) hipHostFree(c->hstat);
    delete c;
    return fail(SEED_ERR_HIP, std::string("seed_create: ") + hipGetErrorString(e));
  }
  *out = c;
  return SEED_OK;
}

seed_status seed_load_weights(seed_ctx* c, const seed_tensor* tensors, int32_t n) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  if (!tensors || n < 0) return fail(SEED_ERR_ARG, "tensors must not be NULL");
  const Plan& p = c->p;
  const auto specs = tensor_specs(p);
  std::map<std::string, int> index;
  for (size_t i = 0; i < specs.size(); ++i) index[specs[i].name] = (int)i;
  std::vector<int> which(n);
  std::vector<bool> seen(specs.size(), false);
  for (int i = 0; i < n; ++i) {
    const seed_tensor& t = tensors[i];
    if (!t.name) return fail(SEED_ERR_ARG, "tensor " + std::to_string(i) + " has no name");
    auto it = index.find(t.name);
    if (it == index.end()) return fail(SEED_ERR_ARG, std::string("unknown tensor '") + t.name + "'");
    const TensorSpec& s = specs[it->second];
    if (seen[it->second]) return fail(SEED_ERR_ARG, std::string("duplicate tensor '") + t.name + "'");
    seen[it->second] = true;
    if (!t.data) return fail(SEED_ERR_ARG, std::string("tensor '") + t.name + "' has no data");
    if (t.dtype != p.cfg.dtype) return fail(SEED_ERR_ARG, std::string("tensor '") + t.name + "' has the wrong dtype");
    if (t.ndim != s.ndim || t.shape[0] != s.d0 || (s.ndim == 2 && t.shape[1] != s.d1))
      return fail(SEED_ERR_ARG, std::string("tensor '") + t.name + "' has the wrong shape");
    which[i] = it->second;
  }
  for (int i = 0; i < n; ++i) {
    seed_status st = load_one(c, tensors[i], specs[which[i]].name);
    if (st != SEED_OK) return st;
    c->loaded[which[i]] = true;
  }
  c->weights_ok = std::all_of(c->loaded.begin(), c->loaded.end(), [](bool b) { return b; });
  return SEED_OK;
}

seed_status seed_prefill(seed_ctx* c, int32_t B, const int32_t* tokens, const int32_t* lens) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  std::vector<int> packed;
  st = check_prompts(c, B, tokens, lens, c->p.cfg.max_draft + 1, packed);
  if (st != SEED_OK) return st;
  st = start_sequences(c, B, lens, c->p.cfg.max_draft + 1);
  if (st != SEED_OK) return st;
  c->sim_accept = -1;
  c->eos = -1;
  st = c->p.cfg.dtype == SEED_BF16 ? do_prefill<uint16_t>(c, packed) : do_prefill<float>(c, packed);
  if (st != SEED_OK) return st;
  HIPCHK(hipStreamSynchronize(c->s));
  c->prefilled = true;
  return SEED_OK;
}

static seed_status check_step(seed_ctx* c, int32_t k, int64_t growth) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (!c->prefilled) return fail(SEED_ERR_STATE, "call seed_prefill first");
  if (k < 0 || k > c->p.cfg.max_draft) return fail(SEED_ERR_ARG, "k must be in [0, max_draft]");
  for (int b = 0; b < c->B; ++b)
    if ((int64_t)c->t_upper[b] + growth > c->p.cfg.max_ctx)
      return fail(SEED_ERR_CAPACITY, "sequence " + std::to_string(b) + " would pass max_ctx");
  for (int b = 0; b < c->B; ++b) {
    st = ensure_blocks(c, b, (int)std::min<int64_t>(c->p.cfg.max_ctx, c->t_upper[b] + growth));
    if (st != SEED_OK) return st;
  }
  return SEED_OK;
}

seed_status seed_draft(seed_ctx* c, int32_t k, int32_t* drafts, float* logits) {
  seed_status st = check_step(c, k, (int64_t)k + 1);
  if (st != SEED_OK) return st;
  if (k < 1) return fail(SEED_ERR_ARG, "seed_draft needs k >= 1");
  if (c->p.cfg.dtype == SEED_BF16) enqueue_draft<uint16_t>(c, k, logits, false);
  else enqueue_draft<float>(c, k, logits, false);
  HIPCHK(hipGetLastError());
  if (drafts) {
    std::vector<int> d((size_t)c->B * c->p.dstride);
    HIPCHK(hipMemcpyAsync(d.data(), c->ws<int>(c->p.o_drafts), d.size() * 4, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    for (int b = 0; b < c->B; ++b)
      for (int i = 0; i < k; ++i) drafts[b * k + i] = d[(size_t)b * c->p.dstride + 1 + i];
  }
  c->drafts_k = k;
  return SEED_OK;
}

seed_status seed_verify(seed_ctx* c, int32_t k, const int32_t* drafts, int32_t* n_accept, int32_t* bonus, float* logits) {
  seed_status st = check_step(c, k, (int64_t)k + 1);
  if (st != SEED_OK) return st;
  const Plan& p = c->p;
  if (drafts) {
    for (int i = 0; i < c->B * k; ++i)
      if (drafts[i] < 0 || drafts[i] >= p.V) return fail(SEED_ERR_ARG, "draft token out of range");
    for (int b = 0; b < c->B; ++b)
      if (k > 0)
        HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_drafts) + (size_t)b * p.dstride + 1, drafts + (size_t)b * k, k * 4,
                              hipMemcpyHostToDevice, c->s));
  } else if (k > 0 && c->drafts_k != k) {
    return fail(SEED_ERR_STATE, "no drafts of length k since the last commit (call seed_draft or pass drafts)");
  }
  if (p.cfg.dtype == SEED_BF16) enqueue_verify<uint16_t>(c, k, -1, logits, false);
  else enqueue_verify<float>(c, k, -1, logits, false);
  HIPCHK(hipGetLastError());
  std::vector<int> na(c->B), bo(c->B);
  HIPCHK(hipMemcpyAsync(na.data(), c->ws<int>(p.o_nacc), c->B * 4, hipMemcpyDeviceToHost, c->s));
  HIPCHK(hipMemcpyAsync(bo.data(), c->ws<int>(p.o_bonus), c->B * 4, hipMemcpyDeviceToHost, c->s));
  st = read_t(c);
  if (st != SEED_OK) return st;
  if (n_accept) std::copy(na.begin(), na.end(), n_accept);
  if (bonus) std::copy(bo.begin(), bo.end(), bonus);
  c->drafts_k = -1;
  return SEED_OK;
}

seed_status seed_rounds(seed_ctx* c, int32_t k, int32_t n_rounds, int32_t use_graph) {
  if (n_rounds < 0) return fail(SEED_ERR_ARG, "n_rounds must be >= 0");
  if (c && c->prefilled) {
    // refresh the upper bounds if the worst case would not fit
    for (int b = 0; b < c->B; ++b)
      if ((int64_t)c->t_upper[b] + (int64_t)n_rounds * (k + 1) + k + 1 > c->p.cfg.max_ctx) {
        seed_status st = read_t(c);
        if (st != SEED_OK) return st;
        break;
      }
  }
  seed_status st = check_step(c, k, (int64_t)n_rounds * (k + 1) + k + 1);
  if (st != SEED_OK) return st;
  st = c->p.cfg.dtype == SEED_BF16 ? run_rounds<uint16_t>(c, k, n_rounds, use_graph != 0)
                                   : run_rounds<float>(c, k, n_rounds, use_graph != 0);
  if (st != SEED_OK) return st;
  for (int b = 0; b < c->B; ++b) c->t_upper[b] += n_rounds * (k + 1);
  c->drafts_k = -1;
  return SEED_OK;
}

seed_status seed_generate(seed_ctx* c, int32_t B, const int32_t* tokens, const int32_t* lens, const seed_gen_opts* opts,
                          int32_t* out, int32_t* counts, seed_stats* stats) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (!opts || !out || !counts) return fail(SEED_ERR_ARG, "opts, out and counts must not be NULL");
  const Plan& p = c->p;
  const int k = opts->k;
  if (k < 0 || k > p.cfg.max_draft) return fail(SEED_ERR_ARG, "k must be in [0, max_draft]");
  if (opts->max_new < 1) return fail(SEED_ERR_ARG, "max_new must be >= 1");
  if (opts->sim_accept < -1 || opts->sim_accept > k) return fail(SEED_ERR_ARG, "sim_accept must be -1 or in [0, k]");
  if (opts->sim_accept >= 0 && !opts->forced_trace) return fail(SEED_ERR_ARG, "sim_accept needs forced_trace");
  if (opts->eos_id < -1 || opts->eos_id >= p.V) return fail(SEED_ERR_ARG, "eos_id out of range");
  std::vector<int> packed;
  // a finished sequence keeps running rounds at its final position: room for 2k+1 more
  const int extra = opts->max_new + 2 * k + 1;
  st = check_prompts(c, B, tokens, lens, extra, packed);
  if (st != SEED_OK) return st;
  if (opts->sim_accept >= 0)
    for (int64_t i = 0; i < (int64_t)B * opts->max_new; ++i)
      if (opts->forced_trace[i] < 0 || opts->forced_trace[i] >= p.V)
        return fail(SEED_ERR_ARG, "forced_trace token out of range at " + std::to_string(i));
  // every argument is checked: from here on the previous decoding state is replaced
  st = start_sequences(c, B, lens, extra);
  if (st != SEED_OK) return st;
  c->eos = opts->eos_id;
  c->sim_accept = -1;

  CallEvents ce;
  HIPCHK(ce.create());
  hipEvent_t e0 = ce.e[0], e1 = ce.e[1], e2 = ce.e[2];
  HIPCHK(hipEventRecord(e0, c->s));
  st = p.cfg.dtype == SEED_BF16 ? do_prefill<uint16_t>(c, packed) : do_prefill<float>(c, packed);
  if (st != SEED_OK) return st;
  c->prefilled = true;
  // limits and the forced trace
  std::vector<int> limit(B);
  for (int b = 0; b < B; ++b) limit[b] = lens[b] + opts->max_new;
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_limit), limit.data(), B * 4, hipMemcpyHostToDevice, c->s));
  if (opts->sim_accept >= 0) {
    std::vector<int> tr((size_t)B * p.tstride, 0);
    for (int b = 0; b < B; ++b)
      for (int i = 0; i < opts->max_new; ++i)
        tr[(size_t)b * p.tstride + lens[b] + i] = opts->forced_trace[(size_t)b * opts->max_new + i];
    HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_trace), tr.data(), tr.size() * 4, hipMemcpyHostToDevice, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    c->sim_accept = opts->sim_accept;
  }
  HIPCHK(hipEventRecord(e1, c->s));
  // rounds: every round commits >= 1 token per live sequence; launch the number of rounds the
  // observed tokens-per-round rate predicts, then re-check
  double rate = k + 1;
  std::vector<int> t(B), active(B), t0(B);
  while (true) {
    HIPCHK(hipMemcpyAsync(t.data(), c->ws<int>(p.o_t), B * 4, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipMemcpyAsync(active.data(), c->ws<int>(p.o_active), B * 4, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    int rem = 0, slowest = -1;
    for (int b = 0; b < B; ++b)
      if (active[b] && limit[b] - t[b] > rem) { rem = limit[b] - t[b]; slowest = b; }
    if (slowest < 0) break;
    const int n = std::max(1, (int)std::ceil(rem / rate));
    t0 = t;
    st = p.cfg.dtype == SEED_BF16 ? run_rounds<uint16_t>(c, k, n, opts->use_graph != 0)
                                  : run_rounds<float>(c, k, n, opts->use_graph != 0);
    if (st != SEED_OK) return st;
    HIPCHK(hipMemcpyAsync(t.data(), c->ws<int>(p.o_t), B * 4, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    const double gained = t[slowest] - t0[slowest];
    rate = std::max(1.0, std::min((double)(k + 1), gained / n));
  }
  HIPCHK(hipEventRecord(e2, c->s));
  HIPCHK(hipEventSynchronize(e2));
  // outputs
  std::vector<int> tok((size_t)B * p.tstride);
  HIPCHK(hipMemcpy(tok.data(), c->ws<int>(p.o_tokens), tok.size() * 4, hipMemcpyDeviceToHost));
  HIPCHK(hipMemcpy(t.data(), c->ws<int>(p.o_t), B * 4, hipMemcpyDeviceToHost));
  c->t_upper = t;
  for (int b = 0; b < B; ++b) {
    const int n = std::min(t[b] - lens[b], opts->max_new);
    counts[b] = n;
    for (int i = 0; i < opts->max_new; ++i) out[(size_t)b * opts->max_new + i] = i < n ? tok[(size_t)b * p.tstride + lens[b] + i] : -1;
  }
  if (stats) {
    int rounds = 0;
    long long cnt[2];
    HIPCHK(hipMemcpy(&rounds, c->ws<int>(p.o_rounds), 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(cnt, c->ws<long long>(p.o_counters), 16, hipMemcpyDeviceToHost));
    stats->rounds = rounds;
    stats->drafted = cnt[0];
    stats->accepted = cnt[1];
    float ms1 = 0.f, ms2 = 0.f;
    HIPCHK(hipEventElapsedTime(&ms1, e0, e1));
    HIPCHK(hipEventElapsedTime(&ms2, e1, e2));
    stats->prefill_ms = ms1;
    stats->decode_ms = ms2;
    if (stats->n_accept_log && stats->n_accept_log_cap > 0) {
      const int64_t rows = std::min<int64_t>({(int64_t)rounds, stats->n_accept_log_cap, (int64_t)p.log_cap});
      HIPCHK(hipMemcpy(stats->n_accept_log, c->ws<int>(p.o_log), rows * B * 4, hipMemcpyDeviceToHost));
    }
    st = phase_medians(c, rounds, k, &stats->verify_ms, &stats->draft_ms);
    if (st != SEED_OK) return st;
  }
  c->sim_accept = -1;
  c->drafts_k = -1;
  return SEED_OK;
}

seed_status seed_verify_tree(seed_ctx* c, int32_t n, const int32_t* tokens, const int32_t* parents, int32_t* path,
                             int32_t* path_len, int32_t* bonus, float* logits) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (!c->prefilled) return fail(SEED_ERR_STATE, "call seed_prefill first");
  if (c->B != 1) return fail(SEED_ERR_UNSUPPORTED, "tree verification runs one sequence (B = 1)");
  const Plan& p = c->p;
  if (n < 1 || n > MAX_ROWS) return fail(SEED_ERR_ARG, "the tree needs 1..64 nodes");
  if (!tokens || !parents) return fail(SEED_ERR_ARG, "tokens and parents must not be NULL");
  // shape: node 0 is the root; nodes 1..D the top-1 chain (parent i-1); later nodes are leaves
  // whose parent is the root or a chain node
  if (parents[0] != -1) return fail(SEED_ERR_ARG, "node 0 must be the root (parent -1)");
  int D = 0;
  while (D + 1 < n && parents[D + 1] == D) ++D;
  std::vector<int> host(3 * MAX_ROWS, 0);
  for (int i = 0; i < n; ++i) {
    if (tokens[i] < 0 || tokens[i] >= p.V) return fail(SEED_ERR_ARG, "tree token out of range at node " + std::to_string(i));
    if (i > D && (parents[i] < 0 || parents[i] >= D))
      return fail(SEED_ERR_ARG, "node " + std::to_string(i) + ": a node after the chain must hang off the root or a chain node other than the last");
    host[i] = tokens[i];
    host[MAX_ROWS + i] = parents[i];
    host[2 * MAX_ROWS + i] = i <= D ? i : parents[i] + 1;
  }
  if ((int64_t)c->t_upper[0] + n + 1 > p.cfg.max_ctx) return fail(SEED_ERR_CAPACITY, "the tree would pass max_ctx");
  st = ensure_blocks(c, 0, c->t_upper[0] + n + 1);
  if (st != SEED_OK) return st;
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_tree), host.data(), host.size() * 4, hipMemcpyHostToDevice, c->s));
  if (p.cfg.dtype == SEED_BF16) enqueue_verify_tree<uint16_t>(c, n, logits, false);
  else enqueue_verify_tree<float>(c, n, logits, false);
  HIPCHK(hipGetLastError());
  std::vector<int> out(2 + MAX_ROWS);
  HIPCHK(hipMemcpyAsync(out.data(), c->ws<int>(p.o_tree_out), out.size() * 4, hipMemcpyDeviceToHost, c->s));
  st = read_t(c);
  if (st != SEED_OK) return st;
  if (path_len) *path_len = out[0];
  if (bonus) *bonus = out[1];
  if (path) std::copy(out.begin() + 2, out.begin() + 2 + out[0], path);
  c->drafts_k = -1;
  return SEED_OK;
}

void seed_tree_defaults(seed_tree_opts* o, int32_t max_depth) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->tau = 0.7f;
  o->max_depth = max_depth;
  o->n_levels = 3;
  o->thr[0] = 0.95f; o->thr[1] = 0.8f; o->thr[2] = 0.5f;
  o->k[0] = 1; o->k[1] = 3; o->k[2] = 5;
  o->k_rest = 10;
  o->max_nodes = MAX_ROWS;
}

seed_status seed_draft_tree(seed_ctx* c, const seed_tree_opts* opts, int32_t* tokens, int32_t* parents,
                            int32_t* n_nodes, float* p0, float* logits) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (!c->prefilled) return fail(SEED_ERR_STATE, "call seed_prefill first");
  st = check_tree_opts(c, opts, c->B);
  if (st != SEED_OK) return st;
  if (!tokens || !parents || !n_nodes) return fail(SEED_ERR_ARG, "tokens, parents and n_nodes must not be NULL");
  const Plan& p = c->p;
  const seed_tree_opts o = *opts;
  if ((int64_t)c->t_upper[0] + o.max_nodes + 1 > p.cfg.max_ctx) return fail(SEED_ERR_CAPACITY, "the tree would pass max_ctx");
  st = ensure_blocks(c, 0, c->t_upper[0] + o.max_nodes + 1);
  if (st != SEED_OK) return st;
  int depth = 0;
  for (int i = 1; i <= o.max_depth; ++i) {
    float* lg = logits ? logits + (size_t)(i - 1) * p.V : c->ws<float>(p.o_dlog);
    if (p.cfg.dtype == SEED_BF16) enqueue_tree_step<uint16_t>(c, o, i, lg, false);
    else enqueue_tree_step<float>(c, o, i, lg, false);
    HIPCHK(hipGetLastError());
    int stopped = 0;
    HIPCHK(hipMemcpyAsync(&stopped, c->ws<int>(p.o_tdraft) + TREE_MAX_STEPS * (TOPK_MAX + 2), 4, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    depth = i;
    if (stopped) break;
  }
  std::vector<int> tree(3 * MAX_ROWS + 1);
  std::vector<float> pr(TREE_MAX_STEPS);
  HIPCHK(hipMemcpyAsync(tree.data(), c->ws<int>(p.o_tree), tree.size() * 4, hipMemcpyDeviceToHost, c->s));
  HIPCHK(hipMemcpyAsync(pr.data(), c->ws<int>(p.o_tdraft) + TREE_MAX_STEPS * (TOPK_MAX + 1), TREE_MAX_STEPS * 4,
                        hipMemcpyDeviceToHost, c->s));
  HIPCHK(hipStreamSynchronize(c->s));
  const int n = tree[3 * MAX_ROWS];
  if (n < depth + 1 || n > o.max_nodes) return fail(SEED_ERR_HIP, "drafted tree size out of range");
  *n_nodes = n;
  std::copy(tree.begin(), tree.begin() + n, tokens);
  std::copy(tree.begin() + MAX_ROWS, tree.begin() + MAX_ROWS + n, parents);
  if (p0) std::copy(pr.begin() + 1, pr.begin() + 1 + depth, p0);
  c->drafts_k = -1;
  return SEED_OK;
}

seed_status seed_generate_tree(seed_ctx* c, const int32_t* tokens, int32_t len, const seed_tree_opts* topts,
                               const seed_gen_opts* opts, int32_t* out, int32_t* count, seed_stats* stats) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (!topts || !opts || !out || !count) return fail(SEED_ERR_ARG, "topts, opts, out and count must not be NULL");
  const Plan& p = c->p;
  const int max_new = opts->max_new;
  if (max_new < 1) return fail(SEED_ERR_ARG, "max_new must be >= 1");
  if (opts->eos_id < -1 || opts->eos_id >= p.V) return fail(SEED_ERR_ARG, "eos_id out of range");
  if (topts->max_nodes < 2 || topts->max_nodes > MAX_ROWS) return fail(SEED_ERR_ARG, "max_nodes must be in [2, 64]");
  if (opts->sim_accept < -1 || opts->sim_accept > topts->max_depth)
    return fail(SEED_ERR_ARG, "sim_accept must be -1 or in [0, max_depth]");
  if (opts->sim_accept >= 0 && !opts->forced_trace) return fail(SEED_ERR_ARG, "sim_accept needs forced_trace");
  std::vector<int> packed;
  // a finished sequence may still draft one more round's first step: room for two trees
  const int extra = max_new + 2 * (topts->max_nodes + 1);
  st = check_prompts(c, 1, tokens, &len, extra, packed);
  if (st != SEED_OK) return st;
  st = check_tree_opts(c, topts, 1);
  if (st != SEED_OK) return st;
  if (opts->sim_accept >= 0)
    for (int i = 0; i < max_new; ++i)
      if (opts->forced_trace[i] < 0 || opts->forced_trace[i] >= p.V)
        return fail(SEED_ERR_ARG, "forced_trace token out of range at " + std::to_string(i));
  // every argument is checked: from here on the previous decoding state is replaced
  st = start_sequences(c, 1, &len, extra);
  if (st != SEED_OK) return st;
  c->eos = opts->eos_id;
  c->sim_accept = -1;
  CallEvents ce;
  HIPCHK(ce.create());
  hipEvent_t e0 = ce.e[0], e1 = ce.e[1], e2 = ce.e[2];
  HIPCHK(hipEventRecord(e0, c->s));
  st = p.cfg.dtype == SEED_BF16 ? do_prefill<uint16_t>(c, packed) : do_prefill<float>(c, packed);
  if (st != SEED_OK) return st;
  c->prefilled = true;
  const int limit = len + max_new;
  HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_limit), &limit, 4, hipMemcpyHostToDevice, c->s));
  std::vector<int> tr;
  if (opts->sim_accept >= 0) {
    tr.assign(p.tstride, 0);
    for (int i = 0; i < max_new; ++i) tr[len + i] = opts->forced_trace[i];
    HIPCHK(hipMemcpyAsync(c->ws<int>(p.o_trace), tr.data(), tr.size() * 4, hipMemcpyHostToDevice, c->s));
    c->sim_accept = opts->sim_accept;
  }
  HIPCHK(hipEventRecord(e1, c->s));
  HIPCHK(hipStreamSynchronize(c->s));
  int rounds_run = 0;
  st = p.cfg.dtype == SEED_BF16 ? tree_rounds<uint16_t>(c, *topts, opts->use_graph != 0, 0, &rounds_run)
                                : tree_rounds<float>(c, *topts, opts->use_graph != 0, 0, &rounds_run);
  c->sim_accept = -1;
  if (st != SEED_OK) return st;
  HIPCHK(hipEventRecord(e2, c->s));
  HIPCHK(hipEventSynchronize(e2));
  std::vector<int> tok(p.tstride);
  int t = 0;
  HIPCHK(hipMemcpy(tok.data(), c->ws<int>(p.o_tokens), tok.size() * 4, hipMemcpyDeviceToHost));
  HIPCHK(hipMemcpy(&t, c->ws<int>(p.o_t), 4, hipMemcpyDeviceToHost));
  c->t_upper.assign(1, t);
  const int n = std::min(t - len, max_new);
  *count = n;
  for (int i = 0; i < max_new; ++i) out[i] = i < n ? tok[len + i] : -1;
  if (stats) {
    int rounds = 0;
    long long cnt[2];
    HIPCHK(hipMemcpy(&rounds, c->ws<int>(p.o_rounds), 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(cnt, c->ws<long long>(p.o_counters), 16, hipMemcpyDeviceToHost));
    stats->rounds = rounds;
    stats->drafted = cnt[0];
    stats->accepted = cnt[1];
    float ms1 = 0.f, ms2 = 0.f;
    HIPCHK(hipEventElapsedTime(&ms1, e0, e1));
    HIPCHK(hipEventElapsedTime(&ms2, e1, e2));
    stats->prefill_ms = ms1;
    stats->decode_ms = ms2;
    if (stats->n_accept_log && stats->n_accept_log_cap > 0) {
      const int64_t rows = std::min<int64_t>({(int64_t)rounds, stats->n_accept_log_cap, (int64_t)p.log_cap});
      HIPCHK(hipMemcpy(stats->n_accept_log, c->ws<int>(p.o_log), rows * 4, hipMemcpyDeviceToHost));
    }
    // a round's drafting steps vary here: draft_ms is the whole drafting phase of a round
    st = phase_medians(c, rounds, 1, &stats->verify_ms, &stats->draft_ms);
    if (st != SEED_OK) return st;
  }
  c->drafts_k = -1;
  return SEED_OK;
}

seed_status seed_spec_kv_bytes(const seed_config* cfg, size_t* bytes) {
  seed_status st = validate(cfg);
  if (st != SEED_OK) return st;
  if (!bytes) return fail(SEED_ERR_ARG, "bytes must not be NULL");
  *bytes = spec_kv_bytes(make_plan(*cfg));
  return SEED_OK;
}

}  // extern "C"

namespace {

// seed_spec_forward with the pass's own cache at skv (skv_blocks blocks per decoder layer).
seed_status spec_forward_impl(seed_ctx* c, int32_t n, const int32_t* tokens, int32_t block, void* skv, int skv_blocks,
                              float* logits, float* row_nll, double* loss) {
  std::vector<int> packed;
  seed_status st = check_prompts(c, 1, tokens, &n, 1, packed);
  if (st != SEED_OK) return st;
  st = start_sequences(c, 1, &n, 1);
  if (st != SEED_OK) return st;
  c->sim_accept = -1;
  c->eos = -1;
  const bool bf = c->p.cfg.dtype == SEED_BF16;
  st = bf ? do_prefill<uint16_t>(c, packed) : do_prefill<float>(c, packed);
  if (st != SEED_OK) return st;
  c->prefilled = true;
  st = bf ? do_spec<uint16_t>(c, n, block, skv, skv_blocks, logits) : do_spec<float>(c, n, block, skv, skv_blocks, logits);
  if (st != SEED_OK) return st;
  if (row_nll || loss) {
    float* nll = row_nll ? row_nll : c->ws<float>(c->p.o_nll);
    launch_row_nll(logits, n - 1, c->p.V, c->ws<int>(c->p.o_tokens) + 1, nll, c->s);
    HIPCHK(hipGetLastError());
    if (loss) {
      std::vector<float> h(n - 1);
      HIPCHK(hipMemcpyAsync(h.data(), nll, (size_t)(n - 1) * 4, hipMemcpyDeviceToHost, c->s));
      HIPCHK(hipStreamSynchronize(c->s));
      double sum = 0.0;
      for (float v : h) sum += v;
      *loss = sum;
    }
  }
  HIPCHK(hipStreamSynchronize(c->s));
  return SEED_OK;
}

}  // namespace

extern "C" {

seed_status seed_spec_forward(seed_ctx* c, int32_t n, const int32_t* tokens, int32_t block, void* shallow_kv,
                              float* logits, float* row_nll, double* loss) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (n < 2) return fail(SEED_ERR_ARG, "the sequence needs at least two tokens");
  if (block < 1) return fail(SEED_ERR_ARG, "block must be >= 1");
  if (!shallow_kv || !logits) return fail(SEED_ERR_ARG, "shallow_kv and logits must not be NULL");
  if ((uintptr_t)shallow_kv & 255) return fail(SEED_ERR_ARG, "shallow_kv must be 256-byte aligned");
  return spec_forward_impl(c, n, tokens, block, shallow_kv, c->p.blocks_per_seq, logits, row_nll, loss);
}

seed_status seed_spec_forward_noalloc(seed_ctx* c, int32_t n, const int32_t* tokens, int32_t block, float* logits,
                                      float* row_nll, double* loss) {
  seed_status st = check_ready(c);
  if (st != SEED_OK) return st;
  if (n < 2) return fail(SEED_ERR_ARG, "the sequence needs at least two tokens");
  if (block < 1) return fail(SEED_ERR_ARG, "block must be >= 1");
  if (!logits) return fail(SEED_ERR_ARG, "logits must not be NULL");
  if (!c->scratch_dev) return fail(SEED_ERR_HIP, "the library's scratch array has no device address on this GPU");
  // the pass's cache sized to this sequence (positions 0..n-2) instead of max_ctx
  const int blocks = cdiv(n, 16);
  const size_t need = spec_cache_bytes(c->p, blocks);
  if (need > NOALLOC_SCRATCH_BYTES)
    return fail(SEED_ERR_CAPACITY, "the pass needs " + std::to_string(need) + " bytes of scratch; the fixed array holds " +
                                       std::to_string(NOALLOC_SCRATCH_BYTES) + " (use seed_spec_forward with a buffer)");
  // no timing events here (creating them allocates)
  const int timed_id = c->timed_id;
  c->timed_id = -1;
  st = spec_forward_impl(c, n, tokens, block, c->scratch_dev, blocks, logits, row_nll, loss);
  c->timed_id = timed_id;
  return st;
}

seed_status seed_get_tokens(seed_ctx* c, int32_t b, int32_t* out, int32_t cap, int32_t* len) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  if (!c->prefilled) return fail(SEED_ERR_STATE, "call seed_prefill first");
  if (b < 0 || b >= c->B) return fail(SEED_ERR_ARG, "sequence index out of range");
  if (!len) return fail(SEED_ERR_ARG, "len must not be NULL");
  seed_status st = read_t(c);
  if (st != SEED_OK) return st;
  const int t = c->t_upper[b];
  *len = t;
  if (out && cap > 0) {
    HIPCHK(hipMemcpy(out, c->ws<int>(c->p.o_tokens) + (size_t)b * c->p.tstride, std::min(cap, t) * 4, hipMemcpyDeviceToHost));
  }
  return SEED_OK;
}

seed_status seed_read_kv(seed_ctx* c, int32_t b, int32_t layer, int32_t pos0, int32_t n, void* k_out, void* v_out) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  if (!c->prefilled) return fail(SEED_ERR_STATE, "call seed_prefill first");
  const Plan& p = c->p;
  if (b < 0 || b >= c->B) return fail(SEED_ERR_ARG, "sequence index out of range");
  if (layer < 0 || layer >= p.L) return fail(SEED_ERR_ARG, "layer out of range");
  if (!k_out || !v_out) return fail(SEED_ERR_ARG, "k_out and v_out must not be NULL");
  const int have = (int)c->seq_blocks[b].size() * 16;
  if (pos0 < 0 || n < 0 || (int64_t)pos0 + n > have)
    return fail(SEED_ERR_ARG, "positions [" + std::to_string(pos0) + ", " + std::to_string((int64_t)pos0 + n) +
                                  ") exceed the sequence's cache blocks (" + std::to_string(have) + " positions)");
  // one block holds K [n_kv][16][hd] then V^T [n_kv][hd][16] of 16 positions
  const size_t es = p.esize, per = (size_t)p.NKV * 16 * p.HD * es;
  std::vector<char> blk(2 * per);
  char* ko = static_cast<char*>(k_out);
  char* vo = static_cast<char*>(v_out);
  for (int pos = pos0; pos < pos0 + n;) {
    const int bi = pos >> 4, id = c->seq_blocks[b][bi];
    const char* src = c->KV + ((size_t)layer * p.n_blocks + id) * 2 * per;
    HIPCHK(hipMemcpyAsync(blk.data(), src, 2 * per, hipMemcpyDeviceToHost, c->s));
    HIPCHK(hipStreamSynchronize(c->s));
    for (; pos < pos0 + n && (pos >> 4) == bi; ++pos) {
      const int s = pos & 15;
      const size_t row = (size_t)(pos - pos0) * p.NKV * p.HD * es;
      for (int h = 0; h < p.NKV; ++h) {
        std::memcpy(ko + row + (size_t)h * p.HD * es, blk.data() + ((size_t)h * 16 + s) * p.HD * es, p.HD * es);
        for (int d = 0; d < p.HD; ++d)
          std::memcpy(vo + row + ((size_t)h * p.HD + d) * es, blk.data() + per + (((size_t)h * p.HD + d) * 16 + s) * es, es);
      }
    }
  }
  return SEED_OK;
}

seed_status seed_kernel_timing(seed_ctx* c, int32_t kernel_id, int32_t enable) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  HIPCHK(drain_timing(c));
  c->timed_id = enable ? kernel_id : -1;
  c->timed_launches = 0;
  c->timed_ms = 0.0;
  return SEED_OK;
}

seed_status seed_kernel_timing_read(seed_ctx* c, int64_t* launches, double* total_ms) {
  if (!c) return fail(SEED_ERR_ARG, "ctx is NULL");
  HIPCHK(drain_timing(c));
  if (launches) *launches = c->timed_launches;
  if (total_ms) *total_ms = c->timed_ms;
  return SEED_OK;
}

void seed_destroy(seed_ctx* c) {
  if (!c) return;
  hipStreamSynchronize(c->s);
  for (auto& kv : c->graphs) hipGraphExecDestroy(kv.second);
  for (auto& kv : c->tree_step_graphs) hipGraphExecDestroy(kv.second);
  for (auto& kv : c->tree_verify_graphs) hipGraphExecDestroy(kv.second);
  if (c->hstat) hipHostFree(c->hstat);
  for (auto& t : c->pending) { hipEventDestroy(t.a); hipEventDestroy(t.b); }
  for (auto& t : c->pool) { hipEventDestroy(t.a); hipEventDestroy(t.b); }
  delete c;
}

}  // extern "C"
