// Confidence-aware dynamic drafting (Method, Adaptive Drafting with Tree-Based Verification;
// appendix "Confidence-Aware Dynamic Drafting", Fig. 3 left): after each drafting step, the top-1
// probability p0 of the step's logits and its k highest-ranked tokens, k from the top-p table of
// p0; drafting stops after a step with p0 < tau (or at the depth / node limits) and the tree is
// then packed for tree-based verification: root, top-1 chain in depth order, then the other
// candidates by depth and rank.
//
// Ranking: larger logit first, equal logits by lower token id. Two stages: TOPK_PARTS waves each
// rank a contiguous chunk of the vocabulary (chunk maximum, sum of exp(z - chunk maximum), the
// chunk's k_max best), then one workgroup merges the partials in a fixed order.
#include "device_common.h"

namespace seedk {

__device__ __forceinline__ bool ranks_before(float v, int i, float w, int j) {
  return v > w || (v == w && (unsigned)i < (unsigned)j);   // id -1 (none) ranks after every id
}

__device__ __forceinline__ void wave_best(float& v, int& i) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(i, off);
    if (ranks_before(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

constexpr int TOPK_PER_LANE = 16;   // logits per lane in the first stage (V <= 256 * 64 * 16)

// First stage: wave g ranks logits [g * chunk, (g + 1) * chunk); lane l holds ids
// g * chunk + 64 j + l (coalesced).
__global__ void __launch_bounds__(64) k_topk_partial(TreeDraftArgs a) {
  if (a.step > 1 && a.dstate[0]) return;   // drafting already stopped this round
  const int g = blockIdx.x, lane = threadIdx.x;
  const int per = a.chunk >> 6;
  const int base = g * a.chunk + lane;
  float v[TOPK_PER_LANE];
  float mx = NEG_INF;
#pragma unroll
  for (int j = 0; j < TOPK_PER_LANE; ++j) {
    const int id = base + 64 * j;
    v[j] = (j < per && id < a.V) ? a.logits[id] : NEG_INF;
    mx = fmaxf(mx, v[j]);
  }
  mx = wave_max(mx);   // finite: every chunk holds at least one logit
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < TOPK_PER_LANE; ++j) sum += (v[j] == NEG_INF) ? 0.f : expf(v[j] - mx);
  sum = wave_sum(sum);
  unsigned taken = 0;
  for (int r = 0; r < a.k_max; ++r) {
    float bv = NEG_INF;
    int bi = -1, bj = -1;
#pragma unroll
    for (int j = 0; j < TOPK_PER_LANE; ++j) {
      const int id = base + 64 * j;
      if (j < per && id < a.V && !((taken >> j) & 1u) && ranks_before(v[j], id, bv, bi)) {
        bv = v[j];
        bi = id;
        bj = j;
      }
    }
    float wv = bv;
    int wi = bi;
    wave_best(wv, wi);
    if (bj >= 0 && wi == bi) taken |= 1u << bj;   // the lane holding the winner drops it
    if (lane == 0) {
      a.pval[g * TOPK_MAX + r] = wv;
      a.pidx[g * TOPK_MAX + r] = wi;
    }
  }
  if (lane == 0) {
    a.pmax[g] = mx;
    a.psum[g] = sum;
  }
}

// Second stage (one workgroup): p0 = 1 / sum_v exp(z_v - max z), the fan-out k, the k best of the
// partials, then the drafting state; on a stop, the packed tree.
__global__ void __launch_bounds__(256) k_topk_finalize(TreeDraftArgs a, int G) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int stopped = a.step > 1 ? a.dstate[0] : 0;
  if (stopped) return;
  const int nodes0 = a.step > 1 ? a.dstate[1] : 1;
  __shared__ float s_f[4];
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  __shared__ int s_win[TOPK_MAX];
  __shared__ int s_cand[TREE_MAX_STEPS * TOPK_MAX];
  __shared__ int s_kcnt[TREE_MAX_STEPS];
  __shared__ int s_root, s_tag;
  // every global input is requested up front, in one round trip: the partials (thread t holds
  // candidates t, t + 256, ... of the G x TOPK_MAX table), chunk maxima and sums, and for the
  // packing the earlier steps' candidates and fan-outs, the root and the round tag
  constexpr int PER = TOPK_PARTS * TOPK_MAX / 256;
  const int nc = G * TOPK_MAX;
  float cv[PER];
  int ci[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int c = tid + 256 * u;
    const bool ok = c < nc && (c & (TOPK_MAX - 1)) < a.k_max;
    cv[u] = ok ? a.pval[c] : NEG_INF;
    ci[u] = ok ? a.pidx[c] : -1;
  }
  const float pm = tid < G ? a.pmax[tid] : NEG_INF;
  const float ps = tid < G ? a.psum[tid] : 0.f;
  for (int i = tid; i < a.step * TOPK_MAX; i += 256) s_cand[i] = a.cand[i];
  if (tid < a.step) s_kcnt[tid] = a.kcnt[tid];
  if (tid == 0) {
    s_root = a.drafts[0];
    s_tag = *a.rounds;
  }
  // global maximum, then the sum of exponentials (waves and partials in a fixed order)
  float m = wave_max(pm);
  if (lane == 0) s_f[w] = m;
  __syncthreads();
  const float M = fmaxf(fmaxf(s_f[0], s_f[1]), fmaxf(s_f[2], s_f[3]));
  __syncthreads();
  float sv = tid < G ? ps * expf(pm - M) : 0.f;
  sv = wave_sum(sv);
  if (lane == 0) s_f[w] = sv;
  __syncthreads();
  const float S = ((s_f[0] + s_f[1]) + s_f[2]) + s_f[3];
  const float p0 = 1.f / S;   // the top-1 logit is M
  int k = a.k_rest;
  for (int j = 0; j < a.n_levels; ++j)
    if (p0 > a.thr[j]) {
      k = a.kk[j];
      break;
    }
  k = min(k, a.max_nodes - nodes0);
  // the k best of the partial candidates, one block-wide arg-max per rank
  for (int r = 0; r < k; ++r) {
    float bv = NEG_INF;
    int bi = -1;
#pragma unroll
    for (int u = 0; u < PER; ++u)
      if (ci[u] >= 0 && ranks_before(cv[u], ci[u], bv, bi)) {
        bv = cv[u];
        bi = ci[u];
      }
    float wv = bv;
    int wi = bi;
    wave_best(wv, wi);
    if (lane == 0) {
      s_v[w] = wv;
      s_i[w] = wi;
    }
    __syncthreads();
    float xv = s_v[0];
    int xi = s_i[0];
#pragma unroll
    for (int q = 1; q < 4; ++q)
      if (ranks_before(s_v[q], s_i[q], xv, xi)) {
        xv = s_v[q];
        xi = s_i[q];
      }
#pragma unroll
    for (int u = 0; u < PER; ++u)
      if (ci[u] == xi) ci[u] = -1;   // token ids are unique: only the winner's holder matches
    if (tid == 0) s_win[r] = xi;
    __syncthreads();
  }
  if (tid != 0) return;
  const int step = a.step;
  for (int r = 0; r < k; ++r) a.cand[step * TOPK_MAX + r] = s_win[r];
  a.kcnt[step] = k;
  a.p0[step] = p0;
  a.drafts[step] = s_win[0];
  const int nodes = nodes0 + k;
  const int stop = (p0 < a.tau) || step >= a.max_depth || nodes >= a.max_nodes;
  a.dstate[0] = stop;
  a.dstate[1] = nodes;
  if (!stop) return;
  // pack: node 0 the root, nodes 1..D the chain, then each step's other candidates by rank
  int* tok = a.tree;
  int* par = a.tree + 64;
  int* dep = a.tree + 128;
  tok[0] = s_root;
  par[0] = -1;
  dep[0] = 0;
  for (int d = 1; d <= step; ++d) {
    tok[d] = (d == step) ? s_win[0] : s_cand[d * TOPK_MAX];
    par[d] = d - 1;
    dep[d] = d;
  }
  int n = step + 1;
  for (int d = 1; d <= step; ++d) {
    const int kd = (d == step) ? k : s_kcnt[d];
    for (int r = 1; r < kd; ++r) {
      tok[n] = (d == step) ? s_win[r] : s_cand[d * TOPK_MAX + r];
      par[n] = d - 1;
      dep[n] = d;
      ++n;
    }
  }
  a.tree[192] = n;
  if (a.hstat) {
    a.hstat[1] = n;
    a.hstat[2] = step;
    __threadfence_system();
    a.hstat[0] = s_tag;
  }
}

int tree_topk_chunk(int V) {
  const int per = (V + TOPK_PARTS * 64 - 1) / (TOPK_PARTS * 64);
  return per * 64;
}

void launch_tree_topk(const TreeDraftArgs& a, hipStream_t s) {
  const int G = (a.V + a.chunk - 1) / a.chunk;
  hipLaunchKernelGGL(k_topk_partial, dim3(G), dim3(64), 0, s, a);
  hipLaunchKernelGGL(k_topk_finalize, dim3(1), dim3(256), 0, s, a, G);
}

}  // namespace seedk
