// Row setup + embedding gather, acceptance/commit, and load-time helpers.
#include "device_common.h"

#include <algorithm>

namespace seedk {

// ---------------------------------------------------------------------------------------------
// Row setup for a pass: pick each row's sequence, position and token (Algorithm 2: drafts feed
// X_draft[i-1], verification feeds X_draft[0..d]; prefill and the drafting objective's pass of
// Algorithm 1 feed the sequence itself), gather the raw embedding H^0 = W_in x from
// the packed table into the fp32 residual stream, and write its per-16-feature sums of squares.
// ---------------------------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_setup(SetupArgs a) {
  const int m = blockIdx.x;
  __shared__ int s_tok, s_pos, s_seq, s_slot;
  if (a.stamp && m == 0 && threadIdx.x == 0) {
    const long long now = (long long)__builtin_amdgcn_s_memrealtime();
    const int r = *a.rounds;
    if (r >= 0 && r < a.stamp_cap) a.stamp[(size_t)r * 3 + a.stamp_col] = now;
  }
  if (threadIdx.x == 0) {
    int b, pos, tok, slot = -1;
    if (a.mode == SETUP_PREFILL || a.mode == SETUP_SPEC) {
      b = a.pf_seq;
      pos = a.pf_pos0 + m;
      tok = a.tokens[b * a.tstride + pos];
    } else if (a.mode == SETUP_DRAFT) {
      b = m;
      pos = a.t[b] - 1 + (a.step - 1);
      tok = a.drafts[b * a.dstride + a.step - 1];
    } else if (a.mode == SETUP_TREE) {
      // packed draft tree (Tree-Based Verification): node m at rotary position p + depth,
      // cached at slot p + m
      b = 0;
      pos = a.t[0] - 1 + a.tree_depth[m];
      slot = a.t[0] - 1 + m;
      tok = a.tree_tok[m];
      // benchmark mode: chain nodes 1..a take the greedy trace, node a+1 a token that is not it
      if (a.sim_accept >= 0 && m >= 1 && a.tree_depth[m] == m && m <= a.sim_accept + 1) {
        const int tr = a.trace[pos];
        tok = (m <= a.sim_accept) ? tr : (tr + 1) % a.vocab;
        a.tree_tok[m] = tok;
      }
    } else {
      b = m / a.R;
      const int r = m - b * a.R;
      pos = a.t[b] - 1 + r;
      tok = a.drafts[b * a.dstride + r];
      if (a.sim_accept >= 0 && r >= 1 && r <= a.sim_accept + 1) {
        const int tr = a.trace[b * a.tstride + pos];
        tok = (r <= a.sim_accept) ? tr : (tr + 1) % a.vocab;
        a.drafts[b * a.dstride + r] = tok;
      }
    }
    if (slot < 0) slot = pos;
    a.row_seq[m] = b;
    a.row_pos[m] = pos;
    a.row_slot[m] = slot;
    s_tok = tok;
    s_pos = pos;
    s_seq = b;
    s_slot = slot;
  }
  __syncthreads();
  const int tok = s_tok;
  {
    // the row's KV block and RoPE angles, read once per pass by every layer's QKV epilogue
    const int pos = s_pos, half = a.head_dim >> 1, slot = s_slot;
    // keys/values go to the row's cache slot; the block-causal drafter pass writes to a cache of
    // its own, indexed by position (block id = position / 16)
    if (threadIdx.x == 0) a.row_blk[m] = a.mode == SETUP_SPEC ? (slot >> 4) : a.bt[s_seq * a.bt_stride + (slot >> 4)];
    for (int i = threadIdx.x; i < half; i += blockDim.x) {
      a.row_rope[(size_t)m * a.head_dim + i] = a.rope_cos[(size_t)pos * half + i];
      a.row_rope[(size_t)m * a.head_dim + half + i] = a.rope_sin[(size_t)pos * half + i];
    }
  }
  const int KT = a.H >> 5;
  const T* E = reinterpret_cast<const T*>(a.E);
  const int nt = tok >> 4, rr = tok & 15;
  for (int j = threadIdx.x; j < (a.H >> 4); j += blockDim.x) {
    const int k0 = j * 16, kt = k0 >> 5, kg = (k0 >> 3) & 3;
    const T* src = E + ((size_t)nt * KT + kt) * 512 + (rr + 16 * kg) * 8;
    float v0[8], v1[8];
    ET<T>::to_f32(ET<T>::load(src), v0);
    ET<T>::to_f32(ET<T>::load(src + 128), v1);   // lane + 16 => next 8 features
    float* hp = a.h + (size_t)m * a.H + k0;
    float* xgp = a.xg + (size_t)m * a.H + k0;
    const float* gp = a.gain + k0;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) { hp[i] = v0[i]; xgp[i] = v0[i] * gp[i]; s += v0[i] * v0[i]; }
#pragma unroll
    for (int i = 0; i < 8; ++i) { hp[8 + i] = v1[i]; xgp[8 + i] = v1[i] * gp[8 + i]; s += v1[i] * v1[i]; }
    a.ssq[(size_t)m * (a.H >> 4) + j] = s;
  }
}

// ---------------------------------------------------------------------------------------------
// Greedy acceptance and commit (Algorithm 2): n_accept = longest prefix with g_{i-1} ==
// X_draft[i], append X_draft[1..n_accept] and the bonus token g_{n_accept}, advance t. The
// cache needs no work: positions >= the new t-1 are simply treated as invalid.
// ---------------------------------------------------------------------------------------------
__global__ void __launch_bounds__(64) k_accept(DevState st, int B, int k) {
  __shared__ int s_round;
  if (threadIdx.x == 0) s_round = *st.rounds;
  __syncthreads();
  const int b = threadIdx.x;
  if (b < B) {
    int logv = -1;
    if (st.active[b]) {
      const int R = k + 1;
      int t = st.t[b];
      int* dr = st.drafts + b * st.dstride;
      const int* gv = st.vtok + b * R;
      int n = 0;
      while (n < k && gv[n] == dr[n + 1]) ++n;
      const int bonus = gv[n];
      int* tk = st.tokens + b * st.tstride;
      int stop = 0, ncommit = n + 1;
      for (int i = 0; i < n + 1; ++i) {
        const int tv = (i < n) ? dr[i + 1] : bonus;
        tk[t + i] = tv;
        if (st.eos >= 0 && tv == st.eos) { ncommit = i + 1; stop = 1; break; }
      }
      t += ncommit;
      st.t[b] = t;
      dr[0] = tk[t - 1];
      st.nacc[b] = n;
      st.bonus[b] = bonus;
      if (stop || t >= st.limit[b]) st.active[b] = 0;
      atomicAdd(reinterpret_cast<unsigned long long*>(&st.counters[0]), (unsigned long long)k);
      atomicAdd(reinterpret_cast<unsigned long long*>(&st.counters[1]), (unsigned long long)n);
      logv = n;
    }
    if (s_round < st.log_cap) st.nacc_log[(size_t)s_round * B + b] = logv;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    *st.rounds = s_round + 1;
    if (st.stamp && s_round < st.stamp_cap) st.stamp[(size_t)s_round * 3 + 2] = (long long)__builtin_amdgcn_s_memrealtime();
  }
}

// ---------------------------------------------------------------------------------------------
// Tree acceptance and commit (Tree-Based Verification, one sequence): from the root, move to the
// child whose token equals the verifier's argmax at the current node while one exists; append
// the accepted tokens and the bonus token (the argmax at the last node reached). The nodes of the
// top-1 chain are cached at the positions of their depths already (node d of the chain has
// depth d); an accepted leaf is not, and k_kv_move copies its keys/values there in every layer.
// out: [0] path length, [1] bonus, [2 + i] path nodes, [TREE_MOVE] leaf to move (0 = none),
// [TREE_MOVE + 1] p = the old pending token's position.
// ---------------------------------------------------------------------------------------------
static constexpr int TREE_MOVE = 2 + 64;

__global__ void __launch_bounds__(64) k_accept_tree(DevState st, int n, const int* tok, const int* par,
                                                   const int* depth, int* out, int* hstat) {
  if (threadIdx.x != 0) return;
  const int s_round = *st.rounds;
  int logv = -1;
  out[0] = 0;
  out[1] = -1;
  out[TREE_MOVE] = 0;
  if (st.active[0]) {
    int t = st.t[0];
    out[TREE_MOVE + 1] = t - 1;
    int node = 0, len = 0;
    for (;;) {
      const int g = st.vtok[node];
      int nxt = -1;
      for (int c = 1; c < n; ++c)
        if (par[c] == node && tok[c] == g) { nxt = c; break; }
      if (nxt < 0) break;
      out[2 + len] = nxt;
      ++len;
      node = nxt;
    }
    const int bonus = st.vtok[node];
    if (node != depth[node]) out[TREE_MOVE] = node;
    int* tk = st.tokens;
    int stop = 0, ncommit = len + 1;
    for (int i = 0; i < len + 1; ++i) {
      const int tv = (i < len) ? tok[out[2 + i]] : bonus;
      tk[t + i] = tv;
      if (st.eos >= 0 && tv == st.eos) { ncommit = i + 1; stop = 1; break; }
    }
    t += ncommit;
    st.t[0] = t;
    st.drafts[0] = tk[t - 1];
    st.nacc[0] = len;
    st.bonus[0] = bonus;
    if (stop || t >= st.limit[0]) st.active[0] = 0;
    st.counters[0] += n - 1;
    st.counters[1] += len;
    out[0] = len;
    out[1] = bonus;
    logv = len;
  }
  if (s_round < st.log_cap) st.nacc_log[s_round] = logv;
  *st.rounds = s_round + 1;
  if (st.stamp && s_round < st.stamp_cap) st.stamp[(size_t)s_round * 3 + 2] = (long long)__builtin_amdgcn_s_memrealtime();
  if (hstat) {   // host-visible: the sequence's length and liveness, tagged with the round count
    hstat[5] = st.t[0];
    hstat[6] = st.active[0];
    __threadfence_system();
    hstat[4] = s_round + 1;
  }
}

// Copies the keys/values of cache slot p + leaf to position p + depth(leaf) in every layer, when
// k_accept_tree asked for it.
template <typename T>
__global__ void __launch_bounds__(256) k_kv_move(const int* depth, const int* out, T* kv, int n_layers, int n_blocks,
                                                 int n_kv, int head_dim, const int* bt) {
  const int leaf = out[TREE_MOVE];
  if (leaf == 0) return;
  const int p = out[TREE_MOVE + 1];
  const int from = p + leaf, to = p + depth[leaf];
  const int per_layer = 2 * n_kv * head_dim;   // K and V values of one position
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n_layers * per_layer; e += gridDim.x * blockDim.x) {
    const int l = e / per_layer, r = e - l * per_layer;
    const int kvs = r / (n_kv * head_dim), r2 = r - kvs * n_kv * head_dim, h = r2 / head_dim, d = r2 - h * head_dim;
    const size_t fb = (((size_t)l * n_blocks + bt[from >> 4]) * 2 + kvs) * n_kv + h;
    const size_t tb = (((size_t)l * n_blocks + bt[to >> 4]) * 2 + kvs) * n_kv + h;
    if (kvs == 0) kv[tb * 16 * head_dim + (to & 15) * head_dim + d] = kv[fb * 16 * head_dim + (from & 15) * head_dim + d];
    else kv[tb * head_dim * 16 + d * 16 + (to & 15)] = kv[fb * head_dim * 16 + d * 16 + (from & 15)];
  }
}

// ---------------------------------------------------------------------------------------------
// Negative log-likelihood of each row's target under the softmax of its logits (the per-position
// term of L_spec, Algorithm 1): one workgroup per row, one pass over the row. Each thread keeps a
// running (max m, sum of exp(x - m)) over steps of 16 values (four 16-byte loads in flight); the
// pairs are then merged across the wave and the workgroup, each merge rescaling both sums to the
// larger maximum.
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ void lse_merge(float& m, float& s, float mo, float so) {
  const float mn = fmaxf(m, mo);
  if (mn == NEG_INF) return;   // both empty
  s = (m == NEG_INF ? 0.f : s * __expf(m - mn)) + (mo == NEG_INF ? 0.f : so * __expf(mo - mn));
  m = mn;
}

__global__ void __launch_bounds__(256) k_row_nll(const float* logits, int V, const int* target, float* nll) {
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* z = logits + (size_t)r * V;
  __shared__ float s_m[4], s_s[4];
  float m = NEG_INF, s = 0.f;
  auto step = [&](const float (&x)[16]) {
    float cm = x[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) cm = fmaxf(cm, x[i]);
    float acc = 0.f;
    if (cm != NEG_INF) {
#pragma unroll
      for (int i = 0; i < 16; ++i) acc += x[i] == NEG_INF ? 0.f : __expf(x[i] - cm);
    }
    lse_merge(m, s, cm, acc);
  };
  if ((V & 3) == 0) {   // rows start 16-byte aligned
    const int V4 = V >> 2;
    const float4* z4 = reinterpret_cast<const float4*>(z);
    for (int j0 = 0; j0 < V4; j0 += 4 * 256) {
      float x[16];
#pragma unroll
      for (int u = 0; u < 4; ++u) {   // unconditional (clamped) loads; slots past the row are masked
        const int idx = j0 + u * 256 + tid;
        const float4 v = z4[min(idx, V4 - 1)];
        const bool ok = idx < V4;
        x[4 * u + 0] = ok ? v.x : NEG_INF;
        x[4 * u + 1] = ok ? v.y : NEG_INF;
        x[4 * u + 2] = ok ? v.z : NEG_INF;
        x[4 * u + 3] = ok ? v.w : NEG_INF;
      }
      step(x);
    }
  } else {
    for (int j0 = 0; j0 < V; j0 += 16 * 256) {
      float x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int idx = j0 + u * 256 + tid;
        x[u] = idx < V ? z[idx] : NEG_INF;
      }
      step(x);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) lse_merge(m, s, __shfl_xor(m, o), __shfl_xor(s, o));
  if (lane == 0) {
    s_m[wave] = m;
    s_s[wave] = s;
  }
  __syncthreads();
  if (tid == 0) {
    float mm = s_m[0], ss = s_s[0];
    for (int w = 1; w < 4; ++w) lse_merge(mm, ss, s_m[w], s_s[w]);
    nll[r] = mm + logf(ss) - z[target[r]];
  }
}

// ---------------------------------------------------------------------------------------------
// Load-time helpers.
// ---------------------------------------------------------------------------------------------
template <typename T>
__global__ void k_pack(const T* src, T* dst, const int* dst_row, int rows, int K) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int groups = K >> 3;
  if (gid >= (long long)rows * groups) return;
  const int r = (int)(gid / groups), kq = (int)(gid - (long long)r * groups);
  const int k = kq * 8, n = dst_row[r];
  const int KT = K >> 5, nt = n >> 4, rr = n & 15, kt = k >> 5, kg = (k >> 3) & 3;
  const T* s = src + (size_t)r * K + k;
  T* d = dst + ((size_t)nt * KT + kt) * 512 + (rr + 16 * kg) * 8;
#pragma unroll
  for (int j = 0; j < 8; ++j) d[j] = s[j];
}

__global__ void k_to_f32(const void* src, int is_bf16, float* dst, long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  dst[i] = is_bf16 ? bf2f(reinterpret_cast<const uint16_t*>(src)[i]) : reinterpret_cast<const float*>(src)[i];
}

__global__ void k_fill_u32(uint32_t* dst, uint32_t v, long long n) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
    dst[i] = v;
}

// ---------------------------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------------------------
template <typename T>
void launch_setup(const SetupArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_setup<T>), dim3(a.M), dim3(256), 0, s, a);
}

void launch_accept(const DevState& st, int B, int k, hipStream_t s) {
  hipLaunchKernelGGL(k_accept, dim3(1), dim3(64), 0, s, st, B, k);
}

void launch_accept_tree(const DevState& st, int n, const int* tree_tok, const int* tree_par, const int* tree_depth,
                        int* out, void* kv, int n_layers, int n_blocks, int n_kv, int head_dim, int esize,
                        const int* bt, int* hstat, hipStream_t s) {
  hipLaunchKernelGGL(k_accept_tree, dim3(1), dim3(64), 0, s, st, n, tree_tok, tree_par, tree_depth, out, hstat);
  const int blocks = std::max(1, std::min(256, (n_layers * 2 * n_kv * head_dim + 255) / 256));
  if (esize == 2)
    hipLaunchKernelGGL(k_kv_move<uint16_t>, dim3(blocks), dim3(256), 0, s, tree_depth, (const int*)out,
                       reinterpret_cast<uint16_t*>(kv), n_layers, n_blocks, n_kv, head_dim, bt);
  else
    hipLaunchKernelGGL(k_kv_move<float>, dim3(blocks), dim3(256), 0, s, tree_depth, (const int*)out,
                       reinterpret_cast<float*>(kv), n_layers, n_blocks, n_kv, head_dim, bt);
}

void launch_row_nll(const float* logits, int rows, int V, const int* target, float* nll, hipStream_t s) {
  if (rows > 0) hipLaunchKernelGGL(k_row_nll, dim3(rows), dim3(256), 0, s, logits, V, target, nll);
}

template <typename T>
void launch_pack(const void* src, void* dst, const int* dst_row, int rows, int K, hipStream_t s) {
  const long long n = (long long)rows * (K >> 3);
  hipLaunchKernelGGL((k_pack<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const T*>(src), reinterpret_cast<T*>(dst), dst_row, rows, K);
}

void launch_to_f32(const void* src, int src_is_bf16, float* dst, long long n, hipStream_t s) {
  hipLaunchKernelGGL(k_to_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, src_is_bf16, dst, n);
}

void launch_fill_u32(void* dst, unsigned value, long long n_words, hipStream_t s) {
  long long blocks = (n_words + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<uint32_t*>(dst), value, n_words);
}

template void launch_setup<uint16_t>(const SetupArgs&, hipStream_t);
template void launch_setup<float>(const SetupArgs&, hipStream_t);
template void launch_pack<uint16_t>(const void*, void*, const int*, int, int, hipStream_t);
template void launch_pack<float>(const void*, void*, const int*, int, int, hipStream_t);

}  // namespace seedk
