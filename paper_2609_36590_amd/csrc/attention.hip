// Paged split-KV attention on MFMA for the verify, draft and prefill passes.
//
// The unit of work is one 16-position paged KV block (a "tile"). A wave takes a run of `tpw`
// consecutive tiles of one (sequence b, KV head h, row-block rb); a workgroup of 4 waves takes 4
// consecutive runs, one "group" of span = 64 * tpw absolute positions. The queries of a
// row-block (G query heads x RB rows, <= 32 query vectors) are the MFMA B operand:
//   S^T = K Q^T     16x16x32 MFMAs, the block's K rows as the A operand (k = head dim);
//   O^T += V^T P^T  16x16x16 MFMAs, the block's transposed V as the A operand (k = positions).
// After S^T, lane (qv, kg) holds the scores of positions 4kg..4kg+3 of the tile for query vector
// qv, which is exactly the k-slot layout O^T needs for P^T: no cross-lane shuffle of P.
// The queries' B-operand fragments (bf16 hi/lo) are built once per workgroup into LDS and read
// per tile, so that a wave's registers hold only its tiles' K/V fragments and two waves fit per
// SIMD even with 4 tiles per wave and 32 query vectors.
// Positions later than a query's own are masked; a wave keeps an online softmax (base 2) over its
// tiles. The 4 waves' partials are merged left to right in LDS and written as the group partial
// (o, m, l), or as the final output when the pass sees a single group.
//
// The tree variant verifies a packed draft tree (Tree-Based Verification): node i of the tree sits
// at rotary position p + depth(i) and cache slot p + i, the top-1 chain first, so a node's
// ancestors are exactly the positions below its rotary position; it attends to those and to its
// own slot.
//
// The block-causal variant (SPEC) computes the drafter pass of the speculative drafting objective
// (Algorithm 1, Fig. 2 right): row q attends to the deep cache at positions below its block start
// s and to the pass's own keys/values (a second, position-indexed cache) at s..q. Tiles that
// hold positions of both kinds for some row are contracted with both caches and selected per
// (query, position).
//
// k_attn_combine merges the group partials of each query vector with a fixed tree: lane j of an
// 8-lane team merges groups j, j+8, j+16, ... left to right, then the 8 results are merged
// pairwise (0+1, 2+3, ..; then 01+23, ..). A tile, run or group with no visible position is an
// exact identity of every merge, and the tree's shape depends only on absolute group indices, so
// a query's result depends only on the positions it attends to, not on how many rows share the
// pass: verify rows and plain greedy decoding give bit-identical outputs, and so do a sequence
// decoded alone and inside a batch.
#include "device_common.h"

#include <algorithm>

namespace seedk {

static constexpr int ATT_WAVES = 4;
static constexpr int CMB_LANES = 8;
static constexpr int CMB_INFLIGHT = 4;   // group partials in flight per lane (8 measured slower)

// 16-position contraction (k = 16) for O^T: 4 stored elements per lane as the A operand, 4 fp32
// probabilities per lane as the B operand (bf16 hi/lo pair, or fp32 for fp32 caches).
template <typename T>
struct PV;

template <>
struct PV<uint16_t> {
  typedef __attribute__((ext_vector_type(4))) short s16x4;
  struct A { uint2 v; };
  struct B { s16x4 hi, lo; };
  __device__ static A load(const uint16_t* p) { return A{*reinterpret_cast<const uint2*>(p)}; }
  __device__ static B split(const float x[4]) {
    B r;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint16_t h = f2bf(x[j]);
      r.hi[j] = (short)h;
      r.lo[j] = (short)f2bf(x[j] - bf2f(h));
    }
    return r;
  }
  __device__ static void mma(f32x4& acc, const A& a, const B& b) {
    const s16x4 av = __builtin_bit_cast(s16x4, a.v);
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, b.hi, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, b.lo, acc, 0, 0, 0);
  }
};

template <>
struct PV<float> {
  struct A { float4 v; };
  struct B { float x[4]; };
  __device__ static A load(const float* p) { return A{*reinterpret_cast<const float4*>(p)}; }
  __device__ static B split(const float x[4]) { return B{{x[0], x[1], x[2], x[3]}}; }
  __device__ static void mma(f32x4& acc, const A& a, const B& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.x, b.x[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.y, b.x[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.z, b.x[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.w, b.x[3], acc, 0, 0, 0);
  }
};

enum AttnMode { ATT_CAUSAL = 0, ATT_SPEC = 1, ATT_TREE = 2 };

template <typename T, int HD, int QT, int TPW, int MODE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_attention(AttnArgs a) {
  constexpr bool SPEC = MODE == ATT_SPEC;
  // packed draft tree: a row sees positions below its rotary position (the committed prefix and
  // its ancestors on the top-1 chain) and its own cache slot
  constexpr bool TREE = MODE == ATT_TREE;
  constexpr int DS = HD / 32;    // 32-dim steps of S^T
  constexpr int DT = HD / 16;    // 16-dim tiles of O^T
  constexpr int PS = HD + 4;     // floats per query vector in a group partial
  constexpr int SPAN = ATT_WAVES * TPW * 16;
  // run partials for the in-group merge; rows padded by 4 floats so that the 16 query lanes
  // reading one column fall in different banks
  // run partials for the in-group merge, [wave][query vector][HD + 4] (+ m, l), sized by the
  // launcher for the launch's query vectors per row-block; rows padded by 4 floats so that the 16
  // query lanes reading one column fall in different banks
  extern __shared__ __attribute__((aligned(16))) float att_lds[];
  const int NQ = a.nq_alloc;
  float* s_o = att_lds;                               // [ATT_WAVES][NQ][HD + 4]
  float* s_ml = att_lds + ATT_WAVES * NQ * (HD + 4);  // [ATT_WAVES][NQ][2]
#define S_O(w_, q_, d_) s_o[((w_) * NQ + (q_)) * (HD + 4) + (d_)]
#define S_ML(w_, q_, i_) s_ml[((w_) * NQ + (q_)) * 2 + (i_)]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tl = lane & 15, kg = lane >> 4;
  const int g = blockIdx.x;
  const int h = blockIdx.y % a.n_kv, rb = blockIdx.y / a.n_kv;
  const int b = blockIdx.z;
  const int r0 = rb * a.RB;
  if (r0 >= a.R) return;
  const int nr = min(a.RB, a.R - r0);
  const int nqv = nr * a.G;
  const int mrow0 = b * a.R + r0;
  const int qstride = a.n_heads * HD;
  const int P0 = (g * ATT_WAVES + wave) * TPW * 16;   // first position of this wave's run
  const T* kvp = reinterpret_cast<const T*>(a.kv);
  const int* btp = a.bt + b * a.bt_stride;   // the grid covers exactly bt_stride * 16 positions
  const size_t layer_base = (size_t)a.layer * a.n_blocks;

  // ---- round trip 1: the last row's position, the run's block-table entries, the queries ----
  const int maxpos = TREE ? a.row_slot[mrow0 + nr - 1] : a.row_pos[mrow0 + nr - 1];
  // block-causal pass: the first and last rows' block starts bound which tiles need which cache
  const int s_first = SPEC ? (a.row_pos[mrow0] / a.s_block) * a.s_block : 0;
  const int s_last = SPEC ? (maxpos / a.s_block) * a.s_block : 0;
  int blk[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) blk[t] = btp[(P0 >> 4) + t];
  // positions of the lane's query columns qv = qt*16 + tl (loaded from a valid row, masked later)
  int qpos[QT], qstart[QT], qslot[QT];
  bool qok[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qv = qt * 16 + tl;
    qok[qt] = qv < nqv;
    const int rl = qok[qt] ? qv / a.G : 0;
    qpos[qt] = a.row_pos[mrow0 + rl];
    qslot[qt] = TREE ? a.row_slot[mrow0 + rl] : 0;
  }
  // the queries, shared by the 4 waves: thread i loads the 8 values of B-operand slots
  // i, i + 256, .. (slot (qt, ds, lane) = query column qt*16 + (lane & 15), dims ds*32 +
  // (lane >> 4)*8 .. +7), branch-free from a valid row
  constexpr int QSLOTS = QT * DS * 64, QPT = (QSLOTS + 255) / 256;
  float qraw[QPT][8];
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int sl = u * 256 + (int)threadIdx.x, sc = sl < QSLOTS ? sl : 0;
    const int qv = (sc / (DS * 64)) * 16 + (sc & 15), ds = (sc / 64) % DS, kq = (sc >> 4) & 3;
    const int rl = qv < nqv ? qv / a.G : 0, gq = qv < nqv ? qv - rl * a.G : 0;
    load8(a.q + (size_t)(mrow0 + rl) * qstride + (h * a.G + gq) * HD + ds * 32 + kq * 8, qraw[u]);
  }
  __builtin_amdgcn_sched_barrier(0);
  const int n_groups = maxpos / SPAN + 1;
  if (g >= n_groups) return;
  const int n_live = P0 > maxpos ? 0 : min(TPW, ((maxpos - P0) >> 4) + 1);   // tiles with a visible position

  // ---- round trip 2: the run's K and V tiles ----
  // K: lane (tl, kg) holds K[position tl][d = ds*32 + kg*8 + j]; V^T: lane holds V[positions
  // 4kg..4kg+3][d = dt*16 + tl] (the cache keeps V transposed per block)
  typename ET<T>::A kf[TPW][DS];
  typename PV<T>::A vf[TPW][DT];
  // block-causal pass: the pass's own keys/values of the same tiles, and which caches each tile
  // needs (deep: some row's block starts after the tile's first position; shallow: some row's
  // block starts at or before its last position)
  typename ET<T>::A kfs[SPEC ? TPW : 1][DS];
  typename PV<T>::A vfs[SPEC ? TPW : 1][DT];
  bool need_deep[TPW], need_sh[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int T0 = P0 + 16 * t;
    need_deep[t] = !SPEC || T0 < s_last;
    need_sh[t] = SPEC && T0 + 15 >= s_first;
    if (t < n_live && need_deep[t]) {
      const T* kp = kvp + (((layer_base + blk[t]) * 2 + 0) * a.n_kv + h) * 16 * HD + tl * HD + kg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[t][ds] = ET<T>::load(kp + ds * 32);
      const T* vp = kvp + (((layer_base + blk[t]) * 2 + 1) * a.n_kv + h) * HD * 16 + tl * 16 + 4 * kg;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vf[t][dt] = PV<T>::load(vp + dt * 16 * 16);
    }
    if constexpr (SPEC) {
      if (t < n_live && need_sh[t]) {
        const T* sp = reinterpret_cast<const T*>(a.skv);
        const size_t sb = (size_t)a.s_layer * a.s_n_blocks + (T0 >> 4);
        const T* kp = sp + ((sb * 2 + 0) * a.n_kv + h) * 16 * HD + tl * HD + kg * 8;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) kfs[t][ds] = ET<T>::load(kp + ds * 32);
        const T* vp = sp + ((sb * 2 + 1) * a.n_kv + h) * HD * 16 + tl * 16 + 4 * kg;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) vfs[t][dt] = PV<T>::load(vp + dt * 16 * 16);
      }
    }
  }
  // keep every K/V load here, ahead of all arithmetic: left to itself the scheduler trades them
  // for registers and sinks them into the MFMA sequence, one round trip at a time
  __builtin_amdgcn_sched_barrier(0);

  // ---- queries scaled by log2(e)/sqrt(d), as bf16 hi/lo B operands, parked in LDS (in the
  // space of the run partials, which are written only after the last tile) so that the K/V
  // fragments of every tile fit the registers of two waves per SIMD ----
  typedef typename ET<T>::B QB;
  QB* s_q = reinterpret_cast<QB*>(att_lds);   // the launcher sizes the buffer for these too
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int sl = u * 256 + (int)threadIdx.x;
    if (sl < QSLOTS) {
      const bool ok = (sl / (DS * 64)) * 16 + (sl & 15) < nqv;
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = ok ? qraw[u][j] * a.scale_log2 : 0.f;
      s_q[sl] = ET<T>::split(x);
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    if (!qok[qt]) {
      qpos[qt] = -1;
      qslot[qt] = -1;
    }
    // block-causal pass: positions below qstart come from the deep cache
    qstart[qt] = SPEC ? (qpos[qt] / a.s_block) * a.s_block : 0;
  }
  __syncthreads();
  // read per use: an offset the compiler cannot see through keeps it from hoisting the fragments
  // of every tile into registers (which would cost the second wave per SIMD again)
  int q_off = 0;
  auto qf = [&](int qt, int ds) -> QB { return s_q[q_off + (qt * DS + ds) * 64 + lane]; };

  // ---- online softmax over the run's tiles, left to right ----
  float m_c[QT], l_c[QT];
  f32x4 o_c[QT][DT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_c[qt] = NEG_INF;
    l_c[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o_c[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    if (t >= n_live) break;
    asm volatile("" : "+v"(q_off));
    f32x4 sacc[QT], ssh[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      sacc[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
      ssh[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (need_deep[t]) {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) ET<T>::mma(sacc[qt], kf[t][ds], qf(qt, ds));
    }
    if constexpr (SPEC) {
      if (need_sh[t]) {
#pragma unroll
        for (int ds = 0; ds < DS; ++ds)
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) ET<T>::mma(ssh[qt], kfs[t][ds], qf(qt, ds));
      }
    }
    typename PV<T>::B pf[QT], pfs[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float s[4], mx = NEG_INF;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int pos = P0 + 16 * t + 4 * kg + i;
        if constexpr (SPEC) s[i] = (pos > qpos[qt]) ? NEG_INF : (pos < qstart[qt] ? sacc[qt][i] : ssh[qt][i]);
        else if constexpr (TREE) s[i] = (pos < qpos[qt] || pos == qslot[qt]) ? sacc[qt][i] : NEG_INF;
        else s[i] = (pos <= qpos[qt]) ? sacc[qt][i] : NEG_INF;
        mx = fmaxf(mx, s[i]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_n = fmaxf(m_c[qt], mx);
      // m_n = -inf: nothing visible so far; the running state stays the identity
      const float alpha = (m_c[qt] == NEG_INF) ? 0.f : exp2f(m_c[qt] - m_n);
      float p[4], sum = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = (m_n == NEG_INF) ? 0.f : exp2f(s[i] - m_n);
        sum += p[i];
      }
      sum += __shfl_xor(sum, 16);
      sum += __shfl_xor(sum, 32);
      l_c[qt] = l_c[qt] * alpha + sum;
      m_c[qt] = m_n;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) o_c[qt][dt][i] *= alpha;
      if constexpr (SPEC) {
        float pd[4], ps[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool deep = P0 + 16 * t + 4 * kg + i < qstart[qt];
          pd[i] = deep ? p[i] : 0.f;
          ps[i] = deep ? 0.f : p[i];
        }
        pf[qt] = PV<T>::split(pd);
        pfs[qt] = PV<T>::split(ps);
      } else {
        pf[qt] = PV<T>::split(p);
      }
    }
    if (need_deep[t]) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) PV<T>::mma(o_c[qt][dt], vf[t][dt], pf[qt]);
    }
    if constexpr (SPEC) {
      if (need_sh[t]) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) PV<T>::mma(o_c[qt][dt], vfs[t][dt], pfs[qt]);
      }
    }
  }

  // ---- merge the group's 4 runs left to right: every wave parks its run partial in LDS (lane
  // (qv, kg) holds dims dt*16 + 4kg..+3), then thread e merges query vector e / (HD/4),
  // columns 4*(e mod HD/4).., run 0 first ----
  __syncthreads();   // every wave is done with the query fragments under s_o
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qv = qt * 16 + tl;
    if (qv >= nqv) continue;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(&S_O(wave, qv, dt * 16 + 4 * kg)) =
          make_float4(o_c[qt][dt][0], o_c[qt][dt][1], o_c[qt][dt][2], o_c[qt][dt][3]);
    if (kg == 0) {
      S_ML(wave, qv, 0) = m_c[qt];
      S_ML(wave, qv, 1) = l_c[qt];
    }
  }
  __syncthreads();
  float* part = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.n_groups_max + g) * 32) * PS;
  constexpr int HD4 = HD / 4;
  for (int e = threadIdx.x; e < nqv * HD4; e += blockDim.x) {
    const int qv = e / HD4, d = (e - qv * HD4) * 4;
    const float4 v0 = *reinterpret_cast<const float4*>(&S_O(0, qv, d));
    float m_r = S_ML(0, qv, 0), l_r = S_ML(0, qv, 1), o_r[4] = {v0.x, v0.y, v0.z, v0.w};
#pragma unroll
    for (int w = 1; w < ATT_WAVES; ++w) {
      const float4 v = *reinterpret_cast<const float4*>(&S_O(w, qv, d));
      const float oc[4] = {v.x, v.y, v.z, v.w};
      softmax_merge(m_r, l_r, o_r, S_ML(w, qv, 0), S_ML(w, qv, 1), oc, 4);
    }
    if (n_groups == 1) {
      // the only group: the merge of groups reduces to o / l for it (weight 1), so finish here
      const int rl = qv / a.G, gq = qv - rl * a.G;
      *reinterpret_cast<float4*>(a.out + (size_t)(mrow0 + rl) * qstride + (h * a.G + gq) * HD + d) =
          make_float4(o_r[0] / l_r, o_r[1] / l_r, o_r[2] / l_r, o_r[3] / l_r);
    } else {
      float* pp = part + (size_t)qv * PS;
      *reinterpret_cast<float4*>(pp + d) = make_float4(o_r[0], o_r[1], o_r[2], o_r[3]);
      if (d == 0) *reinterpret_cast<float2*>(pp + HD) = make_float2(m_r, l_r);
    }
  }
}

#undef S_O
#undef S_ML

// Merge of the group partials: an 8-lane team per (query vector, 4 columns). Lane j merges groups
// j, j+8, .. left to right from the identity (4 groups' loads in flight at a time), then the team
// merges pairwise with a fixed butterfly; both lanes of a pair compute merge(lower, upper).
template <int HD>
__global__ void __launch_bounds__(256) k_attn_combine(AttnArgs a) {
  constexpr int PS = HD + 4, HD4 = HD / 4;
  const int h = blockIdx.y % a.n_kv, rb = blockIdx.y / a.n_kv;
  const int b = blockIdx.z;
  const int r0 = rb * a.RB;
  if (r0 >= a.R) return;
  const int nr = min(a.RB, a.R - r0);
  const int nqv = nr * a.G;
  const int mrow0 = b * a.R + r0;
  const int gid = blockIdx.x * blockDim.x + threadIdx.x;
  const int item = gid / CMB_LANES, j = gid % CMB_LANES;
  const int qv = item / HD4, d = (item - qv * HD4) * 4;
  if (qv >= nqv) return;   // the 8 lanes of an item leave together
  // the same group count as k_attention: a tree's rows reach their cache slots, not positions
  const int n_groups = (a.tree ? a.row_slot[mrow0 + nr - 1] : a.row_pos[mrow0 + nr - 1]) / a.span + 1;
  if (n_groups == 1) return;   // k_attention wrote the final output
  const float* pq = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.n_groups_max) * 32 + qv) * PS;
  float m_r = NEG_INF, l_r = 0.f, o_r[4] = {0.f, 0.f, 0.f, 0.f};
  for (int g0 = j; g0 < n_groups; g0 += CMB_INFLIGHT * CMB_LANES) {
    float4 ov[CMB_INFLIGHT];
    float2 ml[CMB_INFLIGHT];
#pragma unroll
    for (int u = 0; u < CMB_INFLIGHT; ++u) {
      const float* pp = pq + (size_t)min(g0 + u * CMB_LANES, n_groups - 1) * 32 * PS;
      ov[u] = *reinterpret_cast<const float4*>(pp + d);
      ml[u] = *reinterpret_cast<const float2*>(pp + HD);
    }
#pragma unroll
    for (int u = 0; u < CMB_INFLIGHT; ++u) {
      if (g0 + u * CMB_LANES < n_groups) {
        const float oc[4] = {ov[u].x, ov[u].y, ov[u].z, ov[u].w};
        softmax_merge(m_r, l_r, o_r, ml[u].x, ml[u].y, oc, 4);
      }
    }
  }
#pragma unroll
  for (int s = 1; s < CMB_LANES; s <<= 1) {
    const float pm = __shfl_xor(m_r, s), pl = __shfl_xor(l_r, s);
    float po[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) po[i] = __shfl_xor(o_r[i], s);
    const bool upper = j & s;
    float am = upper ? pm : m_r, al = upper ? pl : l_r, ao[4], bo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ao[i] = upper ? po[i] : o_r[i];
      bo[i] = upper ? o_r[i] : po[i];
    }
    softmax_merge(am, al, ao, upper ? m_r : pm, upper ? l_r : pl, bo, 4);
    m_r = am;
    l_r = al;
#pragma unroll
    for (int i = 0; i < 4; ++i) o_r[i] = ao[i];
  }
  if (j == 0) {
    const int rl = qv / a.G, gq = qv - rl * a.G;
    *reinterpret_cast<float4*>(a.out + (size_t)(mrow0 + rl) * a.n_heads * HD + (h * a.G + gq) * HD + d) =
        make_float4(o_r[0] / l_r, o_r[1] / l_r, o_r[2] / l_r, o_r[3] / l_r);
  }
}

// Causal attention of a wide single-sequence pass (the prompt's prefill, more than 64 rows at a
// time). The decode kernel above spreads a row-block's positions over groups of workgroups and
// merges their partials in a second launch, which suits a few rows over a long cache; across a
// whole prompt it re-reads every key/value once per 32-query-vector row-block and writes a partial
// per group. Here a workgroup owns 64 query vectors (64 / G rows of the G query heads of one KV
// head, one 16-vector tile per wave) and each wave streams every visible 16-position tile in
// order with an online softmax (the same per-tile contractions, masking and base-2 softmax as the
// decode kernel), so the output is written directly: no partials, no merge launch, and each tile
// is fetched from memory once per workgroup (the four waves read it from the CU's cache).
// Tiles are loaded two ahead into registers; every load is issued unconditionally (a tile past the
// last visible one reloads that tile and is fully masked), and the block table is staged in LDS so
// that no key/value address waits on a global load.
// The block-causal variant (SPEC: the drafting objective's decoder pass) contracts every tile with
// both caches, the deep one below each query's block start and the pass's own one from there to
// the query, and selects per (query, position) as the decode kernel's SPEC variant does.
template <typename T, int HD, bool SPEC>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_attention_prefill(AttnArgs a) {
  constexpr int DS = HD / 32, DT = HD / 16, NC = SPEC ? 2 : 1;
  extern __shared__ int s_bt[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tl = lane & 15, kg = lane >> 4;
  const int rows_wg = 64 / a.G;
  const int n_rbp = (a.R + rows_wg - 1) / rows_wg;
  // the row-blocks with the most tiles first, so that the short ones fill the tail
  const int rbp = n_rbp - 1 - (int)blockIdx.x / a.n_kv, h = (int)blockIdx.x % a.n_kv;
  const int r0 = rbp * rows_wg, nr = min(rows_wg, a.R - r0);
  const int maxpos = a.row_pos[r0 + nr - 1];
  const int t_last = maxpos >> 4;
  for (int i0 = 0; i0 <= t_last; i0 += 4 * (int)blockDim.x) {   // 4 entries per thread in flight
    int e[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) e[u] = a.bt[min(i0 + u * (int)blockDim.x + (int)threadIdx.x, t_last)];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * (int)blockDim.x + (int)threadIdx.x;
      if (i <= t_last) s_bt[i] = e[u];
    }
  }

  // this lane's query vector qv = wave*16 + tl: row qv / G, head qv % G of the KV head's group
  const int qv = wave * 16 + tl;
  const bool qok = qv < nr * a.G;
  const int rl = qok ? qv / a.G : 0, gq = qok ? qv - (qv / a.G) * a.G : 0;
  const int qpos = qok ? a.row_pos[r0 + rl] : -1;
  const int qstart = SPEC ? (qpos < 0 ? 0 : (qpos / a.s_block) * a.s_block) : 0;
  const int qstride = a.n_heads * HD;
  const float* qp = a.q + (size_t)(r0 + rl) * qstride + (h * a.G + gq) * HD;
  typename ET<T>::B qf[DS];
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) {
    float x[8];
    load8(qp + ds * 32 + kg * 8, x);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = qok ? x[j] * a.scale_log2 : 0.f;
    qf[ds] = ET<T>::split(x);
  }
  // positions split over a.pf_split workgroups: this one streams tiles [t0, t_end) and, when the
  // pass is split, writes an unnormalised partial that k_prefill_merge combines
  const int n_split = a.pf_split, ks = blockIdx.y;
  const int t0 = ks * (t_last + 1) / n_split, t_end = (ks + 1) * (t_last + 1) / n_split;
  const size_t pidx = ((size_t)ks * a.R + r0 + rl) * a.n_heads + h * a.G + gq;   // (split, row, head)
  if (t_end <= t0) {   // no tile here (every wave of the workgroup takes this branch): the merge's identity
    if (qok) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<float4*>(a.pf_o + pidx * HD + dt * 16 + 4 * kg) = make_float4(0.f, 0.f, 0.f, 0.f);
      if (kg == 0) *reinterpret_cast<float2*>(a.pf_ml + pidx * 2) = make_float2(NEG_INF, 0.f);
    }
    return;
  }
  __syncthreads();   // the block table is in LDS

  const T* kvp = reinterpret_cast<const T*>(a.kv);
  const size_t layer_base = (size_t)a.layer * a.n_blocks;
  typedef typename ET<T>::A KA;
  typedef typename PV<T>::A VA;
  // cache 0: the deep cache through the block table; cache 1 (SPEC): the pass's own, by position
  auto load_tile = [&](KA (&kf)[NC][DS], VA (&vf)[NC][DT], int t) {
    const int tc = min(t, t_end - 1);
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const T* base = cc == 0 ? kvp : reinterpret_cast<const T*>(a.skv);
      const size_t blk = cc == 0 ? layer_base + s_bt[tc] : (size_t)a.s_layer * a.s_n_blocks + tc;
      const T* kp = base + ((blk * 2 + 0) * a.n_kv + h) * 16 * HD + tl * HD + kg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[cc][ds] = ET<T>::load(kp + ds * 32);
      const T* vp = base + ((blk * 2 + 1) * a.n_kv + h) * HD * 16 + tl * 16 + 4 * kg;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vf[cc][dt] = PV<T>::load(vp + dt * 16 * 16);
    }
  };
  float m_c = NEG_INF, l_c = 0.f;
  f32x4 o_c[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o_c[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto consume = [&](const KA (&kf)[NC][DS], const VA (&vf)[NC][DT], int t) {
    f32x4 sacc[NC];
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      sacc[cc] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) ET<T>::mma(sacc[cc], kf[cc][ds], qf[ds]);
    }
    float sv[4], mx = NEG_INF;
    const bool tv = t < t_end;   // a tile past this workgroup's range is masked whole
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int pos = 16 * t + 4 * kg + i;
      if constexpr (SPEC) sv[i] = (!tv || pos > qpos) ? NEG_INF : (pos < qstart ? sacc[0][i] : sacc[1][i]);
      else sv[i] = (tv && pos <= qpos) ? sacc[0][i] : NEG_INF;
      mx = fmaxf(mx, sv[i]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_n = fmaxf(m_c, mx);
    const float alpha = (m_c == NEG_INF) ? 0.f : exp2f(m_c - m_n);
    float pr[4], sum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pr[i] = (m_n == NEG_INF) ? 0.f : exp2f(sv[i] - m_n);
      sum += pr[i];
    }
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    l_c = l_c * alpha + sum;
    m_c = m_n;
    typename PV<T>::B pf[NC];
    if constexpr (SPEC) {
      float pd[4], ps[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool deep = 16 * t + 4 * kg + i < qstart;
        pd[i] = deep ? pr[i] : 0.f;
        ps[i] = deep ? 0.f : pr[i];
      }
      pf[0] = PV<T>::split(pd);
      pf[NC - 1] = PV<T>::split(ps);
    } else {
      pf[0] = PV<T>::split(pr);
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o_c[dt][i] *= alpha;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) PV<T>::mma(o_c[dt], vf[cc][dt], pf[cc]);
    }
  };

  if constexpr (sizeof(T) == 2) {
    // bf16 caches: each tile is fetched once per workgroup (one 16-byte key chunk and one value
    // chunk per thread and cache) and staged in LDS, from which every wave reads its fragments,
    // instead of each wave fetching the whole tile for itself (a quarter of the memory requests).
    // RD register stages keep RD - 1 tiles in flight; tiles alternate between two LDS slots, one
    // barrier per tile. Key chunk c of position row r sits at column c ^ kswz(r) of its row and
    // value chunk c of dim row d at c ^ ((d >> 3) & 1), so the 16 rows a fragment read touches fall
    // on distinct banks.
    constexpr int CPR = HD / 8;            // 16-byte chunks per key row (one position)
    constexpr int NKC = 16 * CPR;          // key chunks per tile and cache
    constexpr int NCH = 2 * NKC;           // key and value chunks per tile and cache
    constexpr int TB = NCH * 16;           // bytes per tile and cache
    constexpr int CPT = NC * NCH / 256;    // chunks per thread and tile
    static_assert(NC * NCH % 256 == 0, "whole chunks per thread");
    constexpr int RD = 4;                  // register stages r0..r3 below
    char* stage = reinterpret_cast<char*>(s_bt) + prefill_bt_bytes(a.bt_stride);
    auto kswz = [](int r) { return (r * CPR / 16) % CPR; };
    auto gload = [&](u32x4 (&rg)[CPT], int t) __attribute__((always_inline)) {
      const int tc = min(t, t_end - 1);
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int q = u * 256 + (int)threadIdx.x, cc = q / NCH, qq = q - cc * NCH;
        const T* base = cc == 0 ? kvp : reinterpret_cast<const T*>(a.skv);
        const size_t blk = cc == 0 ? layer_base + s_bt[tc] : (size_t)a.s_layer * a.s_n_blocks + tc;
        const int r = qq / CPR, kc = (qq % CPR) ^ kswz(r);
        const int d = (qq - NKC) >> 1, vc = ((qq - NKC) & 1) ^ ((d >> 3) & 1);
        const T* src = qq < NKC ? base + ((blk * 2 + 0) * a.n_kv + h) * 16 * HD + r * HD + kc * 8
                                : base + ((blk * 2 + 1) * a.n_kv + h) * HD * 16 + d * 16 + vc * 8;
        rg[u] = *reinterpret_cast<const u32x4*>(src);
      }
    };
    auto lstore = [&](const u32x4 (&rg)[CPT], int slot) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < CPT; ++u)   // chunk q = cc * NCH + qq at byte 16 q of the slot
        *reinterpret_cast<u32x4*>(stage + (size_t)slot * NC * TB + (size_t)(u * 256 + threadIdx.x) * 16) = rg[u];
    };
    auto lfrag = [&](KA (&kf)[NC][DS], VA (&vf)[NC][DT], int slot) __attribute__((always_inline)) {
      const char* sb = stage + (size_t)slot * NC * TB;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
#pragma unroll
        for (int ds = 0; ds < DS; ++ds)
          kf[cc][ds].v = *reinterpret_cast<const uint4*>(sb + cc * TB + tl * (HD * 2) + ((ds * 4 + kg) ^ kswz(tl)) * 16);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const int d = dt * 16 + tl;
          vf[cc][dt].v = *reinterpret_cast<const uint2*>(sb + cc * TB + NKC * 16 + d * 32 +
                                                          (((kg >> 1) ^ ((d >> 3) & 1)) * 16) + (kg & 1) * 8);
        }
      }
    };
    // register stages, named so that every index is a constant (tile j lives in stage j mod RD)
    u32x4 r0[CPT], r1[CPT], r2[CPT], r3[CPT];
    gload(r0, t0);   // each tile's loads strictly after the previous tile's
    __builtin_amdgcn_sched_barrier(0);
    gload(r1, t0 + 1);
    __builtin_amdgcn_sched_barrier(0);
    gload(r2, t0 + 2);
    __builtin_amdgcn_sched_barrier(0);
    gload(r3, t0 + 3);
    __builtin_amdgcn_sched_barrier(0);
    lstore(r0, 0);
    gload(r0, t0 + RD);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // tile tt from slot (tt - t0) & 1 (past t_end: the last tile again, every position masked); then tile
    // tt + 1, fetched RD - 1 tiles ago into stage `next`, into the other slot (whose previous tile
    // every wave finished before the last barrier), and `next` refilled with tile tt + 1 + RD
    auto step = [&](int tt, int slot, u32x4 (&next)[CPT]) __attribute__((always_inline)) {
      KA kf[NC][DS];
      VA vf[NC][DT];
      lfrag(kf, vf, slot);
      consume(kf, vf, tt);
      __builtin_amdgcn_sched_barrier(0);
      lstore(next, slot ^ 1);
      gload(next, tt + 1 + RD);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
    };
    for (int t = t0; t < t_end; t += RD) {
      step(t, 0, r1);
      step(t + 1, 1, r2);
      step(t + 2, 0, r3);
      step(t + 3, 1, r0);
    }
  } else {
    KA ka[NC][DS], kb[NC][DS];
    VA va[NC][DT], vb[NC][DT];
    // tile 0's loads strictly before tile 1's, here as in the loop: if the scheduler issued them
    // in the other order, the first use of tile 0 would have to wait for both tiles on every
    // iteration
    load_tile(ka, va, t0);
    __builtin_amdgcn_sched_barrier(0);
    load_tile(kb, vb, t0 + 1);
    __builtin_amdgcn_sched_barrier(0);
    for (int t = t0; t < t_end; t += 2) {
      consume(ka, va, t);
      load_tile(ka, va, t + 2);
      __builtin_amdgcn_sched_barrier(0);
      consume(kb, vb, t + 1);   // past t_last: the last tile again, every position masked
      load_tile(kb, vb, t + 3);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // lane (qv, kg) holds dims dt*16 + 4kg .. +3 of query vector qv
  if (qok && n_split == 1) {
    float* op = a.out + (size_t)(r0 + rl) * qstride + (h * a.G + gq) * HD;
    const float inv = 1.f / l_c;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(op + dt * 16 + 4 * kg) =
          make_float4(o_c[dt][0] * inv, o_c[dt][1] * inv, o_c[dt][2] * inv, o_c[dt][3] * inv);
  } else if (qok) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(a.pf_o + pidx * HD + dt * 16 + 4 * kg) =
          make_float4(o_c[dt][0], o_c[dt][1], o_c[dt][2], o_c[dt][3]);
    if (kg == 0) *reinterpret_cast<float2*>(a.pf_ml + pidx * 2) = make_float2(m_c, l_c);
  }
}

// The partials of a split one-launch pass merged in split order (the online-softmax merge),
// normalised and written: one thread per (row, head, 4 dims).
__global__ void __launch_bounds__(256) k_prefill_merge(AttnArgs a) {
  const int hd4 = a.head_dim / 4;
  const long long rh_n = (long long)a.R * a.n_heads;
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= rh_n * hd4) return;
  const long long rh = e / hd4;   // row * n_heads + head
  const int d = (int)(e - rh * hd4) * 4;
  float m = NEG_INF, l = 0.f, o[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < a.pf_split; ++k) {
    const size_t pi = (size_t)k * rh_n + rh;
    const float2 ml = *reinterpret_cast<const float2*>(a.pf_ml + pi * 2);
    const float4 v = *reinterpret_cast<const float4*>(a.pf_o + pi * a.head_dim + d);
    const float ov[4] = {v.x, v.y, v.z, v.w};
    softmax_merge(m, l, o, ml.x, ml.y, ov, 4);
  }
  const float inv = 1.f / l;
  *reinterpret_cast<float4*>(a.out + rh * a.head_dim + d) = make_float4(o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
}

template <typename Kern>
static void launch_kernel(Kern k, dim3 grid, hipStream_t s, const LaunchEvents* ev, const AttnArgs& a,
                          size_t lds = 0) {
  if (ev) hipExtLaunchKernelGGL(k, grid, dim3(256), (uint32_t)lds, s, ev->start, ev->stop, 0, a);
  else hipLaunchKernelGGL(k, grid, dim3(256), lds, s, a);
}

// LDS of one attention workgroup: the 4 waves' run partials for the launch's query vectors per
// row-block (at most 32), and at least the queries' B-operand fragments parked there first
template <typename T, int HD, int QT>
static size_t attention_lds(int nq) {
  const size_t parts = (size_t)ATT_WAVES * nq * (HD + 4) * 4 + (size_t)ATT_WAVES * nq * 2 * 4;
  const size_t qfrag = (size_t)QT * (HD / 32) * 64 * sizeof(typename ET<T>::B);
  return std::max(parts, qfrag);
}

template <typename T, int HD, int QT, int MODE>
static void launch_attention_qt(const AttnArgs& a0, hipStream_t s, const LaunchEvents* ev) {
  AttnArgs a = a0;
  a.nq_alloc = std::min(a.RB, a.R) * a.G;   // query vectors of the widest row-block
  const size_t lds = attention_lds<T, HD, QT>(a.nq_alloc);
  const dim3 grid(a.n_groups_max, a.n_kv * a.n_rb, a.B);
  switch (a.span) {
    case 64: launch_kernel(k_attention<T, HD, QT, 1, MODE>, grid, s, ev, a, lds); break;
    case 128: launch_kernel(k_attention<T, HD, QT, 2, MODE>, grid, s, ev, a, lds); break;
    default: launch_kernel(k_attention<T, HD, QT, 4, MODE>, grid, s, ev, a, lds); break;
  }
}

template <typename T, int HD>
static void launch_attention_hd(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  const bool q2 = std::min(a.RB, a.R) * a.G > 16;
  if (a.s_block > 0) {
    if (q2) launch_attention_qt<T, HD, 2, ATT_SPEC>(a, s, ev);
    else launch_attention_qt<T, HD, 1, ATT_SPEC>(a, s, ev);
  } else if (a.tree) {
    if (q2) launch_attention_qt<T, HD, 2, ATT_TREE>(a, s, ev);
    else launch_attention_qt<T, HD, 1, ATT_TREE>(a, s, ev);
  } else {
    if (q2) launch_attention_qt<T, HD, 2, ATT_CAUSAL>(a, s, ev);
    else launch_attention_qt<T, HD, 1, ATT_CAUSAL>(a, s, ev);
  }
}

// One sequence: 64 positions per group up to 4096 (at its ~1.2k-position context, 1024-token
// prompt, 128-position groups leave half the 160 workgroups of a launch out: verification
// attention 7.9 -> 9.6 us per layer). Several sequences fill the chip sooner: 64 up to 2048, then
// 128 (batch 8 at ~2300 positions: verification attention 19.7 -> 17.4 us per layer and its merge
// 9.3 -> 7.6 us against 64; 256 gave 19.3). 256 beyond 8192 positions (16k contexts).
int attention_span(int max_ctx, int max_batch) {
  const int small = max_batch == 1 ? 4096 : 2048;
  return max_ctx <= small ? 64 : (max_ctx <= 8192 ? 128 : 256);
}

template <typename T>
void launch_attention(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  if (a.head_dim == 128) launch_attention_hd<T, 128>(a, s, ev);
  else launch_attention_hd<T, 64>(a, s, ev);
}

// LDS of one prefill workgroup: the block table, then (bf16) two tile slots of both caches
static size_t prefill_lds(const AttnArgs& a, bool bf16) {
  const size_t tile = (size_t)2 * 16 * a.head_dim * 2 * (a.s_block > 0 ? 2 : 1);
  return prefill_bt_bytes(a.bt_stride) + (bf16 ? 2 * tile : 0);
}

bool attention_prefill_supported(const AttnArgs& a) {
  // the block table must fit LDS beside the tile slots (capacities up to ~131k positions); longer
  // ones take the split-KV kernel
  return a.B == 1 && a.G >= 1 && 64 % a.G == 0 && (a.head_dim == 128 || a.head_dim == 64) && !a.tree &&
         prefill_lds(a, true) <= 65536;
}

template <typename T>
void launch_attention_prefill(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  const int rows_wg = 64 / a.G;
  const dim3 grid((unsigned)(((a.R + rows_wg - 1) / rows_wg) * a.n_kv), (unsigned)a.pf_split);
  const size_t lds = prefill_lds(a, sizeof(T) == 2);
  const LaunchEvents e0{ev ? ev->start : nullptr, nullptr}, e1{nullptr, ev ? ev->stop : nullptr};
  const LaunchEvents* ea = ev ? (a.pf_split > 1 ? &e0 : ev) : nullptr;
  if (a.s_block > 0) {
    if (a.head_dim == 128) launch_kernel(k_attention_prefill<T, 128, true>, grid, s, ea, a, lds);
    else launch_kernel(k_attention_prefill<T, 64, true>, grid, s, ea, a, lds);
  } else {
    if (a.head_dim == 128) launch_kernel(k_attention_prefill<T, 128, false>, grid, s, ea, a, lds);
    else launch_kernel(k_attention_prefill<T, 64, false>, grid, s, ea, a, lds);
  }
  if (a.pf_split > 1) {
    const long long items = (long long)a.R * a.n_heads * (a.head_dim / 4);
    launch_kernel(k_prefill_merge, dim3((unsigned)((items + 255) / 256)), s, ev ? &e1 : nullptr, a);
  }
}

bool attention_needs_combine(const AttnArgs& a) { return a.n_groups_max > 1; }

void launch_attn_combine(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  const int items = 32 * (a.head_dim / 4) * CMB_LANES;
  const dim3 grid((items + 255) / 256, a.n_kv * a.n_rb, a.B);
  if (a.head_dim == 128) launch_kernel(k_attn_combine<128>, grid, s, ev, a);
  else launch_kernel(k_attn_combine<64>, grid, s, ev, a);
}

template void launch_attention<uint16_t>(const AttnArgs&, hipStream_t, const LaunchEvents*);
template void launch_attention<float>(const AttnArgs&, hipStream_t, const LaunchEvents*);
template void launch_attention_prefill<uint16_t>(const AttnArgs&, hipStream_t, const LaunchEvents*);
template void launch_attention_prefill<float>(const AttnArgs&, hipStream_t, const LaunchEvents*);

}  // namespace seedk
