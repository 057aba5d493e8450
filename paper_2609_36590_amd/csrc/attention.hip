// Paged split-KV attention on MFMA for the verify, draft and prefill passes.
//
// k_attention: one workgroup = 4 waves = one group of 256 absolute positions (4 chunks of 64) for
// one (sequence b, KV head h, row-block rb). The queries of a row-block (G query heads x RB rows,
// <= 32) are the MFMA B operand. Per chunk, a wave computes S^T = K Q^T with the paged K block
// rows as the A operand, masks positions later than each query's own, takes the chunk softmax in
// base 2, and forms O^T = V^T P^T with the transposed V block as the A operand. The wave issues
// its block-table reads together with the row positions, then all K/V loads of its chunk and the
// query loads, so it waits for two memory round trips. The group's 4 chunks are merged left to
// right in LDS and written as one partial (o, m, l), or as the final output when the rows see a
// single group.
//
// k_attn_combine merges the group partials of each query left to right. A chunk or group with no
// visible position is an exact identity of the merge, so a query's result depends only on the
// positions it attends to, not on how many rows share the pass (verify rows vs plain greedy
// decoding give bit-identical outputs).
//
// Position tile pt (16 positions) of chunk base P0, MFMA row r <-> position
//   P0 + 32*(pt>>1) + 8*(r>>2) + (r&3) + 4*(pt&1),
// so after S^T the lane group kg holds positions 8kg..8kg+7 of each 32-position step, which is
// exactly the k-slot layout O^T needs for P^T: no cross-lane shuffle of P.
#include "device_common.h"

#include <algorithm>

namespace seedk {

static constexpr int ATT_CHUNK = 64;
static constexpr int ATT_WAVES = 4;
static constexpr int ATT_GROUP = ATT_CHUNK * ATT_WAVES;

__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int HD, bool COHERENT>
__device__ void merge_groups(const AttnArgs& a, const float* part0, int e, int n_groups, int mrow0, int h);

template <typename T, int HD, int QT>
__global__ void __launch_bounds__(256) k_attention(AttnArgs a) {
  constexpr int DS = HD / 32;    // 32-dim steps of S^T
  constexpr int DT = HD / 16;    // 16-dim tiles of O^T
  constexpr int PS = HD + 4;     // floats per query vector in a group partial
  // chunk partials for the in-group merge; rows padded by 4 floats so that the 16 query lanes
  // reading one column fall in different banks
  __shared__ float s_o[ATT_WAVES][32][HD + 4];
  __shared__ float s_ml[ATT_WAVES][32][2];
  __shared__ int s_last;
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
  const int P0 = (g * ATT_WAVES + wave) * ATT_CHUNK;
  const T* kvp = reinterpret_cast<const T*>(a.kv);
  const int* btp = a.bt + b * a.bt_stride;   // the grid covers exactly bt_stride * 16 positions
  const size_t layer_base = (size_t)a.layer * a.n_blocks;

  // ---- round trip 1: the last row's position and this wave's block-table entries ----
  const int maxpos = a.row_pos[mrow0 + nr - 1];
  int kblk[4], vblk[2];
#pragma unroll
  for (int pt = 0; pt < 4; ++pt) kblk[pt] = btp[(P0 + 32 * (pt >> 1) + 8 * (tl >> 2) + (tl & 3) + 4 * (pt & 1)) >> 4];
#pragma unroll
  for (int s = 0; s < 2; ++s) vblk[s] = btp[(P0 + 32 * s + 8 * kg) >> 4];
  // queries (lane column qv = qt*16 + tl, k-slots d = ds*32 + kg*8 + j) and their positions:
  // loaded branch-free from a valid row, masked when converted
  float qraw[QT][DS][8];
  int qpos[QT];
  bool qok[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qv = qt * 16 + tl;
    qok[qt] = qv < nqv;
    const int rl = qok[qt] ? qv / a.G : 0, gq = qok[qt] ? qv - rl * a.G : 0;
    qpos[qt] = a.row_pos[mrow0 + rl];
    const float* qp = a.q + (size_t)(mrow0 + rl) * qstride + (h * a.G + gq) * HD + kg * 8;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) load8(qp + ds * 32, qraw[qt][ds]);
  }
  __builtin_amdgcn_sched_barrier(0);
  const int n_groups = maxpos / ATT_GROUP + 1;
  if (g >= n_groups) return;
  const bool live = P0 <= maxpos;

  // ---- round trip 2: the chunk's K and V, then the queries ----
  typename ET<T>::A kf[4][DS];
  typename ET<T>::A vf[2][DT];
  if (live) {
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) {
      const int pos = P0 + 32 * (pt >> 1) + 8 * (tl >> 2) + (tl & 3) + 4 * (pt & 1);
      const T* kp = kvp + (((layer_base + kblk[pt]) * 2 + 0) * a.n_kv + h) * 16 * HD + (pos & 15) * HD + kg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[pt][ds] = ET<T>::load(kp + ds * 32);
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int pos = P0 + 32 * s + 8 * kg;
      const T* vp = kvp + (((layer_base + vblk[s]) * 2 + 1) * a.n_kv + h) * HD * 16 + tl * 16 + (pos & 15);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vf[s][dt] = ET<T>::load(vp + dt * 16 * 16);
    }
  }
  // keep every K/V load here, ahead of all arithmetic: left to itself the scheduler trades them
  // for registers and sinks them into the MFMA sequence, one round trip at a time
  __builtin_amdgcn_sched_barrier(0);

  // ---- queries scaled by log2(e)/sqrt(d), as bf16 hi/lo B operands ----
  typename ET<T>::B qf[QT][DS];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    if (!(live && qok[qt])) qpos[qt] = -1;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = (live && qok[qt]) ? qraw[qt][ds][j] * a.scale_log2 : 0.f;
      qf[qt][ds] = ET<T>::split(x);
    }
  }

  float m_c[QT], l_c[QT];
  float o_c[QT][DT][4];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_c[qt] = NEG_INF;
    l_c[qt] = 0.f;
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) o_c[qt][dt][i] = 0.f;

  if (live) {
    // ---- S^T = K Q^T ----
    f32x4 sacc[4][QT];
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) {
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) sacc[pt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) ET<T>::mma(sacc[pt][qt], kf[pt][ds], qf[qt][ds]);
    }
    // ---- mask + chunk softmax (base 2) ----
    float p[QT][4][4];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float mx = NEG_INF;
#pragma unroll
      for (int pt = 0; pt < 4; ++pt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int pos = P0 + 32 * (pt >> 1) + 8 * kg + i + 4 * (pt & 1);
          const float s = (pos <= qpos[qt]) ? sacc[pt][qt][i] : NEG_INF;
          p[qt][pt][i] = s;
          mx = fmaxf(mx, s);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      float sum = 0.f;
#pragma unroll
      for (int pt = 0; pt < 4; ++pt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = (mx == NEG_INF) ? 0.f : exp2f(p[qt][pt][i] - mx);
          p[qt][pt][i] = e;
          sum += e;
        }
      sum += __shfl_xor(sum, 16);
      sum += __shfl_xor(sum, 32);
      m_c[qt] = mx;
      l_c[qt] = sum;
    }
    // ---- O^T = V^T P^T ----
    typename ET<T>::B pf[QT][2];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        float x[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          x[j] = p[qt][2 * s][j];
          x[j + 4] = p[qt][2 * s + 1][j];
        }
        pf[qt][s] = ET<T>::split(x);
      }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        f32x4 oacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 2; ++s) ET<T>::mma(oacc, vf[s][dt], pf[qt][s]);
#pragma unroll
        for (int i = 0; i < 4; ++i) o_c[qt][dt][i] = oacc[i];
      }
  }

  // ---- merge the group's 4 chunks left to right: every wave parks its chunk partial in LDS,
  // then thread e merges query vector e / (HD/4), columns 4*(e mod HD/4).., chunk 0 first ----
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qv = qt * 16 + tl;
    if (qv >= nqv) continue;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(&s_o[wave][qv][dt * 16 + 4 * kg]) =
          make_float4(o_c[qt][dt][0], o_c[qt][dt][1], o_c[qt][dt][2], o_c[qt][dt][3]);
    if (kg == 0) {
      s_ml[wave][qv][0] = m_c[qt];
      s_ml[wave][qv][1] = l_c[qt];
    }
  }
  __syncthreads();
  float* part = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.n_groups_max + g) * 32) * PS;
  constexpr int HD4 = HD / 4;
  for (int e = threadIdx.x; e < nqv * HD4; e += blockDim.x) {
    const int qv = e / HD4, d = (e - qv * HD4) * 4;
    const float4 v0 = *reinterpret_cast<const float4*>(&s_o[0][qv][d]);
    float m_r = s_ml[0][qv][0], l_r = s_ml[0][qv][1], o_r[4] = {v0.x, v0.y, v0.z, v0.w};
#pragma unroll
    for (int w = 1; w < ATT_WAVES; ++w) {
      const float4 v = *reinterpret_cast<const float4*>(&s_o[w][qv][d]);
      const float oc[4] = {v.x, v.y, v.z, v.w};
      softmax_merge(m_r, l_r, o_r, s_ml[w][qv][0], s_ml[w][qv][1], oc, 4);
    }
    if (n_groups == 1) {
      // the only group: the merge of groups reduces to o / l for it (weight 1), so finish here
      const int rl = qv / a.G, gq = qv - rl * a.G;
      *reinterpret_cast<float4*>(a.out + (size_t)(mrow0 + rl) * qstride + (h * a.G + gq) * HD + d) =
          make_float4(o_r[0] / l_r, o_r[1] / l_r, o_r[2] / l_r, o_r[3] / l_r);
    } else if (a.fused_combine) {
      // agent-coherent stores (written through to the level every XCD reads from): the merge of
      // groups runs in this launch
      float* pp = part + (size_t)qv * PS;
#pragma unroll
      for (int i = 0; i < 4; ++i) store_coherent(pp + d + i, o_r[i]);
      if (d == 0) {
        store_coherent(pp + HD, m_r);
        store_coherent(pp + HD + 1, l_r);
      }
    } else {
      // plain stores: k_attn_combine reads them after this launch has ended
      float* pp = part + (size_t)qv * PS;
      *reinterpret_cast<float4*>(pp + d) = make_float4(o_r[0], o_r[1], o_r[2], o_r[3]);
      if (d == 0) *reinterpret_cast<float2*>(pp + HD) = make_float2(m_r, l_r);
    }
  }
  if (n_groups == 1 || !a.fused_combine) return;

  // ---- fused combine: the last group of (b, h, rb) to finish merges all group partials ----
  // Every wave waits for its coherent stores to complete before the barrier; then one relaxed
  // agent-scope count per workgroup (no L2 write-back or invalidate is needed: the partials
  // travel through coherent stores and loads).
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int* cnt = a.cnt + (b * a.n_kv + h) * a.n_rb + rb;
  if (threadIdx.x == 0)
    s_last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_groups - 1;
  __syncthreads();
  if (!s_last) return;
  const float* part0 = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.n_groups_max) * 32) * PS;
  for (int e = threadIdx.x; e < nqv * (HD / 4); e += blockDim.x)
    merge_groups<HD, true>(a, part0, e, n_groups, mrow0, h);
  if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Merge the group partials of query vector e / (HD/4), columns 4*(e mod HD/4).., left to right
// (online softmax merge from the identity, fixed order) and write the normalised output. Each
// batch of 8 groups is loaded at once; COHERENT reads them with agent-coherent loads (the fused
// combine inside k_attention reads partials other workgroups wrote during the same launch).
template <int HD, bool COHERENT>
__device__ void merge_groups(const AttnArgs& a, const float* part0, int e, int n_groups, int mrow0, int h) {
  constexpr int PS = HD + 4, HD4 = HD / 4;
  const int qv = e / HD4, d = (e - qv * HD4) * 4;
  const float* pq = part0 + (size_t)qv * PS;
  float m_r = NEG_INF, l_r = 0.f, o_r[4] = {0.f, 0.f, 0.f, 0.f};
  for (int g0 = 0; g0 < n_groups; g0 += 8) {
    float mg[8], lg[8], og[8][4];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float* pp = pq + (size_t)min(g0 + u, n_groups - 1) * 32 * PS;
      if (COHERENT) {
#pragma unroll
        for (int i = 0; i < 4; ++i) og[u][i] = load_coherent(pp + d + i);
        mg[u] = load_coherent(pp + HD);
        lg[u] = load_coherent(pp + HD + 1);
      } else {
        const float4 v = *reinterpret_cast<const float4*>(pp + d);
        const float2 ml = *reinterpret_cast<const float2*>(pp + HD);
        og[u][0] = v.x; og[u][1] = v.y; og[u][2] = v.z; og[u][3] = v.w;
        mg[u] = ml.x;
        lg[u] = ml.y;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (g0 + u < n_groups) softmax_merge(m_r, l_r, o_r, mg[u], lg[u], og[u], 4);
  }
  const int rl = qv / a.G, gq = qv - rl * a.G;
  *reinterpret_cast<float4*>(a.out + (size_t)(mrow0 + rl) * a.n_heads * HD + (h * a.G + gq) * HD + d) =
      make_float4(o_r[0] / l_r, o_r[1] / l_r, o_r[2] / l_r, o_r[3] / l_r);
}

// Separate merge of the group partials (contexts that can span many groups): thread e of the
// grid's x extent owns one (query vector, 4 columns).
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
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= nqv * HD4) return;
  const int n_groups = a.row_pos[mrow0 + nr - 1] / ATT_GROUP + 1;
  if (n_groups == 1) return;   // k_attention wrote the final output
  const float* part0 = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.n_groups_max) * 32) * PS;
  merge_groups<HD, false>(a, part0, e, n_groups, mrow0, h);
}

template <typename T, int HD>
static void launch_attention_hd(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  const dim3 grid(a.n_groups_max, a.n_kv * a.n_rb, a.B);
  if (std::min(a.RB, a.R) * a.G > 16) {
    if (ev) hipExtLaunchKernelGGL((k_attention<T, HD, 2>), grid, dim3(256), 0, s, ev->start, ev->stop, 0, a);
    else hipLaunchKernelGGL((k_attention<T, HD, 2>), grid, dim3(256), 0, s, a);
  } else {
    if (ev) hipExtLaunchKernelGGL((k_attention<T, HD, 1>), grid, dim3(256), 0, s, ev->start, ev->stop, 0, a);
    else hipLaunchKernelGGL((k_attention<T, HD, 1>), grid, dim3(256), 0, s, a);
  }
}

template <int HD>
static void launch_attn_combine_hd(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  const dim3 cgrid((32 * HD / 4 + 255) / 256, a.n_kv * a.n_rb, a.B);
  if (ev) hipExtLaunchKernelGGL((k_attn_combine<HD>), cgrid, dim3(256), 0, s, ev->start, ev->stop, 0, a);
  else hipLaunchKernelGGL((k_attn_combine<HD>), cgrid, dim3(256), 0, s, a);
}

template <typename T>
void launch_attention(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  if (a.head_dim == 128) launch_attention_hd<T, 128>(a, s, ev);
  else launch_attention_hd<T, 64>(a, s, ev);
}

bool attention_needs_combine(const AttnArgs& a) { return a.n_groups_max > 1 && !a.fused_combine; }

void launch_attn_combine(const AttnArgs& a, hipStream_t s, const LaunchEvents* ev) {
  if (a.head_dim == 128) launch_attn_combine_hd<128>(a, s, ev);
  else launch_attn_combine_hd<64>(a, s, ev);
}

template void launch_attention<uint16_t>(const AttnArgs&, hipStream_t, const LaunchEvents*);
template void launch_attention<float>(const AttnArgs&, hipStream_t, const LaunchEvents*);

}  // namespace seedk
