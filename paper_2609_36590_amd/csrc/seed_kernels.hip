// gfx950 kernels of the SEED draft-verify decode path.
//
// Precision: weights and the KV cache are bf16 (or fp32 for fp32 models); every activation, the
// residual stream, softmax and logits are fp32. MFMA consumes the stored operand (weights or
// K/V) exactly and the fp32 activation as a bf16 hi/lo pair (x = hi + lo), which keeps products
// within ~2^-16 of fp32 at the cost of a second MFMA (the path is HBM-bound, so MFMA time is
// not on the critical path).
//
// Determinism: the reduction order of every output depends only on the weight shape (N, K) and
// on absolute positions, never on how many rows share a pass. A row therefore gets bit-identical
// logits whether it is verified alone (plain greedy decoding, d = 0) or with d drafts.
#include "kernels.h"

#include <math.h>

namespace seedk {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

static constexpr float NEG_INF = -__builtin_huge_valf();

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------------------------------------
// Element traits: A-operand fragments (8 stored elements per lane) and the B-operand (8 fp32
// activations per lane). The MFMA sums over k; A and B agree on which logical k each
// (lane, j) slot carries, so any fixed slot assignment is a valid contraction.
// ---------------------------------------------------------------------------------------------
template <typename T>
struct ET;

template <>
struct ET<uint16_t> {
  struct A { uint4 v; };
  struct B { bf16x8 hi, lo; };
  __device__ static A load(const uint16_t* p) { return A{*reinterpret_cast<const uint4*>(p)}; }
  __device__ static B split(const float x[8]) {
    B r;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      __bf16 h = (__bf16)x[j];
      r.hi[j] = h;
      r.lo[j] = (__bf16)(x[j] - (float)h);
    }
    return r;
  }
  __device__ static void mma(f32x4& acc, const A& a, const B& b) {
    bf16x8 av = __builtin_bit_cast(bf16x8, a.v);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, b.hi, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, b.lo, acc, 0, 0, 0);
  }
  __device__ static void to_f32(const A& a, float out[8]) {
    const uint32_t w[4] = {a.v.x, a.v.y, a.v.z, a.v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[2 * j] = __uint_as_float(w[j] << 16);
      out[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
  __device__ static uint16_t from_f32(float f) { return f2bf(f); }
};

template <>
struct ET<float> {
  struct A { float4 a, b; };
  struct B { float x[8]; };
  __device__ static A load(const float* p) {
    return A{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
  }
  __device__ static B split(const float x[8]) {
    B r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r.x[j] = x[j];
    return r;
  }
  __device__ static void mma(f32x4& acc, const A& a, const B& b) {
    const float av[8] = {a.a.x, a.a.y, a.a.z, a.a.w, a.b.x, a.b.y, a.b.z, a.b.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], b.x[j], acc, 0, 0, 0);
  }
  __device__ static void to_f32(const A& a, float out[8]) {
    out[0] = a.a.x; out[1] = a.a.y; out[2] = a.a.z; out[3] = a.a.w;
    out[4] = a.b.x; out[5] = a.b.y; out[6] = a.b.z; out[7] = a.b.w;
  }
  __device__ static float from_f32(float f) { return f; }
};

__device__ __forceinline__ unsigned long long argmax_key(float v, int idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // order-preserving map of floats
  return ((unsigned long long)u << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)idx);
}

__device__ __forceinline__ void load8(const float* p, float x[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// ---------------------------------------------------------------------------------------------
// Linear epilogues. Y(nl, m, c) is the finished fp32 output of row c of the workgroup's local
// n-tile nl for activation row m.
// ---------------------------------------------------------------------------------------------
template <typename T, int EPI>
__device__ void linear_epilogue(const LinArgs& a, const float* Y, int y_nl_stride, int y_m_stride) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n_tiles = a.N >> 4;
  const int M = a.M;
#define YV(nl_, m_, c_) Y[(nl_) * y_nl_stride + (m_) * y_m_stride + (c_)]
  if constexpr (EPI == EPI_RESID) {
    for (int e = tid; e < a.NT * M; e += nthr) {
      const int nl = e / M, m = e - nl * M;
      const int nt = blockIdx.x * a.NT + nl;
      if (nt >= n_tiles) continue;
      float* hp = a.h + (size_t)m * a.N + nt * 16;
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const float v = hp[c] + YV(nl, m, c);
        hp[c] = v;
        s += v * v;
      }
      a.ssq_out[(size_t)m * n_tiles + nt] = s;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int F = a.N >> 1;
    for (int e = tid; e < a.NT * M * 8; e += nthr) {
      const int nl = e / (M * 8), r = e - nl * M * 8, m = r >> 3, c = r & 7;
      const int nt = blockIdx.x * a.NT + nl;
      if (nt >= n_tiles) continue;
      const float g = YV(nl, m, c), u = YV(nl, m, c + 8);
      a.act[(size_t)m * F + nt * 8 + c] = g / (1.f + __expf(-g)) * u;
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int HD = a.head_dim, tpd = HD >> 4, half = HD >> 1;
    const int q_tiles = a.n_heads * tpd, k_tiles = a.n_kv * tpd;
    T* kvp = reinterpret_cast<T*>(a.kv);
    for (int e = tid; e < a.NT * M * 16; e += nthr) {
      const int nl = e / (M * 16), r = e - nl * M * 16, m = r >> 4, c = r & 15;
      const int nt = blockIdx.x * a.NT + nl;
      if (nt >= n_tiles) continue;
      int sec, lt;
      if (nt < q_tiles) { sec = 0; lt = nt; }
      else if (nt < q_tiles + k_tiles) { sec = 1; lt = nt - q_tiles; }
      else { sec = 2; lt = nt - q_tiles - k_tiles; }
      const int head = lt / tpd, j = lt - head * tpd;
      const int d = (c < 8) ? 8 * j + c : half + 8 * j + (c - 8);
      const int pos = a.row_pos[m];
      float y = YV(nl, m, c);
      if (sec < 2) {
        const int fi = 8 * j + (c & 7);
        const float cs = a.rope_cos[(size_t)pos * half + fi];
        const float sn = a.rope_sin[(size_t)pos * half + fi];
        const float partner = YV(nl, m, c ^ 8);
        y = (c < 8) ? (y * cs - partner * sn) : (y * cs + partner * sn);
      }
      if (sec == 0) {
        a.q[(size_t)m * a.n_heads * HD + head * HD + d] = y;
      } else {
        const int b = a.row_seq[m];
        const int blk = a.bt[b * a.bt_stride + (pos >> 4)];
        const size_t base = ((size_t)(a.layer * a.n_blocks + blk) * 2 + (sec - 1)) * a.n_kv + head;
        if (sec == 1) kvp[base * 16 * HD + (pos & 15) * HD + d] = ET<T>::from_f32(y);
        else kvp[base * HD * 16 + d * 16 + (pos & 15)] = ET<T>::from_f32(y);
      }
    }
  } else {  // EPI_HEAD
    if (a.logits) {
      for (int e = tid; e < a.NT * M * 16; e += nthr) {
        const int nl = e / (M * 16), r = e - nl * M * 16, m = r >> 4, c = r & 15;
        const int nt = blockIdx.x * a.NT + nl;
        if (nt >= n_tiles) continue;
        a.logits[(long long)m * a.ld_logits + nt * 16 + c] = YV(nl, m, c);
      }
    }
    for (int m = tid; m < M; m += nthr) {
      float best = NEG_INF;
      int bi = -1;
      for (int nl = 0; nl < a.NT; ++nl) {
        const int nt = blockIdx.x * a.NT + nl;
        if (nt >= n_tiles) break;
        for (int c = 0; c < 16; ++c) {
          const float v = YV(nl, m, c);
          if (bi < 0 || v > best) { best = v; bi = nt * 16 + c; }
        }
      }
      if (bi >= 0) atomicMax(&a.keys[m], argmax_key(best, bi));
    }
    __shared__ int s_last;
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const unsigned prev = atomicAdd(a.counter, 1u);
      s_last = (prev == gridDim.x - 1);
    }
    __syncthreads();
    if (s_last) {
      __threadfence();
      for (int m = tid; m < M; m += nthr) {
        const unsigned long long key = atomicExch(&a.keys[m], 0ull);
        a.tok_out[m * a.tok_stride] = (int)(0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull));
      }
      if (tid == 0) atomicExch(a.counter, 0u);
    }
  }
#undef YV
}

// Sum of squares of row m from the per-16-feature partials, in a fixed order.
__device__ __forceinline__ float row_rsqrt(const LinArgs& a, int m) {
  const float* sp = a.ssq + (size_t)m * a.nssq;
  float s = 0.f;
  for (int j = 0; j < a.nssq; ++j) s += sp[j];
  return rsqrtf(s / (float)a.K + a.eps);
}

// ---------------------------------------------------------------------------------------------
// Weight-streaming skinny GEMM on MFMA: Y[M, N] = X[M, K] W^T, M <= 16*TT.
// Workgroup = NT*KS waves; wave (nl, ks) streams n-tile blockIdx.x*NT+nl over the ks-th
// contiguous range of k-tiles. Partials are reduced across ks in LDS in ks order.
// ---------------------------------------------------------------------------------------------
template <typename T, int PRO, int EPI, int TT>
__global__ void __launch_bounds__(1024) k_linear_mfma(LinArgs a) {
  extern __shared__ float smem[];
  __shared__ float s_rs[64];
  float* s_red = smem;         // [NW][M][16]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int KT = a.K >> 5, n_tiles = a.N >> 4;
  const int M = a.M;
  if constexpr (PRO == PRO_NORM) {
    for (int m = tid; m < M; m += blockDim.x) s_rs[m] = row_rsqrt(a, m);
    __syncthreads();
  }
  const int nl = wave / a.KS, ks = wave - nl * a.KS;
  const int nt = blockIdx.x * a.NT + nl;
  const int tl = lane & 15, kg = lane >> 4;
  f32x4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nt < n_tiles) {
    const int kt0 = (ks * KT) / a.KS, kt1 = ((ks + 1) * KT) / a.KS;
    const T* wp = reinterpret_cast<const T*>(a.W) + (size_t)nt * KT * 512 + lane * 8;
    const float* xp[TT];
    float rs[TT];
    bool ok[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int tok = tt * 16 + tl;
      ok[tt] = tok < M;
      xp[tt] = a.X + (size_t)(ok[tt] ? tok : 0) * a.ldx + kg * 8;
      rs[tt] = 1.f;
      if constexpr (PRO == PRO_NORM) rs[tt] = ok[tt] ? s_rs[tok] : 0.f;
    }
    const float* gp = (PRO == PRO_NORM) ? a.gain + kg * 8 : nullptr;
    constexpr int U = (TT <= 1) ? 4 : 2;
    int kt = kt0;
    for (; kt + U <= kt1; kt += U) {
      typename ET<T>::A w[U];
      float x[U][TT][8];
#pragma unroll
      for (int u = 0; u < U; ++u) w[u] = ET<T>::load(wp + (size_t)(kt + u) * 512);
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          if (ok[tt]) load8(xp[tt] + (kt + u) * 32, x[u][tt]);
          else {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[u][tt][j] = 0.f;
          }
        }
      }
      if constexpr (PRO == PRO_NORM) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          float g[8];
          load8(gp + (kt + u) * 32, g);
#pragma unroll
          for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int j = 0; j < 8; ++j) x[u][tt][j] = (x[u][tt][j] * rs[tt]) * g[j];
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) ET<T>::mma(acc[tt], w[u], ET<T>::split(x[u][tt]));
    }
    for (; kt < kt1; ++kt) {
      const typename ET<T>::A w = ET<T>::load(wp + (size_t)kt * 512);
      float g[8];
      if constexpr (PRO == PRO_NORM) load8(gp + kt * 32, g);
#pragma unroll
      for (int tt = 0; tt < TT; ++tt) {
        float x[8];
        if (ok[tt]) load8(xp[tt] + kt * 32, x);
        else {
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = 0.f;
        }
        if constexpr (PRO == PRO_NORM) {
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = (x[j] * rs[tt]) * g[j];
        }
        ET<T>::mma(acc[tt], w, ET<T>::split(x));
      }
    }
  }
  // lane (tl, kg) holds rows 4*kg+i of the n-tile for token tt*16+tl
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int tok = tt * 16 + tl;
    if (tok < M) {
      float* dst = s_red + ((size_t)wave * M + tok) * 16 + 4 * kg;
      dst[0] = acc[tt][0]; dst[1] = acc[tt][1]; dst[2] = acc[tt][2]; dst[3] = acc[tt][3];
    }
  }
  __syncthreads();
  for (int e = tid; e < a.NT * M * 16; e += blockDim.x) {
    const int nl2 = e / (M * 16), r = e - nl2 * M * 16;
    float y = 0.f;
    for (int k2 = 0; k2 < a.KS; ++k2) y += s_red[(size_t)(nl2 * a.KS + k2) * M * 16 + r];
    s_red[(size_t)(nl2 * a.KS) * M * 16 + r] = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, s_red, a.KS * M * 16, 16);
}

// ---------------------------------------------------------------------------------------------
// Weight-streaming GEMV on the vector ALUs (one activation row): same tiles and waves as the
// MFMA kernel; lane (tl, kg) accumulates row tl over its k-slots, then the four k-groups are
// added across lanes and the KS partials in LDS.
// ---------------------------------------------------------------------------------------------
template <typename T, int PRO, int EPI>
__global__ void __launch_bounds__(1024) k_linear_valu(LinArgs a) {
  extern __shared__ float smem[];
  float* s_x = smem;                // [K]
  float* s_red = smem + a.K;        // [NW][16]
  __shared__ float s_rs;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int KT = a.K >> 5, n_tiles = a.N >> 4;
  if constexpr (PRO == PRO_NORM) {
    if (tid == 0) s_rs = row_rsqrt(a, 0);
    __syncthreads();
    const float rs = s_rs;
    for (int k = tid; k < a.K; k += blockDim.x) s_x[k] = (a.X[k] * rs) * a.gain[k];
  } else {
    for (int k = tid; k < a.K; k += blockDim.x) s_x[k] = a.X[k];
  }
  __syncthreads();
  const int nl = wave / a.KS, ks = wave - nl * a.KS;
  const int nt = blockIdx.x * a.NT + nl;
  const int kg = lane >> 4;
  float acc = 0.f;
  if (nt < n_tiles) {
    const int kt0 = (ks * KT) / a.KS, kt1 = ((ks + 1) * KT) / a.KS;
    const T* wp = reinterpret_cast<const T*>(a.W) + (size_t)nt * KT * 512 + lane * 8;
    const float* xs = s_x + kg * 8;
    int kt = kt0;
    for (; kt + 4 <= kt1; kt += 4) {
      typename ET<T>::A w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) w[u] = ET<T>::load(wp + (size_t)(kt + u) * 512);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float wf[8], xv[8];
        ET<T>::to_f32(w[u], wf);
        load8(xs + (kt + u) * 32, xv);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaf(wf[j], xv[j], acc);
      }
    }
    for (; kt < kt1; ++kt) {
      float wf[8], xv[8];
      ET<T>::to_f32(ET<T>::load(wp + (size_t)kt * 512), wf);
      load8(xs + kt * 32, xv);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc = fmaf(wf[j], xv[j], acc);
    }
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  if (lane < 16) s_red[wave * 16 + lane] = acc;
  __syncthreads();
  for (int e = tid; e < a.NT * 16; e += blockDim.x) {
    const int nl2 = e >> 4, c = e & 15;
    float y = 0.f;
    for (int k2 = 0; k2 < a.KS; ++k2) y += s_red[(nl2 * a.KS + k2) * 16 + c];
    s_red[(nl2 * a.KS) * 16 + c] = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, s_red, a.KS * 16, 16);
}

// ---------------------------------------------------------------------------------------------
// Paged attention on MFMA, one wave per (sequence b, KV head h, row-block rb, chunk group g).
// The queries of a row-block (G heads x RB rows <= 32) are the B operand. For each chunk of 64
// absolute positions: S^T = K Q^T (A = K rows from the paged cache), mask positions > the
// query's own, chunk softmax in base 2, then O^T = V^T P^T (A = V^T from the transposed V
// block). Chunks are merged left to right with the online-softmax rule; a fully masked chunk
// is the exact identity of that merge, so the result for a query depends only on the positions
// it sees, not on how many rows share the pass.
//
// Position tile pt (16 positions) of chunk base P0, MFMA row r <-> position
//   P0 + 32*(pt>>1) + 8*(r>>2) + (r&3) + 4*(pt&1),
// so after S^T the lane group kg holds positions 8kg..8kg+7 of each 32-position step, which is
// exactly the k-slot layout the O^T MFMA needs for P^T: no cross-lane shuffle of P.
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ void softmax_merge(float& m_r, float& l_r, float* o_r, float m_c, float l_c,
                                              const float* o_c, int n) {
  const float m_n = fmaxf(m_r, m_c);
  const float ar = (m_r == NEG_INF) ? 0.f : exp2f(m_r - m_n);
  const float ac = (m_c == NEG_INF) ? 0.f : exp2f(m_c - m_n);
  l_r = l_r * ar + l_c * ac;
  for (int i = 0; i < n; ++i) o_r[i] = o_r[i] * ar + o_c[i] * ac;
  m_r = m_n;
}

template <typename T, int HD, bool FLASH>
__global__ void __launch_bounds__(64) k_attention(AttnArgs a) {
  constexpr int DS = HD / 32;    // 32-dim steps of S^T
  constexpr int DT = HD / 16;    // 16-dim tiles of O^T
  const int lane = threadIdx.x, tl = lane & 15, kg = lane >> 4;
  const int g = blockIdx.x;
  const int h = blockIdx.y % a.n_kv, rb = blockIdx.y / a.n_kv;
  const int b = blockIdx.z;
  const int r0 = rb * a.RB;
  if (r0 >= a.R) return;
  const int nr = min(a.RB, a.R - r0);
  const int nqv = nr * a.G;
  const int mrow0 = b * a.R + r0;
  const int maxpos = a.row_pos[mrow0 + nr - 1];
  const int n_chunks = (maxpos >> 6) + 1;
  int c0, c1;
  if (FLASH) { c0 = 0; c1 = n_chunks; }
  else {
    c0 = g * a.S;
    if (c0 >= n_chunks) return;
    c1 = min(n_chunks, c0 + a.S);
  }
  const int QT = nqv > 16 ? 2 : 1;
  const int qstride = a.n_heads * HD;

  // queries: lane column qv = qt*16 + tl, k-slots d = ds*32 + kg*8 + j, pre-scaled by log2(e)/sqrt(d)
  typename ET<T>::B qf[2][DS];
  int qpos[2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int qv = qt * 16 + tl;
    const bool ok = qt < QT && qv < nqv;
    const int rl = qv / a.G, gq = qv - rl * a.G;
    const int m = mrow0 + (ok ? rl : 0);
    qpos[qt] = ok ? a.row_pos[m] : -1;
    const float* qp = a.q + (size_t)m * qstride + (h * a.G + gq) * HD;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      float x[8];
      if (ok) {
        load8(qp + ds * 32 + kg * 8, x);
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] *= a.scale_log2;
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = 0.f;
      }
      qf[qt][ds] = ET<T>::split(x);
    }
  }

  const T* kvp = reinterpret_cast<const T*>(a.kv);
  const int* btp = a.bt + b * a.bt_stride;
  const size_t layer_base = (size_t)a.layer * a.n_blocks;

  float m_r[2] = {NEG_INF, NEG_INF}, l_r[2] = {0.f, 0.f};
  float o_r[2][DT][4];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) o_r[qt][dt][i] = 0.f;

  for (int c = c0; c < c1; ++c) {
    const int P0 = c * 64;
    // ---- S^T = K Q^T over 4 position tiles ----
    f32x4 sacc[4][2];
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) {
      sacc[pt][0] = f32x4{0.f, 0.f, 0.f, 0.f};
      sacc[pt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int pos = P0 + 32 * (pt >> 1) + 8 * (tl >> 2) + (tl & 3) + 4 * (pt & 1);
      const int blk = btp[pos >> 4];
      const T* kp = kvp + (((layer_base + blk) * 2 + 0) * a.n_kv + h) * 16 * HD + (pos & 15) * HD + kg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const typename ET<T>::A kf = ET<T>::load(kp + ds * 32);
        ET<T>::mma(sacc[pt][0], kf, qf[0][ds]);
        if (QT > 1) ET<T>::mma(sacc[pt][1], kf, qf[1][ds]);
      }
    }
    // ---- mask + chunk softmax (base 2) ----
    float p[2][4][4];
    float m_c[2], l_c[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
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
    typename ET<T>::B pf[2][2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
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
    float o_c[2][DT][4];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      f32x4 oacc0 = {0.f, 0.f, 0.f, 0.f}, oacc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int pos = P0 + 32 * s + 8 * kg;
        const int blk = btp[pos >> 4];
        const T* vp = kvp + (((layer_base + blk) * 2 + 1) * a.n_kv + h) * HD * 16 + (dt * 16 + tl) * 16 + (pos & 15);
        const typename ET<T>::A vf = ET<T>::load(vp);
        ET<T>::mma(oacc0, vf, pf[0][s]);
        if (QT > 1) ET<T>::mma(oacc1, vf, pf[1][s]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        o_c[0][dt][i] = oacc0[i];
        o_c[1][dt][i] = oacc1[i];
      }
    }
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) softmax_merge(m_r[qt], l_r[qt], &o_r[qt][0][0], m_c[qt], l_c[qt], &o_c[qt][0][0], DT * 4);
  }

  // lane (tl, kg) holds o for query column qt*16+tl, dims dt*16 + 4*kg + i
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int qv = qt * 16 + tl;
    if (qt >= QT || qv >= nqv) continue;
    if (FLASH) {
      const int rl = qv / a.G, gq = qv - rl * a.G;
      float* op = a.out + (size_t)(mrow0 + rl) * qstride + (h * a.G + gq) * HD;
      const float inv = 1.f / l_r[qt];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<float4*>(op + dt * 16 + 4 * kg) =
            make_float4(o_r[qt][dt][0] * inv, o_r[qt][dt][1] * inv, o_r[qt][dt][2] * inv, o_r[qt][dt][3] * inv);
    } else {
      float* pp = a.part + ((((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.chunk_groups + g) * 32 + qv) * (HD + 4);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<float4*>(pp + dt * 16 + 4 * kg) =
            make_float4(o_r[qt][dt][0], o_r[qt][dt][1], o_r[qt][dt][2], o_r[qt][dt][3]);
      if (kg == 0) {
        pp[HD] = m_r[qt];
        pp[HD + 1] = l_r[qt];
      }
    }
  }
}

// Merge the chunk-group partials of one (row, query head), left to right.
__global__ void __launch_bounds__(128) k_combine(AttnArgs a) {
  const int hq = blockIdx.x, m = blockIdx.y, d = threadIdx.x;
  const int HD = a.head_dim;
  if (d >= HD) return;
  const int b = m / a.R, r = m - b * a.R;
  const int rb = r / a.RB, rl = r - rb * a.RB;
  const int h = hq / a.G, gq = hq - h * a.G;
  const int qv = rl * a.G + gq;
  const int r0 = rb * a.RB, nr = min(a.RB, a.R - r0);
  const int maxpos = a.row_pos[b * a.R + r0 + nr - 1];
  const int n_chunks = (maxpos >> 6) + 1;
  const int n_groups = (n_chunks + a.S - 1) / a.S;
  float m_r = NEG_INF, l_r = 0.f, o_r = 0.f;
  const float* pp = a.part + (((size_t)(b * a.n_kv + h) * a.n_rb + rb) * a.chunk_groups * 32 + qv) * (HD + 4);
  for (int gi = 0; gi < n_groups; ++gi) {
    const float* q = pp + (size_t)gi * 32 * (HD + 4);
    const float oc = q[d];
    softmax_merge(m_r, l_r, &o_r, q[HD], q[HD + 1], &oc, 1);
  }
  a.out[(size_t)m * a.n_heads * HD + hq * HD + d] = o_r / l_r;
}

// ---------------------------------------------------------------------------------------------
// Row setup for a pass: pick each row's sequence, position and token (Algorithm 2: drafts feed
// X_draft[i-1], verification feeds X_draft[0..d]), gather the raw embedding H^0 = W_in x from
// the packed table into the fp32 residual stream, and write its per-16-feature sums of squares.
// ---------------------------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_setup(SetupArgs a) {
  const int m = blockIdx.x;
  __shared__ int s_tok;
  if (threadIdx.x == 0) {
    int b, pos, tok;
    if (a.mode == SETUP_PREFILL) {
      b = a.pf_seq;
      pos = a.pf_pos0 + m;
      tok = a.tokens[b * a.tstride + pos];
    } else if (a.mode == SETUP_DRAFT) {
      b = m;
      pos = a.t[b] - 1 + (a.step - 1);
      tok = a.drafts[b * a.dstride + a.step - 1];
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
    a.row_seq[m] = b;
    a.row_pos[m] = pos;
    s_tok = tok;
  }
  __syncthreads();
  const int tok = s_tok;
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
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) { hp[i] = v0[i]; s += v0[i] * v0[i]; }
#pragma unroll
    for (int i = 0; i < 8; ++i) { hp[8 + i] = v1[i]; s += v1[i] * v1[i]; }
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
  if (threadIdx.x == 0) *st.rounds = s_round + 1;
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
size_t linear_lds_bytes(int M, int K, int NT, int KS, bool valu) {
  const int NW = NT * KS;
  if (valu) return (size_t)(K + NW * 16) * sizeof(float);
  return (size_t)(NW * M * 16) * sizeof(float);
}

template <typename T, int PRO, int EPI>
static void launch_linear_pe(const LinArgs& a, bool valu, hipStream_t s) {
  const int n_tiles = a.N >> 4;
  const dim3 grid((n_tiles + a.NT - 1) / a.NT);
  const dim3 block(64 * a.NT * a.KS);
  const size_t lds = linear_lds_bytes(a.M, a.K, a.NT, a.KS, valu);
  if (valu) {
    hipLaunchKernelGGL((k_linear_valu<T, PRO, EPI>), grid, block, lds, s, a);
    return;
  }
  const int TT = (a.M + 15) / 16;
  switch (TT) {
    case 1: hipLaunchKernelGGL((k_linear_mfma<T, PRO, EPI, 1>), grid, block, lds, s, a); break;
    case 2: hipLaunchKernelGGL((k_linear_mfma<T, PRO, EPI, 2>), grid, block, lds, s, a); break;
    case 3: hipLaunchKernelGGL((k_linear_mfma<T, PRO, EPI, 3>), grid, block, lds, s, a); break;
    default: hipLaunchKernelGGL((k_linear_mfma<T, PRO, EPI, 4>), grid, block, lds, s, a); break;
  }
}

template <typename T>
void launch_linear(const LinArgs& a, int prologue, int epilogue, bool valu, hipStream_t s) {
  if (prologue == PRO_NORM) {
    switch (epilogue) {
      case EPI_QKV: launch_linear_pe<T, PRO_NORM, EPI_QKV>(a, valu, s); break;
      case EPI_SWIGLU: launch_linear_pe<T, PRO_NORM, EPI_SWIGLU>(a, valu, s); break;
      default: launch_linear_pe<T, PRO_NORM, EPI_HEAD>(a, valu, s); break;
    }
  } else {
    launch_linear_pe<T, PRO_PLAIN, EPI_RESID>(a, valu, s);
  }
}

template <typename T>
void launch_attention(const AttnArgs& a, bool flash, hipStream_t s) {
  const dim3 grid(flash ? 1 : a.chunk_groups, a.n_kv * a.n_rb, a.B);
  if (a.head_dim == 128) {
    if (flash) hipLaunchKernelGGL((k_attention<T, 128, true>), grid, dim3(64), 0, s, a);
    else hipLaunchKernelGGL((k_attention<T, 128, false>), grid, dim3(64), 0, s, a);
  } else {
    if (flash) hipLaunchKernelGGL((k_attention<T, 64, true>), grid, dim3(64), 0, s, a);
    else hipLaunchKernelGGL((k_attention<T, 64, false>), grid, dim3(64), 0, s, a);
  }
}

void launch_combine(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_combine, dim3(a.n_heads, a.B * a.R), dim3(a.head_dim), 0, s, a);
}

template <typename T>
void launch_setup(const SetupArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_setup<T>), dim3(a.M), dim3(256), 0, s, a);
}

void launch_accept(const DevState& st, int B, int k, hipStream_t s) {
  hipLaunchKernelGGL(k_accept, dim3(1), dim3(64), 0, s, st, B, k);
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

template <typename T, int PRO, int EPI>
static void allow_big_lds(int bytes) {
  const void* fns[] = {reinterpret_cast<const void*>(&k_linear_valu<T, PRO, EPI>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 1>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 2>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 3>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 4>)};
  for (const void* f : fns) (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

// Every launch stays within 64 KB of dynamic LDS; where the device allows more, opt in anyway
// (failures are harmless and cleared).
hipError_t configure_kernels(int bf16) {
  int dev = 0, optin = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipGetLastError();
  if (hipDeviceGetAttribute(&optin, hipDeviceAttributeSharedMemPerBlockOptin, dev) == hipSuccess && optin > 65536) {
    if (bf16) {
      allow_big_lds<uint16_t, PRO_NORM, EPI_QKV>(optin); allow_big_lds<uint16_t, PRO_NORM, EPI_SWIGLU>(optin);
      allow_big_lds<uint16_t, PRO_NORM, EPI_HEAD>(optin); allow_big_lds<uint16_t, PRO_PLAIN, EPI_RESID>(optin);
    } else {
      allow_big_lds<float, PRO_NORM, EPI_QKV>(optin); allow_big_lds<float, PRO_NORM, EPI_SWIGLU>(optin);
      allow_big_lds<float, PRO_NORM, EPI_HEAD>(optin); allow_big_lds<float, PRO_PLAIN, EPI_RESID>(optin);
    }
  }
  (void)hipGetLastError();
  return hipSuccess;
}

template void launch_linear<uint16_t>(const LinArgs&, int, int, bool, hipStream_t);
template void launch_linear<float>(const LinArgs&, int, int, bool, hipStream_t);
template void launch_attention<uint16_t>(const AttnArgs&, bool, hipStream_t);
template void launch_attention<float>(const AttnArgs&, bool, hipStream_t);
template void launch_setup<uint16_t>(const SetupArgs&, hipStream_t);
template void launch_setup<float>(const SetupArgs&, hipStream_t);
template void launch_pack<uint16_t>(const void*, void*, const int*, int, int, hipStream_t);
template void launch_pack<float>(const void*, void*, const int*, int, int, hipStream_t);

}  // namespace seedk
