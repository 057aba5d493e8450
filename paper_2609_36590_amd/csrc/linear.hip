// Weight-streaming linear kernels (MFMA skinny GEMM) with fused RMSNorm scale, RoPE + paged-KV
// write, residual, SwiGLU and LM-head argmax epilogues.
//
//  * k_linear_lds    M <= 16 rows: the activation rows are staged once per workgroup in LDS as MFMA
//                    B-operand slots, so the vector-memory path carries weight tiles only.
//  * k_linear_mfma   any M (prefill, large batches): activation fragments are read from global
//                    memory next to each weight tile.
//
// Both compute every output with the same arithmetic: wave ks of the KS K-splits accumulates its
// k-range in k order on MFMA, and the KS partial sums are added in S consecutive groups
// (y = sum_s (sum_{k in group s} p_k), each sum left to right, starting from 0). The split (KS, S)
// depends only on the weight shape (N, K), so a row's output is bit-identical whatever kernel
// runs it and however many rows share the pass: verifying d drafts gives the same logits, row by
// row, as plain greedy decoding (d = 0). (k_linear_lds supports S == 1 only.)
#include "device_common.h"

#include <algorithm>

namespace seedk {

// n-group of pass j of this workgroup: g0 + j * gs
struct Grp {
  int g0, gs;
};

// ---------------------------------------------------------------------------------------------
// Epilogues. Y(lt, m, c) is the finished fp32 output (column c of local tile lt = j*NT + nl, row
// m). Element e of the (lt, m, c) space is handled by thread e mod blockDim; the global values an
// element needs (residual, gain, KV block, RoPE angles) are loaded for the thread's first element
// at kernel start, before the weight stream, so the epilogue itself costs no extra round trip.
// ---------------------------------------------------------------------------------------------
struct EpiPre {
  float h, g;        // EPI_RESID: residual value and next-norm gain
  int pos, blk;      // EPI_QKV: position and KV block of the row
  float cs, sn;      // EPI_QKV: RoPE cos/sin for the element's rotary pair
};

__device__ __forceinline__ void epi_coords(const LinArgs& a, Grp gr, int e, int& lt, int& m, int& c, int& nt) {
  const int per = a.M * 16;
  lt = e / per;
  const int r = e - lt * per;
  m = r >> 4;
  c = r & 15;
  const int j = lt / a.NT, nl = lt - j * a.NT;
  nt = (gr.g0 + j * gr.gs) * a.NT + nl;
}

// QKV section of n-tile nt: 0 = q, 1 = k, 2 = v; (head, j) = tile j of that head (dims 8j..8j+7
// and head_dim/2+8j..+7, so rotary partners share the tile).
__device__ __forceinline__ void qkv_tile(const LinArgs& a, int nt, int& sec, int& head, int& j) {
  const int tpd = a.head_dim >> 4, q_tiles = a.n_heads * tpd, k_tiles = a.n_kv * tpd;
  int lt;
  if (nt < q_tiles) { sec = 0; lt = nt; }
  else if (nt < q_tiles + k_tiles) { sec = 1; lt = nt - q_tiles; }
  else { sec = 2; lt = nt - q_tiles - k_tiles; }
  head = lt / tpd;
  j = lt - head * tpd;
}

template <int EPI>
__device__ __forceinline__ void epi_load(const LinArgs& a, Grp gr, int e, EpiPre& p) {
  int lt, m, c, nt;
  epi_coords(a, gr, e, lt, m, c, nt);
  if (e >= a.NJ * a.NT * a.M * 16 || nt >= (a.N >> 4)) return;
  if constexpr (EPI == EPI_RESID) {
    p.h = a.h[(size_t)m * a.N + nt * 16 + c];
    p.g = a.gain_next[nt * 16 + c];
  } else if constexpr (EPI == EPI_QKV) {
    int sec, head, j;
    qkv_tile(a, nt, sec, head, j);
    p.pos = a.row_slot[m];   // the cache slot (the rotary position enters through row_rope)
    p.blk = a.row_blk[m];
    const int fi = 8 * j + (c & 7);
    p.cs = a.row_rope[(size_t)m * a.head_dim + fi];
    p.sn = a.row_rope[(size_t)m * a.head_dim + (a.head_dim >> 1) + fi];
  }
}

template <typename T, int EPI>
__device__ void linear_epilogue(const LinArgs& a, Grp gr, const float* Y, int y_lt_stride, const EpiPre& pre) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n_tiles = a.N >> 4;
  const int M = a.M;
  const int total = a.NJ * a.NT * M * 16;
#define YV(lt_, m_, c_) Y[(lt_) * y_lt_stride + (m_) * 16 + (c_)]
  if constexpr (EPI == EPI_RESID || EPI == EPI_QKV) {
    // nthr is a multiple of 64 and total of 16, so the 16 columns of one (lt, m) are 16 aligned
    // lanes of one wave in the same iteration (the ssq butterfly below stays inside them)
    for (int e = tid; e < total; e += nthr) {
      int lt, m, c, nt;
      epi_coords(a, gr, e, lt, m, c, nt);
      if (nt >= n_tiles) continue;
      EpiPre p = pre;
      if (e != tid) epi_load<EPI>(a, gr, e, p);
      if constexpr (EPI == EPI_RESID) {
        const float v = p.h + YV(lt, m, c);
        const size_t off = (size_t)m * a.N + nt * 16 + c;
        a.h[off] = v;
        a.xg[off] = v * p.g;
        float s = v * v;
        s += __shfl_xor(s, 8);
        s += __shfl_xor(s, 4);
        s += __shfl_xor(s, 2);
        s += __shfl_xor(s, 1);
        if (c == 0) a.ssq_out[(size_t)m * n_tiles + nt] = s;
      } else {
        const int HD = a.head_dim, half = HD >> 1;
        int sec, head, j;
        qkv_tile(a, nt, sec, head, j);
        const int d = (c < 8) ? 8 * j + c : half + 8 * j + (c - 8);
        float y = YV(lt, m, c);
        if (sec < 2) {
          const float partner = YV(lt, m, c ^ 8);
          y = (c < 8) ? (y * p.cs - partner * p.sn) : (y * p.cs + partner * p.sn);
        }
        if (sec == 0) {
          a.q[(size_t)m * a.n_heads * HD + head * HD + d] = y;
        } else {
          T* kvp = reinterpret_cast<T*>(a.kv);
          const size_t base = ((size_t)(a.layer * a.n_blocks + p.blk) * 2 + (sec - 1)) * a.n_kv + head;
          if (sec == 1) kvp[base * 16 * HD + (p.pos & 15) * HD + d] = ET<T>::from_f32(y);
          else kvp[base * HD * 16 + d * 16 + (p.pos & 15)] = ET<T>::from_f32(y);
        }
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int F = a.N >> 1;
    for (int e = tid; e < a.NJ * a.NT * M * 8; e += nthr) {
      const int lt = e / (M * 8), r = e - lt * M * 8, m = r >> 3, c = r & 7;
      const int j = lt / a.NT, nt = (gr.g0 + j * gr.gs) * a.NT + (lt - j * a.NT);
      if (nt >= n_tiles) continue;
      const float g = YV(lt, m, c), u = YV(lt, m, c + 8);
      a.act[(size_t)m * F + nt * 8 + c] = g / (1.f + __expf(-g)) * u;
    }
  } else {  // EPI_HEAD
    if (a.logits) {
      for (int e = tid; e < total; e += nthr) {
        int lt, m, c, nt;
        epi_coords(a, gr, e, lt, m, c, nt);
        if (nt >= n_tiles) continue;
        a.logits[(long long)m * a.ld_logits + nt * 16 + c] = YV(lt, m, c);
      }
    }
    // argmax of each row over each pass's n-group (lowest token id among equal maxima): one wave
    // per (pass, row), lane-strided candidates, then a butterfly; the partial of n-group g goes to
    // slot g and k_argmax_finalize reduces the slots (none when the caller wants the logits only)
    const int lane = tid & 63, wave = tid >> 6, nw = nthr >> 6;
    for (int q = wave; a.amax_val && q < a.NJ * M; q += nw) {
      const int j = q / M, m = q - j * M;
      const int grp = gr.g0 + j * gr.gs;
      if (grp * a.NT >= n_tiles) continue;
      const int n_cand = min(a.NT, n_tiles - grp * a.NT) * 16;
      const int id0 = grp * a.NT * 16;
      float best = NEG_INF;
      int bi = -1;
      for (int jc = lane; jc < n_cand; jc += 64) {
        const float v = YV(j * a.NT + (jc >> 4), m, jc & 15);
        if (bi < 0 || v > best) { best = v; bi = id0 + jc; }
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(best, o);
        const int oi = __shfl_xor(bi, o);
        if (oi >= 0 && (bi < 0 || ov > best || (ov == best && oi < bi))) { best = ov; bi = oi; }
      }
      if (lane == 0) {
        a.amax_val[(size_t)m * a.amax_stride + grp] = best;
        a.amax_idx[(size_t)m * a.amax_stride + grp] = bi;
      }
    }
  }
#undef YV
}

// RMSNorm scale of row m from its per-16-feature sums of squares. Lane partials (lane-strided,
// pre-loaded in ssv when available) are combined by a fixed xor tree, so the value does not
// depend on which wave computes it or on how many rows share the pass.
__device__ __forceinline__ float wave_row_scale(const LinArgs& a, int m, const float* ssv, bool pre) {
  const int lane = threadIdx.x & 63;
  float s;
  if (pre) {
    s = ((ssv[0] + ssv[1]) + ssv[2]) + ssv[3];
  } else {
    s = 0.f;
    for (int j = lane; j < a.nssq; j += 64) s += a.ssq[(size_t)m * a.nssq + j];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  return rsqrtf(s / (float)a.K + a.eps);
}

__device__ __forceinline__ bool preload_row_ssq(const LinArgs& a, int m, float ssv[4]) {
  const int lane = threadIdx.x & 63;
  if (m >= a.M || a.nssq > 256) return false;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = lane + 64 * i;
    ssv[i] = j < a.nssq ? a.ssq[(size_t)m * a.nssq + j] : 0.f;
  }
  return true;
}

// sum of n consecutive wave partials (stride `per` floats), left to right from 0
__device__ __forceinline__ float sum_partials(const float* p, int n, int per) {
  float t = 0.f;
  for (int k = 0; k < n; ++k) t += p[(size_t)k * per];
  return t;
}

__host__ __device__ inline size_t lds_x_bytes(int M, int nkt) { return (size_t)nkt * 4 * M * 32 + 32; }

// ---------------------------------------------------------------------------------------------
// Skinny GEMM with the activation rows in LDS: Y[M, N] = X[M, K] W^T, M <= 16 (one MFMA tile).
//
// The workgroup (NT * KS/S waves) issues its first weight tiles, then stages the X columns of its
// K-slice into LDS as MFMA B-operand slots: slot (kt, kg, r) = 32 bytes holding
// x[r][32kt + 8kg .. +7] (bf16 hi/lo pair for bf16 weights, fp32 otherwise), plus one zero slot
// for the token columns r >= M. Waves then stream weight tiles with P in flight, reading their B
// operands from LDS.
//
// Work: the workgroup makes NJ passes over n-groups blockIdx.x + j*gridDim.x (NT n-tiles each);
// wave (nl, ks) covers k-range ks of n-tile nl of every pass, as one continuous stream. All KS
// K-splits of an n-tile run in one workgroup (the runtime uses this kernel only with S == 1).
// ---------------------------------------------------------------------------------------------
template <typename T, int PRO, int EPI, bool ALIAS>
__global__ void __launch_bounds__(1024) k_linear_lds(LinArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int P = 8;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int NW = a.NT * a.KS;
  const int KT = a.K >> 5, n_tiles = a.N >> 4, M = a.M;
  const int nl = wave / a.KS, ks = wave - nl * a.KS;
  const int tl = lane & 15, kg = lane >> 4;
  const Grp gr{(int)blockIdx.x, (int)gridDim.x};
  const int kt0 = (ks * KT) / a.KS, nk = ((ks + 1) * KT) / a.KS - kt0;
  int nj = 0;
  while (nj < a.NJ && (gr.g0 + nj * gr.gs) * a.NT + nl < n_tiles) ++nj;
  const int Sw = nj * nk;  // weight tiles this wave streams
  const T* w0 = reinterpret_cast<const T*>(a.W) + ((size_t)(gr.g0 * a.NT + nl) * KT + kt0) * 512 + lane * 8;
  const size_t wj = (size_t)gr.gs * a.NT * KT * 512;  // elements from one pass's n-tile to the next

  // ---- weight prefetch ----
  typename ET<T>::A wb[P];
  int jI = 0, iI = 0;  // pass / k-tile of the next tile to issue
  auto issue = [&](int slot) {
    wb[slot] = ET<T>::load_nt(w0 + jI * wj + (size_t)iI * 512);
    if (++iI == nk) { iI = 0; ++jI; }
  };
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (p < Sw) issue(p);

  EpiPre epre{};
  epi_load<EPI>(a, gr, tid, epre);
  float ssv[4] = {0.f, 0.f, 0.f, 0.f};
  bool pre = false;
  if constexpr (PRO == PRO_NORM) pre = preload_row_ssq(a, wave, ssv);

  // ---- stage X into LDS (loads first, then the LDS writes) ----
  const size_t zero_off = (size_t)KT * 4 * M * 32;
  // partials [NJ][NW][M][16] and the row scales: after the staged rows, or (when both do not fit)
  // over them once the stream is done
  constexpr bool alias = ALIAS;
  float* part = reinterpret_cast<float*>(alias ? lds : lds + lds_x_bytes(M, KT));
  float* s_rs = part + (size_t)a.NJ * NW * M * 16;
  {
    // two batches of 2 items per thread per round trip: both batches' loads are issued before
    // either is written, so a workgroup whose rows take several batches (O at 5 rows, the LM head
    // at more than 3) pays half the round trips. Loads are branch-free (items past the end reload
    // the last one and are not written) and none is issued after a wait: a load under a branch
    // makes the compiler wait for every load in flight before each write, and a surplus load
    // issued after the first wait would add a round trip to the one-batch case.
    const int row_items = KT * 4, items = M * row_items, bs = 2 * (int)blockDim.x;
    float xa[2][8], xb[2][8];
    auto ld = [&](float (&xv)[2][8], int q0) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int q = min(q0 + u * (int)blockDim.x + tid, items - 1);
        const int r = q / row_items, rem = q - r * row_items;
        load8(a.X + (size_t)r * a.ldx + (size_t)rem * 8, xv[u]);
      }
    };
    auto st = [&](const float (&xv)[2][8], int q0) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int q = q0 + u * (int)blockDim.x + tid;
        if (q < items) {
          const int r = q / row_items, rem = q - r * row_items;
          ET<T>::to_lds(lds + ((size_t)rem * M + r) * 32, xv[u]);
        }
      }
    };
    if constexpr (!ALIAS) {
      if (items <= bs) {   // one batch (both paths finish their loads before they merge)
        ld(xa, 0);
        st(xa, 0);
      } else {
        for (int q0 = 0; q0 < items; q0 += 2 * bs) {
          ld(xa, q0);
          ld(xb, q0 + bs);
          st(xa, q0);
          st(xb, q0 + bs);
        }
      }
    } else {
      // one batch per round trip, loads under the item bound: with this variant's pass registers
      // the forms above make the compiler wait for every weight tile of the ring below
      for (int q0 = 0; q0 < items; q0 += bs) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int q = q0 + u * (int)blockDim.x + tid;
          if (q < items) {
            const int r = q / row_items, rem = q - r * row_items;
            load8(a.X + (size_t)r * a.ldx + (size_t)rem * 8, xa[u]);
          }
        }
        st(xa, q0);
      }
    }
    if (tid < 2) *reinterpret_cast<float4*>(lds + zero_off + tid * 16) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();

  // ---- stream ----
  const bool live_col = tl < M;
  const char* xa = lds + (live_col ? ((size_t)kt0 * 4 * M + (size_t)kg * M + tl) * 32 : zero_off);
  const size_t xs = live_col ? (size_t)4 * M * 32 : 0;  // bytes per k-tile
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  f32x4 done[ALIAS ? LDS_MAX_PASSES : 1];   // finished passes, kept until the staged rows are no longer read
  int jC = 0, iC = 0;  // pass / k-tile of the next tile to consume
  auto consume = [&](int slot) {
    ET<T>::mma(acc, wb[slot], ET<T>::from_lds(xa + iC * xs));
    if (++iC == nk) {
      if constexpr (!ALIAS) {
        if (live_col) {
          float* dst = part + ((size_t)(jC * NW + wave) * M + tl) * 16 + 4 * kg;
          dst[0] = acc[0]; dst[1] = acc[1]; dst[2] = acc[2]; dst[3] = acc[3];
        }
      } else {
#pragma unroll
        for (int q = 0; q < (ALIAS ? LDS_MAX_PASSES : 1); ++q)
          if (q == jC) done[q] = acc;
      }
      acc = f32x4{0.f, 0.f, 0.f, 0.f};
      iC = 0;
      ++jC;
    }
  };
  int s0 = 0;
  for (; s0 + 2 * P <= Sw; s0 += P) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      consume(p);
      issue(p);
      // keep each refill next to its consumption (the scheduler would otherwise sink all refills
      // below the last MFMA and drain the pipeline once per P tiles)
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (s0 + p < Sw) {
      consume(p);
      if (s0 + p + P < Sw) issue(p);
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (s0 + P + p < Sw) consume(p);

  if constexpr (ALIAS) {
    __syncthreads();   // every wave is done with the staged rows
    if (live_col) {
#pragma unroll
      for (int q = 0; q < (ALIAS ? LDS_MAX_PASSES : 1); ++q)
        if (q < nj) {
          float* dst = part + ((size_t)(q * NW + wave) * M + tl) * 16 + 4 * kg;
          dst[0] = done[q][0]; dst[1] = done[q][1]; dst[2] = done[q][2]; dst[3] = done[q][3];
        }
    }
  }

  // ---- sums over the K-splits (in ks order), RMSNorm row scale, epilogue ----
  if constexpr (PRO == PRO_NORM) {
    for (int m = wave; m < M; m += NW) {
      const float r = wave_row_scale(a, m, ssv, pre && m == wave);
      if (lane == 0) s_rs[m] = r;
    }
  }
  __syncthreads();
  const int per = M * 16;
  for (int e = tid; e < a.NJ * a.NT * per; e += blockDim.x) {
    const int lt = e / per, r = e - lt * per;
    const int j = lt / a.NT, nl2 = lt - j * a.NT;
    float* src = part + (size_t)(j * NW + nl2 * a.KS) * per + r;
    float y = sum_partials(src, a.KS, per);
    if constexpr (PRO == PRO_NORM) y *= s_rs[r >> 4];
    *src = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, gr, part, a.KS * per, epre);
}

// ---------------------------------------------------------------------------------------------
// Skinny GEMM with activation fragments from global memory: Y[M, N] = X[M, K] W^T, M <= 16*TT.
// Workgroup = NT*KS waves; wave (nl, ks) streams n-tile blockIdx.x*NT+nl over the ks-th
// contiguous range of k-tiles; each wave keeps P weight tiles in flight together with the
// matching activation fragments, refilling a slot right after taking its data (vector memory
// returns in issue order, so every wait is for the oldest slot only). Lanes past the last row
// read row 0 (branch-free issue) and are zeroed when consumed.
// ---------------------------------------------------------------------------------------------
template <typename T, int PRO, int EPI, int TT>
__global__ void __launch_bounds__(1024) k_linear_mfma(LinArgs a) {
  extern __shared__ float smem[];
  __shared__ float s_rs[64];
  float* s_red = smem;         // [NW][M][16]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int NW = a.NT * a.KS;
  const int KT = a.K >> 5, n_tiles = a.N >> 4;
  const int M = a.M;
  const int nl = wave / a.KS, ks = wave - nl * a.KS;
  const int nt = blockIdx.x * a.NT + nl;
  const int tl = lane & 15, kg = lane >> 4;
  const Grp gr{(int)blockIdx.x, (int)gridDim.x};
  EpiPre epre{};
  epi_load<EPI>(a, gr, tid, epre);
  float ssv[4] = {0.f, 0.f, 0.f, 0.f};
  bool pre = false;
  if constexpr (PRO == PRO_NORM) pre = preload_row_ssq(a, wave, ssv);
  f32x4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nt < n_tiles) {
    const int kt0 = (ks * KT) / a.KS, kt1 = ((ks + 1) * KT) / a.KS;
    const int nk = kt1 - kt0;
    const T* wp = reinterpret_cast<const T*>(a.W) + ((size_t)nt * KT + kt0) * 512 + lane * 8;
    const float* xp[TT];
    bool ok[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int tok = tt * 16 + tl;
      ok[tt] = tok < M;
      xp[tt] = a.X + (size_t)(ok[tt] ? tok : 0) * a.ldx + kg * 8 + kt0 * 32;
    }
    constexpr int P = (TT <= 1) ? 4 : (TT == 2 ? 3 : 2);
    typename ET<T>::A wb[P];
    float xb[P][TT][8];
    auto issue = [&](int slot, int j) {
      wb[slot] = ET<T>::load_nt(wp + (size_t)j * 512);
#pragma unroll
      for (int tt = 0; tt < TT; ++tt) load8(xp[tt] + j * 32, xb[slot][tt]);
    };
    auto consume = [&](int slot) {
#pragma unroll
      for (int tt = 0; tt < TT; ++tt) {
        float x[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) x[q] = ok[tt] ? xb[slot][tt][q] : 0.f;
        ET<T>::mma(acc[tt], wb[slot], ET<T>::split(x));
      }
    };
#pragma unroll
    for (int i = 0; i < P; ++i)
      if (i < nk) issue(i, i);
    int base = 0;
    for (; base + 2 * P <= nk; base += P) {
#pragma unroll
      for (int i = 0; i < P; ++i) {
        consume(i);
        issue(i, base + i + P);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int i = 0; i < P; ++i)
      if (base + i < nk) {
        consume(i);
        if (base + i + P < nk) issue(i, base + i + P);
      }
#pragma unroll
    for (int i = 0; i < P; ++i)
      if (base + P + i < nk) consume(i);
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
  if constexpr (PRO == PRO_NORM) {
    for (int m = wave; m < M; m += NW) {
      const float r = wave_row_scale(a, m, ssv, pre && m == wave);
      if (lane == 0) s_rs[m] = r;
    }
  }
  __syncthreads();
  const int per = M * 16, KSs = a.KS / a.S;
  for (int e = tid; e < a.NT * per; e += blockDim.x) {
    const int nl2 = e / per, r = e - nl2 * per;
    float* src = s_red + (size_t)(nl2 * a.KS) * per + r;
    float y = 0.f;
    for (int s2 = 0; s2 < a.S; ++s2) y += sum_partials(src + (size_t)s2 * KSs * per, KSs, per);
    if constexpr (PRO == PRO_NORM) y *= s_rs[r >> 4];
    *src = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, gr, s_red, a.KS * per, epre);
}

// ---------------------------------------------------------------------------------------------
// Wide passes (16 < M <= 64 rows: batched verification, prefill, the drafting objective's pass):
// the K split runs across workgroups. Workgroup (n-group g, k-range ks) stages the activation
// columns of its k-range only (they fit LDS where the whole K of M rows does not) and its NT
// waves stream one n-tile each over that range, exactly as wave (nl, ks) of the narrow kernels
// does (same tiles, same order, same B slots), for TT token tiles of 16 rows. The range partials
// go to global memory; k_splitk_reduce adds them in k-range order from 0 and runs the epilogue,
// so every row gets the bit-identical output of the narrow kernels.
// ---------------------------------------------------------------------------------------------
template <typename T, int TT, int XI, int PRO>
__global__ void __launch_bounds__(512) k_linear_splitk(LinArgs a, float* part) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int P = 8;
  const int tid = threadIdx.x, lane = tid & 63, nl = tid >> 6;
  const int KT = a.K >> 5, n_tiles = a.N >> 4, M = a.M;
  const int tl = lane & 15, kg = lane >> 4;
  const int ks = blockIdx.y;
  const int kt0 = (ks * KT) / a.KS, nk = ((ks + 1) * KT) / a.KS - kt0;
  const int nt = blockIdx.x * a.NT + nl;
  const bool live = nt < n_tiles;
  const T* w0 = reinterpret_cast<const T*>(a.W) + ((size_t)(live ? nt : 0) * KT + kt0) * 512 + lane * 8;

  // ---- the k-range's activations first (cache hits: issued ahead of the weight tiles they do
  // not queue behind the weights' HBM round trip), XI items per thread, branch-free: item
  // q = (i*4 + kg)*M + r is slot q = x[r][32(kt0+i) + 8kg .. +7]; items past the end load item 0
  // and go to a dummy slot ----
  const int items = nk * 4 * M;
  float xv[XI][8];
#pragma unroll
  for (int u = 0; u < XI; ++u) {
    const int q = u * (int)blockDim.x + tid, qc = q < items ? q : 0;
    const int r = qc % M, rest = qc / M;
    load8(a.X + (size_t)r * a.ldx + (size_t)kt0 * 32 + rest * 8, xv[u]);
  }

  // ---- weight prefetch (slots past the range re-read its last tile, never consumed) ----
  typename ET<T>::A wb[P];
#pragma unroll
  for (int p = 0; p < P; ++p) wb[p] = ET<T>::load_nt(w0 + (size_t)min(p, nk - 1) * 512);

  const size_t zero_off = (size_t)items * 32;
#pragma unroll
  for (int u = 0; u < XI; ++u) {
    const int q = u * (int)blockDim.x + tid;
    ET<T>::to_lds(lds + (q < items ? (size_t)q * 32 : zero_off + 32), xv[u]);
  }
  // items beyond XI per thread (shapes the launcher could not cover up front)
  for (int q = XI * (int)blockDim.x + tid; q < items; q += blockDim.x) {
    const int r = q % M, rest = q / M;
    float x[8];
    load8(a.X + (size_t)r * a.ldx + (size_t)kt0 * 32 + rest * 8, x);
    ET<T>::to_lds(lds + (size_t)q * 32, x);
  }
  if (tid < 2) *reinterpret_cast<float4*>(lds + zero_off + tid * 16) = make_float4(0.f, 0.f, 0.f, 0.f);
  __syncthreads();

  // ---- stream the range: TT token tiles per weight tile ----
  const char* xa[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int m = tt * 16 + tl;
    xa[tt] = lds + (m < M ? ((size_t)kg * M + m) * 32 : zero_off);
  }
  const size_t xs = (size_t)4 * M * 32;   // bytes per k-tile
  f32x4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto consume = [&](int slot, int i) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int m = tt * 16 + tl;
      ET<T>::mma(acc[tt], wb[slot], ET<T>::from_lds(xa[tt] + (m < M ? i * xs : 0)));
    }
  };
  int s0 = 0;
  for (; s0 + 2 * P <= nk; s0 += P) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      consume(p, s0 + p);
      wb[p] = ET<T>::load_nt(w0 + (size_t)(s0 + p + P) * 512);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (s0 + p < nk) {
      consume(p, s0 + p);
      if (s0 + p + P < nk) wb[p] = ET<T>::load_nt(w0 + (size_t)(s0 + p + P) * 512);
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (s0 + P + p < nk) consume(p, s0 + P + p);

  // ---- the RMSNorm row scales, once per launch (workgroup (0, 0)), for the reduction ----
  if constexpr (PRO == PRO_NORM) {
    if (blockIdx.x == 0 && blockIdx.y == 0) {
      const float ssv[4] = {0.f, 0.f, 0.f, 0.f};
      for (int m = nl; m < M; m += a.NT) {
        const float r = wave_row_scale(a, m, ssv, false);
        if (lane == 0) a.part_rs[m] = r;
      }
    }
  }
  // ---- range partial: part[ks][m][n], lane (tl, kg) holds features 4kg..4kg+3 of token tt*16+tl ----
  if (live) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int m = tt * 16 + tl;
      if (m < M)
        *reinterpret_cast<float4*>(part + ((size_t)ks * M + m) * a.N + nt * 16 + 4 * kg) =
            make_float4(acc[tt][0], acc[tt][1], acc[tt][2], acc[tt][3]);
    }
  }
}

// Sum of the k-range partials (k-range order, from 0), RMSNorm row scale, epilogue. Workgroup g
// handles n-tiles g*NT .. g*NT+NT-1 of all M rows (a.NT, a.NJ = 1 describe that layout to the
// shared epilogue); the launcher gives it one thread per output element.
template <typename T, int PRO, int EPI>
__global__ void __launch_bounds__(1024) k_splitk_reduce(LinArgs a, const float* part) {
  extern __shared__ float Y[];   // [NT][M][16]
  const int tid = threadIdx.x;
  const int M = a.M, n_tiles = a.N >> 4;
  const Grp gr{(int)blockIdx.x, (int)gridDim.x};
  EpiPre epre{};
  epi_load<EPI>(a, gr, tid, epre);
  const int per = M * 16;
  for (int e = tid; e < a.NT * per; e += blockDim.x) {
    const int lt = e / per, r = e - lt * per, m = r >> 4, c = r & 15;
    const int nt = blockIdx.x * a.NT + lt;
    // all k-range partials in flight at once, then added in k-range order from 0 (the order of
    // sum_partials)
    const float* pp = part + (size_t)m * a.N + min(nt, n_tiles - 1) * 16 + c;
    const size_t stride = (size_t)M * a.N;
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = k < a.KS ? pp[k * stride] : 0.f;
    float y = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (k < a.KS) y += v[k];
    for (int k = 16; k < a.KS; ++k) y += pp[k * stride];
    if constexpr (PRO == PRO_NORM) y *= a.part_rs[m];   // row scale from the split-K launch
    Y[e] = nt < n_tiles ? y : 0.f;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, gr, Y, per, epre);
}

// ---------------------------------------------------------------------------------------------
// Wide passes (more than 64 rows: the prompt's prefill and the drafting objective's decoder
// pass): a compute-bound MFMA GEMM, Y[M, N] = X[M, K] W^T. A workgroup owns WIDE_WN n-tiles
// (16 output features each) x WIDE_WM token tiles (16 rows each); its 8 waves form a 4 x 2 grid,
// wave (wn, wm) accumulating WN/4 n-tiles for token tiles 4wm..4wm+3, so each weight fragment
// feeds 4 token tiles and each activation fragment WN/4 n-tiles. WN (8, 12, 16 or 20) is chosen
// per projection so that the grid fills whole rounds of one workgroup per CU: the cost is rounds x
// WN (gate/up's 1216 n-tiles: 20 gives 2 rounds of 488 workgroups where 16 gives 3 of 608; QKV's
// 384: 12 gives one round of 256; the 2560-wide O and down stay at 8, 160 workgroups). K runs in
// chunks of WIDE_CK k-tiles: a chunk's activation rows are staged in LDS as bf16 hi/lo B-operand
// slots, double-buffered (chunk c+1's global loads are issued before chunk c is consumed and
// written to the other buffer after it), and the weight fragments of chunk c+1 are loaded into
// registers while chunk c is consumed. Every output is one MFMA chain over all of K in k order
// (these passes write the prompt's cache and the drafting objective's logits, which no decode
// pass has to reproduce bit for bit).
// Workgroup order: the token tiles of one n-group are consecutive workgroups of one XCD (workgroup
// w runs on XCD w mod 8), so that n-group's weights come from HBM once and from that XCD's L2 for
// its other token tiles. The finished tile goes through the same epilogues as the narrow kernels,
// 8 (or 4) n-tiles at a time.
// ---------------------------------------------------------------------------------------------
constexpr int WIDE_WM = 8;    // token tiles per workgroup (128 rows)
constexpr int WIDE_CK = 2;    // k-tiles per staged chunk
// n-tiles per epilogue group: 8 (the head's argmax partials are per 8 n-tiles), or 4 for workgroup
// widths that are not a multiple of 8 (their epilogues are all tile-local)
constexpr int wide_epi_nt(int wn) { return wn % 8 == 0 ? 8 : 4; }
constexpr int WIDE_ROWS_TILE = WIDE_WM * 16;
constexpr size_t WIDE_CHUNK_BYTES = (size_t)WIDE_CK * 4 * WIDE_ROWS_TILE * 32;   // one staging buffer
constexpr size_t WIDE_LDS = 2 * WIDE_CHUNK_BYTES;   // = 8 n-tiles x 128 rows x 16 fp32 outputs (the epilogue)

// A staging buffer's B-operand slots. bf16: two planes, the 16-byte hi halves of all slots, then
// the lo halves, so that the 16 lanes of a fragment read (consecutive slots) cover 256 contiguous
// bytes (interleaved 32-byte slots would put lanes tl and tl + 8 on the same banks); fp32: 32-byte
// slots of 8 values.
template <typename T>
__device__ __forceinline__ void wide_store_half(char* buf, int q, int hf, const float4 x) {
  if constexpr (sizeof(T) == 2) {
    const float v[4] = {x.x, x.y, x.z, x.w};
    bf16x4 h, l;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      __bf16 t = (__bf16)v[j];
      h[j] = t;
      l[j] = (__bf16)(v[j] - (float)t);
    }
    *reinterpret_cast<bf16x4*>(buf + (size_t)q * 16 + hf * 8) = h;
    *reinterpret_cast<bf16x4*>(buf + WIDE_CHUNK_BYTES / 2 + (size_t)q * 16 + hf * 8) = l;
  } else {
    ET<T>::to_lds_half(buf + (size_t)q * 32, hf, x);
  }
}

template <typename T>
__device__ __forceinline__ typename ET<T>::B wide_load_slot(const char* buf, int q) {
  if constexpr (sizeof(T) == 2) {
    return typename ET<T>::B{*reinterpret_cast<const bf16x8*>(buf + (size_t)q * 16),
                             *reinterpret_cast<const bf16x8*>(buf + WIDE_CHUNK_BYTES / 2 + (size_t)q * 16)};
  } else {
    return ET<T>::from_lds(buf + (size_t)q * 32);
  }
}

// row-indexed arguments of rows m0.. of a pass
__device__ __forceinline__ LinArgs wide_rows(const LinArgs& a0, int m0, int Mt, int epi_nt) {
  LinArgs a = a0;
  const int n_tiles = a0.N >> 4;
  a.M = Mt;
  a.X = a0.X + (size_t)m0 * a0.ldx;
  if (a0.ssq) a.ssq = a0.ssq + (size_t)m0 * a0.nssq;
  if (a0.h) a.h = a0.h + (size_t)m0 * a0.N;
  if (a0.xg) a.xg = a0.xg + (size_t)m0 * a0.N;
  if (a0.ssq_out) a.ssq_out = a0.ssq_out + (size_t)m0 * n_tiles;
  if (a0.act) a.act = a0.act + (size_t)m0 * (a0.N >> 1);
  if (a0.q) a.q = a0.q + (size_t)m0 * a0.n_heads * a0.head_dim;
  if (a0.row_pos) a.row_pos = a0.row_pos + m0;
  if (a0.row_slot) a.row_slot = a0.row_slot + m0;
  if (a0.row_blk) a.row_blk = a0.row_blk + m0;
  if (a0.row_rope) a.row_rope = a0.row_rope + (size_t)m0 * a0.head_dim;
  if (a0.logits) a.logits = a0.logits + (long long)m0 * a0.ld_logits;
  if (a0.amax_val) a.amax_val = a0.amax_val + (size_t)m0 * a0.amax_stride;
  if (a0.amax_idx) a.amax_idx = a0.amax_idx + (size_t)m0 * a0.amax_stride;
  a.NT = epi_nt;
  a.KS = 1;
  a.S = 1;
  a.NJ = 1;
  return a;
}

template <typename T, int PRO, int EPI, int WIDE_WN, bool SPLIT>
__global__ void __launch_bounds__(512) k_linear_wide(LinArgs a0) {
  constexpr int NI = WIDE_WN / 4;   // n-tiles per wave
  extern __shared__ __attribute__((aligned(16))) char lds[];
  __shared__ float s_rs[WIDE_ROWS_TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tl = lane & 15, kg = lane >> 4;
  const int KTF = a0.K >> 5, n_tiles = a0.N >> 4;
  const int NG = (n_tiles + WIDE_WN - 1) / WIDE_WN;
  const int MT = (a0.M + WIDE_ROWS_TILE - 1) / WIDE_ROWS_TILE;
  // SPLIT: K in a0.KS k-ranges, each (n-group, k-range) pair a virtual n-group of its own
  const int S = SPLIT ? a0.KS : 1;
  // workgroup -> (virtual n-group, token tile): the MT token tiles of virtual n-group gv share the
  // XCD gv mod 8
  const int b = blockIdx.x, xcd = b & 7, r = b >> 3;
  const int mt = r % MT, gv = (r / MT) * 8 + xcd;
  if (gv >= NG * S) return;   // padding of the grid to whole XCD rounds; the workgroup leaves together
  const int g = gv / S, ks = gv - g * S;
  const int kt0 = (ks * KTF) / S, KT = ((ks + 1) * KTF) / S - kt0;   // this workgroup's k-tiles
  const int m0 = mt * WIDE_ROWS_TILE;
  const int Mt = min(WIDE_ROWS_TILE, a0.M - m0);
  constexpr int EPI_NT = wide_epi_nt(WIDE_WN);
  const LinArgs a = wide_rows(a0, m0, Mt, EPI_NT);
  const int wn = wave & 3, wm = wave >> 2;

  // weight fragments of n-tiles g*WN + NI*wn + i (past the last n-tile: the last one, never stored)
  const T* wp[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int nt = min(g * WIDE_WN + NI * wn + i, n_tiles - 1);
    wp[i] = reinterpret_cast<const T*>(a.W) + ((size_t)nt * KTF + kt0) * 512 + lane * 8;
  }
  const float* X = a.X + (size_t)kt0 * 32;
  // staged slot q = (ktl*4 + kg') * 128 + row holds x[row][32 (c*CK + ktl) + 8 kg' .. +7]; rows past
  // the tile's last row read its last row (their outputs are never stored). A chunk is read as
  // (8 rows x one k-tile) blocks, one per wave and load: lane (r, e) takes floats 4e..4e+3 of the
  // k-tile in row r, so a load touches 8 cache lines (not 64 rows' pieces), and its LDS stores
  // (half e&1 of slot kg' = e/2) fall on 16 distinct 8-byte bank positions.
  const int NC = (KT + WIDE_CK - 1) / WIDE_CK;
  constexpr int XP = 2 * WIDE_CK;   // 16-byte pieces per thread and chunk (16 x CK blocks / 8 waves)
  static_assert(XP * 512 * 16 == WIDE_ROWS_TILE * WIDE_CK * 32 * 4, "chunk pieces");
  float4 xv[XP];
  auto stage_load = [&](int c) {
#pragma unroll
    for (int u = 0; u < XP; ++u) {
      const int blk = u * 8 + wave, ktl = blk % WIDE_CK;
      const int rr = min((blk / WIDE_CK) * 8 + (lane >> 3), Mt - 1);
      const int kt = min(c * WIDE_CK + ktl, KT - 1);
      xv[u] = *reinterpret_cast<const float4*>(X + (size_t)rr * a.ldx + kt * 32 + (lane & 7) * 4);
    }
  };
  auto stage_store = [&](int c) {
    char* buf = lds + (size_t)(c & 1) * WIDE_CHUNK_BYTES;
#pragma unroll
    for (int u = 0; u < XP; ++u) {
      const int blk = u * 8 + wave, ktl = blk % WIDE_CK, row = (blk / WIDE_CK) * 8 + (lane >> 3);
      const int q = (ktl * 4 + ((lane & 7) >> 1)) * WIDE_ROWS_TILE + row;
      wide_store_half<T>(buf, q, lane & 1, xv[u]);
    }
  };
  typename ET<T>::A wa[NI][WIDE_CK], wb[NI][WIDE_CK];
  auto wload = [&](typename ET<T>::A (&w)[NI][WIDE_CK], int c) {
#pragma unroll
    for (int kk = 0; kk < WIDE_CK; ++kk) {
      const int kt = min(c * WIDE_CK + kk, KT - 1);
#pragma unroll
      for (int i = 0; i < NI; ++i) w[i][kk] = ET<T>::load(wp[i] + (size_t)kt * 512);
    }
  };
  f32x4 acc[NI][4];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto consume = [&](const typename ET<T>::A (&w)[NI][WIDE_CK], int c) {
    const char* buf = lds + (size_t)(c & 1) * WIDE_CHUNK_BYTES;
    const int nk = min(WIDE_CK, KT - c * WIDE_CK);
#pragma unroll
    for (int kk = 0; kk < WIDE_CK; ++kk) {
      if (kk < nk) {
        typename ET<T>::B xb[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          xb[j] = wide_load_slot<T>(buf, (kk * 4 + kg) * WIDE_ROWS_TILE + (wm * 4 + j) * 16 + tl);
#pragma unroll
        for (int i = 0; i < NI; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) ET<T>::mma(acc[i][j], w[i][kk], xb[j]);
      }
    }
  };

  stage_load(0);
  wload(wa, 0);
  stage_store(0);
  __syncthreads();
  // chunk c (weights in wa, activations in buffer 0), then chunk c+1 (wb, buffer 1). The next
  // chunk's loads are issued unconditionally (indices clamped to the last k-tile; a chunk past the
  // end is staged but never consumed): under a data-dependent branch the compiler's wait counts
  // merge the path without the loads, and every chunk then waits for all loads in flight,
  // including the prefetch just issued.
  for (int c = 0; c < NC; c += 2) {
    stage_load(c + 1);
    wload(wb, c + 1);
    consume(wa, c);
    stage_store(c + 1);
    __syncthreads();
    stage_load(c + 2);
    wload(wa, c + 2);
    consume(wb, c + 1);
    stage_store(c + 2);
    __syncthreads();
  }

  if constexpr (SPLIT) {
    // the k-range's partial tile: part[ks][row][feature] over the pass's rows, added in k-range
    // order by k_wide_splitk_reduce, which runs the epilogue
    float* pp = a0.part + ((size_t)ks * a0.M + m0) * a0.N;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int nt = g * WIDE_WN + NI * wn + i;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = (wm * 4 + j) * 16 + tl;
        if (nt < n_tiles && row < Mt)
          *reinterpret_cast<float4*>(pp + (size_t)row * a0.N + nt * 16 + 4 * kg) =
              make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      }
    }
    return;
  }

  // RMSNorm row scales, then the tile in groups of EPI_NT n-tiles through the staging buffers:
  // Y[lt][row][16], lane (tl, kg) holding features 4kg..4kg+3 of its n-tile for row (4wm+j)*16 + tl
  if constexpr (PRO == PRO_NORM) {
    const float ssv[4] = {0.f, 0.f, 0.f, 0.f};
    for (int m = wave; m < Mt; m += 8) {
      const float rs = wave_row_scale(a, m, ssv, false);
      if (lane == 0) s_rs[m] = rs;
    }
  }
  float* Y = reinterpret_cast<float*>(lds);
  constexpr int YS = WIDE_ROWS_TILE * 16;   // floats per local n-tile
  constexpr int HALVES = WIDE_WN / EPI_NT;
#pragma unroll
  for (int half = 0; half < HALVES; ++half) {
    const Grp gr{HALVES * g + half, HALVES * NG};   // n-tiles (HALVES g + half) * EPI_NT + local tile
    EpiPre epre{};
    epi_load<EPI>(a, gr, tid, epre);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int lt = NI * wn + i;   // a wave's n-tiles may straddle two groups
      if (lt / EPI_NT == half) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<float4*>(Y + (size_t)(lt % EPI_NT) * YS + ((wm * 4 + j) * 16 + tl) * 16 + 4 * kg) =
              make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      }
    }
    __syncthreads();
    if constexpr (PRO == PRO_NORM) {
      for (int e = tid; e < EPI_NT * Mt * 16; e += 512) {
        const int lt = e / (Mt * 16), rem = e - lt * Mt * 16;
        Y[(size_t)lt * YS + rem] *= s_rs[rem >> 4];
      }
      __syncthreads();
    }
    linear_epilogue<T, EPI>(a, gr, Y, YS, epre);
    __syncthreads();   // the epilogue is done with Y before the next group overwrites it
  }
}

// k-range partials of a split wide pass (the residual projections) added in k-range order from 0,
// then the residual epilogue of linear_epilogue (h += y, xg = h * gain of the next norm, and the
// per-16-feature sums of squares in the same xor order): a workgroup per 128 features x
// WIDE_RED_ROWS rows, 4 rows per thread with all their loads issued before the first store, each
// row's 128 features read and written as one contiguous 512-byte run.
constexpr int WIDE_RED_ROWS = 16;
__global__ void __launch_bounds__(512) k_wide_splitk_resid(LinArgs a, const float* part) {
  constexpr int RPT = WIDE_RED_ROWS / 4;   // rows per thread
  const int tid = threadIdx.x, f = tid & 127, rsub = tid >> 7;
  const int n_tiles = a.N >> 4, nt = blockIdx.x * 8 + (f >> 4);
  const int m0 = blockIdx.y * WIDE_RED_ROWS;
  const size_t stride = (size_t)a.M * a.N;
  const int S = a.KS;
  if (nt >= n_tiles) return;   // whole 16-lane groups leave together
  const int col = nt * 16 + (f & 15);
  const float g = a.gain_next[col];
  float v[RPT][WIDE_SPLIT_MAX], h[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int m = min(m0 + rsub + 4 * i, a.M - 1);   // rows past the pass re-read its last row, never stored
    const size_t off = (size_t)m * a.N + col;
#pragma unroll
    for (int k = 0; k < WIDE_SPLIT_MAX; ++k) v[i][k] = k < S ? part[k * stride + off] : 0.f;
    h[i] = a.h[off];
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int m = m0 + rsub + 4 * i;   // uniform across the wave (a wave is 64 features of one row)
    float y = 0.f;
#pragma unroll
    for (int k = 0; k < WIDE_SPLIT_MAX; ++k)
      if (k < S) y += v[i][k];
    const float hv = h[i] + y;
    float s = hv * hv;
    s += __shfl_xor(s, 8);
    s += __shfl_xor(s, 4);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 1);
    if (m < a.M) {
      const size_t off = (size_t)m * a.N + col;
      a.h[off] = hv;
      a.xg[off] = hv * g;
      if ((f & 15) == 0) a.ssq_out[(size_t)m * n_tiles + nt] = s;
    }
  }
}

// Reduce per-n-group argmax partials of one row; lowest token id wins among equal maxima.
__global__ void __launch_bounds__(256) k_argmax_finalize(const float* val, const int* idx, int stride, int n_parts,
                                                         int* tok_out, int tok_stride) {
  const int m = blockIdx.x, tid = threadIdx.x;
  __shared__ float s_v[256];
  __shared__ int s_i[256];
  float best = NEG_INF;
  int bi = -1;
  for (int j = tid; j < n_parts; j += blockDim.x) {
    const float v = val[(size_t)m * stride + j];
    const int i = idx[(size_t)m * stride + j];
    if (i >= 0 && (bi < 0 || v > best || (v == best && i < bi))) { best = v; bi = i; }
  }
  s_v[tid] = best;
  s_i[tid] = bi;
  __syncthreads();
  for (int o = blockDim.x / 2; o > 0; o >>= 1) {
    if (tid < o) {
      const float v = s_v[tid + o];
      const int i = s_i[tid + o];
      if (i >= 0 && (s_i[tid] < 0 || v > s_v[tid] || (v == s_v[tid] && i < s_i[tid]))) { s_v[tid] = v; s_i[tid] = i; }
    }
    __syncthreads();
  }
  if (tid == 0) tok_out[m * tok_stride] = s_i[0] < 0 ? 0 : s_i[0];
}

// ---------------------------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------------------------
// Waves (n-tiles) per workgroup of the split-K kernel: 8, or fewer (down to 4) where that gives
// the busiest CU at least 30% fewer weight tiles with the grid's workgroups spread evenly over the
// 256 CUs: the 2560-wide projections (down: 160 n-tiles x 16 k-ranges make 320 workgroups of 8,
// so 64 CUs stream two, against 512 of 5, two on every CU; O: 160 workgroups of 8 leave 96 CUs
// idle, 256 of 5 fill them). Measured: verify down 17.9 -> 16.0 us at 5 rows, O 16.4 -> 15.4 us at
// 40 rows; QKV (384 n-tiles, 25% by this count) was slower with 6. Each wave's work and summation
// order are the same for any choice.
static int splitk_nt(int n_tiles, int ks) {
  constexpr int CUS = 256;
  auto cost = [&](int nt) {   // weight tiles per k-range on the busiest CU
    const long long wgs = (long long)((n_tiles + nt - 1) / nt) * ks;
    return (wgs + CUS - 1) / CUS * nt;
  };
  int best = 8;
  for (int nt = 7; nt >= 4; --nt)
    if (cost(nt) < cost(best)) best = nt;
  return 10 * cost(best) <= 7 * cost(8) ? best : 8;
}

size_t linear_lds_bytes(int M, int K, int NT, int KS, int S, int NJ, int kind) {
  (void)S;
  if (kind == LIN_LDS) {
    const size_t x = lds_x_bytes(M, K >> 5), part = (size_t)(NJ * NT * KS * M + 1) * 16 * sizeof(float);
    return x + part <= linear_lds_limit() ? x + part : std::max(x, part);
  }
  if (kind == LIN_SPLITK) {
    const int nk_max = ((K >> 5) + KS - 1) / KS;
    return (size_t)nk_max * 4 * M * 32 + 64;
  }
  if (kind == LIN_WIDE) return WIDE_LDS;
  return (size_t)(NT * KS * M * 16) * sizeof(float);
}

// ---------------------------------------------------------------------------------------------
// LM head for 16 < M <= 64 rows (batched verification, draft trees of more than 16 nodes): the
// activation rows of all M tokens do not fit LDS whole (4 bytes per element as MFMA B slots), so
// they are staged in chunks of HEAD_CK k-tiles, double-buffered: the loads of chunk c+1 are issued
// before chunk c is consumed and written to the other buffer after it. Each of the 8 waves
// streams one n-tile over all of K in k order (KS = 1, as the narrow kernel does for any M), for TT
// token tiles of 16 rows, so every row's logits are bit-identical to a pass of fewer rows. A
// workgroup has HEAD_WIDE_NT = 16 waves (n-tiles), so the 40 staged rows of a batch-8 verification
// are read by 594 workgroups instead of 1187 (the argmax partials are per 16-n-tile group; the
// maximum over them is the same).
// ---------------------------------------------------------------------------------------------
constexpr int HEAD_CK = 8;   // k-tiles per staged chunk (= the weight ring depth)
static size_t g_lds_limit = 65536;   // dynamic LDS one workgroup may use (set by configure_kernels)

template <typename T, int TT, int NW>
__global__ void __launch_bounds__(NW * 64) k_linear_head_chunked(LinArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  __shared__ float s_rs[64];
  constexpr int P = HEAD_CK;
  constexpr int NTH = NW * 64;
  constexpr int XI = (HEAD_CK * 4 * 16 * TT + NTH - 1) / NTH;   // staged items per thread and chunk
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int KT = a.K >> 5, n_tiles = a.N >> 4, M = a.M;
  const int tl = lane & 15, kg = lane >> 4;
  const Grp gr{(int)blockIdx.x, (int)gridDim.x};
  const int nt = blockIdx.x * a.NT + wave;
  const T* w0 = reinterpret_cast<const T*>(a.W) + (size_t)(nt < n_tiles ? nt : 0) * KT * 512 + lane * 8;
  const size_t chunk_bytes = (size_t)HEAD_CK * 4 * M * 32;
  const size_t zero_off = 2 * chunk_bytes;
  const int NC = (KT + HEAD_CK - 1) / HEAD_CK;

  EpiPre epre{};
  epi_load<EPI_HEAD>(a, gr, tid, epre);
  float ssv[4] = {0.f, 0.f, 0.f, 0.f};
  const bool pre = preload_row_ssq(a, wave, ssv);

  // chunk c's items q = (ktl*4 + kg)*M + r hold x[r][32(c*CK + ktl) + 8kg .. +7]; loaded branch-free
  // (items past the chunk reload item 0 and are not written)
  float xv[XI][8];
  auto stage_load = [&](int c) {
    const int nkc = min(HEAD_CK, KT - c * HEAD_CK), items = nkc * 4 * M;
#pragma unroll
    for (int u = 0; u < XI; ++u) {
      const int q = u * NTH + tid, qc = q < items ? q : 0;
      const int r = qc % M, rest = qc / M;
      load8(a.X + (size_t)r * a.ldx + (size_t)c * HEAD_CK * 32 + rest * 8, xv[u]);
    }
  };
  auto stage_store = [&](int c) {
    const int nkc = min(HEAD_CK, KT - c * HEAD_CK), items = nkc * 4 * M;
    char* buf = lds + (c & 1) * chunk_bytes;
#pragma unroll
    for (int u = 0; u < XI; ++u) {
      const int q = u * NTH + tid;
      if (q < items) ET<T>::to_lds(buf + (size_t)q * 32, xv[u]);
    }
  };

  stage_load(0);
  typename ET<T>::A wb[P];
#pragma unroll
  for (int p = 0; p < P; ++p) wb[p] = ET<T>::load_nt(w0 + (size_t)min(p, KT - 1) * 512);
  stage_store(0);
  if (tid < 2) *reinterpret_cast<float4*>(lds + zero_off + tid * 16) = make_float4(0.f, 0.f, 0.f, 0.f);
  __syncthreads();

  f32x4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // every load below is issued unconditionally (the last chunk is reloaded past the end, weight
  // tiles past K re-read the last one, neither is consumed): a load under a data-dependent branch
  // makes the compiler's wait counts assume the path without it, and every refill would then wait
  // for the whole ring
  for (int c = 0; c < NC; ++c) {
    stage_load(min(c + 1, NC - 1));
    const char* buf = lds + (c & 1) * chunk_bytes;
    const int nkc = min(HEAD_CK, KT - c * HEAD_CK);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      if (p < nkc) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          const int m = tt * 16 + tl;
          const char* xb = m < M ? buf + ((size_t)(p * 4 + kg) * M + m) * 32 : lds + zero_off;
          ET<T>::mma(acc[tt], wb[p], ET<T>::from_lds(xb));
        }
      }
      const int nxt = c * HEAD_CK + p + P;
      wb[p] = ET<T>::load_nt(w0 + (size_t)min(nxt, KT - 1) * 512);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (c + 1 < NC) stage_store(c + 1);
    __syncthreads();
  }

  // lane (tl, kg) holds features 4kg..4kg+3 of token tt*16+tl: Y[wave][m][16] over the buffers
  float* Y = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int m = tt * 16 + tl;
    if (m < M) {
      float* dst = Y + ((size_t)wave * M + m) * 16 + 4 * kg;
      dst[0] = acc[tt][0]; dst[1] = acc[tt][1]; dst[2] = acc[tt][2]; dst[3] = acc[tt][3];
    }
  }
  for (int m = wave; m < M; m += a.NT) {
    const float r = wave_row_scale(a, m, ssv, pre && m == wave);
    if (lane == 0) s_rs[m] = r;
  }
  __syncthreads();
  const int per = M * 16;
  for (int e = tid; e < a.NT * per; e += blockDim.x) {
    float y = sum_partials(Y + e, 1, per);   // the one k-range, as the narrow kernel adds it
    y *= s_rs[(e % per) >> 4];
    Y[e] = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI_HEAD>(a, gr, Y, per, epre);
}

size_t head_chunked_lds(int M) { return 2 * (size_t)HEAD_CK * 4 * M * 32 + 32; }

// a launch, optionally stamping timing events at the kernel's start and end
template <typename K, typename... Args>
static void launch(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, const LaunchEvents* ev, Args... args) {
  if (ev) hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, ev->start, ev->stop, 0, args...);
  else hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
}

// Workgroup width (n-tiles) of a wide pass: the candidate with the lowest rounds x width x
// per-tile cost, one workgroup per CU (the kernel holds ~200-240 registers per lane). The per-tile
// cost falls with width, since an activation fragment feeds WN/4 n-tiles (128-feature tiles were
// measured about 1.35x slower per tile than 256-feature ones). The LM head keeps 16 when it ranks
// its logits (its argmax partials are per 8 n-tiles); only the tile-local epilogues take 12 (QKV)
// or 20 (gate/up, the head writing logits only).
template <int EPI>
static int wide_width(int n_tiles, int MT, bool argmax) {
  const bool local = EPI != EPI_HEAD || !argmax;   // every epilogue group tile-local
  const int cands[] = {16, 8, (EPI == EPI_SWIGLU || (EPI == EPI_HEAD && local)) ? 20 : 0, EPI == EPI_QKV ? 12 : 0};
  int best = n_tiles >= 192 ? 16 : 8;
  long long best_cost = -1;
  for (int wn : cands) {
    if (wn == 0 || (!local && wn != 16 && n_tiles >= 192)) continue;
    const int per_tile = wn == 8 ? 135 : wn == 12 ? 112 : wn == 16 ? 100 : 95;
    const long long wgs = (long long)((n_tiles + wn - 1) / wn) * MT;
    const long long cost = (wgs + 255) / 256 * wn * per_tile;
    if (best_cost < 0 || cost < best_cost || (cost == best_cost && wn > best)) {
      best = wn;
      best_cost = cost;
    }
  }
  return best;
}

// K-ranges of a residual projection's wide pass (8-n-tile workgroups): as many as keep the
// workgroups of a 1024-row pass (8 token tiles) within two per CU (two 64 KB-LDS workgroups fit one
// CU), at most WIDE_SPLIT_MAX. The count depends on the shape only, so a row's output does not
// depend on the pass's row count. The 2560-wide projections of the 4B model (20 n-groups) take 3:
// 480 workgroups; measured on its 1024-token prefill: 26.7 ms unsplit, 27.3 / 24.7 / 25.5 ms with
// 2 / 3 / 4 k-ranges (2 leaves 64 CUs with two workgroups and the rest with one, 4 needs a third).
static int wide_split(int n_tiles, int KT) {
  constexpr int SLOTS = 2 * 256, MT_REF = 8;
  const int ng = (n_tiles + 7) / 8;
  const int S = std::max(1, std::min(SLOTS / (ng * MT_REF), WIDE_SPLIT_MAX));
  return std::min(S, KT);
}

template <typename T, int PRO, int EPI>
static void launch_linear_pe(const LinArgs& a0, int kind, hipStream_t s, const LaunchEvents* ev) {
  LinArgs a = a0;
  const int n_tiles = a.N >> 4;
  const int n_groups = (n_tiles + a.NT - 1) / a.NT;
  if (kind == LIN_LDS) {
    const dim3 grid((n_groups + a.NJ - 1) / a.NJ);
    const dim3 block(64 * a.NT * a.KS);
    const size_t lds = linear_lds_bytes(a.M, a.K, a.NT, a.KS, a.S, a.NJ, kind);
    const bool alias = lds < lds_x_bytes(a.M, a.K >> 5) + (size_t)(a.NJ * a.NT * a.KS * a.M + 1) * 16 * sizeof(float);
    if (alias) launch(k_linear_lds<T, PRO, EPI, true>, grid, block, lds, s, ev, a);
    else launch(k_linear_lds<T, PRO, EPI, false>, grid, block, lds, s, ev, a);
    return;
  }
  if (kind == LIN_WIDE) {
    const int MT = (a.M + WIDE_ROWS_TILE - 1) / WIDE_ROWS_TILE;
    const int wn = wide_width<EPI>(n_tiles, MT, a.amax_val != nullptr);
    const int NG = (n_tiles + wn - 1) / wn;
    const dim3 grid((unsigned)((NG + 7) / 8 * 8 * MT)), block(512);
    if constexpr (PRO == PRO_PLAIN && EPI == EPI_RESID) {
      const int S = wn == 8 ? wide_split(n_tiles, a.K >> 5) : 1;
      if (S > 1) {
        a.KS = S;
        const LaunchEvents e0{ev ? ev->start : nullptr, nullptr}, e1{nullptr, ev ? ev->stop : nullptr};
        launch(k_linear_wide<T, PRO, EPI, 8, true>, dim3((unsigned)((NG * S + 7) / 8 * 8 * MT)), block, WIDE_LDS, s,
               ev ? &e0 : nullptr, a);
        const dim3 rgrid((unsigned)((n_tiles + 7) / 8), (unsigned)((a.M + WIDE_RED_ROWS - 1) / WIDE_RED_ROWS));
        launch(k_wide_splitk_resid, rgrid, block, 0, s, ev ? &e1 : nullptr, a, (const float*)a.part);
        return;
      }
    }
    switch (wn) {
      case 20: if constexpr (EPI == EPI_SWIGLU || EPI == EPI_HEAD) launch(k_linear_wide<T, PRO, EPI, 20, false>, grid, block, WIDE_LDS, s, ev, a); break;
      case 12: if constexpr (EPI == EPI_QKV) launch(k_linear_wide<T, PRO, EPI, 12, false>, grid, block, WIDE_LDS, s, ev, a); break;
      case 16: launch(k_linear_wide<T, PRO, EPI, 16, false>, grid, block, WIDE_LDS, s, ev, a); break;
      default: launch(k_linear_wide<T, PRO, EPI, 8, false>, grid, block, WIDE_LDS, s, ev, a); break;
    }
    return;
  }
  if (kind == LIN_SPLITK) {
    const int nk_max = ((a.K >> 5) + a.KS - 1) / a.KS;
    LinArgs b = a;
    b.NT = splitk_nt(n_tiles, a.KS);
    b.NJ = 1;
    const dim3 grid((n_tiles + b.NT - 1) / b.NT, a.KS), block(64 * b.NT);
    const size_t lds = (size_t)nk_max * 4 * a.M * 32 + 64;   // + zero slot + dummy slot
    const LaunchEvents e0{ev ? ev->start : nullptr, nullptr}, e1{nullptr, ev ? ev->stop : nullptr};
    const int xi = (nk_max * 4 * a.M + (int)block.x - 1) / (int)block.x <= 4 ? 4 : 8;
    const LaunchEvents* e = ev ? &e0 : nullptr;
    switch ((a.M + 15) / 16 * 16 + xi) {
      case 20: launch(k_linear_splitk<T, 1, 4, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 24: launch(k_linear_splitk<T, 1, 8, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 36: launch(k_linear_splitk<T, 2, 4, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 40: launch(k_linear_splitk<T, 2, 8, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 52: launch(k_linear_splitk<T, 3, 4, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 56: launch(k_linear_splitk<T, 3, 8, PRO>, grid, block, lds, s, e, b, a.part); break;
      case 68: launch(k_linear_splitk<T, 4, 4, PRO>, grid, block, lds, s, e, b, a.part); break;
      default: launch(k_linear_splitk<T, 4, 8, PRO>, grid, block, lds, s, e, b, a.part); break;
    }
    // one output element per thread (the epilogue loads each thread's row data up front)
    LinArgs r = a;
    r.NT = 1;
    r.NJ = 1;
    const int rthreads = (a.M * 16 + 63) / 64 * 64;
    launch(k_splitk_reduce<T, PRO, EPI>, dim3(n_tiles), dim3(rthreads), (size_t)a.M * 16 * sizeof(float), s,
           ev ? &e1 : nullptr, r, (const float*)a.part);
    return;
  }
  a.NJ = 1;
  const dim3 grid(n_groups), block(64 * a.NT * a.KS);
  const int TT = (a.M + 15) / 16;
  if constexpr (EPI == EPI_HEAD) {
    if (a.M > 16 && a.KS == 1 && a.NT == HEAD_WIDE_NT && a.S == 1 && head_chunked_lds(a.M) <= g_lds_limit) {
      const size_t lds_h = head_chunked_lds(a.M);
      switch (TT) {
        case 2: launch(k_linear_head_chunked<T, 2, HEAD_WIDE_NT>, grid, block, lds_h, s, ev, a); break;
        case 3: launch(k_linear_head_chunked<T, 3, HEAD_WIDE_NT>, grid, block, lds_h, s, ev, a); break;
        default: launch(k_linear_head_chunked<T, 4, HEAD_WIDE_NT>, grid, block, lds_h, s, ev, a); break;
      }
      return;
    }
  }
  const size_t lds = linear_lds_bytes(a.M, a.K, a.NT, a.KS, a.S, 1, kind);
  switch (TT) {
    case 1: launch(k_linear_mfma<T, PRO, EPI, 1>, grid, block, lds, s, ev, a); break;
    case 2: launch(k_linear_mfma<T, PRO, EPI, 2>, grid, block, lds, s, ev, a); break;
    case 3: launch(k_linear_mfma<T, PRO, EPI, 3>, grid, block, lds, s, ev, a); break;
    default: launch(k_linear_mfma<T, PRO, EPI, 4>, grid, block, lds, s, ev, a); break;
  }
}

template <typename T>
void launch_linear(const LinArgs& a, int prologue, int epilogue, int kind, hipStream_t s, const LaunchEvents* ev) {
  if (prologue == PRO_NORM) {
    switch (epilogue) {
      case EPI_QKV: launch_linear_pe<T, PRO_NORM, EPI_QKV>(a, kind, s, ev); break;
      case EPI_SWIGLU: launch_linear_pe<T, PRO_NORM, EPI_SWIGLU>(a, kind, s, ev); break;
      default: launch_linear_pe<T, PRO_NORM, EPI_HEAD>(a, kind, s, ev); break;
    }
  } else {
    launch_linear_pe<T, PRO_PLAIN, EPI_RESID>(a, kind, s, ev);
  }
}

void launch_argmax_finalize(const float* val, const int* idx, int stride, int n_parts, int M, int* tok_out,
                            int tok_stride, hipStream_t s) {
  hipLaunchKernelGGL(k_argmax_finalize, dim3(M), dim3(256), 0, s, val, idx, stride, n_parts, tok_out, tok_stride);
}

template <typename T, int PRO, int EPI>
static bool allow_big_lds(int bytes) {
  const void* fns[] = {reinterpret_cast<const void*>(&k_linear_lds<T, PRO, EPI, false>),
                       reinterpret_cast<const void*>(&k_linear_lds<T, PRO, EPI, true>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 1, 4, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 1, 8, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 2, 4, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 2, 8, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 3, 4, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 3, 8, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 4, 4, PRO>),
                       reinterpret_cast<const void*>(&k_linear_splitk<T, 4, 8, PRO>),
                       reinterpret_cast<const void*>(&k_linear_head_chunked<T, 2, HEAD_WIDE_NT>),
                       reinterpret_cast<const void*>(&k_linear_head_chunked<T, 3, HEAD_WIDE_NT>),
                       reinterpret_cast<const void*>(&k_linear_head_chunked<T, 4, HEAD_WIDE_NT>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 1>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 2>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 3>),
                       reinterpret_cast<const void*>(&k_linear_mfma<T, PRO, EPI, 4>),
                       reinterpret_cast<const void*>(&k_linear_wide<T, PRO, EPI, 16, false>),
                       reinterpret_cast<const void*>(&k_linear_wide<T, PRO, EPI, 8, false>)};
  bool ok = true;
  for (const void* f : fns) ok &= hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess;
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_HEAD)
    ok &= hipFuncSetAttribute(reinterpret_cast<const void*>(&k_linear_wide<T, PRO, EPI, 20, false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess;
  if constexpr (EPI == EPI_QKV)
    ok &= hipFuncSetAttribute(reinterpret_cast<const void*>(&k_linear_wide<T, PRO, EPI, 12, false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess;
  if constexpr (PRO == PRO_PLAIN && EPI == EPI_RESID)
    ok &= hipFuncSetAttribute(reinterpret_cast<const void*>(&k_linear_wide<T, PRO, EPI, 8, true>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess;
  return ok;
}


// Dynamic LDS available to one linear workgroup: the device's per-block limit, raised to the
// opt-in limit when every linear kernel accepted it (failed opt-ins are cleared and ignored).
hipError_t configure_kernels(int bf16) {
  int dev = 0, base = 0, optin = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipGetLastError();
  if (hipDeviceGetAttribute(&base, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && base > 0)
    g_lds_limit = (size_t)base;
  if (hipDeviceGetAttribute(&optin, hipDeviceAttributeSharedMemPerBlockOptin, dev) == hipSuccess &&
      (size_t)optin > g_lds_limit) {
    bool ok;
    if (bf16) {
      ok = allow_big_lds<uint16_t, PRO_NORM, EPI_QKV>(optin) & allow_big_lds<uint16_t, PRO_NORM, EPI_SWIGLU>(optin) &
           allow_big_lds<uint16_t, PRO_NORM, EPI_HEAD>(optin) & allow_big_lds<uint16_t, PRO_PLAIN, EPI_RESID>(optin);
    } else {
      ok = allow_big_lds<float, PRO_NORM, EPI_QKV>(optin) & allow_big_lds<float, PRO_NORM, EPI_SWIGLU>(optin) &
           allow_big_lds<float, PRO_NORM, EPI_HEAD>(optin) & allow_big_lds<float, PRO_PLAIN, EPI_RESID>(optin);
    }
    if (ok) g_lds_limit = (size_t)optin;
  }
  (void)hipGetLastError();
  return hipSuccess;
}

size_t linear_lds_limit() { return g_lds_limit; }

template void launch_linear<uint16_t>(const LinArgs&, int, int, int, hipStream_t, const LaunchEvents*);
template void launch_linear<float>(const LinArgs&, int, int, int, hipStream_t, const LaunchEvents*);

}  // namespace seedk
