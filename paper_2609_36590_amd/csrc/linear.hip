// Weight-streaming linear kernels (MFMA skinny GEMM, VALU GEMV) with fused RMSNorm,
// RoPE + paged-KV write, residual, SwiGLU and LM-head argmax epilogues.
#include "device_common.h"

namespace seedk {

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
      float* xgp = a.xg + (size_t)m * a.N + nt * 16;
      const float* gn = a.gain_next + nt * 16;
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const float v = hp[c] + YV(nl, m, c);
        hp[c] = v;
        xgp[c] = v * gn[c];
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
    // per-workgroup argmax (lowest token id among equal maxima), reduced by a finalize kernel
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
      a.amax_val[(size_t)m * a.amax_stride + blockIdx.x] = best;
      a.amax_idx[(size_t)m * a.amax_stride + blockIdx.x] = bi;
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

// ---------------------------------------------------------------------------------------------
// Weight-streaming skinny GEMM on MFMA: Y[M, N] = X[M, K] W^T, M <= 16*TT.
// Workgroup = NT*KS waves; wave (nl, ks) streams n-tile blockIdx.x*NT+nl over the ks-th
// contiguous range of k-tiles. Partials are reduced across ks in LDS in ks order.
//
// Streaming: each wave keeps P k-tiles in flight, the weight tile (non-temporal) together with
// the matching activation fragment, and refills a slot right after taking its data. Vector
// memory returns complete in issue order, so issuing an operand together with its weight tile
// keeps every wait at "oldest slot only".
//
// RMSNorm consumers get x*g already formed by the producer of x and apply the row scale rs to
// the reduced sums (y = rs * sum_k W (x*g)).
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
    constexpr int P = (TT <= 1) ? 8 : (TT == 2 ? 4 : (TT == 3 ? 3 : 2));
    typename ET<T>::A wb[P];
    float xb[P][TT][8];
    // lanes past the last row read row 0 (branch-free issue) and are zeroed when consumed
    auto issue = [&](int slot, int j) {
      wb[slot] = ET<T>::load_nt(wp + (size_t)j * 512);
#pragma unroll
      for (int tt = 0; tt < TT; ++tt) load8(xp[tt] + j * 32, xb[slot][tt]);
    };
#pragma unroll
    for (int i = 0; i < P; ++i) issue(i, min(i, nk - 1));
    // consume a slot, then refill the same registers: no register copies, so every wait is
    // for the oldest slot only
    int base = 0;
    for (; base + P <= nk; base += P) {
#pragma unroll
      for (int i = 0; i < P; ++i) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          float x[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) x[q] = ok[tt] ? xb[i][tt][q] : 0.f;
          ET<T>::mma(acc[tt], wb[i], ET<T>::split(x));
        }
        issue(i, min(base + i + P, nk - 1));
      }
    }
#pragma unroll
    for (int i = 0; i < P; ++i)
      if (base + i < nk) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          float x[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) x[q] = ok[tt] ? xb[i][tt][q] : 0.f;
          ET<T>::mma(acc[tt], wb[i], ET<T>::split(x));
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
  if constexpr (PRO == PRO_NORM) {
    for (int m = wave; m < M; m += NW) {
      const float r = wave_row_scale(a, m, ssv, pre && m == wave);
      if (lane == 0) s_rs[m] = r;
    }
  }
  __syncthreads();
  for (int e = tid; e < a.NT * M * 16; e += blockDim.x) {
    const int nl2 = e / (M * 16), r = e - nl2 * M * 16;
    float y = 0.f;
    for (int k2 = 0; k2 < a.KS; ++k2) y += s_red[(size_t)(nl2 * a.KS + k2) * M * 16 + r];
    if constexpr (PRO == PRO_NORM) y *= s_rs[r >> 4];
    s_red[(size_t)(nl2 * a.KS) * M * 16 + r] = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, s_red, a.KS * M * 16, 16);
}

// ---------------------------------------------------------------------------------------------
// Weight-streaming GEMV on the vector ALUs (one activation row): same tiles and waves as the
// MFMA kernel; lane (tl, kg) accumulates row tl over its k-slots, then the four k-groups are
// added across lanes and the KS partials in LDS. The activation row sits in LDS; the weight
// stream keeps P tiles in flight from the first instruction on.
// ---------------------------------------------------------------------------------------------
template <typename T, int PRO, int EPI>
__global__ void __launch_bounds__(1024) k_linear_valu(LinArgs a) {
  extern __shared__ float smem[];
  float* s_x = smem;                // [K]
  float* s_red = smem + a.K;        // [NW][16]
  __shared__ float s_rs;
  constexpr int P = 8;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int KT = a.K >> 5, n_tiles = a.N >> 4;
  const int nl = wave / a.KS, ks = wave - nl * a.KS;
  const int nt = blockIdx.x * a.NT + nl;
  const int kg = lane >> 4;
  const bool live = nt < n_tiles;
  const int kt0 = (ks * KT) / a.KS, kt1 = ((ks + 1) * KT) / a.KS;
  const int nk = kt1 - kt0;
  const T* wp = reinterpret_cast<const T*>(a.W) + ((size_t)(live ? nt : 0) * KT + kt0) * 512 + lane * 8;
  typename ET<T>::A wb[P];
  if (live) {
#pragma unroll
    for (int i = 0; i < P; ++i) wb[i] = ET<T>::load_nt(wp + (size_t)min(i, nk - 1) * 512);
  }
  float ssv[4] = {0.f, 0.f, 0.f, 0.f};
  bool pre = false;
  if constexpr (PRO == PRO_NORM) pre = (wave == 0) && preload_row_ssq(a, 0, ssv);
  for (int k = tid; k < a.K; k += blockDim.x) s_x[k] = a.X[k];
  __syncthreads();
  float acc = 0.f;
  if (live) {
    const float* xs = s_x + kg * 8 + kt0 * 32;
    auto step = [&](const typename ET<T>::A& w, int j) {
      float wf[8], xv[8];
      ET<T>::to_f32(w, wf);
      load8(xs + j * 32, xv);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc = fmaf(wf[q], xv[q], acc);
    };
    int base = 0;
    for (; base + P <= nk; base += P) {
#pragma unroll
      for (int i = 0; i < P; ++i) {
        step(wb[i], base + i);
        wb[i] = ET<T>::load_nt(wp + (size_t)min(base + i + P, nk - 1) * 512);
      }
    }
#pragma unroll
    for (int i = 0; i < P; ++i)
      if (base + i < nk) step(wb[i], base + i);
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  if (lane < 16) s_red[wave * 16 + lane] = acc;
  if constexpr (PRO == PRO_NORM) {
    if (wave == 0) {
      const float r = wave_row_scale(a, 0, ssv, pre);
      if (lane == 0) s_rs = r;
    }
  }
  __syncthreads();
  for (int e = tid; e < a.NT * 16; e += blockDim.x) {
    const int nl2 = e >> 4, c = e & 15;
    float y = 0.f;
    for (int k2 = 0; k2 < a.KS; ++k2) y += s_red[(nl2 * a.KS + k2) * 16 + c];
    if constexpr (PRO == PRO_NORM) y *= s_rs;
    s_red[(nl2 * a.KS) * 16 + c] = y;
  }
  __syncthreads();
  linear_epilogue<T, EPI>(a, s_red, a.KS * 16, 16);
}

// Reduce per-workgroup argmax partials of one row; lowest token id wins among equal maxima.
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

void launch_argmax_finalize(const float* val, const int* idx, int stride, int n_parts, int M, int* tok_out,
                            int tok_stride, hipStream_t s) {
  hipLaunchKernelGGL(k_argmax_finalize, dim3(M), dim3(256), 0, s, val, idx, stride, n_parts, tok_out, tok_stride);
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

}  // namespace seedk
