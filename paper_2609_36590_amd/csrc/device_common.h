// Device-side helpers shared by the gfx950 kernels of the SEED decode path.
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
#pragma once
#include "kernels.h"

#include <math.h>

namespace seedk {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

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
  // streaming (non-temporal) load for data read once per pass: weights
  __device__ static A load_nt(const uint16_t* p) {
    const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return A{make_uint4(t.x, t.y, t.z, t.w)};
  }
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
  // B operand kept in LDS as 32 bytes per lane slot: 8 bf16 hi, then 8 bf16 lo
  __device__ static void to_lds(char* p, const float x[8]) {
    const B b = split(x);
    *reinterpret_cast<bf16x8*>(p) = b.hi;
    *reinterpret_cast<bf16x8*>(p + 16) = b.lo;
  }
  __device__ static B from_lds(const char* p) {
    return B{*reinterpret_cast<const bf16x8*>(p), *reinterpret_cast<const bf16x8*>(p + 16)};
  }
  // half `hf` (values 4hf..4hf+3) of a slot: the same bytes to_lds writes for them
  __device__ static void to_lds_half(char* p, int hf, const float4 x) {
    const float v[4] = {x.x, x.y, x.z, x.w};
    bf16x4 h, l;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      __bf16 t = (__bf16)v[j];
      h[j] = t;
      l[j] = (__bf16)(v[j] - (float)t);
    }
    *reinterpret_cast<bf16x4*>(p + hf * 8) = h;
    *reinterpret_cast<bf16x4*>(p + 16 + hf * 8) = l;
  }
};

template <>
struct ET<float> {
  struct A { float4 a, b; };
  struct B { float x[8]; };
  __device__ static A load(const float* p) {
    return A{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
  }
  __device__ static A load_nt(const float* p) {
    const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p) + 1);
    return A{make_float4(a[0], a[1], a[2], a[3]), make_float4(b[0], b[1], b[2], b[3])};
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
  // B operand kept in LDS as 32 bytes per lane slot: 8 fp32
  __device__ static void to_lds(char* p, const float x[8]) {
    reinterpret_cast<float4*>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
  }
  __device__ static B from_lds(const char* p) {
    const float4 u = reinterpret_cast<const float4*>(p)[0], v = reinterpret_cast<const float4*>(p)[1];
    return B{{u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w}};
  }
  __device__ static void to_lds_half(char* p, int hf, const float4 x) { reinterpret_cast<float4*>(p)[hf] = x; }
};

__device__ __forceinline__ void load8(const float* p, float x[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// Online-softmax merge (base 2) of a partial (m_c, l_c, o_c) into a running (m_r, l_r, o_r).
// A partial with m = -inf (nothing visible) is an exact identity of this merge.
__device__ __forceinline__ void softmax_merge(float& m_r, float& l_r, float* o_r, float m_c, float l_c,
                                              const float* o_c, int n) {
  const float m_n = fmaxf(m_r, m_c);
  const float ar = (m_r == NEG_INF) ? 0.f : exp2f(m_r - m_n);
  const float ac = (m_c == NEG_INF) ? 0.f : exp2f(m_c - m_n);
  l_r = l_r * ar + l_c * ac;
  for (int i = 0; i < n; ++i) o_r[i] = o_r[i] * ar + o_c[i] * ac;
  m_r = m_n;
}

}  // namespace seedk
