// Device helpers shared by the libtrace kernels (gfx950 / CDNA4).
//
// MFMA fragment conventions (the GPU parity tests in tests/ check every use of them):
//   v_mfma_f32_16x16x32_bf16: lane l holds A[row l%16][k (l/16)*8 + j], j < 8, and
//     B[k (l/16)*8 + j][col l%16]; the 16x16 fp32 result lands in lane l as
//     rows 4*(l/16) + r (r < 4) of column l%16.
//   v_mfma_f32_16x16x4_f32: lane l holds A[row l%16][k l/16] and B[k l/16][col l%16],
//     same result layout.
// Every fragment is 16 bytes per lane: 8 bf16, or 4 fp32 covering four chained
// 16x16x4 steps.  A "k-step" is therefore 32 (bf16) or 16 (fp32) k values, and
// lane l reads bytes [(l/16)*16, (l/16)*16 + 16) of the k-step's 64-byte slice of
// its row.  The k order inside a step is the same for A and B, so the products
// pair up exactly as in the plain sum over k.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

#define TRACE_LOG2E 1.4426950408889634f

// fp32 -> bf16 bits, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ float round_bf(float f) { return bf2f(f2bf(f)); }

template <bool BF> struct Mma;

template <> struct Mma<true> {
  typedef uint16_t T;            // storage of one operand element (bf16 bits)
  static constexpr int KS = 32;  // k values per fragment step
  static constexpr int EPF = 8;  // elements per lane per fragment
  __device__ static __forceinline__ void run(f32x4& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                0, 0);
  }
  __device__ static __forceinline__ T cvt(float x) { return f2bf(x); }
  __device__ static __forceinline__ float val(T x) { return bf2f(x); }
};

template <> struct Mma<false> {
  typedef float T;
  static constexpr int KS = 16;
  static constexpr int EPF = 4;
  __device__ static __forceinline__ void run(f32x4& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
  __device__ static __forceinline__ T cvt(float x) { return x; }
  __device__ static __forceinline__ float val(T x) { return x; }
};

// Eight consecutive operand elements -> fp32.
__device__ __forceinline__ void load8(const uint16_t* p, float* out) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float* out) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
  out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
}
// fp32 x8 -> eight operand elements at p (16 or 32 bytes, aligned).
__device__ __forceinline__ void store8(uint16_t* p, const float* in) {
  uint4 v;
  v.x = (uint32_t)f2bf(in[0]) | ((uint32_t)f2bf(in[1]) << 16);
  v.y = (uint32_t)f2bf(in[2]) | ((uint32_t)f2bf(in[3]) << 16);
  v.z = (uint32_t)f2bf(in[4]) | ((uint32_t)f2bf(in[5]) << 16);
  v.w = (uint32_t)f2bf(in[6]) | ((uint32_t)f2bf(in[7]) << 16);
  *reinterpret_cast<uint4*>(p) = v;
}
__device__ __forceinline__ void store8(float* p, const float* in) {
  *reinterpret_cast<float4*>(p) = make_float4(in[0], in[1], in[2], in[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(in[4], in[5], in[6], in[7]);
}

// Exact-erf GELU of Eq. 3: u * Phi(u), Phi(u) = erfc(-u / sqrt 2) / 2.
__device__ __forceinline__ float gelu_f(float u) { return u * (0.5f * erfcf(-u * 0.70710678118654752f)); }
// d/du [u Phi(u)] = Phi(u) + u phi(u).
__device__ __forceinline__ float gelu_grad_f(float u) {
  float Phi = 0.5f * erfcf(-u * 0.70710678118654752f);
  float phi = expf(-0.5f * u * u) * 0.3989422804014327f;
  return Phi + u * phi;
}

// GELU with erf by Abramowitz & Stegun, Handbook of Mathematical Functions,
// 7.1.28: erf(x) = 1 - (1 + a1 x + ... + a6 x^6)^-16 for x >= 0, |error| <= 3e-7.
// GELU(u) = u (1 + erf(u/sqrt2)) / 2 = (u + |u| - |u| / p(|u|/sqrt2)^16) / 2.
// Absolute error <= 1.5e-7 |u|; used where the exact form is not required.
__device__ __forceinline__ float gelu_as(float u) {
  const float au = fabsf(u);
  const float x = au * 0.70710678118654752f;
  float p = fmaf(4.30638e-5f, x, 2.765672e-4f);
  p = fmaf(p, x, 1.520143e-4f);
  p = fmaf(p, x, 9.2705272e-3f);
  p = fmaf(p, x, 4.22820123e-2f);
  p = fmaf(p, x, 7.05230784e-2f);
  p = fmaf(p, x, 1.0f);
  p = p * p;
  p = p * p;
  p = p * p;
  p = p * p;
  const float r = __builtin_amdgcn_rcpf(p);
  return 0.5f * fmaf(-au, r, u + au);
}

// 2 GELU(u) by the same 7.1.28 formula, with the 1/sqrt2 folded into the
// coefficients (b_i = a_i / 2^(i/2), a polynomial in |u|) and the factor 1/2
// left to the caller: 2 GELU(u) = u + |u| - |u| / p(|u|)^16.  Twelve vector
// operations and one reciprocal; |error| <= 7.5e-7 max(1, |u|).
__device__ __forceinline__ float gelu2_as(float u) {
  const float au = fabsf(u);
  float p = fmaf(5.382975e-6f, au, 4.889063564e-5f);
  p = fmaf(p, au, 3.8003575e-5f);
  p = fmaf(p, au, 3.277626324e-3f);
  p = fmaf(p, au, 2.114100615e-2f);
  p = fmaf(p, au, 4.986734697e-2f);
  p = fmaf(p, au, 1.0f);
  p = p * p;
  p = p * p;
  p = p * p;
  p = p * p;
  const float r = __builtin_amdgcn_rcpf(p);
  return fmaf(-au, r, u + au);
}

// 2 GELU(u) = u + |u| - |u| erfc(|u|/sqrt2), with erfc(a/sqrt2) = 2^P(a) and P
// of degree 5, fitted on a in [0, 4 sqrt2] minimax in |u| times the error of
// erfc (a linear program over 8001 points).  P decreases beyond that range (its
// leading coefficient is negative), so 2^P falls to 0 with no clamp.  |error| <=
// 6.8e-7 max(1, |u|) in fp32 (the 7.1.28 form: 7.2e-7).  Eight vector operations,
// the exp2 among them, against thirteen.
__device__ __forceinline__ float gelu2_ex(float u) {
  const float a = fabsf(u);
  float q = fmaf(-5.1878412099e-04f, a, 7.3867838681e-03f);
  q = fmaf(q, a, -5.2537328834e-02f);
  q = fmaf(q, a, -4.5927711224e-01f);
  q = fmaf(q, a, -1.1510829986e+00f);
  q = fmaf(q, a, -8.5913516831e-07f);
  return fmaf(-a, __builtin_amdgcn_exp2f(q), u + a);
}

// GELU'(u) = Phi(u) + u phi(u) with Phi from the same 7.1.28 formula,
// Phi(u) = (1 + sgn(u) (1 - p(|u|)^-16)) / 2, and phi(u) = exp(-u^2/2)/sqrt(2 pi)
// by the hardware base-2 exponential; |error| <= 4e-7 (1 + |u|).  About 18
// vector operations where gelu_grad_f spends erfc and exp.
__device__ __forceinline__ float gelu_grad_as(float u) {
  const float au = fabsf(u);
  float p = fmaf(5.382975e-6f, au, 4.889063564e-5f);
  p = fmaf(p, au, 3.8003575e-5f);
  p = fmaf(p, au, 3.277626324e-3f);
  p = fmaf(p, au, 2.114100615e-2f);
  p = fmaf(p, au, 4.986734697e-2f);
  p = fmaf(p, au, 1.0f);
  p = p * p;
  p = p * p;
  p = p * p;
  p = p * p;
  const float h = 0.5f * __builtin_amdgcn_rcpf(p);  // (1 - erf(|u|/sqrt2)) / 2
  const float Phi = u >= 0.f ? 1.f - h : h;
  const float phi = 0.3989422804014327f * __builtin_amdgcn_exp2f(-0.7213475204444817f * u * u);
  return fmaf(u, phi, Phi);
}

// two fp32 -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
  bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Cross-lane reductions on the DPP path (no LDS traffic).  Within aligned
// groups of 4 lanes: quad permutations xor 1 and xor 2; groups of 8 add the
// mirrored half-row (lane i <-> 7 - i), which pairs each quad with the other.
// Each step is one VALU instruction with the DPP operand (v op v[perm]); the
// s_nop gives the two wait states a DPP read needs after a VALU write of its
// source.  (The builtin form leaves a separate DPP move and, for the maximum,
// two canonicalising operations per step.)
#define TRACE_DPP_STEP(NAME, OP, CTRL)                                                                   \
  __device__ __forceinline__ float NAME(float v) {                                                     \
    float r;                                                                                           \
    asm("s_nop 1\n\t" OP " %0, %1, %1 " CTRL " row_mask:0xf bank_mask:0xf" : "=v"(r) : "v"(v));        \
    return r;                                                                                          \
  }
TRACE_DPP_STEP(dpp_add_x1, "v_add_f32_dpp", "quad_perm:[1,0,3,2]")
TRACE_DPP_STEP(dpp_add_x2, "v_add_f32_dpp", "quad_perm:[2,3,0,1]")
TRACE_DPP_STEP(dpp_add_hm, "v_add_f32_dpp", "row_half_mirror")
TRACE_DPP_STEP(dpp_max_x1, "v_max_f32_dpp", "quad_perm:[1,0,3,2]")
TRACE_DPP_STEP(dpp_max_x2, "v_max_f32_dpp", "quad_perm:[2,3,0,1]")
TRACE_DPP_STEP(dpp_max_hm, "v_max_f32_dpp", "row_half_mirror")
#undef TRACE_DPP_STEP
template <int G>  // G = 4 or 8 lanes
__device__ __forceinline__ float group_sum(float v) {
  v = dpp_add_x2(dpp_add_x1(v));
  if constexpr (G == 8) v = dpp_add_hm(v);
  return v;
}
template <int G>
__device__ __forceinline__ float group_max(float v) {
  v = dpp_max_x2(dpp_max_x1(v));
  if constexpr (G == 8) v = dpp_max_hm(v);
  return v;
}

__device__ __forceinline__ float wave_sum16(float v) {  // over the 16 lanes sharing l/16
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  return v;
}
__device__ __forceinline__ float wave_max16(float v) {
  v = fmaxf(v, __shfl_xor(v, 1, 64));
  v = fmaxf(v, __shfl_xor(v, 2, 64));
  v = fmaxf(v, __shfl_xor(v, 4, 64));
  v = fmaxf(v, __shfl_xor(v, 8, 64));
  return v;
}
