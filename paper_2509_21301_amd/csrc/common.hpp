// Shared device helpers for the gfx950 kernels: bf16 storage, MFMA operand packing, reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // bf16 storage (upper 16 bits of an IEEE float)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define NOVA_DEV __device__ __forceinline__

NOVA_DEV float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// float -> bf16, round to nearest even (gfx950 converts in hardware, v_cvt_pk_bf16_f32).
NOVA_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Two floats -> two bf16 in one dword (a in the low half), one conversion instruction.
NOVA_DEV uint32_t pack2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Activation element types: bf16 (storage bf16_t) or fp32.
template <typename T> NOVA_DEV float to_f(T v);
template <> NOVA_DEV float to_f<bf16_t>(bf16_t v) { return bf2f(v); }
template <> NOVA_DEV float to_f<float>(float v) { return v; }
template <typename T> NOVA_DEV T from_f(float v);
template <> NOVA_DEV bf16_t from_f<bf16_t>(float v) { return f2bf(v); }
template <> NOVA_DEV float from_f<float>(float v) { return v; }

// 8 bf16 held as 4 dwords; converts to the MFMA operand type.
struct alignas(16) Frag8 { uint32_t w[4]; };
NOVA_DEV bf16x8 as_bf16x8(const Frag8& f) { return __builtin_bit_cast(bf16x8, f); }
NOVA_DEV Frag8 zero_frag() { Frag8 f; f.w[0] = f.w[1] = f.w[2] = f.w[3] = 0u; return f; }

// Split 8 floats into a bf16 high part and a bf16 low part (x ~= hi + lo to about 2^-17 relative).
NOVA_DEV void split8(const float* x, Frag8& hi, Frag8& lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bf16_t h0 = f2bf(x[2 * i]), h1 = f2bf(x[2 * i + 1]);
    hi.w[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    lo.w[i] = pack2(x[2 * i] - bf2f(h0), x[2 * i + 1] - bf2f(h1));
  }
}

NOVA_DEV f32x4 mfma16(const Frag8& a, const Frag8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}
NOVA_DEV f32x16 mfma32(const Frag8& a, const Frag8& b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

NOVA_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
NOVA_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Rotary angle pos * theta^(-2c/D), evaluated in double and reduced to [0, 2pi) before the
// fp32 sine/cosine, so that the rotation stays accurate at long positions.
NOVA_DEV void rope_sincos(int pos, int c, int D, float theta, float* sn, float* cs) {
  const double inv = exp2(-(2.0 * c / D) * log2((double)theta));
  double ang = (double)pos * inv;
  ang -= 6.283185307179586 * floor(ang * 0.15915494309189535);
  sincosf((float)ang, sn, cs);
}

// erf by the rational approximation of Abramowitz & Stegun, formula 7.1.26 (after Hastings):
// erf(a) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-a^2), t = 1 / (1 + p a), a >= 0,
// absolute error at most 1.5e-7; odd in x.  One reciprocal and one exp, no branches, which makes
// the GELU epilogue of the vision MLP several times cheaper than the library erf.
NOVA_DEV float erf_as(float x) {
  const float a = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, a, 1.0f));
  const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f),
                                      -0.284496736f), 0.254829592f);
  return copysignf(1.0f - poly * __expf(-a * a), x);
}
NOVA_DEV float gelu_erf(float x) { return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f)); }
NOVA_DEV float silu(float x) { return x / (1.0f + __expf(-x)); }

// Kernel timing categories (host side).
enum NovaKernelKind { NK_GEMM = 0, NK_ATTN = 1, NK_GEMV = 2, NK_DECATTN = 3, NK_MISC = 4, NK_COUNT = 5 };
