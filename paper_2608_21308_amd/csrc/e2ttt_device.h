// Device-side building blocks shared by the E2-TTT gfx950 kernels.
//
// MFMA tiles are 16x16.  The accumulator ("D") layout of a 16x16 tile is:
// lane l = 16 g + c (g = l / 16, c = l % 16) holds rows 4 g + r (r = 0..3) of
// column c.  A K-step of an MFMA takes, from every lane, a fragment of the
// row (A operand) or column (B operand) numbered c, covering the contraction
// indices {k0 + 16 h + 4 g + r}: h = 0..NH-1, r = 0..3.  The A and B operands
// use the same (lane group, slot) -> k assignment, so the hardware sum over k
// is unchanged; with this assignment a D tile whose ROW index is the
// contraction index is directly usable (after conversion) as half of a bf16
// fragment or as a whole fp32 fragment, without going through LDS.
//
//   bf16: v_mfma_f32_16x16x32_bf16, K-step 32 = two 16-row halves, 8 bf16/lane
//   fp32: v_mfma_f32_16x16x4_f32 x 4, K-step 16, one float per lane per MFMA
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace e2ttt {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4;

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Keeps the instruction scheduler from moving work across this point; used
// between fully unrolled iterations so that operand loads of later
// iterations are not hoisted (which would raise register pressure).
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Returns p unchanged but opaque to the optimiser, so that addresses derived
// from it are formed where they are used instead of being hoisted out of the
// chunk loop and kept live in registers for its whole duration.
template <class T>
__device__ __forceinline__ T* opaque_ptr(T* p) {
  asm volatile("" : "+s"(p));
  return p;
}
// Same for a per-lane integer (kept in a VGPR).
__device__ __forceinline__ int opaque_lane(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Thread indices re-derived behind an opaque copy of threadIdx.x.  A kernel
// phase that starts with E2TTT_LANE_IDS forms its per-lane address arithmetic
// inside the phase; without it the compiler hoists every such address to the
// kernel entry and keeps dozens of them live (or spilled) across the chunk loop.
#define E2TTT_LANE_IDS                                                \
  const int tid = ::e2ttt::opaque_lane((int)threadIdx.x);             \
  const int lane = tid & 63, g = lane >> 4, c = lane & 15, l16 = c;   \
  (void)tid; (void)lane; (void)g; (void)c; (void)l16

template <bool BF> struct OpT;

template <> struct OpT<true> {
  using E = __bf16;                 // element type of LDS operands
  using Q = bf16x4;                 // four consecutive contraction indices
  static constexpr int KC = 32;     // contraction indices per K-step
  static constexpr int NH = 2;      // quads per fragment
  // Row padding of LDS operands: 4 elements (8 bytes), so that row strides
  // are 2 (mod 4) dwords.  Fragment reads (paired 8-byte loads, 16 lanes on
  // 16 consecutive rows per LDS cycle) then touch 32 distinct banks; with a
  // 16-byte pad (stride 0 mod 4) pairs of rows 8 apart share banks.
  static constexpr int PAD = 4;
  struct Frag { Q h[2]; };
  static __device__ __forceinline__ Q cvt(f32x4 x) {
    return Q{(__bf16)x[0], (__bf16)x[1], (__bf16)x[2], (__bf16)x[3]};
  }
  static __device__ __forceinline__ E to_e(float x) { return (__bf16)x; }
  static __device__ __forceinline__ float from_e(E x) { return (float)x; }
  static __device__ __forceinline__ f32x4 mma(f32x4 acc, const Frag& a, const Frag& b) {
    bf16x8 av = __builtin_shufflevector(a.h[0], a.h[1], 0, 1, 2, 3, 4, 5, 6, 7);
    bf16x8 bv = __builtin_shufflevector(b.h[0], b.h[1], 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
  }
};

template <> struct OpT<false> {
  using E = float;
  using Q = f32x4;
  static constexpr int KC = 16;
  static constexpr int NH = 1;
  static constexpr int PAD = 4;
  struct Frag { Q h[1]; };
  static __device__ __forceinline__ Q cvt(f32x4 x) { return x; }
  static __device__ __forceinline__ E to_e(float x) { return x; }
  static __device__ __forceinline__ float from_e(E x) { return x; }
  static __device__ __forceinline__ f32x4 mma(f32x4 acc, const Frag& a, const Frag& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.h[0][0], b.h[0][0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.h[0][1], b.h[0][1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.h[0][2], b.h[0][2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.h[0][3], b.h[0][3], acc, 0, 0, 0);
    return acc;
  }
};

// Fragment of row `row` of a row-major LDS array (leading dimension ld, in
// elements) whose columns are the contraction index, for the K-step at k0.
template <bool BF>
__device__ __forceinline__ typename OpT<BF>::Frag lds_frag(const typename OpT<BF>::E* base,
                                                            int ld, int row, int k0, int g) {
  using O = OpT<BF>;
  typename O::Frag f;
#pragma unroll
  for (int h = 0; h < O::NH; ++h)
    f.h[h] = *reinterpret_cast<const typename O::Q*>(base + row * ld + k0 + 16 * h + 4 * g);
  return f;
}

// --------------------------------------------------------------- activations
// Reciprocal and reciprocal square root on the hardware units (1 ulp).
__device__ __forceinline__ float rcp_f(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float rsq_f(float x) { return __builtin_amdgcn_rsqf(x); }

// GELU(x) = x Phi(x) with Phi the standard normal CDF, evaluated through
// h = Phi(-|x|) = erfc(|x| / sqrt(2)) / 2 and e = exp(-x^2 / 2).  erfc comes
// from Abramowitz & Stegun, Handbook of Mathematical Functions, eq. 7.1.26:
// erfc(z) = t (a1 + a2 t + ... + a5 t^4) exp(-z^2), t = 1 / (1 + p z), z >= 0,
// absolute error at most 1.5e-7.  Here p is pre-multiplied by 1/sqrt(2) and
// the a_k by 1/2, so h = t poly(t) e.  One reciprocal and one exponential
// serve GELU and both of its derivatives:
//   GELU(x)   = max(x, 0) - |x| h
//   GELU'(x)  = Phi(x) + x phi(x),   Phi(x) = 1 - h for x >= 0, h otherwise
//   GELU''(x) = phi(x) (2 - x^2),    phi(x) = e / sqrt(2 pi).
struct GeluParts {
  float h, e, x2;
};
__device__ __forceinline__ GeluParts gelu_parts(float x) {
  GeluParts r;
  r.x2 = x * x;
  r.e = __builtin_amdgcn_exp2f(r.x2 * -0.7213475204444817f);   // 2^(-x^2 log2(e) / 2)
  const float t = rcp_f(fmaf(fabsf(x), 0.23164189f, 1.0f));
  float p = 0.5307027f;
  p = fmaf(p, t, -0.72657603f);
  p = fmaf(p, t, 0.7107069f);
  p = fmaf(p, t, -0.14224836f);
  p = fmaf(p, t, 0.1274148f);
  r.h = (p * t) * r.e;
  return r;
}
__device__ __forceinline__ float gelu_from(float x, const GeluParts& g) {
  return fmaf(-fabsf(x), g.h, fmaxf(x, 0.0f));
}
__device__ __forceinline__ float gelu_f(float x) { return gelu_from(x, gelu_parts(x)); }
// Phi(x) = 1/2 + sign(x) (1/2 - h), branch- and compare-free (a compare per
// element would hold a scalar register pair per element in flight).
__device__ __forceinline__ float gelu_cdf(float x, const GeluParts& g) {
  return 0.5f + copysignf(0.5f - g.h, x);
}
// GELU and GELU'.
struct Act2 {
  float f, d1;
};
__device__ __forceinline__ Act2 gelu2(float x) {
  const GeluParts g = gelu_parts(x);
  return Act2{gelu_from(x, g), fmaf(x * 0.3989423f, g.e, gelu_cdf(x, g))};
}
__device__ __forceinline__ float sigm_f(float x) { return rcp_f(1.0f + __expf(-x)); }
__device__ __forceinline__ float silu_f(float x) { return x * sigm_f(x); }
__device__ __forceinline__ float silu_d1(float x) {
  const float s = sigm_f(x);
  return s * (1.0f + x * (1.0f - s));
}
__device__ __forceinline__ float silu_d2(float x) {
  const float s = sigm_f(x);
  return s * (1.0f - s) * (2.0f + x * (1.0f - 2.0f * s));
}

// An activation with its first two derivatives from one evaluation of the
// transcendental part (one erfc for GELU, one sigmoid for SiLU).
struct Act3 {
  float f, d1, d2;
};
__device__ __forceinline__ Act3 gelu3(float x) {
  const GeluParts g = gelu_parts(x);
  const float pdf = 0.3989423f * g.e;
  return Act3{gelu_from(x, g), fmaf(x, pdf, gelu_cdf(x, g)), pdf * (2.0f - g.x2)};
}
__device__ __forceinline__ Act3 silu3(float x) {
  const float s = sigm_f(x);
  return Act3{x * s, s * (1.0f + x * (1.0f - s)), s * (1.0f - s) * (2.0f + x * (1.0f - 2.0f * s))};
}

// ------------------------------------------------------------- reductions
// DPP lane permutations within a row of 16 lanes (no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
// Sum over the 16 lanes of a DPP row (lanes 16 k .. 16 k + 15); every lane of
// the row receives the sum.
__device__ __forceinline__ float group16_sum(float v) {
  v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);   // row_half_mirror
  v += dpp_f<0x140>(v);   // row_mirror
  return v;
}
// Reduce-scatter of eight values over the 16 lanes of a DPP row: with l16 the
// lane's index in its row and b3 b2 b1 b0 its bits, the lane returns the row
// sum of v[4 b3 + 2 b2 + b1].  Each step pairs lanes that differ in one bit
// (row_mirror: bit 3, row_half_mirror: bit 2, quad perms: bits 1 and 0); a
// lane keeps the half of its values its bit selects and adds the partner's
// copy of that half: 22 VALU operations instead of the 32 of eight group16_sum.
__device__ __forceinline__ float row16_reduce_scatter8(const float (&v)[8], int l16) {
  const bool b3 = (l16 & 8) != 0, b2 = (l16 & 4) != 0, b1 = (l16 & 2) != 0;
  float u[4], h[2];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float keep = b3 ? v[4 + k] : v[k], send = b3 ? v[k] : v[4 + k];
    u[k] = keep + dpp_f<0x140>(send);   // row_mirror
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float keep = b2 ? u[2 + k] : u[k], send = b2 ? u[k] : u[2 + k];
    h[k] = keep + dpp_f<0x141>(send);   // row_half_mirror
  }
  const float keep = b1 ? h[1] : h[0], send = b1 ? h[0] : h[1];
  const float x = keep + dpp_f<0x4E>(send);   // quad_perm [2,3,0,1]
  return x + dpp_f<0xB1>(x);                  // quad_perm [1,0,3,2]
}
// Sum over all 64 lanes, returned to every lane (all lanes must be active).
__device__ __forceinline__ float wave_sum(float v) {
  const int b = __float_as_int(group16_sum(v));
  return (__int_as_float(__builtin_amdgcn_readlane(b, 0)) +
          __int_as_float(__builtin_amdgcn_readlane(b, 16))) +
         (__int_as_float(__builtin_amdgcn_readlane(b, 32)) +
          __int_as_float(__builtin_amdgcn_readlane(b, 48)));
}

// --------------------------------------------------------- streaming access
// Global loads and stores of data a launch touches once (token rows, outputs,
// chunk-start checkpoints, saved activations and LayerNorm rows) are marked
// non-temporal: the L2 evicts those lines first, so that they do not push out
// the exchange slots through which the workgroups of a unit swap partial sums
// every chunk (those stay L2-resident and never need to reach HBM).
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
template <class T>
__device__ __forceinline__ void st_stream(T* p, const T& v) {
  __builtin_nontemporal_store(v, p);
}
template <class T>
__device__ __forceinline__ T ld_stream(const T* p) {
  return __builtin_nontemporal_load(p);
}
__device__ __forceinline__ uint4 ld_stream16(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld_stream16f(const float* p) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

// ----------------------------------------------------------- io element load
template <bool BF> struct IoT;
// (stores are streaming: outputs and gradients are written once per launch)
template <> struct IoT<true> {
  using T = __bf16;
  static __device__ __forceinline__ float ld(const T* p) { return (float)*p; }
  static __device__ __forceinline__ void st(T* p, float x) { st_stream(p, (__bf16)x); }
  // four consecutive values, one 8-byte store (p 8-byte aligned)
  static __device__ __forceinline__ void st4(T* p, f32x4 x) {
    st_stream(reinterpret_cast<bf16x4*>(p),
              bf16x4{(__bf16)x[0], (__bf16)x[1], (__bf16)x[2], (__bf16)x[3]});
  }
};
template <> struct IoT<false> {
  using T = float;
  static __device__ __forceinline__ float ld(const T* p) { return *p; }
  static __device__ __forceinline__ void st(T* p, float x) { st_stream(p, x); }
  // four consecutive values, one 16-byte store (p 16-byte aligned)
  static __device__ __forceinline__ void st4(T* p, f32x4 x) {
    st_stream(reinterpret_cast<f32x4*>(p), x);
  }
};

}  // namespace e2ttt
