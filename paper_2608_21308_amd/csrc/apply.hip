// Evaluation of the fast-weight net at a given state, o = f_W(q) (eq. (6):
// the output of a token is the net at its chunk's start state).  Streaming
// decode answers each new token this way from the current chunk-start state
// and advances the state with the chunk update once C tokens have arrived.
//
// One workgroup per (unit, group of up to TT tokens).  The work is a pair of
// matrix-vector products per token over a state that is read once per
// workgroup, so it is bound by HBM reads of W (fp32, P floats per unit):
//   0. every lane issues all of its loads of the state at once (the whole
//      P floats of the unit are in flight together; a workgroup is otherwise
//      latency-bound on a single unit's 2 d dh floats).
//   1. hidden: for every hidden row j, h_j = W1[j,:] . q (SwiGLU: the gate and
//      up rows together).  D/4 lanes hold one row as float4 pieces (a wave
//      reads 64/(D/4) whole rows per load, fully coalesced) and sum their
//      partial dots over a DPP row; the activation goes to LDS.
//   2. output: for every row i of W2 (Wd), y_i = W2[i,:] . a, one wave per
//      row, each lane holding four consecutive hidden indices (one float4
//      load), summed over the wave.
//   3. LayerNorm over the D outputs of each token and the residual, one wave
//      per token; written in the io type.
#include <math.h>

#include "e2ttt.h"
#include "e2ttt_device.h"
#include "e2ttt_internal.h"

namespace e2ttt {
namespace {

constexpr int kApplyWaves = 8;

// Sum over groups of L consecutive lanes (L = 4 or 16), returned to every lane of the group.
template <int L>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(L == 4 || L == 16, "row group of 4 or 16 lanes");
  if constexpr (L == 16) {
    return group16_sum(v);
  } else {
    v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
    return v;
  }
}

__device__ __forceinline__ float gelu_exact(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
__device__ __forceinline__ float silu_exact(float x) { return x / (1.0f + expf(-x)); }

template <int D, bool BF, int FW, int TT>
__global__ void __launch_bounds__(64 * kApplyWaves) apply_kernel(ApplyArgs a) {
  using Io = IoT<BF>;
  using E = typename Io::T;
  constexpr int NWV = kApplyWaves;
  constexpr int L = D / 4;                                   // lanes per row of W1
  constexpr int RPI = 64 / L;                                // W1 rows per wave per load
  constexpr int NR1 = (kApplyMaxDh + NWV * RPI - 1) / (NWV * RPI);  // W1 loads per lane
  constexpr int NR2 = D / NWV;                               // W2 rows per wave
  static_assert(D % NWV == 0 && 4 * 64 >= kApplyMaxDh, "one float4 of W2 per lane and row");
  __shared__ float qs[TT][D];
  __shared__ float hs[TT][kApplyMaxDh];
  __shared__ float ys[TT][D];

  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long u = blockIdx.x / a.groups;
  const int t0 = (int)(blockIdx.x % a.groups) * TT;
  const int nt = min(TT, a.T - t0);
  const E* q = static_cast<const E*>(a.q) + (u * a.T + t0) * D;
  E* out = static_cast<E*>(a.out) + (u * a.T + t0) * D;
  const float* w = a.w + u * a.P;
  const int dh = a.dh;
  const float* w2 = w + (long)(FW == 0 ? 1 : 2) * dh * D;   // W2 (MLP) or Wd (SwiGLU)

  // Every load of this workgroup's share of the state is issued up front, so
  // the whole state (P floats) is in flight at once.
  const int c4 = lane % L, rsub = lane / L;
  f32x4 w1r[NR1], w3r[NR1], w2r[NR2];
#pragma unroll
  for (int k = 0; k < NR1; ++k) {
    const int r = (k * NWV + wv) * RPI + rsub;
    w1r[k] = zero4();
    w3r[k] = zero4();
    if (r < dh) {
      w1r[k] = *reinterpret_cast<const f32x4*>(w + (long)r * D + 4 * c4);
      if constexpr (FW == 1)
        w3r[k] = *reinterpret_cast<const f32x4*>(w + (long)(dh + r) * D + 4 * c4);
    }
  }
  const int j4 = 4 * lane;
  if ((dh & 3) == 0) {   // rows of W2 start 16-byte aligned
#pragma unroll
    for (int k = 0; k < NR2; ++k) {
      const int i = k * NWV + wv;
      w2r[k] = (j4 < dh) ? *reinterpret_cast<const f32x4*>(w2 + (long)i * dh + j4) : zero4();
    }
  } else {
#pragma unroll
    for (int k = 0; k < NR2; ++k) {
      const int i = k * NWV + wv;
#pragma unroll
      for (int e = 0; e < 4; ++e) w2r[k][e] = (j4 + e < dh) ? w2[(long)i * dh + j4 + e] : 0.0f;
    }
  }

  for (int x = threadIdx.x; x < TT * D; x += 64 * NWV) {
    const int t = x / D, i = x % D;
    qs[t][i] = (t < nt) ? Io::ld(q + (long)t * D + i) : 0.0f;
  }
  __syncthreads();

  // 1. hidden rows: h = W1 q (SwiGLU: g = Wg q, up = Wu q), activation to LDS
  f32x4 qv[TT];
#pragma unroll
  for (int t = 0; t < TT; ++t)
    qv[t] = f32x4{qs[t][4 * c4], qs[t][4 * c4 + 1], qs[t][4 * c4 + 2], qs[t][4 * c4 + 3]};
#pragma unroll
  for (int k = 0; k < NR1; ++k) {
    const int r0 = (k * NWV + wv) * RPI;
    if (r0 >= dh) break;   // uniform over the wave
    const int r = r0 + rsub;
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      const float h = group_sum<L>(w1r[k][0] * qv[t][0] + w1r[k][1] * qv[t][1] +
                                   w1r[k][2] * qv[t][2] + w1r[k][3] * qv[t][3]);
      if constexpr (FW == 0) {
        if (r < dh && c4 == 0) hs[t][r] = gelu_exact(h);
      } else {
        const float up = group_sum<L>(w3r[k][0] * qv[t][0] + w3r[k][1] * qv[t][1] +
                                      w3r[k][2] * qv[t][2] + w3r[k][3] * qv[t][3]);
        if (r < dh && c4 == 0) hs[t][r] = silu_exact(h) * up;
      }
    }
  }
  __syncthreads();

  // 2. output rows: y_i = W2[i,:] . a, lane holding hidden indices 4 lane .. 4 lane + 3
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    f32x4 av = zero4();
    if (j4 < dh) {
#pragma unroll
      for (int e = 0; e < 4; ++e) av[e] = (j4 + e < dh) ? hs[t][j4 + e] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < NR2; ++k) {
      const float y = wave_sum(w2r[k][0] * av[0] + w2r[k][1] * av[1] + w2r[k][2] * av[2] +
                               w2r[k][3] * av[3]);
      if (lane == 0) ys[t][k * NWV + wv] = y;
    }
  }
  __syncthreads();

  // 3. LayerNorm (biased variance) and residual, one wave per token
  for (int t = wv; t < nt; t += NWV) {
    const bool act = lane < D;
    const float y = act ? ys[t][lane] : 0.0f;
    float o = y;
    if (a.resln) {
      const float mean = wave_sum(y) * (1.0f / D);
      const float dv = act ? y - mean : 0.0f;
      const float var = wave_sum(dv * dv) * (1.0f / D);
      const float z = dv / sqrtf(var + a.eps);
      const int ic = lane < D ? lane : 0;
      o = qs[t][ic] + (a.ln_a ? fmaf(a.ln_a[(u % a.H) * D + ic], z, a.ln_b[(u % a.H) * D + ic]) : z);
    }
    if (act) Io::st(out + (long)t * D + lane, o);
  }
}

// Head dim 128 (the paper's 1.3B model), hidden width up to 512: a unit's
// state (up to 0.5 MB) does not fit in registers, so it streams through them
// in batches, each batch's loads issued together before any of them is used.
//   1. hidden rows: 32 lanes hold one W1 row as float4 pieces (two rows per
//      wave per load), UB rows of each wave in flight at once; the partial
//      dots are summed over the 32 lanes.
//   2. output rows: one wave per row, each lane holding hidden indices
//      4 lane + 256 h (h < NQ), four rows' loads in flight at once.
//   3. LayerNorm and residual, one wave per token, two elements per lane.
constexpr int kApplyMaxDh128 = 512;

template <bool BF, int FW, int TT>
__global__ void __launch_bounds__(64 * kApplyWaves) apply128_kernel(ApplyArgs a) {
  using Io = IoT<BF>;
  using E = typename Io::T;
  constexpr int D = 128, NWV = kApplyWaves;
  constexpr int RPI = 2;                                   // W1 rows per wave per load
  constexpr int UB = 8;                                    // W1 loads in flight per lane
  constexpr int NQ = kApplyMaxDh128 / 256;                 // W2 float4 per lane and row
  constexpr int RB = 4;                                    // W2 rows in flight per wave
  __shared__ float qs[TT][D];
  __shared__ float hs[TT][kApplyMaxDh128];
  __shared__ float ys[TT][D];

  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long u = blockIdx.x / a.groups;
  const int t0 = (int)(blockIdx.x % a.groups) * TT;
  const int nt = min(TT, a.T - t0);
  const E* q = static_cast<const E*>(a.q) + (u * a.T + t0) * D;
  E* out = static_cast<E*>(a.out) + (u * a.T + t0) * D;
  const float* w = a.w + u * a.P;
  const int dh = a.dh;
  const float* w2 = w + (long)(FW == 0 ? 1 : 2) * dh * D;   // W2 (MLP) or Wd (SwiGLU)

  for (int x = threadIdx.x; x < TT * D; x += 64 * NWV) {
    const int t = x / D, i = x % D;
    qs[t][i] = (t < nt) ? Io::ld(q + (long)t * D + i) : 0.0f;
  }
  for (int x = threadIdx.x; x < TT * kApplyMaxDh128; x += 64 * NWV) hs[x / kApplyMaxDh128][x % kApplyMaxDh128] = 0.0f;
  __syncthreads();

  // 1. hidden rows
  const int c4 = lane & 31, rsub = lane >> 5;
  f32x4 qv[TT];
#pragma unroll
  for (int t = 0; t < TT; ++t)
    qv[t] = f32x4{qs[t][4 * c4], qs[t][4 * c4 + 1], qs[t][4 * c4 + 2], qs[t][4 * c4 + 3]};
  const int nstep = (dh + NWV * RPI - 1) / (NWV * RPI);
  for (int s0 = 0; s0 < nstep; s0 += UB) {
    f32x4 wr[UB], ur[UB];
#pragma unroll
    for (int k = 0; k < UB; ++k) {
      const int r = ((s0 + k) * NWV + wv) * RPI + rsub;
      wr[k] = zero4();
      ur[k] = zero4();
      if (r < dh) {
        wr[k] = *reinterpret_cast<const f32x4*>(w + (long)r * D + 4 * c4);
        if constexpr (FW == 1)
          ur[k] = *reinterpret_cast<const f32x4*>(w + (long)(dh + r) * D + 4 * c4);
      }
    }
#pragma unroll
    for (int k = 0; k < UB; ++k) {
      const int r0 = ((s0 + k) * NWV + wv) * RPI;
      if (r0 >= dh) break;   // uniform over the wave
      const int r = r0 + rsub;
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        float h = group16_sum(wr[k][0] * qv[t][0] + wr[k][1] * qv[t][1] + wr[k][2] * qv[t][2] +
                              wr[k][3] * qv[t][3]);
        h += __shfl_xor(h, 16);
        if constexpr (FW == 0) {
          if (r < dh && c4 == 0) hs[t][r] = gelu_exact(h);
        } else {
          float up = group16_sum(ur[k][0] * qv[t][0] + ur[k][1] * qv[t][1] +
                                 ur[k][2] * qv[t][2] + ur[k][3] * qv[t][3]);
          up += __shfl_xor(up, 16);
          if (r < dh && c4 == 0) hs[t][r] = silu_exact(h) * up;
        }
      }
    }
  }
  __syncthreads();

  // 2. output rows: y_i = W2[i,:] . a
  f32x4 av[TT][NQ];
#pragma unroll
  for (int t = 0; t < TT; ++t)
#pragma unroll
    for (int h = 0; h < NQ; ++h) {
      const int j = 4 * lane + 256 * h;
      av[t][h] = f32x4{hs[t][j], hs[t][j + 1], hs[t][j + 2], hs[t][j + 3]};
    }
  const bool al16 = (dh & 3) == 0;   // rows of W2 start 16-byte aligned
  for (int k0 = 0; k0 < D / NWV; k0 += RB) {
    f32x4 wr[RB][NQ];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const float* row = w2 + (long)((k0 + b) * NWV + wv) * dh;
#pragma unroll
      for (int h = 0; h < NQ; ++h) {
        const int j = 4 * lane + 256 * h;
        if (al16 && j + 3 < dh) {
          wr[b][h] = *reinterpret_cast<const f32x4*>(row + j);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) wr[b][h][e] = (j + e < dh) ? row[j + e] : 0.0f;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        float p = 0.0f;
#pragma unroll
        for (int h = 0; h < NQ; ++h)
          p += wr[b][h][0] * av[t][h][0] + wr[b][h][1] * av[t][h][1] +
               wr[b][h][2] * av[t][h][2] + wr[b][h][3] * av[t][h][3];
        const float y = wave_sum(p);
        if (lane == 0) ys[t][(k0 + b) * NWV + wv] = y;
      }
  }
  __syncthreads();

  // 3. LayerNorm (biased variance) and residual, one wave per token
  for (int t = wv; t < nt; t += NWV) {
    const float y0 = ys[t][lane], y1 = ys[t][lane + 64];
    float o0 = y0, o1 = y1;
    if (a.resln) {
      const float mean = wave_sum(y0 + y1) * (1.0f / D);
      const float d0 = y0 - mean, d1 = y1 - mean;
      const float var = wave_sum(d0 * d0 + d1 * d1) * (1.0f / D);
      const float inv = 1.0f / sqrtf(var + a.eps);
      float z0 = d0 * inv, z1 = d1 * inv;
      if (a.ln_a) {
        const long ho = (u % a.H) * D;
        z0 = fmaf(a.ln_a[ho + lane], z0, a.ln_b[ho + lane]);
        z1 = fmaf(a.ln_a[ho + lane + 64], z1, a.ln_b[ho + lane + 64]);
      }
      o0 = qs[t][lane] + z0;
      o1 = qs[t][lane + 64] + z1;
    }
    Io::st(out + (long)t * D + lane, o0);
    Io::st(out + (long)t * D + lane + 64, o1);
  }
}

template <int D, bool BF, int FW, int TT>
hipError_t launch(const ApplyArgs& a, hipStream_t s) {
  const long blocks = a.U * a.groups;
  hipLaunchKernelGGL((apply_kernel<D, BF, FW, TT>), dim3((unsigned)blocks),
                     dim3(64 * kApplyWaves), 0, s, a);
  return hipGetLastError();
}

template <bool BF, int FW, int TT>
hipError_t launch128(const ApplyArgs& a, hipStream_t s) {
  const long blocks = a.U * a.groups;
  hipLaunchKernelGGL((apply128_kernel<BF, FW, TT>), dim3((unsigned)blocks),
                     dim3(64 * kApplyWaves), 0, s, a);
  return hipGetLastError();
}

template <int D, bool BF, int FW>
hipError_t launch_tt(ApplyArgs a, hipStream_t s) {
  if constexpr (D == 128) {
    if (a.T == 1) {
      a.groups = 1;
      return launch128<BF, FW, 1>(a, s);
    }
    a.groups = (a.T + 3) / 4;
    return launch128<BF, FW, 4>(a, s);
  } else {
    if (a.T == 1) {
      a.groups = 1;
      return launch<D, BF, FW, 1>(a, s);
    }
    a.groups = (a.T + 7) / 8;
    return launch<D, BF, FW, 8>(a, s);
  }
}

}  // namespace

hipError_t launch_apply(const ChainConfig& cfg, int fw, ApplyArgs a, hipStream_t s) {
  if (a.T < 1 || a.dh > (cfg.d == 128 ? kApplyMaxDh128 : kApplyMaxDh)) return hipErrorInvalidValue;
  if (cfg.bf && cfg.d == 128)
    return fw == 0 ? launch_tt<128, true, 0>(a, s) : launch_tt<128, true, 1>(a, s);
  if (cfg.bf && cfg.d == 64)
    return fw == 0 ? launch_tt<64, true, 0>(a, s) : launch_tt<64, true, 1>(a, s);
  if (!cfg.bf && cfg.d == 16)
    return fw == 0 ? launch_tt<16, false, 0>(a, s) : launch_tt<16, false, 1>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace e2ttt
