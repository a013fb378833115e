// Scalar kernels of the E2-TTT chunk transition and their backward.
//
// Forward (Prop. 1, eq. (9)-(11)), per chunk of length L with 1-based token t:
//   b~_t = prod_{i>t} beta_i,  g~_t = prod_{i>t} gamma_i   (suffix products)
//   S_t  = b~_t R_t = sum_{i>=t} (prod_{t<j<=i} beta_j) g~_i
//        satisfies S_L = 1, S_t = g~_t + beta_{t+1} S_{t+1}
//   K^W_t = eta_t S_t,  K^M_t = eta_t b~_t
//   carry = (g~_0, b~_0 R_1 = beta_1 S_1, b~_0)
// The paper evaluates the suffix products in log space and forms R_t as a sum
// of ratios g~_i / b~_i; here the products are formed by a multiplicative
// wave scan (every factor lies in (0, 1], so nothing overflows, and underflow
// to zero is the exact limit) and S_t by an affine wave scan, which never
// divides and stays finite for beta -> 0 where the ratio form is 0/0.
//
// Chunk-averaged rule (the ablation baseline, eqs. (4)-(5) with mean factors):
//   K^W_t = K^M_t = eta_t,  carry = (mean gamma, mean beta, mean beta),
// with the backward  d eta_t = dK^W_t + dK^M_t,  d beta_t = (dcm + dcb) / L,
// d gamma_t = dcw / L.
//
// One wave64 handles one (unit, chunk); lane tau holds token t = tau + 1.
#include <hip/hip_runtime.h>

#include "e2ttt_internal.h"

namespace e2ttt {

namespace {

struct ChunkScalars {
  float e, b, gm;      // this lane's eta, beta, gamma (padding: 0, 1, 1)
  float pb, pg;        // inclusive suffix products of beta, gamma
  float bt, gt;        // exclusive suffix products (b~_t, g~_t)
  float S;             // S_t
};

__device__ __forceinline__ ChunkScalars chunk_scalars(const float* eta, const float* beta,
                                                      const float* gamma, long base, int len,
                                                      int lane) {
  ChunkScalars s;
  const bool valid = lane < len;
  s.e = valid ? eta[base + lane] : 0.0f;
  s.b = valid ? beta[base + lane] : 1.0f;
  s.gm = (valid && gamma) ? gamma[base + lane] : 1.0f;
  float pb = s.b, pg = s.gm;
#pragma unroll
  for (int k = 1; k < 64; k <<= 1) {
    float ob = __shfl_down(pb, k, 64);
    float og = __shfl_down(pg, k, 64);
    if (lane + k < 64) { pb *= ob; pg *= og; }
  }
  s.pb = pb;
  s.pg = pg;
  float bt = __shfl_down(pb, 1, 64), gt = __shfl_down(pg, 1, 64);
  if (lane == 63) { bt = 1.0f; gt = 1.0f; }
  s.bt = bt;
  s.gt = gt;
  // reverse affine scan S_t = A_t + B_t S_{t+1}
  const float bnext = __shfl_down(s.b, 1, 64);
  float A, B;
  if (lane < len - 1) { A = gt; B = bnext; }
  else if (lane == len - 1) { A = 1.0f; B = 0.0f; }
  else { A = 0.0f; B = 0.0f; }
#pragma unroll
  for (int k = 1; k < 64; k <<= 1) {
    float oA = __shfl_down(A, k, 64);
    float oB = __shfl_down(B, k, 64);
    if (lane + k < 64) { A = A + B * oA; B = B * oB; }
  }
  s.S = A;
  return s;
}

// Ascending affine scan x_tau = a_tau + b_tau x_{tau-1} (b_0 is ignored).
__device__ __forceinline__ float affine_scan_up(float a, float b, int lane) {
  if (lane == 0) b = 0.0f;
#pragma unroll
  for (int k = 1; k < 64; k <<= 1) {
    float oa = __shfl_up(a, k, 64);
    float ob = __shfl_up(b, k, 64);
    if (lane >= k) { a = a + b * oa; b = b * ob; }
  }
  return a;
}

// Sum over the wave (butterfly, the same order on every lane).
__device__ __forceinline__ float wave_total(float v) {
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) v += __shfl_xor(v, k, 64);
  return v;
}

// Chunks longer than a wave (C up to 512): the wave walks the chunk's 64-token
// segments from the last to the first, carrying the products of the later
// segments' factors (for the suffix products) and S at the next segment's
// first token (for the affine recursion S_t = g~_t + beta_{t+1} S_{t+1}).
constexpr int kMaxSeg = 8;   // 512 / 64

struct LongScalars {
  float S[kMaxSeg], bt[kMaxSeg], gt[kMaxSeg];   // per segment, this lane's token
  float carry[3];                                // (g~_0, beta_1 S_1, b~_0)
};

// One lane's token of every segment of a long chunk (eta, beta, gamma, with
// the neutral values 0, 1, 1 past the chunk's end).  Every load goes out at
// once, from an index clamped to the chunk's first token so that it stays in
// bounds; the segment walks below then run on registers (loads issued segment
// by segment would each wait a full memory round trip).
struct LongInputs {
  float e[kMaxSeg], b[kMaxSeg], g[kMaxSeg];
};
__device__ __forceinline__ void long_inputs(const float* eta, const float* beta,
                                            const float* gamma, long base, int len, int lane,
                                            LongInputs& x) {
#pragma unroll
  for (int seg = 0; seg < kMaxSeg; ++seg) {
    const bool valid = seg * 64 + lane < len;
    const long i = valid ? base + seg * 64 + lane : base;
    const float e = eta[i], b = beta[i], g = gamma ? gamma[i] : 1.0f;
    x.e[seg] = valid ? e : 0.0f;
    x.b[seg] = valid ? b : 1.0f;
    x.g[seg] = valid ? g : 1.0f;
  }
}

__device__ __forceinline__ void long_scalars(const LongInputs& x, int len, int lane,
                                             LongScalars& o) {
  float cb = 1.0f, cg = 1.0f;           // products of beta, gamma over the later segments
  float s_next = 0.0f, b_next = 1.0f;   // S and beta at the next segment's first token
  const int nseg = (len + 63) / 64;
#pragma unroll
  for (int seg = kMaxSeg - 1; seg >= 0; --seg) {
    if (seg >= nseg) continue;          // uniform
    const int n = min(64, len - seg * 64);
    const float b = x.b[seg];
    const float gm = x.g[seg];
    float pb = b, pg = gm;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
      const float ob = __shfl_down(pb, k, 64), og = __shfl_down(pg, k, 64);
      if (lane + k < 64) { pb *= ob; pg *= og; }
    }
    float bt = __shfl_down(pb, 1, 64), gt = __shfl_down(pg, 1, 64);
    if (lane == 63) { bt = 1.0f; gt = 1.0f; }
    bt *= cb;                            // exclusive suffix products over the whole chunk
    gt *= cg;
    const float bnext = __shfl_down(b, 1, 64);
    float A, B;
    if (lane < n - 1) { A = gt; B = bnext; }
    else if (lane == n - 1) {
      if (seg == nseg - 1) { A = 1.0f; B = 0.0f; }
      else { A = gt + b_next * s_next; B = 0.0f; }
    } else { A = 0.0f; B = 0.0f; }
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
      const float oA = __shfl_down(A, k, 64), oB = __shfl_down(B, k, 64);
      if (lane + k < 64) { A = A + B * oA; B = B * oB; }
    }
    o.S[seg] = A;
    o.bt[seg] = bt;
    o.gt[seg] = gt;
    s_next = __shfl(A, 0, 64);
    b_next = __shfl(b, 0, 64);
    cb *= __shfl(pb, 0, 64);
    cg *= __shfl(pg, 0, 64);
  }
  o.carry[0] = cg;
  o.carry[1] = b_next * s_next;
  o.carry[2] = cb;
}

__device__ void coeff_fwd_long(const CoeffFwdArgs& a, long wid, long base, int len, int lane) {
  LongInputs x;
  long_inputs(a.eta, a.beta, a.gamma, base, len, lane, x);
  LongScalars o;
  long_scalars(x, len, lane, o);
  const int nseg = (len + 63) / 64;
#pragma unroll
  for (int seg = 0; seg < kMaxSeg; ++seg) {
    if (seg >= nseg) break;
    const long sb = base + seg * 64;
    if (lane < min(64, len - seg * 64)) {
      const float e = x.e[seg];
      a.kw[sb + lane] = e * o.S[seg];
      a.km[sb + lane] = e * o.bt[seg];
    }
  }
  if (lane == 0) {
    a.carry[wid * 3 + 0] = o.carry[0];
    a.carry[wid * 3 + 1] = o.carry[1];
    a.carry[wid * 3 + 2] = o.carry[2];
  }
}

__global__ void __launch_bounds__(256) coeff_fwd_kernel(CoeffFwdArgs a) {
  // the chain kernel that follows on this stream starts from cleared sync words
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < a.nzero; i += (long)gridDim.x * 256)
    a.zero[i] = 0u;
  const long wid = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= a.nwork) return;
  const int lane = threadIdx.x & 63;
  const long u = wid / a.NC;
  const int r = (int)(wid % a.NC);
  const int s0 = r * a.C;
  const int len = min(a.C, a.T - s0);
  const long base = u * a.T + s0;
  if (a.averaged) {
    float bpart = 0.0f, gpart = 0.0f;
    for (int t0 = 0; t0 < len; t0 += 64) {
      const bool valid = t0 + lane < len;
      const float e = valid ? a.eta[base + t0 + lane] : 0.0f;
      bpart += valid ? a.beta[base + t0 + lane] : 0.0f;
      gpart += valid ? (a.gamma ? a.gamma[base + t0 + lane] : 1.0f) : 0.0f;
      if (valid) {
        a.kw[base + t0 + lane] = e;
        a.km[base + t0 + lane] = e;
      }
    }
    const float bsum = wave_total(bpart), gsum = wave_total(gpart);
    const float inv = 1.0f / (float)len;
    if (lane == 0) {
      a.carry[wid * 3 + 0] = gsum * inv;
      a.carry[wid * 3 + 1] = bsum * inv;
      a.carry[wid * 3 + 2] = bsum * inv;
    }
    return;
  }
  if (len > 64) {
    coeff_fwd_long(a, wid, base, len, lane);
    return;
  }
  ChunkScalars s = chunk_scalars(a.eta, a.beta, a.gamma, base, len, lane);
  if (lane < len) {
    a.kw[base + lane] = s.e * s.S;
    a.km[base + lane] = s.e * s.bt;
  }
  if (lane == 0) {
    a.carry[wid * 3 + 0] = s.pg;
    a.carry[wid * 3 + 1] = s.b * s.S;
    a.carry[wid * 3 + 2] = s.pb;
  }
}

// Backward of the map (eta, beta, gamma) -> (K^W, K^M, carry) given the
// adjoints kwb, kmb (per token) and carryb (per chunk).  Reverse mode through
// the same scans:  S-bar accumulates through an ascending affine scan, and the
// suffix-product adjoints are pushed to the factors with ascending affine
// scans as well (no division by beta or gamma).
// Backward of a long chunk: the same adjoint recursions as the single-wave
// kernel below, walked over the chunk's segments from the first to the last
// (every scan is ascending); each segment's scans start from the previous
// segment's last values (S-hat, Y, Z, and the previous token's beta, gamma and
// K^M eta), which enter lane 0 as x_0 = a_0 + b_0 x_{-1}.
// Token t's adjoints of K^W and K^M summed over the ns workgroup slots, in
// slot order from slot 0.  The slot loop runs to the largest ns with every
// load issued (slot index clamped to ns - 1, in bounds) and the surplus
// slots added as zeros, so the loads go out together instead of one slot
// per memory round trip.
constexpr int kMaxSlots = 8;
__device__ __forceinline__ void sum_slots(const CoeffBwdArgs& a, long t, bool valid, float& kw,
                                          float& km) {
  float w[kMaxSlots], m[kMaxSlots];
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    const long o = (long)min(sl, a.ns - 1) * a.tok_slot + t;
    w[sl] = a.kwb[o];
    m[sl] = a.kmb[o];
  }
  kw = 0.0f;
  km = 0.0f;
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    if (valid && sl < a.ns) {
      kw += w[sl];
      km += m[sl];
    }
  }
}

__device__ void coeff_bwd_long(const CoeffBwdArgs& a, long wid, long base, int len, int lane,
                               float cwb, float cmb, float cbb) {
  LongInputs x;
  long_inputs(a.eta, a.beta, a.gamma, base, len, lane, x);
  // the token adjoints of every segment, summed over the workgroup slots
  float kwv[kMaxSeg], kmv[kMaxSeg];
#pragma unroll
  for (int seg = 0; seg < kMaxSeg; ++seg) {
    const bool valid = seg * 64 + lane < len;
    sum_slots(a, valid ? base + seg * 64 + lane : base, valid, kwv[seg], kmv[seg]);
  }
  LongScalars o;
  long_scalars(x, len, lane, o);
  const int nseg = (len + 63) / 64;
  float sh_last = 0.0f, kme_last = 0.0f, b_last = 1.0f, g_last = 1.0f, y_last = 0.0f,
        z_last = 0.0f;
#pragma unroll
  for (int seg = 0; seg < kMaxSeg; ++seg) {
    if (seg >= nseg) break;
    const long sb = base + seg * 64;
    const int n = min(64, len - seg * 64);
    const bool valid = lane < n;
    const float e = x.e[seg];
    const float b = x.b[seg];
    const float gm = x.g[seg];
    const float kwb = kwv[seg], kmb = kmv[seg];
    const float S = o.S[seg], bt = o.bt[seg], gt = o.gt[seg];
    const bool t0 = seg == 0 && lane == 0;            // the chunk's first token
    const float etab = kwb * S + kmb * bt;
    float Sb = kwb * e;
    float betab = 0.0f;
    if (t0) { Sb += cmb * b; betab = cmb * S; }
    if (seg > 0 && lane == 0) Sb += b * sh_last;
    const float Sh = affine_scan_up(Sb, b, lane);
    float Sh_prev = __shfl_up(Sh, 1, 64);
    float kme_prev = __shfl_up(kmb * e, 1, 64);
    float b_prev = __shfl_up(b, 1, 64);
    float g_prev = __shfl_up(gm, 1, 64);
    if (lane == 0) { Sh_prev = sh_last; kme_prev = kme_last; b_prev = b_last; g_prev = g_last; }
    if (!t0) betab += Sh_prev * S;
    float btb = t0 ? cbb : kme_prev;
    float gtb = t0 ? cwb : Sh_prev;
    if (seg > 0 && lane == 0) { btb += b_prev * y_last; gtb += g_prev * z_last; }
    const float Y = affine_scan_up(btb, b_prev, lane);
    const float Z = affine_scan_up(gtb, g_prev, lane);
    betab += bt * Y;
    if (valid) {
      a.d_eta[sb + lane] = etab;
      a.d_beta[sb + lane] = betab;
      if (a.d_gamma) a.d_gamma[sb + lane] = gt * Z;
    }
    sh_last = __shfl(Sh, 63, 64);
    kme_last = __shfl(kmb * e, 63, 64);
    b_last = __shfl(b, 63, 64);
    g_last = __shfl(gm, 63, 64);
    y_last = __shfl(Y, 63, 64);
    z_last = __shfl(Z, 63, 64);
  }
}

// LONGC: chunks longer than one wave's 64 tokens (a separate instantiation,
// so that the short-chunk kernel keeps its small register footprint).
template <bool LONGC>
__global__ void __launch_bounds__(256) coeff_bwd_kernel(CoeffBwdArgs a) {
  const long wid = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= a.nwork) return;
  const int lane = threadIdx.x & 63;
  const long u = wid / a.NC;
  const int r = (int)(wid % a.NC);
  const int s0 = r * a.C;
  const int len = min(a.C, a.T - s0);
  const long base = u * a.T + s0;
  const bool valid = lane < len;
  // the chain kernel leaves one partial per workgroup of a unit; sum them
  float kwb, kmb, cwb = 0.0f, cmb = 0.0f, cbb = 0.0f;
  sum_slots(a, valid ? base + lane : base, valid, kwb, kmb);
  float cv[kMaxSlots][3];
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    const long o = (long)min(sl, a.ns - 1) * a.chk_slot + wid * 3;
    cv[sl][0] = a.carryb[o];
    cv[sl][1] = a.carryb[o + 1];
    cv[sl][2] = a.carryb[o + 2];
  }
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    if (sl < a.ns) {
      cwb += cv[sl][0];
      cmb += cv[sl][1];
      cbb += cv[sl][2];
    }
  }
  if (a.averaged) {
    const float inv = 1.0f / (float)len;
    for (int t0 = 0; t0 < len; t0 += 64) {
      const int t = t0 + lane;
      if (t >= len) continue;
      float kw2 = 0.0f, km2 = 0.0f;
      for (int sl = 0; sl < a.ns; ++sl) {
        kw2 += a.kwb[sl * a.tok_slot + base + t];
        km2 += a.kmb[sl * a.tok_slot + base + t];
      }
      a.d_eta[base + t] = kw2 + km2;
      a.d_beta[base + t] = (cmb + cbb) * inv;
      if (a.d_gamma) a.d_gamma[base + t] = cwb * inv;
    }
    return;
  }
  if (LONGC && len > 64) {
    coeff_bwd_long(a, wid, base, len, lane, cwb, cmb, cbb);
    return;
  }
  ChunkScalars s = chunk_scalars(a.eta, a.beta, a.gamma, base, len, lane);

  const float etab = kwb * s.S + kmb * s.bt;
  // S-bar and the direct beta_1 term of carry_m = beta_1 S_1
  float Sb = kwb * s.e;
  float betab = 0.0f;
  if (lane == 0) { Sb += cmb * s.b; betab = cmb * s.S; }
  // S^_tau = Sb_tau + beta_tau S^_{tau-1}
  const float Sh = affine_scan_up(Sb, s.b, lane);
  const float Sh_prev = __shfl_up(Sh, 1, 64);
  if (lane >= 1) betab += Sh_prev * s.S;           // S_{t-1} = g~_{t-1} + beta_t S_t
  // adjoints of the exclusive suffix products b~_{tau}, g~_{tau} (tau = 0..len-1)
  const float kme_prev = __shfl_up(kmb * s.e, 1, 64);
  const float btb = (lane == 0) ? cbb : kme_prev;
  const float gtb = (lane == 0) ? cwb : Sh_prev;
  const float b_prev = __shfl_up(s.b, 1, 64);
  const float g_prev = __shfl_up(s.gm, 1, 64);
  const float Y = affine_scan_up(btb, b_prev, lane);
  const float Z = affine_scan_up(gtb, g_prev, lane);
  betab += s.bt * Y;
  const float gammab = s.gt * Z;
  if (valid) {
    a.d_eta[base + lane] = etab;
    a.d_beta[base + lane] = betab;
    if (a.d_gamma) a.d_gamma[base + lane] = gammab;
  }
}

__global__ void __launch_bounds__(256) zero_words_kernel(unsigned* p, long n) {
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) p[i] = 0u;
}

}  // namespace

hipError_t launch_zero_words(unsigned* p, long n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)min(64L, (n + 255) / 256);
  hipLaunchKernelGGL(zero_words_kernel, dim3(blocks), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

hipError_t launch_coeff_fwd(const CoeffFwdArgs& a, hipStream_t stream) {
  const unsigned blocks = (unsigned)((a.nwork + 3) / 4);
  hipLaunchKernelGGL(coeff_fwd_kernel, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_coeff_bwd(const CoeffBwdArgs& a, hipStream_t stream) {
  if (a.ns < 1 || a.ns > kMaxSlots) return hipErrorInvalidValue;
  const unsigned blocks = (unsigned)((a.nwork + 3) / 4);
  if (a.C > 64)
    hipLaunchKernelGGL(coeff_bwd_kernel<true>, dim3(blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(coeff_bwd_kernel<false>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace e2ttt
