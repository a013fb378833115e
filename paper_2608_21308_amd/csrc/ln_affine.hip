// Gradients of the learnable LayerNorm affine (f = x + a LN(y) + b, a and b
// per head) after the backward chain.  Per head h and column i, summed over
// the batch and every token t:
//   d_a = sum  dO_t z_q,t  +  zbar_t (e_t - a z_k,t)
//   d_b = sum  dO_t  -  a zbar_t,          e_t = v_t - k_t - a z_k,t - b,
// the first terms from the outputs o = q + a z_q + b, the second from the
// inner-loss gradients through e = v - f(k) (zbar is the adjoint of a e that
// the backward chain wrote for every token row; z_k, z_q are the LayerNorm
// outputs the forward saved).
//
// Two passes, both in a fixed order so that results are reproducible: one
// workgroup per (unit, block of kAffineTokBlock tokens) sums its block into a
// partial; then one thread per (head, column) adds the partials of that head's
// units over the batch and the token blocks.  Bound by streaming the six
// [U][T][d] tensors once.
#include "e2ttt_device.h"
#include "e2ttt_internal.h"

namespace e2ttt {
namespace {

constexpr int kAffineThreads = 256;

template <bool BF>
__global__ void __launch_bounds__(kAffineThreads) affine_part_kernel(AffineGradArgs a) {
  using Io = IoT<BF>;
  using E = typename Io::T;
  const int d = a.d;
  const int nb = (a.T + kAffineTokBlock - 1) / kAffineTokBlock;
  const long u = blockIdx.x / nb;
  const int tb = (int)(blockIdx.x % nb);
  const int h = (int)(u % a.H);
  const int rows = kAffineThreads / d;              // token rows handled per pass
  const int i = threadIdx.x % d, r0 = threadIdx.x / d;
  const float la = a.ln_a[h * d + i], lb = a.ln_b[h * d + i];
  const int t_lo = tb * kAffineTokBlock, t_hi = min(a.T, t_lo + kAffineTokBlock);
  float ga = 0.0f, gb = 0.0f;
  for (int t = t_lo + r0; t < t_hi; t += rows) {
    const long e = (u * a.T + t) * d + i;
    const float dO = Io::ld(static_cast<const E*>(a.d_out) + e);
    const float zq = ld_stream(a.zq + e), zk = ld_stream(a.zk + e), zb = ld_stream(a.zbar + e);
    const float ev = Io::ld(static_cast<const E*>(a.v) + e) - Io::ld(static_cast<const E*>(a.k) + e) -
                     fmaf(la, zk, lb);
    ga += dO * zq + zb * (ev - la * zk);
    gb += dO - la * zb;
  }
  // sum the rows that share a column, in row order
  __shared__ float sa[kAffineThreads], sb[kAffineThreads];
  sa[threadIdx.x] = ga;
  sb[threadIdx.x] = gb;
  __syncthreads();
  if (threadIdx.x < d) {
    float xa = 0.0f, xb = 0.0f;
    for (int r = 0; r < rows; ++r) {
      xa += sa[r * d + threadIdx.x];
      xb += sb[r * d + threadIdx.x];
    }
    float* p = a.part + ((u * nb + tb) * 2) * d;
    p[threadIdx.x] = xa;
    p[d + threadIdx.x] = xb;
  }
}

__global__ void __launch_bounds__(kAffineThreads) affine_sum_kernel(AffineGradArgs a) {
  const int d = a.d;
  const int nb = (a.T + kAffineTokBlock - 1) / kAffineTokBlock;
  const long x = (long)blockIdx.x * kAffineThreads + threadIdx.x;   // (head, which, column)
  if (x >= (long)a.H * 2 * d) return;
  const int h = (int)(x / (2 * d)), which = (int)((x / d) % 2), i = (int)(x % d);
  const long B = a.U / a.H;
  float s = 0.0f;
  for (long b = 0; b < B; ++b) {
    const long u = b * a.H + h;
    for (int tb = 0; tb < nb; ++tb) s += a.part[((u * nb + tb) * 2 + which) * d + i];
  }
  (which == 0 ? a.d_ln_a : a.d_ln_b)[h * d + i] = s;
}

}  // namespace

hipError_t launch_affine_grad(const AffineGradArgs& a, hipStream_t stream) {
  if (a.d < 1 || kAffineThreads % a.d != 0) return hipErrorInvalidValue;
  const long nb = (a.T + kAffineTokBlock - 1) / kAffineTokBlock;
  const long blocks = a.U * nb;
  if (a.bf)
    hipLaunchKernelGGL(affine_part_kernel<true>, dim3((unsigned)blocks), dim3(kAffineThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL(affine_part_kernel<false>, dim3((unsigned)blocks), dim3(kAffineThreads), 0,
                       stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long n = (long)a.H * 2 * a.d;
  hipLaunchKernelGGL(affine_sum_kernel, dim3((unsigned)((n + kAffineThreads - 1) / kAffineThreads)),
                     dim3(kAffineThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace e2ttt
