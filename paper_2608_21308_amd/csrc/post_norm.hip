// Post-chunk L2 normalisation of the fast weights (App. B.1): the target norm
// of every row, i.e. the norm that row has in the unit's initial weights.
//
// Rows are counted as the chain kernels count them, in packing order: the dh
// rows of each first-layer matrix ([dh][d], a hidden unit's d input weights),
// then the d rows of the second-layer matrix ([d][dh], an output's dh
// weights), R = (nmat - 1) dh + d per unit.  Every row is contiguous in the
// packed parameters, so one wave reads a row with unit stride and reduces it.
#include "e2ttt_device.h"
#include "e2ttt_internal.h"

namespace e2ttt {
namespace {

constexpr int kNormWaves = 4;

__global__ void __launch_bounds__(64 * kNormWaves)
    norm_targets_kernel(const float* __restrict__ w_in, float* __restrict__ tgt, long nrows_all,
                        long R, int d, int dh, int nf, long P) {
  const long row = (long)blockIdx.x * kNormWaves + (threadIdx.x >> 6);
  if (row >= nrows_all) return;   // uniform over the wave
  const int lane = threadIdx.x & 63;
  const long u = row / R, r = row % R;
  const long first = (long)nf * dh;
  const float* src = w_in + u * P + (r < first ? r * d : first * d + (r - first) * dh);
  const int cols = r < first ? d : dh;
  float s = 0.0f;
  for (int c = lane; c < cols; c += 64) s = fmaf(src[c], src[c], s);
  s = wave_sum(s);
  if (lane == 0) tgt[row] = __builtin_sqrtf(s);
}

}  // namespace

hipError_t launch_norm_targets(const float* w_in, float* tgt, long U, int d, int dh, int nmat,
                               long P, hipStream_t stream) {
  const long R = (long)(nmat - 1) * dh + d;
  const long n = U * R;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(norm_targets_kernel, dim3((unsigned)((n + kNormWaves - 1) / kNormWaves)),
                     dim3(64 * kNormWaves), 0, stream, w_in, tgt, n, R, d, dh, nmat - 1, P);
  return hipGetLastError();
}

}  // namespace e2ttt
