// Gate parameterization of Sec. 4 (eqs. (12)-(14)) and its backward: an
// elementwise map over the tokens, bound by HBM traffic (the forward reads
// three logits and writes three gates per token, the backward reads six
// values and writes three).
#include <math.h>

#include "e2ttt.h"
#include "e2ttt_internal.h"

namespace e2ttt {
namespace {

// sigmoid(x) and sigmoid(-x) = 1 - sigmoid(x), each without cancellation.
struct Sig {
  float s, sm;
};
__device__ __forceinline__ Sig sigmoid2(float x) {
  const float e = expf(-fabsf(x));      // in (0, 1]
  const float r = 1.0f / (1.0f + e);
  Sig o;
  o.s = (x >= 0.0f) ? r : e * r;
  o.sm = (x >= 0.0f) ? e * r : r;
  return o;
}
// log sigmoid(x) = min(x, 0) - log1p(exp(-|x|))
__device__ __forceinline__ float log_sigmoid(float x) {
  return fminf(x, 0.0f) - log1pf(expf(-fabsf(x)));
}

struct GateArgs {
  float eta_base, alpha_base, inv_tau;
  long n;
  const float* l_eta;
  const float* l_beta;
  const float* l_alpha;   // nullable
  float* eta;
  float* beta;
  float* gamma;           // nullable iff l_alpha is
  const float* d_eta;
  const float* d_beta;
  const float* d_gamma;   // nullable iff l_alpha is
  float* d_l_eta;
  float* d_l_beta;
  float* d_l_alpha;       // nullable iff l_alpha is
};

__global__ void __launch_bounds__(256) gates_fwd_kernel(GateArgs a) {
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += stride) {
    const float eta = a.eta_base * sigmoid2(a.l_eta[i]).s;
    a.eta[i] = eta;
    a.beta[i] = expf(log_sigmoid(a.l_beta[i]) * a.inv_tau);
    if (a.l_alpha) a.gamma[i] = 1.0f - eta * (a.alpha_base * sigmoid2(a.l_alpha[i]).s);
  }
}

// eta = eb s_e, beta = exp(log s_b / tau), alpha = ab s_a, gamma = 1 - eta alpha:
//   d l_eta   = (d_eta - alpha d_gamma) eb s_e (1 - s_e)
//   d l_alpha = -eta d_gamma ab s_a (1 - s_a)
//   d l_beta  = d_beta beta (1 - s_b) / tau
__global__ void __launch_bounds__(256) gates_bwd_kernel(GateArgs a) {
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += stride) {
    const Sig se = sigmoid2(a.l_eta[i]);
    const float eta = a.eta_base * se.s;
    float deta = a.d_eta[i];
    if (a.l_alpha) {
      const Sig sa = sigmoid2(a.l_alpha[i]);
      const float alpha = a.alpha_base * sa.s, dg = a.d_gamma[i];
      deta -= alpha * dg;
      a.d_l_alpha[i] = -eta * dg * a.alpha_base * sa.s * sa.sm;
    }
    a.d_l_eta[i] = deta * a.eta_base * se.s * se.sm;
    const Sig sb = sigmoid2(a.l_beta[i]);
    const float beta = expf(log_sigmoid(a.l_beta[i]) * a.inv_tau);
    a.d_l_beta[i] = a.d_beta[i] * beta * sb.sm * a.inv_tau;
  }
}

bool params_ok(const e2ttt_gate_params* p) {
  return isfinite(p->eta_base) && isfinite(p->alpha_base) && isfinite(p->tau) &&
         p->eta_base >= 0.0f && p->alpha_base >= 0.0f && p->tau > 0.0f;
}

int grid_for(long n) {
  const long blocks = (n + 255) / 256;
  return (int)(blocks < 2048 ? (blocks > 0 ? blocks : 1) : 2048);
}

}  // namespace
}  // namespace e2ttt

using namespace e2ttt;

extern "C" e2ttt_status e2ttt_gates_forward(const e2ttt_gate_params* params, int64_t n,
                                            const float* l_eta, const float* l_beta,
                                            const float* l_alpha, float* eta, float* beta,
                                            float* gamma, void* stream) {
  if (!params) return E2TTT_ERR_NULL_ARG;
  if (n < 0 || !params_ok(params)) return E2TTT_ERR_BAD_SHAPE;
  if (n == 0) return E2TTT_OK;
  if (!l_eta || !l_beta || !eta || !beta) return E2TTT_ERR_NULL_ARG;
  if ((l_alpha == nullptr) != (gamma == nullptr)) return E2TTT_ERR_NULL_ARG;
  GateArgs a{};
  a.eta_base = params->eta_base;
  a.alpha_base = params->alpha_base;
  a.inv_tau = 1.0f / params->tau;
  a.n = n;
  a.l_eta = l_eta; a.l_beta = l_beta; a.l_alpha = l_alpha;
  a.eta = eta; a.beta = beta; a.gamma = gamma;
  hipLaunchKernelGGL(gates_fwd_kernel, dim3(grid_for(n)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? E2TTT_OK : E2TTT_ERR_HIP;
}

extern "C" e2ttt_status e2ttt_gates_backward(const e2ttt_gate_params* params, int64_t n,
                                             const float* l_eta, const float* l_beta,
                                             const float* l_alpha, const float* d_eta,
                                             const float* d_beta, const float* d_gamma,
                                             float* d_l_eta, float* d_l_beta, float* d_l_alpha,
                                             void* stream) {
  if (!params) return E2TTT_ERR_NULL_ARG;
  if (n < 0 || !params_ok(params)) return E2TTT_ERR_BAD_SHAPE;
  if (n == 0) return E2TTT_OK;
  if (!l_eta || !l_beta || !d_eta || !d_beta || !d_l_eta || !d_l_beta) return E2TTT_ERR_NULL_ARG;
  const bool ga = l_alpha != nullptr;
  if (ga != (d_gamma != nullptr) || ga != (d_l_alpha != nullptr)) return E2TTT_ERR_NULL_ARG;
  GateArgs a{};
  a.eta_base = params->eta_base;
  a.alpha_base = params->alpha_base;
  a.inv_tau = 1.0f / params->tau;
  a.n = n;
  a.l_eta = l_eta; a.l_beta = l_beta; a.l_alpha = l_alpha;
  a.d_eta = d_eta; a.d_beta = d_beta; a.d_gamma = d_gamma;
  a.d_l_eta = d_l_eta; a.d_l_beta = d_l_beta; a.d_l_alpha = d_l_alpha;
  hipLaunchKernelGGL(gates_bwd_kernel, dim3(grid_for(n)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? E2TTT_OK : E2TTT_ERR_HIP;
}
