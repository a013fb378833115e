// Internal declarations shared by the host API and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace e2ttt {

struct CoeffFwdArgs {
  const float* eta;
  const float* beta;
  const float* gamma;   // nullable (gamma = 1)
  float* kw;            // [U][T]
  float* km;            // [U][T]
  float* carry;         // [U][NC][3]
  int T, C, NC;
  long nwork;           // U * NC
};

struct CoeffBwdArgs {
  const float* eta;
  const float* beta;
  const float* gamma;   // nullable
  const float* kwb;     // [U][T]   adjoint of K^W
  const float* kmb;     // [U][T]   adjoint of K^M
  const float* carryb;  // [U][NC][3] adjoint of the carries
  float* d_eta;
  float* d_beta;
  float* d_gamma;       // nullable iff gamma is
  int T, C, NC;
  long nwork;
};

// Chain kernels: one workgroup per (batch, head) unit, looping over chunks.
struct ChainArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* w_in;    // [U][P]
  const float* m_in;    // [U][P], nullable
  const float* kw;      // [U][T]
  const float* km;      // [U][T]
  const float* carry;   // [U][NC][3]
  // forward
  void* out;            // [U][T][d]
  float* w_out;
  float* m_out;
  // backward
  const void* d_out;
  const float* d_w_out; // nullable
  const float* d_m_out; // nullable
  void* dq;
  void* dk;
  void* dv;
  float* d_w_in;
  float* d_m_in;
  float* kwb;           // [U][T] adjoint of K^W (written by the backward chain)
  float* kmb;
  float* carryb;        // [U][NC][3]
  // chunk-start checkpoints (operand precision, kernel register order),
  // nullable in the forward
  void* ckpt;
  long ckpt_stride;     // bytes per (unit, chunk, W-or-M) block
  int T, C, NC, dh;
  long P;               // parameters per unit (unpadded)
  int resln;            // 1: f = x + LN(y); 0: f = y
  float eps;
};

// Kernel configuration chosen by the host for a descriptor.
struct ChainConfig {
  int fw;     // 0 MLP, 1 SwiGLU
  int d;      // head dim (template)
  int nw;     // waves per workgroup
  int njb;    // 16-wide hidden blocks per wave
  int ntb;    // 16-row token blocks per chunk
  int bf;     // 1: bf16 MFMA operands and io; 0: fp32
};

hipError_t launch_coeff_fwd(const CoeffFwdArgs& a, hipStream_t stream);
hipError_t launch_coeff_bwd(const CoeffBwdArgs& a, hipStream_t stream);
// Return hipErrorInvalidValue when no kernel exists for `cfg`.
hipError_t launch_chain_fwd(const ChainConfig& cfg, const ChainArgs& a, long units,
                            hipStream_t stream);
hipError_t launch_chain_bwd(const ChainConfig& cfg, const ChainArgs& a, long units,
                            hipStream_t stream);
// Bytes of one checkpoint block (W or M of one unit at one chunk start).
long chain_ckpt_bytes(const ChainConfig& cfg);

}  // namespace e2ttt
