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
  unsigned* zero;       // nullable: words cleared by this kernel (pair sync words)
  long nzero;
  int averaged;         // 1: chunk-averaged rule (K^W = K^M = eta, mean beta / gamma carries)
};

struct CoeffBwdArgs {
  const float* eta;
  const float* beta;
  const float* gamma;   // nullable
  const float* kwb;     // [ns][U][T]   adjoint of K^W (summed over the slots)
  const float* kmb;     // [ns][U][T]   adjoint of K^M
  const float* carryb;  // [ns][U][NC][3] adjoint of the carries
  float* d_eta;
  float* d_beta;
  float* d_gamma;       // nullable iff gamma is
  int T, C, NC;
  long nwork;
  int ns;               // partial slots of kwb, kmb, carryb (one per workgroup of a unit)
  long tok_slot;        // elements between slots of kwb / kmb (U T)
  long chk_slot;        // elements between slots of carryb (U NC 3)
  int averaged;         // as CoeffFwdArgs::averaged
};

// Chain kernels: one or two workgroups per (batch, head) unit, looping over chunks.
struct ChainArgs {
  long U;               // units
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
  float* kwb;           // [NS][U][T] adjoint of K^W, one partial per rank
  float* kmb;
  float* carryb;        // [NS][U][NC][3]
  // chunk-start checkpoints (operand precision, kernel register order),
  // nullable in the forward
  void* ckpt;
  long ckpt_stride;     // bytes per (unit, chunk, rank, W-or-M) block
  // query-side activations A_Q and GELU'(H_Q) of every chunk (GELU MLP), saved
  // by the forward for the backward's output branch (nullable in the forward;
  // layout: SavedAct in chain_common.h)
  void* asave;
  long as_stride;       // bytes per (unit, chunk tile, rank) block
  // backward of chunks longer than one tile: per workgroup, the MFMA operand
  // copies of the adjoint state at the chunk end (that of W, then that of M,
  // in the operand type and the register-tile order of the state), kept by
  // the chunk's first processed tile for its other tiles; room for two blocks
  // of chain_frz_floats(cfg) floats (the fp32 path fills both, bf16 half)
  float* bfrz;
  // forward of chunks longer than one tile with operands re-formed from the
  // state (SwiGLU on bf16): per workgroup, the chunk-start weights W_0 (fp32,
  // register-tile order), chain_frz_floats(cfg) floats each
  float* w0blk;
  // LN outputs saved by the forward for the backward (nullable in the forward):
  // Z = LN(Y) (Y itself without the residual LN) [U][T][d], 1/sigma [U][T]
  float* zk;
  float* rk;
  float* zq;
  float* rq;
  // two workgroups per unit: exchange slots and sync words (pair_xchg.h)
  float* xbuf;
  unsigned* sync;
  long npairs;
  long long wait_ticks;  // limit of every bounded wait between ranks (100 MHz counter ticks)
  int T, C, NC, dh;
  long P;               // parameters per unit (unpadded)
  int resln;            // 1: f = x + LN(y); 0: f = y
  float eps;
  // learnable LayerNorm affine, f = x + a LN(y) + b, per head [H][d] fp32
  // (nullable together: no affine); unit u belongs to head u mod H
  const float* ln_a;
  const float* ln_b;
  int H;
  // backward with the affine: the adjoint of a * e for every token row
  // [U][T][d] fp32, rows [rank share] written by each rank
  float* ln_zbar;
  // post-chunk L2 normalisation of the fast-weight rows (nullable: off).
  // Rows in packing order: the first-layer matrices' dh rows each, then the
  // second layer's d rows, R = (NMAT - 1) dh + d per unit.
  const float* norm_tgt;  // [U][R] target norms (the rows of w_in)
  float* norm_pre;        // [U][NC][R] norms before the normalisation (forward, saving)
  float* norm_rbar;       // [U][NS][R] backward: what flows into the targets, per rank
  float* nxbuf;           // [groups][NS][2][d] second-layer row sums of each rank
  long ckpt_nc;           // checkpoint blocks per unit: NC, or NC + 1 (the final state)
};
// Post-chunk normalisation: the target norms of every unit's rows from w_in.
hipError_t launch_norm_targets(const float* w_in, float* tgt, long U, int d, int dh, int nmat,
                               long P, hipStream_t stream);

// The affine's gradients from the saved and written rows (ln_affine.hip):
// per head h and column i, over the batch and all tokens,
//   d_a = sum dO z_q + zbar (e - a z_k),  d_b = sum dO - a zbar,
//   e = v - k - a z_k - b.
struct AffineGradArgs {
  const void* d_out;    // [U][T][d] io
  const void* k;
  const void* v;
  const float* zk;      // [U][T][d] fp32 (saved by the forward)
  const float* zq;
  const float* zbar;    // [U][T][d] fp32 (written by the backward chain)
  const float* ln_a;    // [H][d]
  const float* ln_b;
  float* part;          // [U][NB][2][d] partial sums per token block
  float* d_ln_a;        // [H][d]
  float* d_ln_b;
  long U;
  int H, T, d, bf;
};
constexpr int kAffineTokBlock = 256;
hipError_t launch_affine_grad(const AffineGradArgs& a, hipStream_t stream);

// Kernel configuration chosen by the host for a descriptor.
struct ChainConfig {
  int fw;     // 0 MLP, 1 SwiGLU
  int d;      // head dim (template)
  int nw;     // waves per workgroup
  int njb;    // 16-wide hidden blocks per wave
  int ntb;    // 16-row token blocks per chunk
  int bf;     // 1: bf16 MFMA operands and io; 0: fp32
  int ns;     // workgroups per unit (1, or 2 with a cooperative launch)
  int pn;     // 1: with the post-chunk normalisation of the fast weights
};

// Net evaluation at a given state (e2ttt_apply): per unit, T tokens of q at
// one state w of P floats.
struct ApplyArgs {
  const void* q;        // [U][T][d] io
  const float* w;       // [U][P]
  void* out;            // [U][T][d] io
  long U;
  int T, dh;
  int groups;           // token groups per unit (set by the launcher)
  long P;
  int resln;
  float eps;
  const float* ln_a;    // LayerNorm affine per head [H][d], nullable together
  const float* ln_b;
  int H;
};
constexpr int kApplyMaxDh = 256;

hipError_t launch_coeff_fwd(const CoeffFwdArgs& a, hipStream_t stream);
hipError_t launch_coeff_bwd(const CoeffBwdArgs& a, hipStream_t stream);
// Return hipErrorInvalidValue when no kernel exists for `cfg`.
hipError_t launch_chain_fwd(const ChainConfig& cfg, const ChainArgs& a, hipStream_t stream);
hipError_t launch_chain_bwd(const ChainConfig& cfg, const ChainArgs& a, hipStream_t stream);
// the instantiations with the post-chunk normalisation (cfg.pn; the two above
// forward to these)
hipError_t launch_chain_fwd_pn(const ChainConfig& cfg, const ChainArgs& a, hipStream_t stream);
hipError_t launch_chain_bwd_pn(const ChainConfig& cfg, const ChainArgs& a, hipStream_t stream);
int chain_fwd_blocks_per_cu_pn(const ChainConfig& cfg);
int chain_bwd_blocks_per_cu_pn(const ChainConfig& cfg);
// Returns hipErrorInvalidValue for a head dim / io type / width without a kernel.
hipError_t launch_apply(const ChainConfig& cfg, int fw, ApplyArgs a, hipStream_t stream);
// Clears n words (a kernel, so that it may be captured in a graph).
hipError_t launch_zero_words(unsigned* p, long n, hipStream_t stream);
// Pairs a cooperative launch of the chain kernel can hold at once (multiple of 8).
long chain_max_pairs(const ChainConfig& cfg, bool backward);
// Bytes of one checkpoint block (W or M of one unit's workgroup at one chunk start).
long chain_ckpt_bytes(const ChainConfig& cfg);
// floats of one workgroup's fp32 state block (register-tile order): the unit of
// the long-chunk buffers bfrz and w0blk
long chain_frz_floats(const ChainConfig& cfg);
// Bytes of one saved-activation block (one unit's workgroup, one chunk); 0 when
// the backward recomputes the activations instead (SwiGLU).
long chain_saved_act_bytes(const ChainConfig& cfg);
// Floats of one rank's exchange slot set (both parities).
long chain_xchg_floats(const ChainConfig& cfg, bool backward);

}  // namespace e2ttt
