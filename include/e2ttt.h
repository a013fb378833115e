/*
 * e2ttt.h -- C ABI of the MI355X (gfx950) E2-TTT chunk-parallel fast-weight update.
 *
 * Method: arxiv 2608.21308, "Rethinking Expressivity and Efficiency in
 * Test-Time Training".  The library computes, for every (batch, head) unit
 * independently, the chunk update of Algorithm 1:
 *   - chunk-start outputs  o_t = f_{W_0}(q_t)                  (eq. (6))
 *   - per-token gradients  G_t = -grad_W 1/2||f_{W_0}(k_t) - v_t||^2 at the
 *     chunk-start weights (Sec. 3.1)
 *   - the closed-form transition of Prop. 1 (eq. (10)-(11))
 *       M_C = b~_0 M_0 + sum_t K^M_t G_t
 *       W_C = g~_0 W_0 + b~_0 R_1 M_0 + sum_t K^W_t G_t
 *     which equals the per-token recurrence M_t = beta_t M_{t-1} + eta_t G_t,
 *     W_t = gamma_t W_{t-1} + M_t (eq. (7)) at every chunk end,
 * and the state (W, M) is carried from chunk to chunk.  The fast-weight net f
 * is the GELU MLP f(x) = x + LN(W2 GELU(W1 x)) or the SwiGLU net
 * f(x) = x + LN(Wd (SiLU(Wg x) * (Wu x))) of Sec. 4 (LayerNorm with biased
 * variance, eps = ln_eps, and optionally a learnable affine per head,
 * E2TTT_FLAG_LN_AFFINE).  GELU is x Phi(x) with the normal CDF; the
 * chunk kernels evaluate Phi through the rational erfc of Abramowitz & Stegun
 * eq. 7.1.26 (absolute error at most 1.5e-7, so a relative error of Phi that
 * grows for x << 0 where Phi itself is tiny), e2ttt_apply through erff.
 *
 * Conventions shared by every entry point:
 *   - Every tensor pointer is a DEVICE pointer (hipMalloc'd or equivalent) on
 *     the current HIP device; all work is enqueued on `stream` (a hipStream_t,
 *     NULL = the default stream) and the call returns without waiting.
 *   - The caller owns every buffer; the library never allocates, frees or
 *     keeps state between calls and is safe to call from several host threads
 *     on distinct streams.
 *   - Every argument check runs before anything is launched; on an error
 *     return nothing has been written.  Errors raised by kernels while they
 *     run surface on the stream as HIP errors.
 *   - Results are bitwise reproducible run to run (no floating-point atomics).
 *   - For the wider nets (d = 64: GELU MLP with dh > 128, SwiGLU with
 *     dh > 64; d = 128: dh > 64) each unit is split over two to eight
 *     workgroups that swap partial sums through the workspace (or the
 *     backward scratch); those
 *     kernels are launched cooperatively, so a call may wait for the whole
 *     device.  Calls that share a workspace or scratch buffer must not run
 *     concurrently.
 *
 * Tensor layouts (row-major, C order):
 *   q, k, v, out, d_out, dq, dk, dv : [B][H][T][d]   element type desc.io
 *   eta, beta, gamma, d_eta, ...    : [B][H][T]      float32
 *   w_*, m_*, d_w_*, d_m_*          : [B][H][P]      float32, P parameters per unit
 * Packing of the P fast-weight parameters of one unit (row-major, W x rule):
 *   GELU MLP : W1[dh][d], then W2[d][dh]                       P = 2 d dh
 *   SwiGLU   : Wg[dh][d], then Wu[dh][d], then Wd[d][dh]        P = 3 d dh
 *   (Wg, Wu, Wd are the paper's W1, W2, W3 of the SwiGLU net.)
 *
 * Supported shapes: io = BF16 with d = 64 (dh <= 256 for the MLP, <= 192 for
 * SwiGLU) or d = 128 (dh <= 512), or io = F32 with d = 16
 * (dh <= 128); dh is padded inside the library to a multiple of 16;
 * 1 <= chunk <= 512 (the paper's C = 512), forward and backward; a chunk
 * longer than the kernels' token tile (64 rows, 32 at d = 128) runs as
 * consecutive tiles that all take gradients and outputs at the chunk-start
 * weights; e2ttt_apply takes d <= 64; T >= 1 with
 * a ragged last chunk of T mod chunk tokens allowed (Prop. 1 holds for any
 * chunk length).
 * bf16 tensors use MFMA bf16 operands with fp32 accumulation and fp32 state;
 * f32 tensors use fp32 MFMA throughout.  Anything else returns
 * E2TTT_ERR_UNSUPPORTED.
 */
#ifndef E2TTT_H
#define E2TTT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  E2TTT_OK = 0,
  E2TTT_ERR_NULL_ARG = 1,              /* a required pointer is NULL             */
  E2TTT_ERR_BAD_SHAPE = 2,             /* a size is <= 0 or inconsistent          */
  E2TTT_ERR_UNSUPPORTED = 3,           /* valid but outside the supported set     */
  E2TTT_ERR_WORKSPACE_TOO_SMALL = 4,   /* workspace / scratch smaller than needed */
  E2TTT_ERR_HIP = 5,                   /* a HIP launch failed                     */
  E2TTT_ERR_DEVICE = 6                 /* a bounded device-side wait expired      */
} e2ttt_status;
/* E2TTT_ERR_DEVICE: a bounded wait between the workgroups of a unit expired
 * (after 2 s, or the limit set by E2TTT_WAIT_LIMIT_US), the grid was drained
 * and the results of that call are undefined.  The kernels record it in a
 * status word of the workspace (forward) or scratch (backward) buffer;
 * e2ttt_wait_status reads it.  With the environment variable
 * E2TTT_DEBUG_SYNC=1 (read at every call) every call also waits for its
 * kernels and returns it. */

typedef enum { E2TTT_FW_GELU_MLP = 0, E2TTT_FW_SWIGLU = 1 } e2ttt_fw;

/* Element type of q, k, v, out, d_out, dq, dk, dv. */
typedef enum { E2TTT_DT_F32 = 0, E2TTT_DT_BF16 = 1 } e2ttt_dtype;

/* f(x) = y (the bare matrix net) instead of f(x) = x + LN(y). */
#define E2TTT_FLAG_NO_RESIDUAL_LN 0x1u
/* Chunk-averaged update rule instead of the closed form of Prop. 1: the
 * ablation baseline of Sec. 5 (Tables 4 and 5) that collapses the per-token
 * momentum and decay factors of a chunk to their means, after the chunk-level
 * momentum of eqs. (4)-(5).  Per chunk of L tokens, with beta_bar and
 * gamma_bar the means of beta_t and gamma_t over the chunk (gamma NULL:
 * gamma_bar = 1, which is eqs. (4)-(5) exactly):
 *   M_C = beta_bar M_0 + sum_t eta_t G_t,   W_C = gamma_bar W_0 + M_C,
 * that is K^W_t = K^M_t = eta_t and carry (gamma_bar, beta_bar, beta_bar).
 * Outputs, gradients and every other convention are unchanged (all entry
 * points that take a descriptor honour the flag). */
#define E2TTT_FLAG_CHUNK_AVERAGED 0x2u
/* Learnable LayerNorm affine of the fast-weight net (Sec. 4's LayerNorm with
 * an elementwise weight and bias per head, slow weights shared by the batch):
 *   f(x) = x + a * LN(y) + b,   a, b in R^d per head.
 * Calls with this flag take a and b (and return their gradients) through the
 * *_ln entry points below; the plain entry points return E2TTT_ERR_NULL_ARG
 * for it.  Not combinable with E2TTT_FLAG_NO_RESIDUAL_LN (E2TTT_ERR_BAD_SHAPE). */
#define E2TTT_FLAG_LN_AFFINE 0x4u
/* Post-chunk L2 normalisation of the fast weights (App. B.1, after LaCT): at
 * every chunk end, after the update of Prop. 1, each row of each fast-weight
 * matrix, taken over the matrix's input dimension (W1 / Wg / Wu: a hidden
 * unit's d weights; W2 / Wd: an output's dh weights), is rescaled to the norm
 * of the same row of the unit's initial weights w_in; a row of norm zero is
 * left as it is, the momentum is not normalised.  Chunk-start states, outputs
 * and w_out are then those of the normalised weights; the backward includes
 * the normalisation and its targets' dependence on w_in.  (The paper gives no
 * axis or target; this is the reading taken.  Off by default: with it the
 * closed form no longer equals the plain token recurrence.) */
#define E2TTT_FLAG_POST_NORM 0x8u

typedef struct {
  int32_t B, H, T;      /* batch, heads, tokens                        */
  int32_t d, dh;        /* head dim, fast-weight hidden width          */
  int32_t chunk;        /* chunk length C                              */
  int32_t fw;           /* e2ttt_fw                                    */
  int32_t io;           /* e2ttt_dtype                                 */
  uint32_t flags;       /* E2TTT_FLAG_*                                */
  float ln_eps;         /* LayerNorm epsilon (> 0 unless NO_RESIDUAL_LN) */
} e2ttt_desc;

/* Parameters per unit (P above), or 0 for a bad descriptor. */
size_t e2ttt_param_count(const e2ttt_desc* desc);

/* Bytes of `workspace` that e2ttt_chunk_forward needs.  With
 * save_for_backward != 0 the workspace also keeps what the backward reuses
 * (per-token scalar kernels, chunk-start checkpoints of W and M in the
 * operand precision, the LayerNorm outputs and inverse deviations of the key
 * and query passes, and for the GELU MLP the query-side activations and GELU
 * derivatives), and the same buffer, untouched, must then be passed to
 * e2ttt_chunk_backward.  Returns 0 for a bad descriptor. */
size_t e2ttt_workspace_bytes(const e2ttt_desc* desc, int save_for_backward);

/* Bytes of `scratch` that e2ttt_chunk_backward needs (0 for a bad descriptor). */
size_t e2ttt_backward_scratch_bytes(const e2ttt_desc* desc);

/*
 * Forward: Algorithm 1 over every chunk of every unit.
 *   q, k, v   [B][H][T][d] io     queries, keys, values (k, v feed the inner
 *                                 loss, q the outputs)
 *   eta, beta [B][H][T]   f32     learning rate and momentum gates, eq. (7)
 *   gamma     [B][H][T]   f32     decay gate; NULL means gamma = 1
 *   w_in      [B][H][P]   f32     initial fast weights W (chunk-start state of chunk 0)
 *   m_in      [B][H][P]   f32     initial momentum M; NULL means zero
 *   out       [B][H][T][d] io     o_t = f_{W_0}(q_t) with W_0 the start state of t's chunk
 *   w_out, m_out [B][H][P] f32    state after the last token
 *   workspace, workspace_bytes    caller-owned device memory, at least
 *                                 e2ttt_workspace_bytes(desc, save_for_backward)
 * w_out / m_out may alias w_in / m_in only when save_for_backward == 0.
 * q, k, v, out and workspace must be 16-byte aligned (else E2TTT_ERR_BAD_SHAPE).
 */
e2ttt_status e2ttt_chunk_forward(const e2ttt_desc* desc, const void* q, const void* k,
                                 const void* v, const float* eta, const float* beta,
                                 const float* gamma, const float* w_in, const float* m_in,
                                 void* out, float* w_out, float* m_out, void* workspace,
                                 size_t workspace_bytes, int save_for_backward, void* stream);

/*
 * Backward of  sum_t <d_out_t, o_t> + <d_w_out, W_T> + <d_m_out, M_T>
 * with respect to every input of the forward (reverse mode through the chunk
 * chain; the paper trains with autograd through the same computation).
 *   q .. m_in         the forward's inputs, unchanged
 *   workspace         as left by e2ttt_chunk_forward(..., save_for_backward = 1)
 *   d_out             [B][H][T][d] io   gradient of the outputs
 *   d_w_out, d_m_out  [B][H][P] f32     gradient of the final state; NULL = zero
 *   dq, dk, dv        [B][H][T][d] io
 *   d_eta, d_beta     [B][H][T] f32
 *   d_gamma           [B][H][T] f32; must be NULL iff gamma is NULL
 *   d_w_in, d_m_in    [B][H][P] f32     gradient of the initial state
 *   scratch           at least e2ttt_backward_scratch_bytes(desc) bytes
 * q, k, v, workspace, d_out, dq, dk, dv and scratch must be 16-byte aligned
 * (else E2TTT_ERR_BAD_SHAPE).
 */
e2ttt_status e2ttt_chunk_backward(const e2ttt_desc* desc, const void* q, const void* k,
                                  const void* v, const float* eta, const float* beta,
                                  const float* gamma, const float* w_in, const float* m_in,
                                  const void* workspace, size_t workspace_bytes,
                                  const void* d_out, const float* d_w_out, const float* d_m_out,
                                  void* dq, void* dk, void* dv, float* d_eta, float* d_beta,
                                  float* d_gamma, float* d_w_in, float* d_m_in, void* scratch,
                                  size_t scratch_bytes, void* stream);

/*
 * Scalar kernels of every chunk (Prop. 1, eq. (9)-(11)), exposed on their own
 * so that callers (and tests) can inspect them:
 *   kw, km      [B][H][T] f32   K^W_t = eta_t b~_t R_t and K^M_t = eta_t b~_t
 *   carry       [B][H][NC][3] f32, NC = ceil(T / chunk): (g~_0, b~_0 R_1, b~_0)
 * gamma NULL means gamma = 1.
 */
e2ttt_status e2ttt_chunk_coeffs(const e2ttt_desc* desc, const float* eta, const float* beta,
                                const float* gamma, float* kw, float* km, float* carry,
                                void* stream);

/*
 * Net evaluation at a given state: out_t = f_W(q_t) for T tokens per unit, all
 * at the unit's one state W.  This is how a token's output is formed (eq. (6):
 * the net at the start state of the token's chunk, Table 1), exposed for
 * streaming decode: while a chunk fills, each arriving token is answered from
 * the current chunk-start state with this call (T = 1), and once C tokens have
 * arrived e2ttt_chunk_forward over those C tokens (w_in, m_in = the current
 * state) gives the next chunk-start state.  Outputs and states then agree
 * with those of one e2ttt_chunk_forward over the whole sequence within the
 * bf16 / fp32 tolerances (the two evaluate GELU's Phi differently, above).
 *   desc   as for the chunk calls (same supported set); desc.T is the number
 *          of tokens per unit to evaluate; desc.chunk is checked but unused
 *   q      [B][H][T][d] io
 *   w      [B][H][P]   f32, 16-byte aligned (else E2TTT_ERR_BAD_SHAPE)
 *   out    [B][H][T][d] io; may not overlap q or w
 * fp32 arithmetic on the fp32 state (GELU through erff); no workspace.
 */
e2ttt_status e2ttt_apply(const e2ttt_desc* desc, const void* q, const float* w, void* out,
                         void* stream);

/*
 * Gate parameterization of Sec. 4 ("Input-Dependent Dynamics", eqs. (12)-(14)):
 * per token, from the outputs l_eta, l_beta, l_alpha of the three linear heads,
 *   eta   = eta_base * sigmoid(l_eta)                       (12)
 *   beta  = sigmoid(l_beta)^(1 / tau)                       (13)
 *   alpha = alpha_base * sigmoid(l_alpha),  gamma = 1 - eta * alpha   (14)
 * (the paper trains with eta_base = 0.01, tau = 32, alpha_base = 0.1, App. B.1).
 * The outputs are the gate arrays e2ttt_chunk_forward takes, and the backward
 * maps the gate gradients e2ttt_chunk_backward returns to the logits.
 *   n                       number of tokens (B H T); 0 is a no-op
 *   l_eta, l_beta, l_alpha  [n] f32 device arrays; l_alpha NULL means no decay
 *                           gate (gamma = 1): gamma, d_gamma and d_l_alpha must
 *                           then be NULL too
 *   eta, beta, gamma        [n] f32 outputs
 * Errors: a required pointer NULL (or one of the alpha-side pointers given
 * without l_alpha) -> E2TTT_ERR_NULL_ARG; n < 0, tau <= 0 or a negative or
 * non-finite base -> E2TTT_ERR_BAD_SHAPE.  Caller-owned buffers, no workspace.
 */
typedef struct {
  float eta_base;    /* >= 0 */
  float alpha_base;  /* >= 0 */
  float tau;         /* > 0 */
} e2ttt_gate_params;

e2ttt_status e2ttt_gates_forward(const e2ttt_gate_params* params, int64_t n, const float* l_eta,
                                 const float* l_beta, const float* l_alpha, float* eta,
                                 float* beta, float* gamma, void* stream);

/* Backward of e2ttt_gates_forward: given d_eta, d_beta, d_gamma [n] f32 (for
 * example from e2ttt_chunk_backward), the gradients d_l_eta, d_l_beta,
 * d_l_alpha [n] f32 of the logits.  Same pointer rules as the forward. */
e2ttt_status e2ttt_gates_backward(const e2ttt_gate_params* params, int64_t n,
                                  const float* l_eta, const float* l_beta, const float* l_alpha,
                                  const float* d_eta, const float* d_beta, const float* d_gamma,
                                  float* d_l_eta, float* d_l_beta, float* d_l_alpha,
                                  void* stream);

/*
 * Status of the bounded waits between the workgroups of a unit in the last
 * e2ttt_chunk_forward that used `workspace` and the last e2ttt_chunk_backward
 * that used `scratch` (either may be NULL, not both).  Waits for `stream`
 * first (the calls must have been enqueued there or be complete), then reads
 * the status words: E2TTT_ERR_DEVICE when a wait of either call expired (its
 * results are undefined), E2TTT_OK otherwise (always for descriptors that run
 * one workgroup per unit).  Each call clears its buffer's word when it starts.
 * The wait limit is 2 s; the environment variable E2TTT_WAIT_LIMIT_US (a
 * decimal count of microseconds, read at every call) sets another; a limit of
 * 0 makes every wait give up before it reads the peer's flag, which lets a
 * test force the expiry without any kernel failing.
 */
e2ttt_status e2ttt_wait_status(const e2ttt_desc* desc, const void* workspace,
                               const void* scratch, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * e2ttt_chunk_forward with save_for_backward = 0 on a workspace the library
 * owns, a device array of E2TTT_STATIC_WORKSPACE_BYTES on each GPU it runs
 * on, held until the process ends.  Inputs, outputs and their rules are those
 * of e2ttt_chunk_forward.  A descriptor whose workspace
 * (e2ttt_workspace_bytes(desc, 0)) exceeds E2TTT_STATIC_WORKSPACE_BYTES
 * returns E2TTT_ERR_WORKSPACE_TOO_SMALL before anything is launched.  The call
 * allocates nothing.  Every call on a GPU shares that GPU's array: calls that
 * overlap on one GPU race (enqueue them on one stream, or wait between them).
 * e2ttt_wait_status cannot read its status word (the array is the library's);
 * E2TTT_DEBUG_SYNC=1 reports an expired wait from the call itself.
 */
#define E2TTT_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
e2ttt_status e2ttt_chunk_forward_static(const e2ttt_desc* desc, const void* q, const void* k,
                                        const void* v, const float* eta, const float* beta,
                                        const float* gamma, const float* w_in, const float* m_in,
                                        void* out, float* w_out, float* m_out, void* stream);

/*
 * The chunk calls and the net evaluation with the learnable LayerNorm affine
 * (E2TTT_FLAG_LN_AFFINE in desc.flags): the same arguments as e2ttt_chunk_forward,
 * e2ttt_chunk_backward and e2ttt_apply, plus
 *   ln_weight, ln_bias    [H][d] f32 device arrays: a and b of each head (unit
 *                         (b, h) uses row h); required with the flag
 *   d_ln_weight, d_ln_bias [H][d] f32 (backward only): the gradients of a and b,
 *                         summed over the batch and all tokens (overwritten)
 * Without the flag every one of these pointers must be NULL, and the calls
 * equal the plain ones.  The backward's scratch (e2ttt_backward_scratch_bytes,
 * which reads the flag) then also holds, per token row, the adjoint the
 * affine's gradients are summed from, and one partial sum per block of 256
 * tokens; ln_weight and ln_bias must be 16-byte aligned (else E2TTT_ERR_BAD_SHAPE).
 */
e2ttt_status e2ttt_chunk_forward_ln(const e2ttt_desc* desc, const float* ln_weight,
                                    const float* ln_bias, const void* q, const void* k,
                                    const void* v, const float* eta, const float* beta,
                                    const float* gamma, const float* w_in, const float* m_in,
                                    void* out, float* w_out, float* m_out, void* workspace,
                                    size_t workspace_bytes, int save_for_backward, void* stream);
e2ttt_status e2ttt_chunk_backward_ln(const e2ttt_desc* desc, const float* ln_weight,
                                     const float* ln_bias, const void* q, const void* k,
                                     const void* v, const float* eta, const float* beta,
                                     const float* gamma, const float* w_in, const float* m_in,
                                     const void* workspace, size_t workspace_bytes,
                                     const void* d_out, const float* d_w_out,
                                     const float* d_m_out, void* dq, void* dk, void* dv,
                                     float* d_eta, float* d_beta, float* d_gamma, float* d_w_in,
                                     float* d_m_in, float* d_ln_weight, float* d_ln_bias,
                                     void* scratch, size_t scratch_bytes, void* stream);
e2ttt_status e2ttt_apply_ln(const e2ttt_desc* desc, const float* ln_weight, const float* ln_bias,
                            const void* q, const float* w, void* out, void* stream);

/* Static description of a status code. */
const char* e2ttt_status_str(e2ttt_status status);

#ifdef __cplusplus
}
#endif

#endif /* E2TTT_H */
