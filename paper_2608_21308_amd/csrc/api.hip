// Host side of the C ABI declared in include/e2ttt.h: argument validation,
// workspace planning and kernel dispatch.  Nothing here allocates memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdlib>

#include "e2ttt.h"
#include "e2ttt_internal.h"
#include "pair_xchg.h"

namespace {

using namespace e2ttt;

constexpr size_t kAlign = 256;
// Upper bound on workgroup groups (two to eight workgroups sharing a unit) of
// one cooperative launch; more units are taken in turn by the same groups.
constexpr long kMaxPairs = 128;

// Chunks of up to 512 tokens (the paper's setting); a chunk longer than the
// kernels' 64-row tile runs as consecutive tiles at the chunk-start weights,
// forward and backward.
constexpr int kMaxChunk = 512;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// The kernels move token rows, checkpoints and partial sums as 16-byte vectors.
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Plan {
  long U = 0, T = 0, NC = 0, P = 0;
  ChainConfig cfg{};
  long npairs = 0;        // groups the exchange buffers are sized for (ns workgroups per unit)
  // forward workspace
  size_t off_kw = 0, off_km = 0, off_carry = 0, off_sync = 0, off_xbuf = 0, off_w0 = 0;
  size_t ws_bytes = 0;
  size_t off_ckpt = 0, off_zk = 0, off_rk = 0, off_zq = 0, off_rq = 0, ws_bytes_save = 0;
  // post-chunk normalisation: targets and exchange (forward), norms before it (saving)
  size_t off_ntgt = 0, off_nx = 0, off_npre = 0;
  long nrows = 0, ckpt_nc = 0;
  bool post_norm = false;
  bool w0b = false;       // the forward keeps W_0 per workgroup (long chunks re-forming operands)
  long ckpt_stride = 0;
  size_t off_as = 0;
  long as_stride = 0;
  long tpc = 1;           // 64-row tiles per chunk (chunks longer than one tile)
  // backward scratch
  size_t off_kwb = 0, off_kmb = 0, off_carryb = 0, off_bsync = 0, off_bxbuf = 0, off_frz = 0;
  size_t off_zbar = 0, off_apart = 0;   // LayerNorm affine: written rows and partial sums
  size_t off_rbar = 0, off_bnx = 0;      // post-chunk normalisation (backward)
  size_t scratch_bytes = 0;
  bool affine = false;
};

e2ttt_status select_config(const e2ttt_desc& d, ChainConfig& cfg) {
  cfg.fw = d.fw;
  cfg.d = d.d;
  cfg.bf = (d.io == E2TTT_DT_BF16) ? 1 : 0;
  const int nblk = (d.dh + 15) / 16;
  cfg.ns = 1;
  if (cfg.bf && d.d == 128) {
    // head dim 128 (the paper's 1.3B model, 2048 / 16 heads): the state of 64
    // hidden columns per workgroup (four waves, one per SIMD) and 32-row token
    // tiles (longer chunks run as consecutive tiles) fit LDS; wider nets spread
    // over 2, 4, 6 (SwiGLU) or 8 workgroups
    cfg.ntb = 2;
    cfg.nw = 4;
    cfg.njb = 1;
    if (nblk <= 4) cfg.ns = 1;
    else if (nblk <= 8) cfg.ns = 2;
    else if (nblk <= 16) cfg.ns = 4;
    else if (d.fw == E2TTT_FW_SWIGLU && nblk <= 24) cfg.ns = 6;
    else if (nblk <= 32) cfg.ns = 8;
    else return E2TTT_ERR_UNSUPPORTED;
  } else if (cfg.bf) {
    if (d.d != 64) return E2TTT_ERR_UNSUPPORTED;
    cfg.ntb = 4;
    if (nblk <= 4) { cfg.nw = 4; cfg.njb = 1; }
    else if (d.fw == E2TTT_FW_GELU_MLP && nblk <= 8) { cfg.nw = 8; cfg.njb = 1; }
    else if (d.fw == E2TTT_FW_GELU_MLP && nblk <= 16) { cfg.nw = 8; cfg.njb = 1; cfg.ns = 2; }
    // SwiGLU keeps three matrices of state per wave: one wave per SIMD (four
    // waves per workgroup) holds them without spilling, so wider nets spread
    // over two or three workgroups of 64 hidden columns each
    else if (d.fw == E2TTT_FW_SWIGLU && nblk <= 8) { cfg.nw = 4; cfg.njb = 1; cfg.ns = 2; }
    else if (d.fw == E2TTT_FW_SWIGLU && nblk <= 12) { cfg.nw = 4; cfg.njb = 1; cfg.ns = 3; }
    else return E2TTT_ERR_UNSUPPORTED;
  } else {
    if (d.d != 16) return E2TTT_ERR_UNSUPPORTED;
    cfg.ntb = (d.chunk <= 16) ? 1 : 4;
    if (nblk <= 4) { cfg.nw = 4; cfg.njb = 1; }
    else if (nblk <= 8) { cfg.nw = 8; cfg.njb = 1; }
    else return E2TTT_ERR_UNSUPPORTED;
  }
  return E2TTT_OK;
}

e2ttt_status make_plan(const e2ttt_desc* desc, Plan& pl) {
  if (!desc) return E2TTT_ERR_NULL_ARG;
  const e2ttt_desc& d = *desc;
  if (d.B < 1 || d.H < 1 || d.T < 1 || d.d < 1 || d.dh < 1 || d.chunk < 1)
    return E2TTT_ERR_BAD_SHAPE;
  if (d.fw != E2TTT_FW_GELU_MLP && d.fw != E2TTT_FW_SWIGLU) return E2TTT_ERR_UNSUPPORTED;
  if (d.io != E2TTT_DT_F32 && d.io != E2TTT_DT_BF16) return E2TTT_ERR_UNSUPPORTED;
  if (d.flags & ~(E2TTT_FLAG_NO_RESIDUAL_LN | E2TTT_FLAG_CHUNK_AVERAGED | E2TTT_FLAG_LN_AFFINE |
                  E2TTT_FLAG_POST_NORM))
    return E2TTT_ERR_UNSUPPORTED;
  if (!(d.flags & E2TTT_FLAG_NO_RESIDUAL_LN) && !(d.ln_eps > 0.0f)) return E2TTT_ERR_BAD_SHAPE;
  // the affine belongs to the LayerNorm of the residual form
  if ((d.flags & E2TTT_FLAG_LN_AFFINE) && (d.flags & E2TTT_FLAG_NO_RESIDUAL_LN))
    return E2TTT_ERR_BAD_SHAPE;
  if (d.chunk > kMaxChunk) return E2TTT_ERR_UNSUPPORTED;
  const long U = (long)d.B * d.H;
  if (U > INT_MAX || (long)d.T * d.d > (1L << 40) / U) return E2TTT_ERR_UNSUPPORTED;
  e2ttt_status st = select_config(d, pl.cfg);
  if (st != E2TTT_OK) return st;
  pl.cfg.pn = (d.flags & E2TTT_FLAG_POST_NORM) ? 1 : 0;
  pl.U = U;
  pl.T = d.T;
  pl.NC = (d.T + d.chunk - 1) / d.chunk;
  pl.P = (d.fw == E2TTT_FW_GELU_MLP ? 2L : 3L) * d.d * d.dh;
  const size_t tok = (size_t)U * d.T * sizeof(float);
  const size_t chk = (size_t)U * pl.NC * 3 * sizeof(float);
  const long ns = pl.cfg.ns;
  pl.npairs = (ns > 1) ? std::min((U + 7) / 8 * 8, kMaxPairs) : 0;
  const size_t sync_b = (ns > 1) ? (size_t)sync_words(pl.npairs, (int)ns) * sizeof(unsigned) : 0;
  pl.off_kw = 0;
  pl.off_km = align_up(tok);
  pl.off_carry = pl.off_km + align_up(tok);
  pl.off_sync = pl.off_carry + align_up(chk);
  pl.off_xbuf = pl.off_sync + align_up(sync_b);
  const int cm_rows = 16 * pl.cfg.ntb;
  pl.tpc = (d.chunk > cm_rows) ? (d.chunk + cm_rows - 1) / cm_rows : 1;
  const long nwg = (ns > 1) ? pl.npairs * ns : U;   // workgroups of a chain launch
  pl.off_w0 = pl.off_xbuf +
              align_up((size_t)pl.npairs * ns * chain_xchg_floats(pl.cfg, false) * sizeof(float));
  // long chunks on bf16 whose products re-form W_0's operands from the state
  // (SwiGLU, and the MLP at head dim 128): the forward's per-workgroup copy of W_0
  pl.w0b = pl.tpc > 1 && pl.cfg.bf && (pl.cfg.fw == E2TTT_FW_SWIGLU || d.d > 64);
  pl.off_ckpt =
      pl.off_w0 + (pl.w0b ? align_up((size_t)nwg * chain_frz_floats(pl.cfg) * sizeof(float)) : 0);
  pl.post_norm = (d.flags & E2TTT_FLAG_POST_NORM) != 0;
  pl.nrows = (d.fw == E2TTT_FW_GELU_MLP ? 1L : 2L) * d.dh + d.d;
  const size_t ngroups = (size_t)std::max(pl.npairs, 1L);
  pl.off_ntgt = pl.off_ckpt;
  pl.off_nx = pl.off_ntgt + (pl.post_norm ? align_up((size_t)U * pl.nrows * sizeof(float)) : 0);
  pl.off_ckpt = pl.off_nx +
                (pl.post_norm ? align_up(ngroups * ns * 2 * d.d * sizeof(float)) : 0);
  pl.ws_bytes = pl.off_ckpt;
  pl.ckpt_stride = chain_ckpt_bytes(pl.cfg);
  // with the normalisation the backward also reads the final state (one more block)
  pl.ckpt_nc = pl.NC + (pl.post_norm ? 1 : 0);
  const size_t tokd = tok * d.d;
  pl.off_npre = pl.off_ckpt + align_up((size_t)U * pl.ckpt_nc * ns * 2 * pl.ckpt_stride);
  pl.off_zk = pl.off_npre +
              (pl.post_norm ? align_up((size_t)U * pl.NC * pl.nrows * sizeof(float)) : 0);
  pl.off_rk = pl.off_zk + align_up(tokd);
  pl.off_zq = pl.off_rk + align_up(tok);
  pl.off_rq = pl.off_zq + align_up(tokd);
  pl.as_stride = chain_saved_act_bytes(pl.cfg);
  pl.off_as = pl.off_rq + align_up(tok);
  pl.ws_bytes_save = pl.off_as + align_up((size_t)U * pl.NC * pl.tpc * ns * pl.as_stride);
  pl.off_kwb = 0;
  pl.off_kmb = align_up(ns * tok);
  pl.off_carryb = pl.off_kmb + align_up(ns * tok);
  pl.off_bsync = pl.off_carryb + align_up(ns * chk);
  pl.off_bxbuf = pl.off_bsync + align_up(sync_b);
  pl.off_frz =
      pl.off_bxbuf +
      align_up((size_t)pl.npairs * ns * chain_xchg_floats(pl.cfg, true) * sizeof(float));
  pl.off_zbar =
      pl.off_frz +
      (pl.tpc > 1 ? align_up((size_t)nwg * 2 * chain_frz_floats(pl.cfg) * sizeof(float)) : 0);
  pl.affine = (d.flags & E2TTT_FLAG_LN_AFFINE) != 0;
  pl.off_apart = pl.off_zbar + (pl.affine ? align_up(tokd) : 0);
  const long nb = (d.T + kAffineTokBlock - 1) / kAffineTokBlock;
  pl.off_rbar =
      pl.off_apart + (pl.affine ? align_up((size_t)U * nb * 2 * d.d * sizeof(float)) : 0);
  // one copy per rank (each accumulates its own rows)
  pl.off_bnx = pl.off_rbar + (pl.post_norm ? align_up((size_t)U * ns * pl.nrows * sizeof(float)) : 0);
  pl.scratch_bytes =
      pl.off_bnx + (pl.post_norm ? align_up(ngroups * ns * 2 * d.d * sizeof(float)) : 0);
  return E2TTT_OK;
}

// The affine pointers agree with the descriptor: all given with the flag
// (gradients only in the backward), none without it.
e2ttt_status check_affine(const Plan& pl, const float* a, const float* b, bool backward,
                          const float* ga, const float* gb) {
  if (pl.affine) {
    if (!a || !b || (backward && (!ga || !gb))) return E2TTT_ERR_NULL_ARG;
    if (!aligned16(a) || !aligned16(b)) return E2TTT_ERR_BAD_SHAPE;
  } else if (a || b || ga || gb) {
    return E2TTT_ERR_BAD_SHAPE;
  }
  return E2TTT_OK;
}

int averaged(const e2ttt_desc* d) { return (d->flags & E2TTT_FLAG_CHUNK_AVERAGED) ? 1 : 0; }

e2ttt_status hip_status(hipError_t e) { return e == hipSuccess ? E2TTT_OK : E2TTT_ERR_HIP; }

// Bound of every wait between the workgroups of a unit, in ticks of the
// 100 MHz real-time counter: 2 s, or E2TTT_WAIT_LIMIT_US microseconds when
// that variable holds a decimal count (read at every call).
long long wait_ticks() {
  const char* s = std::getenv("E2TTT_WAIT_LIMIT_US");
  if (!s || !*s) return kTimeoutTicks;
  char* end = nullptr;
  const long long us = std::strtoll(s, &end, 10);
  if (*end != '\0' || us < 0) return kTimeoutTicks;
  return std::min(us, 600000000LL) * 100;
}

// E2TTT_DEBUG_SYNC=1 (read at every call)
bool debug_sync() {
  const char* s = std::getenv("E2TTT_DEBUG_SYNC");
  return s && s[0] == '1';
}

// With E2TTT_DEBUG_SYNC=1 every call waits for its kernels and, for the
// two-workgroup kernels, reads the status word of the pair exchange.
e2ttt_status finish(hipError_t e, hipStream_t s, const unsigned* sync = nullptr) {
  if (e != hipSuccess) return E2TTT_ERR_HIP;
  if (debug_sync()) {
    if (hipStreamSynchronize(s) != hipSuccess) return E2TTT_ERR_HIP;
    if (sync) {
      unsigned st = 0;
      if (hipMemcpy(&st, sync, sizeof(st), hipMemcpyDeviceToHost) != hipSuccess)
        return E2TTT_ERR_HIP;
      if (st != 0) return E2TTT_ERR_DEVICE;
    }
  }
  return E2TTT_OK;
}

// Pairs for one cooperative launch: what the buffers were sized for, capped by
// what the device holds at once.  0 when the device cannot hold eight pairs.
long launch_pairs(const Plan& pl, bool backward) {
  return std::min(pl.npairs, chain_max_pairs(pl.cfg, backward));
}

}  // namespace

namespace e2ttt {

int chain_fwd_blocks_per_cu(const ChainConfig& cfg);
int chain_bwd_blocks_per_cu(const ChainConfig& cfg);

long chain_max_pairs(const ChainConfig& cfg, bool backward) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const int nb = backward ? chain_bwd_blocks_per_cu(cfg) : chain_fwd_blocks_per_cu(cfg);
  return ((long)nb * cus / (cfg.ns > 1 ? cfg.ns : 1)) / 8 * 8;
}

long chain_xchg_floats(const ChainConfig& cfg, bool backward) {
  // per rank, in units of 16 ntb x d floats: backward two parities of the fp32
  // dYh partial and the dk, dq partials in the operand type (bf16: one unit for
  // both); forward at most two slots of Y_K and one of Y_Q
  return (backward ? (cfg.bf ? 4L : 6L) : 3L) * 16 * cfg.ntb * cfg.d;
}

long chain_frz_floats(const ChainConfig& cfg) {
  // one workgroup's share of the state: nmat matrices of 16 nw njb hidden columns x d
  return (cfg.fw == 0 ? 2L : 3L) * 16 * cfg.nw * cfg.njb * cfg.d;
}

}  // namespace e2ttt

namespace {

template <class Tp> Tp* at(void* base, size_t off) {
  return reinterpret_cast<Tp*>(static_cast<char*>(base) + off);
}
template <class Tp> const Tp* at(const void* base, size_t off) {
  return reinterpret_cast<const Tp*>(static_cast<const char*>(base) + off);
}

}  // namespace

extern "C" {

size_t e2ttt_param_count(const e2ttt_desc* desc) {
  Plan pl;
  return make_plan(desc, pl) == E2TTT_OK ? (size_t)pl.P : 0;
}

size_t e2ttt_workspace_bytes(const e2ttt_desc* desc, int save_for_backward) {
  Plan pl;
  if (make_plan(desc, pl) != E2TTT_OK) return 0;
  return save_for_backward ? pl.ws_bytes_save : pl.ws_bytes;
}

size_t e2ttt_backward_scratch_bytes(const e2ttt_desc* desc) {
  Plan pl;
  if (make_plan(desc, pl) != E2TTT_OK) return 0;
  return pl.scratch_bytes;
}

const char* e2ttt_status_str(e2ttt_status s) {
  switch (s) {
    case E2TTT_OK: return "ok";
    case E2TTT_ERR_NULL_ARG: return "a required pointer is NULL";
    case E2TTT_ERR_BAD_SHAPE: return "a size is not positive or the arguments are inconsistent";
    case E2TTT_ERR_UNSUPPORTED: return "shape, dtype or flags outside the supported set";
    case E2TTT_ERR_WORKSPACE_TOO_SMALL: return "workspace or scratch buffer too small";
    case E2TTT_ERR_HIP: return "a HIP launch failed";
    case E2TTT_ERR_DEVICE: return "a device-side wait between the two workgroups of a unit expired";
  }
  return "unknown status";
}

e2ttt_status e2ttt_chunk_coeffs(const e2ttt_desc* desc, const float* eta, const float* beta,
                                const float* gamma, float* kw, float* km, float* carry,
                                void* stream) {
  Plan pl;
  e2ttt_status st = make_plan(desc, pl);
  if (st != E2TTT_OK) return st;
  if (!eta || !beta || !kw || !km || !carry) return E2TTT_ERR_NULL_ARG;
  CoeffFwdArgs c{eta, beta, gamma, kw, km, carry, (int)pl.T, desc->chunk, (int)pl.NC,
                 pl.U * pl.NC, nullptr, 0, averaged(desc)};
  hipStream_t s = static_cast<hipStream_t>(stream);
  return finish(launch_coeff_fwd(c, s), s);
}

e2ttt_status e2ttt_apply(const e2ttt_desc* desc, const void* q, const float* w, void* out,
                         void* stream) {
  return e2ttt_apply_ln(desc, nullptr, nullptr, q, w, out, stream);
}

e2ttt_status e2ttt_apply_ln(const e2ttt_desc* desc, const float* ln_weight, const float* ln_bias,
                            const void* q, const float* w, void* out, void* stream) {
  Plan pl;
  e2ttt_status st = make_plan(desc, pl);
  if (st != E2TTT_OK) return st;
  if (!q || !w || !out) return E2TTT_ERR_NULL_ARG;
  st = check_affine(pl, ln_weight, ln_bias, false, nullptr, nullptr);
  if (st != E2TTT_OK) return st;
  if (reinterpret_cast<uintptr_t>(w) % 16 != 0) return E2TTT_ERR_BAD_SHAPE;
  if (desc->dh > (desc->d == 128 ? 512 : kApplyMaxDh)) return E2TTT_ERR_UNSUPPORTED;
  if (pl.U * ((pl.T + 7) / 8) > INT_MAX) return E2TTT_ERR_UNSUPPORTED;
  ApplyArgs a{};
  a.q = q; a.w = w; a.out = out;
  a.U = pl.U;
  a.T = (int)pl.T;
  a.dh = desc->dh;
  a.P = pl.P;
  a.resln = (desc->flags & E2TTT_FLAG_NO_RESIDUAL_LN) ? 0 : 1;
  a.eps = desc->ln_eps;
  a.ln_a = ln_weight;
  a.ln_b = ln_bias;
  a.H = desc->H;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return finish(launch_apply(pl.cfg, desc->fw, a, s), s);
}

e2ttt_status e2ttt_chunk_forward(const e2ttt_desc* desc, const void* q, const void* k,
                                 const void* v, const float* eta, const float* beta,
                                 const float* gamma, const float* w_in, const float* m_in,
                                 void* out, float* w_out, float* m_out, void* workspace,
                                 size_t workspace_bytes, int save_for_backward, void* stream) {
  return e2ttt_chunk_forward_ln(desc, nullptr, nullptr, q, k, v, eta, beta, gamma, w_in, m_in,
                                out, w_out, m_out, workspace, workspace_bytes, save_for_backward,
                                stream);
}

e2ttt_status e2ttt_chunk_forward_ln(const e2ttt_desc* desc, const float* ln_weight,
                                    const float* ln_bias, const void* q, const void* k,
                                    const void* v, const float* eta, const float* beta,
                                    const float* gamma, const float* w_in, const float* m_in,
                                    void* out, float* w_out, float* m_out, void* workspace,
                                    size_t workspace_bytes, int save_for_backward, void* stream) {
  Plan pl;
  e2ttt_status st = make_plan(desc, pl);
  if (st != E2TTT_OK) return st;
  if (!q || !k || !v || !eta || !beta || !w_in || !out || !w_out || !m_out || !workspace)
    return E2TTT_ERR_NULL_ARG;
  st = check_affine(pl, ln_weight, ln_bias, false, nullptr, nullptr);
  if (st != E2TTT_OK) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(workspace))
    return E2TTT_ERR_BAD_SHAPE;
  if (workspace_bytes < (save_for_backward ? pl.ws_bytes_save : pl.ws_bytes))
    return E2TTT_ERR_WORKSPACE_TOO_SMALL;
  if (save_for_backward && (w_out == w_in || (m_in && m_out == m_in))) return E2TTT_ERR_BAD_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* kw = at<float>(workspace, pl.off_kw);
  float* km = at<float>(workspace, pl.off_km);
  float* carry = at<float>(workspace, pl.off_carry);
  unsigned* sync = pl.cfg.ns > 1 ? at<unsigned>(workspace, pl.off_sync) : nullptr;
  const long np = pl.cfg.ns > 1 ? launch_pairs(pl, false) : 0;
  if (pl.cfg.ns > 1 && np < 8) return E2TTT_ERR_UNSUPPORTED;
  CoeffFwdArgs c{eta, beta, gamma, kw, km, carry, (int)pl.T, desc->chunk, (int)pl.NC,
                 pl.U * pl.NC, sync, sync ? sync_words(np, pl.cfg.ns) : 0, averaged(desc)};
  hipError_t e = launch_coeff_fwd(c, s);
  if (e != hipSuccess) return E2TTT_ERR_HIP;
  if (pl.post_norm) {
    e = launch_norm_targets(w_in, at<float>(workspace, pl.off_ntgt), pl.U, desc->d, desc->dh,
                            pl.cfg.fw == E2TTT_FW_GELU_MLP ? 2 : 3, pl.P, s);
    if (e != hipSuccess) return E2TTT_ERR_HIP;
  }
  ChainArgs a{};
  a.U = pl.U;
  a.q = q; a.k = k; a.v = v;
  a.w_in = w_in; a.m_in = m_in;
  a.kw = kw; a.km = km; a.carry = carry;
  a.out = out; a.w_out = w_out; a.m_out = m_out;
  a.ckpt = save_for_backward ? at<char>(workspace, pl.off_ckpt) : nullptr;
  a.ckpt_stride = pl.ckpt_stride;
  if (save_for_backward) {
    a.asave = pl.as_stride ? at<char>(workspace, pl.off_as) : nullptr;
    a.as_stride = pl.as_stride;
    a.zk = at<float>(workspace, pl.off_zk);
    a.rk = at<float>(workspace, pl.off_rk);
    a.zq = at<float>(workspace, pl.off_zq);
    a.rq = at<float>(workspace, pl.off_rq);
  }
  a.xbuf = at<float>(workspace, pl.off_xbuf);
  a.w0blk = pl.w0b ? at<float>(workspace, pl.off_w0) : nullptr;
  a.sync = sync;
  a.npairs = np;
  a.wait_ticks = wait_ticks();
  a.T = (int)pl.T; a.C = desc->chunk; a.NC = (int)pl.NC; a.dh = desc->dh; a.P = pl.P;
  a.resln = (desc->flags & E2TTT_FLAG_NO_RESIDUAL_LN) ? 0 : 1;
  a.eps = desc->ln_eps;
  a.ln_a = ln_weight;
  a.ln_b = ln_bias;
  a.H = desc->H;
  a.ckpt_nc = pl.ckpt_nc;
  if (pl.post_norm) {
    a.norm_tgt = at<float>(workspace, pl.off_ntgt);
    a.nxbuf = at<float>(workspace, pl.off_nx);
    a.norm_pre = save_for_backward ? at<float>(workspace, pl.off_npre) : nullptr;
  }
  return finish(launch_chain_fwd(pl.cfg, a, s), s, sync);
}

e2ttt_status e2ttt_chunk_backward(const e2ttt_desc* desc, const void* q, const void* k,
                                  const void* v, const float* eta, const float* beta,
                                  const float* gamma, const float* w_in, const float* m_in,
                                  const void* workspace, size_t workspace_bytes,
                                  const void* d_out, const float* d_w_out, const float* d_m_out,
                                  void* dq, void* dk, void* dv, float* d_eta, float* d_beta,
                                  float* d_gamma, float* d_w_in, float* d_m_in, void* scratch,
                                  size_t scratch_bytes, void* stream) {
  return e2ttt_chunk_backward_ln(desc, nullptr, nullptr, q, k, v, eta, beta, gamma, w_in, m_in,
                                 workspace, workspace_bytes, d_out, d_w_out, d_m_out, dq, dk, dv,
                                 d_eta, d_beta, d_gamma, d_w_in, d_m_in, nullptr, nullptr,
                                 scratch, scratch_bytes, stream);
}

e2ttt_status e2ttt_chunk_backward_ln(const e2ttt_desc* desc, const float* ln_weight,
                                     const float* ln_bias, const void* q, const void* k,
                                     const void* v, const float* eta, const float* beta,
                                     const float* gamma, const float* w_in, const float* m_in,
                                     const void* workspace, size_t workspace_bytes,
                                     const void* d_out, const float* d_w_out,
                                     const float* d_m_out, void* dq, void* dk, void* dv,
                                     float* d_eta, float* d_beta, float* d_gamma, float* d_w_in,
                                     float* d_m_in, float* d_ln_weight, float* d_ln_bias,
                                     void* scratch, size_t scratch_bytes, void* stream) {
  Plan pl;
  e2ttt_status st = make_plan(desc, pl);
  if (st != E2TTT_OK) return st;
  st = check_affine(pl, ln_weight, ln_bias, true, d_ln_weight, d_ln_bias);
  if (st != E2TTT_OK) return st;
  if (!q || !k || !v || !eta || !beta || !w_in || !workspace || !d_out || !dq || !dk || !dv ||
      !d_eta || !d_beta || !d_w_in || !d_m_in || !scratch)
    return E2TTT_ERR_NULL_ARG;
  if ((gamma == nullptr) != (d_gamma == nullptr)) return E2TTT_ERR_BAD_SHAPE;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(workspace) ||
      !aligned16(d_out) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv) || !aligned16(scratch))
    return E2TTT_ERR_BAD_SHAPE;
  if (workspace_bytes < pl.ws_bytes_save || scratch_bytes < pl.scratch_bytes)
    return E2TTT_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned* sync = pl.cfg.ns > 1 ? at<unsigned>(scratch, pl.off_bsync) : nullptr;
  const long np = pl.cfg.ns > 1 ? launch_pairs(pl, true) : 0;
  if (pl.cfg.ns > 1 && np < 8) return E2TTT_ERR_UNSUPPORTED;
  if (sync && launch_zero_words(sync, sync_words(np, pl.cfg.ns), s) != hipSuccess)
    return E2TTT_ERR_HIP;
  ChainArgs a{};
  a.U = pl.U;
  a.q = q; a.k = k; a.v = v;
  a.w_in = w_in; a.m_in = m_in;
  a.kw = at<float>(workspace, pl.off_kw);
  a.km = at<float>(workspace, pl.off_km);
  a.carry = at<float>(workspace, pl.off_carry);
  a.ckpt = const_cast<char*>(at<char>(workspace, pl.off_ckpt));
  a.ckpt_stride = pl.ckpt_stride;
  a.asave = pl.as_stride ? const_cast<char*>(at<char>(workspace, pl.off_as)) : nullptr;
  a.as_stride = pl.as_stride;
  a.zk = const_cast<float*>(at<float>(workspace, pl.off_zk));
  a.rk = const_cast<float*>(at<float>(workspace, pl.off_rk));
  a.zq = const_cast<float*>(at<float>(workspace, pl.off_zq));
  a.rq = const_cast<float*>(at<float>(workspace, pl.off_rq));
  a.xbuf = at<float>(scratch, pl.off_bxbuf);
  a.sync = sync;
  a.npairs = np;
  a.wait_ticks = wait_ticks();
  a.d_out = d_out; a.d_w_out = d_w_out; a.d_m_out = d_m_out;
  a.dq = dq; a.dk = dk; a.dv = dv;
  a.d_w_in = d_w_in; a.d_m_in = d_m_in;
  a.kwb = at<float>(scratch, pl.off_kwb);
  a.kmb = at<float>(scratch, pl.off_kmb);
  a.carryb = at<float>(scratch, pl.off_carryb);
  a.bfrz = pl.tpc > 1 ? at<float>(scratch, pl.off_frz) : nullptr;
  a.T = (int)pl.T; a.C = desc->chunk; a.NC = (int)pl.NC; a.dh = desc->dh; a.P = pl.P;
  a.resln = (desc->flags & E2TTT_FLAG_NO_RESIDUAL_LN) ? 0 : 1;
  a.eps = desc->ln_eps;
  a.ln_a = ln_weight;
  a.ln_b = ln_bias;
  a.H = desc->H;
  a.ln_zbar = pl.affine ? at<float>(scratch, pl.off_zbar) : nullptr;
  a.ckpt_nc = pl.ckpt_nc;
  if (pl.post_norm) {
    a.norm_tgt = at<float>(workspace, pl.off_ntgt);
    a.norm_pre = const_cast<float*>(at<float>(workspace, pl.off_npre));
    a.norm_rbar = at<float>(scratch, pl.off_rbar);
    a.nxbuf = at<float>(scratch, pl.off_bnx);
  }
  hipError_t e = launch_chain_bwd(pl.cfg, a, s);
  if (e != hipSuccess) return E2TTT_ERR_HIP;
  CoeffBwdArgs cb{eta, beta, gamma, a.kwb, a.kmb, a.carryb, d_eta, d_beta, d_gamma,
                  (int)pl.T, desc->chunk, (int)pl.NC, pl.U * pl.NC, pl.cfg.ns,
                  pl.U * pl.T, pl.U * pl.NC * 3, averaged(desc)};
  e = launch_coeff_bwd(cb, s);
  if (e == hipSuccess && pl.affine) {
    AffineGradArgs g{d_out, k, v, a.zk, a.zq, a.ln_zbar, ln_weight, ln_bias,
                     at<float>(scratch, pl.off_apart), d_ln_weight, d_ln_bias, pl.U, desc->H,
                     (int)pl.T, desc->d, pl.cfg.bf};
    e = launch_affine_grad(g, s);
  }
  return finish(e, s, sync);
}

e2ttt_status e2ttt_wait_status(const e2ttt_desc* desc, const void* workspace,
                               const void* scratch, void* stream) {
  Plan pl;
  e2ttt_status st = make_plan(desc, pl);
  if (st != E2TTT_OK) return st;
  if (!workspace && !scratch) return E2TTT_ERR_NULL_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipStreamSynchronize(s) != hipSuccess) return E2TTT_ERR_HIP;
  if (pl.cfg.ns == 1) return E2TTT_OK;   // one workgroup per unit: no waits
  unsigned word[2] = {0u, 0u};
  if (workspace && hipMemcpy(&word[0], at<unsigned>(workspace, pl.off_sync), sizeof(unsigned),
                             hipMemcpyDeviceToHost) != hipSuccess)
    return E2TTT_ERR_HIP;
  if (scratch && hipMemcpy(&word[1], at<unsigned>(scratch, pl.off_bsync), sizeof(unsigned),
                           hipMemcpyDeviceToHost) != hipSuccess)
    return E2TTT_ERR_HIP;
  return (word[0] != 0u || word[1] != 0u) ? E2TTT_ERR_DEVICE : E2TTT_OK;
}

}  // extern "C"
