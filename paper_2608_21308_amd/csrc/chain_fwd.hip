// Forward chain kernel: Algorithm 1 of the paper over every chunk of a unit.
//
// Per chunk (tokens t < len, the state (W_0, M_0) in registers):
//   H  = K W1^T              contraction over i, state tiles as operand   (a3)
//   A  = act(H)               GELU, or SiLU(Hg) * Hu for SwiGLU
//   Y  = A W2^T               contraction over j, A and W2 staged in LDS
//   Z  = LN(Y), E = V - K - Z, dY = LN backward of E            (a4, the g_t)
//   dA = dY W2,  dH = dA * act'(H)                                          (a4)
//   W  <- cw W + cm M + sum_t K^W_t G_t,   M <- cb M + sum_t K^M_t G_t      (a5, a6)
//        with sum_t K_t G_t = (dY^T diag(K) A, dH^T diag(K) K): MFMAs that
//        accumulate straight into the state tiles
//   O  = Q + LN(act(Q W1^T) W2^T)     outputs from the chunk-start weights (a7)
// The new state stays in registers for the next chunk (a8).
//
// Chunks longer than the CM-row tile (C up to 512) run as consecutive tiles of
// one chunk: every tile takes its gradients and outputs at the chunk-start
// weights (the operand copies formed at the chunk's first tile), the state is
// scaled by the carries once, at the first tile, and every tile accumulates
// its sum_t K_t G_t into it, so the chunk end is Prop. 1 over all C tokens.
//
// With NS workgroups per unit (pair_xchg.h) each holds a share of the hidden
// columns; the j-contractions Y_K and Y_Q then give partial sums that the
// ranks swap.  The Q-side first layer and Y_Q run between posting the Y_K
// partial and waiting for the peers', so the exchange overlaps that work; the
// Y_Q swap is waited for only at the end of the chunk.  Every rank adds the
// partials in rank order, so all see bitwise identical Y_K and dY.
#include <algorithm>

#include "chain_common.h"
#include "pair_xchg.h"

// The instantiations with the post-chunk normalisation of the fast weights are
// compiled in a translation unit of their own (chain_fwd_pn.hip defines this
// as 1 and includes this file), in parallel with the plain ones.
#ifndef E2TTT_CHAIN_PN
#define E2TTT_CHAIN_PN 0
#endif
#if E2TTT_CHAIN_PN
#define E2TTT_PN_NAME(f) f##_pn
#else
#define E2TTT_PN_NAME(f) f
#endif

namespace e2ttt {

namespace {

template <class S>
struct FwdSmemBase {
  using E = typename S::E;
  static constexpr int BYTES =
      (3 * S::CM * S::LDD + S::D * S::LDC + S::CM * S::LDH + S::D * S::LDH + S::CM * S::LDD +
       2 * S::D * S::LDC) * (int)sizeof(E) + 2 * S::CM * S::D * 4 + 2 * S::CM * 4 + 64;
  // a separate Q-side activation buffer when it fits in LDS
  static constexpr bool Q2 = BYTES + S::CM * S::LDH * (int)sizeof(E) <= 160 * 1024;
};

template <class S>
struct FwdSmem {
  using E = typename S::E;
  static constexpr bool Q2 = FwdSmemBase<S>::Q2;
  alignas(16) E xk[S::CM * S::LDD];
  alignas(16) E xq[S::CM * S::LDD];
  alignas(16) E xv[S::CM * S::LDD];
  alignas(16) E kt[S::D * S::LDC];    // K^T, layout [i][t] (it_idx)
  alignas(16) E alds[S::CM * S::LDH]; // activations A[t][j] (this workgroup's columns)
  alignas(16) E alds2[Q2 ? S::CM * S::LDH : 8]; // Q-side activations (else alds)
  alignas(16) E w2[S::D * S::LDH];    // second-layer weights W2[i][j] (bf16/fp32 copy of W_0)
  alignas(16) E dy[S::CM * S::LDD];   // dY[t][i]
  alignas(16) E dytw[S::D * S::LDC];  // K^W_t dY[t][i], layout [i][t] (it_idx)
  alignas(16) E dytm[S::D * S::LDC];  // K^M_t dY[t][i]
  alignas(16) float y[S::CM * S::D];  // Y_K (partial over this workgroup's columns)
  alignas(16) float yq[S::CM * S::D]; // Y_Q (partial)
  alignas(16) float kw[S::CM];
  alignas(16) float km[S::CM];
  float carry[4];
  int word[2];
};

// Exchange slots of one rank: NPK slots of Y_K (one per parity) and one of
// Y_Q, CM x D floats each.  A slot is rewritten only after every peer has
// finished reading it, by the order of the waits, with one slot of Y_Q: a
// peer reads a rank's Y_Q of tile n in its outputs phase, before it posts its
// Y_K of tile n + 1 (whose post waits for those loads), and the rank writes
// its Y_Q of tile n + 1 only after waiting for that post.  Likewise one slot
// of Y_K where the peers load its rows right after their wait for it (before
// posting their Y_Q of the same tile, which the rank waits for before the next
// Y_K); where the row phases read Y_K from the slots later in the tile (after
// that post), Y_K alternates between two slots.  Fewer slots keep the
// exchange's working set in the XCD's L2.
template <class S, int NPK>
__device__ __forceinline__ float* fwd_slot_k(float* xbuf, long p, int rank, int parity) {
  return xbuf + ((p * S::NS + rank) * (NPK + 1) + (NPK == 2 ? parity : 0)) * (long)S::CM * S::D;
}
template <class S, int NPK>
__device__ __forceinline__ float* fwd_slot_q(float* xbuf, long p, int rank) {
  return xbuf + ((p * S::NS + rank) * (NPK + 1) + NPK) * (long)S::CM * S::D;
}

// LONG: chunks longer than the CM-row tile (a separate instantiation, so that
// the common case keeps W_0's operand copies dead between chunks).
template <class S, bool LONG, bool PN>
__global__ void __launch_bounds__(S::NT, 1) chain_fwd_kernel(ChainArgs a) {
  using O = typename S::O;
  using IO = IoT<S::BF>;
  constexpr int D = S::D, NJB = S::NJB, NTB = S::NTB, NIB = S::NIB, NMAT = S::NMAT;
  constexpr int SEC = NMAT - 1;  // index of the second-layer matrix
  // MLP on the bf16 path: the bf16 high / low parts of W_0 are formed once per
  // chunk (checkpoint, LDS copy of W2, and the K-side, Q-side and dA products
  // share them); the wider SwiGLU state re-forms them per use instead
  constexpr bool PRESPLIT = S::BF && S::FW == 0 && S::D <= 64;
  // fp32 path: the chunk's sum_t K_t G_t accumulates apart from the state and
  // joins it in one addition at the chunk end (one rounding of W and M per
  // chunk instead of one per contraction step); W itself stays W_0 for the
  // whole chunk and is the products' operand, also across a long chunk's tiles
  constexpr bool SEPDELTA = !S::BF;
  // SwiGLU on the bf16 path re-forms W_0's operands at every product.  In a
  // long chunk's later tiles the state has already taken the chunk's first
  // updates, so those products read W_0 back from the fp32 copy (register-tile
  // order, lane-private) that the chunk's first tile leaves in this
  // workgroup's block.
  constexpr bool RELOAD = LONG && S::BF && !PRESPLIT;
  constexpr long NB0 = (long)NMAT * NJB * NIB * S::NT;   // f32x4 per block
  f32x4* const w0blk =
      RELOAD ? reinterpret_cast<f32x4*>(E2TTT_ARG(w0blk)) + (long)blockIdx.x * NB0 : nullptr;
  constexpr int EPL = D / 16;    // head elements per lane in the row phases
  constexpr int RPW = row_share<S>();  // output rows written by one rank (last: fewer)
  constexpr int NPEER = S::NS - 1;
  // the peers' rows of Y_K and Y_Q are loaded right after the waits (so that
  // they arrive under the next contraction) while they are few; with many
  // peers or wide rows that would hold too many registers, and each row
  // phase loads them where it adds them
  constexpr bool PEER_EARLY = NPEER * EPL <= 8 && S::D <= 64;
  constexpr int NPK = PEER_EARLY ? 1 : 2;   // Y_K slots per rank
  __shared__ FwdSmem<S> sm;
  static_assert(sizeof(FwdSmem<S>) <= 160 * 1024, "LDS budget");

  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int T = a.T, C = a.C, NC = a.NC, dh = a.dh;
  const int TPC = LONG ? (C + S::CM - 1) / S::CM : 1;   // tiles per chunk
  const int TL = LONG ? S::CM : C;                       // tokens per tile
  const float inv_d = 1.0f / D;

  PairX<S::NS> px;
  px.init(a.sync, a.npairs, sm.word, a.wait_ticks);
  const int rank = px.rank;
  const int j0 = rank * S::DHP;
  const long NP = (S::NS > 1) ? a.npairs : (long)gridDim.x;
  const int rlo = rank * RPW;
  const int rhi = min(S::CM, rlo + RPW);
  long nch = 0;   // chunks processed by this workgroup (exchange parity)

  // hidden columns [DHP, DHK) of the j-operands stay zero for the whole run
  if constexpr (S::DHK > S::DHP) {
    jq_zero_cols<S, S::LDH, S::DHK>(sm.alds, S::NTB, sm.w2, S::NIB, S::DHP);
    if constexpr (FwdSmem<S>::Q2) jq_zero_cols<S, S::LDH, S::DHK>(sm.alds2, S::NTB, sm.alds2, 0, S::DHP);
  }

  // inputs of the next chunk, loaded one chunk ahead
  TileRegs<S> pk, pq, pv;
  float pkw = 0.0f, pkm = 0.0f, pcar = 0.0f;
  auto prefetch = [&](long uu, int rc, int kt) {
    E2TTT_LANE_IDS;
    const int st = LONG ? rc * C + kt * TL : rc * C;
    const long r0 = uu * T + st;
    const int ln = LONG ? min(TL, min(T, (rc + 1) * C) - st) : min(C, T - st);
    pk.load(E2TTT_ARG(k), r0, ln, tid);
    pq.load(E2TTT_ARG(q), r0, ln, tid);
    pv.load(E2TTT_ARG(v), r0, ln, tid);
    if (tid < S::CM) {
      pkw = (tid < ln) ? E2TTT_ARG(kw)[r0 + tid] : 0.0f;
      pkm = (tid < ln) ? E2TTT_ARG(km)[r0 + tid] : 0.0f;
    }
    if (tid < 3) pcar = E2TTT_ARG(carry)[(uu * NC + rc) * 3 + tid];
  };

  for (long u = px.p; u < a.U; u += NP) {
    StateTiles<S> W, M;
    SplitTiles<S> WS;   // bf16 hi / lo parts of W_0 (PRESPLIT)
    StateTiles<S> XW, XM;   // the chunk's sum_t K_t G_t (SEPDELTA)
    {
      E2TTT_LANE_IDS;
      load_state<S>(W, E2TTT_ARG(w_in) + u * a.P, dh, j0, w, g, c);
      load_state<S>(M, E2TTT_ARG(m_in) ? E2TTT_ARG(m_in) + u * a.P : nullptr, dh, j0, w, g, c);
    }
    prefetch(u, 0, 0);

    // tile kt of chunk r (always kt = 0 unless LONG)
    for (int r = 0, kt = 0; r < NC; ++nch) {
      const int s0 = LONG ? r * C + kt * TL : r * C;
      const int cend = LONG ? min(T, (r + 1) * C) : 0;
      const bool first = !LONG || kt == 0;         // the chunk's first tile
      const int len = LONG ? min(TL, cend - s0) : min(C, T - s0);
      const bool more = LONG && s0 + TL < cend;    // another tile of this chunk follows
      const int rc = r, kc = kt;                   // this tile
      if (more) ++kt; else { ++r; kt = 0; }
      const long row0 = u * T + s0;
      const int par = (int)(nch & 1);
      const unsigned seq0 = px.seq_now();
      // -------------------------------------------------------- stage (a1)
      {
      E2TTT_LANE_IDS;
      pk.store(sm.xk, tid);
      pq.store(sm.xq, tid);
      pv.store(sm.xv, tid);
      if (tid < S::CM) {
        sm.kw[tid] = pkw;
        sm.km[tid] = pkm;
      }
      if (tid < 3) sm.carry[tid] = pcar;
      if (first) {
      if constexpr (PRESPLIT) split_state<S>(WS, W);
      if constexpr (RELOAD) {
        if (more) {
#pragma unroll
          for (int m = 0; m < NMAT; ++m)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
              for (int ib = 0; ib < NIB; ++ib)
                w0blk[((m * NJB + jj) * NIB + ib) * S::NT + tid] = W.t[m][jj][ib];
        }
      }
      if constexpr (SEPDELTA) {
#pragma unroll
        for (int m = 0; m < NMAT; ++m)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
              XW.t[m][jj][ib] = zero4();
              XM.t[m][jj][ib] = zero4();
            }
      }
      if (E2TTT_ARG(ckpt)) {
        char* cb = static_cast<char*>(E2TTT_ARG(ckpt)) +
                   ((u * E2TTT_ARG(ckpt_nc) + rc) * S::NS + rank) * 2 * E2TTT_ARG(ckpt_stride);
        if constexpr (PRESPLIT) store_ckpt_q<S>(WS.hi, cb, w, lane);
        else store_ckpt<S>(W, cb, w, lane);
        store_ckpt<S>(M, cb + E2TTT_ARG(ckpt_stride), w, lane);
      }
      // second-layer weights of W_0 into LDS as the j-contraction operand
#pragma unroll
      for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
          jq_put<S, S::LDH>(sm.w2, ib, g, 16 * (w * NJB + jj) + c,
                            as_quad<S>(PRESPLIT ? WS.hi[SEC][jj][ib] : O::cvt(W.t[SEC][jj][ib])));
      }
      opaque_state<S>(W);
      opaque_state<S>(M);
      }
      __syncthreads();
      if (r < NC) prefetch(u, r, kt);              // the next tile (r, kt advanced above)

      // operand of the chunk's products (W_0: W is not updated before the chunk end
      // on the fp32 path, nor before the transition below on the others)
      StateTiles<S> W0r;   // RELOAD: W_0 tiles of the matrices the next product takes
      auto w0_mats = [&](int m0, int m1) {
        E2TTT_LANE_IDS;
#pragma unroll
        for (int m = 0; m < NMAT; ++m) {
          if (m < m0 || m > m1) continue;
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib)
              W0r.t[m][jj][ib] = first ? W.t[m][jj][ib]
                                       : w0blk[((m * NJB + jj) * NIB + ib) * S::NT + tid];
        }
      };
      const StateTiles<S>& Wop = RELOAD ? W0r : W;

      // ------------------------------------------- K-side forward (a3)
      // act'(H) kept for dH: MLP GELU'(H); SwiGLU (Hu SiLU'(Hg), SiLU(Hg))
      f32x4 H[NTB][NJB];
      f32x4 Hu[NTB][(S::FW == 1) ? NJB : 1];
      typename O::Q AK[NTB][NJB];          // act(H) as operand quads (rows t)
      if constexpr (RELOAD) w0_mats(0, 1);
      {
      E2TTT_LANE_IDS;
      transpose_to_it<S>(sm.kt, sm.xk, tid);
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj) {
          f32x4 acc = zero4(), accu = zero4();
#pragma unroll
          for (int p = 0; p < S::KS_D; ++p) {
            auto af = lds_frag<S::BF>(sm.xk, S::LDD, 16 * tb + c, p * S::KC, g);
            if constexpr (PRESPLIT) acc = mma_split<S>(acc, af, WS.hi[0][jj], WS.lo[0][jj], p);
            else acc = mma_state<S>(acc, af, &Wop.t[0][jj][0], p, 1);
            if constexpr (S::FW == 1) accu = mma_state<S>(accu, af, &Wop.t[1][jj][0], p, 1);
          }
          f32x4 act, d1, d2;
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            if constexpr (S::FW == 0) {
              const Act2 ga = gelu2(acc[rr]);
              act[rr] = ga.f;
              d1[rr] = ga.d1;
            } else {
              const float hg = acc[rr], hu = accu[rr], sg = sigm_f(hg);
              d2[rr] = hg * sg;                              // SiLU(Hg)
              d1[rr] = hu * sg * (1.0f + hg * (1.0f - sg));  // Hu SiLU'(Hg)
              act[rr] = d2[rr] * hu;
            }
          }
          H[tb][jj] = d1;
          if constexpr (S::FW == 1) Hu[tb][jj] = d2;
          AK[tb][jj] = O::cvt(act);
          jq_put<S, S::LDH>(sm.alds, tb, g, 16 * (w * NJB + jj) + c, AK[tb][jj]);
          sched_fence();
        }
      }
      __syncthreads();

      {
        E2TTT_LANE_IDS;
        jgemm_to_lds<S>(sm.alds, sm.w2, sm.y, w, g, c,   // Y_K (partial)
                        (S::NS > 1) ? fwd_slot_k<S, NPK>(E2TTT_ARG(xbuf), px.xs, rank, par) : nullptr);
      }
      px.post();                                          // seq0 + 1: Y_K
      // without a separate Q-side buffer, alds is rewritten below
      if constexpr (!FwdSmem<S>::Q2 && S::NS == 1) __syncthreads();
      typename S::E* const aq = FwdSmem<S>::Q2 ? sm.alds2 : sm.alds;

      // ------------------- Q-side first layer and Y_Q (a7), overlapping the swap
      // (MLP, saving for the backward: A_Q and GELU'(H_Q) of every tile)
      typename O::Q qsa[S::FW == 0 ? NTB : 1][NJB];
      f32x4 qsd[S::FW == 0 ? NTB : 1][NJB];
      if constexpr (RELOAD) w0_mats(0, 1);
      {
      E2TTT_LANE_IDS;
      opaque_state<S>(W);
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj) {
          f32x4 acc = zero4(), accu = zero4();
#pragma unroll
          for (int p = 0; p < S::KS_D; ++p) {
            auto af = lds_frag<S::BF>(sm.xq, S::LDD, 16 * tb + c, p * S::KC, g);
            if constexpr (PRESPLIT) acc = mma_split<S>(acc, af, WS.hi[0][jj], WS.lo[0][jj], p);
            else acc = mma_state<S>(acc, af, &Wop.t[0][jj][0], p, 1);
            if constexpr (S::FW == 1) accu = mma_state<S>(accu, af, &Wop.t[1][jj][0], p, 1);
          }
          f32x4 act, d1;
          if (S::FW == 0 && E2TTT_ARG(asave)) {   // GELU and GELU', saved for the backward
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
              const Act2 ga = gelu2(acc[rr]);
              act[rr] = ga.f;
              d1[rr] = ga.d1;
            }
          } else {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
              if constexpr (S::FW == 0) act[rr] = gelu_f(acc[rr]);
              else act[rr] = silu_f(acc[rr]) * accu[rr];
            }
          }
          const auto aquad = O::cvt(act);
          jq_put<S, S::LDH>(aq, tb, g, 16 * (w * NJB + jj) + c, aquad);
          if constexpr (S::FW == 0) {   // stored after the Y_Q post below
            qsa[tb][jj] = aquad;
            qsd[tb][jj] = d1;
          }
          sched_fence();
        }
      }
      // The peer's Y_K was posted before its Q-side; waiting here (a barrier,
      // which also completes the Q-side activations) lets the loads of its
      // rows for every LN step run under the Y_Q contraction.
      constexpr int NIT = (S::CM + 4 * S::NW - 1) / (4 * S::NW);
      float pyv[S::NS > 1 && PEER_EARLY ? NIT : 1][S::NS > 1 ? NPEER : 1][EPL];
      if constexpr (S::NS > 1) {
        px.wait_for(seq0 + 1, sm.word);                   // peers' Y_K
        E2TTT_LANE_IDS;
#pragma unroll
        for (int k = 0; k < (PEER_EARLY ? NPEER : 0); ++k) {
          const float* peer = fwd_slot_k<S, NPK>(E2TTT_ARG(xbuf), px.xs, other_rank(k, rank), par);
#pragma unroll
          for (int it_ = 0; it_ < NIT; ++it_) {
            const int t0 = 4 * w + it_ * 4 * S::NW;
            if (t0 < S::CM)
              load_row_xchg<EPL>(pyv[it_][k], E2TTT_ARG(xbuf), peer,
                                 (t0 + (lane >> 4)) * D + l16 * EPL);
          }
        }
      } else {
        __syncthreads();
      }
      {
        E2TTT_LANE_IDS;
        jgemm_to_lds<S>(aq, sm.w2, sm.yq, w, g, c,        // Y_Q (partial)
                        (S::NS > 1) ? fwd_slot_q<S, NPK>(E2TTT_ARG(xbuf), px.xs, rank) : nullptr);
      }
      px.post();                                          // seq0 + 2: Y_Q
      // the saved query side goes out after the post, so that the post's wait
      // for this chunk's stores does not include it
      if (S::FW == 0 && E2TTT_ARG(asave)) {
        E2TTT_LANE_IDS;
        const SavedAct<S> sv(static_cast<char*>(E2TTT_ARG(asave)) +
                             (((u * NC + rc) * TPC + kc) * S::NS + rank) * E2TTT_ARG(as_stride));
#pragma unroll
        for (int tb = 0; tb < (S::FW == 0 ? NTB : 0); ++tb)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            const int qi = SavedAct<S>::idx(tb, jj, w, lane);
            st_stream(sv.aq() + qi, qsa[tb][jj]);
            st_stream(sv.d1q() + qi, DerivQ<S::BF>::pack(qsd[tb][jj]));
          }
      }

      // ------------------------------- LN and activation gradients (a4)
      // Four token rows per wave step: lanes 16 r .. 16 r + 15 hold row t0 + r,
      // EPL consecutive head elements each; row sums are 16-lane DPP reductions.
      const float cw = sm.carry[0], cm = sm.carry[1], cbv = sm.carry[2];
      {
        E2TTT_LANE_IDS;
        // this lane's rows of the rows [rlo, rhi), kept for the backward,
        // are written after the loop, so that no global store sits between
        // the peer's rows and their use
        float zsave[NIT][EPL], rsave[NIT];
        bool keep[NIT];
#pragma unroll
        for (int it_ = 0; it_ < NIT; ++it_) {
          const int t0 = 4 * w + it_ * 4 * S::NW;
          if (t0 < S::CM) {
          const int t = t0 + (lane >> 4);
          float yv[EPL], e[EPL], z[EPL], dyv[EPL];
          float s1 = 0.0f, sig = 1.0f;
#pragma unroll
          for (int q = 0; q < EPL; ++q) yv[q] = sm.y[t * D + l16 * EPL + q];
          if constexpr (S::NS > 1 && PEER_EARLY) {
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              float pv[NPEER];
#pragma unroll
              for (int k = 0; k < NPEER; ++k) pv[k] = pyv[it_][k][q];
              yv[q] = sum_ranks<S::NS>(yv[q], pv, rank);
            }
          } else if constexpr (S::NS > 1) {
            // every rank's partial from its slot (this rank's too), added in
            // rank order as sum_ranks does: the same sum on every rank
#pragma unroll
            for (int r = 0; r < S::NS; ++r) {
              float pr[EPL];
              load_row_xchg<EPL>(pr, E2TTT_ARG(xbuf),
                                 fwd_slot_k<S, NPK>(E2TTT_ARG(xbuf), px.xs, r, par),
                                 t * D + l16 * EPL);
#pragma unroll
              for (int q = 0; q < EPL; ++q) yv[q] = (r == 0) ? pr[q] : yv[q] + pr[q];
            }
          }
#pragma unroll
          for (int q = 0; q < EPL; ++q) s1 += yv[q];
          if (E2TTT_ARG(resln)) {
            const float mu = group16_sum(s1) * inv_d;
            float s2 = 0.0f;
#pragma unroll
            for (int q = 0; q < EPL; ++q) { yv[q] -= mu; s2 += yv[q] * yv[q]; }
            sig = rsq_f(group16_sum(s2) * inv_d + E2TTT_ARG(eps));   // 1 / sigma
            float se = 0.0f, sez = 0.0f;
            if (E2TTT_ARG(ln_a)) {
              // f = k + a z + b: the LayerNorm backward takes a (v - f)
              float la[EPL], lb[EPL];
              const long ho = (u % E2TTT_ARG(H)) * D + l16 * EPL;
              load_row_part<EPL>(la, E2TTT_ARG(ln_a) + ho);
              load_row_part<EPL>(lb, E2TTT_ARG(ln_b) + ho);
#pragma unroll
              for (int q = 0; q < EPL; ++q) {
                const int i = l16 * EPL + q;
                z[q] = yv[q] * sig;
                const float r = O::from_e(sm.xv[t * S::LDD + i]) - O::from_e(sm.xk[t * S::LDD + i]);
                e[q] = la[q] * (r - fmaf(la[q], z[q], lb[q]));
                se += e[q];
                sez += e[q] * z[q];
              }
            } else {
#pragma unroll
              for (int q = 0; q < EPL; ++q) {
                const int i = l16 * EPL + q;
                z[q] = yv[q] * sig;
                e[q] = O::from_e(sm.xv[t * S::LDD + i]) - O::from_e(sm.xk[t * S::LDD + i]) - z[q];
                se += e[q];
                sez += e[q] * z[q];
              }
            }
            const float me = group16_sum(se) * inv_d, mez = group16_sum(sez) * inv_d;
#pragma unroll
            for (int q = 0; q < EPL; ++q) dyv[q] = (e[q] - me - z[q] * mez) * sig;
          } else {
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              z[q] = yv[q];
              dyv[q] = O::from_e(sm.xv[t * S::LDD + l16 * EPL + q]) - yv[q];
            }
          }
          keep[it_] = t >= rlo && t < rhi && t < len;
#pragma unroll
          for (int q = 0; q < EPL; ++q) zsave[it_][q] = z[q];
          rsave[it_] = sig;
          const float kwt = sm.kw[t], kmt = sm.km[t];
          store_row_ti<S, EPL>(sm.dy, S::LDD, t, l16 * EPL, dyv);
          store_row_it<S, EPL>(sm.dytw, t, l16 * EPL, dyv, kwt);
          store_row_it<S, EPL>(sm.dytm, t, l16 * EPL, dyv, kmt);
                  }
        }
        if (E2TTT_ARG(zk)) {
#pragma unroll
          for (int it_ = 0; it_ < NIT; ++it_) {
            const int t = 4 * w + it_ * 4 * S::NW + (lane >> 4);
            if (t < S::CM && keep[it_]) {
              // (SwiGLU, at the register limit, keeps element stores: with the
              // vector store the three-workgroup variant spilled 57 VGPRs)
              if constexpr (S::FW == 0) {
                store_row_io<IoT<false>, EPL>(E2TTT_ARG(zk) + (row0 + t) * D + l16 * EPL,
                                              zsave[it_]);
              } else {
#pragma unroll
                for (int q = 0; q < EPL; ++q)
                  st_stream(E2TTT_ARG(zk) + (row0 + t) * D + l16 * EPL + q, zsave[it_][q]);
              }
              if (l16 == 0) st_stream(E2TTT_ARG(rk) + row0 + t, rsave[it_]);
            }
          }
        }
      }
      // The peer's Y_Q was posted before its LN phase: wait for it here (the
      // barrier that ends the LN phase) and load its rows of the outputs, so
      // that they arrive under dA and the state update.
      constexpr int NITO = (RPW + 4 * S::NW - 1) / (4 * S::NW);
      float pyq[S::NS > 1 && PEER_EARLY ? NITO : 1][S::NS > 1 ? NPEER : 1][EPL];
      if constexpr (S::NS > 1) {
        px.wait_for(seq0 + 2, sm.word);                   // peers' Y_Q
        E2TTT_LANE_IDS;
#pragma unroll
        for (int k = 0; k < (PEER_EARLY ? NPEER : 0); ++k) {
          const float* peer = fwd_slot_q<S, NPK>(E2TTT_ARG(xbuf), px.xs, other_rank(k, rank));
#pragma unroll
          for (int it_ = 0; it_ < NITO; ++it_) {
            const int t0 = rlo + 4 * w + it_ * 4 * S::NW;
            if (t0 < rhi)
              load_row_xchg<EPL>(pyq[it_][k], E2TTT_ARG(xbuf), peer,
                                 (t0 + (lane >> 4)) * D + l16 * EPL);
          }
        }
      } else {
        __syncthreads();
      }

      // ---------------------------------- dA = dY W2, first-layer deltas (a4)
      opaque_state<S>(W);
      if constexpr (RELOAD) w0_mats(SEC, SEC);
      // first-layer update operands K^W_t dH[t][j] and K^M_t dH[t][j] (the scalar
      // kernels go on dH, so that the other operand is K^T, exact in bf16); for
      // the MLP on the bf16 path they are split into bf16 high and low parts
      constexpr bool SPLIT_UPD = S::BF && S::FW == 0;
      constexpr int NU = (S::FW == 1) ? 2 : 1;            // first-layer matrices
      typename O::Q DW[NU][NTB][NJB], DM[NU][NTB][NJB];
      typename O::Q DWl[SPLIT_UPD ? NU : 1][NTB][NJB], DMl[SPLIT_UPD ? NU : 1][NTB][NJB];
      {
      E2TTT_LANE_IDS;
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj) {
          f32x4 da = zero4();
#pragma unroll
          for (int p = 0; p < S::KS_D; ++p) {
            auto af = lds_frag<S::BF>(sm.dy, S::LDD, 16 * tb + c, p * S::KC, g);
            if constexpr (PRESPLIT) da = mma_split<S>(da, af, WS.hi[SEC][jj], WS.lo[SEC][jj], p);
            else da = mma_state<S>(da, af, &Wop.t[SEC][jj][0], p, 1);
          }
          f32x4 dh[NU];
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            dh[0][rr] = da[rr] * H[tb][jj][rr];
            if constexpr (S::FW == 1) dh[1][rr] = da[rr] * Hu[tb][jj][rr];
          }
          const f32x4 kwv = *reinterpret_cast<const f32x4*>(&sm.kw[16 * tb + 4 * g]);
          const f32x4 kmv = *reinterpret_cast<const f32x4*>(&sm.km[16 * tb + 4 * g]);
#pragma unroll
          for (int m = 0; m < NU; ++m) {
            const f32x4 vw = kwv * dh[m], vm = kmv * dh[m];
            DW[m][tb][jj] = O::cvt(vw);
            DM[m][tb][jj] = O::cvt(vm);
            if constexpr (SPLIT_UPD) {
              DWl[m][tb][jj] = O::cvt(vw - quad_f32(DW[m][tb][jj]));
              DMl[m][tb][jj] = O::cvt(vm - quad_f32(DM[m][tb][jj]));
            }
          }
          sched_fence();
        }
      }

      // ------------------- closed-form transition (a5, a6): scale, then accumulate
      StateTiles<S>& AW = SEPDELTA ? XW : W;   // accumulation targets
      StateTiles<S>& AM = SEPDELTA ? XM : M;
      if (!SEPDELTA && first) {
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
          for (int ib = 0; ib < NIB; ++ib) {
            W.t[m][jj][ib] = cw * W.t[m][jj][ib] + cm * M.t[m][jj][ib];
            M.t[m][jj][ib] = cbv * M.t[m][jj][ib];
          }
      }
      {
      E2TTT_LANE_IDS;
#pragma unroll
      for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
          for (int p = 0; p < S::KS_C; ++p) {
            typename O::Frag bA;
#pragma unroll
            for (int h = 0; h < S::NH; ++h) bA.h[h] = AK[S::NH * p + h][jj];
            const int row = 16 * ib + c, k0 = p * S::KC;
            // second layer: sum_t K_t dY[t][i] A[t][j]
            AW.t[SEC][jj][ib] = O::mma(AW.t[SEC][jj][ib], it_frag<S>(sm.dytw, row, k0, g), bA);
            AM.t[SEC][jj][ib] = O::mma(AM.t[SEC][jj][ib], it_frag<S>(sm.dytm, row, k0, g), bA);
            // first layer(s): sum_t k[t][i] (K_t dH[t][j])
            auto kf = it_frag<S>(sm.kt, row, k0, g);
#pragma unroll
            for (int m = 0; m < NU; ++m) {
              typename O::Frag bw, bm;
#pragma unroll
              for (int h = 0; h < S::NH; ++h) {
                bw.h[h] = DW[m][S::NH * p + h][jj];
                bm.h[h] = DM[m][S::NH * p + h][jj];
              }
              AW.t[m][jj][ib] = O::mma(AW.t[m][jj][ib], kf, bw);
              AM.t[m][jj][ib] = O::mma(AM.t[m][jj][ib], kf, bm);
              if constexpr (SPLIT_UPD) {
#pragma unroll
                for (int h = 0; h < S::NH; ++h) {
                  bw.h[h] = DWl[m][S::NH * p + h][jj];
                  bm.h[h] = DMl[m][S::NH * p + h][jj];
                }
                AW.t[m][jj][ib] = O::mma(AW.t[m][jj][ib], kf, bw);
                AM.t[m][jj][ib] = O::mma(AM.t[m][jj][ib], kf, bm);
              }
            }
          }
      }
      if (SEPDELTA && !more) {   // chunk end: W_C = cw W_0 + cm M_0 + dW, M_C = cb M_0 + dM
#pragma unroll
        for (int m = 0; m < NMAT; ++m)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
              W.t[m][jj][ib] = (cw * W.t[m][jj][ib] + cm * M.t[m][jj][ib]) + XW.t[m][jj][ib];
              M.t[m][jj][ib] = cbv * M.t[m][jj][ib] + XM.t[m][jj][ib];
            }
      }

      // ------------- post-chunk normalisation of the fast-weight rows (chunk end)
      if (PN && !more) {
        E2TTT_LANE_IDS;
        constexpr int NF = NMAT - 1;
        const long R = (long)NF * dh + D;
        const float* tg = E2TTT_ARG(norm_tgt) + u * R;
        float* npre = E2TTT_ARG(norm_pre) ? E2TTT_ARG(norm_pre) + (u * NC + rc) * R : nullptr;
        // first-layer rows: hidden unit j's d weights are the tile column of
        // lanes c, c + 16, c + 32, c + 48
#pragma unroll
        for (int m = 0; m < NF; ++m)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            float s2 = 0.0f;
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
              for (int r = 0; r < 4; ++r) s2 = fmaf(W.t[m][jj][ib][r], W.t[m][jj][ib][r], s2);
            s2 += __shfl_xor(s2, 16);
            s2 += __shfl_xor(s2, 32);
            const int j = j0 + 16 * (w * NJB + jj) + c;
            const float sc = (j < dh && s2 > 0.0f) ? tg[(long)m * dh + j] * rsq_f(s2) : 1.0f;
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) W.t[m][jj][ib] *= sc;
            if (npre && g == 0 && j < dh) npre[(long)m * dh + j] = __builtin_sqrtf(s2);
          }
        // second-layer rows: output i's dh weights span the lanes, the waves and
        // the ranks; partial sums through LDS (the Y_K buffer, free here) and,
        // between ranks, the exchange, added in rank order on every rank
        static_assert(S::CM >= S::NW + 1, "LDS room for the row sums");
        float* part = sm.y;   // [NW][D] wave partials, then [D] scales
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float s2 = 0.0f;
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
              s2 = fmaf(W.t[SEC][jj][ib][r], W.t[SEC][jj][ib][r], s2);
            s2 = group16_sum(s2);
            if (c == 0) part[w * D + 16 * ib + 4 * g + r] = s2;
          }
        __syncthreads();
        float tot = 0.0f;
        if (tid < D)
          for (int ww = 0; ww < S::NW; ++ww) tot += part[ww * D + tid];
        if constexpr (S::NS > 1) {
          float* nx = E2TTT_ARG(nxbuf);
          if (tid < D) nx[((px.xs * S::NS + rank) * 2 + par) * D + tid] = tot;
          px.post();
          px.wait_for(px.seq_now(), sm.word);
          if (tid < D) {
            tot = 0.0f;
            for (int rr = 0; rr < S::NS; ++rr)
              tot += ld_xchg(nx, nx + ((px.xs * S::NS + rr) * 2 + par) * D, tid);
          }
        }
        if (tid < D) {
          part[S::NW * D + tid] = tot > 0.0f ? tg[(long)NF * dh + tid] * rsq_f(tot) : 1.0f;
          if (npre && rank == 0) npre[(long)NF * dh + tid] = __builtin_sqrtf(tot);
        }
        __syncthreads();
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float sc = part[S::NW * D + 16 * ib + 4 * g + r];
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj) W.t[SEC][jj][ib][r] *= sc;
          }
      }

      // ------------------------------------------------- outputs (a7)
      {
        E2TTT_LANE_IDS;
        using IOT = typename IO::T;
        IOT* outp = reinterpret_cast<IOT*>(E2TTT_ARG(out)) + row0 * D;
#pragma unroll
        for (int it_ = 0; it_ < NITO; ++it_) {
          const int t0 = rlo + 4 * w + it_ * 4 * S::NW;
          if (t0 < rhi) {
          const int t = t0 + (lane >> 4);
          float yv[EPL], f[EPL];
          float s1 = 0.0f, sig = 1.0f;
#pragma unroll
          for (int q = 0; q < EPL; ++q) yv[q] = sm.yq[t * D + l16 * EPL + q];
          if constexpr (S::NS > 1 && PEER_EARLY) {
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              float pv[NPEER];
#pragma unroll
              for (int k = 0; k < NPEER; ++k) pv[k] = pyq[it_][k][q];
              yv[q] = sum_ranks<S::NS>(yv[q], pv, rank);
            }
          } else if constexpr (S::NS > 1) {
            // every rank's partial from its slot (this rank's too), added in
            // rank order as sum_ranks does: the same sum on every rank
#pragma unroll
            for (int r = 0; r < S::NS; ++r) {
              float pr[EPL];
              load_row_xchg<EPL>(pr, E2TTT_ARG(xbuf), fwd_slot_q<S, NPK>(E2TTT_ARG(xbuf), px.xs, r),
                                 t * D + l16 * EPL);
#pragma unroll
              for (int q = 0; q < EPL; ++q) yv[q] = (r == 0) ? pr[q] : yv[q] + pr[q];
            }
          }
#pragma unroll
          for (int q = 0; q < EPL; ++q) s1 += yv[q];
          if (E2TTT_ARG(resln)) {
            const float mu = group16_sum(s1) * inv_d;
            float s2 = 0.0f;
#pragma unroll
            for (int q = 0; q < EPL; ++q) { yv[q] -= mu; s2 += yv[q] * yv[q]; }
            sig = rsq_f(group16_sum(s2) * inv_d + E2TTT_ARG(eps));   // 1 / sigma
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              yv[q] *= sig;                                 // Z_Q
              f[q] = O::from_e(sm.xq[t * S::LDD + l16 * EPL + q]) + yv[q];
            }
            if (E2TTT_ARG(ln_a)) {                          // f = q + a Z_Q + b
              float la[EPL], lb[EPL];
              const long ho = (u % E2TTT_ARG(H)) * D + l16 * EPL;
              load_row_part<EPL>(la, E2TTT_ARG(ln_a) + ho);
              load_row_part<EPL>(lb, E2TTT_ARG(ln_b) + ho);
#pragma unroll
              for (int q = 0; q < EPL; ++q)
                f[q] = O::from_e(sm.xq[t * S::LDD + l16 * EPL + q]) + fmaf(la[q], yv[q], lb[q]);
            }
          } else {
#pragma unroll
            for (int q = 0; q < EPL; ++q) f[q] = yv[q];
          }
          if (t < len) {
            store_row_io<IO, EPL>(outp + (long)t * D + l16 * EPL, f);
            if (E2TTT_ARG(zq)) {
              store_row_io<IoT<false>, EPL>(E2TTT_ARG(zq) + (row0 + t) * D + l16 * EPL, yv);
              if (l16 == 0) st_stream(E2TTT_ARG(rq) + row0 + t, sig);
            }
          }
                  }
        }
      }
      __syncthreads();
    }

    {
      E2TTT_LANE_IDS;
      // with the normalisation the backward also needs the final (normalised)
      // weights: one more checkpoint block, W only
      if (PN && E2TTT_ARG(ckpt))
        store_ckpt<S>(W, static_cast<char*>(E2TTT_ARG(ckpt)) +
                             ((u * E2TTT_ARG(ckpt_nc) + NC) * S::NS + rank) * 2 *
                                 E2TTT_ARG(ckpt_stride), w, lane);
      store_state<S>(W, E2TTT_ARG(w_out) + u * a.P, dh, j0, w, g, c);
      store_state<S>(M, E2TTT_ARG(m_out) + u * a.P, dh, j0, w, g, c);
    }
  }
}

template <class S, bool LONG, bool PN>
int occupancy() {
  int v = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, chain_fwd_kernel<S, LONG, PN>, S::NT, 0) !=
      hipSuccess)
    v = 0;
  return v;
}

template <class S>
int max_blocks_per_cu() {
  static int nb = [] {
    // one launch geometry serves both chunk-length instantiations
    constexpr bool PN = E2TTT_CHAIN_PN;
    return std::min(occupancy<S, false, PN>(), occupancy<S, true, PN>());
  }();
  return nb;
}

template <class S, bool LONG, bool PN>
hipError_t launch_as(const ChainArgs& a, hipStream_t stream) {
  if constexpr (S::NS == 1) {
    hipLaunchKernelGGL((chain_fwd_kernel<S, LONG, PN>), dim3((unsigned)a.U), dim3(S::NT), 0, stream,
                       a);
    return hipGetLastError();
  } else {
    ChainArgs b = a;
    void* args[] = {&b};
    return hipLaunchCooperativeKernel((const void*)chain_fwd_kernel<S, LONG, PN>,
                                      dim3((unsigned)(S::NS * a.npairs)), dim3(S::NT), args, 0,
                                      stream);
  }
}

template <class S>
hipError_t launch(const ChainArgs& a, hipStream_t stream) {
  // the post-chunk normalisation is a separate instantiation, so that the
  // kernels without it carry none of its registers
  constexpr bool PN = E2TTT_CHAIN_PN;
  if ((a.norm_tgt != nullptr) != PN) return hipErrorInvalidValue;
  if (a.C <= S::CM) return launch_as<S, false, PN>(a, stream);
  // a long chunk whose products re-form W_0 from the state needs the W_0 blocks
  if (S::BF && (S::FW == 1 || S::D > 64) && !a.w0blk) return hipErrorInvalidValue;
  return launch_as<S, true, PN>(a, stream);
}

}  // namespace

#define E2TTT_CASE(FW, D, NW, NJB, NTB, BF, NS)                                          \
  if (cfg.fw == FW && cfg.d == D && cfg.nw == NW && cfg.njb == NJB && cfg.ntb == NTB && \
      cfg.bf == BF && cfg.ns == NS)                                                     \
    return launch<Shape<FW, D, NW, NJB, NTB, BF, NS>>(a, stream);

hipError_t E2TTT_PN_NAME(launch_chain_fwd)(const ChainConfig& cfg, const ChainArgs& a,
                                      hipStream_t stream) {
#if !E2TTT_CHAIN_PN
  if (cfg.pn) return launch_chain_fwd_pn(cfg, a, stream);
#endif
#include "chain_variants.inc"
  return hipErrorInvalidValue;
}
#undef E2TTT_CASE

#define E2TTT_CASE(FW, D, NW, NJB, NTB, BF, NS)                                          \
  if (cfg.fw == FW && cfg.d == D && cfg.nw == NW && cfg.njb == NJB && cfg.ntb == NTB && \
      cfg.bf == BF && cfg.ns == NS)                                                     \
    return max_blocks_per_cu<Shape<FW, D, NW, NJB, NTB, BF, NS>>();

int E2TTT_PN_NAME(chain_fwd_blocks_per_cu)(const ChainConfig& cfg) {
#if !E2TTT_CHAIN_PN
  if (cfg.pn) return chain_fwd_blocks_per_cu_pn(cfg);
#endif
#include "chain_variants.inc"
  return 0;
}
#undef E2TTT_CASE

#if !E2TTT_CHAIN_PN
long chain_ckpt_bytes(const ChainConfig& cfg) {
  const long nmat = (cfg.fw == 0) ? 2 : 3;
  return nmat * 16L * cfg.nw * cfg.njb * cfg.d * (cfg.bf ? 2 : 4);
}

long chain_saved_act_bytes(const ChainConfig& cfg) {
  if (cfg.fw != 0) return 0;
  // SavedAct: an operand quad (A_Q) and a derivative quad per lane and tile,
  // 8 bytes each on the bf16 path (bf16, fp16), 16 on the fp32 path
  return (long)cfg.ntb * cfg.njb * cfg.nw * 64 * (cfg.bf ? 2 * 8 : 2 * 16);
}

#endif  // !E2TTT_CHAIN_PN

}  // namespace e2ttt
