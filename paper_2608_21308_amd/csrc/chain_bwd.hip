// Backward chain kernel: reverse mode through Algorithm 1, one workgroup per
// (batch, head) unit, chunks in reverse order.
//
// The adjoint state (Wb, Mb) = (dL/dW_C, dL/dM_C) of the current chunk lives in
// MFMA accumulator tiles (same layout as the forward state).  For a chunk with
// start state (W_0, M_0) (read back from the forward's checkpoints), scalar
// kernels K^W, K^M and carries (cw, cm, cb):
//   W_C = cw W_0 + cm M_0 + sum_t K^W_t G_t,   M_C = cb M_0 + sum_t K^M_t G_t,
//   o_t = f_{W_0}(q_t),   G_t = G(W_0, k_t, v_t) = -grad_W 1/2||f_{W_0}(k_t) - v_t||^2,
// the adjoints are
//   dK^W_t = <Wb, G_t>, dK^M_t = <Mb, G_t>, dcw = <Wb, W_0>, dcm = <Wb, M_0>, dcb = <Mb, M_0>
//   dM_0 = cm Wb + cb Mb
//   dW_0 = cw Wb + d/dW_0 sum_t <Gb_t, G_t> + d/dW_0 sum_t <do_t, o_t>,  Gb_t = K^W_t Wb + K^M_t Mb
// and d/dk_t, d/dv_t, d/dq_t follow from the same two terms.  The terms
// through G_t are second order (Hessian-vector products); they are formed by
// differentiating the first-order gradient graph once more:
//   G_t = (dH_t k_t^T, dY_t a_t^T) with dY = LN backward of e = v - f, dA = dY W2,
//   dH = dA * act'(H); with p = Gb1 k (over i), p2 = Gb2 a (over j), r1 = Gb1^T dH
//   (over j), r2 = Gb2^T dY (over i), the reverse pass through
//   dH -> dA -> dY -> (e, Z, sigma) -> Y -> A -> H -> (W_0, k) gives
//   Wb2 += dY^T dAh + Yh^T A,  Wb1 += K^T Hh,  dk = r1 - eh + Hh W1,  dv = eh,
//   dAh = p act'(H), Hh = p dA act''(H) + (r2 + Yh W2) act'(H),
//   eh = LNb(dYh),  dYh = p2 + dAh W2^T,  Yh = LNb(zh) + sigh Z / d,
//   zh = -(dYh mean(eZ) + e mean(dYh Z))/sigma - eh,  sigh = -sum(dYh dY)/sigma,
// where LNb(x) = (x - mean x - Z mean(x Z)) / sigma (per token, over the head dim).
// SwiGLU and the bare net (no residual LN) follow the same pattern.
#include <algorithm>

#include "chain_common.h"
#include "pair_xchg.h"

// The instantiations with the post-chunk normalisation of the fast weights are
// compiled in a translation unit of their own (chain_bwd_pn.hip defines this
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
struct BwdLayout {
  using E = typename S::E;
  static constexpr int JH = (S::DHK > 128) ? 2 : 1;     // hidden halves per j-round
  static constexpr int JWD = S::DHK / JH;                // hidden width of one half
  static constexpr int LDJ = JWD + S::O::PAD;
  static_assert(!S::BF || LDJ % 16 == 4, "bf16 j-round quad rows 4 (mod 16) quads apart");
  static_assert(JWD % S::KC == 0, "half width must be a multiple of the K-step");
  static_assert(JWD % (16 * S::NJB) == 0, "a wave's hidden slice must lie in one half");
  static constexpr int TD = S::CM * S::LDD * (int)sizeof(E);   // [t][i]
  static constexpr int DT = S::D * S::LDC * (int)sizeof(E);    // [i][t] (it_idx)
  static constexpr int TDX = (TD > DT) ? TD : DT;
  static constexpr int TJ = S::CM * LDJ * (int)sizeof(E);      // [t][j] half
  static constexpr int IJ = S::D * LDJ * (int)sizeof(E);       // [i][j] half
  static constexpr int F = S::CM * S::D * 4;                   // fp32 [t][i]
  static constexpr int R1 = (2 * TDX > F) ? 2 * TDX : F;
  static constexpr int A16(int x) { return (x + 15) / 16 * 16; }
  // region offsets (bytes)
  static constexpr int XK = 0;                   // K [t][i]            | out branch: Q [t][i]
  static constexpr int JW = A16(XK + TD);        // j-round weight half [i][j]
  static constexpr int JA = A16(JW + IJ);        // j-round activation half [t][j]
  static constexpr int YK = A16(JA + TJ);        // fp32 Y -> Z          | out branch: Y_Q
  static constexpr int EK = A16(YK + F);         // fp32 E -> eh
  static constexpr int RR = A16(EK + F);         // V | dY (t,i) ; dYh fp32 ; K^T ; dO
  static constexpr int DYT = A16(RR + R1);       // dY^T [i][t]          | out branch: Yb_Q^T
  static constexpr int YH = A16(DYT + DT);       // Yh [t][i]            | out branch: Yb_Q
  static constexpr int YHT = A16(YH + TD);       // Yh^T [i][t]          | out branch: Q^T
  static constexpr int ROW = A16(YHT + DT);       // per token: 1/sigma, mean(e Z)
  // Until P7 writes Yh, the Yh / Yh^T regions are free: a second j-round
  // weight buffer there lets two j-rounds over the same activations share
  // one pass (jround2)
  static constexpr int JW2 = YH;
  static constexpr bool J2 = (JH == 1) && (ROW - YH >= IJ);
  static constexpr int KB = A16(ROW + S::CM * 8);          // dK^W, dK^M partials [2][NW][CM]
  static constexpr int CB = A16(KB + 2 * S::NW * S::CM * 4);  // carry adjoint partials [NW][4]
  static constexpr int SC = A16(CB + S::NW * 16);          // kw[CM], km[CM], carry[4]
  static constexpr int BASE = A16(SC + (2 * S::CM + 4) * 4);
  // Hh of P4 (completed in P8) kept in LDS when it fits: one float4 per lane
  // per token block and first-layer matrix (lane-private, conflict-free)
  static constexpr int HHB = (S::FW == 0 ? 1 : 2) * S::NTB * S::NW * 64 * 16;
  static constexpr bool HH_LDS = BASE + HHB <= 160 * 1024;
  static constexpr int HHR = BASE;
  static constexpr int TOTAL = HH_LDS ? BASE + HHB : BASE;
  static_assert(TOTAL <= 160 * 1024, "LDS budget of the backward chain kernel");
  // j-round output items per wave: (token block, head block pair) items
  static constexpr int NITEM = S::NTB * (S::NIB / S::IBB);
  static constexpr int JIT = (NITEM + S::NW - 1) / S::NW;
};

template <class S>
struct JAcc {
  f32x4 v[BwdLayout<S>::JIT][S::IBB];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int a = 0; a < BwdLayout<S>::JIT; ++a)
#pragma unroll
      for (int b = 0; b < S::IBB; ++b) v[a][b] = zero4();
  }
};

// j-round: out[t][i] (+)= rowscale[t] * sum_j Act[t][j] Wt[i][j] over the full
// hidden range.  Act and Wt are register tiles of every wave: act(tb, jj) is
// the tile (rows t, column j) and wt(ib, jj) the tile (rows i, column j).
// Both are written to the half-width LDS buffers one half at a time.  With a
// single half (JH == 1) and WRITE_ACT false, ja already holds Act (written by
// the caller or by the previous j-round) and only Wt is written.
template <class S, bool WRITE_ACT = true, class FA, class FWT>
__device__ __forceinline__ void jround(JAcc<S>& out, const float* rowscale, typename S::E* ja,
                                       typename S::E* jw, FA act, FWT wt, int w, int g, int c) {
  using L = BwdLayout<S>;
  using O = typename S::O;
  constexpr int NI = S::NIB / S::IBB;
  JAcc<S> tmp;
  tmp.zero();
#pragma unroll
  for (int half = 0; half < L::JH; ++half) {
    // columns of this half beyond the padded hidden width belong to no wave;
    // they may hold the previous half's values and must read as zero
    const int validw = S::DHP - half * L::JWD;
    if (validw < L::JWD) jq_zero_cols<S, L::LDJ, L::JWD>(ja, S::NTB, jw, S::NIB, validw);
    const int col0 = 16 * w * S::NJB - half * L::JWD;   // this wave's first column in the half
    if (col0 >= 0 && col0 < L::JWD) {
#pragma unroll
      for (int jj = 0; jj < S::NJB; ++jj) {
        const int col = col0 + 16 * jj + c;
        if (WRITE_ACT || L::JH > 1) {
#pragma unroll
          for (int tb = 0; tb < S::NTB; ++tb) jq_put<S, L::LDJ>(ja, tb, g, col, as_quad<S>(act(tb, jj)));
        }
#pragma unroll
        for (int ib = 0; ib < S::NIB; ++ib) jq_put<S, L::LDJ>(jw, ib, g, col, as_quad<S>(wt(ib, jj)));
      }
    }
    __syncthreads();
#pragma unroll
    for (int a = 0; a < L::JIT; ++a) {
      const int it = w + a * S::NW;
      if (it < L::NITEM) {
        const int tb = it / NI, ib0 = (it % NI) * S::IBB;
        const typename S::E* pa = jq_lane<S, L::LDJ>(ja, tb, g, c);
        const typename S::E* pb[S::IBB];
#pragma unroll
        for (int b = 0; b < S::IBB; ++b) pb[b] = jq_lane<S, L::LDJ>(jw, ib0 + b, g, c);
#pragma unroll
        for (int p = 0; p < L::JWD / S::KC; ++p) {
          auto af = jq_frag<S>(pa, p * S::KC);
#pragma unroll
          for (int b = 0; b < S::IBB; ++b) {
            auto bf = jq_frag<S>(pb[b], p * S::KC);
            tmp.v[a][b] = O::mma(tmp.v[a][b], af, bf);
          }
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI;
#pragma unroll
      for (int b = 0; b < S::IBB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float s = rowscale ? rowscale[16 * tb + 4 * g + r] : 1.0f;
          out.v[a][b][r] += s * tmp.v[a][b][r];
        }
    }
  }
}

// Two j-rounds over the same activations in one pass (single hidden half):
// out[t][i] += rs1[t] sum_j Act[t][j] Wt1[i][j] + rs2[t] sum_j Act[t][j] Wt2[i][j].
// jw2 is a second weight buffer; WRITE_ACT as for jround.
template <class S, bool WRITE_ACT, class FA, class FW1, class FW2>
__device__ __forceinline__ void jround2(JAcc<S>& out, const float* rs1, const float* rs2,
                                        typename S::E* ja, typename S::E* jw, typename S::E* jw2,
                                        FA act, FW1 wt1, FW2 wt2, int w, int g, int c) {
  using L = BwdLayout<S>;
  using O = typename S::O;
  static_assert(L::JH == 1, "jround2 needs a single hidden half");
  constexpr int NI = S::NIB / S::IBB;
  JAcc<S> t1, t2;
  t1.zero();
  t2.zero();
  // padding columns beyond the hidden width read as zero
  constexpr int NZ = L::JWD - S::DHP;
  if constexpr (NZ > 0) {
    jq_zero_cols<S, L::LDJ, L::JWD>(ja, S::NTB, jw, S::NIB, S::DHP);
    jq_zero_cols<S, L::LDJ, L::JWD>(jw2, 0, jw2, S::NIB, S::DHP);
  }
#pragma unroll
  for (int jj = 0; jj < S::NJB; ++jj) {
    const int col = 16 * (w * S::NJB + jj) + c;
    if constexpr (WRITE_ACT) {
#pragma unroll
      for (int tb = 0; tb < S::NTB; ++tb) jq_put<S, L::LDJ>(ja, tb, g, col, as_quad<S>(act(tb, jj)));
    }
#pragma unroll
    for (int ib = 0; ib < S::NIB; ++ib) {
      jq_put<S, L::LDJ>(jw, ib, g, col, as_quad<S>(wt1(ib, jj)));
      jq_put<S, L::LDJ>(jw2, ib, g, col, as_quad<S>(wt2(ib, jj)));
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI, ib0 = (it % NI) * S::IBB;
      const typename S::E* pa = jq_lane<S, L::LDJ>(ja, tb, g, c);
      const typename S::E* pb1[S::IBB];
      const typename S::E* pb2[S::IBB];
#pragma unroll
      for (int b = 0; b < S::IBB; ++b) {
        pb1[b] = jq_lane<S, L::LDJ>(jw, ib0 + b, g, c);
        pb2[b] = jq_lane<S, L::LDJ>(jw2, ib0 + b, g, c);
      }
#pragma unroll
      for (int p = 0; p < L::JWD / S::KC; ++p) {
        auto af = jq_frag<S>(pa, p * S::KC);
#pragma unroll
        for (int b = 0; b < S::IBB; ++b) {
          auto b1 = jq_frag<S>(pb1[b], p * S::KC);
          auto b2 = jq_frag<S>(pb2[b], p * S::KC);
          t1.v[a][b] = O::mma(t1.v[a][b], af, b1);
          t2.v[a][b] = O::mma(t2.v[a][b], af, b2);
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI;
#pragma unroll
      for (int b = 0; b < S::IBB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tb + 4 * g + r;
          out.v[a][b][r] += rs1[t] * t1.v[a][b][r] + rs2[t] * t2.v[a][b][r];
        }
    }
  }
}

// Write (or add to global io) the j-round output tiles: dst[t][i] = out + extra[t][i].
template <class S, class FX>
__device__ __forceinline__ void jacc_store_io(const JAcc<S>& out, void* dst, long row0, int len,
                                              FX extra, int w, int g, int c) {
  using L = BwdLayout<S>;
  using IO = IoT<S::BF>;
  constexpr int NI = S::NIB / S::IBB;
  typename IO::T* p = reinterpret_cast<typename IO::T*>(dst) + row0 * S::D;
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI, ib0 = (it % NI) * S::IBB;
#pragma unroll
      for (int b = 0; b < S::IBB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tb + 4 * g + r, i = 16 * (ib0 + b) + c;
          if (t < len) IO::st(p + (long)t * S::D + i, out.v[a][b][r] + extra(t, i));
        }
    }
  }
}

// Write the j-round output tiles to a slot's dk or dq partial: out + extra(t, i),
// rounded to E, in accumulator order: the quad at quad offset (t / 4) D + i
// holds rows 4 (t / 4) .. + 3 of column i (one 8- or 16-byte store per tile
// and lane instead of four element stores).
template <class S, class FX>
__device__ __forceinline__ void jacc_store_part(const JAcc<S>& out, typename S::E* dst, FX extra,
                                                int w, int g, int c) {
  using L = BwdLayout<S>;
  constexpr int NI = S::NIB / S::IBB;
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI, ib0 = (it % NI) * S::IBB;
#pragma unroll
      for (int b = 0; b < S::IBB; ++b) {
        const int i = 16 * (ib0 + b) + c;
        f32x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = out.v[a][b][r] + extra(16 * tb + 4 * g + r, i);
        *reinterpret_cast<typename S::O::Q*>(dst + ((4 * tb + g) * S::D + i) * 4) = S::O::cvt(v);
      }
    }
  }
}

// Write the j-round output tiles to an fp32 [CM][D] buffer: dst[t][i] = out + extra(t, i).
template <class S, class FX>
__device__ __forceinline__ void jacc_store_f32(const JAcc<S>& out, float* dst, FX extra, int w,
                                               int g, int c) {
  using L = BwdLayout<S>;
  constexpr int NI = S::NIB / S::IBB;
#pragma unroll
  for (int a = 0; a < L::JIT; ++a) {
    const int it = w + a * S::NW;
    if (it < L::NITEM) {
      const int tb = it / NI, ib0 = (it % NI) * S::IBB;
#pragma unroll
      for (int b = 0; b < S::IBB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tb + 4 * g + r, i = 16 * (ib0 + b) + c;
          dst[t * S::D + i] = out.v[a][b][r] + extra(t, i);
        }
    }
  }
}

// Exchange slot of one rank for one parity: the dYh partial (CM x D floats),
// then the dk and dq partials (CM x D each) in the operand type E.  dk and dq
// leave the kernel in the io type, which is E, so their partials travel in it
// too (bf16 on the bf16 path: half the bytes, which keeps more of the slots in
// the XCD's L2); they are widened and added in fp32 and rounded once more.
template <class S>
__device__ __forceinline__ float* bwd_slot(float* xbuf, long p, int rank, int parity) {
  constexpr long PART = (long)S::CM * S::D * (1 + 2 * (long)sizeof(typename S::E) / 4);
  return xbuf + ((p * S::NS + rank) * 2 + parity) * PART;
}
// The dk (sec = 1) or dq (sec = 2) partial of a slot.
template <class S>
__device__ __forceinline__ typename S::E* bwd_part(float* slot, int sec) {
  return reinterpret_cast<typename S::E*>(slot + S::CM * S::D) + (sec - 1) * S::CM * S::D;
}

// dk and dq of one chunk from the ranks' partials, added in rank order (rank
// 0's carries the -eh and dO terms), rows [rlo, min(CM, rlo + RPW)) below len
// (rlo and RPW are multiples of 4).  An item is one row quad of one column:
// one quad load per rank, four element stores, each coalesced over the wave's
// 64 consecutive columns.  load() issues every rank's partial quads and
// store() widens, adds and writes them, so that the loads travel while the
// caller works in between: a partial added as soon as it is loaded would
// wait for each load in turn, and every such wait also waits for whatever
// memory operations were issued before it.  The raw quads take as many
// registers as the sums with two ranks; with more ranks, load() adds them
// itself once all are in flight.
template <class S>
struct FlushDkDq {
  using Q = typename S::O::Q;
  static constexpr int RPW = row_share<S>();
  static_assert(RPW % 4 == 0, "row shares in whole row quads");
  static constexpr int NV = (RPW / 4) * S::D;
  static constexpr int NPT = (NV + S::NT - 1) / S::NT;   // items per thread
  static constexpr bool RAW = S::NS <= 2;                // sums formed in store()
  Q raw[RAW ? NPT : 1][2][RAW ? S::NS : 1];
  f32x4 x[RAW ? 1 : NPT][2];

  __device__ __forceinline__ void load(long p, int parity, int tid) {
    Q q[NPT][2][S::NS];
#pragma unroll
    for (int a = 0; a < NPT; ++a) {
      // the item's quad; items past the rank's share or the tile (the last
      // rank's share may extend beyond CM rows) read quad 0 and are not stored
      const int qi = q0 + tid + a * S::NT;
      const int qs = (tid + a * S::NT < NV && qi < (S::CM / 4) * S::D) ? qi : 0;
#pragma unroll
      for (int sec = 1; sec <= 2; ++sec)
#pragma unroll
        for (int rk = 0; rk < S::NS; ++rk)
          q[a][sec - 1][rk] = ld_xchg(E2TTT_ARG(xbuf),
              reinterpret_cast<const Q*>(bwd_part<S>(bwd_slot<S>(E2TTT_ARG(xbuf), p, rk, parity), sec)),
              qs);
    }
    if constexpr (RAW) {
#pragma unroll
      for (int a = 0; a < NPT; ++a)
#pragma unroll
        for (int sec = 0; sec < 2; ++sec)
#pragma unroll
          for (int rk = 0; rk < S::NS; ++rk) raw[a][sec][rk] = q[a][sec][rk];
    } else {
      sched_fence();   // every load issued before the first sum waits for one
#pragma unroll
      for (int a = 0; a < NPT; ++a)
#pragma unroll
        for (int sec = 0; sec < 2; ++sec) x[a][sec] = sum_quads(q[a][sec]);
    }
  }
  __device__ __forceinline__ void store(long row0, int len, int rlo, int tid) const {
    using IO = IoT<S::BF>;
    const int tend = min(len, min(S::CM, rlo + RPW));
    typename IO::T* dk = reinterpret_cast<typename IO::T*>(E2TTT_ARG(dk)) + row0 * S::D;
    typename IO::T* dq = reinterpret_cast<typename IO::T*>(E2TTT_ARG(dq)) + row0 * S::D;
#pragma unroll
    for (int a = 0; a < NPT; ++a) {
      const int v = tid + a * S::NT;
      const int tq = rlo / 4 + v / S::D, i = v % S::D;
      if (v >= NV || 4 * tq >= tend) continue;
#pragma unroll
      for (int sec = 1; sec <= 2; ++sec) {
        typename IO::T* d = (sec == 1) ? dk : dq;
        f32x4 xs;
        if constexpr (RAW) xs = sum_quads(raw[a][sec - 1]);
        else xs = x[a][sec - 1];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * tq + r < tend) IO::st(d + (4 * tq + r) * S::D + i, xs[r]);
      }
    }
  }
  // the ranks' partials widened and added in rank order, from zero
  static __device__ __forceinline__ f32x4 sum_quads(const Q (&qr)[S::NS]) {
    f32x4 acc = zero4();
#pragma unroll
    for (int rk = 0; rk < S::NS; ++rk) acc += quad_f32(qr[rk]);
    return acc;
  }
  int q0 = 0;   // quad index of the rank's first row quad, set with the loads
};
template <class S>
__device__ __forceinline__ void flush_dkdq(long p, int parity, long row0, int len, int rlo,
                                           int tid) {
  FlushDkDq<S> f;
  f.q0 = (rlo / 4) * S::D;
  f.load(p, parity, tid);
  f.store(row0, len, rlo, tid);
}

// LONG: chunks longer than the CM-row tile.  Their tiles are processed last
// to first; every tile's P4 needs the adjoint state at the chunk end (Wb_C,
// Mb_C) as its product operands, while P8 and P9 add the tile's contributions
// to the adjoint of W_0.  So the chunk's first processed tile (its last) keeps
// the operand copies of Wb_C and Mb_C in a per-workgroup buffer, applies the
// transition Wb_0 = cw Wb_C (+ contributions), Mb_0 = cm Wb_C + cb Mb_C right
// after its P4 as a one-tile chunk does, and every tile adds its contributions
// to Wb; the chunk's other tiles take their P4 operands from the buffer.
template <class S, bool LONG, bool PN>
__global__ void __launch_bounds__(S::NT, 1) chain_bwd_kernel(ChainArgs a) {
  using O = typename S::O;
  using E = typename S::E;
  using Q = typename O::Q;
  using L = BwdLayout<S>;
  constexpr int D = S::D, NJB = S::NJB, NTB = S::NTB, NIB = S::NIB, NMAT = S::NMAT, NW = S::NW;
  constexpr int SEC = NMAT - 1;      // second-layer matrix
  constexpr int NF = NMAT - 1;       // number of first-layer matrices
  constexpr bool SW = S::FW == 1;
  constexpr int EPL = D / 16;        // head elements per lane in row phases
  constexpr int RPW = row_share<S>(); // rows of dv, dk, dq written by one rank (last: fewer)
  constexpr int NPEER = S::NS - 1;
  // the peers' dYh rows are loaded right after the swap while they are few;
  // with many peers or wide rows (head dim 128) that would hold too many
  // registers, and P7 loads every rank's partial where it adds them
  constexpr bool PEER_EARLY = NPEER * EPL <= 8 && S::D <= 64;
  __shared__ __attribute__((aligned(16))) unsigned char smem[L::TOTAL];
  __shared__ int sword[2];
  E* xk = reinterpret_cast<E*>(smem + L::XK);
  E* jw = reinterpret_cast<E*>(smem + L::JW);
  E* ja = reinterpret_cast<E*>(smem + L::JA);
  float* yk = reinterpret_cast<float*>(smem + L::YK);
  float* ek = reinterpret_cast<float*>(smem + L::EK);
  unsigned char* rr = smem + L::RR;
  E* dyt = reinterpret_cast<E*>(smem + L::DYT);
  E* yh = reinterpret_cast<E*>(smem + L::YH);
  E* yht = reinterpret_cast<E*>(smem + L::YHT);
  float* row = reinterpret_cast<float*>(smem + L::ROW);
  float* kb = reinterpret_cast<float*>(smem + L::KB);
  float* cbp = reinterpret_cast<float*>(smem + L::CB);
  float* skw = reinterpret_cast<float*>(smem + L::SC);
  float* skm = skw + S::CM;
  float* scar = skm + S::CM;

  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int T = a.T, C = a.C, NC = a.NC, dh = a.dh;
  const float inv_d = 1.0f / D;
  const bool resln = E2TTT_ARG(resln) != 0;
  const int TPC = LONG ? (C + S::CM - 1) / S::CM : 1;   // tiles per chunk
  const int TL = LONG ? S::CM : C;                       // tokens per tile
  auto ntiles = [&](int rc) { return LONG ? (min(T, (rc + 1) * C) - rc * C + TL - 1) / TL : 1; };
  constexpr int NB = NMAT * NJB * NIB * S::NT;            // float4 per frozen block
  // LONG: the operand copies of Wb_C, then of Mb_C (NB quads each, register-tile order)
  Q* const frz = LONG ? reinterpret_cast<Q*>(reinterpret_cast<f32x4*>(E2TTT_ARG(bfrz)) + (long)blockIdx.x * 2 * NB)
                      : nullptr;

  PairX<S::NS> px;
  px.init(a.sync, a.npairs, sword, a.wait_ticks);
  const int rank = px.rank;
  const int j0 = rank * S::DHP;
  const long NP = (S::NS > 1) ? a.npairs : (long)gridDim.x;
  const int rlo = rank * RPW;
  const int rhi = min(S::CM, rlo + RPW);
  float* const kwb_slot = E2TTT_ARG(kwb) + rank * a.U * T;
  float* const kmb_slot = E2TTT_ARG(kmb) + rank * a.U * T;
  float* const carryb_slot = E2TTT_ARG(carryb) + rank * a.U * NC * 3;
  long nch = 0;   // chunks processed by this workgroup (exchange parity)

  // inputs loaded ahead of use: the K side of the next chunk during the output
  // branch, the Q side of this chunk during P7
  TileRegs<S> pK, pV, pQ, pD;
  F32TileRegs<S> pZ, pZq;
  float pkw = 0.0f, pkm = 0.0f, prk = 0.0f, prq = 0.0f, pcar = 0.0f;
  auto prefetch_k = [&](long uu, int rc, int kt) {
    E2TTT_LANE_IDS;
    const int st = LONG ? rc * C + kt * TL : rc * C;
    const long r0 = uu * T + st;
    const int ln = LONG ? min(TL, min(T, (rc + 1) * C) - st) : min(C, T - st);
    pK.load(E2TTT_ARG(k), r0, ln, tid);
    pV.load(E2TTT_ARG(v), r0, ln, tid);
    pZ.load(E2TTT_ARG(zk), r0, ln, tid);
    if (tid < S::CM) {
      pkw = (tid < ln) ? E2TTT_ARG(kw)[r0 + tid] : 0.0f;
      pkm = (tid < ln) ? E2TTT_ARG(km)[r0 + tid] : 0.0f;
      prk = (tid < ln) ? ld_stream(E2TTT_ARG(rk) + r0 + tid) : 0.0f;
    }
    if (tid < 3) pcar = E2TTT_ARG(carry)[(uu * NC + rc) * 3 + tid];
  };
  auto prefetch_q = [&](long uu, int rc, int kt) {
    E2TTT_LANE_IDS;
    const int st = LONG ? rc * C + kt * TL : rc * C;
    const long r0 = uu * T + st;
    const int ln = LONG ? min(TL, min(T, (rc + 1) * C) - st) : min(C, T - st);
    pQ.load(E2TTT_ARG(q), r0, ln, tid);
    pD.load(E2TTT_ARG(d_out), r0, ln, tid);
    pZq.load(E2TTT_ARG(zq), r0, ln, tid);
    if (tid < S::CM) prq = (tid < ln) ? ld_stream(E2TTT_ARG(rq) + r0 + tid) : 0.0f;
  };

  for (long u = px.p; u < a.U; u += NP) {
    // adjoint of the final state
    StateTiles<S> Wb, Mb;
    {
      E2TTT_LANE_IDS;
      load_state<S>(Wb, E2TTT_ARG(d_w_out) ? E2TTT_ARG(d_w_out) + u * a.P : nullptr, dh, j0, w, g, c);
      load_state<S>(Mb, E2TTT_ARG(d_m_out) ? E2TTT_ARG(d_m_out) + u * a.P : nullptr, dh, j0, w, g, c);
    }
    // the tile whose dk, dq partials are not yet combined (first token, length)
    int pend_s0 = -1, pend_len = 0, pend_par = 0;
    prefetch_k(u, NC - 1, ntiles(NC - 1) - 1);

    // tile kt of chunk r, last to first (always kt = 0 unless LONG)
    for (int r = NC - 1, kt = ntiles(NC - 1) - 1; r >= 0; ++nch) {
      const int s0 = LONG ? r * C + kt * TL : r * C;
      const int cend = LONG ? min(T, (r + 1) * C) : 0;
      const int len = LONG ? min(TL, cend - s0) : min(C, T - s0);
      const bool firstp = !LONG || s0 + TL >= cend;   // the chunk's first tile processed (its last)
      const int rc = r, kc = kt;                      // this tile
      if (kt > 0) --kt;
      else if (--r >= 0) kt = ntiles(r) - 1;
      const long row0 = u * T + s0;
      const int par = (int)(nch & 1);

      // ---- reverse of the post-chunk normalisation at this chunk's end (the
      // chunk's first tile processed).  The normalised row is W_r = t_r u_r
      // (t_r its target norm, n_r its norm before, u_r the unit direction),
      // so Wb_r, the adjoint of W_r, becomes that of the row before:
      //   Wb_r <- (t_r / n_r) Wb_r - (W_r / n_r) (A_r / t_r),  A_r = <W_r, Wb_r>,
      // and <u_r, Wb_r> = A_r / t_r is what flows into t_r (summed over the
      // chunks, and applied to d_w_in at the unit's end).  W_r is the next
      // chunk's checkpoint (the final state's for the last chunk).  A row the
      // forward left alone (n_r = 0) keeps its adjoint; one sent to zero
      // (t_r = 0) gets none.
      if (PN && firstp) {
        E2TTT_LANE_IDS;
        const long R = (long)NF * dh + D;
        const float* tg = E2TTT_ARG(norm_tgt) + u * R;
        const float* npre = E2TTT_ARG(norm_pre) + (u * NC + rc) * R;
        float* rbar = E2TTT_ARG(norm_rbar) + (u * S::NS + rank) * R;
        const bool init = rc == NC - 1;
        const char* ckN = static_cast<const char*>(E2TTT_ARG(ckpt)) +
                          ((u * E2TTT_ARG(ckpt_nc) + rc + 1) * S::NS + rank) * 2 *
                              E2TTT_ARG(ckpt_stride);
        // first-layer rows: hidden unit j is the tile column of lanes c + 16 g
#pragma unroll
        for (int m = 0; m < NF; ++m) {
          Q wn[NJB][NIB];
          load_ckpt_mat<S>(wn, ckN, m, w, lane);
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            float A = 0.0f;
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
              const f32x4 x = quad_f32(wn[jj][ib]);
#pragma unroll
              for (int q = 0; q < 4; ++q) A = fmaf(x[q], Wb.t[m][jj][ib][q], A);
            }
            A += __shfl_xor(A, 16);
            A += __shfl_xor(A, 32);
            const int j = j0 + 16 * (w * NJB + jj) + c;
            float s1 = 1.0f, s2 = 0.0f, dot = 0.0f;
            if (j < dh) {
              const float t = tg[(long)m * dh + j], n = npre[(long)m * dh + j];
              if (n > 0.0f) {
                s1 = t / n;
                if (t > 0.0f) { dot = A / t; s2 = dot / n; }
              }
              if (g == 0) rbar[(long)m * dh + j] = init ? dot : rbar[(long)m * dh + j] + dot;
            }
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib)
              Wb.t[m][jj][ib] = s1 * Wb.t[m][jj][ib] - s2 * quad_f32(wn[jj][ib]);
          }
        }
        // second-layer rows: output i's weights span the lanes, the waves and
        // the ranks; partial sums through LDS (Y's buffer, not yet staged)
        // and, between ranks, the exchange, added in rank order on every rank
        static_assert(S::CM >= NW + 2, "LDS room for the row sums");
        float* part = yk;   // [NW][D] wave partials, then [2][D] row factors
        Q wn[NJB][NIB];
        load_ckpt_mat<S>(wn, ckN, SEC, w, lane);
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
          float A[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            const f32x4 x = quad_f32(wn[jj][ib]);
#pragma unroll
            for (int q = 0; q < 4; ++q) A[q] = fmaf(x[q], Wb.t[SEC][jj][ib][q], A[q]);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float v = group16_sum(A[q]);
            if (c == 0) part[w * D + 16 * ib + 4 * g + q] = v;
          }
        }
        __syncthreads();
        float A = 0.0f;
        if (tid < D)
          for (int ww = 0; ww < NW; ++ww) A += part[ww * D + tid];
        if constexpr (S::NS > 1) {
          float* nx = E2TTT_ARG(nxbuf);
          if (tid < D) nx[((px.xs * S::NS + rank) * 2 + par) * D + tid] = A;
          px.post();
          px.wait_for(px.seq_now(), sword);
          if (tid < D) {
            A = 0.0f;
            for (int rr = 0; rr < S::NS; ++rr)
              A += ld_xchg(nx, nx + ((px.xs * S::NS + rr) * 2 + par) * D, tid);
          }
        }
        if (tid < D) {
          const float t = tg[(long)NF * dh + tid], n = npre[(long)NF * dh + tid];
          float s1 = 1.0f, s2 = 0.0f, dot = 0.0f;
          if (n > 0.0f) {
            s1 = t / n;
            if (t > 0.0f) { dot = A / t; s2 = dot / n; }
          }
          part[NW * D + tid] = s1;
          part[(NW + 1) * D + tid] = s2;
          rbar[(long)NF * dh + tid] = init ? dot : rbar[(long)NF * dh + tid] + dot;
        }
        __syncthreads();
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
          const f32x4 s1 = *reinterpret_cast<const f32x4*>(&part[NW * D + 16 * ib + 4 * g]);
          const f32x4 s2 = *reinterpret_cast<const f32x4*>(&part[(NW + 1) * D + 16 * ib + 4 * g]);
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
            Wb.t[SEC][jj][ib] = s1 * Wb.t[SEC][jj][ib] - s2 * quad_f32(wn[jj][ib]);
        }
        __syncthreads();   // part (Y's buffer) is staged next
      }

      // the exchange sequence of this tile starts after the normalisation's
      const unsigned seq0 = px.seq_now();
      const char* ckW = static_cast<const char*>(E2TTT_ARG(ckpt)) +
                        ((u * E2TTT_ARG(ckpt_nc) + rc) * S::NS + rank) * 2 * E2TTT_ARG(ckpt_stride);
      const char* ckM = ckW + E2TTT_ARG(ckpt_stride);

      // chunk-start weights W_0 (kept for the whole chunk), issued first so
      // that P0 and P3 hide them; momentum M_0 (for the carry adjoints after
      // P3) follows after P0, so that the two bursts of loads each drain under
      // a phase
      Q w0q[NMAT][NJB][NIB], m0q[NMAT][NJB][NIB];
      {
        E2TTT_LANE_IDS;
#pragma unroll
        for (int m = 0; m < NMAT; ++m) load_ckpt_mat<S>(w0q[m], ckW, m, w, lane);
      }

      // ---------------------------------------------------------- P0: stage
      E* xv = reinterpret_cast<E*>(rr);
      {
        E2TTT_LANE_IDS;
        pK.store(xk, tid);
        pV.store(xv, tid);
        pZ.store(yk, tid);                       // Z (or Y without the residual LN)
        if (tid < S::CM) {
          skw[tid] = pkw;
          skm[tid] = pkm;
          row[2 * tid] = prk;                    // 1 / sigma
        }
        if (tid < 3) scar[tid] = pcar;
      }
      __syncthreads();
      {
        E2TTT_LANE_IDS;
#pragma unroll
        for (int m = 0; m < NMAT; ++m) load_ckpt_mat<S>(m0q[m], ckM, m, w, lane);
      }

      // --------------------- P3: e, dY (first order, from the saved LN output)
      E* dyl = reinterpret_cast<E*>(rr + L::TDX);   // dY [t][i]
      {
      E2TTT_LANE_IDS;
#pragma unroll
      for (int it_ = 0; it_ < (S::CM + 4 * NW - 1) / (4 * NW); ++it_) {
        const int t0 = 4 * w + it_ * 4 * NW;
        if (t0 < S::CM) {
        const int t = t0 + (lane >> 4);
        float z[EPL], e[EPL], dyv[EPL];
        float mez = 0.0f;
#pragma unroll
        for (int q = 0; q < EPL; ++q) z[q] = yk[t * D + l16 * EPL + q];
        if (resln) {
          const float sig = row[2 * t];
          float se = 0.0f, sez = 0.0f;
          if (E2TTT_ARG(ln_a)) {
            // f = k + a z + b: e below is a (v - f), what the LayerNorm backward takes
            float la[EPL], lb[EPL];
            const long ho = (u % E2TTT_ARG(H)) * D + l16 * EPL;
            load_row_part<EPL>(la, E2TTT_ARG(ln_a) + ho);
            load_row_part<EPL>(lb, E2TTT_ARG(ln_b) + ho);
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              const int i = l16 * EPL + q;
              const float r = O::from_e(xv[t * S::LDD + i]) - O::from_e(xk[t * S::LDD + i]);
              e[q] = la[q] * (r - fmaf(la[q], z[q], lb[q]));
              se += e[q];
              sez += e[q] * z[q];
            }
          } else {
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              const int i = l16 * EPL + q;
              e[q] = O::from_e(xv[t * S::LDD + i]) - O::from_e(xk[t * S::LDD + i]) - z[q];
              se += e[q];
              sez += e[q] * z[q];
            }
          }
          const float me = group16_sum(se) * inv_d;
          mez = group16_sum(sez) * inv_d;
#pragma unroll
          for (int q = 0; q < EPL; ++q) dyv[q] = (e[q] - me - z[q] * mez) * sig;
        } else {
#pragma unroll
          for (int q = 0; q < EPL; ++q) {
            e[q] = O::from_e(xv[t * S::LDD + l16 * EPL + q]) - z[q];
            dyv[q] = e[q];
            z[q] = 0.0f;
          }
        }
#pragma unroll
        for (int q = 0; q < EPL; ++q) {
          const int i = l16 * EPL + q;
          yk[t * D + i] = z[q];
          ek[t * D + i] = e[q];
        }
        store_row_ti<S, EPL>(dyl, S::LDD, t, l16 * EPL, dyv);
        store_row_it<S, EPL>(dyt, t, l16 * EPL, dyv);
        if (l16 == 0) row[2 * t + 1] = mez;
              }
      }
      }
      __syncthreads();

      // ------------- carry adjoints: <Wb, W_0>, <Wb, M_0>, <Mb, M_0> (per wave)
      if (firstp) {
        E2TTT_LANE_IDS;
        float pcw = 0.0f, pcm = 0.0f, pcb = 0.0f;
#pragma unroll
        for (int m = 0; m < NMAT; ++m) {
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
              const f32x4 w0 = quad_f32(w0q[m][jj][ib]), m0 = quad_f32(m0q[m][jj][ib]);
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                pcw += Wb.t[m][jj][ib][q] * w0[q];
                pcm += Wb.t[m][jj][ib][q] * m0[q];
                pcb += Mb.t[m][jj][ib][q] * m0[q];
              }
            }
        }
        pcw = wave_sum(pcw);
        pcm = wave_sum(pcm);
        pcb = wave_sum(pcb);
        if (lane == 0) { cbp[w * 4 + 0] = pcw; cbp[w * 4 + 1] = pcm; cbp[w * 4 + 2] = pcb; }
        if constexpr (LONG) {   // Wb_C, Mb_C operands for the chunk's other tiles
#pragma unroll
          for (int m = 0; m < NMAT; ++m)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
              for (int ib = 0; ib < NIB; ++ib) {
                const long idx = ((m * NJB + jj) * NIB + ib) * S::NT + tid;
                frz[idx] = O::cvt(Wb.t[m][jj][ib]);
                frz[NB + idx] = O::cvt(Mb.t[m][jj][ib]);
              }
        }
      }

      // ----------- P4: first-order deltas, scalar-kernel adjoints, Hessian terms
      // For every tile: H = K W1^T and A = act(H) (recomputed from the checkpoint),
      // dA = dY W2, dH = dA act'(H);  u = K Wb1^T, K Mb1^T;
      // rW = dY Wb2, dY Mb2;  dK^W += rowsum(dH uW + A rW), dK^M likewise;
      // p = K^W uW + K^M uM (= d(Phi)/d(dH)), r2 = K^W rW + K^M rM (direct a-term);
      // dAh = p act'(H);  Hh = p dA act''(H) + r2 act'(H)  (the Yh W2 term is added in P8)
      // MLP with one j-round half: dH goes straight into the j-round act buffer
      constexpr bool DH_LDS = (NF == 1) && (L::JH == 1);
      Q Akq[NTB][NJB];
      // act'(H) factors: MLP GELU'(H); SwiGLU Hu SiLU'(Hg), SiLU(Hg)
      f32x4 D1[NF][NTB][NJB];
      Q dHq[DH_LDS ? 1 : NF][NTB][NJB];
      Q dAhq[NTB][NJB];
      // Hh, in LDS when it fits (hh_at), else in registers
      f32x4 HhR[L::HH_LDS ? 1 : NF][L::HH_LDS ? 1 : NTB][L::HH_LDS ? 1 : NJB];
      f32x4* const hhlds = reinterpret_cast<f32x4*>(smem + L::HHR);
      auto hh_at = [&](int m, int tb, int jj, int ln) -> f32x4& {
        if constexpr (L::HH_LDS)
          return hhlds[((m * NTB + tb) * NW + w) * 64 + ln];
        else
          return HhR[m][tb][jj];
      };
      // operand copies of the adjoint state, formed once for all token blocks
      // of P4 and the j-rounds after it
      Q wbq[NMAT][NJB][NIB], mbq[NMAT][NJB][NIB];
      {
        const auto& w1q = w0q;            // first-layer matrices m < NF
        const auto& w2q = w0q[SEC];
        opaque_state<S>(Wb);
        opaque_state<S>(Mb);
        if (LONG && !firstp) {   // Wb, Mb hold the chunk's W_0 adjoints by now
          E2TTT_LANE_IDS;
#pragma unroll
          for (int m = 0; m < NMAT; ++m)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
              for (int ib = 0; ib < NIB; ++ib) {
                const long idx = ((m * NJB + jj) * NIB + ib) * S::NT + tid;
                wbq[m][jj][ib] = frz[idx];
                mbq[m][jj][ib] = frz[NB + idx];
              }
        } else {
#pragma unroll
          for (int m = 0; m < NMAT; ++m)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
              for (int ib = 0; ib < NIB; ++ib) {
                wbq[m][jj][ib] = O::cvt(Wb.t[m][jj][ib]);
                mbq[m][jj][ib] = O::cvt(Mb.t[m][jj][ib]);
              }
        }
        // The products of token block (tb, jj) (dA, rW, rM, then hk, uW, uM of
        // each first-layer matrix) are issued one item ahead of the arithmetic
        // that uses them, in the same scheduling region, so that the matrix
        // cores work on the next item while the VALU evaluates this one.
        constexpr int NPR = 3 + 3 * NF, NITEM4 = NTB * NJB;
        auto p4_products = [&](int tb, int jj, f32x4 (&r)[NPR]) {
          E2TTT_LANE_IDS;
#pragma unroll
          for (int x = 0; x < NPR; ++x) r[x] = zero4();
#pragma unroll
          for (int p = 0; p < S::KS_D; ++p) {
            auto fy = lds_frag<S::BF>(dyl, S::LDD, 16 * tb + c, p * S::KC, g);
            auto fk = lds_frag<S::BF>(xk, S::LDD, 16 * tb + c, p * S::KC, g);
            typename O::Frag b2, bw, bm;
#pragma unroll
            for (int h = 0; h < S::NH; ++h) {
              b2.h[h] = w2q[jj][S::NH * p + h];
              bw.h[h] = wbq[SEC][jj][S::NH * p + h];
              bm.h[h] = mbq[SEC][jj][S::NH * p + h];
            }
            r[0] = O::mma(r[0], fy, b2);
            r[1] = O::mma(r[1], fy, bw);
            r[2] = O::mma(r[2], fy, bm);
#pragma unroll
            for (int m = 0; m < NF; ++m) {
#pragma unroll
              for (int h = 0; h < S::NH; ++h) {
                b2.h[h] = w1q[m][jj][S::NH * p + h];
                bw.h[h] = wbq[m][jj][S::NH * p + h];
                bm.h[h] = mbq[m][jj][S::NH * p + h];
              }
              r[3 + m] = O::mma(r[3 + m], fk, b2);
              r[3 + NF + m] = O::mma(r[3 + NF + m], fk, bw);
              r[3 + 2 * NF + m] = O::mma(r[3 + 2 * NF + m], fk, bm);
            }
          }
        };
        f32x4 pcur[NPR], pnext[NPR];
        p4_products(0, 0, pcur);
        sched_fence();
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          E2TTT_LANE_IDS;
          float kwp[4] = {0.0f, 0.0f, 0.0f, 0.0f}, kmp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            const int it4 = tb * NJB + jj;
            if (it4 + 1 < NITEM4) p4_products((it4 + 1) / NJB, (it4 + 1) % NJB, pnext);
            const f32x4 dA = pcur[0], rW = pcur[1], rM = pcur[2];
            f32x4 uW[NF], uM[NF], hk[NF];
#pragma unroll
            for (int m = 0; m < NF; ++m) {
              hk[m] = pcur[3 + m];
              uW[m] = pcur[3 + NF + m];
              uM[m] = pcur[3 + 2 * NF + m];
            }
            f32x4 dH[NF], dAh, hh[NF], Af;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int t = 16 * tb + 4 * g + q;
              const float kwv = skw[t], kmv = skm[t];
              const float r2 = kwv * rW[q] + kmv * rM[q];
              if constexpr (!SW) {
                const Act3 ga = gelu3(hk[0][q]);
                Af[q] = ga.f;
                D1[0][tb][jj][q] = ga.d1;
                dH[0][q] = dA[q] * ga.d1;
                const float pp = kwv * uW[0][q] + kmv * uM[0][q];
                dAh[q] = pp * ga.d1;
                hh[0][q] = pp * dA[q] * ga.d2 + r2 * ga.d1;
                kwp[q] += dH[0][q] * uW[0][q] + Af[q] * rW[q];
                kmp[q] += dH[0][q] * uM[0][q] + Af[q] * rM[q];
              } else {
                const float hg = hk[0][q], hu = hk[1][q];
                const Act3 sa = silu3(hg);
                const float sg = sa.f, s1 = sa.d1, s2 = sa.d2;
                Af[q] = sg * hu;
                D1[0][tb][jj][q] = hu * s1;
                D1[1][tb][jj][q] = sg;
                dH[0][q] = dA[q] * hu * s1;
                dH[1][q] = dA[q] * sg;
                const float pg = kwv * uW[0][q] + kmv * uM[0][q];
                const float pu = kwv * uW[1][q] + kmv * uM[1][q];
                dAh[q] = pg * hu * s1 + pu * sg;
                hh[0][q] = pg * dA[q] * hu * s2 + pu * dA[q] * s1 + r2 * hu * s1;
                hh[1][q] = pg * dA[q] * s1 + r2 * sg;
                kwp[q] += dH[0][q] * uW[0][q] + dH[1][q] * uW[1][q] + Af[q] * rW[q];
                kmp[q] += dH[0][q] * uM[0][q] + dH[1][q] * uM[1][q] + Af[q] * rM[q];
              }
            }
#pragma unroll
            for (int m = 0; m < NF; ++m) hh_at(m, tb, jj, lane) = hh[m];
            if constexpr (DH_LDS) {
              jq_put<S, L::LDJ>(ja, tb, g, 16 * (w * NJB + jj) + c, O::cvt(dH[0]));
            } else {
#pragma unroll
              for (int m = 0; m < NF; ++m) dHq[m][tb][jj] = O::cvt(dH[m]);
            }
            dAhq[tb][jj] = O::cvt(dAh);
            Akq[tb][jj] = O::cvt(Af);
            if (it4 + 1 < NITEM4) {
#pragma unroll
              for (int x = 0; x < NPR; ++x) pcur[x] = pnext[x];
            }
            sched_fence();
          }
          // per-wave row partials of dK^W, dK^M for this token block: after the
          // reduce-scatter, lane c (even) holds the row sum of dK^W (c < 8) or
          // dK^M (c >= 8) for row 4 g + (c / 2) mod 4
          {
            const float vals[8] = {kwp[0], kwp[1], kwp[2], kwp[3], kmp[0], kmp[1], kmp[2], kmp[3]};
            const float sred = row16_reduce_scatter8(vals, c);
            if ((c & 1) == 0)
              kb[(((c >> 3) & 1) * NW + w) * S::CM + 16 * tb + 4 * g + ((c >> 1) & 3)] = sred;
          }
        }
      }
      // direct terms through the state adjoint, over the hidden index:
      //   r1 = K^W (dH Wb1) + K^M (dH Mb1)  (into dK),  p2 = K^W (A Wb2^T) + K^M (A Mb2^T)  (into dYh)
      JAcc<S> dkacc, dyhacc;
      dkacc.zero();
      dyhacc.zero();
      {
      E2TTT_LANE_IDS;
      // (with a single j-round half the two rounds of a pair share the act buffer)
      E* const jw2 = reinterpret_cast<E*>(smem + L::JW2);
#pragma unroll
      for (int m = 0; m < NF; ++m) {
        const int mq = DH_LDS ? 0 : m;
        if constexpr (L::J2) {
          jround2<S, !DH_LDS>(dkacc, skw, skm, ja, jw, jw2,
                              [&](int tb, int jj) { return dHq[mq][tb][jj]; },
                              [&](int ib, int jj) { return wbq[m][jj][ib]; },
                              [&](int ib, int jj) { return mbq[m][jj][ib]; }, w, g, c);
        } else {
          jround<S, !DH_LDS>(dkacc, skw, ja, jw,
                             [&](int tb, int jj) { return dHq[mq][tb][jj]; },
                             [&](int ib, int jj) { return wbq[m][jj][ib]; }, w, g, c);
          jround<S, false>(dkacc, skm, ja, jw,
                           [&](int tb, int jj) { return dHq[mq][tb][jj]; },
                           [&](int ib, int jj) { return mbq[m][jj][ib]; }, w, g, c);
        }
      }
      if constexpr (L::J2) {
        jround2<S, true>(dyhacc, skw, skm, ja, jw, jw2, [&](int tb, int jj) { return Akq[tb][jj]; },
                         [&](int ib, int jj) { return wbq[SEC][jj][ib]; },
                         [&](int ib, int jj) { return mbq[SEC][jj][ib]; }, w, g, c);
      } else {
        jround<S>(dyhacc, skw, ja, jw, [&](int tb, int jj) { return Akq[tb][jj]; },
                  [&](int ib, int jj) { return wbq[SEC][jj][ib]; }, w, g, c);
        jround<S, false>(dyhacc, skm, ja, jw, [&](int tb, int jj) { return Akq[tb][jj]; },
                         [&](int ib, int jj) { return mbq[SEC][jj][ib]; }, w, g, c);
      }
      }

      // ------------------------------------ P5: adjoint state transition
      // (LONG: once per chunk, at its first tile processed)
      if (!LONG || firstp) {
        const float cw = scar[0], cm = scar[1], cbv = scar[2];
#pragma unroll
        for (int m = 0; m < NMAT; ++m)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
              const f32x4 wb = Wb.t[m][jj][ib];
              Mb.t[m][jj][ib] = cm * wb + cbv * Mb.t[m][jj][ib];
              Wb.t[m][jj][ib] = cw * wb;
            }
      }

      // --------------------------- P6: dYh = p2 + dAh W2^T  (into RR, fp32)
      float* dyh = reinterpret_cast<float*>(rr);
      {
        E2TTT_LANE_IDS;
        const auto& w2q = w0q[SEC];
        jround<S>(dyhacc, nullptr, ja, jw, [&](int tb, int jj) { return dAhq[tb][jj]; },
                  [&](int ib, int jj) { return w2q[jj][ib]; }, w, g, c);
        jacc_store_f32<S>(dyhacc, dyh, [](int, int) { return 0.0f; }, w, g, c);
      }
      __syncthreads();
      constexpr int P7IT = (S::CM + 4 * NW - 1) / (4 * NW);
      FlushDkDq<S> flush;
      float pdyh[S::NS > 1 && PEER_EARLY ? P7IT : 1][S::NS > 1 ? NPEER : 1][EPL];
      if constexpr (S::NS > 1) {
        E2TTT_LANE_IDS;
        float* mine = bwd_slot<S>(E2TTT_ARG(xbuf), px.xs, rank, par);
#pragma unroll 1
        for (int v = tid; v < S::CM * D / 4; v += S::NT)
          reinterpret_cast<float4*>(mine)[v] = reinterpret_cast<const float4*>(dyh)[v];
        px.post();                                  // seq0 + 1: dYh partial, previous tile's dk, dq
        px.wait_for(seq0 + 1, sword);               // the peers'
        // the peers' rows of every P7 step, loaded before the global stores
        // below (which would otherwise order each step's loads after them)
#pragma unroll
        for (int k = 0; k < (PEER_EARLY ? NPEER : 0); ++k) {
          const float* dyh_peer = bwd_slot<S>(E2TTT_ARG(xbuf), px.xs, other_rank(k, rank), par);
#pragma unroll
          for (int it_ = 0; it_ < P7IT; ++it_) {
            const int t0 = 4 * w + it_ * 4 * NW;
            if (t0 < S::CM)
              load_row_xchg<EPL>(pdyh[it_][k], E2TTT_ARG(xbuf), dyh_peer,
                                 (t0 + (lane >> 4)) * D + l16 * EPL);
          }
        }
        // the previous chunk's dk / dq: partials read now (their latency
        // overlaps the peers' rows'), rows written after P7's first row step
        if (pend_s0 >= 0) {
          flush.q0 = (rlo / 4) * S::D;
          flush.load(px.xs, pend_par, tid);
        }
      }

      // ------------------------------------- P7: LayerNorm second order
      // every earlier memory operation complete (the first row step waits for
      // the peers' rows, issued before the flush, anyway): stated through the
      // builtin, so that the compiler knows it and the second row step does
      // not wait again, for the tile loads issued between the steps
      __builtin_amdgcn_s_waitcnt(0x0F70);
      {
        E2TTT_LANE_IDS;
        using IOT = typename IoT<S::BF>::T;
        IOT* dvp = reinterpret_cast<IOT*>(E2TTT_ARG(dv)) + row0 * D;
#pragma unroll
        for (int it_ = 0; it_ < P7IT; ++it_) {
          const int t0 = 4 * w + it_ * 4 * NW;
          if (t0 < S::CM) {
          const int t = t0 + (lane >> 4);
          float dyhv[EPL], e[EPL], eh[EPL], yhv[EPL];
#pragma unroll
          for (int q = 0; q < EPL; ++q) {
            dyhv[q] = dyh[t * D + l16 * EPL + q];
            e[q] = ek[t * D + l16 * EPL + q];
          }
          if constexpr (S::NS > 1 && PEER_EARLY) {
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              float pv[NPEER];
#pragma unroll
              for (int k = 0; k < NPEER; ++k) pv[k] = pdyh[it_][k][q];
              dyhv[q] = sum_ranks<S::NS>(dyhv[q], pv, rank);
            }
          } else if constexpr (S::NS > 1) {
            // every rank's partial from its slot (this rank's too), added in
            // rank order as sum_ranks does: the same sum on every rank
            sum_rows_xchg<S::NS, EPL>(dyhv, E2TTT_ARG(xbuf),
                                      [&](int r) { return bwd_slot<S>(E2TTT_ARG(xbuf), px.xs, r, par); },
                                      t * D + l16 * EPL);
          }
          if (resln) {
            float z[EPL], dyv[EPL], zh[EPL];
            const float sig = row[2 * t], mez = row[2 * t + 1];
            float se = 0.0f, m1 = 0.0f, m2 = 0.0f;
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              z[q] = yk[t * D + l16 * EPL + q];
              se += e[q];
              m1 += dyhv[q];
              m2 += dyhv[q] * z[q];
            }
            const float me = group16_sum(se) * inv_d;
            m1 = group16_sum(m1) * inv_d;
            m2 = group16_sum(m2) * inv_d;
            float sdd = 0.0f;
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              dyv[q] = (e[q] - me - z[q] * mez) * sig;
              eh[q] = (dyhv[q] - m1 - z[q] * m2) * sig;
              sdd += dyhv[q] * dyv[q];
            }
            const float sh = -group16_sum(sdd) * sig;
            float n1 = 0.0f, n2 = 0.0f;
#pragma unroll
            for (int q = 0; q < EPL; ++q) zh[q] = -(dyhv[q] * mez + e[q] * m2) * sig;
            if (E2TTT_ARG(ln_a)) {
              // with f = k + a z + b: e's adjoint is a eh (dv, and -a eh into dk), and z
              // takes -a^2 eh; eh itself (the adjoint of a e) is kept for the
              // affine's gradients
              float la[EPL];
              load_row_part<EPL>(la, E2TTT_ARG(ln_a) + (u % E2TTT_ARG(H)) * D + l16 * EPL);
              if (t < len && t >= rlo && t < rhi)
                store_row_io<IoT<false>, EPL>(E2TTT_ARG(ln_zbar) + (row0 + t) * D + l16 * EPL, eh);
#pragma unroll
              for (int q = 0; q < EPL; ++q) {
                zh[q] -= la[q] * la[q] * eh[q];
                eh[q] *= la[q];
              }
            } else {
#pragma unroll
              for (int q = 0; q < EPL; ++q) zh[q] -= eh[q];
            }
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              n1 += zh[q];
              n2 += zh[q] * z[q];
            }
            n1 = group16_sum(n1) * inv_d;
            n2 = group16_sum(n2) * inv_d;
#pragma unroll
            for (int q = 0; q < EPL; ++q) yhv[q] = (zh[q] - n1 - z[q] * n2) * sig + sh * z[q] * inv_d;
          } else {
#pragma unroll
            for (int q = 0; q < EPL; ++q) { eh[q] = dyhv[q]; yhv[q] = -eh[q]; }
          }
#pragma unroll
          for (int q = 0; q < EPL; ++q) ek[t * D + l16 * EPL + q] = eh[q];
          if (t < len && t >= rlo && t < rhi)
            store_row_io<IoT<S::BF>, EPL>(dvp + (long)t * D + l16 * EPL, eh);
          store_row_ti<S, EPL>(yh, S::LDD, t, l16 * EPL, yhv);
          store_row_it<S, EPL>(yht, t, l16 * EPL, yhv);
                  }
          // the output branch's tiles, issued after the first row step: issued
          // before it, the wait for the peers' rows (whose count of later
          // memory operations the compiler loses over the flush loop) waited
          // for these loads from HBM as well; issued here, they drain from the
          // memory pipeline while the next row step computes
          if (it_ == 0) {
            prefetch_q(u, rc, kc);
            if (S::NS > 1 && pend_s0 >= 0) flush.store(u * T + pend_s0, pend_len, rlo, tid);
          }
        }
      }
      // MLP: A_Q and GELU'(H_Q) as the forward formed them (its query side at
      // W_0, GELU' packed), in flight during P8
      Q Aqq[NTB][NJB];
      typename DerivQ<S::BF>::T D1p[SW ? 1 : NTB][SW ? 1 : NJB];
      if constexpr (!SW) {
        E2TTT_LANE_IDS;
        const SavedAct<S> sv(static_cast<char*>(E2TTT_ARG(asave)) +
                             (((u * NC + rc) * TPC + kc) * S::NS + rank) * E2TTT_ARG(as_stride));
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            const int qi = SavedAct<S>::idx(tb, jj, w, lane);
            Aqq[tb][jj] = ld_stream(sv.aq() + qi);
            D1p[tb][jj] = ld_stream(sv.d1q() + qi);
          }
      }
      __syncthreads();

      // ---------- P8: Hh += (Yh W2) act'(H); accumulate into Wb; dk = r1 - eh + Hh W1
      {
        E2TTT_LANE_IDS;
        // K^T into RR for the first-layer accumulation
        E* xkt = reinterpret_cast<E*>(rr);
        transpose_to_it<S>(xkt, xk, tid);
        const auto& w2q = w0q[SEC];
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
          for (int jj = 0; jj < NJB; ++jj) {
            f32x4 ah = zero4();
#pragma unroll
            for (int p = 0; p < S::KS_D; ++p) {
              auto af = lds_frag<S::BF>(yh, S::LDD, 16 * tb + c, p * S::KC, g);
              typename O::Frag bf;
#pragma unroll
              for (int h = 0; h < S::NH; ++h) bf.h[h] = w2q[jj][S::NH * p + h];
              ah = O::mma(ah, af, bf);
            }
#pragma unroll
            for (int m = 0; m < NF; ++m) {
              f32x4 hv = hh_at(m, tb, jj, lane);
#pragma unroll
              for (int q = 0; q < 4; ++q) hv[q] += ah[q] * D1[m][tb][jj][q];
              hh_at(m, tb, jj, lane) = hv;
            }
            sched_fence();
          }
        __syncthreads();   // xkt complete
        // Wb2 += dY^T dAh + Yh^T A ;  Wb1 += K^T Hh
        opaque_state<S>(Wb);
        Q hhq[NF][NTB][NJB];   // Hh as operand quads, for every head block and the dk round
#pragma unroll
        for (int m = 0; m < NF; ++m)
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj) hhq[m][tb][jj] = O::cvt(hh_at(m, tb, jj, lane));
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
          for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
            for (int p = 0; p < S::KS_C; ++p) {
              typename O::Frag bd, ba;
#pragma unroll
              for (int h = 0; h < S::NH; ++h) {
                bd.h[h] = dAhq[S::NH * p + h][jj];
                ba.h[h] = Akq[S::NH * p + h][jj];
              }
              const int rowi = 16 * ib + c, k0 = p * S::KC;
              Wb.t[SEC][jj][ib] = O::mma(Wb.t[SEC][jj][ib], it_frag<S>(dyt, rowi, k0, g), bd);
              Wb.t[SEC][jj][ib] = O::mma(Wb.t[SEC][jj][ib], it_frag<S>(yht, rowi, k0, g), ba);
              auto fk = it_frag<S>(xkt, rowi, k0, g);
#pragma unroll
              for (int m = 0; m < NF; ++m) {
                typename O::Frag bh;
#pragma unroll
                for (int h = 0; h < S::NH; ++h) bh.h[h] = hhq[m][S::NH * p + h][jj];
                Wb.t[m][jj][ib] = O::mma(Wb.t[m][jj][ib], fk, bh);
              }
            }
            sched_fence();
          }
        // dk += Hh W1 (over the hidden index)
#pragma unroll
        for (int m = 0; m < NF; ++m) {
          const auto& w1q = w0q[m];
          jround<S>(dkacc, nullptr, ja, jw, [&](int tb, int jj) { return hhq[m][tb][jj]; },
                    [&](int ib, int jj) { return w1q[jj][ib]; }, w, g, c);
        }
        const float ksign = (resln && rank == 0) ? -1.0f : 0.0f;
        if constexpr (S::NS > 1) {
          jacc_store_part<S>(dkacc, bwd_part<S>(bwd_slot<S>(E2TTT_ARG(xbuf), px.xs, rank, par), 1),
                            [&](int t, int i) { return ksign * ek[t * D + i]; }, w, g, c);
        } else {
          jacc_store_io<S>(dkacc, E2TTT_ARG(dk), row0, len,
                           [&](int t, int i) { return ksign * ek[t * D + i]; }, w, g, c);
        }
      }
      __syncthreads();

      // -------------------------------------------- P9: output branch
      {
        E2TTT_LANE_IDS;
        E* xq = xk;                                      // Q [t][i]
        E* xdo = reinterpret_cast<E*>(rr);               // dO [t][i]
        E* ybq = yh;                                     // Yb_Q [t][i]
        E* ybqt = dyt;                                   // Yb_Q^T [i][t]
        E* xqt = yht;                                    // Q^T [i][t]
        // act'(H_Q) factors, as D1 above (SwiGLU: recomputed below; the MLP's
        // GELU'(H_Q) was loaded packed with A_Q at the end of P7)
        f32x4 D1q[SW ? NF : 1][SW ? NTB : 1][SW ? NJB : 1];
        pQ.store(xq, tid);
        pD.store(xdo, tid);
        pZq.store(yk, tid);                             // Z_Q (or Y_Q)
        if (tid < S::CM) row[2 * tid] = prq;
        __syncthreads();
        if (r >= 0) prefetch_k(u, r, kt);              // the next tile (r, kt advanced above)
        transpose_to_it<S>(xqt, xq, tid);
        // Yb_Q = LN backward of dO at the Q rows (dO itself when there is no LN)
#pragma unroll
        for (int it_ = 0; it_ < (S::CM + 4 * NW - 1) / (4 * NW); ++it_) {
          const int t0 = 4 * w + it_ * 4 * NW;
          if (t0 < S::CM) {
          const int t = t0 + (lane >> 4);
          float dov[EPL], yb[EPL];
#pragma unroll
          for (int q = 0; q < EPL; ++q) dov[q] = O::from_e(xdo[t * S::LDD + l16 * EPL + q]);
          if (resln) {
            const float sig = row[2 * t];
            float z[EPL], m1 = 0.0f, m2 = 0.0f;
            if (E2TTT_ARG(ln_a)) {   // o = q + a z_q + b: the LayerNorm backward takes a dO
              float la[EPL];
              load_row_part<EPL>(la, E2TTT_ARG(ln_a) + (u % E2TTT_ARG(H)) * D + l16 * EPL);
#pragma unroll
              for (int q = 0; q < EPL; ++q) dov[q] *= la[q];
            }
#pragma unroll
            for (int q = 0; q < EPL; ++q) {
              z[q] = yk[t * D + l16 * EPL + q];
              m1 += dov[q];
              m2 += dov[q] * z[q];
            }
            m1 = group16_sum(m1) * inv_d;
            m2 = group16_sum(m2) * inv_d;
#pragma unroll
            for (int q = 0; q < EPL; ++q) yb[q] = (dov[q] - m1 - z[q] * m2) * sig;
          } else {
#pragma unroll
            for (int q = 0; q < EPL; ++q) yb[q] = dov[q];
          }
          store_row_ti<S, EPL>(ybq, S::LDD, t, l16 * EPL, yb);
          store_row_it<S, EPL>(ybqt, t, l16 * EPL, yb);
                  }
        }
        if constexpr (SW) {   // the SwiGLU query side is recomputed from W_0
          const auto& w1q = w0q;
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj) {
              f32x4 acc[NF];
#pragma unroll
              for (int m = 0; m < NF; ++m) acc[m] = zero4();
#pragma unroll
              for (int p = 0; p < S::KS_D; ++p) {
                auto af = lds_frag<S::BF>(xq, S::LDD, 16 * tb + c, p * S::KC, g);
#pragma unroll
                for (int m = 0; m < NF; ++m) {
                  typename O::Frag bf;
#pragma unroll
                  for (int h = 0; h < S::NH; ++h) bf.h[h] = w1q[m][jj][S::NH * p + h];
                  acc[m] = O::mma(acc[m], af, bf);
                }
              }
              f32x4 act;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const float hg = acc[0][q], hu = acc[1][q], sg = sigm_f(hg);
                D1q[1][tb][jj][q] = hg * sg;
                D1q[0][tb][jj][q] = hu * sg * (1.0f + hg * (1.0f - sg));
                act[q] = hg * sg * hu;
              }
              Aqq[tb][jj] = O::cvt(act);
              sched_fence();
            }
        }
        __syncthreads();
        // Ab_Q = Yb_Q W2;  Hb_Q = Ab_Q act'(H_Q);  Wb2 += Yb_Q^T A_Q;  Wb1 += Q^T Hb_Q
        Q Hbq[NF][NTB][NJB];
        {
          const auto& w2q = w0q[SEC];
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj) {
              f32x4 ab = zero4();
#pragma unroll
              for (int p = 0; p < S::KS_D; ++p) {
                auto af = lds_frag<S::BF>(ybq, S::LDD, 16 * tb + c, p * S::KC, g);
                typename O::Frag bf;
#pragma unroll
                for (int h = 0; h < S::NH; ++h) bf.h[h] = w2q[jj][S::NH * p + h];
                ab = O::mma(ab, af, bf);
              }
              f32x4 hb[NF];
              if constexpr (SW) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                  for (int m = 0; m < NF; ++m) hb[m][q] = ab[q] * D1q[m][tb][jj][q];
              } else {
                const f32x4 d1 = DerivQ<S::BF>::unpack(D1p[tb][jj]);
#pragma unroll
                for (int q = 0; q < 4; ++q) hb[0][q] = ab[q] * d1[q];
              }
#pragma unroll
              for (int m = 0; m < NF; ++m) Hbq[m][tb][jj] = O::cvt(hb[m]);
              sched_fence();
            }
        }
        opaque_state<S>(Wb);
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
          for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
            for (int p = 0; p < S::KS_C; ++p) {
              typename O::Frag ba;
#pragma unroll
              for (int h = 0; h < S::NH; ++h) ba.h[h] = Aqq[S::NH * p + h][jj];
              const int rowi = 16 * ib + c, k0 = p * S::KC;
              Wb.t[SEC][jj][ib] = O::mma(Wb.t[SEC][jj][ib], it_frag<S>(ybqt, rowi, k0, g), ba);
              auto fq = it_frag<S>(xqt, rowi, k0, g);
#pragma unroll
              for (int m = 0; m < NF; ++m) {
                typename O::Frag bh;
#pragma unroll
                for (int h = 0; h < S::NH; ++h) bh.h[h] = Hbq[m][S::NH * p + h][jj];
                Wb.t[m][jj][ib] = O::mma(Wb.t[m][jj][ib], fq, bh);
              }
            }
            sched_fence();
          }
        // dq = dO (residual) + Hb_Q W1 (over the hidden index)
        JAcc<S> dqacc;
        dqacc.zero();
#pragma unroll
        for (int m = 0; m < NF; ++m) {
          const auto& w1q = w0q[m];
          jround<S>(dqacc, nullptr, ja, jw, [&](int tb, int jj) { return Hbq[m][tb][jj]; },
                    [&](int ib, int jj) { return w1q[jj][ib]; }, w, g, c);
        }
        const float qsign = (resln && rank == 0) ? 1.0f : 0.0f;
        if constexpr (S::NS > 1) {
          jacc_store_part<S>(dqacc, bwd_part<S>(bwd_slot<S>(E2TTT_ARG(xbuf), px.xs, rank, par), 2),
                            [&](int t, int i) { return qsign * O::from_e(xdo[t * S::LDD + i]); },
                            w, g, c);
        } else {
          jacc_store_io<S>(dqacc, E2TTT_ARG(dq), row0, len,
                           [&](int t, int i) { return qsign * O::from_e(xdo[t * S::LDD + i]); },
                           w, g, c);
        }
      }

      // ------------------------------ P10: scalar-kernel adjoints of this chunk
      {
      E2TTT_LANE_IDS;
#pragma unroll 1
      for (int t = tid; t < len; t += S::NT) {
        float sw = 0.0f, sm2 = 0.0f;
        for (int ww = 0; ww < NW; ++ww) {
          sw += kb[(0 * NW + ww) * S::CM + t];
          sm2 += kb[(1 * NW + ww) * S::CM + t];
        }
        kwb_slot[row0 + t] = sw;
        kmb_slot[row0 + t] = sm2;
      }
      if (firstp && tid < 3) {
        float sacc = 0.0f;
        for (int ww = 0; ww < NW; ++ww) sacc += cbp[ww * 4 + tid];
        carryb_slot[(u * NC + rc) * 3 + tid] = sacc;
      }
      }
      // The dk, dq partials stored above go out with the next post (the next
      // tile's dYh post, or the one after the unit's last tile): the peers
      // read them only after that post anyway, and a post here would wait
      // for every memory operation in flight (the next tile's loads among
      // them).  The barrier guards the LDS regions that the next tile's
      // staging rewrites.
      __syncthreads();
      if constexpr (S::NS > 1) {
        pend_s0 = s0;
        pend_len = len;
        pend_par = par;
      }
    }

    if constexpr (S::NS > 1) {
      E2TTT_LANE_IDS;
      px.post();                                    // the last tile's dk, dq partials
      px.wait_for(px.seq_now(), sword);             // the peers'
      if (pend_s0 >= 0)
        flush_dkdq<S>(px.xs, pend_par, u * T + pend_s0, pend_len, rlo, tid);
      __syncthreads();
    }
    // w_in also sets the targets t_r = |w_in,r|: d_w_in,r += (sum over the
    // chunks of A_r / t_r) w_in,r / t_r
    if (PN) {
      E2TTT_LANE_IDS;
      const long R = (long)NF * dh + D;
      const float* tg = E2TTT_ARG(norm_tgt) + u * R;
      const float* rbar = E2TTT_ARG(norm_rbar) + (u * S::NS + rank) * R;
      // the second-layer factors through LDS (each was written by thread tid)
      if (tid < D) {
        const float t = tg[(long)NF * dh + tid];
        yk[tid] = t > 0.0f ? rbar[(long)NF * dh + tid] / t : 0.0f;
      }
      __syncthreads();
      StateTiles<S> X;
      load_state<S>(X, E2TTT_ARG(w_in) + u * a.P, dh, j0, w, g, c);
#pragma unroll
      for (int m = 0; m < NF; ++m)
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj) {
          // the factor of column j, read by the lane that wrote it (g = 0, lane c)
          const int j = j0 + 16 * (w * NJB + jj) + c;
          float f = 0.0f;
          if (g == 0 && j < dh) {
            const float t = tg[(long)m * dh + j];
            f = t > 0.0f ? rbar[(long)m * dh + j] / t : 0.0f;
          }
          f = __shfl(f, c);
#pragma unroll
          for (int ib = 0; ib < NIB; ++ib) Wb.t[m][jj][ib] += f * X.t[m][jj][ib];
        }
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        const f32x4 f = *reinterpret_cast<const f32x4*>(&yk[16 * ib + 4 * g]);
#pragma unroll
        for (int jj = 0; jj < NJB; ++jj) Wb.t[SEC][jj][ib] += f * X.t[SEC][jj][ib];
      }
      __syncthreads();   // yk is staged by the next unit
    }
    {
      E2TTT_LANE_IDS;
      store_state<S>(Wb, E2TTT_ARG(d_w_in) + u * a.P, dh, j0, w, g, c);
      store_state<S>(Mb, E2TTT_ARG(d_m_in) + u * a.P, dh, j0, w, g, c);
    }
  }
}

template <class S, bool LONG, bool PN>
int occupancy() {
  int v = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, chain_bwd_kernel<S, LONG, PN>, S::NT, 0) !=
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
    hipLaunchKernelGGL((chain_bwd_kernel<S, LONG, PN>), dim3((unsigned)a.U), dim3(S::NT), 0, stream,
                       a);
    return hipGetLastError();
  } else {
    ChainArgs b = a;
    void* args[] = {&b};
    return hipLaunchCooperativeKernel((const void*)chain_bwd_kernel<S, LONG, PN>,
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
  if (!a.bfrz) return hipErrorInvalidValue;
  return launch_as<S, true, PN>(a, stream);
}

}  // namespace

#define E2TTT_CASE(FW, D, NW, NJB, NTB, BF, NS)                                          \
  if (cfg.fw == FW && cfg.d == D && cfg.nw == NW && cfg.njb == NJB && cfg.ntb == NTB && \
      cfg.bf == BF && cfg.ns == NS)                                                     \
    return launch<Shape<FW, D, NW, NJB, NTB, BF, NS>>(a, stream);

hipError_t E2TTT_PN_NAME(launch_chain_bwd)(const ChainConfig& cfg, const ChainArgs& a,
                                      hipStream_t stream) {
#if !E2TTT_CHAIN_PN
  if (cfg.pn) return launch_chain_bwd_pn(cfg, a, stream);
#endif
#include "chain_variants.inc"
  return hipErrorInvalidValue;
}
#undef E2TTT_CASE

#define E2TTT_CASE(FW, D, NW, NJB, NTB, BF, NS)                                          \
  if (cfg.fw == FW && cfg.d == D && cfg.nw == NW && cfg.njb == NJB && cfg.ntb == NTB && \
      cfg.bf == BF && cfg.ns == NS)                                                     \
    return max_blocks_per_cu<Shape<FW, D, NW, NJB, NTB, BF, NS>>();

int E2TTT_PN_NAME(chain_bwd_blocks_per_cu)(const ChainConfig& cfg) {
#if !E2TTT_CHAIN_PN
  if (cfg.pn) return chain_bwd_blocks_per_cu_pn(cfg);
#endif
#include "chain_variants.inc"
  return 0;
}
#undef E2TTT_CASE

}  // namespace e2ttt
