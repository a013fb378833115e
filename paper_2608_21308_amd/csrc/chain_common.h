// Shape constants and register-resident state handling shared by the forward
// and backward chain kernels.
//
// NS workgroups (1 to 8) own one (batch, head) unit for the whole sequence;
// rank r of them holds the hidden columns [r DHP, (r+1) DHP).  Its NW waves
// split that range: wave w owns the local hidden columns j in
// [16 w NJB, 16 (w+1) NJB).  Every fast-weight matrix is held as 16x16
// MFMA accumulator tiles with the head index i as the tile ROW and the hidden
// index j as the tile COLUMN:
//   first-layer matrices (MLP W1, SwiGLU Wg and Wu, stored [dh][d]) as W^T,
//   the second-layer matrix (MLP W2, SwiGLU Wd, stored [d][dh]) as W.
// With that orientation every update sum_t c_t delta_t x_t^T of Prop. 1 is an
// MFMA whose accumulator IS the state tile, and every contraction over i of a
// token tile with a state matrix takes the state tile directly as operand.
#pragma once

#include "e2ttt_device.h"
#include "e2ttt_internal.h"

namespace e2ttt {

template <int FW_, int D_, int NW_, int NJB_, int NTB_, bool BF_, int NS_>
struct Shape {
  static constexpr int FW = FW_;
  static constexpr int D = D_;
  static constexpr int NW = NW_;
  static constexpr int NJB = NJB_;
  static constexpr int NTB = NTB_;
  static constexpr bool BF = BF_;
  static constexpr int NS = NS_;              // workgroups per unit
  using O = OpT<BF>;
  using E = typename O::E;
  static constexpr int KC = O::KC;
  static constexpr int NH = O::NH;
  static constexpr int NIB = D / 16;          // 16-row blocks over the head dim
  static constexpr int CM = 16 * NTB;         // token rows per chunk tile
  static constexpr int DHP = 16 * NW * NJB;   // padded hidden width of one workgroup
  static constexpr int DHK = ((DHP + KC - 1) / KC) * KC;  // hidden extent of LDS operands
  static constexpr int NMAT = (FW == 0) ? 2 : 3;
  static constexpr int NT = NW * 64;
  static constexpr int LDD = D + O::PAD;      // [t][i] operands
  static constexpr int LDC = CM + O::PAD;     // [i][t] operands
  static constexpr int LDH = DHK + O::PAD;    // [t][j] and [i][j] operands
  static constexpr int KS_D = D / KC;         // K-steps over i
  static constexpr int KS_C = CM / KC;        // K-steps over t
  static constexpr int KS_H = DHK / KC;       // K-steps over j
  static constexpr int IBB = (NIB >= 2) ? 2 : 1;  // head blocks per wave item in j-contractions
  static constexpr int CKPT = NMAT * DHP * D; // checkpoint elements per state
  static_assert(D % KC == 0, "head dim must be a multiple of the K-step");
  static_assert(CM % KC == 0, "chunk tile must be a multiple of the K-step");
};

// Token rows of a chunk tile whose outputs one of the NS ranks of a unit
// writes: rows [rank R, min(CM, (rank + 1) R)), R a multiple of four so that
// the four-row steps of the row phases never straddle two ranks.
template <class S>
__host__ __device__ constexpr int row_share() {
  return ((S::CM + S::NS - 1) / S::NS + 3) / 4 * 4;
}

// State tiles of one wave: T[m][jj][ib] is the tile (rows i = 16 ib + 4 g + r,
// column j = j0 + 16 (w NJB + jj) + c, j0 = rank DHP) of matrix m.
template <class S>
struct StateTiles {
  f32x4 t[S::NMAT][S::NJB][S::NIB];
};

// Marks every state tile as possibly modified, so that conversions of the
// tiles made before this point are not reused (and kept live) after it.
template <class S>
__device__ __forceinline__ void opaque_state(StateTiles<S>& st) {
#pragma unroll
  for (int m = 0; m < S::NMAT; ++m)
#pragma unroll
    for (int jj = 0; jj < S::NJB; ++jj)
#pragma unroll
      for (int ib = 0; ib < S::NIB; ++ib) asm volatile("" : "+v"(st.t[m][jj][ib]));
}

// A field of the chain kernels' argument block (their only parameter, at
// offset 0 of the kernel-argument segment), read from that segment where it
// is used.  Read as `a.field`, every pointer of the block stays in scalar
// registers for the whole kernel; with the chunk loop's own scalar values that
// overflows the scalar register file, and the compiler parks the block in
// vector-register lanes and reads whole register tuples back at every use.
// A scalar load at the use (one instruction, served from the scalar cache)
// keeps each value live only where it is needed.
template <class T>
__device__ __forceinline__ T chain_arg(int off) {
  typedef __attribute__((address_space(4))) const char KChar;
  KChar* kp = (KChar*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(kp));
  return *reinterpret_cast<__attribute__((address_space(4))) const T*>(kp + off);
}
#define E2TTT_ARG(f) \
  ::e2ttt::chain_arg<decltype(::e2ttt::ChainArgs::f)>((int)offsetof(::e2ttt::ChainArgs, f))

// Element (i, j) of matrix m of one unit's P parameters lives at
//   first layer  [dh][d]: m dh d + j d + i
//   second layer [d][dh]: (NMAT-1) dh d + i dh + j.
// The per-lane part of the offset is formed once and kept opaque so that the
// compiler does not materialise one 64-bit address per element.
template <class S, bool STORE>
__device__ __forceinline__ void state_io(StateTiles<S>& st, const float* src, float* dst,
                                         int dh, int j0, int w, int g, int c) {
  constexpr int D = S::D;
  const int jl = j0 + 16 * w * S::NJB + c;                 // this lane's first hidden column
  const int l1 = opaque_lane(jl * D + 4 * g);              // first-layer lane offset
  const int l2 = opaque_lane(4 * g * dh + jl);             // second-layer lane offset
#pragma unroll
  for (int m = 0; m < S::NMAT; ++m)
#pragma unroll
    for (int jj = 0; jj < S::NJB; ++jj) {
      const bool ok = (jl + 16 * jj) < dh;
#pragma unroll
      for (int ib = 0; ib < S::NIB; ++ib) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          long off;
          if (m < S::NMAT - 1) off = (long)m * dh * D + l1 + jj * 16 * D + 16 * ib + r;
          else off = (long)(S::NMAT - 1) * dh * D + l2 + (long)(16 * ib + r) * dh + 16 * jj;
          if constexpr (STORE) {
            if (ok) dst[off] = st.t[m][jj][ib][r];
          } else {
            st.t[m][jj][ib][r] = (ok && src) ? src[off] : 0.0f;
          }
        }
      }
    }
}

template <class S>
__device__ __forceinline__ void load_state(StateTiles<S>& st, const float* src, int dh, int j0,
                                           int w, int g, int c) {
  state_io<S, false>(st, src, nullptr, dh, j0, w, g, c);
}

template <class S>
__device__ __forceinline__ void store_state(StateTiles<S>& st, float* dst, int dh, int j0, int w,
                                            int g, int c) {
  state_io<S, true>(st, nullptr, dst, dh, j0, w, g, c);
}

// Checkpoint blocks hold the chunk-start state in the operand precision
// (bf16 on the bf16 path, fp32 on the fp32 path) and in register order: quad
// ((m NJB + jj) NIB + ib) NW 64 + w 64 + lane, so that writes and reads are
// one 8- or 16-byte access per lane and fully coalesced.
template <class S>
__device__ __forceinline__ void store_ckpt(const StateTiles<S>& st, void* dst, int w, int lane) {
  using Q = typename S::O::Q;
  Q* lp = reinterpret_cast<Q*>(dst) + opaque_lane(w * 64 + lane);
#pragma unroll
  for (int m = 0; m < S::NMAT; ++m)
#pragma unroll
    for (int jj = 0; jj < S::NJB; ++jj)
#pragma unroll
      for (int ib = 0; ib < S::NIB; ++ib)
        st_stream(lp + ((m * S::NJB + jj) * S::NIB + ib) * S::NW * 64, S::O::cvt(st.t[m][jj][ib]));
}

// Quads of matrix m of a checkpoint block, for this lane.
template <class S>
__device__ __forceinline__ void load_ckpt_mat(typename S::O::Q (&q)[S::NJB][S::NIB],
                                              const void* src, int m, int w, int lane) {
  using Q = typename S::O::Q;
  const Q* lp = reinterpret_cast<const Q*>(src) + opaque_lane(w * 64 + lane);
#pragma unroll
  for (int jj = 0; jj < S::NJB; ++jj)
#pragma unroll
    for (int ib = 0; ib < S::NIB; ++ib)
      q[jj][ib] = ld_stream(lp + ((m * S::NJB + jj) * S::NIB + ib) * S::NW * 64);
}

template <class Q>
__device__ __forceinline__ f32x4 quad_f32(const Q& q) {
  return f32x4{(float)q[0], (float)q[1], (float)q[2], (float)q[3]};
}
// bf16 quads widen by moving each half-word into the high half of a word: one
// shift or mask per element, read straight from the packed pair.
__device__ __forceinline__ f32x4 quad_f32(const bf16x4& q) {
  typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
  const u32x2 u = __builtin_bit_cast(u32x2, q);
  return f32x4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
               __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
}

// An operand quad from fp32 values (converted) or from a quad already in the
// operand precision (passed through).
template <class S>
__device__ __forceinline__ typename S::O::Q as_quad(const f32x4& x) {
  return S::O::cvt(x);
}
template <class S, class Q,
          typename std::enable_if<!std::is_same<Q, f32x4>::value, int>::type = 0>
__device__ __forceinline__ Q as_quad(const Q& q) {
  return q;
}

// Operand fragment whose contraction index is the tile ROW of `tiles`
// (tiles[k-block]) for K-step p.
template <class S>
__device__ __forceinline__ typename S::O::Frag tile_frag(const f32x4* tiles, int p,
                                                         int stride) {
  typename S::O::Frag f;
#pragma unroll
  for (int h = 0; h < S::NH; ++h) f.h[h] = S::O::cvt(tiles[(S::NH * p + h) * stride]);
  return f;
}

// acc += af * (fragment of fp32 state tiles, as operand).  On the bf16 path
// the state operand is split into bf16 high and low parts (x = hi + lo to
// about 16 significant bits) and both are multiplied: one more MFMA and a few
// conversions buy an operand as precise as the fp32 state for the products
// whose rounding drives the drift of the chunk chain.
template <class S>
__device__ __forceinline__ f32x4 mma_state(f32x4 acc, const typename S::O::Frag& af,
                                           const f32x4* tiles, int p, int stride) {
  using O = typename S::O;
  if constexpr (S::BF) {
    typename O::Frag hi, lo;
#pragma unroll
    for (int h = 0; h < S::NH; ++h) {
      const f32x4 v = tiles[(S::NH * p + h) * stride];
      hi.h[h] = O::cvt(v);
      lo.h[h] = O::cvt(v - quad_f32(hi.h[h]));
    }
    acc = O::mma(acc, af, hi);
    return O::mma(acc, af, lo);
  } else {
    return O::mma(acc, af, tile_frag<S>(tiles, p, stride));
  }
}

// bf16 high and low parts (x = hi + lo to about 16 significant bits) of
// every state tile, formed once per chunk when the same state is an MFMA
// operand several times; the high part is also the operand-precision copy
// (checkpoint, LDS operand).
template <class S>
struct SplitTiles {
  typename S::O::Q hi[S::NMAT][S::NJB][S::NIB];
  typename S::O::Q lo[S::NMAT][S::NJB][S::NIB];
};
template <class S>
__device__ __forceinline__ void split_state(SplitTiles<S>& sp, const StateTiles<S>& st) {
#pragma unroll
  for (int m = 0; m < S::NMAT; ++m)
#pragma unroll
    for (int jj = 0; jj < S::NJB; ++jj)
#pragma unroll
      for (int ib = 0; ib < S::NIB; ++ib) {
        const f32x4 v = st.t[m][jj][ib];
        sp.hi[m][jj][ib] = S::O::cvt(v);
        sp.lo[m][jj][ib] = S::O::cvt(v - quad_f32(sp.hi[m][jj][ib]));
      }
}
// acc += af * (hi + lo) for K-step p of the pre-split tiles of one (m, jj).
template <class S>
__device__ __forceinline__ f32x4 mma_split(f32x4 acc, const typename S::O::Frag& af,
                                           const typename S::O::Q* hi,
                                           const typename S::O::Q* lo, int p) {
  typename S::O::Frag fh, fl;
#pragma unroll
  for (int h = 0; h < S::NH; ++h) {
    fh.h[h] = hi[S::NH * p + h];
    fl.h[h] = lo[S::NH * p + h];
  }
  acc = S::O::mma(acc, af, fh);
  return S::O::mma(acc, af, fl);
}
// Checkpoint block from pre-converted quads (same layout as store_ckpt).
template <class S>
__device__ __forceinline__ void store_ckpt_q(const typename S::O::Q (&q)[S::NMAT][S::NJB][S::NIB],
                                             void* dst, int w, int lane) {
  using Q = typename S::O::Q;
  Q* lp = reinterpret_cast<Q*>(dst) + opaque_lane(w * 64 + lane);
#pragma unroll
  for (int m = 0; m < S::NMAT; ++m)
#pragma unroll
    for (int jj = 0; jj < S::NJB; ++jj)
#pragma unroll
      for (int ib = 0; ib < S::NIB; ++ib)
        st_stream(lp + ((m * S::NJB + jj) * S::NIB + ib) * S::NW * 64, q[m][jj][ib]);
}

// EPL consecutive fp32 values from global memory (one vector load when EPL = 4).
template <int EPL>
__device__ __forceinline__ void load_row_part(float (&dst)[EPL], const float* src) {
  if constexpr (EPL == 4) {
    const float4 v = *reinterpret_cast<const float4*>(src);
    dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
  } else {
#pragma unroll
    for (int q = 0; q < EPL; ++q) dst[q] = src[q];
  }
}

// Saved activation derivatives: fp16 quads on the bf16 path (2^-11 relative,
// below the bf16 rounding of the MFMA operands they scale), fp32 on the fp32 path.
template <bool BF> struct DerivQ {
  using T = f16x4;
  static __device__ __forceinline__ T pack(f32x4 v) { return __builtin_convertvector(v, f16x4); }
  static __device__ __forceinline__ f32x4 unpack(T v) { return __builtin_convertvector(v, f32x4); }
};
template <> struct DerivQ<false> {
  using T = f32x4;
  static __device__ __forceinline__ T pack(f32x4 v) { return v; }
  static __device__ __forceinline__ f32x4 unpack(T v) { return v; }
};

// Layout of one saved-activation block (one unit's workgroup, one chunk; GELU
// MLP): two sections of NQ entries in register order, entry
// ((tb NJB + jj) NW + w) 64 + lane: A_Q (operand quads), then GELU'(H_Q).
template <class S>
struct SavedAct {
  using Q = typename S::O::Q;
  using DQ = typename DerivQ<S::BF>::T;
  static constexpr int NQ = S::NTB * S::NJB * S::NW * 64;
  char* base;
  __device__ SavedAct(void* block) : base(static_cast<char*>(block)) {}
  static __device__ __forceinline__ int idx(int tb, int jj, int w, int lane) {
    return ((tb * S::NJB + jj) * S::NW + w) * 64 + lane;
  }
  __device__ Q* aq() const { return reinterpret_cast<Q*>(base); }
  __device__ DQ* d1q() const { return reinterpret_cast<DQ*>(base + (long)NQ * sizeof(Q)); }
};

// 16 bytes into a padded [t][i] row.  Rows of the bf16 path are only 8-byte
// aligned (the row padding is 8 bytes), so the vector goes out as two 8-byte
// stores there.
template <class S>
__device__ __forceinline__ void store_row16(typename S::E* dst, const uint4& x) {
  if constexpr ((S::LDD * sizeof(typename S::E)) % 16 == 0) {
    *reinterpret_cast<uint4*>(dst) = x;
  } else {
    reinterpret_cast<uint2*>(dst)[0] = make_uint2(x.x, x.y);
    reinterpret_cast<uint2*>(dst)[1] = make_uint2(x.z, x.w);
  }
}

// Operands of the contractions over the hidden index (the forward's Y = A W2^T,
// the backward's j-rounds).  Both operands (activations [t][j], weights [i][j])
// come from accumulator-layout tiles: lane (g, c) of a wave holds rows
// 4 g .. 4 g + 3 of a 16-row block at one hidden column.  On the bf16 path
// that quad is stored with one 8-byte write, quad (block b, row quad q, hidden
// column k) at quad offset (4 b + q) LD + k (the bytes of a [16 NB][LD]
// array), and a lane's operand fragment (row c of block b, contraction indices
// k0 + 16 h + 4 g + 0..3 for h = 0, 1, the order lds_frag reads) comes back
// through two transposing LDS reads (ds_read_b64_tr_b16: within each group of
// 16 lanes, lane c receives element c mod 4 of the quads addressed by lanes
// 4 r + c / 4, r = 0..3; measured on the MI355X).  With LD = 4 (mod 16) the
// stores (16 lanes on 16 consecutive quads) and the reads (four quad rows, four
// consecutive quads each) fall on 32 distinct banks.  On the fp32 path the
// arrays stay row-major, one element per store.
template <class S, int LD>
__device__ __forceinline__ void jq_put(typename S::E* buf, int blk, int g, int k,
                                       const typename S::O::Q& v) {
  static_assert(!S::BF || LD % 16 == 4, "bf16 quad rows 4 (mod 16) quads apart");
  if constexpr (S::BF) {
    *reinterpret_cast<typename S::O::Q*>(buf + ((4 * blk + g) * LD + k) * 4) = v;
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) buf[(16 * blk + 4 * g + r) * LD + k] = v[r];
  }
}
// A lane's read position in block blk of a j-round operand array (formed once
// per block; the K-steps then add constant offsets).
template <class S, int LD>
__device__ __forceinline__ const typename S::E* jq_lane(const typename S::E* buf, int blk, int g,
                                                        int c) {
  if constexpr (S::BF) return buf + ((4 * blk + (c & 3)) * LD + 4 * g + (c >> 2)) * 4;
  else return buf + (16 * blk + c) * LD + 4 * g;
}
// The operand fragment at K-step offset k0 from a lane's read position.
template <class S>
__device__ __forceinline__ typename S::O::Frag jq_frag(const typename S::E* pos, int k0) {
  typename S::O::Frag f;
  if constexpr (S::BF) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s4* lds_s4;
#pragma unroll
    for (int h = 0; h < S::O::NH; ++h) {
      typename S::E* p = const_cast<typename S::E*>(pos) + (k0 + 16 * h) * 4;
      f.h[h] = __builtin_bit_cast(typename S::O::Q, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)p));
    }
  } else {
#pragma unroll
    for (int h = 0; h < S::O::NH; ++h)
      f.h[h] = *reinterpret_cast<const typename S::O::Q*>(pos + k0 + 16 * h);
  }
  return f;
}
// Zero quads at hidden columns [k_lo, KW) of nb_a + nb_w 16-row blocks of two
// operand arrays (columns no wave owns must read as zero).
template <class S, int LD, int KW>
__device__ __forceinline__ void jq_zero_cols(typename S::E* a, int nb_a, typename S::E* b, int nb_w,
                                             int k_lo) {
  const int nz = KW - k_lo;
  const typename S::O::Q z = S::O::cvt(zero4());
#pragma unroll 1
  for (int idx = threadIdx.x; idx < 4 * (nb_a + nb_w) * nz; idx += S::NT) {
    const int rq = idx / nz, k = k_lo + idx % nz;
    if (rq < 4 * nb_a) jq_put<S, LD>(a, rq / 4, rq % 4, k, z);
    else jq_put<S, LD>(b, (rq - 4 * nb_a) / 4, (rq - 4 * nb_a) % 4, k, z);
  }
}

// [i][t] operands (rows i = head index, columns t = token, the contraction
// index of the state updates).  On the bf16 path they use the quad layout of
// the hidden-index operands above with the token as the K index: quad (head
// block b, head quad q, token t) holds heads 16 b + 4 q .. + 3 of token t, so
// a row phase that holds four consecutive head indices of one token writes
// them with one 8-byte store, and a fragment comes back through the
// transposing reads.  On the fp32 path each row's 4-element quads are
// permuted instead: element (i, t) sits at quad (t / 4) ^ ((i / 16) mod 4) of
// row i, so that the element stores of 16 lanes on rows 4 apart fall on 16
// LDS banks rather than 4; fragment reads stay single paired loads (the
// permutation only moves the lane's quad within its K-step).
template <class S>
__device__ __forceinline__ int it_idx(int i, int t) {
  return i * S::LDC + ((((t >> 2) ^ (i >> 4)) & 3) | ((t >> 2) & ~3)) * 4 + (t & 3);
}
template <class S>
__device__ __forceinline__ typename S::O::Frag it_frag(const typename S::E* base, int row, int k0,
                                                       int g) {
  if constexpr (S::BF) return jq_frag<S>(jq_lane<S, S::LDC>(base, row >> 4, g, row & 15), k0);
  else return lds_frag<S::BF>(base, S::LDC, row, k0, g ^ ((row >> 4) & 3));
}

// Row-phase stores: a lane holds EPL consecutive head indices i0 .. i0+EPL-1
// (i0 a multiple of EPL) of token row t.
// Into a [t][i] operand array (leading dimension ld): one 8-byte store per
// four bf16 values (the rows are 8-byte aligned), element stores otherwise.
template <class S, int EPL>
__device__ __forceinline__ void store_row_ti(typename S::E* dst, int ld, int t, int i0,
                                             const float (&v)[EPL]) {
  if constexpr (S::BF && EPL % 4 == 0) {
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k)
      *reinterpret_cast<typename S::O::Q*>(dst + t * ld + i0 + 4 * k) =
          S::O::cvt(f32x4{v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]});
  } else {
#pragma unroll
    for (int q = 0; q < EPL; ++q) dst[t * ld + i0 + q] = S::O::to_e(v[q]);
  }
}
// Into an [i][t] operand array (it_idx layout), each value scaled by `sc`:
// the EPL rows lie in one 16-row block, so they share the quad permutation and
// sit at one base address plus multiples of the row stride; on the bf16 path
// two values are converted per instruction.
template <class S, int EPL>
__device__ __forceinline__ void store_row_it(typename S::E* dst, int t, int i0,
                                             const float (&v)[EPL], float sc = 1.0f) {
  static_assert(16 % EPL == 0 || EPL % 16 == 0, "a lane's head indices in whole 16-row blocks");
  if constexpr (S::BF && EPL % 4 == 0) {
    // bf16: four consecutive head indices of one token are one quad of the
    // transposed-read layout: one 8-byte store each
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k) {
      const int i = i0 + 4 * k;
      jq_put<S, S::LDC>(dst, i >> 4, (i >> 2) & 3, t,
                        S::O::cvt(f32x4{sc * v[4 * k], sc * v[4 * k + 1], sc * v[4 * k + 2],
                                        sc * v[4 * k + 3]}));
    }
  } else {
    const int b = it_idx<S>(i0, t);
#pragma unroll
    for (int q = 0; q < EPL; ++q) dst[b + q * S::LDC] = S::O::to_e(sc * v[q]);
  }
}
// EPL consecutive values of a row to global memory (io element type T, or
// fp32): four values per vector store when EPL allows (dst 8- or 16-byte aligned).
template <class IO, int EPL>
__device__ __forceinline__ void store_row_io(typename IO::T* dst, const float (&v)[EPL]) {
  if constexpr (EPL % 4 == 0) {
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k)
      IO::st4(dst + 4 * k, f32x4{v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]});
  } else {
#pragma unroll
    for (int q = 0; q < EPL; ++q) IO::st(dst + q, v[q]);
  }
}

// [t][i] -> [i][t] (it_idx layout) copy of a CM x D operand tile, four tokens
// of one head index per item (one quad store).
template <class S>
__device__ __forceinline__ void transpose_to_it(typename S::E* dst, const typename S::E* src,
                                                int tid) {
  if constexpr (S::BF) {
    // bf16: a row quad of [t][i] (four consecutive head indices of one token)
    // is a quad of the transposed-read layout as it stands: copied whole
#pragma unroll 1
    for (int idx = tid; idx < S::CM * (S::D / 4); idx += S::NT) {
      const int t = idx / (S::D / 4), i = 4 * (idx % (S::D / 4));
      jq_put<S, S::LDC>(dst, i >> 4, (i >> 2) & 3, t,
                        *reinterpret_cast<const typename S::O::Q*>(src + t * S::LDD + i));
    }
    return;
  }
#pragma unroll 1
  for (int idx = tid; idx < S::D * (S::CM / 4); idx += S::NT) {
    const int i = idx % S::D, t0 = 4 * (idx / S::D);
    typename S::O::Q qv;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) qv[q4] = src[(t0 + q4) * S::LDD + i];
    *reinterpret_cast<typename S::O::Q*>(&dst[it_idx<S>(i, t0)]) = qv;
  }
}

// Copy a CM x D token tile (rows < len, zero beyond) from global io memory to
// LDS in 16-byte vectors (the io element type equals the LDS element type).
template <class S>
__device__ __forceinline__ void stage_tile(typename S::E* dst, const void* src, long row0,
                                           int len, int tid) {
  using IOT = typename IoT<S::BF>::T;
  static_assert(sizeof(IOT) == sizeof(typename S::E), "io and operand types differ");
  constexpr int VE = 16 / sizeof(IOT);
  constexpr int NV = S::CM * S::D / VE;
  const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const IOT*>(src) + row0 * S::D);
#pragma unroll 1
  for (int v = tid; v < NV; v += S::NT) {
    const int e = v * VE, t = e / S::D, i = e % S::D;
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (t < len) x = p[v];
    store_row16<S>(dst + t * S::LDD + i, x);
  }
}

// A CM x D token tile held in registers (16-byte vectors, rows < len, zero
// beyond): the next chunk's inputs are loaded while the current chunk runs and
// written to LDS when it starts, so their global-memory latency is hidden.
template <class S>
struct TileRegs {
  static constexpr int VE = 16 / (int)sizeof(typename S::E);   // elements per vector
  static constexpr int NV = S::CM * S::D / VE;
  static constexpr int PER = (NV + S::NT - 1) / S::NT;
  uint4 v[PER];

  __device__ __forceinline__ void load(const void* src, long row0, int len, int tid) {
    using IOT = typename IoT<S::BF>::T;
    static_assert(sizeof(IOT) == sizeof(typename S::E), "io and operand types differ");
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const IOT*>(src) + row0 * S::D);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = (tid + k * S::NT) * VE;
      v[k] = make_uint4(0u, 0u, 0u, 0u);
      if (e < S::CM * S::D && e / S::D < len) v[k] = ld_stream16(p + tid + k * S::NT);
    }
  }
  __device__ __forceinline__ void store(typename S::E* dst, int tid) const {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = (tid + k * S::NT) * VE;
      if (e < S::CM * S::D) store_row16<S>(dst + (e / S::D) * S::LDD + e % S::D, v[k]);
    }
  }
};

// The same for an fp32 CM x D tile (saved LayerNorm outputs), stored to a
// dense [CM][D] fp32 LDS array.
template <class S>
struct F32TileRegs {
  static constexpr int NV = S::CM * S::D / 4;
  static constexpr int PER = (NV + S::NT - 1) / S::NT;
  float4 v[PER];

  __device__ __forceinline__ void load(const float* src, long row0, int len, int tid) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = (tid + k * S::NT) * 4;
      v[k] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (e < S::CM * S::D && e / S::D < len) v[k] = ld_stream16f(src + row0 * S::D + 4 * (tid + k * S::NT));
    }
  }
  __device__ __forceinline__ void store(float* dst, int tid) const {
#pragma unroll
    for (int k = 0; k < PER; ++k)
      if (tid + k * S::NT < NV) reinterpret_cast<float4*>(dst)[tid + k * S::NT] = v[k];
  }
};

// Y[t][i] = sum_j A[t][j] Wt[i][j]  (j-contraction, both operands in LDS as
// quads, stored with jq_put<S, S::LDH>),
// written to y (fp32 [CM][D]) and, when given, in the same layout to `slot`
// in global memory.  Work is split into (token block, head block pair) items
// over the waves.
template <class S>
__device__ __forceinline__ void jgemm_to_lds(const typename S::E* A, const typename S::E* Wt,
                                             float* y, int w, int g, int c,
                                             float* slot = nullptr) {
  constexpr int NI = S::NIB / S::IBB;
  for (int it = w; it < S::NTB * NI; it += S::NW) {
    const int tb = it / NI, ib0 = (it % NI) * S::IBB;
    f32x4 acc[S::IBB];
#pragma unroll
    for (int b = 0; b < S::IBB; ++b) acc[b] = zero4();
    const typename S::E* pa = jq_lane<S, S::LDH>(A, tb, g, c);
    const typename S::E* pb[S::IBB];
#pragma unroll
    for (int b = 0; b < S::IBB; ++b) pb[b] = jq_lane<S, S::LDH>(Wt, ib0 + b, g, c);
#pragma unroll
    for (int p = 0; p < S::KS_H; ++p) {
      auto af = jq_frag<S>(pa, p * S::KC);
#pragma unroll
      for (int b = 0; b < S::IBB; ++b) {
        auto bf = jq_frag<S>(pb[b], p * S::KC);
        acc[b] = S::O::mma(acc[b], af, bf);
      }
    }
#pragma unroll
    for (int b = 0; b < S::IBB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = (16 * tb + 4 * g + r) * S::D + 16 * (ib0 + b) + c;
        y[e] = acc[b][r];
        if (slot) slot[e] = acc[b][r];
      }
  }
}

}  // namespace e2ttt
