// E2-TTT fp64 CPU oracle.  TEST INFRASTRUCTURE ONLY.
//
// This file is the checker, not the product.  Only the test-suite, the smoke
// check and the CPU-baseline leg of the benchmark load it.  It shares no code,
// header, table or helper with the HIP library: it is written from the paper's
// definitions, in the paper's order, as a plain token-by-token loop in double
// precision.
//
// What it computes (arxiv 2608.21308):
//   * Fast-weight net f_W (Sec. 4, "Fast-weight Network"): GELU MLP
//     f(x) = x + LN(W2 GELU(W1 x)) or SwiGLU f(x) = x + LN(Wd (SiLU(Wg x) * (Wu x))),
//     LayerNorm with biased variance, explicit eps, exact erf GELU.
//     Flag bit 0 drops "x + LN(.)" so that f(x) is the bare matrix net.
//     Optionally a learnable per-head LayerNorm affine (flag bit 2):
//     f(x) = x + a * LN(y) + b with a, b in R^d, slow weights of the head.
//   * Optionally (flag bit 3) the post-chunk L2 normalisation of the fast
//     weights (App. B.1, after Zhang et al.): at every chunk end each row of
//     each fast-weight matrix, taken over the matrix's input dimension, is
//     rescaled to the norm that row has in the unit's initial weights w_in;
//     the momentum is left as it is.  A row of norm zero is left as it is;
//     a row whose target is zero becomes zero.
//   * Inner loss L_t = 1/2 ||f_W(k_t) - v_t||^2 (Sec. 2, eq. (1); the paper
//     names MSE without a constant, see the readings list in the design notes).
//   * Per-token recurrence with gradients frozen at the chunk-start weights
//     (Sec. 3.1, eq. (7)):  M_t = beta_t M_{t-1} + eta_t G_t,
//                           W_t = gamma_t W_{t-1} + M_t,
//     G_t = -grad_W L(f_{W_0}(k_t), v_t), W_0 = state at the chunk start.
//   * Outputs from the chunk-start weights, o_t = f_{W_0}(q_t) (eq. (6),
//     Table 1 "output computed from chunk start").
//   * Backward: reverse mode over that same token loop.  The second-order terms
//     (how G_t moves with W_0, k_t, v_t) are obtained with forward-mode dual
//     numbers run through the first-order gradient code: seeding W_0 with the
//     direction Gbar_t gives the Hessian-vector product (the Hessian of L is
//     symmetric) and the tangent of grad_k L, grad_v L gives the mixed terms.
//     No second derivative is written by hand.
//   * Scalar kernels (Sec. 3.2, eq. (8)-(11), App. A): the per-token weights of
//     G_t in W_C and M_C and the three carries, evaluated straight from the
//     unrolled sums of eq. (8) (products and sums, no division, O(C^2)).
//
// Layout of one unit's P fast-weight parameters (row-major, W x convention):
//   MLP:    W1[dh][d], W2[d][dh]                    P = 2 d dh
//   SwiGLU: Wg[dh][d], Wu[dh][d], Wd[d][dh]         P = 3 d dh
// Tensors are [B][H][T][d] (q, k, v, out), [B][H][T] (gates), [B][H][P] (state).
#include <cmath>
#include <cstring>
#include <vector>
#include <omp.h>

namespace {

// ---------------------------------------------------------------- dual numbers
struct Dual {
  double v, d;
  Dual() : v(0), d(0) {}
  Dual(double x) : v(x), d(0) {}
  Dual(double x, double dx) : v(x), d(dx) {}
};
inline Dual operator+(Dual a, Dual b) { return Dual(a.v + b.v, a.d + b.d); }
inline Dual operator-(Dual a, Dual b) { return Dual(a.v - b.v, a.d - b.d); }
inline Dual operator-(Dual a) { return Dual(-a.v, -a.d); }
inline Dual operator*(Dual a, Dual b) { return Dual(a.v * b.v, a.d * b.v + a.v * b.d); }
inline Dual operator/(Dual a, Dual b) {
  return Dual(a.v / b.v, (a.d * b.v - a.v * b.d) / (b.v * b.v));
}
inline Dual& operator+=(Dual& a, Dual b) { a = a + b; return a; }
inline Dual& operator-=(Dual& a, Dual b) { a = a - b; return a; }
inline Dual exp_(Dual a) { double e = std::exp(a.v); return Dual(e, e * a.d); }
inline Dual erf_(Dual a) {
  const double c = 2.0 / std::sqrt(M_PI);
  return Dual(std::erf(a.v), c * std::exp(-a.v * a.v) * a.d);
}
inline Dual sqrt_(Dual a) { double s = std::sqrt(a.v); return Dual(s, a.d / (2.0 * s)); }
inline double exp_(double a) { return std::exp(a); }
inline double erf_(double a) { return std::erf(a); }
inline double sqrt_(double a) { return std::sqrt(a); }

// --------------------------------------------------------- activation functions
// GELU with the exact normal CDF: gelu(x) = x Phi(x).
template <class T> T gelu(T x) { return 0.5 * x * (1.0 + erf_(x * (1.0 / std::sqrt(2.0)))); }
// d/dx gelu(x) = Phi(x) + x phi(x).
template <class T> T gelu_grad(T x) {
  const double inv_sqrt_2pi = 1.0 / std::sqrt(2.0 * M_PI);
  return 0.5 * (1.0 + erf_(x * (1.0 / std::sqrt(2.0)))) + x * (inv_sqrt_2pi * exp_(-0.5 * x * x));
}
template <class T> T sigmoid(T x) { return 1.0 / (1.0 + exp_(-x)); }
template <class T> T silu(T x) { return x * sigmoid(x); }
// d/dx silu(x) = s (1 + x (1 - s)), s = sigmoid(x).
template <class T> T silu_grad(T x) { T s = sigmoid(x); return s * (1.0 + x * (1.0 - s)); }

struct Net {
  int d, dh, fw;     // fw: 0 = GELU MLP, 1 = SwiGLU
  bool resln;        // true: f(x) = x + a * LN(y) + b; false: f(x) = y
  double eps;
  const double* lna = nullptr;   // LayerNorm affine a[d] of the unit's head (nullptr: a = 1)
  const double* lnb = nullptr;   // and b[d] (nullptr: b = 0)
  long P() const { return (fw == 0 ? 2L : 3L) * d * dh; }
  double a(int i) const { return lna ? lna[i] : 1.0; }
  double b(int i) const { return lnb ? lnb[i] : 0.0; }
};

// f_W(x) and, when fbar != nullptr, its vector-Jacobian product:
//   Wbar += (df/dW)^T fbar,  xbar = (df/dx)^T fbar,
//   and, when given, lnabar += (df/da)^T fbar, lnbbar += (df/db)^T fbar for
//   the LayerNorm affine.
// Every intermediate is recomputed here; the code is the definition written out.
template <class T>
void net_eval(const Net& n, const T* W, const T* x, T* f, const T* fbar, T* Wbar, T* xbar,
              T* lnabar = nullptr, T* lnbbar = nullptr) {
  const int d = n.d, dh = n.dh;
  std::vector<T> h(dh), hu(dh), a(dh), y(d), z(d);
  const T* W1 = W;                       // MLP W1 / SwiGLU Wg   [dh][d]
  const T* Wu = W + (long)dh * d;        // SwiGLU Wu            [dh][d]
  const T* W2 = (n.fw == 0) ? W + (long)dh * d : W + 2L * dh * d;  // W2 / Wd [d][dh]
  for (int j = 0; j < dh; ++j) {
    T s = 0.0;
    for (int i = 0; i < d; ++i) s += W1[(long)j * d + i] * x[i];
    h[j] = s;
    if (n.fw == 1) {
      T su = 0.0;
      for (int i = 0; i < d; ++i) su += Wu[(long)j * d + i] * x[i];
      hu[j] = su;
      a[j] = silu(h[j]) * hu[j];
    } else {
      a[j] = gelu(h[j]);
    }
  }
  for (int i = 0; i < d; ++i) {
    T s = 0.0;
    for (int j = 0; j < dh; ++j) s += W2[(long)i * dh + j] * a[j];
    y[i] = s;
  }
  T sigma = 1.0;
  if (n.resln) {
    T mu = 0.0;
    for (int i = 0; i < d; ++i) mu += y[i];
    mu = mu * (1.0 / d);
    T var = 0.0;
    for (int i = 0; i < d; ++i) var += (y[i] - mu) * (y[i] - mu);
    var = var * (1.0 / d);
    sigma = sqrt_(var + n.eps);
    for (int i = 0; i < d; ++i) {
      z[i] = (y[i] - mu) / sigma;
      f[i] = x[i] + n.a(i) * z[i] + n.b(i);
    }
  } else {
    for (int i = 0; i < d; ++i) f[i] = y[i];
  }
  if (!fbar) return;

  // ---- reverse pass
  std::vector<T> ybar(d), abar(dh), hbar(dh), hubar(dh);
  for (int i = 0; i < d; ++i) xbar[i] = 0.0;
  if (n.resln) {
    // f = x + a z + b  ->  xbar = fbar, zbar = a fbar, abar += fbar z, bbar += fbar;
    // z = (y - mean y)/sigma  ->  ybar = (zbar - mean zbar - z mean(zbar z)) / sigma.
    std::vector<T> zbar(d);
    T m1 = 0.0, m2 = 0.0;
    for (int i = 0; i < d; ++i) {
      zbar[i] = n.a(i) * fbar[i];
      m1 += zbar[i];
      m2 += zbar[i] * z[i];
      if (lnabar) lnabar[i] += fbar[i] * z[i];
      if (lnbbar) lnbbar[i] += fbar[i];
    }
    m1 = m1 * (1.0 / d);
    m2 = m2 * (1.0 / d);
    for (int i = 0; i < d; ++i) {
      xbar[i] = fbar[i];
      ybar[i] = (zbar[i] - m1 - z[i] * m2) / sigma;
    }
  } else {
    for (int i = 0; i < d; ++i) ybar[i] = fbar[i];
  }
  T* W1bar = Wbar;
  T* Wubar = Wbar + (long)dh * d;
  T* W2bar = (n.fw == 0) ? Wbar + (long)dh * d : Wbar + 2L * dh * d;
  for (int j = 0; j < dh; ++j) {
    T s = 0.0;
    for (int i = 0; i < d; ++i) {
      s += W2[(long)i * dh + j] * ybar[i];
      W2bar[(long)i * dh + j] += ybar[i] * a[j];
    }
    abar[j] = s;
    if (n.fw == 1) {
      hbar[j] = abar[j] * hu[j] * silu_grad(h[j]);
      hubar[j] = abar[j] * silu(h[j]);
    } else {
      hbar[j] = abar[j] * gelu_grad(h[j]);
    }
  }
  for (int j = 0; j < dh; ++j) {
    for (int i = 0; i < d; ++i) {
      W1bar[(long)j * d + i] += hbar[j] * x[i];
      xbar[i] += W1[(long)j * d + i] * hbar[j];
      if (n.fw == 1) {
        Wubar[(long)j * d + i] += hubar[j] * x[i];
        xbar[i] += Wu[(long)j * d + i] * hubar[j];
      }
    }
  }
}

// Gradients of the inner loss L = 1/2 ||f_W(k) - v||^2 with respect to W, k, v
// and, when ga / gb are given, the LayerNorm affine a, b.
template <class T>
void loss_grad(const Net& n, const T* W, const T* k, const T* v, T* gW, T* gk, T* gv,
               T* ga = nullptr, T* gb = nullptr) {
  const int d = n.d;
  std::vector<T> f(d), r(d);
  net_eval<T>(n, W, k, f.data(), nullptr, nullptr, nullptr);
  for (int i = 0; i < d; ++i) { r[i] = f[i] - v[i]; gv[i] = -r[i]; }
  const long P = n.P();
  for (long p = 0; p < P; ++p) gW[p] = 0.0;
  if (ga) for (int i = 0; i < d; ++i) { ga[i] = 0.0; gb[i] = 0.0; }
  net_eval<T>(n, W, k, f.data(), r.data(), gW, gk, ga, gb);
}

struct Problem {
  int B, H, T, C;
  Net net;
  bool post_norm = false;   // L2-normalise the fast-weight rows at every chunk end
  long units() const { return (long)B * H; }
};

// Rows of the fast-weight matrices for the post-chunk normalisation: row r of
// a matrix laid out [rows][cols] with the input index as the column (W x rule):
// MLP W1 [dh][d], W2 [d][dh]; SwiGLU Wg, Wu [dh][d], Wd [d][dh].  Calls
// f(offset of the row's first element, number of columns) for every row.
template <class F>
void for_each_row(const Net& n, F f) {
  const int nmat = n.fw == 0 ? 2 : 3;
  long off = 0;
  for (int m = 0; m < nmat; ++m) {
    const bool second = (m == nmat - 1);
    const int rows = second ? n.d : n.dh, cols = second ? n.dh : n.d;
    for (int r = 0; r < rows; ++r) f(off + (long)r * cols, cols);
    off += (long)rows * cols;
  }
}

double row_norm(const double* x, int cols) {
  double s = 0.0;
  for (int c = 0; c < cols; ++c) s += x[c] * x[c];
  return std::sqrt(s);
}

// W <- every row rescaled from its norm to the norm of the same row of W_init.
void post_chunk_normalise(const Net& n, const double* w_init, double* W) {
  for_each_row(n, [&](long off, int cols) {
    const double nr = row_norm(W + off, cols);
    if (nr == 0.0) return;
    const double s = row_norm(w_init + off, cols) / nr;
    for (int c = 0; c < cols; ++c) W[off + c] *= s;
  });
}

// Reverse of post_chunk_normalise at the pre-normalisation weights Wpre:
// Wbar (the adjoint of the normalised rows) becomes the adjoint of Wpre, and
// w_init_bar receives what flows into the targets (norm of w_init's rows):
// with u = Wpre_r / |Wpre_r| and t_r = |w_init_r|, the normalised row is t_r u,
// so  Wpre_r_bar = (t_r / |Wpre_r|) (Wbar_r - u <u, Wbar_r>)  and
// w_init_r_bar += <u, Wbar_r> w_init_r / t_r.
void post_chunk_normalise_bwd(const Net& n, const double* w_init, const double* Wpre, double* Wbar,
                              double* w_init_bar) {
  for_each_row(n, [&](long off, int cols) {
    const double nr = row_norm(Wpre + off, cols);
    if (nr == 0.0) return;                      // left as it was: identity
    const double t = row_norm(w_init + off, cols);
    double dot = 0.0;
    for (int c = 0; c < cols; ++c) dot += Wpre[off + c] / nr * Wbar[off + c];
    for (int c = 0; c < cols; ++c) Wbar[off + c] = t / nr * (Wbar[off + c] - Wpre[off + c] / nr * dot);
    if (t > 0.0)
      for (int c = 0; c < cols; ++c) w_init_bar[off + c] += dot * w_init[off + c] / t;
  });
}

// Per-unit forward; optionally records the chunk-start states for the backward.
void unit_forward(const Problem& pb, const double* q, const double* k, const double* v,
                  const double* eta, const double* beta, const double* gamma,
                  const double* w_in, const double* m_in, double* out, double* w_out,
                  double* m_out, std::vector<double>* starts) {
  const Net& n = pb.net;
  const int d = n.d, T = pb.T, C = pb.C;
  const long P = n.P();
  std::vector<double> W(w_in, w_in + P), M(P, 0.0), W0(P), G(P), gk(d), gv(d);
  if (m_in) std::memcpy(M.data(), m_in, sizeof(double) * P);
  std::vector<double> fbuf(d);
  for (int s0 = 0; s0 < T; s0 += C) {
    const int len = (T - s0 < C) ? T - s0 : C;
    W0 = W;
    if (starts) {
      starts->insert(starts->end(), W.begin(), W.end());
      starts->insert(starts->end(), M.begin(), M.end());
    }
    for (int t = s0; t < s0 + len; ++t)      // o_t = f_{W_0}(q_t)
      net_eval<double>(n, W0.data(), q + (long)t * d, out + (long)t * d, nullptr, nullptr, nullptr);
    for (int t = s0; t < s0 + len; ++t) {    // token-by-token recurrence, gradient at W_0
      loss_grad<double>(n, W0.data(), k + (long)t * d, v + (long)t * d, G.data(), gk.data(), gv.data());
      const double e = eta[t], b = beta[t], g = gamma ? gamma[t] : 1.0;
      for (long p = 0; p < P; ++p) {
        M[p] = b * M[p] + e * (-G[p]);
        W[p] = g * W[p] + M[p];
      }
    }
    if (pb.post_norm) post_chunk_normalise(n, w_in, W.data());
  }
  std::memcpy(w_out, W.data(), sizeof(double) * P);
  std::memcpy(m_out, M.data(), sizeof(double) * P);
}

// Per-unit backward of
//   Loss = sum_t <d_out_t, o_t> + <d_w_out, W_T> + <d_m_out, M_T>
// by reverse mode over the token loop of unit_forward.
void unit_backward(const Problem& pb, const double* q, const double* k, const double* v,
                   const double* eta, const double* beta, const double* gamma,
                   const double* w_in, const double* m_in, const double* d_out,
                   const double* d_w_out, const double* d_m_out, double* dq, double* dk,
                   double* dv, double* d_eta, double* d_beta, double* d_gamma,
                   double* d_w_in, double* d_m_in, double* d_lna, double* d_lnb) {
  const Net& n = pb.net;
  const int d = n.d, T = pb.T, C = pb.C;
  const long P = n.P();
  const int NC = (T + C - 1) / C;
  std::vector<double> starts, scratch_out((long)T * d), wo(P), mo(P);
  starts.reserve((size_t)NC * 2 * P);
  unit_forward(pb, q, k, v, eta, beta, gamma, w_in, m_in, scratch_out.data(), wo.data(), mo.data(),
               &starts);

  std::vector<double> Wbar(P, 0.0), Mbar(P, 0.0);
  if (d_w_out) std::memcpy(Wbar.data(), d_w_out, sizeof(double) * P);
  if (d_m_out) std::memcpy(Mbar.data(), d_m_out, sizeof(double) * P);

  std::vector<double> Ws, Ms, Gs;        // token states W_t, M_t (t = 0..len) and G_t
  std::vector<double> gk(d), gv(d), fb(d), xb(d);
  std::vector<Dual> Wd(P), gWd(P), kd(d), vd(d), gkd(d), gvd(d), gad(d), gbd(d);
  std::vector<double> Gbar, winit_bar(P, 0.0);
  for (int c = NC - 1; c >= 0; --c) {
    const int s0 = c * C;
    const int len = (T - s0 < C) ? T - s0 : C;
    const double* W0 = starts.data() + (size_t)c * 2 * P;
    const double* M0 = W0 + P;
    // recompute the chunk: G_t at W_0 and the token states
    Ws.assign((size_t)(len + 1) * P, 0.0);
    Ms.assign((size_t)(len + 1) * P, 0.0);
    Gs.assign((size_t)len * P, 0.0);
    std::memcpy(Ws.data(), W0, sizeof(double) * P);
    std::memcpy(Ms.data(), M0, sizeof(double) * P);
    for (int i = 0; i < len; ++i) {
      const int t = s0 + i;
      double* Gt = Gs.data() + (size_t)i * P;
      loss_grad<double>(n, W0, k + (long)t * d, v + (long)t * d, Gt, gk.data(), gv.data());
      for (long p = 0; p < P; ++p) Gt[p] = -Gt[p];
      const double e = eta[t], b = beta[t], g = gamma ? gamma[t] : 1.0;
      const double* Wp = Ws.data() + (size_t)i * P;
      const double* Mp = Ms.data() + (size_t)i * P;
      double* Wn = Ws.data() + (size_t)(i + 1) * P;
      double* Mn = Ms.data() + (size_t)(i + 1) * P;
      for (long p = 0; p < P; ++p) {
        Mn[p] = b * Mp[p] + e * Gt[p];
        Wn[p] = g * Wp[p] + Mn[p];
      }
    }
    // the chunk end was normalised: Wbar is the adjoint of the normalised
    // weights, turned into that of the token loop's last state
    if (pb.post_norm)
      post_chunk_normalise_bwd(n, w_in, Ws.data() + (size_t)len * P, Wbar.data(),
                               winit_bar.data());
    // reverse through the token loop
    Gbar.assign((size_t)len * P, 0.0);
    for (int i = len - 1; i >= 0; --i) {
      const int t = s0 + i;
      const double e = eta[t], b = beta[t], g = gamma ? gamma[t] : 1.0;
      const double* Wp = Ws.data() + (size_t)i * P;      // W_{t-1}
      const double* Mp = Ms.data() + (size_t)i * P;      // M_{t-1}
      const double* Gt = Gs.data() + (size_t)i * P;
      double* Gb = Gbar.data() + (size_t)i * P;
      // W_t = g W_{t-1} + M_t
      double sg = 0.0;
      for (long p = 0; p < P; ++p) { Mbar[p] += Wbar[p]; sg += Wbar[p] * Wp[p]; Wbar[p] *= g; }
      // M_t = b M_{t-1} + e G_t
      double sb = 0.0, se = 0.0;
      for (long p = 0; p < P; ++p) {
        sb += Mbar[p] * Mp[p];
        se += Mbar[p] * Gt[p];
        Gb[p] = e * Mbar[p];
        Mbar[p] *= b;
      }
      if (d_gamma) d_gamma[t] = sg;
      d_beta[t] = sb;
      d_eta[t] = se;
    }
    // G_t = G(W_0, k_t, v_t): push Gbar_t into W_0, k_t, v_t with dual numbers.
    for (int i = 0; i < len; ++i) {
      const int t = s0 + i;
      const double* Gb = Gbar.data() + (size_t)i * P;
      for (long p = 0; p < P; ++p) Wd[p] = Dual(W0[p], Gb[p]);
      for (int j = 0; j < d; ++j) { kd[j] = Dual(k[(long)t * d + j]); vd[j] = Dual(v[(long)t * d + j]); }
      loss_grad<Dual>(n, Wd.data(), kd.data(), vd.data(), gWd.data(), gkd.data(), gvd.data(),
                      gad.data(), gbd.data());
      // G = -grad_W L, so d<Gbar, G>/dW0 = -(tangent of grad_W L), likewise for k, v
      // and the affine a, b.
      for (long p = 0; p < P; ++p) Wbar[p] -= gWd[p].d;
      for (int j = 0; j < d; ++j) {
        dk[(long)t * d + j] = -gkd[j].d;
        dv[(long)t * d + j] = -gvd[j].d;
        if (d_lna) { d_lna[j] -= gad[j].d; d_lnb[j] -= gbd[j].d; }
      }
    }
    // o_t = f_{W_0}(q_t)
    std::vector<double> Wob(P, 0.0);
    for (int i = 0; i < len; ++i) {
      const int t = s0 + i;
      net_eval<double>(n, W0, q + (long)t * d, fb.data(), d_out + (long)t * d, Wob.data(),
                       dq + (long)t * d, d_lna, d_lnb);
    }
    for (long p = 0; p < P; ++p) Wbar[p] += Wob[p];
  }
  for (long p = 0; p < P; ++p) Wbar[p] += winit_bar[p];   // w_in also sets the targets
  std::memcpy(d_w_in, Wbar.data(), sizeof(double) * P);
  std::memcpy(d_m_in, Mbar.data(), sizeof(double) * P);
}

bool make_problem(Problem& pb, int B, int H, int T, int d, int dh, int C, int fw, int flags,
                  double eps) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || dh < 1 || C < 1 || (fw != 0 && fw != 1)) return false;
  pb.B = B; pb.H = H; pb.T = T; pb.C = C;
  pb.net.d = d; pb.net.dh = dh; pb.net.fw = fw;
  pb.net.resln = (flags & 1) == 0;
  pb.net.eps = eps;
  pb.post_norm = (flags & 8) != 0;
  return true;
}

// The problem of unit u: the affine of its head h = u mod H (ln_a, ln_b are
// [H][d]; either may be NULL: a = 1, b = 0).
Problem unit_problem(const Problem& pb, long u, const double* ln_a, const double* ln_b) {
  Problem q = pb;
  const long h = u % pb.H;
  q.net.lna = ln_a ? ln_a + h * pb.net.d : nullptr;
  q.net.lnb = ln_b ? ln_b + h * pb.net.d : nullptr;
  return q;
}

}  // namespace

extern "C" {

// Number of fast-weight parameters per unit, or -1 for a bad kind.
long e2ttt_oracle_param_count(int d, int dh, int fw) {
  if (fw == 0) return 2L * d * dh;
  if (fw == 1) return 3L * d * dh;
  return -1;
}

// Forward over all B*H units.  Returns 0, or -1 on a bad argument.
// ln_a, ln_b: the LayerNorm affine per head, [H][d], each NULL for a = 1 / b = 0.
int e2ttt_oracle_forward(int B, int H, int T, int d, int dh, int C, int fw, int flags, double eps,
                         const double* q, const double* k, const double* v, const double* eta,
                         const double* beta, const double* gamma, const double* w_in,
                         const double* m_in, const double* ln_a, const double* ln_b, double* out,
                         double* w_out, double* m_out, int nthreads) {
  Problem pb;
  if (!make_problem(pb, B, H, T, d, dh, C, fw, flags, eps)) return -1;
  if (!q || !k || !v || !eta || !beta || !w_in || !out || !w_out || !m_out) return -1;
  if ((ln_a || ln_b) && !pb.net.resln) return -1;   // the affine belongs to the LayerNorm
  const long P = pb.net.P();
  const long U = pb.units();
  if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
  for (long u = 0; u < U; ++u) {
    const long tok = u * T;
    unit_forward(unit_problem(pb, u, ln_a, ln_b), q + tok * d, k + tok * d, v + tok * d,
                 eta + tok, beta + tok,
                 gamma ? gamma + tok : nullptr, w_in + u * P, m_in ? m_in + u * P : nullptr,
                 out + tok * d, w_out + u * P, m_out + u * P, nullptr);
  }
  return 0;
}

// Backward over all B*H units (see unit_backward for the loss).  d_w_out,
// d_m_out and m_in may be NULL (zero); d_gamma must be NULL iff gamma is NULL;
// d_ln_a, d_ln_b ([H][d], summed over the batch) must be given iff ln_a and
// ln_b are (both or neither).
int e2ttt_oracle_backward(int B, int H, int T, int d, int dh, int C, int fw, int flags, double eps,
                          const double* q, const double* k, const double* v, const double* eta,
                          const double* beta, const double* gamma, const double* w_in,
                          const double* m_in, const double* ln_a, const double* ln_b,
                          const double* d_out, const double* d_w_out, const double* d_m_out,
                          double* dq, double* dk, double* dv, double* d_eta, double* d_beta,
                          double* d_gamma, double* d_w_in, double* d_m_in, double* d_ln_a,
                          double* d_ln_b, int nthreads) {
  Problem pb;
  if (!make_problem(pb, B, H, T, d, dh, C, fw, flags, eps)) return -1;
  if (!q || !k || !v || !eta || !beta || !w_in || !d_out || !dq || !dk || !dv || !d_eta ||
      !d_beta || !d_w_in || !d_m_in)
    return -1;
  if ((gamma == nullptr) != (d_gamma == nullptr)) return -1;
  const bool aff = ln_a || ln_b;
  if (aff && (!ln_a || !ln_b || !d_ln_a || !d_ln_b || !pb.net.resln)) return -1;
  const long P = pb.net.P();
  const long U = pb.units();
  // the affine gradients of every unit, summed over the batch afterwards in order
  std::vector<double> ga(aff ? U * d : 0, 0.0), gb(aff ? U * d : 0, 0.0);
  if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
  for (long u = 0; u < U; ++u) {
    const long tok = u * T;
    unit_backward(unit_problem(pb, u, ln_a, ln_b), q + tok * d, k + tok * d, v + tok * d,
                  eta + tok, beta + tok,
                  gamma ? gamma + tok : nullptr, w_in + u * P, m_in ? m_in + u * P : nullptr,
                  d_out + tok * d, d_w_out ? d_w_out + u * P : nullptr,
                  d_m_out ? d_m_out + u * P : nullptr, dq + tok * d, dk + tok * d, dv + tok * d,
                  d_eta + tok, d_beta + tok, d_gamma ? d_gamma + tok : nullptr, d_w_in + u * P,
                  d_m_in + u * P, aff ? ga.data() + u * d : nullptr,
                  aff ? gb.data() + u * d : nullptr);
  }
  if (aff) {
    for (long i = 0; i < (long)H * d; ++i) { d_ln_a[i] = 0.0; d_ln_b[i] = 0.0; }
    for (long u = 0; u < U; ++u)
      for (int i = 0; i < d; ++i) {
        d_ln_a[(u % H) * d + i] += ga[u * d + i];
        d_ln_b[(u % H) * d + i] += gb[u * d + i];
      }
  }
  return 0;
}

// Scalar kernels of one chunk of length C (Prop. 1), from the unrolled sums of
// eq. (8) with the suffix-product convention of eq. (9):
//   kw[t] = eta_t * sum_{j=t}^{C} prod_{i=t+1}^{j} beta_i prod_{q=j+1}^{C} gamma_q
//   km[t] = eta_t * prod_{i=t+1}^{C} beta_i
//   cw = prod_{i=1}^{C} gamma_i
//   cm = sum_{j=1}^{C} prod_{i=1}^{j} beta_i prod_{q=j+1}^{C} gamma_q
//   cb = prod_{i=1}^{C} beta_i
// gamma may be NULL (gamma = 1).  carry = {cw, cm, cb}.
int e2ttt_oracle_chunk_coeffs(int C, const double* eta, const double* beta, const double* gamma,
                              double* kw, double* km, double* carry) {
  if (C < 1 || !eta || !beta || !kw || !km || !carry) return -1;
  auto g = [&](int i) { return gamma ? gamma[i - 1] : 1.0; };  // 1-based token index
  auto b = [&](int i) { return beta[i - 1]; };
  auto prod_b = [&](int lo, int hi) { double p = 1.0; for (int i = lo; i <= hi; ++i) p *= b(i); return p; };
  auto prod_g = [&](int lo, int hi) { double p = 1.0; for (int i = lo; i <= hi; ++i) p *= g(i); return p; };
  for (int t = 1; t <= C; ++t) {
    double s = 0.0;
    for (int j = t; j <= C; ++j) s += prod_b(t + 1, j) * prod_g(j + 1, C);
    kw[t - 1] = eta[t - 1] * s;
    km[t - 1] = eta[t - 1] * prod_b(t + 1, C);
  }
  double cm = 0.0;
  for (int j = 1; j <= C; ++j) cm += prod_b(1, j) * prod_g(j + 1, C);
  carry[0] = prod_g(1, C);
  carry[1] = cm;
  carry[2] = prod_b(1, C);
  return 0;
}

// f_W(x) for one unit and a batch of n rows x[n][d] (used by the tests to pin
// special cases such as "eta = 0 leaves every output at f_{W_in}(q_t)").
// ln_a, ln_b: the LayerNorm affine a[d], b[d] (NULL: a = 1, b = 0).
int e2ttt_oracle_net(int d, int dh, int fw, int flags, double eps, const double* W,
                     const double* ln_a, const double* ln_b, int n, const double* x, double* f) {
  Net net;
  net.d = d; net.dh = dh; net.fw = fw; net.resln = (flags & 1) == 0; net.eps = eps;
  net.lna = ln_a; net.lnb = ln_b;
  if (d < 1 || dh < 1 || (fw != 0 && fw != 1) || n < 0 || !W || !x || !f) return -1;
  for (int r = 0; r < n; ++r)
    net_eval<double>(net, W, x + (long)r * d, f + (long)r * d, nullptr, nullptr, nullptr);
  return 0;
}

// Negative inner-loss gradients G = -grad_W L at W for rows (k, v), one per row
// (G is [n][P]); used by the tests to pin the closed form of Prop. 1.
int e2ttt_oracle_neg_grad(int d, int dh, int fw, int flags, double eps, const double* W,
                          const double* ln_a, const double* ln_b, int n, const double* k,
                          const double* v, double* G) {
  Net net;
  net.d = d; net.dh = dh; net.fw = fw; net.resln = (flags & 1) == 0; net.eps = eps;
  net.lna = ln_a; net.lnb = ln_b;
  if (d < 1 || dh < 1 || (fw != 0 && fw != 1) || n < 0 || !W || !k || !v || !G) return -1;
  const long P = net.P();
  std::vector<double> gk(d), gv(d);
  for (int r = 0; r < n; ++r) {
    double* Gr = G + (long)r * P;
    loss_grad<double>(net, W, k + (long)r * d, v + (long)r * d, Gr, gk.data(), gv.data());
    for (long p = 0; p < P; ++p) Gr[p] = -Gr[p];
  }
  return 0;
}

}  // extern "C"
