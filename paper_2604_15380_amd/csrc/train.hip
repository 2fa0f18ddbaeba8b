// One FP64 training step of PaiNN on energies and forces (section "Flagship
// Training of Top HPO Models"; Table "Lead PaiNN model configuration": MAE
// loss, force weight ~94.8, AdamW, FP64).
//
// Loss over a batch of B structures and N atoms (F = -dE/dx):
//   L = (1/B) sum_b |E_b - E*_b| + lambda (1/(3N)) sum_ic |F_ic - F*_ic|
// Gradient (the residual signs held fixed):
//   dL/dtheta = sum_b c_b dE_b/dtheta - d/dtheta (u . dE/dx),
//   c_b = sign(E_b - E*_b) / B,  u = lambda sign(F - F*) / (3N).
//
// Two passes over the same kernels, templated on the scalar type S:
//  A (S = double): forward, then the reverse pass to the positions: E, F;
//    then the loss, c and u.
//  B (S = Dual, a value and a first-order tangent): the forward with the
//    positions moving along -u, then the reverse pass to the weights seeded
//    with dE_b = 1 + eps c_b.  The reverse pass is linear in its seed, so the
//    tangent of the weight gradient it returns is
//      sum_b c_b dE_b/dtheta + d/deps [dE/dtheta](x - eps u) = dL/dtheta.
//    (forward-mode differentiation of the reverse pass: a Hessian-vector
//    product in mixed position/weight coordinates, with no second reverse.)
// Then AdamW (Loshchilov & Hutter, ICLR 2019) on the FP64 weights.
//
// Weights live in one flat FP64 array in the weight file's order at the
// model's own width F.  Every weight gradient is a reduction over atoms or
// edges computed by one launch in a fixed order (no atomics), so a step is
// deterministic.  The kernels are plain FP64 vector-ALU code with LDS tiles:
// a training batch of the lead model (25 structures) is small.
#include <math.h>
#include <string.h>

#include <new>

#include "internal.h"

namespace {

struct Dual {
  double v, d;
};
__device__ inline Dual operator+(Dual a, Dual b) { return {a.v + b.v, a.d + b.d}; }
__device__ inline Dual operator-(Dual a, Dual b) { return {a.v - b.v, a.d - b.d}; }
__device__ inline Dual operator-(Dual a) { return {-a.v, -a.d}; }
__device__ inline Dual operator*(Dual a, Dual b) { return {a.v * b.v, a.v * b.d + a.d * b.v}; }
__device__ inline Dual operator*(Dual a, double b) { return {a.v * b, a.d * b}; }
__device__ inline Dual operator*(double a, Dual b) { return {a * b.v, a * b.d}; }
__device__ inline Dual operator+(Dual a, double b) { return {a.v + b, a.d}; }
__device__ inline Dual operator+(double a, Dual b) { return {a + b.v, b.d}; }
__device__ inline Dual operator-(double a, Dual b) { return {a - b.v, -b.d}; }
__device__ inline Dual operator-(Dual a, double b) { return {a.v - b, a.d}; }
__device__ inline Dual operator/(Dual a, Dual b) {
  const double q = a.v / b.v;
  return {q, (a.d - q * b.d) / b.v};
}
__device__ inline Dual operator/(double a, Dual b) {
  const double q = a / b.v;
  return {q, -q * b.d / b.v};
}
__device__ inline Dual operator/(Dual a, double b) { return {a.v / b, a.d / b}; }
__device__ inline Dual& operator+=(Dual& a, Dual b) { a = a + b; return a; }
__device__ inline Dual& operator-=(Dual& a, Dual b) { a = a - b; return a; }
__device__ inline Dual dexp(Dual a) {
  const double e = exp(a.v);
  return {e, e * a.d};
}
__device__ inline Dual dsin(Dual a) { return {sin(a.v), cos(a.v) * a.d}; }
__device__ inline Dual dcos(Dual a) { return {cos(a.v), -sin(a.v) * a.d}; }
__device__ inline Dual dsqrt(Dual a) {
  const double r = sqrt(a.v);
  return {r, a.d / (2.0 * r)};
}
__device__ inline double dexp(double a) { return exp(a); }
__device__ inline double dsin(double a) { return sin(a); }
__device__ inline double dcos(double a) { return cos(a); }
__device__ inline double dsqrt(double a) { return sqrt(a); }

// value part, gradient part (the tangent of a Dual; the value of a double)
__device__ inline double val(double x) { return x; }
__device__ inline double val(Dual x) { return x.v; }
__device__ inline double part(double x) { return x; }
__device__ inline double part(Dual x) { return x.d; }
template <class S> __device__ inline S cst(double x);
template <> __device__ inline double cst<double>(double x) { return x; }
template <> __device__ inline Dual cst<Dual>(double x) { return {x, 0.0}; }
template <class S> __device__ inline S mk(double v, double d);
template <> __device__ inline double mk<double>(double v, double) { return v; }
template <> __device__ inline Dual mk<Dual>(double v, double d) { return {v, d}; }

template <class S> __device__ inline S silu(S x) { return x / (1.0 + dexp(-x)); }
template <class S> __device__ inline S dsilu(S x) {
  const S sg = 1.0 / (1.0 + dexp(-x));
  return sg * (1.0 + x * (1.0 - sg));
}

constexpr int TB = 256;
inline unsigned blocks(size_t n, int t = TB) { return (unsigned)((n + t - 1) / t); }
// most row chunks of one weight-gradient reduction (k_tr_wgrad)
constexpr int WG_CHUNKS = 32;

// ---- dense layers ------------------------------------------------------------
// Y[r][o] = sum_k X[r][k] W(o, k) (+ b[o] on the value part) (+ ADD[r][o]),
// W(o, k) = W[o * wo + k * wk] (wo = din, wk = 1 for a layer stored
// [out, in]; wo = 1, wk = dout_of_the_layer for its transpose); with SILU,
// Z keeps the pre-activation and Y = silu(Z).  Rows [lo, hi) with lo, hi from
// `range` (device) when given, else [0, rows).  32 x 32 output tiles, 2 x 2 per
// thread, k in steps of 32 through LDS.
template <class S, bool SILU>
__global__ void __launch_bounds__(256) k_tr_dense(int rows, const int32_t* __restrict__ range, int din, int dout,
                                                  const S* __restrict__ X, int ldx, const double* __restrict__ W,
                                                  long long wo, long long wk, const double* __restrict__ b,
                                                  const S* __restrict__ add, int ldadd, S* __restrict__ Z,
                                                  S* __restrict__ Y, int ldy) {
  __shared__ S Xs[32][33];
  __shared__ double Ws[32][33];
  const int lo = range ? range[0] : 0, hi = range ? range[1] : rows;
  const int r0 = lo + blockIdx.x * 32, o0 = blockIdx.y * 32;
  if (r0 >= hi) return;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  S acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = cst<S>(0.0);
  for (int k0 = 0; k0 < din; k0 += 32) {
    for (int q = threadIdx.x; q < 1024; q += 256) {
      const int rr = q >> 5, kk = q & 31, r = r0 + rr, k = k0 + kk;
      Xs[rr][kk] = (r < hi && k < din) ? X[(size_t)r * ldx + k] : cst<S>(0.0);
      const int o = o0 + rr;
      Ws[rr][kk] = (o < dout && k < din) ? W[(long long)o * wo + (long long)k * wk] : 0.0;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const S x0 = Xs[2 * ty][kk], x1 = Xs[2 * ty + 1][kk];
      const double w0 = Ws[2 * tx][kk], w1 = Ws[2 * tx + 1][kk];
      acc[0][0] += x0 * w0;
      acc[0][1] += x0 * w1;
      acc[1][0] += x1 * w0;
      acc[1][1] += x1 * w1;
    }
    __syncthreads();
  }
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) {
      const int r = r0 + 2 * ty + i, o = o0 + 2 * tx + j;
      if (r >= hi || o >= dout) continue;
      S y = acc[i][j];
      if (b) y = y + b[o];
      if (add) y = y + add[(size_t)r * ldadd + o];
      if (SILU) {
        Z[(size_t)r * ldy + o] = y;
        y = silu(y);
      }
      Y[(size_t)r * ldy + o] = y;
    }
}

// Weight gradient over rows [lo, hi): G[o][k] = part( sum_r sc[r] A[r][o] B[r][k] )
// for k < din, and with a bias the column k = din, where B is taken as 1:
// Gb[o] = part( sum_r sc[r] A[r][o] ) (sc may be null: 1).  The rows are cut
// into gridDim.z chunks of `rch`; chunk z writes its partial sums to
// Pz[z][o][kb] (kb < din + 1), and k_tr_wgrad_sum adds the chunks in order,
// so the result does not depend on scheduling.
template <class S>
__global__ void __launch_bounds__(256) k_tr_wgrad(int rows, const int32_t* __restrict__ range, int dout, int din,
                                                  int dinb, int rch, const S* __restrict__ A, int lda,
                                                  const S* __restrict__ Bm, int ldb, const S* __restrict__ sc,
                                                  double* __restrict__ Pz) {
  __shared__ S As[32][33];
  __shared__ S Bs[32][33];
  const int lo0 = range ? range[0] : 0, hi0 = range ? range[1] : rows;
  const int lo = lo0 + blockIdx.z * rch, hi = min(hi0, lo + rch);
  const int k0 = blockIdx.x * 32, o0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  S acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = cst<S>(0.0);
  for (int rb = lo; rb < hi; rb += 32) {
    for (int q = threadIdx.x; q < 1024; q += 256) {
      const int rr = q >> 5, cc = q & 31, r = rb + rr;
      const int o = o0 + cc, k = k0 + cc;
      S a = (r < hi && o < dout) ? A[(size_t)r * lda + o] : cst<S>(0.0);
      if (sc && r < hi) a = a * sc[r];
      As[rr][cc] = a;
      Bs[rr][cc] = (r < hi && k < din) ? Bm[(size_t)r * ldb + k] : (r < hi && k == din) ? cst<S>(1.0) : cst<S>(0.0);
    }
    __syncthreads();
#pragma unroll 8
    for (int rr = 0; rr < 32; ++rr) {
      const S a0 = As[rr][2 * ty], a1 = As[rr][2 * ty + 1];
      const S b0 = Bs[rr][2 * tx], b1 = Bs[rr][2 * tx + 1];
      acc[0][0] += a0 * b0;
      acc[0][1] += a0 * b1;
      acc[1][0] += a1 * b0;
      acc[1][1] += a1 * b1;
    }
    __syncthreads();
  }
  double* P = Pz + (size_t)blockIdx.z * dout * dinb;
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) {
      const int o = o0 + 2 * ty + i, k = k0 + 2 * tx + j;
      if (o < dout && k < dinb) P[(size_t)o * dinb + k] = part(acc[i][j]);
    }
}

// G[o][k] = sum over the chunks z (in order) of Pz[z][o][k], k < din; the
// bias column k = din (when dinb > din) into Gb[o].
__global__ void k_tr_wgrad_sum(int nz, int dout, int din, int dinb, const double* __restrict__ Pz,
                               double* __restrict__ G, double* __restrict__ Gb) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)dout * dinb) return;
  const int o = (int)(idx / dinb), k = (int)(idx % dinb);
  double acc = 0.0;
  for (int z = 0; z < nz; ++z) acc += Pz[(size_t)z * dout * dinb + idx];
  if (k < din) G[(size_t)o * din + k] = acc;
  else Gb[o] = acc;
}

// Y[r][o] *= silu'(Z[r][o]) for rows [lo, hi), width n (row strides ld).
template <class S>
__global__ void k_tr_mul_dsilu(int rows, const int32_t* __restrict__ range, int n, S* __restrict__ Y, int ldy,
                               const S* __restrict__ Z, int ldz) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  const int lo = range ? range[0] : 0, hi = range ? range[1] : rows;
  const size_t r = lo + idx / n;
  if ((long long)r >= hi) return;
  const int o = (int)(idx % n);
  Y[r * ldy + o] = Y[r * ldy + o] * dsilu(Z[r * ldz + o]);
}

template <class S>
__global__ void k_tr_zero(size_t n, S* __restrict__ p) {
  const size_t i = (size_t)blockIdx.x * TB + threadIdx.x;
  if (i < n) p[i] = cst<S>(0.0);
}

template <class S>
__global__ void k_tr_copy(size_t n, const S* __restrict__ src, S* __restrict__ dst) {
  const size_t i = (size_t)blockIdx.x * TB + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

__global__ void k_tr_zero_d(size_t n, double* __restrict__ p) {
  const size_t i = (size_t)blockIdx.x * TB + threadIdx.x;
  if (i < n) p[i] = 0.0;
}

// ---- geometry, embedding -------------------------------------------------------
// Per edge: r = x_j - x_i + t (with tangent dpos_j - dpos_i), d, rhat, the
// radial basis g_k(d) and the cosine cutoff f_c(d) (the edge set has d < r_c).
// With DERIV (the real pass) also d, g_k'(d) and f_c'(d).
template <class S, bool DERIV>
__global__ void k_tr_geom(long long E, int K, double rc, int rbf, const int32_t* __restrict__ recv,
                          const int32_t* __restrict__ col, const int32_t* __restrict__ shift,
                          const int32_t* __restrict__ atom_struct, const double* __restrict__ pos,
                          const double* __restrict__ cell, const double* __restrict__ dpos, S* __restrict__ rhat,
                          S* __restrict__ basis, S* __restrict__ fc, double* __restrict__ dist,
                          double* __restrict__ dbasis, double* __restrict__ dfc) {
  const long long e = (long long)blockIdx.x * TB + threadIdx.x;
  if (e >= E) return;
  const int i = recv[e], j = col[e], sh = shift[e];
  const double* Cl = cell + 9 * atom_struct[i];
  const double n[3] = {(double)(int8_t)(sh & 0xff), (double)(int8_t)((sh >> 8) & 0xff),
                       (double)(int8_t)((sh >> 16) & 0xff)};
  S r[3];
  for (int c = 0; c < 3; ++c) {
    const double t = (n[0] * Cl[c] + n[1] * Cl[3 + c]) + n[2] * Cl[6 + c];
    const double x = (pos[3 * j + c] - pos[3 * i + c]) + t;
    r[c] = mk<S>(x, dpos ? dpos[3 * j + c] - dpos[3 * i + c] : 0.0);
  }
  const S d = dsqrt((r[0] * r[0] + r[1] * r[1]) + r[2] * r[2]);
  for (int c = 0; c < 3; ++c) rhat[3 * e + c] = r[c] / d;
  const double pi = 3.14159265358979323846;
  fc[e] = 0.5 * (dcos(d * (pi / rc)) + 1.0);
  if (DERIV) {
    dist[e] = val(d);
    dfc[e] = -0.5 * (pi / rc) * sin(val(d) * (pi / rc));
  }
  if (rbf == 0) {
    const double delta = rc / (K - 1), gamma = 1.0 / (2.0 * delta * delta);
    for (int k = 0; k < K; ++k) {
      const S x = d - k * delta;
      const S g = dexp(-gamma * (x * x));
      basis[(size_t)e * K + k] = g;
      if (DERIV) dbasis[(size_t)e * K + k] = -2.0 * gamma * val(x) * val(g);
    }
  } else {
    for (int k = 0; k < K; ++k) {
      const double w = (k + 1) * (pi / rc);
      basis[(size_t)e * K + k] = dsin(d * w) / d;
      if (DERIV) {
        const double dv = val(d);
        dbasis[(size_t)e * K + k] = w * cos(w * dv) / dv - sin(w * dv) / (dv * dv);
      }
    }
  }
}

template <class S>
__global__ void k_tr_embed(int N, int F, const int32_t* __restrict__ species, const double* __restrict__ emb,
                           S* __restrict__ s, S* __restrict__ v) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t i = idx / F;
  const int f = (int)(idx % F);
  s[idx] = cst<S>(emb[(size_t)species[i] * F + f]);
  for (int c = 0; c < 3; ++c) v[(i * 3 + c) * F + f] = cst<S>(0.0);
}

// ---- message -----------------------------------------------------------------
// Per (receiver i, channel f), over the receiver's CSR row:
//   s_mid = s + sum_e h^s_j w^s_e,  v_mid[c] = v[c] + sum_e (v_j[c] h^v_j w^v_e + rhat_e[c] h^r_j w^r_e)
// with w_e = f_c(d_e) lin_e, lin_e = W_f g(d_e) + b_f.
template <class S>
__global__ void k_tr_message(int N, int F, const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col,
                             const S* __restrict__ h, const S* __restrict__ s, const S* __restrict__ v,
                             const S* __restrict__ lin, const S* __restrict__ fc, const S* __restrict__ rhat,
                             S* __restrict__ s_mid, S* __restrict__ v_mid) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const int i = (int)(idx / F), f = (int)(idx % F);
  const size_t F3 = 3 * (size_t)F;
  S ds = cst<S>(0.0), dv[3] = {cst<S>(0.0), cst<S>(0.0), cst<S>(0.0)};
  for (int e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
    const size_t j = col[e];
    const S w = fc[e];
    const S ws = w * lin[e * F3 + f], wv = w * lin[e * F3 + F + f], wr = w * lin[e * F3 + 2 * F + f];
    ds += h[j * F3 + f] * ws;
    const S hv = h[j * F3 + F + f] * wv, hr = h[j * F3 + 2 * F + f] * wr;
    for (int c = 0; c < 3; ++c) dv[c] += v[(j * 3 + c) * F + f] * hv + rhat[3 * (size_t)e + c] * hr;
  }
  s_mid[idx] = s[idx] + ds;
  for (int c = 0; c < 3; ++c) v_mid[((size_t)i * 3 + c) * F + f] = v[((size_t)i * 3 + c) * F + f] + dv[c];
}

// Reverse of the message per (sender j, channel f), over the edges whose
// sender is j (t_edge order): dE/dh_j, dE/dv_j (the residual plus the
// message's share) and per edge dE/dw_e; g_s, g_v are dE/ds_mid, dE/dv_mid.
template <class S>
__global__ void k_tr_message_bwd(int N, int F, const int32_t* __restrict__ t_ptr, const int32_t* __restrict__ t_edge,
                                 const int32_t* __restrict__ recv, const S* __restrict__ h, const S* __restrict__ v,
                                 const S* __restrict__ lin, const S* __restrict__ fc, const S* __restrict__ rhat,
                                 const S* __restrict__ g_s, const S* __restrict__ g_v, S* __restrict__ g_h,
                                 S* __restrict__ g_v_out, S* __restrict__ g_w) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t j = idx / F;
  const int f = (int)(idx % F);
  const size_t F3 = 3 * (size_t)F;
  const S hs = h[j * F3 + f], hv = h[j * F3 + F + f], hr = h[j * F3 + 2 * F + f];
  S vj[3], gvj[3];
  for (int c = 0; c < 3; ++c) {
    vj[c] = v[(j * 3 + c) * F + f];
    gvj[c] = g_v[(j * 3 + c) * F + f];
  }
  S ghs = cst<S>(0.0), ghv = cst<S>(0.0), ghr = cst<S>(0.0);
  for (int q = t_ptr[j]; q < t_ptr[j + 1]; ++q) {
    const size_t e = t_edge[q], i = recv[e];
    const S w = fc[e];
    const S ws = w * lin[e * F3 + f], wv = w * lin[e * F3 + F + f], wr = w * lin[e * F3 + 2 * F + f];
    const S gsi = g_s[i * F + f];
    S Av = cst<S>(0.0), Ar = cst<S>(0.0);
    for (int c = 0; c < 3; ++c) {
      const S gvi = g_v[(i * 3 + c) * F + f];
      Av += gvi * vj[c];
      Ar += gvi * rhat[3 * e + c];
      gvj[c] += gvi * (hv * wv);
    }
    ghs += gsi * ws;
    ghv += Av * wv;
    ghr += Ar * wr;
    g_w[e * F3 + f] = gsi * hs;
    g_w[e * F3 + F + f] = Av * hv;
    g_w[e * F3 + 2 * F + f] = Ar * hr;
  }
  g_h[j * F3 + f] = ghs;
  g_h[j * F3 + F + f] = ghv;
  g_h[j * F3 + 2 * F + f] = ghr;
  for (int c = 0; c < 3; ++c) g_v_out[(j * 3 + c) * F + f] = gvj[c];
}

// Real pass: per edge (one wave), the layer's share of dE/dd and dE/drhat:
//   dE/dd    += sum_c3 g_w[c3] (f_c'(d) lin[c3] + f_c(d) lin'[c3]),  lin' = W_f g'(d)
//   dE/drhat += sum_f g_v_i[c][f] h^r_j[f] w^r[f]
__global__ void __launch_bounds__(256) k_tr_edge_bwd(long long E, int F, const int32_t* __restrict__ recv,
                                                     const int32_t* __restrict__ col, const double* __restrict__ h,
                                                     const double* __restrict__ lin, const double* __restrict__ linp,
                                                     const double* __restrict__ fc, const double* __restrict__ dfc,
                                                     const double* __restrict__ g_v, const double* __restrict__ g_w,
                                                     double* __restrict__ gd, double* __restrict__ grh) {
  const long long e = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (e >= E) return;
  const size_t F3 = 3 * (size_t)F, i = recv[e], j = col[e];
  const double w = fc[e], dw = dfc[e];
  double a = 0.0, r0 = 0.0, r1 = 0.0, r2 = 0.0;
  for (int c3 = lane; c3 < 3 * F; c3 += 64)
    a += g_w[e * F3 + c3] * (dw * lin[e * F3 + c3] + w * linp[e * F3 + c3]);
  for (int f = lane; f < F; f += 64) {
    const double t = h[j * F3 + 2 * F + f] * (w * lin[e * F3 + 2 * F + f]);
    r0 += g_v[(i * 3 + 0) * F + f] * t;
    r1 += g_v[(i * 3 + 1) * F + f] * t;
    r2 += g_v[(i * 3 + 2) * F + f] * t;
  }
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_down(a, off);
    r0 += __shfl_down(r0, off);
    r1 += __shfl_down(r1, off);
    r2 += __shfl_down(r2, off);
  }
  if (lane == 0) {
    gd[e] += a;
    grh[3 * e] += r0;
    grh[3 * e + 1] += r1;
    grh[3 * e + 2] += r2;
  }
}

// dE/dr per edge, then per atom dE/dx = sum over edges it sends - sum over
// edges it receives; forces = -dE/dx.
__global__ void k_tr_edge_dr(long long E, const double* __restrict__ dist, const double* __restrict__ rhat,
                             const double* __restrict__ gd, const double* __restrict__ grh, double* __restrict__ gr) {
  const long long e = (long long)blockIdx.x * TB + threadIdx.x;
  if (e >= E) return;
  const double* u = rhat + 3 * e;
  const double* q = grh + 3 * e;
  const double dot = (q[0] * u[0] + q[1] * u[1]) + q[2] * u[2];
  for (int c = 0; c < 3; ++c) gr[3 * e + c] = gd[e] * u[c] + (q[c] - dot * u[c]) / dist[e];
}

__global__ void k_tr_forces(int N, const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ t_ptr,
                            const int32_t* __restrict__ t_edge, const double* __restrict__ gr,
                            double* __restrict__ forces) {
  const int a = blockIdx.x * TB + threadIdx.x;
  if (a >= N) return;
  double x[3] = {0.0, 0.0, 0.0};
  for (int q = t_ptr[a]; q < t_ptr[a + 1]; ++q)
    for (int c = 0; c < 3; ++c) x[c] += gr[3 * (size_t)t_edge[q] + c];
  for (int e = row_ptr[a]; e < row_ptr[a + 1]; ++e)
    for (int c = 0; c < 3; ++c) x[c] -= gr[3 * (size_t)e + c];
  for (int c = 0; c < 3; ++c) forces[3 * (size_t)a + c] = -x[c];
}

// ---- update block ---------------------------------------------------------------
// xin = [s_mid ; |V|] with |V| = sqrt(sum_c V[c]^2) (0 where V = 0)
template <class S>
__global__ void k_tr_upd_norm(int N, int F, const S* __restrict__ s_mid, const S* __restrict__ V, S* __restrict__ xin) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t i = idx / F;
  const int f = (int)(idx % F);
  S n2 = cst<S>(0.0);
  for (int c = 0; c < 3; ++c) {
    const S x = V[(i * 3 + c) * F + f];
    n2 += x * x;
  }
  xin[i * 2 * F + f] = s_mid[idx];
  xin[i * 2 * F + F + f] = val(n2) > 0.0 ? dsqrt(n2) : cst<S>(0.0);
}

// v' = v_mid + a_vv U,  s' = s_mid + a_sv <U, V> + a_ss
template <class S>
__global__ void k_tr_upd_post(int N, int F, const S* __restrict__ s_mid, const S* __restrict__ v_mid,
                              const S* __restrict__ U, const S* __restrict__ V, const S* __restrict__ a,
                              S* __restrict__ s_out, S* __restrict__ v_out) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t i = idx / F;
  const int f = (int)(idx % F);
  const S avv = a[i * 3 * F + f], asv = a[i * 3 * F + F + f], ass = a[i * 3 * F + 2 * F + f];
  S uv = cst<S>(0.0);
  for (int c = 0; c < 3; ++c) {
    const size_t q = (i * 3 + c) * F + f;
    uv += U[q] * V[q];
    v_out[q] = v_mid[q] + avv * U[q];
  }
  s_out[idx] = s_mid[idx] + asv * uv + ass;
}

// Reverse of the residual updates: g_a = [sum_c g_v U, g_s <U,V>, g_s];
// g_U[c] = g_v[c] a_vv + g_s a_sv V[c];  g_V[c] = g_s a_sv U[c]
template <class S>
__global__ void k_tr_upd_bwd1(int N, int F, const S* __restrict__ gs, const S* __restrict__ gv,
                              const S* __restrict__ U, const S* __restrict__ V, const S* __restrict__ a,
                              S* __restrict__ g_a, S* __restrict__ gU, S* __restrict__ gV) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t i = idx / F;
  const int f = (int)(idx % F);
  const S avv = a[i * 3 * F + f], asv = a[i * 3 * F + F + f];
  const S g = gs[idx];
  S gavv = cst<S>(0.0), uv = cst<S>(0.0);
  for (int c = 0; c < 3; ++c) {
    const size_t q = (i * 3 + c) * F + f;
    gavv += gv[q] * U[q];
    uv += U[q] * V[q];
    gU[q] = gv[q] * avv + (g * asv) * V[q];
    gV[q] = (g * asv) * U[q];
  }
  g_a[i * 3 * F + f] = gavv;
  g_a[i * 3 * F + F + f] = g * uv;
  g_a[i * 3 * F + 2 * F + f] = g;
}

// g_V[c] += (g_n / |V|) V[c] (0 where |V| = 0);  g_s_mid = g_s + g_in[:, :F]
template <class S>
__global__ void k_tr_upd_bwd2(int N, int F, const S* __restrict__ g_in, const S* __restrict__ xin,
                              const S* __restrict__ V, const S* __restrict__ gs, S* __restrict__ gV,
                              S* __restrict__ gs_mid) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)N * F) return;
  const size_t i = idx / F;
  const int f = (int)(idx % F);
  const S nrm = xin[i * 2 * F + F + f];
  if (val(nrm) > 0.0) {
    const S k = g_in[i * 2 * F + F + f] / nrm;
    for (int c = 0; c < 3; ++c) {
      const size_t q = (i * 3 + c) * F + f;
      gV[q] = gV[q] + k * V[q];
    }
  }
  gs_mid[idx] = gs[idx] + g_in[i * 2 * F + f];
}

// ---- heads -------------------------------------------------------------------
// Atoms grouped by the head of their structure (stable: atom order within a
// head): perm[p] = atom, hstart[h] = first slot of head h, hstart[H] = slots
// in use; atoms of a structure whose id is outside [0, H) get no slot and
// set *bad.
__global__ void k_tr_group(int B, int H, const int32_t* __restrict__ struct_ptr,
                           const int32_t* __restrict__ dataset_id, int32_t* __restrict__ perm,
                           int32_t* __restrict__ hstart, int32_t* __restrict__ bad) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int slot = 0, nbad = 0;
  for (int h = 0; h < H; ++h) {
    hstart[h] = slot;
    for (int b = 0; b < B; ++b) {
      const int d = dataset_id ? dataset_id[b] : 0;
      if (d != h) continue;
      for (int a = struct_ptr[b]; a < struct_ptr[b + 1]; ++a) perm[slot++] = a;
    }
  }
  hstart[H] = slot;
  for (int b = 0; b < B; ++b) {
    const int d = dataset_id ? dataset_id[b] : 0;
    if (d < 0 || d >= H) ++nbad;
  }
  *bad = nbad;
}

template <class S>
__global__ void k_tr_gather(int n, int w, const int32_t* __restrict__ slots, const int32_t* __restrict__ perm,
                            const S* __restrict__ src, S* __restrict__ dst) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  const int used = *slots;
  if (idx >= (size_t)n * w) return;
  const size_t p = idx / w;
  const int o = (int)(idx % w);
  dst[idx] = (long long)p < used ? src[(size_t)perm[p] * w + o] : cst<S>(0.0);
}

template <class S>
__global__ void k_tr_scatter(int n, int w, const int32_t* __restrict__ slots, const int32_t* __restrict__ perm,
                             const S* __restrict__ src, S* __restrict__ dst) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)n * w) return;
  const size_t p = idx / w;
  if ((long long)p >= *slots) return;
  dst[(size_t)perm[p] * w + (int)(idx % w)] = src[idx];
}

// E_b = sum of e over the structure's atoms (atom order)
template <class S>
__global__ void k_tr_energy(int B, const int32_t* __restrict__ struct_ptr, const S* __restrict__ e,
                            double* __restrict__ E) {
  const int b = blockIdx.x * TB + threadIdx.x;
  if (b >= B) return;
  S acc = cst<S>(0.0);
  for (int a = struct_ptr[b]; a < struct_ptr[b + 1]; ++a) acc += e[a];
  E[b] = val(acc);
}

// reverse seed of the per-atom energies: dE_b/de_i = 1 (+ eps c_b in the
// tangent pass), in grouped order
template <class S>
__global__ void k_tr_seed(int N, const int32_t* __restrict__ slots, const int32_t* __restrict__ perm,
                          const int32_t* __restrict__ atom_struct, const double* __restrict__ c, S* __restrict__ g) {
  const int p = blockIdx.x * TB + threadIdx.x;
  if (p >= N) return;
  g[p] = p < *slots ? mk<S>(1.0, c ? c[atom_struct[perm[p]]] : 0.0) : cst<S>(0.0);
}

// embedding gradient: G[z][f] = part(sum of g_s over the atoms of species z)
template <class S>
__global__ void k_tr_emb_grad(int N, int F, int n_species, const int32_t* __restrict__ species,
                              const S* __restrict__ gs, double* __restrict__ G) {
  const size_t idx = (size_t)blockIdx.x * TB + threadIdx.x;
  if (idx >= (size_t)n_species * F) return;
  const int z = (int)(idx / F), f = (int)(idx % F);
  S acc = cst<S>(0.0);
  for (int i = 0; i < N; ++i)
    if (species[i] == z) acc += gs[(size_t)i * F + f];
  G[idx] = part(acc);
}

// ---- loss and optimizer ----------------------------------------------------------
// One workgroup: residuals, the two MAE terms (fixed-order tree sums), the
// energy seeds c_b = sign(r_b) / B and the position tangent -u,
// u = lambda sign(r_F) / (3N).  loss = [L, MAE_E, MAE_F].
__global__ void __launch_bounds__(256) k_tr_loss(int B, int N, double lambda, const double* __restrict__ E,
                                                 const double* __restrict__ E_ref, const double* __restrict__ Fo,
                                                 const double* __restrict__ F_ref, const int32_t* __restrict__ bad,
                                                 double* __restrict__ c, double* __restrict__ dpos,
                                                 double* __restrict__ loss) {
  __shared__ double se[256], sf[256];
  double ae = 0.0, af = 0.0;
  for (int b = threadIdx.x; b < B; b += 256) {
    const double r = E[b] - E_ref[b];
    ae += fabs(r);
    c[b] = (r > 0.0 ? 1.0 : r < 0.0 ? -1.0 : 0.0) / B;
  }
  const double uf = N > 0 ? lambda / (3.0 * N) : 0.0;
  for (int q = threadIdx.x; q < 3 * N; q += 256) {
    const double r = Fo[q] - F_ref[q];
    af += fabs(r);
    dpos[q] = -(r > 0.0 ? 1.0 : r < 0.0 ? -1.0 : 0.0) * uf;
  }
  se[threadIdx.x] = ae;
  sf[threadIdx.x] = af;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) {
      se[threadIdx.x] += se[threadIdx.x + s];
      sf[threadIdx.x] += sf[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double le = B > 0 ? se[0] / B : 0.0, lf = N > 0 ? sf[0] / (3.0 * N) : 0.0;
    const double nan = *bad ? NAN : 0.0;
    loss[0] = le + lambda * lf + nan;
    loss[1] = le + nan;
    loss[2] = lf + nan;
  }
}

__global__ void k_tr_adamw(size_t n, double* __restrict__ th, const double* __restrict__ g, double* __restrict__ m,
                           double* __restrict__ v, double lr, double b1, double b2, double eps, double wd,
                           double bc1, double bc2) {
  const size_t i = (size_t)blockIdx.x * TB + threadIdx.x;
  if (i >= n) return;
  const double gi = g[i];
  const double mi = b1 * m[i] + (1.0 - b1) * gi;
  const double vi = b2 * v[i] + (1.0 - b2) * gi * gi;
  m[i] = mi;
  v[i] = vi;
  th[i] = th[i] * (1.0 - lr * wd) - lr * (mi / bc1) / (sqrt(vi / bc2) + eps);
}

}  // namespace

// ---- host side ---------------------------------------------------------------------
namespace {

painn_status tfail(painn_ctx* ctx, painn_status st, const std::string& msg) {
  if (ctx) ctx->err = msg;
  return st;
}

// Offsets of the arrays of the flat weight vector (file order, width F).
struct TrLayout {
  struct Layer { size_t a[A_PER_LAYER]; };
  size_t emb = 0;
  std::vector<Layer> layers;
  std::vector<size_t> shared_w, shared_b;                 // [m]
  std::vector<std::vector<size_t>> branch_w, branch_b;    // [h][m]
  size_t total = 0;
};

}  // namespace

struct painn_trainer {
  painn_ctx* ctx = nullptr;
  Hyper hp;                 // hp.F = the model's own width
  painn_train_config cfg{};
  TrLayout lay;
  double* theta = nullptr;  // weights [P]
  double* grad = nullptr;   // gradient of the last step [P]
  double* m1 = nullptr;     // AdamW moments
  double* m2 = nullptr;
  long long t = 0;          // steps taken
  void* ws = nullptr;       // workspace
  size_t ws_bytes = 0;
};

namespace {

TrLayout make_layout(const Hyper& hp) {
  TrLayout L;
  const size_t F = hp.F, K = hp.K;
  size_t o = 0;
  L.emb = o;
  o += (size_t)hp.n_species * F;
  L.layers.resize(hp.L);
  for (int l = 0; l < hp.L; ++l) {
    const size_t per[A_PER_LAYER] = {F * F, F, 3 * F * F, 3 * F, 3 * F * K, 3 * F, F * F, F * F,
                                     2 * F * F, F, 3 * F * F, 3 * F};
    for (int a = 0; a < A_PER_LAYER; ++a) {
      L.layers[l].a[a] = o;
      o += per[a];
    }
  }
  size_t din = F;
  for (int d : hp.shared_dims) {
    L.shared_w.push_back(o);
    o += (size_t)d * din;
    L.shared_b.push_back(o);
    o += d;
    din = d;
  }
  L.branch_w.assign(hp.n_heads, {});
  L.branch_b.assign(hp.n_heads, {});
  for (int h = 0; h < hp.n_heads; ++h) {
    size_t di = din;
    for (int d : hp.branch_dims) {
      L.branch_w[h].push_back(o);
      o += (size_t)d * di;
      L.branch_b[h].push_back(o);
      o += d;
      di = d;
    }
  }
  L.total = o;
  return L;
}

// Workspace of one step: every buffer sized for the tangent pass (16-byte
// Dual); the real pass uses the first half of each.
struct TrWs {
  // per layer (L of each): inputs s, v; phi pre-activation and hidden; h;
  // filter lin; after the message s_mid, v_mid; U, V; [s_mid ; |V|]; the gate's
  // pre-activation, hidden and output a
  std::vector<void*> s, v, z1, a1, h, lin, smid, vmid, U, V, xin, za, aa, a;
  void *sL, *vL;                     // after the last layer
  void *rhat, *basis, *fc;           // per edge
  double *dist, *dbasis, *dfc, *linp, *gd, *grh, *gr;   // real pass
  // heads: per shared layer pre-activation and output (atom order); the
  // branch input and per branch layer pre-activation and output (grouped)
  std::vector<void*> shz, shy, brz, bry;
  void *yg, *eg, *e;
  int32_t *perm, *hstart, *bad;
  // reverse
  void *gs, *gv, *gs2, *gv2, *gh, *ga, *gaa, *gin, *gU, *gV, *ga1, *gw, *gx1, *gx2;
  // loss
  double *E, *Fo, *c, *dpos, *lossbuf;
  double* wsum;   // partial sums of the weight-gradient reductions
};

constexpr size_t DS = sizeof(double) * 2;   // bytes per element, sized for Dual

size_t carve(TrWs* w, char* base, const Hyper& hp, int N, long long E, int B) {
  size_t off = 0;
  auto take = [&](size_t elems, size_t eb = DS) -> void* {
    void* p = base ? base + off : nullptr;
    off += (elems * eb + 255) & ~(size_t)255;
    return p;
  };
  const size_t n = N, F = hp.F, e = (size_t)E, K = hp.K;
  int wmax = hp.F;
  for (int d : hp.shared_dims) wmax = d > wmax ? d : wmax;
  for (int d : hp.branch_dims) wmax = d > wmax ? d : wmax;
  auto per = [&](std::vector<void*>& v, size_t elems) {
    v.assign(hp.L, nullptr);
    for (int l = 0; l < hp.L; ++l) v[l] = take(elems);
  };
  per(w->s, n * F);
  per(w->v, 3 * n * F);
  per(w->z1, n * F);
  per(w->a1, n * F);
  per(w->h, 3 * n * F);
  per(w->lin, 3 * e * F);
  per(w->smid, n * F);
  per(w->vmid, 3 * n * F);
  per(w->U, 3 * n * F);
  per(w->V, 3 * n * F);
  per(w->xin, 2 * n * F);
  per(w->za, n * F);
  per(w->aa, n * F);
  per(w->a, 3 * n * F);
  w->sL = take(n * F);
  w->vL = take(3 * n * F);
  w->rhat = take(3 * e);
  w->basis = take(e * K);
  w->fc = take(e);
  w->dist = (double*)take(e, 8);
  w->dbasis = (double*)take(e * K, 8);
  w->dfc = (double*)take(e, 8);
  w->linp = (double*)take(3 * e * F, 8);
  w->gd = (double*)take(e, 8);
  w->grh = (double*)take(3 * e, 8);
  w->gr = (double*)take(3 * e, 8);
  w->shz.assign(hp.shared_dims.size(), nullptr);
  w->shy.assign(hp.shared_dims.size(), nullptr);
  for (size_t m = 0; m < hp.shared_dims.size(); ++m) {
    w->shz[m] = take(n * hp.shared_dims[m]);
    w->shy[m] = take(n * hp.shared_dims[m]);
  }
  w->brz.assign(hp.branch_dims.size(), nullptr);
  w->bry.assign(hp.branch_dims.size(), nullptr);
  for (size_t m = 0; m < hp.branch_dims.size(); ++m) {
    w->brz[m] = take(n * hp.branch_dims[m]);
    w->bry[m] = take(n * hp.branch_dims[m]);
  }
  const int win = hp.shared_dims.empty() ? hp.F : hp.shared_dims.back();
  w->yg = take(n * win);
  w->eg = take(n);
  w->e = take(n);
  w->perm = (int32_t*)take(n + 1, 4);
  w->hstart = (int32_t*)take(hp.n_heads + 1, 4);
  w->bad = (int32_t*)take(1, 4);
  w->gs = take(n * F);
  w->gv = take(3 * n * F);
  w->gs2 = take(n * F);
  w->gv2 = take(3 * n * F);
  w->gh = take(3 * n * F);
  w->ga = take(3 * n * F);
  w->gaa = take(n * F);
  w->gin = take(2 * n * F);
  w->gU = take(3 * n * F);
  w->gV = take(3 * n * F);
  w->ga1 = take(n * F);
  w->gw = take(3 * e * F);
  w->gx1 = take(n * wmax);
  w->gx2 = take(n * wmax);
  w->E = (double*)take(B, 8);
  w->Fo = (double*)take(3 * n, 8);
  w->c = (double*)take(B, 8);
  w->dpos = (double*)take(3 * n, 8);
  w->lossbuf = (double*)take(4, 8);
  // partial-sum scratch: the most row chunks times the widest layer (with
  // its bias column)
  size_t widest = 0;
  auto wid = [&](size_t x) { widest = x > widest ? x : widest; };
  wid(3 * F * (F + 1));
  wid(F * (2 * F + 1));
  wid(3 * F * (K + 1));
  size_t din = F;
  for (int d : hp.shared_dims) { wid((size_t)d * (din + 1)); din = d; }
  {
    size_t di = din;
    for (int d : hp.branch_dims) { wid((size_t)d * (di + 1)); di = d; }
  }
  const long long rmax = (long long)3 * N > (long long)E ? (long long)3 * N : (long long)E;
  long long nzmax = (rmax + 255) / 256;
  nzmax = nzmax < 1 ? 1 : nzmax > WG_CHUNKS ? WG_CHUNKS : nzmax;
  w->wsum = (double*)take((size_t)nzmax * widest, 8);
  return off;
}

dim3 dgrid(int rows, int dout) { return dim3((unsigned)((rows + 31) / 32), (unsigned)((dout + 31) / 32)); }

// Y = X W^T + b for a layer stored [dout, din] at weight offset wofs
template <class S>
void dense(hipStream_t st, const double* th, int rows, const int32_t* range, int din, int dout, const S* X, int ldx,
           size_t wofs, const size_t* bofs, bool silu_on, S* Z, S* Y, int ldy, const S* add = nullptr, int ldadd = 0) {
  if (rows <= 0) return;
  const double* b = bofs ? th + *bofs : nullptr;
  if (silu_on)
    k_tr_dense<S, true><<<dgrid(rows, dout), 256, 0, st>>>(rows, range, din, dout, X, ldx, th + wofs, din, 1, b, add,
                                                           ldadd, Z, Y, ldy);
  else
    k_tr_dense<S, false><<<dgrid(rows, dout), 256, 0, st>>>(rows, range, din, dout, X, ldx, th + wofs, din, 1, b,
                                                            add, ldadd, nullptr, Y, ldy);
}

// GX = GY W (+ ADD) for a layer stored [dout, din]: GX [rows][din]
template <class S>
void dense_t(hipStream_t st, const double* th, int rows, const int32_t* range, int dout, int din, const S* GY, int ldgy,
             size_t wofs, S* GX, int ldgx, const S* add = nullptr, int ldadd = 0) {
  if (rows <= 0) return;
  k_tr_dense<S, false><<<dgrid(rows, din), 256, 0, st>>>(rows, range, dout, din, GY, ldgy, th + wofs, 1, din, nullptr,
                                                         add, ldadd, nullptr, GX, ldgx);
}

// Row chunks of a weight-gradient reduction over `rows` rows: at most
// WG_CHUNKS, of at least 256 rows each.
inline int wg_chunks(long long rows) {
  const long long n = (rows + 255) / 256;
  return n < 1 ? 1 : n > WG_CHUNKS ? WG_CHUNKS : (int)n;
}

// Weight (and bias) gradient of a layer stored [dout, din] at wofs (bias at
// *bofs), reducing over the rows [lo, hi) of A and B (range on the device, or
// all `rows`); `rows` bounds the row count used to cut the chunks.
template <class S>
void wgrad(hipStream_t st, double* G, double* scratch, int rows, const int32_t* range, int dout, int din,
           const S* A, int lda, const S* Bm, int ldb, size_t wofs, const size_t* bofs, const S* sc = nullptr) {
  const int dinb = din + (bofs ? 1 : 0);
  const int nz = wg_chunks(rows);
  const int rch = (rows + nz - 1) / nz;
  k_tr_wgrad<S><<<dim3((unsigned)((dinb + 31) / 32), (unsigned)((dout + 31) / 32), (unsigned)nz), 256, 0, st>>>(
      rows, range, dout, din, dinb, rch < 1 ? 1 : rch, A, lda, Bm, ldb, sc, scratch);
  k_tr_wgrad_sum<<<blocks((size_t)dout * dinb), TB, 0, st>>>(nz, dout, din, dinb, scratch, G + wofs,
                                                            bofs ? G + *bofs : nullptr);
}

// One pass.  Real (S = double): E, F into w.E, w.Fo.  Tangent (S = Dual, with
// w.c and w.dpos from the loss): the gradient into G.
template <class S>
hipError_t run_pass(hipStream_t st, painn_trainer* tr, const painn_graph* g, const int32_t* dataset_id, TrWs& w,
                    double* G) {
  constexpr bool REAL = sizeof(S) == sizeof(double);
  const Hyper& hp = tr->hp;
  const TrLayout& L = tr->lay;
  const double* th = tr->theta;
  const int N = g->N, F = hp.F, K = hp.K, F3 = 3 * F, B = g->B;
  const long long E = g->E;
  if (N == 0) {
    // structures without atoms: zero energy, no force, no gradient
    if (REAL && B > 0) k_tr_zero_d<<<blocks((size_t)B), TB, 0, st>>>((size_t)B, w.E);
    return hipGetLastError();
  }
  // geometry
  if (E > 0)
    k_tr_geom<S, REAL><<<blocks((size_t)E), TB, 0, st>>>(E, K, hp.cutoff, hp.rbf_type, g->recv, g->col, g->shift,
                                                          g->atom_struct, g->pos, g->cell, REAL ? nullptr : w.dpos,
                                                          (S*)w.rhat, (S*)w.basis, (S*)w.fc, w.dist, w.dbasis, w.dfc);
  k_tr_embed<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, g->species, th + L.emb, (S*)w.s[0], (S*)w.v[0]);
  // interaction layers
  for (int l = 0; l < hp.L; ++l) {
    const size_t* a = L.layers[l].a;
    S* s = (S*)w.s[l];
    S* v = (S*)w.v[l];
    dense<S>(st, th, N, nullptr, F, F, s, F, a[A_PHI_W1], &a[A_PHI_B1], true, (S*)w.z1[l], (S*)w.a1[l], F);
    dense<S>(st, th, N, nullptr, F, F3, (S*)w.a1[l], F, a[A_PHI_W2], &a[A_PHI_B2], false, nullptr, (S*)w.h[l], F3);
    if (E > 0)
      dense<S>(st, th, (int)E, nullptr, K, F3, (S*)w.basis, K, a[A_FILT_W], &a[A_FILT_B], false, nullptr,
               (S*)w.lin[l], F3);
    k_tr_message<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, g->row_ptr, g->col, (S*)w.h[l], s, v, (S*)w.lin[l],
                                                          (S*)w.fc, (S*)w.rhat, (S*)w.smid[l], (S*)w.vmid[l]);
    // U, V over the 3N component rows
    dense<S>(st, th, 3 * N, nullptr, F, F, (S*)w.vmid[l], F, a[A_U], nullptr, false, nullptr, (S*)w.U[l], F);
    dense<S>(st, th, 3 * N, nullptr, F, F, (S*)w.vmid[l], F, a[A_V], nullptr, false, nullptr, (S*)w.V[l], F);
    k_tr_upd_norm<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, (S*)w.smid[l], (S*)w.V[l], (S*)w.xin[l]);
    dense<S>(st, th, N, nullptr, 2 * F, F, (S*)w.xin[l], 2 * F, a[A_UPD_W1], &a[A_UPD_B1], true, (S*)w.za[l],
             (S*)w.aa[l], F);
    dense<S>(st, th, N, nullptr, F, F3, (S*)w.aa[l], F, a[A_UPD_W2], &a[A_UPD_B2], false, nullptr, (S*)w.a[l], F3);
    S* s_next = l + 1 < hp.L ? (S*)w.s[l + 1] : (S*)w.sL;
    S* v_next = l + 1 < hp.L ? (S*)w.v[l + 1] : (S*)w.vL;
    k_tr_upd_post<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, (S*)w.smid[l], (S*)w.vmid[l], (S*)w.U[l],
                                                           (S*)w.V[l], (S*)w.a[l], s_next, v_next);
  }
  // heads: shared layers (atom order), then each dataset's branch (grouped)
  const int ns = (int)hp.shared_dims.size(), nb = (int)hp.branch_dims.size(), H = hp.n_heads;
  const S* y = (const S*)w.sL;
  int dy = F;
  for (int m = 0; m < ns; ++m) {
    dense<S>(st, th, N, nullptr, dy, hp.shared_dims[m], y, dy, L.shared_w[m], &L.shared_b[m], true, (S*)w.shz[m],
             (S*)w.shy[m], hp.shared_dims[m]);
    y = (const S*)w.shy[m];
    dy = hp.shared_dims[m];
  }
  if (REAL) k_tr_group<<<1, 64, 0, st>>>(B, H, g->struct_ptr, dataset_id, w.perm, w.hstart, w.bad);
  const int32_t* slots = w.hstart + H;
  k_tr_gather<S><<<blocks((size_t)N * dy), TB, 0, st>>>(N, dy, slots, w.perm, y, (S*)w.yg);
  for (int h = 0; h < H; ++h) {
    const S* x = (const S*)w.yg;
    int dx = dy;
    for (int m = 0; m < nb; ++m) {
      const int d = hp.branch_dims[m];
      dense<S>(st, th, N, w.hstart + h, dx, d, x, dx, L.branch_w[h][m], &L.branch_b[h][m], m + 1 < nb,
               (S*)w.brz[m], (S*)w.bry[m], d);
      x = (const S*)w.bry[m];
      dx = d;
    }
  }
  // per-atom energies (the 1-wide output, grouped) back to atom order
  k_tr_zero<S><<<blocks((size_t)N), TB, 0, st>>>((size_t)N, (S*)w.e);
  k_tr_scatter<S><<<blocks((size_t)N), TB, 0, st>>>(N, 1, slots, w.perm, (const S*)w.bry[nb - 1], (S*)w.e);
  if (REAL) k_tr_energy<S><<<blocks((size_t)B), TB, 0, st>>>(B, g->struct_ptr, (const S*)w.e, w.E);

  // ---- reverse ----
  // heads: seed in grouped order, branch layers per head, then the shared
  // layers in atom order
  S* gcur = (S*)w.gx1;
  S* gnext = (S*)w.gx2;
  k_tr_seed<S><<<blocks((size_t)N), TB, 0, st>>>(N, slots, w.perm, g->atom_struct, REAL ? nullptr : w.c, gcur);
  for (int m = nb - 1; m >= 0; --m) {
    const int dout = hp.branch_dims[m], din = m > 0 ? hp.branch_dims[m - 1] : dy;
    const S* xin = m > 0 ? (const S*)w.bry[m - 1] : (const S*)w.yg;
    for (int h = 0; h < H; ++h) {
      if (!REAL) wgrad<S>(st, G, w.wsum, N, w.hstart + h, dout, din, gcur, dout, xin, din, L.branch_w[h][m], &L.branch_b[h][m]);
      dense_t<S>(st, th, N, w.hstart + h, dout, din, gcur, dout, L.branch_w[h][m], gnext, din);
    }
    if (m > 0)
      k_tr_mul_dsilu<S><<<blocks((size_t)N * din), TB, 0, st>>>(N, nullptr, din, gnext, din, (const S*)w.brz[m - 1],
                                                                 din);
    S* t = gcur;
    gcur = gnext;
    gnext = t;
  }
  // grouped -> atom order (atoms without a head keep a zero gradient)
  k_tr_zero<S><<<blocks((size_t)N * dy), TB, 0, st>>>((size_t)N * dy, gnext);
  k_tr_scatter<S><<<blocks((size_t)N * dy), TB, 0, st>>>(N, dy, slots, w.perm, gcur, gnext);
  {
    S* t = gcur;
    gcur = gnext;
    gnext = t;
  }
  for (int m = ns - 1; m >= 0; --m) {
    const int dout = hp.shared_dims[m], din = m > 0 ? hp.shared_dims[m - 1] : F;
    const S* xin = m > 0 ? (const S*)w.shy[m - 1] : (const S*)w.sL;
    k_tr_mul_dsilu<S><<<blocks((size_t)N * dout), TB, 0, st>>>(N, nullptr, dout, gcur, dout, (const S*)w.shz[m], dout);
    if (!REAL) wgrad<S>(st, G, w.wsum, N, nullptr, dout, din, gcur, dout, xin, din, L.shared_w[m], &L.shared_b[m]);
    dense_t<S>(st, th, N, nullptr, dout, din, gcur, dout, L.shared_w[m], gnext, din);
    S* t = gcur;
    gcur = gnext;
    gnext = t;
  }
  // gcur = dE/ds after the last layer; dE/dv = 0 there
  S* gs = (S*)w.gs;
  S* gv = (S*)w.gv;
  k_tr_copy<S><<<blocks((size_t)N * F), TB, 0, st>>>((size_t)N * F, gcur, gs);
  k_tr_zero<S><<<blocks((size_t)3 * N * F), TB, 0, st>>>((size_t)3 * N * F, gv);
  if (REAL && E > 0) {
    k_tr_zero_d<<<blocks((size_t)E), TB, 0, st>>>((size_t)E, w.gd);
    k_tr_zero_d<<<blocks((size_t)3 * E), TB, 0, st>>>((size_t)3 * E, w.grh);
  }
  S* gs2 = (S*)w.gs2;
  S* gv2 = (S*)w.gv2;
  for (int l = hp.L - 1; l >= 0; --l) {
    const size_t* a = L.layers[l].a;
    // update block: (gs, gv) at s', v' -> (gs2, gv2) at s_mid, v_mid
    k_tr_upd_bwd1<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, gs, gv, (S*)w.U[l], (S*)w.V[l], (S*)w.a[l],
                                                           (S*)w.ga, (S*)w.gU, (S*)w.gV);
    if (!REAL) wgrad<S>(st, G, w.wsum, N, nullptr, F3, F, (S*)w.ga, F3, (S*)w.aa[l], F, a[A_UPD_W2], &a[A_UPD_B2]);
    dense_t<S>(st, th, N, nullptr, F3, F, (S*)w.ga, F3, a[A_UPD_W2], (S*)w.gaa, F);
    k_tr_mul_dsilu<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, nullptr, F, (S*)w.gaa, F, (S*)w.za[l], F);
    if (!REAL) wgrad<S>(st, G, w.wsum, N, nullptr, F, 2 * F, (S*)w.gaa, F, (S*)w.xin[l], 2 * F, a[A_UPD_W1], &a[A_UPD_B1]);
    dense_t<S>(st, th, N, nullptr, F, 2 * F, (S*)w.gaa, F, a[A_UPD_W1], (S*)w.gin, 2 * F);
    k_tr_upd_bwd2<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, (S*)w.gin, (S*)w.xin[l], (S*)w.V[l], gs,
                                                           (S*)w.gV, gs2);
    if (!REAL) {
      wgrad<S>(st, G, w.wsum, 3 * N, nullptr, F, F, (S*)w.gU, F, (S*)w.vmid[l], F, a[A_U], nullptr);
      wgrad<S>(st, G, w.wsum, 3 * N, nullptr, F, F, (S*)w.gV, F, (S*)w.vmid[l], F, a[A_V], nullptr);
    }
    dense_t<S>(st, th, 3 * N, nullptr, F, F, (S*)w.gU, F, a[A_U], gv2, F, gv, F);
    dense_t<S>(st, th, 3 * N, nullptr, F, F, (S*)w.gV, F, a[A_V], gv2, F, gv2, F);
    // message: (gs2, gv2) at s_mid, v_mid -> dE/dh, dE/dv before it (gv), dE/dw
    k_tr_message_bwd<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, F, g->t_ptr, g->t_edge, g->recv, (S*)w.h[l],
                                                              (S*)w.v[l], (S*)w.lin[l], (S*)w.fc, (S*)w.rhat, gs2,
                                                              gv2, (S*)w.gh, gv, (S*)w.gw);
    if (E > 0) {
      if (REAL) {
        // lin' = W_f g'(d) for dE/dd
        k_tr_dense<double, false><<<dgrid((int)E, F3), 256, 0, st>>>((int)E, nullptr, K, F3, w.dbasis, K,
                                                                     th + a[A_FILT_W], K, 1, nullptr, nullptr, 0,
                                                                     nullptr, w.linp, F3);
        k_tr_edge_bwd<<<(unsigned)((E + 3) / 4), 256, 0, st>>>(E, F, g->recv, g->col, (const double*)w.h[l],
                                                               (const double*)w.lin[l], w.linp, (const double*)w.fc,
                                                               w.dfc, (const double*)gv2, (const double*)w.gw, w.gd,
                                                               w.grh);
      } else {
        wgrad<S>(st, G, w.wsum, (int)E, nullptr, F3, K, (S*)w.gw, F3, (S*)w.basis, K, a[A_FILT_W], &a[A_FILT_B], (S*)w.fc);
      }
    }
    // phi: dE/dh -> dE/ds before the message (its residual gs2 added)
    if (!REAL) wgrad<S>(st, G, w.wsum, N, nullptr, F3, F, (S*)w.gh, F3, (S*)w.a1[l], F, a[A_PHI_W2], &a[A_PHI_B2]);
    dense_t<S>(st, th, N, nullptr, F3, F, (S*)w.gh, F3, a[A_PHI_W2], (S*)w.ga1, F);
    k_tr_mul_dsilu<S><<<blocks((size_t)N * F), TB, 0, st>>>(N, nullptr, F, (S*)w.ga1, F, (S*)w.z1[l], F);
    if (!REAL) wgrad<S>(st, G, w.wsum, N, nullptr, F, F, (S*)w.ga1, F, (S*)w.s[l], F, a[A_PHI_W1], &a[A_PHI_B1]);
    dense_t<S>(st, th, N, nullptr, F, F, (S*)w.ga1, F, a[A_PHI_W1], gs, F, gs2, F);
  }
  if (!REAL)
    k_tr_emb_grad<S><<<blocks((size_t)hp.n_species * F), TB, 0, st>>>(N, F, hp.n_species, g->species, gs, G + L.emb);
  if (REAL) {
    if (E > 0)
      k_tr_edge_dr<<<blocks((size_t)E), TB, 0, st>>>(E, w.dist, (const double*)w.rhat, w.gd, w.grh, w.gr);
    k_tr_forces<<<blocks((size_t)N), TB, 0, st>>>(N, g->row_ptr, g->t_ptr, g->t_edge, w.gr, w.Fo);
  }
  return hipGetLastError();
}

}  // namespace

extern "C" {

painn_status painn_trainer_create(painn_ctx* ctx, const painn_model* model, const painn_train_config* cfg,
                                  painn_trainer** out) {
  if (!ctx) return PAINN_E_ARG;
  ctx->err.clear();
  if (!model || !out) return tfail(ctx, PAINN_E_ARG, "null model or output");
  if (model->ctx != ctx) return tfail(ctx, PAINN_E_ARG, "model from another context");
  *out = nullptr;
  painn_train_config c{6.34e-4, 0.9, 0.999, 1e-8, 0.01, 94.8};
  if (cfg) c = *cfg;
  if (!(c.lr >= 0.0) || !(c.beta1 >= 0.0 && c.beta1 < 1.0) || !(c.beta2 >= 0.0 && c.beta2 < 1.0) ||
      !(c.eps > 0.0) || !(c.weight_decay >= 0.0) || !(c.force_weight >= 0.0) || !isfinite(c.lr) ||
      !isfinite(c.eps) || !isfinite(c.weight_decay) || !isfinite(c.force_weight))
    return tfail(ctx, PAINN_E_ARG, "training hyperparameters out of range");
  painn_trainer* tr = new (std::nothrow) painn_trainer();
  if (!tr) return tfail(ctx, PAINN_E_OOM, "host allocation failed");
  tr->ctx = ctx;
  tr->cfg = c;
  tr->hp = model->hp;
  tr->hp.F = model->hp.F_logical;
  tr->lay = make_layout(tr->hp);
  // the model's weights at its own width, in file order
  std::vector<double> host(tr->lay.total);
  const Hyper& hpp = model->hp;
  const int Fp = hpp.F, F = tr->hp.F;
  auto map = [&](int d, size_t x) -> size_t { return d < 0 ? (x / F) * Fp + x % F : x; };
  struct Dim { int rows, cols; };
  std::vector<Dim> dims;
  dims.push_back({hpp.n_species, -1});
  for (int l = 0; l < hpp.L; ++l) {
    const Dim per[A_PER_LAYER] = {{-1, -1}, {-1, 1}, {-3, -1}, {-3, 1}, {-3, hpp.K}, {-3, 1},
                                  {-1, -1}, {-1, -1}, {-1, -2}, {-1, 1}, {-3, -1}, {-3, 1}};
    for (const Dim& d : per) dims.push_back(d);
  }
  int din = -1;
  for (int d : hpp.shared_dims) { dims.push_back({d, din}); dims.push_back({d, 1}); din = d; }
  for (int h = 0; h < hpp.n_heads; ++h) {
    int di = din;
    for (int d : hpp.branch_dims) { dims.push_back({d, di}); dims.push_back({d, 1}); di = d; }
  }
  auto ext = [](int d, int w) { return d < 0 ? (size_t)(-d) * w : (size_t)d; };
  size_t o = 0;
  for (size_t a = 0; a < dims.size(); ++a) {
    const Dim d = dims[a];
    const size_t R = ext(d.rows, F), C = ext(d.cols, F), Cp = ext(d.cols, Fp);
    const double* src = model->master.data() + model->offsets[a];
    for (size_t r = 0; r < R; ++r)
      for (size_t cc = 0; cc < C; ++cc) host[o + r * C + cc] = src[map(d.rows, r) * Cp + map(d.cols, cc)];
    o += R * C;
  }
  (void)hipSetDevice(ctx->device);
  const size_t P = tr->lay.total;
  hipError_t e = hipMalloc((void**)&tr->theta, P * sizeof(double));
  if (e == hipSuccess) e = hipMalloc((void**)&tr->grad, P * sizeof(double));
  if (e == hipSuccess) e = hipMalloc((void**)&tr->m1, P * sizeof(double));
  if (e == hipSuccess) e = hipMalloc((void**)&tr->m2, P * sizeof(double));
  if (e == hipSuccess) e = hipMemcpyAsync(tr->theta, host.data(), P * sizeof(double), hipMemcpyHostToDevice, ctx->stream);
  if (e == hipSuccess) {
    k_tr_zero_d<<<blocks(P), TB, 0, ctx->stream>>>(P, tr->grad);
    k_tr_zero_d<<<blocks(P), TB, 0, ctx->stream>>>(P, tr->m1);
    k_tr_zero_d<<<blocks(P), TB, 0, ctx->stream>>>(P, tr->m2);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);   // the host copy is released on return
  if (e != hipSuccess) {
    (void)hipGetLastError();
    painn_trainer_free(tr);
    return tfail(ctx, PAINN_E_OOM, std::string("trainer allocation: ") + hipGetErrorString(e));
  }
  *out = tr;
  return PAINN_OK;
}

painn_status painn_trainer_free(painn_trainer* tr) {
  if (!tr) return PAINN_OK;
  if (tr->ctx) {
    (void)hipSetDevice(tr->ctx->device);
    (void)hipStreamSynchronize(tr->ctx->stream);
  }
  void* bufs[] = {tr->theta, tr->grad, tr->m1, tr->m2, tr->ws};
  for (void* p : bufs)
    if (p) (void)hipFree(p);
  delete tr;
  return PAINN_OK;
}

painn_status painn_trainer_step(painn_trainer* tr, const painn_graph* g, const int32_t* dataset_id,
                                const double* energy_ref, const double* force_ref, double* loss) {
  if (!tr) return PAINN_E_ARG;
  painn_ctx* ctx = tr->ctx;
  ctx->err.clear();
  if (!g) return tfail(ctx, PAINN_E_ARG, "null graph");
  if (g->ctx != ctx) return tfail(ctx, PAINN_E_ARG, "graph from another context");
  if (!g->valid) return tfail(ctx, PAINN_E_ARG, "graph is not built (its last build failed)");
  if (g->cutoff != tr->hp.cutoff) return tfail(ctx, PAINN_E_ARG, "graph cutoff differs from the model's cutoff");
  if (g->max_neighbors != tr->hp.max_neighbors)
    return tfail(ctx, PAINN_E_ARG, "graph neighbour cap differs from the model's");
  if (g->N > 0 && (g->species_min < 0 || g->species_max >= tr->hp.n_species))
    return tfail(ctx, PAINN_E_SPECIES, "species index outside [0, n_species)");
  if ((g->B > 0 && !energy_ref) || (g->N > 0 && !force_ref))
    return tfail(ctx, PAINN_E_ARG, "null reference energies or forces");
  if (g->E > (1LL << 31) - 1 || 3LL * g->N * tr->hp.F > (1LL << 31) - 1)
    return tfail(ctx, PAINN_E_UNSUPPORTED, "batch too large for one training step");
  (void)hipSetDevice(ctx->device);
  hipStream_t st = ctx->stream;
  painn_graph* gm = const_cast<painn_graph*>(g);
  if (!gm->t_valid && g->N > 0) {
    hipError_t e = hipSuccess;
    size_t cap_a = gm->cap_t_atoms, cap_e = gm->cap_t_edges;
    if ((size_t)g->N + 1 > cap_a || !gm->t_ptr || !gm->t_count) {
      if (gm->t_ptr) { (void)hipFree(gm->t_ptr); gm->t_ptr = nullptr; }
      if (gm->t_count) { (void)hipFree(gm->t_count); gm->t_count = nullptr; }
      cap_a = (size_t)g->N + 1 + (g->N + 1) / 4;
      e = hipMalloc((void**)&gm->t_ptr, cap_a * sizeof(int32_t));
      if (e == hipSuccess) e = hipMalloc((void**)&gm->t_count, cap_a * sizeof(int32_t));
      gm->cap_t_atoms = e == hipSuccess ? cap_a : 0;
    }
    if (e == hipSuccess && ((size_t)g->E + 1 > cap_e || !gm->t_edge)) {
      if (gm->t_edge) { (void)hipFree(gm->t_edge); gm->t_edge = nullptr; }
      cap_e = (size_t)g->E + 1 + (g->E + 1) / 4;
      e = hipMalloc((void**)&gm->t_edge, cap_e * sizeof(int32_t));
      gm->cap_t_edges = e == hipSuccess ? cap_e : 0;
    }
    if (e == hipSuccess) e = launch_transpose(st, ctx->prof, gm);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return tfail(ctx, PAINN_E_HIP, std::string("edge transpose: ") + hipGetErrorString(e));
    }
    gm->t_valid = true;
  }
  TrWs w;
  const size_t need = carve(&w, nullptr, tr->hp, g->N, g->E, g->B);
  if (need > tr->ws_bytes) {
    if (tr->ws) {
      (void)hipStreamSynchronize(st);
      (void)hipFree(tr->ws);
      tr->ws = nullptr;
      tr->ws_bytes = 0;
    }
    const size_t want = need + need / 4;
    if (hipMalloc(&tr->ws, want) != hipSuccess) {
      (void)hipGetLastError();
      return tfail(ctx, PAINN_E_OOM, "training workspace allocation failed");
    }
    tr->ws_bytes = want;
  }
  carve(&w, (char*)tr->ws, tr->hp, g->N, g->E, g->B);
  (void)hipGetLastError();
  const size_t P = tr->lay.total;
  k_tr_zero_d<<<blocks(P), TB, 0, st>>>(P, tr->grad);
  prof_mark(ctx->prof, st, KC_TRAIN_REAL, true);
  hipError_t e = run_pass<double>(st, tr, g, dataset_id, w, nullptr);
  if (e == hipSuccess && g->B > 0) {
    k_tr_loss<<<1, 256, 0, st>>>(g->B, g->N, tr->cfg.force_weight, w.E, energy_ref, w.Fo, force_ref, w.bad, w.c,
                                 w.dpos, loss ? loss : w.lossbuf);
    e = hipGetLastError();
  }
  prof_mark(ctx->prof, st, KC_TRAIN_REAL, false);
  prof_mark(ctx->prof, st, KC_TRAIN_TANGENT, true);
  if (e == hipSuccess) e = run_pass<Dual>(st, tr, g, dataset_id, w, tr->grad);
  prof_mark(ctx->prof, st, KC_TRAIN_TANGENT, false);
  if (e == hipSuccess) {
    tr->t += 1;
    const painn_train_config& c = tr->cfg;
    const double bc1 = 1.0 - pow(c.beta1, (double)tr->t), bc2 = 1.0 - pow(c.beta2, (double)tr->t);
    prof_mark(ctx->prof, st, KC_TRAIN_ADAMW, true);
    k_tr_adamw<<<blocks(P), TB, 0, st>>>(P, tr->theta, tr->grad, tr->m1, tr->m2, c.lr, c.beta1, c.beta2, c.eps,
                                        c.weight_decay, bc1, bc2);
    prof_mark(ctx->prof, st, KC_TRAIN_ADAMW, false);
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return tfail(ctx, PAINN_E_HIP, std::string("training step launch: ") + hipGetErrorString(e));
  }
  return PAINN_OK;
}

painn_status painn_trainer_params(const painn_trainer* tr, int64_t* n_params, double* params, double* grad) {
  if (!tr) return PAINN_E_ARG;
  painn_ctx* ctx = tr->ctx;
  ctx->err.clear();
  if (n_params) *n_params = (int64_t)tr->lay.total;
  (void)hipSetDevice(ctx->device);
  const size_t bytes = tr->lay.total * sizeof(double);
  hipError_t e = hipSuccess;
  if (params) e = hipMemcpyAsync(params, tr->theta, bytes, hipMemcpyDeviceToDevice, ctx->stream);
  if (e == hipSuccess && grad) e = hipMemcpyAsync(grad, tr->grad, bytes, hipMemcpyDeviceToDevice, ctx->stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return tfail(ctx, PAINN_E_HIP, std::string("parameter copy: ") + hipGetErrorString(e));
  }
  return PAINN_OK;
}

}  // extern "C"
