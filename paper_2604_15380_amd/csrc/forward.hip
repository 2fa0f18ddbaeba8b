// Batched PaiNN forward pass on gfx950: embedding, per layer the message
// step (radial filter under a cosine cutoff, scalar/vector messages reduced
// per receiver) and the update step (U/V channel mixing, gate MLP), then the
// per-dataset heads and the per-structure energy sum.  The model is the lead
// PaiNN backbone (section "Flagship Training of Top HPO Models", Table 5) with
// the message and update blocks of the published PaiNN method.
//
// Data layout in HBM (row-major, storage type T of the precision):
//   s [N][F], v [N][3][F] (double buffered), h [N][3F] = [h_s | h_v | h_r],
//   e [N] (accumulation type).  Edges: CSR sorted by receiver.
#include "mfma.h"

namespace {

// ---------------------------------------------------------------- embed ----
template <class P>
__global__ void __launch_bounds__(256) k_embed(int N, int F, const int32_t* __restrict__ species,
                                              const typename P::T* __restrict__ emb,
                                              typename P::T* __restrict__ s,
                                              typename P::T* __restrict__ v) {
  const size_t tot = (size_t)N * F;
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < tot; x += (size_t)gridDim.x * blockDim.x) {
    const size_t i = x / F, f = x % F;
    s[x] = emb[(size_t)species[i] * F + f];
    v[3 * i * F + f] = P::st(0);
    v[3 * i * F + F + f] = P::st(0);
    v[3 * i * F + 2 * F + f] = P::st(0);
  }
}

// Load rows [row0, row0 + rows) of a [N][F] storage array into LDS (row
// stride ld); rows past N are zero.
template <class P, int F>
__device__ __forceinline__ void load_rows(typename P::T* dst, int ld, const typename P::T* src,
                                          size_t row0, int rows, int N) {
  for (int x = threadIdx.x; x < rows * F; x += blockDim.x) {
    const int r = x / F, c = x % F;
    const size_t g = row0 + r;
    dst[r * ld + c] = g < (size_t)N ? src[g * F + c] : P::st(0);
  }
}

// ------------------------------------------------------------------ phi ----
// h = W2 silu(W1 s + b1) + b2 for a tile of 16 RT atoms.
template <class P, int F, int RT>
__device__ __forceinline__ void phi_tile(const typename P::T* X, int ldx, typename P::T* H,
                                         size_t row0, int N, const DenseDev& d1,
                                         const DenseDev& d2, typename P::T* __restrict__ h) {
  using A = typename P::A;
  constexpr int LD = F + P::PAD;
  const int lane = threadIdx.x & 63;
  dense_tiles<P, RT, 4>(X, ldx, d1, [&](int ct, typename P::C* acc) {
    const int col = ct * 16 + (lane & 15);
    const A bias = ((const A*)d1.b)[col];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) H[(r * 16 + P::row(lane, i)) * LD + col] = P::st(silu<A>(acc[r][i] + bias));
  });
  __syncthreads();
  dense_tiles<P, RT, 4>(H, LD, d2, [&](int ct, typename P::C* acc) {
    const int col = ct * 16 + (lane & 15);
    const A bias = ((const A*)d2.b)[col];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) {
        const size_t row = row0 + r * 16 + P::row(lane, i);
        if (row < (size_t)N) h[row * 3 * F + col] = P::st(acc[r][i] + bias);
      }
  });
}

template <class P, int F, int RT>
__global__ void __launch_bounds__(256) k_phi(int N, const typename P::T* __restrict__ s,
                                            typename P::T* __restrict__ h, DenseDev d1, DenseDev d2) {
  constexpr int LD = F + P::PAD;
  __shared__ __attribute__((aligned(16))) typename P::T X[16 * RT * LD];
  __shared__ __attribute__((aligned(16))) typename P::T H[16 * RT * LD];
  const size_t row0 = (size_t)blockIdx.x * 16 * RT;
  load_rows<P, F>(X, LD, s, row0, 16 * RT, N);
  __syncthreads();
  phi_tile<P, F, RT>(X, LD, H, row0, N, d1, d2, h);
}

// -------------------------------------------------------------- message ----
// One workgroup of F threads per receiver i; thread f owns channel f of
// every part.  Per edge e = (i <- j, n):
//   w_e = f_c(d) (Wf g(d) + bf)                 filter, 3F channels
//   ds_i    += h^s_j w^s_e
//   dv_i[c] += v_j[c] h^v_j w^v_e + rhat[c] h^r_j w^r_e
// The K Gaussians times f_c of a chunk of edges are computed once per edge
// (spread over the workgroup) into LDS and broadcast; the filter rows live in
// registers.  The sum over the receiver's edges is a plain in-register
// reduction (the CSR is sorted by receiver), so there are no atomics and the
// result is deterministic.
struct MsgArgs {
  int N, F, K;
  const int32_t* row_ptr;
  const int32_t* col;
  const int32_t* shift;
  const int32_t* atom_struct;
  const double* pos;
  const double* cell;
  double rc, gamma, delta;
  const void* filt;  // [3F][KP+1], accumulation type, column KP = bias
  const void* h;
  const void* v_in;
  void* s;
  void* v_out;
};

constexpr int MSG_CH = 64;  // edges per chunk

template <class P, int KP>
__global__ void __launch_bounds__(256) k_message(MsgArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  constexpr int RS = KP + 4;  // LDS row: KP Gaussians, f_c, 3 zeros
  __shared__ __attribute__((aligned(16))) A eg[MSG_CH * RS];
  __shared__ A er[MSG_CH * 4];
  __shared__ int ej[MSG_CH];
  const int i = blockIdx.x;
  const int f = threadIdx.x;
  const int F = a.F;
  const A* filt = (const A*)a.filt;
  A wS[KP + 1], wV[KP + 1], wR[KP + 1];
#pragma unroll
  for (int k = 0; k <= KP; ++k) {
    wS[k] = filt[(size_t)f * (KP + 1) + k];
    wV[k] = filt[(size_t)(F + f) * (KP + 1) + k];
    wR[k] = filt[(size_t)(2 * F + f) * (KP + 1) + k];
  }
  const T* h = (const T*)a.h;
  const T* vin = (const T*)a.v_in;
  const int b = a.atom_struct[i];
  double C[9];
  for (int k = 0; k < 9; ++k) C[k] = a.cell[9 * b + k];
  const double xi = a.pos[3 * i], yi = a.pos[3 * i + 1], zi = a.pos[3 * i + 2];
  const int e_begin = a.row_ptr[i], e_end = a.row_ptr[i + 1];
  A acc_s = 0, acc_v0 = 0, acc_v1 = 0, acc_v2 = 0;
  const double pi_rc = 3.14159265358979323846 / a.rc;
  for (int e0 = e_begin; e0 < e_end; e0 += MSG_CH) {
    const int cnt = min(MSG_CH, e_end - e0);
    for (int t = f; t < cnt; t += F) {
      const int e = e0 + t;
      const int j = a.col[e];
      const int sh = a.shift[e];
      const double n0 = (double)(int8_t)(sh & 0xff), n1 = (double)(int8_t)((sh >> 8) & 0xff),
                   n2 = (double)(int8_t)((sh >> 16) & 0xff);
      const double rx = (a.pos[3 * j] - xi) + ((n0 * C[0] + n1 * C[3]) + n2 * C[6]);
      const double ry = (a.pos[3 * j + 1] - yi) + ((n0 * C[1] + n1 * C[4]) + n2 * C[7]);
      const double rz = (a.pos[3 * j + 2] - zi) + ((n0 * C[2] + n1 * C[5]) + n2 * C[8]);
      const double d = sqrt(rx * rx + ry * ry + rz * rz);
      const double inv = 1.0 / d;
      er[4 * t + 0] = (A)(rx * inv);
      er[4 * t + 1] = (A)(ry * inv);
      er[4 * t + 2] = (A)(rz * inv);
      er[4 * t + 3] = (A)d;
      ej[t] = j;
      const double fc = d < a.rc ? 0.5 * (cos(d * pi_rc) + 1.0) : 0.0;
      eg[t * RS + KP] = (A)fc;
      eg[t * RS + KP + 1] = 0;
      eg[t * RS + KP + 2] = 0;
      eg[t * RS + KP + 3] = 0;
    }
    __syncthreads();
    for (int x = f; x < cnt * KP; x += F) {
      const int t = x / KP, k = x % KP;
      A g = 0;
      if (k < a.K) {
        const A dd = er[4 * t + 3] - (A)(k * a.delta);
        g = P::ex(-(A)a.gamma * dd * dd) * eg[t * RS + KP];
      }
      eg[t * RS + k] = g;
    }
    __syncthreads();
    for (int t = 0; t < cnt; ++t) {
      const int j = ej[t];
      const A* gp = eg + t * RS;
      A ws = wS[KP] * gp[KP], wv = wV[KP] * gp[KP], wr = wR[KP] * gp[KP];
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        const A gk = gp[k];
        ws += wS[k] * gk;
        wv += wV[k] * gk;
        wr += wR[k] * gk;
      }
      const size_t hb = (size_t)j * 3 * F;
      const A hs = P::ld(h[hb + f]), hv = P::ld(h[hb + F + f]), hr = P::ld(h[hb + 2 * F + f]);
      const A vj0 = P::ld(vin[hb + f]), vj1 = P::ld(vin[hb + F + f]), vj2 = P::ld(vin[hb + 2 * F + f]);
      acc_s += hs * ws;
      const A pv = hv * wv, pr = hr * wr;
      acc_v0 += vj0 * pv + er[4 * t + 0] * pr;
      acc_v1 += vj1 * pv + er[4 * t + 1] * pr;
      acc_v2 += vj2 * pv + er[4 * t + 2] * pr;
    }
    __syncthreads();
  }
  T* s = (T*)a.s;
  T* vout = (T*)a.v_out;
  const size_t ib = (size_t)i * 3 * F;
  s[(size_t)i * F + f] = P::st(P::ld(s[(size_t)i * F + f]) + acc_s);
  vout[ib + f] = P::st(P::ld(vin[ib + f]) + acc_v0);
  vout[ib + F + f] = P::st(P::ld(vin[ib + F + f]) + acc_v1);
  vout[ib + 2 * F + f] = P::st(P::ld(vin[ib + 2 * F + f]) + acc_v2);
}

// --------------------------------------------------------------- update ----
// Tile of 16 atoms, 4 waves.  U[c] = WU v[c], V[c] = WV v[c] for c = x, y, z
// one component at a time (v[c] staged in LDS); U, |V|^2 and <U, V> stay in
// the registers of the wave that owns the feature tile.  Then
// a = W2a silu(W1a [s; |V|] + b1a) + b2a, with each wave computing the
// a_vv / a_sv / a_ss column tiles of its own feature tiles, so the final
//   v[c] += a_vv U[c],  s += a_sv <U, V> + a_ss
// needs no exchange.  Optionally the next layer's phi follows on the new s.
struct UpdArgs {
  int N;
  void* s;
  void* v;
  void* h;
  DenseDev uv, upd1, upd2, phi1, phi2;
};

template <class P, int F, bool FUSE_PHI>
__global__ void __launch_bounds__(256) k_update(UpdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int NFT = F / 16;        // feature tiles
  constexpr int FTW = NFT / 4;       // per wave
  constexpr int LD1 = F + P::PAD, LD2 = 2 * F + P::PAD;
  __shared__ __attribute__((aligned(16))) T VS[16 * LD1];   // v[c] slice, later the MLP hidden
  __shared__ __attribute__((aligned(16))) T SN[16 * LD2];   // [s ; |V|]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t row0 = (size_t)blockIdx.x * 16;
  const int N = a.N;
  T* s = (T*)a.s;
  T* v = (T*)a.v;
  for (int x = threadIdx.x; x < 16 * F; x += blockDim.x) {
    const int r = x / F, c = x % F;
    SN[r * LD2 + c] = row0 + r < (size_t)N ? s[(row0 + r) * F + c] : P::st(0);
  }
  C U[FTW][3], nsq[FTW], pd[FTW];
  for (int q = 0; q < FTW; ++q)
    for (int i = 0; i < 4; ++i) nsq[q][i] = pd[q][i] = 0;
  const int nkb = a.uv.din_p / P::KC;
  const T* Wuv = (const T*)a.uv.w;
  for (int c = 0; c < 3; ++c) {
    __syncthreads();
    for (int x = threadIdx.x; x < 16 * F; x += blockDim.x) {
      const int r = x / F, col = x % F;
      VS[r * LD1 + col] = row0 + r < (size_t)N ? v[(row0 + r) * 3 * F + c * F + col] : P::st(0);
    }
    __syncthreads();
    const T* xp = VS + (lane & 15) * LD1 + (lane >> 4) * P::KPL;
    for (int q = 0; q < FTW; ++q) {
      const int ft = wave + 4 * q;
      C au, av;
      for (int i = 0; i < 4; ++i) au[i] = av[i] = 0;
      const T* wu = Wuv + (size_t)ft * nkb * 64 * P::KPL + (size_t)lane * P::KPL;
      const T* wv = Wuv + (size_t)(NFT + ft) * nkb * 64 * P::KPL + (size_t)lane * P::KPL;
      for (int kb = 0; kb < nkb; ++kb) {
        typename P::Fr x = P::frag(xp + kb * P::KC);
        au = P::mfma(x, P::frag(wu + (size_t)kb * 64 * P::KPL), au);
        av = P::mfma(x, P::frag(wv + (size_t)kb * 64 * P::KPL), av);
      }
      U[q][c] = au;
      for (int i = 0; i < 4; ++i) {
        nsq[q][i] += av[i] * av[i];
        pd[q][i] += au[i] * av[i];
      }
    }
  }
  for (int q = 0; q < FTW; ++q) {
    const int col = (wave + 4 * q) * 16 + (lane & 15);
    for (int i = 0; i < 4; ++i) SN[(P::row(lane, i)) * LD2 + F + col] = P::st(sqrt(nsq[q][i]));
  }
  __syncthreads();
  T* H = VS;
  dense_tiles<P, 1, 4>(SN, LD2, a.upd1, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15);
    const A bias = ((const A*)a.upd1.b)[col];
    for (int i = 0; i < 4; ++i) H[(P::row(lane, i)) * LD1 + col] = P::st(silu<A>(acc[0][i] + bias));
  });
  __syncthreads();
  {
    const int nkb2 = a.upd2.din_p / P::KC;
    const T* W2 = (const T*)a.upd2.w;
    const A* b2 = (const A*)a.upd2.b;
    const T* xp = H + (lane & 15) * LD1 + (lane >> 4) * P::KPL;
    for (int q = 0; q < FTW; ++q) {
      const int ft = wave + 4 * q;
      C avv, asv, ass;
      for (int i = 0; i < 4; ++i) avv[i] = asv[i] = ass[i] = 0;
      const T* w0 = W2 + (size_t)ft * nkb2 * 64 * P::KPL + (size_t)lane * P::KPL;
      const T* w1 = W2 + (size_t)(NFT + ft) * nkb2 * 64 * P::KPL + (size_t)lane * P::KPL;
      const T* w2 = W2 + (size_t)(2 * NFT + ft) * nkb2 * 64 * P::KPL + (size_t)lane * P::KPL;
      for (int kb = 0; kb < nkb2; ++kb) {
        typename P::Fr x = P::frag(xp + kb * P::KC);
        avv = P::mfma(x, P::frag(w0 + (size_t)kb * 64 * P::KPL), avv);
        asv = P::mfma(x, P::frag(w1 + (size_t)kb * 64 * P::KPL), asv);
        ass = P::mfma(x, P::frag(w2 + (size_t)kb * 64 * P::KPL), ass);
      }
      const int col = ft * 16 + (lane & 15);
      const A bvv = b2[col], bsv = b2[F + col], bss = b2[2 * F + col];
      for (int i = 0; i < 4; ++i) {
        const int r = P::row(lane, i);
        const size_t row = row0 + r;
        const A g_vv = avv[i] + bvv, g_sv = asv[i] + bsv, g_ss = ass[i] + bss;
        const A sn = P::ld(SN[r * LD2 + col]) + g_sv * pd[q][i] + g_ss;
        const T st = P::st(sn);
        SN[r * LD2 + col] = st;
        if (row < (size_t)N) {
          s[row * F + col] = st;
          for (int c = 0; c < 3; ++c) {
            const size_t o = row * 3 * F + c * F + col;
            v[o] = P::st(P::ld(v[o]) + g_vv * U[q][c][i]);
          }
        }
      }
    }
  }
  if (FUSE_PHI) {
    __syncthreads();
    phi_tile<P, F, 1>(SN, LD2, VS, row0, N, a.phi1, a.phi2, (T*)a.h);
  }
}

// ---------------------------------------------------------------- heads ----
// Per atom: shared MLP (silu after every layer), then the branch MLP of the
// structure's dataset (silu between layers, last layer linear to a scalar).
// A tile of 16 atoms runs each distinct branch present in it.
struct HeadArgs {
  int N, F, n_heads, ns, nb, lds_s, lds_b;   // row strides of the shared / branch buffers
  const void* s;
  const int32_t* atom_struct;
  const int32_t* dataset_id;
  const void* const* table;  // [n_heads][nb][2] = (packed w, bias)
  DenseDev shared[16];
  int bdin[16], bdout[16];
  void* e;
};

// LDS: X [16][F+PAD] (final s), SA/SB [16][lds_s] (shared layers), B0/B1
// [16][lds_b] (branch hidden layers).
template <class P, int F>
__global__ void __launch_bounds__(256) k_heads(HeadArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  constexpr int LDX = F + P::PAD;
  T* X = (T*)smem;
  T* SA = X + 16 * LDX;
  T* SB = SA + 16 * a.lds_s;
  T* B0 = SB + 16 * a.lds_s;
  T* B1 = B0 + 16 * a.lds_b;
  __shared__ int hd[16];
  __shared__ int heads[16];
  __shared__ int nh;
  __shared__ A eo[16];
  const int lane = threadIdx.x & 63;
  const size_t row0 = (size_t)blockIdx.x * 16;
  const int N = a.N;
  load_rows<P, F>(X, LDX, (const T*)a.s, row0, 16, N);
  if (threadIdx.x < 16) {
    const size_t row = row0 + threadIdx.x;
    int h = -2;                                  // padding row
    if (row < (size_t)N) {
      h = a.dataset_id ? a.dataset_id[a.atom_struct[row]] : 0;
      if (h < 0 || h >= a.n_heads) h = -1;       // invalid id -> NaN energy
    }
    hd[threadIdx.x] = h;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int n = 0;
    for (int r = 0; r < 16; ++r) {
      const int h = hd[r];
      if (h < 0) continue;
      bool seen = false;
      for (int q = 0; q < n; ++q) seen |= heads[q] == h;
      if (!seen) heads[n++] = h;
    }
    nh = n;
  }
  __syncthreads();
  // shared layers: X -> SA -> SB -> SA ...
  const T* S = X;
  int ld_S = LDX;
  for (int m = 0; m < a.ns; ++m) {
    T* dst = (m & 1) ? SB : SA;
    const int lds = a.lds_s;
    dense_tiles<P, 1, 4>(S, ld_S, a.shared[m], [&](int ct, typename P::C* acc) {
      const int col = ct * 16 + (lane & 15);
      const A bias = ((const A*)a.shared[m].b)[col];
      for (int i = 0; i < 4; ++i) dst[(P::row(lane, i)) * lds + col] = P::st(silu<A>(acc[0][i] + bias));
    });
    __syncthreads();
    S = dst;
    ld_S = lds;
  }
  A e_row = 0;
  const int rtid = threadIdx.x;
  for (int q = 0; q < nh; ++q) {
    const int head = heads[q];
    const T* in = S;
    int ld_in = ld_S;
    for (int m = 0; m < a.nb; ++m) {
      DenseDev L;
      L.w = (void*)a.table[((size_t)head * a.nb + m) * 2];
      L.b = (void*)a.table[((size_t)head * a.nb + m) * 2 + 1];
      L.din = a.bdin[m];
      L.dout = a.bdout[m];
      L.din_p = pad32(a.bdin[m]);
      L.dout_p = pad32(a.bdout[m]);
      const bool last = m == a.nb - 1;
      T* dst = (m & 1) ? B1 : B0;
      const int ldb = a.lds_b;
      dense_tiles<P, 1, 4>(in, ld_in, L, [&](int ct, typename P::C* acc) {
        const int col = ct * 16 + (lane & 15);
        const A bias = ((const A*)L.b)[col];
        for (int i = 0; i < 4; ++i) {
          const int r = P::row(lane, i);
          const A y = acc[0][i] + bias;
          if (last) {
            if (col == 0) eo[r] = y;
          } else {
            dst[r * ldb + col] = P::st(silu<A>(y));
          }
        }
      });
      __syncthreads();
      in = dst;
      ld_in = ldb;
    }
    if (rtid < 16 && hd[rtid] == head) e_row = eo[rtid];
    __syncthreads();
  }
  if (rtid < 16) {
    const size_t row = row0 + rtid;
    if (row < (size_t)N) {
      A* e = (A*)a.e;
      e[row] = hd[rtid] == -1 ? (A)NAN : e_row;
    }
  }
}

// ------------------------------------------------------------ energies ----
template <class A>
__global__ void __launch_bounds__(256) k_energy(int B, const int32_t* __restrict__ struct_ptr,
                                               const A* __restrict__ e, double* __restrict__ E) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  double acc = 0.0;
  for (int i = struct_ptr[b]; i < struct_ptr[b + 1]; ++i) acc += (double)e[i];
  E[b] = acc;
}

template <class P>
__global__ void __launch_bounds__(256) k_export(int N, int F, const typename P::T* __restrict__ s,
                                               const typename P::T* __restrict__ v,
                                               double* __restrict__ so, double* __restrict__ vo) {
  const size_t tot = (size_t)N * F;
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < tot; x += (size_t)gridDim.x * blockDim.x) {
    so[x] = (double)P::ld(s[x]);
    const size_t i = x / F, f = x % F;
    for (int c = 0; c < 3; ++c) vo[(3 * i + c) * F + f] = (double)P::ld(v[(3 * i + c) * F + f]);
  }
}

inline int grid_for(size_t n, int per) {
  size_t g = (n + per - 1) / per;
  if (g > 65536) g = 65536;
  return (int)(g ? g : 1);
}

template <class P, int KP>
void launch_message_kp(hipStream_t st, const MsgArgs& a) {
  k_message<P, KP><<<a.N, a.F, 0, st>>>(a);
}

template <class P>
hipError_t launch_message(hipStream_t st, int KP, const MsgArgs& a) {
  switch (KP) {
    case 4: launch_message_kp<P, 4>(st, a); break;
    case 8: launch_message_kp<P, 8>(st, a); break;
    case 12: launch_message_kp<P, 12>(st, a); break;
    case 16: launch_message_kp<P, 16>(st, a); break;
    case 20: launch_message_kp<P, 20>(st, a); break;
    case 24: launch_message_kp<P, 24>(st, a); break;
    case 32: launch_message_kp<P, 32>(st, a); break;
    case 40: launch_message_kp<P, 40>(st, a); break;
    case 48: launch_message_kp<P, 48>(st, a); break;
    case 64: launch_message_kp<P, 64>(st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipSuccess;
}

template <class P, int F>
hipError_t forward_impl(hipStream_t st, ForwardArgs& fa) {
  using T = typename P::T;
  using A = typename P::A;
  const painn_graph* g = fa.g;
  const PrecModel* pm = fa.pm;
  const Hyper& hp = fa.m->hp;
  const int N = g->N;
  constexpr int RT = (sizeof(T) == 8 && F == 256) ? 1 : 2;
  T* s = (T*)fa.s;
  T* v[2] = {(T*)fa.v[0], (T*)fa.v[1]};
  T* h = (T*)fa.h;
  if (N > 0) {
    prof_mark(fa.prof, st, KC_EMBED, true);
    k_embed<P><<<grid_for((size_t)N * F, 256), 256, 0, st>>>(N, F, g->species, (const T*)pm->emb, s, v[0]);
    prof_mark(fa.prof, st, KC_EMBED, false);
    if (fa.stop_layer >= 0) {
      prof_mark(fa.prof, st, KC_PHI, true);
      k_phi<P, F, RT><<<(N + 16 * RT - 1) / (16 * RT), 256, 0, st>>>(N, s, h, pm->layers[0].phi1,
                                                                   pm->layers[0].phi2);
      prof_mark(fa.prof, st, KC_PHI, false);
    }
  }
  int cur = 0;
  const int KP = filter_kp(hp.K);
  for (int l = 0; l <= fa.stop_layer && N > 0; ++l) {
    const LayerDev& Ld = pm->layers[l];
    MsgArgs ma;
    ma.N = N;
    ma.F = F;
    ma.K = hp.K;
    ma.row_ptr = g->row_ptr;
    ma.col = g->col;
    ma.shift = g->shift;
    ma.atom_struct = g->atom_struct;
    ma.pos = g->pos;
    ma.cell = g->cell;
    ma.rc = hp.cutoff;
    ma.delta = hp.cutoff / (hp.K - 1);
    ma.gamma = 1.0 / (2.0 * ma.delta * ma.delta);
    ma.filt = Ld.filt;
    ma.h = h;
    ma.v_in = v[cur];
    ma.s = s;
    ma.v_out = v[cur ^ 1];
    prof_mark(fa.prof, st, KC_MESSAGE, true);
    hipError_t e = launch_message<P>(st, KP, ma);
    prof_mark(fa.prof, st, KC_MESSAGE, false);
    if (e != hipSuccess) return e;
    cur ^= 1;
    UpdArgs ua;
    ua.N = N;
    ua.s = s;
    ua.v = v[cur];
    ua.h = h;
    ua.uv = Ld.uv;
    ua.upd1 = Ld.upd1;
    ua.upd2 = Ld.upd2;
    const bool fuse = l + 1 <= fa.stop_layer;
    prof_mark(fa.prof, st, KC_UPDATE, true);
    if (fuse) {
      ua.phi1 = pm->layers[l + 1].phi1;
      ua.phi2 = pm->layers[l + 1].phi2;
      k_update<P, F, true><<<(N + 15) / 16, 256, 0, st>>>(ua);
    } else {
      k_update<P, F, false><<<(N + 15) / 16, 256, 0, st>>>(ua);
    }
    prof_mark(fa.prof, st, KC_UPDATE, false);
  }
  if (fa.s_out) {
    prof_mark(fa.prof, st, KC_EXPORT, true);
    if (N > 0)
      k_export<P><<<grid_for((size_t)N * F, 256), 256, 0, st>>>(N, F, s, v[cur], fa.s_out, fa.v_out);
    prof_mark(fa.prof, st, KC_EXPORT, false);
    return hipGetLastError();
  }
  if (g->B == 0) return hipGetLastError();
  if (N > 0) {
    HeadArgs ha;
    ha.N = N;
    ha.F = F;
    ha.n_heads = hp.n_heads;
    ha.ns = (int)pm->shared.size();
    ha.nb = (int)hp.branch_dims.size();
    int ds = 32, db = 32;
    for (size_t m = 0; m < pm->shared.size(); ++m) {
      ha.shared[m] = pm->shared[m];
      ds = ds > pad32(hp.shared_dims[m]) ? ds : pad32(hp.shared_dims[m]);
    }
    int di = pm->shared.empty() ? F : hp.shared_dims.back();
    for (int m = 0; m < ha.nb; ++m) {
      ha.bdin[m] = di;
      ha.bdout[m] = hp.branch_dims[m];
      di = hp.branch_dims[m];
      db = db > pad32(di) ? db : pad32(di);
    }
    ha.lds_s = pm->shared.empty() ? 0 : ds + P::PAD;
    ha.lds_b = db + P::PAD;
    ha.s = s;
    ha.atom_struct = g->atom_struct;
    ha.dataset_id = fa.dataset_id;
    ha.table = (const void* const*)pm->head_table;
    ha.e = fa.e;
    const size_t smem = (size_t)16 * ((F + P::PAD) + 2 * ha.lds_s + 2 * ha.lds_b) * sizeof(T);
    // dynamic LDS beyond 64 KiB must be allowed explicitly (the kernel also
    // holds a few hundred bytes of static LDS; 160 KiB per CU in total)
    static size_t lds_allowed = 64 * 1024;
    if (smem > lds_allowed) {
      if (smem > 150 * 1024) return hipErrorInvalidValue;
      hipError_t e = hipFuncSetAttribute((const void*)k_heads<P, F>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return e;
      }
      lds_allowed = smem;
    }
    prof_mark(fa.prof, st, KC_HEADS, true);
    k_heads<P, F><<<(N + 15) / 16, 256, smem, st>>>(ha);
    prof_mark(fa.prof, st, KC_HEADS, false);
  }
  prof_mark(fa.prof, st, KC_ENERGY, true);
  k_energy<A><<<(g->B + 255) / 256, 256, 0, st>>>(g->B, g->struct_ptr, (const A*)fa.e, fa.energies);
  prof_mark(fa.prof, st, KC_ENERGY, false);
  return hipGetLastError();
}

template <class P>
hipError_t forward_prec(hipStream_t st, ForwardArgs& fa) {
  switch (fa.m->hp.F) {
    case 64: return forward_impl<P, 64>(st, fa);
    case 128: return forward_impl<P, 128>(st, fa);
    case 256: return forward_impl<P, 256>(st, fa);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_forward(hipStream_t st, int prec, ForwardArgs& fa) {
  if (prec == PAINN_FP64) return forward_prec<P64>(st, fa);
  if (prec == PAINN_FP32) return forward_prec<P32>(st, fa);
  return forward_prec<PB16>(st, fa);
}
