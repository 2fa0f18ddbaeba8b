// Reverse pass of the batched PaiNN forward on gfx950 (FP64 / FP32):
// forces F_i = -dE/dx_i.  The paper's screening throughput counts energies
// and forces, and its largest single inference gain is computing the force
// gradient in the same pass as the energy (section "Optimizing the Inference
// Pipeline", Fig. 4); this is that gradient written out by hand.
//
// The forward runs with a save area (each layer's s, v, h before the message
// and s, v after it).  Then, with g_X = dE/dX (accumulation type):
//   heads     g_s = readout'(s_L), g_v = 0
//   layer l = L-1 .. 0:
//     update   (g_s, g_v) -> (g_s', g_v') at s, v after the message
//     message  per SENDER j over its incoming edges (the edge list grouped
//              by sender): g_h_j, g_v_j = g_v'_j + message terms, and per
//              edge dE/dd and dE/drhat (accumulated over layers)
//     phi      g_s = g_s' + phi'(s_l)^T g_h         (skipped at l = 0)
//   edges     dE/dr = dE/dd rhat + (dE/drhat - (dE/drhat . rhat) rhat) / d
//   atoms     F_a = sum_{e: receiver a} dE/dr_e - sum_{e: sender a} dE/dr_e
// (r = x_sender - x_receiver + t).  Every sum runs in a fixed order: the
// forces are deterministic.  The graph is held fixed (the cutoff makes every
// message vanish with zero slope at r_c, and the neighbour cap is piecewise
// constant in the positions).  Where |V v| = 0 the norm's gradient is taken
// as zero.
#include "mfma.h"

namespace {

template <class A>
__device__ __forceinline__ A dsilu(A x) {
  const A sg = A(1) / (A(1) + (sizeof(A) == 8 ? (A)exp((double)-x) : (A)expf((float)-x)));
  return sg * (A(1) + x * (A(1) - sg));
}

template <class A>
__global__ void __launch_bounds__(256) k_fill(size_t n, A* __restrict__ p, A value = A(0)) {
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < n; x += (size_t)gridDim.x * blockDim.x)
    p[x] = value;
}

inline int grid_of(size_t n, int per) {
  size_t g = (n + per - 1) / per;
  if (g > 65536) g = 65536;
  return (int)(g ? g : 1);
}

// ------------------------------------------------ edges grouped by sender ----
__global__ void __launch_bounds__(256) k_t_count(long long E, const int32_t* __restrict__ col,
                                                int32_t* __restrict__ cnt) {
  for (long long e = blockIdx.x * (long long)blockDim.x + threadIdx.x; e < E; e += (long long)gridDim.x * blockDim.x)
    atomicAdd(&cnt[col[e]], 1);
}

// Exclusive scan of the N counts into t_ptr[0..N] over blocks of 1024 counts
// (block sums, a one-workgroup scan of those, then each block's own scan);
// the counts are reset to 0 on the way (they become the fill cursors).
__device__ __forceinline__ int t_block_scan(int x, int* sh) {
  // inclusive scan of x over the 256 threads of the workgroup
  sh[threadIdx.x] = x;
  __syncthreads();
  for (int o = 1; o < 256; o *= 2) {
    const int y = threadIdx.x >= o ? sh[threadIdx.x - o] : 0;
    __syncthreads();
    sh[threadIdx.x] += y;
    __syncthreads();
  }
  return sh[threadIdx.x];
}

__global__ void __launch_bounds__(256) k_t_scan_blocks(int N, const int32_t* __restrict__ cnt,
                                                      long long* __restrict__ bsum) {
  __shared__ int sh[256];
  const int base = blockIdx.x * 1024 + threadIdx.x * 4;
  int x = 0;
  for (int k = 0; k < 4; ++k)
    if (base + k < N) x += cnt[base + k];
  const int incl = t_block_scan(x, sh);
  if (threadIdx.x == 255) bsum[blockIdx.x] = incl;
}

__global__ void __launch_bounds__(256) k_t_scan_top(int nblk, long long* __restrict__ bsum, int32_t* __restrict__ ptr,
                                                   int N) {
  __shared__ int sh[256];
  int carry = 0;
  for (int c0 = 0; c0 < nblk; c0 += 256) {
    const int k = c0 + threadIdx.x;
    const int x = k < nblk ? (int)bsum[k] : 0;
    const int incl = t_block_scan(x, sh);
    if (k < nblk) bsum[k] = carry + incl - x;
    carry += sh[255];
    __syncthreads();
  }
  if (threadIdx.x == 0) ptr[N] = carry;
}

__global__ void __launch_bounds__(256) k_t_scan_apply(int N, int32_t* __restrict__ cnt,
                                                     const long long* __restrict__ bsum, int32_t* __restrict__ ptr) {
  __shared__ int sh[256];
  const int base = blockIdx.x * 1024 + threadIdx.x * 4;
  int v[4], x = 0;
  for (int k = 0; k < 4; ++k) {
    v[k] = base + k < N ? cnt[base + k] : 0;
    x += v[k];
  }
  int run = (int)bsum[blockIdx.x] + t_block_scan(x, sh) - x;
  for (int k = 0; k < 4; ++k)
    if (base + k < N) {
      ptr[base + k] = run;
      cnt[base + k] = 0;
      run += v[k];
    }
}

__global__ void __launch_bounds__(256) k_t_fill(long long E, const int32_t* __restrict__ col,
                                               const int32_t* __restrict__ ptr, int32_t* __restrict__ cur,
                                               int32_t* __restrict__ t_edge) {
  for (long long e = blockIdx.x * (long long)blockDim.x + threadIdx.x; e < E; e += (long long)gridDim.x * blockDim.x) {
    const int j = col[e];
    t_edge[ptr[j] + atomicAdd(&cur[j], 1)] = (int32_t)e;
  }
}

// The fill order depends on timing: each sender's edge ids are put in
// ascending order.  One wave per sender: a segment of up to 64 KPT ids is
// held in registers (KPT per lane) and each id goes to its rank, the number
// of smaller ids in the segment (the ids are distinct), counted by walking
// the segment's ids 64 at a time through shuffles.  A segment longer than
// 1,024 ids (more than 16 per lane) is insertion-sorted by one lane.
template <int KPT>
__device__ __forceinline__ void t_rank_sort(int32_t* __restrict__ seg, int n, int lane) {
  int key[KPT], rank[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    key[q] = lane + 64 * q < n ? seg[lane + 64 * q] : 0x7fffffff;
    rank[q] = 0;
  }
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    const int m_end = min(64, n - 64 * q);   // (wave-uniform; <= 0 past the segment)
    for (int m = 0; m < m_end; ++m) {
      const int other = __shfl(key[q], m);
#pragma unroll
      for (int u = 0; u < KPT; ++u) rank[u] += other < key[u];
    }
  }
#pragma unroll
  for (int q = 0; q < KPT; ++q)
    if (lane + 64 * q < n) seg[rank[q]] = key[q];
}

__global__ void __launch_bounds__(256) k_t_sort(int N, const int32_t* __restrict__ ptr, int32_t* __restrict__ t_edge) {
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (j >= N) return;
  const int a = ptr[j], n = ptr[j + 1] - a;
  if (n <= 1) return;
  if (n <= 256) {
    t_rank_sort<4>(t_edge + a, n, lane);
  } else if (n <= 1024) {
    t_rank_sort<16>(t_edge + a, n, lane);
  } else if (lane == 0) {
    for (int x = a + 1; x < a + n; ++x) {
      const int key = t_edge[x];
      int y = x - 1;
      while (y >= a && t_edge[y] > key) {
        t_edge[y + 1] = t_edge[y];
        --y;
      }
      t_edge[y + 1] = key;
    }
  }
}

// ------------------------------------------- edges in sender order, basis ----
// For the position t of the sender-grouped list (edge e = t_edge[t]): the
// basis row of e, its derivative d/dd, and (rhat, receiver).
// The derivative of the row (f_c g_0, .., f_c g_{K-1}, f_c) is
//   f_c' g_k + f_c g_k',  f_c' = -(pi / (2 r_c)) sin(pi d / r_c);
//   Gaussian g_k' = -2 gamma (d - k Delta) g_k;
//   Bessel   g_n' = (n pi / r_c) cos(n pi d / r_c) / d - sin(n pi d / r_c) / d^2.
// Rows E .. E+15 are zero (read by partial chunks).
// DERIV: the derivative row; otherwise the basis row itself, in the layout
// of the filter with its bias column: f_c g_k for k < K, f_c at K (the same
// expressions as the forward's rows of that layout).
template <class P, bool DERIV>
__device__ __forceinline__ void edge_rev_row(long long e, int K, int kcols, double rc, int rbf, double gamma,
                                             double delta, const int32_t* __restrict__ recv,
                                             const int32_t* __restrict__ col, const int32_t* __restrict__ shift,
                                             const int32_t* __restrict__ atom_struct,
                                             const double* __restrict__ pos, const double* __restrict__ cell,
                                             typename P::T* g) {
  using A = typename P::A;
  const int i = recv[e], j = col[e], sh = shift[e];
  const double* Cl = cell + 9 * atom_struct[i];
  const double n0 = (double)(int8_t)(sh & 0xff), n1 = (double)(int8_t)((sh >> 8) & 0xff),
               n2 = (double)(int8_t)((sh >> 16) & 0xff);
  const double rx = (pos[3 * j] - pos[3 * i]) + ((n0 * Cl[0] + n1 * Cl[3]) + n2 * Cl[6]);
  const double ry = (pos[3 * j + 1] - pos[3 * i + 1]) + ((n0 * Cl[1] + n1 * Cl[4]) + n2 * Cl[7]);
  const double rz = (pos[3 * j + 2] - pos[3 * i + 2]) + ((n0 * Cl[2] + n1 * Cl[5]) + n2 * Cl[8]);
  const double d = sqrt(rx * rx + ry * ry + rz * rz);
  const double pi = 3.14159265358979323846;
  const A dd = (A)d;
  const A fc = (A)(d < rc ? 0.5 * (cos(d * (pi / rc)) + 1.0) : 0.0);
  if constexpr (!DERIV) {
    for (int k = 0; k < kcols; ++k) {
      A val = 0;
      if (k < K && rbf == 0) {
        const A t = dd - (A)(k * delta);
        val = P::ex(-(A)gamma * t * t) * fc;
      } else if (k < K) {
        const A arg = (A)((k + 1) * (pi / rc)) * dd;
        val = (sizeof(A) == 8 ? (A)sin((double)arg) : (A)sinf((float)arg)) / dd * fc;
      } else if (k == K) {
        val = fc;
      }
      g[k] = P::st(val);
    }
    return;
  }
  const A dfc = (A)(d < rc ? -0.5 * (pi / rc) * sin(d * (pi / rc)) : 0.0);
  for (int k = 0; k < kcols; ++k) {
    A val = 0;
    if (k < K && rbf == 0) {
      const A u = dd - (A)(k * delta);
      const A gk = P::ex(-(A)gamma * u * u);
      val = dfc * gk + fc * (-(A)(2.0 * gamma) * u * gk);
    } else if (k < K) {
      const A w = (A)((k + 1) * (pi / rc));
      const A arg = w * dd;
      const A sn = sizeof(A) == 8 ? (A)sin((double)arg) : (A)sinf((float)arg);
      const A cs = sizeof(A) == 8 ? (A)cos((double)arg) : (A)cosf((float)arg);
      val = dfc * (sn / dd) + fc * (w * cs / dd - sn / (dd * dd));
    } else if (k == K) {
      val = dfc;
    }
    g[k] = P::st(val);
  }
}

// A workgroup of EP_REV positions stages its rows in LDS and writes each
// array's contiguous slice with 16-byte stores (per thread, the 48-272 byte
// rows would scatter one element per lane per store).
constexpr int EP_REV = 64;

template <class P>
__global__ void __launch_bounds__(EP_REV) k_edge_rev(long long E, int K, int kcols, double rc, int rbf,
                                                    double gamma, double delta,
                                                    const int32_t* __restrict__ t_edge,
                                                    const int32_t* __restrict__ recv,
                                                    const int32_t* __restrict__ col,
                                                    const int32_t* __restrict__ shift,
                                                    const int32_t* __restrict__ atom_struct,
                                                    const double* __restrict__ pos,
                                                    const double* __restrict__ cell,
                                                    const typename P::A* __restrict__ einfo,
                                                    typename P::T* __restrict__ basis_t,
                                                    typename P::T* __restrict__ dbasis_t,
                                                    typename P::A* __restrict__ einfo_t) {
  using T = typename P::T;
  using A = typename P::A;
  extern __shared__ __attribute__((aligned(16))) unsigned char er_smem[];
  const long long t0 = blockIdx.x * (long long)EP_REV;
  const long long t = t0 + threadIdx.x;
  const long long rows = (E + 16 - t0) < EP_REV ? (E + 16 - t0) : EP_REV;
  const size_t n16 = (size_t)rows * kcols * sizeof(T) / 16;   // kcols * sizeof(T) is a multiple of 16
  T* g = (T*)er_smem + (size_t)threadIdx.x * kcols;
  const int e = t < E ? t_edge[t] : -1;
  // the derivative rows (rows E .. E+15: zero)
  if (e >= 0) edge_rev_row<P, true>(e, K, kcols, rc, rbf, gamma, delta, recv, col, shift, atom_struct, pos, cell, g);
  else if (t < E + 16)
    for (int k = 0; k < kcols; ++k) g[k] = P::st(0);
  __syncthreads();
  {
    const uint4* src = (const uint4*)er_smem;
    uint4* dst = (uint4*)(dbasis_t + (size_t)t0 * kcols);
    for (size_t x = threadIdx.x; x < n16; x += EP_REV) dst[x] = src[x];
  }
  __syncthreads();
  // the basis rows (formed here: the forward's own rows may be in another
  // layout, without the bias column or as the in-kernel Gaussians' records)
  if (e >= 0) edge_rev_row<P, false>(e, K, kcols, rc, rbf, gamma, delta, recv, col, shift, atom_struct, pos, cell, g);
  else if (t < E + 16)
    for (int k = 0; k < kcols; ++k) g[k] = P::st(0);
  __syncthreads();
  {
    const uint4* src = (const uint4*)er_smem;
    uint4* dst = (uint4*)(basis_t + (size_t)t0 * kcols);
    for (size_t x = threadIdx.x; x < n16; x += EP_REV) dst[x] = src[x];
  }
  if (e >= 0) {
    A* o = einfo_t + 4 * t;
    o[0] = einfo[4 * (size_t)e];
    o[1] = einfo[4 * (size_t)e + 1];
    o[2] = einfo[4 * (size_t)e + 2];
    if constexpr (sizeof(A) == 4) o[3] = __int_as_float(recv[e]);
    else o[3] = (A)recv[e];
  }
}

// ------------------------------------------------------------ heads, back ----
// One workgroup per tile of 16 atoms of one head (the forward's grouping):
// the layers' pre-activations are recomputed (kept in the per-atom scratch),
// then dE/ds = W_0^T (silu'(z_0) * W_1^T (... silu'(z_{n-2}) * w_out)).
// Waves per workgroup: 16 for wide head layers (the two activation buffers
// fill most of the LDS, so one workgroup per CU must bring the occupancy),
// 4 for narrow ones.
constexpr int HB_NW_WIDE = 16, HB_NW_NARROW = 4, HB_WIDE = 256;

struct HeadBwdArgs {
  int N, ns, nb, F;
  int ldw;                       // LDS row stride of the two buffers
  const void* s;                 // the final s [N][F]
  const int32_t* order;          // null: consecutive atoms, head 0
  const HeadTile* tiles;         // the forward's tiles (any length)
  const HeadPlan* plan;
  const void* const* table;      // [head][layer][2] = (packed w, bias)
  const void* const* tableT;     // [head][layer][2] = (packed w^T, null)
  DenseDev shared[16], sharedT[16];
  int bdin[16], bdout[16];
  int zoff[32];                  // pre-activation offsets in a scratch row
  void* scratch;
  int sw;
  void* xbuf;                    // GX: per-workgroup [2][16][ldw] buffers in global memory
  void* gs;                      // out: dE/ds [N][F]
  void* gh;                      // blended heads: out dE_h/ds [N][H][F] instead
  int H;
};

template <class Q>
__device__ __forceinline__ typename Q::A packed_w0(const DenseDev& L, int k) {
  using P = dense_t<Q>;
  const int kb = k / P::KC, r = k % P::KC;
  return P::ld(((const typename P::T*)L.w)[((size_t)kb * 64 + 16 * (r / P::KPL)) * P::KPL + r % P::KPL]);
}

// The layers' pre-activations of a 16-row sub-tile go to the workgroup's own
// scratch rows (an atom can sit in several tiles at once: one per kept head).
template <class P, int F, int NW>
__device__ void heads_bwd_tile(const HeadBwdArgs& a, int head, const int* idx, typename P::T* const* Y,
                               int lane) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int TM = 16;
  const int nl = a.ns + a.nb;
  auto layer = [&](int m, bool tr) {
    if (m < a.ns) return tr ? a.sharedT[m] : a.shared[m];
    const int mb = m - a.ns;
    DenseDev L;
    const void* const* tab = tr ? a.tableT : a.table;
    L.w = (void*)tab[((size_t)head * a.nb + mb) * 2];
    L.b = (void*)tab[((size_t)head * a.nb + mb) * 2 + 1];
    const int din = mb == 0 ? (a.ns ? a.shared[a.ns - 1].dout : F) : a.bdout[mb - 1];
    const int dout = a.bdout[mb];
    L.din = tr ? dout : din;
    L.dout = tr ? din : dout;
    L.din_p = pad32(L.din);
    L.dout_p = pad32(L.dout);
    return L;
  };
  // the output row of atom g: dE/ds, or dE_h/ds of this head when blended
  A* gs = (A*)a.gs;
  auto out_row = [&](int g) { return a.gh ? (A*)a.gh + ((size_t)g * a.H + head) * F : gs + (size_t)g * F; };
  const DenseDev Lout = layer(nl - 1, false);
  if (nl == 1) {
    for (int x = threadIdx.x; x < TM * F; x += blockDim.x) {
      const int r = x / F, c = x % F;
      if (idx[r] >= 0) out_row(idx[r])[c] = c < Lout.din ? packed_w0<P>(Lout, c) : A(0);
    }
    return;
  }
  A* scr = (A*)a.scratch;
  const T* s = (const T*)a.s;
  for (int x = threadIdx.x; x < TM * F; x += blockDim.x) {
    const int r = x / F, c = x % F;
    Y[0][r * a.ldw + c] = idx[r] >= 0 ? s[(size_t)idx[r] * F + c] : P::st(0);
  }
  __syncthreads();
  int cur = 0;
  // forward through every layer but the output one, keeping z
  for (int m = 0; m + 1 < nl; ++m) {
    const DenseDev L = layer(m, false);
    T* dst = Y[cur ^ 1];
    dense_tiles<P, 1, NW>(Y[cur], a.ldw, L, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      const A bias = ((const A*)L.b)[col];
      for (int i = 0; i < 4; ++i) {
        const int r = P::row(lane, i);
        const A z = acc[0][i] + bias;
        if (idx[r] >= 0) scr[((size_t)blockIdx.x * TM + r) * a.sw + a.zoff[m] + col] = z;
        dst[r * a.ldw + col] = P::st(col < L.dout ? silu<A>(z) : A(0));
      }
    });
    __syncthreads();
    cur ^= 1;
  }
  // delta of the last hidden layer: w_out * silu'(z)
  {
    const int m = nl - 2;
    const int w = pad32(Lout.din);
    for (int x = threadIdx.x; x < TM * w; x += blockDim.x) {
      const int r = x / w, c = x % w;
      A dl = 0;
      if (idx[r] >= 0 && c < Lout.din) dl = packed_w0<P>(Lout, c) * dsilu<A>(scr[((size_t)blockIdx.x * TM + r) * a.sw + a.zoff[m] + c]);
      Y[cur][r * a.ldw + c] = P::st(dl);
    }
  }
  __syncthreads();
  for (int m = nl - 2; m >= 0; --m) {
    const DenseDev LT = layer(m, true);
    T* dst = Y[cur ^ 1];
    dense_tiles<P, 1, NW>(Y[cur], a.ldw, LT, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      for (int i = 0; i < 4; ++i) {
        const int r = P::row(lane, i);
        const int g = idx[r];
        if (m == 0) {
          if (g >= 0 && col < F) out_row(g)[col] = acc[0][i];
        } else {
          A dl = 0;
          if (g >= 0 && col < LT.dout) dl = acc[0][i] * dsilu<A>(scr[((size_t)blockIdx.x * TM + r) * a.sw + a.zoff[m - 1] + col]);
          dst[r * a.ldw + col] = P::st(dl);
        }
      }
    });
    __syncthreads();
    cur ^= 1;
  }
}

// GX: the two activation buffers live in global memory (a region per
// workgroup) when they do not fit the LDS.
template <class P, int F, bool GX, int NW>
__global__ void __launch_bounds__(64 * NW) k_heads_bwd(HeadBwdArgs a) {
  using T = typename P::T;
  constexpr int TM = 16;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* base = GX ? (T*)a.xbuf + (size_t)blockIdx.x * 2 * TM * a.ldw : (T*)smem;
  T* Y[2] = {base, base + TM * a.ldw};
  __shared__ int idx[TM];
  const int lane = threadIdx.x & 63;
  // a persistent grid: workgroup b takes tiles b, b + gridDim.x, ...
  const int ntiles = a.order ? a.plan->n_tiles : (a.N + TM - 1) / TM;
  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int head = 0, begin, end;
    if (a.order) {
      const HeadTile tl = a.tiles[t];
      head = tl.head;
      begin = tl.begin;
      end = tl.end;
    } else {
      begin = t * TM;
      end = min(a.N, begin + TM);
    }
    for (int sub = begin; sub < end; sub += TM) {
      __syncthreads();
      if (threadIdx.x < TM) {
        const int k = sub + threadIdx.x;
        idx[threadIdx.x] = k < end ? (a.order ? a.order[k] : k) : -1;
      }
      __syncthreads();
      heads_bwd_tile<P, F, NW>(a, head, idx, Y, lane);
    }
  }
}
// Blended heads: dE/ds = sum over kept heads h (w_bh >= skip) of w_bh dE_h/ds,
// in head order.
template <class A>
__global__ void __launch_bounds__(256) k_blend_grad(int N, int H, int F, A skip, const int32_t* __restrict__ atom_struct,
                                                   const A* __restrict__ hw, const A* __restrict__ gh,
                                                   A* __restrict__ gs) {
  const size_t tot = (size_t)N * F;
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < tot; x += (size_t)gridDim.x * blockDim.x) {
    const size_t i = x / F, f = x % F;
    const A* w = hw + (size_t)atom_struct[i] * H;
    A y = 0;
    for (int h = 0; h < H; ++h)
      if (w[h] >= skip) y += w[h] * gh[(i * H + h) * F + f];
    gs[x] = y;
  }
}

// ----------------------------------------------------------- update, back ----
// Tile of 16 atoms, 4 waves; LDS R1 [16][3F + PAD], R2 [16][F + PAD].  The
// forward saved U v[c], V v[c], the gate's pre-activation z and a_vv, a_sv,
// so only the transposed products run here:
//   g_a  = [sum_c g_v[c] U[c] | g_s <U, V> | g_s]
//   g_z  = (W2a^T g_a) * silu'(z)
//   [g_s' ; g_n] = W1a^T g_z                 g_s after the message = g_s + g_s'
//   g_U[c] = g_v[c] a_vv + g_s a_sv V[c],  g_V[c] = g_s a_sv U[c] + g_n V[c] / |V|
//   g_v after the message [c] = g_v[c] + [U^T | V^T] [g_U[c] ; g_V[c]]
// The per-atom scratch holds g_n.
// Waves per workgroup of the reverse update and phi kernels: 4, or more
// where the LDS tile leaves room for only one workgroup per CU (measured:
// 16 for FP32; 8 for FP64, whose 3F-wide operands then sit in global memory).
template <class P, int F>
constexpr int ub_nw() {
  return (size_t)16 * (4 * F + 2 * P::PAD) * sizeof(typename P::T) > 64 * 1024
             ? (sizeof(typename P::T) == 8 ? 8 : 16)
             : 4;
}

struct UpdBwdArgs {
  int N;
  const void* uv;    // saved [N][3][2F]: U v[c], V v[c]
  const void* z;     // saved [N][F]
  const void* ag;    // saved [N][2F]: a_vv, a_sv
  const void* gs;    // dE/d(s, v) after the update
  const void* gv;
  void* gs_out;      // dE/d(s, v) after the message
  void* gv_out;
  void* scratch;
  int sw;
  void* xbuf;        // GX: per-workgroup [16][3F + PAD] buffers in global memory
  DenseDev uvT, upd1T, upd2T;
};

// GX: the 3F-wide operand buffer R1 lives in global memory (a region per
// workgroup; the MFMA operand reads go through the caches) when 16 rows of
// 4F do not fit the LDS (FP64 at F = 384).
template <class P, int F, bool GX>
__global__ void __launch_bounds__((64 * ub_nw<P, F>())) k_update_bwd(UpdBwdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int TM = 16, LD1 = 3 * F + P::PAD, LD2 = F + P::PAD;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* R1 = GX ? (T*)a.xbuf + (size_t)blockIdx.x * TM * LD1 : (T*)smem;
  T* R2 = GX ? (T*)smem : R1 + TM * LD1;
  const int lane = threadIdx.x & 63;
  const size_t row0 = (size_t)blockIdx.x * TM;
  const int N = a.N;
  const T* uv = (const T*)a.uv;
  const T* zs = (const T*)a.z;
  const T* ag = (const T*)a.ag;
  const A* gs = (const A*)a.gs;
  const A* gv = (const A*)a.gv;
  A* scr = (A*)a.scratch;
  const int sw = a.sw;
  auto U = [&](size_t i, int c, int f) { return P::ld(uv[(i * 3 + c) * 2 * F + f]); };
  auto V = [&](size_t i, int c, int f) { return P::ld(uv[(i * 3 + c) * 2 * F + F + f]); };
  constexpr int NT = 64 * ub_nw<P, F>(), EPT = (TM * F + NT - 1) / NT;
  constexpr bool PRE = EPT * (int)sizeof(A) <= (NT < 1024 ? 32 : 24);   // 1024 threads leave 128 VGPRs
  // V4: every thread on whole groups of 4 consecutive features: the
  // element-wise passes load 16-byte (FP32) or 32-byte (FP64) vectors, and
  // store them to LDS as such where its rows keep that alignment (FP32)
  constexpr bool V4 = std::is_same<T, A>::value && PRE && (TM * F / 4) % NT == 0;
  constexpr int EPQ = V4 ? TM * F / 4 / NT : 1;
  using Q = Quad<A>;
  auto ldq = [](const void* p) { return *(const Q*)p; };
  auto stq = [](T* d, const Q& q) {
    if constexpr (LD1 % 4 == 0) {
      *(Q*)d = q;
    } else {
      for (int k = 0; k < 4; ++k) d[k] = q.x[k];
    }
  };
  // g_a into R1
  if constexpr (V4) {
#pragma unroll
    for (int e = 0; e < EPQ; ++e) {
      const int x = threadIdx.x + e * NT, r = x / (F / 4), f = (x % (F / 4)) * 4;
      Q gvv, gsv, gss;
      for (int k = 0; k < 4; ++k) gvv.x[k] = gsv.x[k] = gss.x[k] = 0;
      if (row0 + r < (size_t)N) {
        const size_t i = row0 + r;
        A pd[4] = {0, 0, 0, 0};
        for (int c = 0; c < 3; ++c) {
          const Q u = ldq(uv + (i * 3 + c) * 2 * F + f), w = ldq(uv + (i * 3 + c) * 2 * F + F + f);
          const Q g = ldq(gv + i * 3 * F + c * F + f);
          for (int k = 0; k < 4; ++k) {
            pd[k] += u.x[k] * w.x[k];
            gvv.x[k] += g.x[k] * u.x[k];
          }
        }
        gss = ldq(gs + i * F + f);
        for (int k = 0; k < 4; ++k) gsv.x[k] = gss.x[k] * pd[k];
      }
      stq(&R1[r * LD1 + f], gvv);
      stq(&R1[r * LD1 + F + f], gsv);
      stq(&R1[r * LD1 + 2 * F + f], gss);
    }
  } else
  for (int x = threadIdx.x; x < TM * F; x += blockDim.x) {
    const int r = x / F, f = x % F;
    A gvv = 0, gsv = 0, gss = 0;
    if (row0 + r < (size_t)N) {
      const size_t i = row0 + r;
      A pd = 0;
      for (int c = 0; c < 3; ++c) {
        const A u = U(i, c, f);
        pd += u * V(i, c, f);
        gvv += gv[i * 3 * F + c * F + f] * u;
      }
      gss = gs[i * F + f];
      gsv = gss * pd;
    }
    R1[r * LD1 + f] = P::st(gvv);
    R1[r * LD1 + F + f] = P::st(gsv);
    R1[r * LD1 + 2 * F + f] = P::st(gss);
  }
  __syncthreads();
  // g_z = (W2a^T g_a) * silu'(z) into R2
  dense_tiles<P, 1, ub_nw<P, F>(), 3 * F>(R1, LD1, a.upd2T, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15);
    for (int i = 0; i < 4; ++i) {
      const int r = P::row(lane, i);
      A g = 0;
      if (row0 + r < (size_t)N) g = acc[0][i] * dsilu<A>(P::ld(zs[(row0 + r) * F + col]));
      R2[r * LD2 + col] = P::st(g);
    }
  });
  __syncthreads();
  // [g_s' ; g_n] = W1a^T g_z
  A* gs_out = (A*)a.gs_out;
  dense_tiles<P, 1, ub_nw<P, F>(), F>(R2, LD2, a.upd1T, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15);
    for (int i = 0; i < 4; ++i) {
      const int r = P::row(lane, i);
      const size_t g = row0 + r;
      if (g >= (size_t)N) continue;
      if (col < F) gs_out[g * F + col] = gs[g * F + col] + acc[0][i];
      else scr[g * sw + col - F] = acc[0][i];
    }
  });
  __syncthreads();
  // per component: [g_U | g_V] into R1, then [U^T | V^T] [g_U ; g_V]
  A* gv_out = (A*)a.gv_out;
  // the component-independent factors of a thread's elements (the same
  // elements in every component pass) are formed once, in registers, where
  // they fit: g_s a_sv, a_vv, |V| and dE/d|V|
  A gsa_r[PRE ? EPT : 1], avv_r[PRE ? EPT : 1], nv_r[PRE ? EPT : 1], sc_r[PRE ? EPT : 1];
  if constexpr (V4) {
    // element 4e + k of the thread: feature f + k of quad e
#pragma unroll
    for (int e = 0; e < EPQ; ++e) {
      const int x = threadIdx.x + e * NT, r = x / (F / 4), f = (x % (F / 4)) * 4;
      for (int k = 0; k < 4; ++k) gsa_r[4 * e + k] = avv_r[4 * e + k] = nv_r[4 * e + k] = sc_r[4 * e + k] = 0;
      if (row0 + r < (size_t)N) {
        const size_t i = row0 + r;
        const Q v0 = ldq(uv + (i * 3 + 0) * 2 * F + F + f), v1 = ldq(uv + (i * 3 + 1) * 2 * F + F + f),
                v2 = ldq(uv + (i * 3 + 2) * 2 * F + F + f);
        const Q g = ldq(gs + i * F + f), avv = ldq(ag + i * 2 * F + f), asv = ldq(ag + i * 2 * F + F + f);
        for (int k = 0; k < 4; ++k) {
          nv_r[4 * e + k] = sqrt(v0.x[k] * v0.x[k] + v1.x[k] * v1.x[k] + v2.x[k] * v2.x[k]);
          gsa_r[4 * e + k] = g.x[k] * asv.x[k];
          avv_r[4 * e + k] = avv.x[k];
          sc_r[4 * e + k] = scr[i * sw + f + k];
        }
      }
    }
  } else if constexpr (PRE) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int x = threadIdx.x + e * NT, r = x / F, f = x % F;
      gsa_r[e] = avv_r[e] = nv_r[e] = sc_r[e] = 0;
      if (x < TM * F && row0 + r < (size_t)N) {
        const size_t i = row0 + r;
        const A v0 = V(i, 0, f), v1 = V(i, 1, f), v2 = V(i, 2, f);
        nv_r[e] = sqrt(v0 * v0 + v1 * v1 + v2 * v2);
        gsa_r[e] = gs[i * F + f] * P::ld(ag[i * 2 * F + F + f]);
        avv_r[e] = P::ld(ag[i * 2 * F + f]);
        sc_r[e] = scr[i * sw + f];
      }
    }
  }
  for (int c = 0; c < 3; ++c) {
    if constexpr (V4) {
#pragma unroll
      for (int e = 0; e < EPQ; ++e) {
        const int x = threadIdx.x + e * NT, r = x / (F / 4), f = (x % (F / 4)) * 4;
        Q gU, gV;
        for (int k = 0; k < 4; ++k) gU.x[k] = gV.x[k] = 0;
        if (row0 + r < (size_t)N) {
          const size_t i = row0 + r;
          const Q u = ldq(uv + (i * 3 + c) * 2 * F + f), w = ldq(uv + (i * 3 + c) * 2 * F + F + f);
          const Q gvc = ldq(gv + i * 3 * F + c * F + f);
          for (int k = 0; k < 4; ++k) {
            const int q = 4 * e + k;
            gU.x[k] = gvc.x[k] * avv_r[q] + gsa_r[q] * w.x[k];
            gV.x[k] = gsa_r[q] * u.x[k] + (nv_r[q] > A(0) ? sc_r[q] * w.x[k] / nv_r[q] : A(0));
          }
        }
        stq(&R1[r * LD1 + f], gU);
        stq(&R1[r * LD1 + F + f], gV);
      }
    } else if constexpr (PRE) {
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int x = threadIdx.x + e * NT, r = x / F, f = x % F;
        if (x >= TM * F) break;
        A gU = 0, gV = 0;
        if (row0 + r < (size_t)N) {
          const size_t i = row0 + r;
          const A u = U(i, c, f), w = V(i, c, f);
          const A gvc = gv[i * 3 * F + c * F + f];
          gU = gvc * avv_r[e] + gsa_r[e] * w;
          gV = gsa_r[e] * u + (nv_r[e] > A(0) ? sc_r[e] * w / nv_r[e] : A(0));
        }
        R1[r * LD1 + f] = P::st(gU);
        R1[r * LD1 + F + f] = P::st(gV);
      }
    } else {
      for (int x = threadIdx.x; x < TM * F; x += blockDim.x) {
        const int r = x / F, f = x % F;
        A gU = 0, gV = 0;
        if (row0 + r < (size_t)N) {
          const size_t i = row0 + r;
          const A u = U(i, c, f), w = V(i, c, f);
          const A v0 = V(i, 0, f), v1 = V(i, 1, f), v2 = V(i, 2, f);
          const A nv = sqrt(v0 * v0 + v1 * v1 + v2 * v2);
          const A g_s = gs[i * F + f], gvc = gv[i * 3 * F + c * F + f];
          const A avv = P::ld(ag[i * 2 * F + f]), asv = P::ld(ag[i * 2 * F + F + f]);
          gU = gvc * avv + g_s * asv * w;
          gV = g_s * asv * u + (nv > A(0) ? scr[i * sw + f] * w / nv : A(0));
        }
        R1[r * LD1 + f] = P::st(gU);
        R1[r * LD1 + F + f] = P::st(gV);
      }
    }
    __syncthreads();
    dense_tiles<P, 1, ub_nw<P, F>(), 2 * F>(R1, LD1, a.uvT, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      for (int i = 0; i < 4; ++i) {
        const int r = P::row(lane, i);
        const size_t g = row0 + r;
        if (g < (size_t)N) {
          const size_t o = g * 3 * F + c * F + col;
          gv_out[o] = gv[o] + acc[0][i];
        }
      }
    });
    __syncthreads();
  }
}

// -------------------------------------------------------------- phi, back ----
// g_s = g_s' + W1^T ((W2^T g_h) * silu'(W1 s + b1)); tile of 16 atoms.
struct PhiBwdArgs {
  int N;
  const void* s;       // s before the message [N][F]
  const void* gh;      // [N][3F]
  const void* gs_mid;  // [N][F]
  void* gs_out;
  void* scratch;       // per-atom rows of sw elements (FP64 at F = 384 only)
  int sw;
  void* xbuf;          // GX: as for the update
  DenseDev phi1, phi1T, phi2T;
};

template <class P, int F, bool GX>
__global__ void __launch_bounds__((64 * ub_nw<P, F>())) k_phi_bwd(PhiBwdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int TM = 16, LD1 = 3 * F + P::PAD, LD2 = F + P::PAD;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* R1 = GX ? (T*)a.xbuf + (size_t)blockIdx.x * TM * LD1 : (T*)smem;
  T* R2 = GX ? (T*)smem : R1 + TM * LD1;
  const int lane = threadIdx.x & 63;
  const size_t row0 = (size_t)blockIdx.x * TM;
  const int N = a.N;
  stage_rows<P, F, TM>(R2, LD2, (const T*)a.s, F, row0, N);
  stage_rows<P, 3 * F, TM>(R1, LD1, (const A*)a.gh, 3 * F, row0, N);
  __syncthreads();
  // silu'(W1 s + b1) stays in the registers of the lane that formed it (both
  // F-wide layers hand feature tile ct to wave ct % NW, call ct / NW of it)
  // where a wave has at most two tiles; otherwise (FP64 at F = 384) it goes
  // through the per-atom scratch rows.
  constexpr int NW = ub_nw<P, F>(), TPW = (F / 16 + NW - 1) / NW;
  constexpr bool REG = TPW <= 2;
  A* scr = (A*)a.scratch;
  A ds[REG ? TPW : 1][4];
  dense_tiles<P, 1, NW, F>(R2, LD2, a.phi1, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15), k = ct / NW;
    const A bias = ((const A*)a.phi1.b)[col];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const A d = dsilu<A>(acc[0][i] + bias);
      if constexpr (REG) {
#pragma unroll
        for (int j = 0; j < TPW; ++j) ds[j][i] = j == k ? d : ds[j][i];
      } else {
        const int r = P::row(lane, i);
        if (row0 + r < (size_t)N) scr[(row0 + r) * a.sw + col] = d;
      }
    }
  });
  __syncthreads();
  dense_tiles<P, 1, NW, 3 * F>(R1, LD1, a.phi2T, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15), k = ct / NW;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = P::row(lane, i);
      A g = 0;
      if constexpr (REG) {
        A d = ds[0][i];
#pragma unroll
        for (int j = 1; j < TPW; ++j) d = j == k ? ds[j][i] : d;
        g = acc[0][i] * d;
      } else {
        if (row0 + r < (size_t)N) g = acc[0][i] * scr[(row0 + r) * a.sw + col];
      }
      R2[r * LD2 + col] = P::st(row0 + r < (size_t)N ? g : A(0));
    }
  });
  __syncthreads();
  const A* gm = (const A*)a.gs_mid;
  A* go = (A*)a.gs_out;
  dense_tiles<P, 1, ub_nw<P, F>(), F>(R2, LD2, a.phi1T, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15);
    for (int i = 0; i < 4; ++i) {
      const size_t g = row0 + P::row(lane, i);
      if (g < (size_t)N) go[g * F + col] = gm[g * F + col] + acc[0][i];
    }
  });
}

// ---------------------------------------------------------- message, back ----
// Per sender j and channel c, over the edges e = (i <- j) whose sender is j
// (the edge list grouped by sender), with the receiver's g_s' and g_v'
// gathered:
//   A_v = sum_c g_v'_i[c] v_j[c],  A_r = sum_c g_v'_i[c] rhat_e[c]
//   g_h^s_j += g_s'_i w^s,  g_h^v_j += A_v w^v,  g_h^r_j += A_r w^r
//   g_v_j[c] = g_v'_j[c] + sum_e g_v'_i[c] h^v_j w^v
//   dE/dd_e    += sum_ch (g_s'_i h^s_j w'^s + A_v h^v_j w'^v + A_r h^r_j w'^r)
//   dE/drhat_e += sum_ch g_v'_i[.] h^r_j w^r
// with w = f_c (Wf g + bf) and w' = dw/dd.  For 16 edges at a time the
// matrix cores form w and w' (the basis rows and their derivatives against
// the same filter fragments); every lane then works in the accumulator
// layout itself, 4 edges x one channel per feature tile, so the filter never
// leaves the registers.  The per-edge sums over channels go through a
// per-wave LDS transpose (the 16 lanes that share those edges); each wave
// writes its own slot of every edge.
constexpr int MB_RB = 4;   // senders per workgroup (2 and 8 measured the same)

struct MsgBwdArgs {
  int N;
  long long E;
  const int32_t* t_ptr;
  const int32_t* t_edge;
  // in sender order (position t of the sender-grouped list; E + 16 rows)
  const void* basis;
  const void* dbasis;
  const void* einfo;   // rhat, receiver index
  DenseDev filt;
  const void* h;       // layer input h, v (storage type)
  const void* v;
  const void* gs;      // dE/d(s, v) after the message (accumulation type)
  const void* gv;
  void* gh;            // out
  void* gv_out;
  void* eg;            // [E][NW][4]
  int first;           // the first layer: only eg is wanted (g_h, g_v are not written)
  int bg;              // g_s', g_v' gathered by buffer loads (g_v' below 2 GiB)
};

__device__ __forceinline__ int acc_index(float x) { return __float_as_int(x); }
__device__ __forceinline__ int acc_index(double x) { return (int)x; }

// Raw buffer resource over [p, p + bytes) (bytes < 4 GiB): loads at offsets
// past the end read as zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)(uint32_t)bytes, 0x00020000);
}
template <class V>
__device__ __forceinline__ V buf_ld8(__amdgpu_buffer_rsrc_t r, uint32_t off, int soff) {
  return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(r, off, soff, 0));
}
typedef double bwd_d2 __attribute__((ext_vector_type(2)));

// Feature tiles per wave and the waves per SIMD the kernel (FP64) is
// compiled for: one tile, two waves.
template <class P, int F, int KBM>
constexpr int mb_ftw() { return 1; }
template <class P, int F, int KBM>
constexpr int mb_wpe() { return 2; }
// Waves of one feature slice (a workgroup); wide layers take several slices
// in consecutive workgroups.
template <class P, int F, int KBM>
constexpr int mb_nwb() {
  constexpr int nw = F / 16 / mb_ftw<P, F, KBM>();
  return nw <= 8 ? nw : (nw % 8 == 0 ? 8 : 6);
}

// L0: the first layer, where v = 0 and only the per-edge sums are wanted
// (as in the channel-per-lane form below): w^r, w'^s and w'^r only, no g_h,
// g_v.
template <class P, int F, int KBM, bool L0>
__global__ void __launch_bounds__((64 * mb_nwb<P, F, KBM>())) __attribute__((amdgpu_waves_per_eu(mb_wpe<P, F, KBM>())))
k_message_bwd(MsgBwdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  using Fr = typename P::Fr;
  constexpr int FTW = mb_ftw<P, F, KBM>(), NFT = F / 16, NW = NFT / FTW;
  constexpr int NWB = mb_nwb<P, F, KBM>(), SLICES = NW / NWB;
  static_assert(NW % NWB == 0, "feature slices");
  constexpr int kcols = KBM * P::KC;
  const int per_xcd = gridDim.x / 8;
  const int lb = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int lane = threadIdx.x & 63;
  // With one feature tile per wave the register budget is tight (4 waves
  // per SIMD); a wave index the compiler knows to be uniform moves address
  // arithmetic to scalar registers.  With two tiles it has room, and the
  // uniform form measured slower there.
  const int wave_v = (lb % SLICES) * NWB + (threadIdx.x >> 6);
  const int wave = FTW == 1 ? __builtin_amdgcn_readfirstlane(wave_v) : wave_v;
  const T* Wf = (const T*)a.filt.w;
  const T* h = (const T*)a.h;
  const T* vv = (const T*)a.v;
  const A* gs = (const A*)a.gs;
  const A* gv = (const A*)a.gv;
  const A* einfo = (const A*)a.einfo;
  const T* basis = (const T*)a.basis;
  const T* dbasis = (const T*)a.dbasis;
  static_assert(sizeof(A) == 8, "the MFMA form runs FP64");
  using A2 = bwd_d2;
  // At 6 to 9 k-blocks each wave keeps its filter fragments in its own LDS
  // region for the whole kernel (one load each at the start instead of one
  // per chunk from L2; 13.5 KiB per wave at 9; bulk reverse message -8.5 %,
  // molecules -4.7 %).  With 3 they fit in registers (an LDS copy measured
  // 3.5 % slower), past 9 not in the LDS.
  constexpr bool WIMG = KBM >= 6 && KBM <= 9;
  // per wave 16 rows of 64 values for the per-edge sums, or 8 taken in two
  // passes beside the filter copy (+2: the rows' 16-byte groups start on
  // different banks)
  constexpr int RED_LD = 64 + 2, RROWS = WIMG ? 8 : 16;
  __shared__ __attribute__((aligned(16))) A red[NWB * RROWS * RED_LD];
  constexpr int WIMG_N = WIMG ? FTW * 3 * KBM * 64 : 2;
  __shared__ __attribute__((aligned(16))) A wimg[NWB * WIMG_N];
  const __amdgpu_buffer_rsrc_t r_gs = buf_rsrc(gs, a.bg ? (size_t)a.N * F * sizeof(A) : 0);
  const __amdgpu_buffer_rsrc_t r_gv = buf_rsrc(gv, a.bg ? (size_t)a.N * 3 * F * sizeof(A) : 0);
  // the filter's MFMA B fragments: [3 parts x F / 16 tiles][KBM][64 lanes]
  static_assert(P::KPL == 1, "one filter value per lane and k-block");
  const __amdgpu_buffer_rsrc_t r_w = buf_rsrc(Wf, (size_t)3 * NFT * KBM * 64 * sizeof(T));
  const uint32_t lane_w = (uint32_t)lane * sizeof(T);
  A* wi = wimg + (threadIdx.x >> 6) * WIMG_N;
  if constexpr (WIMG) {
#pragma unroll
    for (int q = 0; q < FTW; ++q)
#pragma unroll
      for (int part = 0; part < 3; ++part)
#pragma unroll
        for (int kb = 0; kb < KBM; ++kb) {
          const int ct = part * NFT + FTW * wave + q;
          wi[((q * 3 + part) * KBM + kb) * 64 + lane] =
              buf_ld8<A>(r_w, lane_w, (ct * KBM + kb) * 64 * (int)sizeof(T));
        }
    __builtin_amdgcn_wave_barrier();
  }
  const int j0 = lb / SLICES * MB_RB;
  if (j0 >= a.N) return;
  const int j1 = min(a.N, j0 + MB_RB);
  const int tp_lane = a.t_ptr[j0 + min(lane, j1 - j0)];
  auto tp = [&](int j) { return __builtin_amdgcn_readlane(tp_lane, j - j0); };
  A* gh_out = (A*)a.gh;
  A* gv_out = (A*)a.gv_out;
  A* eg = (A*)a.eg;
  // senders without incoming edges: g_h = 0, g_v = g_v'
  for (int j = j0; j < j1 && !L0; ++j)
    if (tp(j) == tp(j + 1) && lane < 16) {
      const size_t jb = (size_t)j * 3 * F;
#pragma unroll
      for (int q = 0; q < FTW; ++q) {
        const int ch = (FTW * wave + q) * 16 + lane;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          gh_out[jb + k * F + ch] = A(0);
          gv_out[jb + k * F + ch] = gv[jb + k * F + ch];
        }
      }
    }
  auto first_with_edges = [&](int j) {
    while (j < j1 && tp(j) == tp(j + 1)) ++j;
    return j;
  };
  // The block's senders are walked as one stream of chunks of up to 16
  // edges of one sender; each chunk loads its operand rows and edge info at
  // its start.  Per lane: the A rows (position c0 + lane % 16; past the
  // chunk the zero row E) and, for its 4 accumulator rows, edge id,
  // receiver and rhat (past the chunk: receiver 0 and a zero filter, so
  // they add nothing).
  Fr Gan[KBM], Gdn[KBM];
  int ern[4], irn[4];
  A rhn[4][3];
  auto prefetch = [&](int c0, int cnt) {
    const int erA = (lane & 15) < cnt ? c0 + (lane & 15) : (int)a.E;
    const T* gp = basis + (size_t)erA * kcols + (lane >> 4) * P::KPL;
    const T* dp = dbasis + (size_t)erA * kcols + (lane >> 4) * P::KPL;
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) {
      Gan[kb] = P::frag(gp + kb * P::KC);
      Gdn[kb] = P::frag(dp + kb * P::KC);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = P::row(lane, i);
      const bool ok = row < cnt;
      const A* ei = einfo + 4 * (size_t)(ok ? c0 + row : 0);
      ern[i] = ok ? a.t_edge[c0 + row] : -1;
      irn[i] = ok ? acc_index(ei[3]) : 0;
      rhn[i][0] = ok ? ei[0] : A(0);
      rhn[i][1] = ok ? ei[1] : A(0);
      rhn[i][2] = ok ? ei[2] : A(0);
    }
  };
  int j = first_with_edges(j0);
  if (j >= j1) return;
  int c0 = tp(j);
  A acc_h[FTW][3], acc_v[FTW][3];
#pragma unroll
  for (int q = 0; q < FTW; ++q)
#pragma unroll
    for (int k = 0; k < 3; ++k) acc_h[q][k] = acc_v[q][k] = 0;
  while (true) {
    const size_t jb = (size_t)j * 3 * F;
    const int eb = tp(j + 1);
    prefetch(c0, min(16, eb - c0));
    Fr Ga[KBM], Gd[KBM];
    int er[4], ir[4];
    A rh[4][3];
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) {
      Ga[kb] = Gan[kb];
      Gd[kb] = Gdn[kb];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      er[i] = ern[i];
      ir[i] = irn[i];
      rh[i][0] = rhn[i][0];
      rh[i][1] = rhn[i][1];
      rh[i][2] = rhn[i][2];
    }
    // the next chunk: this sender's next 16 edges, else the next sender
    // (found after this chunk, so that its indices are not live across the
    // matrix work)
    const bool last = c0 + 16 >= eb;
    int jn = j, cn = 0;
    bool more = true;
    auto find_next = [&] {
      jn = last ? first_with_edges(j + 1) : j;
      more = jn < j1;
      cn = last ? (more ? tp(jn) : 0) : c0 + 16;
    };
    // the receivers' g_s', g_v' at this lane's channels, all issued before
    // the matrix cores start (they do not depend on the filter)
    // Rows past the chunk must add exactly nothing (not 0 x receiver 0's
    // gradient, which may be NaN): their gathers read zeros.  With buffer
    // loads such a row's offset lies past the buffer, which reads as zero
    // (32-bit offsets, no per-value select); otherwise the values are
    // selected away.
    A gsr[FTW][4], gvr[FTW][4][3];
    if (a.bg) {
#pragma unroll
      for (int q = 0; q < FTW; ++q) {
        const uint32_t ch8 = (uint32_t)((FTW * wave + q) * 16 + (lane & 15)) * sizeof(A);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool live = er[i] >= 0;
          const uint32_t os = live ? (uint32_t)ir[i] * (F * sizeof(A)) + ch8 : 0x80000000u;
          const uint32_t ov = live ? (uint32_t)ir[i] * (3 * F * sizeof(A)) + ch8 : 0x80000000u;
          gsr[q][i] = buf_ld8<A>(r_gs, os, 0);
#pragma unroll
          for (int k = 0; k < 3; ++k) gvr[q][i][k] = buf_ld8<A>(r_gv, ov, k * F * (int)sizeof(A));
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < FTW; ++q) {
        const int ch = (FTW * wave + q) * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const size_t ib = (size_t)ir[i] * 3 * F;
          const bool live = er[i] >= 0;
          const A s0 = gs[(size_t)ir[i] * F + ch];
          const A v0 = gv[ib + ch], v1 = gv[ib + F + ch], v2 = gv[ib + 2 * F + ch];
          gsr[q][i] = live ? s0 : A(0);
          gvr[q][i][0] = live ? v0 : A(0);
          gvr[q][i][1] = live ? v1 : A(0);
          gvr[q][i][2] = live ? v2 : A(0);
        }
      }
    }
    // The filter fragments are buffer loads: the lane's 8 bytes plus the
    // fragment's offset, a scalar (no per-load address arithmetic).  When
    // they are many they stream from the caches chunk by chunk (an opaque
    // copy of the base offset keeps the compiler from hoisting them out of
    // the loops).
    // (With the LDS copy the opaque offset keeps its reads in the loop.)
    int wofs = 0;
    if constexpr (WIMG || FTW * 3 * KBM * (int)sizeof(A) / 4 > 40) asm volatile("" : "+s"(wofs));
    // per-edge partial sums: [dE/dd, dE/drhat x, y, z] x 4 rows
    A vals[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) vals[k] = 0;
#pragma unroll
    for (int q = 0; q < FTW; ++q) {
      C w[3], wd[3];
#pragma unroll
      for (int part = 0; part < 3; ++part) {
        for (int r = 0; r < 4; ++r) w[part][r] = wd[part][r] = 0;
        if (L0 && part == 1) continue;
#pragma unroll
        for (int kb = 0; kb < KBM; ++kb) {
          const int ct = part * NFT + FTW * wave + q;
          Fr bw;
          if constexpr (WIMG) bw = wi[wofs + ((q * 3 + part) * KBM + kb) * 64 + lane];
          else bw = buf_ld8<Fr>(r_w, lane_w, wofs + (ct * KBM + kb) * 64 * (int)sizeof(T));
          if (!L0 || part == 2) w[part] = P::mfma(Ga[kb], bw, w[part]);
          wd[part] = P::mfma(Gd[kb], bw, wd[part]);
        }
      }
      const int ch = (FTW * wave + q) * 16 + (lane & 15);
      const A hs = P::ld(h[jb + ch]), hr = P::ld(h[jb + 2 * F + ch]);
      const A hv = L0 ? A(0) : P::ld(h[jb + F + ch]);
      const A v0 = L0 ? A(0) : P::ld(vv[jb + ch]), v1 = L0 ? A(0) : P::ld(vv[jb + F + ch]);
      const A v2 = L0 ? A(0) : P::ld(vv[jb + 2 * F + ch]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const A g_s = gsr[q][i], g0 = gvr[q][i][0], g1 = gvr[q][i][1], g2 = gvr[q][i][2];
        const A Ar = g0 * rh[i][0] + g1 * rh[i][1] + g2 * rh[i][2];
        const A tr = hr * w[2][i];
        if constexpr (L0) {
          vals[i] += g_s * hs * wd[0][i] + Ar * hr * wd[2][i];
        } else {
          const A Av = g0 * v0 + g1 * v1 + g2 * v2;
          acc_h[q][0] += g_s * w[0][i];
          acc_h[q][1] += Av * w[1][i];
          acc_h[q][2] += Ar * w[2][i];
          const A tv = hv * w[1][i];
          acc_v[q][0] += g0 * tv;
          acc_v[q][1] += g1 * tv;
          acc_v[q][2] += g2 * tv;
          vals[i] += g_s * hs * wd[0][i] + Av * hv * wd[1][i] + Ar * hr * wd[2][i];
        }
        vals[4 + i] += g0 * tr;
        vals[8 + i] += g1 * tr;
        vals[12 + i] += g2 * tr;
      }
    }
    // lane: the wave's total of value (lane % 16) / 4 for its row lane % 4,
    // over the 16 lanes of its row group, through the wave's LDS rows (one
    // write and read per value instead of a butterfly of selects and lane
    // shuffles).  16 rows: value k of every lane in row k, each lane sums 16
    // consecutive entries of its row.  8 rows: two passes, value 8 p + k in
    // row k; lane l sums entries 16 (l / 16) + 8 h .. + 7 (h = bit 3 of l)
    // of row l % 8 and one shuffle adds the other half, so value lane % 16
    // is pass h's row lane % 8.
    {
      A* rw = red + (threadIdx.x >> 6) * (RROWS * RED_LD);
      A sum = 0;
      if constexpr (RROWS == 16) {
#pragma unroll
        for (int k = 0; k < 16; ++k) rw[k * RED_LD + lane] = vals[k];
        __builtin_amdgcn_wave_barrier();
        const A* rr = rw + (lane & 15) * RED_LD + (lane >> 4) * 16;
        A2 t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = *(const A2*)(rr + 2 * u);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int u = 0; u < 8; ++u) sum += t[u][0] + t[u][1];
      } else {
        const A* rr = rw + (lane & 7) * RED_LD + (lane >> 4) * 16 + ((lane >> 3) & 1) * 8;
        A tot[2];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
          for (int k = 0; k < 8; ++k) rw[k * RED_LD + lane] = vals[8 * p + k];
          __builtin_amdgcn_wave_barrier();
          A2 t[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) t[u] = *(const A2*)(rr + 2 * u);
          __builtin_amdgcn_wave_barrier();
          A sp = ((t[0][0] + t[0][1]) + (t[1][0] + t[1][1])) + ((t[2][0] + t[2][1]) + (t[3][0] + t[3][1]));
          sp += __shfl_xor(sp, 8);
          tot[p] = sp;
        }
        sum = (lane & 8) ? tot[1] : tot[0];
      }
      const int k = lane & 15, i = k & 3;
      const int e = i == 0 ? er[0] : i == 1 ? er[1] : i == 2 ? er[2] : er[3];
      // one add per slot per launch, and launches run in layer order: the
      // sums are deterministic; the add does not return, so no wave waits
      if (e >= 0) unsafeAtomicAdd(eg + ((size_t)e * NW + wave) * 4 + (k >> 2), sum);
    }
    find_next();
    if (last && !L0) {
      // the sender's sums over the wave's 4 row groups; lanes < 16 write
#pragma unroll
      for (int q = 0; q < FTW; ++q)
#pragma unroll
        for (int k = 0; k < 3; ++k)
          for (int o = 16; o < 64; o *= 2) {
            acc_h[q][k] += __shfl_xor(acc_h[q][k], o);
            acc_v[q][k] += __shfl_xor(acc_v[q][k], o);
          }
      if (lane < 16) {
        // all loads of g_v' first: the stores may alias them for all the
        // compiler knows, and would otherwise wait for each load in turn
        A gvj[FTW][3];
#pragma unroll
        for (int q = 0; q < FTW; ++q)
#pragma unroll
          for (int k = 0; k < 3; ++k) gvj[q][k] = gv[jb + k * F + (FTW * wave + q) * 16 + lane];
#pragma unroll
        for (int q = 0; q < FTW; ++q) {
          const int ch = (FTW * wave + q) * 16 + lane;
#pragma unroll
          for (int k = 0; k < 3; ++k) {
            gh_out[jb + k * F + ch] = acc_h[q][k];
            gv_out[jb + k * F + ch] = gvj[q][k] + acc_v[q][k];
          }
        }
      }
#pragma unroll
      for (int q = 0; q < FTW; ++q)
#pragma unroll
        for (int k = 0; k < 3; ++k) acc_h[q][k] = acc_v[q][k] = 0;
    }
    if (!more) break;
    j = jn;
    c0 = cn;
  }
}

// Channel-per-lane form of the reverse message (FP32).  A workgroup of
// mbl_nw<F>() waves owns MB_RB2 consecutive senders and a slice of
// 64 mbl_nw<F>() channels (wide layers take several slices in consecutive
// workgroups); each wave owns 64 channels and keeps their filter B fragments
// in registers.
// The block's sender-ordered edges (its senders' rows back to back) stream in
// 16-edge chunks that may span senders.  Per chunk the wave forms the filter
// w and its d-derivative w' on the matrix cores (the same B fragments against
// the basis rows and their derivatives) and parks both in LDS, channel-major;
// then every lane, one channel, walks the chunk's edges.  The receiver of an
// edge is wave-uniform, so each gather of g_s', g_v' reads 256 contiguous
// bytes.  The sender's dE/dh and v terms stay in the lane until its last
// edge.  Every 4 edges the 16 per-edge channel sums (dE/dd and dE/drhat of 4
// edges) are summed over the wave through LDS rows and added to the edges'
// slots of this wave: one add per slot per launch, so the sums are
// deterministic.
constexpr int MB_RB2 = 8;

template <int F>
constexpr int mbl_nw() { return F / 64 < 2 ? F / 64 : 2; }

// L0: the first layer, where v = 0 and only the per-edge sums are wanted
// (h and v of the first layer depend on the species alone): A_v = 0, so the
// filter's v part and its derivative drop out, and dE/dd, dE/drhat need w^r,
// w'^s and w'^r only; no g_h, g_v are formed.
template <class P, int F, int KBM, bool L0>
__global__ void __launch_bounds__((64 * mbl_nw<F>())) __attribute__((amdgpu_waves_per_eu(2)))
k_message_bwd_lane(MsgBwdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  using Fr = typename P::Fr;
  static_assert(sizeof(T) == 4 && sizeof(A) == 4, "FP32 storage and accumulation");
  constexpr int NWB = mbl_nw<F>(), SLICES = F / 64 / NWB, NW = F / 64, NFT = F / 16;
  static_assert(F % 64 == 0 && (F / 64) % NWB == 0, "64-channel waves");
  constexpr int kcols = KBM * P::KC;
  constexpr int BF_REGS = 12 * KBM;
  constexpr int QI = BF_REGS > 100 ? 1 : 2;       // feature tiles whose MFMA chains run together
  constexpr int EG = BF_REGS > 100 ? 4 : 8;       // edges gathered per group (a multiple of 4)
  // LDS tiles of w and w' (3 parts each): channel-major, the chunk's 16 edges
  // per channel as 4 groups of 4 in the order g ^ (((ch >> 1) ^ (ch >> 2)) & 3),
  // so 16-byte accesses by 8 or 16 consecutive lanes hit distinct bank groups
  constexpr int WLD = 16;
  __shared__ __attribute__((aligned(16))) A Wt[NWB][6][64 * WLD];
  // per wave 8 rows of 64 per-edge partial sums (+4: the 16-byte groups
  // that 16 consecutive lanes read fall on distinct banks).  8 rows, not
  // the 16 values at once: with 16 the workgroup's LDS would leave room for
  // two workgroups per CU instead of three.
  constexpr int RLD = 64 + 4;
  __shared__ __attribute__((aligned(16))) A Rd[NWB][8 * RLD];
  auto wslot = [](int ch, int g) { return ch * WLD + 4 * (g ^ (((ch >> 1) ^ (ch >> 2)) & 3)); };
  const int per_xcd = gridDim.x / 8;
  const int lb = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int lane = threadIdx.x & 63, wl = threadIdx.x >> 6;
  const int wave = (lb % SLICES) * NWB + wl;    // this wave's slot among the feature set's NW
  const int c = 64 * wave + lane;               // this lane's channel
  const int j0 = lb / SLICES * MB_RB2;
  if (j0 >= a.N) return;
  const int j1 = min(a.N, j0 + MB_RB2);
  const int tp_lane = a.t_ptr[j0 + min(lane, j1 - j0)];
  auto tp = [&](int j) { return __builtin_amdgcn_readlane(tp_lane, j - j0); };
  const T* Wf = (const T*)a.filt.w;
  const T* h = (const T*)a.h;
  const T* vv = (const T*)a.v;
  const A* gs = (const A*)a.gs;
  const A* gv = (const A*)a.gv;
  const A* einfo = (const A*)a.einfo;
  const T* basis = (const T*)a.basis;
  const T* dbasis = (const T*)a.dbasis;
  A* gh_out = (A*)a.gh;
  A* gv_out = (A*)a.gv_out;
  A* eg = (A*)a.eg;
  // senders without incoming edges: g_h = 0, g_v = g_v'
  if constexpr (!L0)
    for (int j = j0; j < j1; ++j)
      if (tp(j) == tp(j + 1)) {
        const size_t jb = (size_t)j * 3 * F;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          gh_out[jb + k * F + c] = A(0);
          gv_out[jb + k * F + c] = gv[jb + k * F + c];
        }
      }
  const int T0 = tp(j0), T1 = tp(j1);
  if (T0 == T1) return;
  // The filter's B fragments stay in registers unless they are many (a
  // long filter input); then they stream from the caches chunk by chunk (an
  // opaque copy of the pointer keeps the compiler from hoisting them).
  constexpr bool BREG = BF_REGS <= 120;
  Fr Bf[BREG ? 4 : 1][3][BREG ? KBM : 1];
  if constexpr (BREG) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int part = 0; part < 3; ++part)
#pragma unroll
        for (int kb = 0; kb < KBM; ++kb) {
          const int ct = part * NFT + 4 * wave + q;
          Bf[q][part][kb] = P::frag(Wf + ((size_t)(ct * KBM + kb) * 64 + lane) * P::KPL);
        }
  }
  A* wt = Wt[wl][0];
  auto first_with_edges = [&](int j) {
    while (j < j1 && tp(j) == tp(j + 1)) ++j;
    return j;
  };
  // the next chunk's A rows (position cc0 + lane % 16; past the stream's end
  // the zero row E) and, in lanes e < ccnt, edge cc0 + e's id, rhat and
  // receiver
  Fr Gn[KBM], Dn[KBM];
  int idn = -1;
  A exn = 0, eyn = 0, ezn = 0, ern = 0;
  auto prefetch = [&](int cc0, int ccnt) {
    const int r = (lane & 15) < ccnt ? cc0 + (lane & 15) : (int)a.E;
    const T* gp = basis + (size_t)r * kcols + (lane >> 4) * P::KPL;
    const T* dp = dbasis + (size_t)r * kcols + (lane >> 4) * P::KPL;
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) {
      Gn[kb] = P::frag(gp + kb * P::KC);
      Dn[kb] = P::frag(dp + kb * P::KC);
    }
    idn = -1;
    exn = eyn = ezn = ern = 0;
    if (lane < ccnt) {
      const A* ei = einfo + 4 * (size_t)(cc0 + lane);
      idn = a.t_edge[cc0 + lane];
      exn = ei[0];
      eyn = ei[1];
      ezn = ei[2];
      ern = ei[3];
    }
  };
  int c0 = T0;
  prefetch(c0, min(16, T1 - c0));
  // the sender being summed: j, whose edges end at sb; its h and v at this
  // lane's channel
  int j = first_with_edges(j0);
  int sb = tp(j + 1);
  size_t jb = (size_t)j * 3 * F;
  A hs, hv, hr, v0, v1, v2;
  auto load_sender = [&] {
    hs = P::ld(h[jb + c]);
    hr = P::ld(h[jb + 2 * F + c]);
    if constexpr (L0) {
      hv = v0 = v1 = v2 = A(0);
    } else {
      hv = P::ld(h[jb + F + c]);
      v0 = P::ld(vv[jb + c]);
      v1 = P::ld(vv[jb + F + c]);
      v2 = P::ld(vv[jb + 2 * F + c]);
    }
  };
  load_sender();
  A acc_h0 = 0, acc_h1 = 0, acc_h2 = 0, acc_v0 = 0, acc_v1 = 0, acc_v2 = 0;
  auto write_out = [&] {
    if constexpr (L0) return;
    const A g0 = gv[jb + c], g1 = gv[jb + F + c], g2 = gv[jb + 2 * F + c];
    gh_out[jb + c] = acc_h0;
    gh_out[jb + F + c] = acc_h1;
    gh_out[jb + 2 * F + c] = acc_h2;
    gv_out[jb + c] = g0 + acc_v0;
    gv_out[jb + F + c] = g1 + acc_v1;
    gv_out[jb + 2 * F + c] = g2 + acc_v2;
  };
  // edge c0 + e starts the next sender: write sender j out and move on (a
  // wave-uniform branch; the last sender is written after the stream)
  auto next_sender = [&] {
    write_out();
    acc_h0 = acc_h1 = acc_h2 = acc_v0 = acc_v1 = acc_v2 = 0;
    j = first_with_edges(j + 1);
    sb = tp(j + 1);
    jb = (size_t)j * 3 * F;
    load_sender();
  };
  while (true) {
    const int cnt = min(16, T1 - c0);
    Fr Ga[KBM], Gd[KBM];
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) {
      Ga[kb] = Gn[kb];
      Gd[kb] = Dn[kb];
    }
    const int eid = idn;
    const A ex = exn, ey = eyn, ez = ezn, er = ern;
    const int cn = c0 + 16;
    const bool more = cn < T1;
    if (more) prefetch(cn, min(16, T1 - cn));
    // w and w' of 4 feature tiles x 3 parts into LDS
    // (Through an integer and back to a global pointer, as in the MFMA
    // kernel above, so that the loads stay global loads.)
    uintptr_t wbits = (uintptr_t)Wf;
    if constexpr (!BREG) asm volatile("" : "+s"(wbits));
    const T* Wc = (const T*)(const T __attribute__((address_space(1)))*)wbits;
#pragma unroll
    for (int q0 = 0; q0 < 4; q0 += QI) {
      C w[QI][3], wd[QI][3];
#pragma unroll
      for (int q = 0; q < QI; ++q)
#pragma unroll
        for (int part = 0; part < 3; ++part)
          for (int r = 0; r < 4; ++r) w[q][part][r] = wd[q][part][r] = 0;
#pragma unroll
      for (int kb = 0; kb < KBM; ++kb)
#pragma unroll
        for (int q = 0; q < QI; ++q)
#pragma unroll
          for (int part = 0; part < 3; ++part) {
            if (L0 && part == 1) continue;
            Fr b;
            if constexpr (BREG) {
              b = Bf[q0 + q][part][kb];
            } else {
              const int ct = part * NFT + 4 * wave + q0 + q;
              b = P::frag(Wc + ((size_t)(ct * KBM + kb) * 64 + lane) * P::KPL);
            }
            if (!L0 || part == 2) w[q][part] = P::mfma(Ga[kb], b, w[q][part]);
            wd[q][part] = P::mfma(Gd[kb], b, wd[q][part]);
          }
      // this lane's 4 accumulator rows are the 4 consecutive edges of group
      // lane / 16 at one channel: one 16-byte write per part
#pragma unroll
      for (int q = 0; q < QI; ++q) {
        const int o = wslot(16 * (q0 + q) + (lane & 15), lane >> 4);
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          if (L0 && part == 1) continue;
          if (!L0 || part == 2)
            *(f4_t*)(wt + part * 64 * WLD + o) = f4_t{w[q][part][0], w[q][part][1], w[q][part][2], w[q][part][3]};
          *(f4_t*)(wt + (3 + part) * 64 * WLD + o) =
              f4_t{wd[q][part][0], wd[q][part][1], wd[q][part][2], wd[q][part][3]};
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // receivers' g_s', g_v' at this lane's channel for EG edges (past the
    // stream's end the receiver is row 0 and the filter zero)
    A gg[4][EG];
    auto gather = [&](int ebase) {
#pragma unroll
      for (int u = 0; u < EG; ++u) {
        const int i = acc_index(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(er), ebase + u)));
        const size_t ib = (size_t)i * 3 * F;
        gg[0][u] = gs[(size_t)i * F + c];
        gg[1][u] = gv[ib + c];
        gg[2][u] = gv[ib + F + c];
        gg[3][u] = gv[ib + 2 * F + c];
      }
    };
    auto consume = [&](int ebase) {
#pragma unroll
      for (int u4 = 0; u4 < EG; u4 += 4) {
        const int o = wslot(lane, (ebase + u4) / 4);
        f4_t ws4 = {}, wv4 = {}, dv4 = {};
        if constexpr (!L0) {
          ws4 = *(const f4_t*)(wt + o);
          wv4 = *(const f4_t*)(wt + 64 * WLD + o);
          dv4 = *(const f4_t*)(wt + 4 * 64 * WLD + o);
        }
        const f4_t wr4 = *(const f4_t*)(wt + 2 * 64 * WLD + o);
        const f4_t ds4 = *(const f4_t*)(wt + 3 * 64 * WLD + o), dr4 = *(const f4_t*)(wt + 5 * 64 * WLD + o);
        // per edge: [dE/dd, dE/drhat x, y, z] partial sums of this channel
        A vals[16];
#pragma unroll
        for (int uu = 0; uu < 4; ++uu) {
          const int u = u4 + uu, e = ebase + u;
          if (c0 + e == sb && sb < T1) next_sender();
          const A rx = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ex), e));
          const A ry = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ey), e));
          const A rz = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ez), e));
          // past the stream's end: exactly nothing (not 0 x receiver 0's
          // gradient, which may be NaN)
          const bool live = e < cnt;
          const A g_s = live ? gg[0][u] : A(0), g0 = live ? gg[1][u] : A(0);
          const A g1 = live ? gg[2][u] : A(0), g2 = live ? gg[3][u] : A(0);
          const A Ar = g0 * rx + g1 * ry + g2 * rz;
          const A tr = hr * wr4[uu];
          if constexpr (L0) {
            vals[4 * uu] = g_s * hs * ds4[uu] + Ar * hr * dr4[uu];
          } else {
            const A Av = g0 * v0 + g1 * v1 + g2 * v2;
            acc_h0 += g_s * ws4[uu];
            acc_h1 += Av * wv4[uu];
            acc_h2 += Ar * wr4[uu];
            const A tv = hv * wv4[uu];
            acc_v0 += g0 * tv;
            acc_v1 += g1 * tv;
            acc_v2 += g2 * tv;
            vals[4 * uu] = g_s * hs * ds4[uu] + Av * hv * dv4[uu] + Ar * hr * dr4[uu];
          }
          vals[4 * uu + 1] = g0 * tr;
          vals[4 * uu + 2] = g1 * tr;
          vals[4 * uu + 3] = g2 * tr;
        }
        // the 16 values summed over the wave's 64 lanes (channels), 8 at a
        // time through the wave's LDS rows: value k of every lane in row k;
        // lane l sums entries 8 (l % 8) .. 8 (l % 8) + 7 of row l / 8, and
        // shuffles within each 8 lanes finish the row
        A* rw = Rd[wl];
        const A* rr = rw + (lane >> 3) * RLD + (lane & 7) * 8;
        A tot[2];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
          for (int k = 0; k < 8; ++k) rw[k * RLD + lane] = vals[8 * p + k];
          __builtin_amdgcn_wave_barrier();
          const f4_t x = *(const f4_t*)rr, y = *(const f4_t*)(rr + 4);
          __builtin_amdgcn_wave_barrier();
          A t = ((x[0] + x[1]) + (x[2] + x[3])) + ((y[0] + y[1]) + (y[2] + y[3]));
          t += __shfl_xor(t, 1);
          t += __shfl_xor(t, 2);
          t += __shfl_xor(t, 4);
          tot[p] = t;
        }
        // lane 8 r adds values r and 8 + r: (edge, component) = (k / 4, k % 4)
        const int k0 = lane >> 3, k1 = 8 + (lane >> 3);
        const int e0 = __shfl(eid, ebase + u4 + (k0 >> 2)), e1 = __shfl(eid, ebase + u4 + (k1 >> 2));
        if ((lane & 7) == 0) {
          if (e0 >= 0) unsafeAtomicAdd(eg + ((size_t)e0 * NW + wave) * 4 + (k0 & 3), tot[0]);
          if (e1 >= 0) unsafeAtomicAdd(eg + ((size_t)e1 * NW + wave) * 4 + (k1 & 3), tot[1]);
        }
      }
    };
#pragma unroll
    for (int eb0 = 0; eb0 < 16; eb0 += EG)
      if (eb0 < cnt) {
        gather(eb0);
        consume(eb0);
      }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (!more) break;
    c0 = cn;
  }
  write_out();
}

// ------------------------------------------------------------------ forces ----
// dE/dr_e = dE/dd rhat + (dE/drhat - (dE/drhat . rhat) rhat) / d  (FP64
// geometry, the wave slots summed in order).
template <class A>
__global__ void __launch_bounds__(256) k_edge_grad(long long E, int NW, const int32_t* __restrict__ recv,
                                                  const int32_t* __restrict__ col,
                                                  const int32_t* __restrict__ shift,
                                                  const int32_t* __restrict__ atom_struct,
                                                  const double* __restrict__ pos,
                                                  const double* __restrict__ cell,
                                                  const A* __restrict__ eg, double* __restrict__ gr) {
  const long long e = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int i = recv[e], j = col[e], sh = shift[e];
  const double* Cl = cell + 9 * atom_struct[i];
  const double n0 = (double)(int8_t)(sh & 0xff), n1 = (double)(int8_t)((sh >> 8) & 0xff),
               n2 = (double)(int8_t)((sh >> 16) & 0xff);
  const double rx = (pos[3 * j] - pos[3 * i]) + ((n0 * Cl[0] + n1 * Cl[3]) + n2 * Cl[6]);
  const double ry = (pos[3 * j + 1] - pos[3 * i + 1]) + ((n0 * Cl[1] + n1 * Cl[4]) + n2 * Cl[7]);
  const double rz = (pos[3 * j + 2] - pos[3 * i + 2]) + ((n0 * Cl[2] + n1 * Cl[5]) + n2 * Cl[8]);
  const double d = sqrt(rx * rx + ry * ry + rz * rz);
  const double ux = rx / d, uy = ry / d, uz = rz / d;
  double gd = 0, gx = 0, gy = 0, gz = 0;
  for (int w = 0; w < NW; ++w) {
    const A* p = eg + ((size_t)e * NW + w) * 4;
    gd += (double)p[0];
    gx += (double)p[1];
    gy += (double)p[2];
    gz += (double)p[3];
  }
  const double dot = gx * ux + gy * uy + gz * uz;
  gr[3 * e] = gd * ux + (gx - dot * ux) / d;
  gr[3 * e + 1] = gd * uy + (gy - dot * uy) / d;
  gr[3 * e + 2] = gd * uz + (gz - dot * uz) / d;
}

__global__ void __launch_bounds__(256) k_forces(int N, const int32_t* __restrict__ row_ptr,
                                               const int32_t* __restrict__ t_ptr,
                                               const int32_t* __restrict__ t_edge,
                                               const double* __restrict__ gr, double* __restrict__ forces) {
  const int a = blockIdx.x * blockDim.x + threadIdx.x;
  if (a >= N) return;
  double fx = 0, fy = 0, fz = 0;
  for (int e = row_ptr[a]; e < row_ptr[a + 1]; ++e) {
    fx += gr[3 * (size_t)e];
    fy += gr[3 * (size_t)e + 1];
    fz += gr[3 * (size_t)e + 2];
  }
  for (int t = t_ptr[a]; t < t_ptr[a + 1]; ++t) {
    const size_t e = t_edge[t];
    fx -= gr[3 * e];
    fy -= gr[3 * e + 1];
    fz -= gr[3 * e + 2];
  }
  forces[3 * (size_t)a] = fx;
  forces[3 * (size_t)a + 1] = fy;
  forces[3 * (size_t)a + 2] = fz;
}

// ---------------------------------------------------------------- driver ----
template <class K>
hipError_t allow_lds(K kernel, size_t smem) {
  if (smem <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
}

template <class P, int F, int KBM>
void launch_message_bwd_kbm(hipStream_t st, const MsgBwdArgs& ma) {
  if constexpr (sizeof(typename P::T) == 4) {
    constexpr int NWB = mbl_nw<F>(), SLICES = F / 64 / NWB;
    const int blocks = (int)(((long long)(ma.N + MB_RB2 - 1) / MB_RB2 * SLICES + 7) / 8 * 8);
    if (ma.first) k_message_bwd_lane<P, F, KBM, true><<<blocks, 64 * NWB, 0, st>>>(ma);
    else k_message_bwd_lane<P, F, KBM, false><<<blocks, 64 * NWB, 0, st>>>(ma);
  } else {
    constexpr int NWB = mb_nwb<P, F, KBM>(), SLICES = F / 16 / mb_ftw<P, F, KBM>() / NWB;
    const int blocks = (int)(((long long)(ma.N + MB_RB - 1) / MB_RB * SLICES + 7) / 8 * 8);
    if (ma.first) k_message_bwd<P, F, KBM, true><<<blocks, 64 * NWB, 0, st>>>(ma);
    else k_message_bwd<P, F, KBM, false><<<blocks, 64 * NWB, 0, st>>>(ma);
  }
}

// Per-edge slots of the reverse message kernel (one per wave of a feature
// slice set), for a filter input of nkb k-blocks: FP32 runs the
// channel-per-lane form (64 channels per wave).
template <class P, int F>
int message_bwd_slots(int nkb) {
  if constexpr (sizeof(typename P::T) == 4) return F / 64;
  return F / 16 / (nkb == 3 ? mb_ftw<P, F, 3>() : mb_ftw<P, F, 6>());
}

template <class P, int F>
hipError_t launch_message_bwd(hipStream_t st, const MsgBwdArgs& ma, int nkb) {
  switch (nkb) {
    case 3: launch_message_bwd_kbm<P, F, 3>(st, ma); break;
    case 6: launch_message_bwd_kbm<P, F, 6>(st, ma); break;
    case 9: launch_message_bwd_kbm<P, F, 9>(st, ma); break;
    case 12: launch_message_bwd_kbm<P, F, 12>(st, ma); break;
    case 17: launch_message_bwd_kbm<P, F, 17>(st, ma); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class P, int F>
hipError_t backward_impl(hipStream_t st, BackwardArgs& ba) {
  using T = typename P::T;
  using A = typename P::A;
  const painn_graph* g = ba.g;
  const PrecModel* pm = ba.pm;
  const Hyper& hp = ba.m->hp;
  const int N = g->N;
  const long long E = g->E;
  const SaveLayout sv(ba.save, N, F, hp.L, sizeof(T));
  const int kcols = pm->layers[0].filt_mma.din_p;
  const int NW = message_bwd_slots<P, F>(kcols / P::KC);   // per-edge slots (waves of the message kernel)
  if (N == 0) return hipSuccess;
  // LDS of the tile kernels: 16 rows of 3F + F (+ padding), or of F alone
  // with the 3F-wide buffer in global memory
  constexpr bool UGX = (size_t)16 * (4 * F + 2 * P::PAD) * sizeof(T) > 160 * 1024;
  const size_t smem_ub = (size_t)16 * ((UGX ? 0 : 3 * F + P::PAD) + F + P::PAD) * sizeof(T);
  hipError_t e = allow_lds(k_update_bwd<P, F, UGX>, smem_ub);
  if (e == hipSuccess) e = allow_lds(k_phi_bwd<P, F, UGX>, smem_ub);
  if (e != hipSuccess) return e;
  if (E > 0) {
    const double delta = hp.cutoff / (hp.K - 1);
    k_edge_rev<P><<<(unsigned)((E + 16 + EP_REV - 1) / EP_REV), EP_REV, (size_t)EP_REV * kcols * sizeof(T), st>>>(
        E, hp.K, kcols, hp.cutoff, hp.rbf_type, 1.0 / (2.0 * delta * delta), delta, g->t_edge, g->recv, g->col,
        g->shift, g->atom_struct, g->pos, g->cell, (const A*)ba.einfo, (T*)ba.basis_t,
        (T*)ba.dbasis, (A*)ba.einfo_t);
    k_fill<A><<<grid_of((size_t)E * NW * 4, 256), 256, 0, st>>>((size_t)E * NW * 4, (A*)ba.eg);
  }
  k_fill<A><<<grid_of((size_t)N * 3 * F, 256), 256, 0, st>>>((size_t)N * 3 * F, (A*)ba.gv);
  // With dataset ids, an atom of a structure whose id is outside [0, H) is in
  // no head tile: its dE/ds stays NaN, so are its structure's forces (as the
  // forward's energy of that structure).  No edge leaves a structure and
  // every dense product keeps atoms in their own rows, so it stays there.
  if (ba.dataset_id && !ba.blend)
    k_fill<A><<<grid_of((size_t)N * F, 256), 256, 0, st>>>((size_t)N * F, (A*)ba.gs,
                                                           (A)__builtin_nan(""));
  // heads
  prof_mark(ba.prof, st, KC_BWD_HEADS, true);
  {
    HeadBwdArgs ha;
    ha.N = N;
    ha.F = F;
    ha.ns = (int)pm->shared.size();
    ha.nb = (int)hp.branch_dims.size();
    if (ha.ns > 16 || ha.nb > 16 || ha.ns + ha.nb > 32) return hipErrorInvalidValue;
    int wmax = F, off = 0;
    for (int m = 0; m < ha.ns; ++m) {
      ha.shared[m] = pm->shared[m];
      ha.sharedT[m] = pm->sharedT[m];
      wmax = wmax > pad32(hp.shared_dims[m]) ? wmax : pad32(hp.shared_dims[m]);
    }
    for (int m = 0; m < ha.nb; ++m) {
      ha.bdout[m] = hp.branch_dims[m];
      if (m + 1 < ha.nb) wmax = wmax > pad32(hp.branch_dims[m]) ? wmax : pad32(hp.branch_dims[m]);
    }
    for (int m = 0; m + 1 < ha.ns + ha.nb; ++m) {
      ha.zoff[m] = off;
      off += m < ha.ns ? pad32(hp.shared_dims[m]) : pad32(hp.branch_dims[m - ha.ns]);
    }
    if (off > ba.scratch_w) return hipErrorInvalidValue;
    ha.ldw = wmax + P::PAD;
    ha.s = sv.S(hp.L);
    ha.table = (const void* const*)pm->head_table;
    ha.tableT = (const void* const*)pm->head_tableT;
    ha.scratch = ba.scratch;
    ha.sw = ba.scratch_w;
    ha.gs = ba.gs;
    ha.xbuf = ba.xbuf;
    ha.gh = ba.blend ? ba.g_heads : nullptr;
    ha.H = hp.n_heads;
    const bool hgx = (size_t)2 * 16 * ha.ldw * sizeof(T) > 150 * 1024;
    const size_t smem = hgx ? 0 : (size_t)2 * 16 * ha.ldw * sizeof(T);
    const bool wide = wmax >= HB_WIDE;
    e = hgx ? hipSuccess
            : (wide ? allow_lds(k_heads_bwd<P, F, false, HB_NW_WIDE>, smem)
                    : allow_lds(k_heads_bwd<P, F, false, HB_NW_NARROW>, smem));
    if (e != hipSuccess) return e;
    int grid;
    if (ba.dataset_id || ba.blend) {
      // the forward's grouping: tiles of atoms of one head (blended: of
      // every kept (atom, head) entry)
      ha.order = ba.head_order;
      ha.tiles = (const HeadTile*)ba.head_tiles;
      ha.plan = (const HeadPlan*)ba.head_plan;
      grid = (int)(((long long)N * (ba.blend ? hp.n_heads : 1) + 15) / 16) + hp.n_heads;   // >= its tile count
      grid = grid < HB_GRID ? grid : HB_GRID;
    } else {
      ha.order = nullptr;
      ha.tiles = nullptr;
      ha.plan = nullptr;
      grid = (N + 15) / 16;
      grid = grid < HB_GRID ? grid : HB_GRID;
    }
    if (hgx && (size_t)grid * 2 * 16 * ha.ldw * sizeof(T) > ba.xbuf_bytes) return hipErrorInvalidValue;
    if (hgx) k_heads_bwd<P, F, true, HB_NW_WIDE><<<grid, 64 * HB_NW_WIDE, 0, st>>>(ha);
    else if (wide) k_heads_bwd<P, F, false, HB_NW_WIDE><<<grid, 64 * HB_NW_WIDE, smem, st>>>(ha);
    else k_heads_bwd<P, F, false, HB_NW_NARROW><<<grid, 64 * HB_NW_NARROW, smem, st>>>(ha);
    if (ba.blend)
      k_blend_grad<A><<<grid_of((size_t)N * F, 256), 256, 0, st>>>(N, hp.n_heads, F, (A)ba.skip, g->atom_struct,
                                                                    (const A*)ba.hw, (const A*)ba.g_heads,
                                                                    (A*)ba.gs);
  }
  prof_mark(ba.prof, st, KC_BWD_HEADS, false);
  const int tiles = (N + 15) / 16;
  for (int l = hp.L - 1; l >= 0; --l) {
    const LayerDev& Ld = pm->layers[l];
    UpdBwdArgs ua;
    ua.N = N;
    ua.uv = sv.UV(l);
    ua.z = sv.Z(l);
    ua.ag = sv.Agate(l);
    ua.gs = ba.gs;
    ua.gv = ba.gv;
    ua.gs_out = ba.gs2;
    ua.gv_out = ba.gv2;
    ua.scratch = ba.scratch;
    ua.sw = ba.scratch_w;
    ua.uvT = Ld.uvT;
    ua.upd1T = Ld.upd1T;
    ua.upd2T = Ld.upd2T;
    ua.xbuf = ba.xbuf;
    if (UGX && (size_t)tiles * 16 * (3 * F + P::PAD) * sizeof(T) > ba.xbuf_bytes) return hipErrorInvalidValue;
    prof_mark(ba.prof, st, KC_BWD_UPDATE, true);
    k_update_bwd<P, F, UGX><<<tiles, 64 * ub_nw<P, F>(), smem_ub, st>>>(ua);
    prof_mark(ba.prof, st, KC_BWD_UPDATE, false);
    MsgBwdArgs ma;
    ma.N = N;
    ma.E = E;
    ma.t_ptr = g->t_ptr;
    ma.t_edge = g->t_edge;
    ma.basis = ba.basis_t;
    ma.dbasis = ba.dbasis;
    ma.einfo = ba.einfo_t;
    ma.filt = Ld.filt_mma;
    ma.h = sv.H(l);
    ma.v = sv.V(l);
    ma.gs = ba.gs2;
    ma.gv = ba.gv2;
    ma.gh = ba.gh;
    ma.gv_out = ba.gv;
    ma.eg = ba.eg;
    ma.first = l == 0;
    ma.bg = (size_t)N * 3 * F * sizeof(A) < ((size_t)1 << 31);
    prof_mark(ba.prof, st, KC_BWD_MESSAGE, true);
    e = launch_message_bwd<P, F>(st, ma, kcols / P::KC);
    prof_mark(ba.prof, st, KC_BWD_MESSAGE, false);
    if (e != hipSuccess) return e;
    if (l > 0) {
      PhiBwdArgs pa;
      pa.N = N;
      pa.s = sv.S(l);
      pa.gh = ba.gh;
      pa.gs_mid = ba.gs2;
      pa.gs_out = ba.gs;
      pa.scratch = ba.scratch;
      pa.sw = ba.scratch_w;
      pa.phi1 = Ld.phi1;
      pa.phi1T = Ld.phi1T;
      pa.phi2T = Ld.phi2T;
      pa.xbuf = ba.xbuf;
      prof_mark(ba.prof, st, KC_BWD_PHI, true);
      k_phi_bwd<P, F, UGX><<<tiles, 64 * ub_nw<P, F>(), smem_ub, st>>>(pa);
      prof_mark(ba.prof, st, KC_BWD_PHI, false);
    }
  }
  prof_mark(ba.prof, st, KC_FORCE, true);
  if (E > 0)
    k_edge_grad<A><<<(unsigned)((E + 255) / 256), 256, 0, st>>>(E, NW, g->recv, g->col, g->shift, g->atom_struct,
                                                                 g->pos, g->cell, (const A*)ba.eg, ba.gr);
  k_forces<<<(N + 255) / 256, 256, 0, st>>>(N, g->row_ptr, g->t_ptr, g->t_edge, ba.gr, ba.forces);
  prof_mark(ba.prof, st, KC_FORCE, false);
  return hipGetLastError();
}

template <class P>
hipError_t backward_prec(hipStream_t st, BackwardArgs& ba) {
  switch (ba.m->hp.F) {
    case 64: return backward_impl<P, 64>(st, ba);
    case 128: return backward_impl<P, 128>(st, ba);
    case 256: return backward_impl<P, 256>(st, ba);
    case 384: return backward_impl<P, 384>(st, ba);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_backward(hipStream_t st, int prec, BackwardArgs& ba) {
  if (prec == PAINN_FP64) return backward_prec<P64>(st, ba);
  if (prec == PAINN_FP32) return backward_prec<P32>(st, ba);
  return hipErrorInvalidValue;
}

hipError_t launch_transpose(hipStream_t st, Profiler* p, painn_graph* g) {
  const int N = g->N;
  const long long E = g->E;
  prof_mark(p, st, KC_TRANSPOSE, true);
  k_fill<int32_t><<<grid_of((size_t)N + 1, 256), 256, 0, st>>>((size_t)N + 1, g->t_count);
  if (E > 0) k_t_count<<<grid_of((size_t)E, 256), 256, 0, st>>>(E, g->col, g->t_count);
  // the graph's scan buffer (at least (N + 1023) / 1024 + 1 entries) holds
  // the block sums; the graph build that used it has finished on this stream
  const int nblk = (N + 1023) / 1024;
  if (nblk > 0) k_t_scan_blocks<<<nblk, 256, 0, st>>>(N, g->t_count, g->scan_tmp);
  k_t_scan_top<<<1, 256, 0, st>>>(nblk, g->scan_tmp, g->t_ptr, N);
  if (nblk > 0) k_t_scan_apply<<<nblk, 256, 0, st>>>(N, g->t_count, g->scan_tmp, g->t_ptr);
  if (E > 0) {
    k_t_fill<<<grid_of((size_t)E, 256), 256, 0, st>>>(E, g->col, g->t_ptr, g->t_count, g->t_edge);
    k_t_sort<<<(N + 3) / 4, 256, 0, st>>>(N, g->t_ptr, g->t_edge);
  }
  prof_mark(p, st, KC_TRANSPOSE, false);
  return hipGetLastError();
}
