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
#include <type_traits>

#include "mfma.h"

namespace {

// ---------------------------------------------------------------- embed ----
// s = emb[species], v = 0 (when v is given) and, when h is given, layer 0's
// h = h0[species] (the species' row of the phi table: phi acts on each row
// by itself, so the row is what phi gives for the atom's own s).  Each
// thread moves 4 consecutive elements of a row (F is a multiple of 64).
template <class P, int F>
__global__ void __launch_bounds__(256) k_embed(int N, const int32_t* __restrict__ species,
                                              const typename P::T* __restrict__ emb,
                                              const typename P::T* __restrict__ h0,
                                              typename P::T* __restrict__ s,
                                              typename P::T* __restrict__ v,
                                              typename P::T* __restrict__ h) {
  using T = typename P::T;
  using Q = Quad<T>;
  constexpr int F4 = F / 4;
  const size_t tot = (size_t)N * F4;
  Q zero;
  for (int k = 0; k < 4; ++k) zero.x[k] = P::st(0);
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < tot; x += (size_t)gridDim.x * blockDim.x) {
    const size_t i = x / F4, f = (x % F4) * 4;
    const size_t z = (size_t)species[i];
    *(Q*)(s + i * F + f) = *(const Q*)(emb + z * F + f);
    if (v) {
      *(Q*)(v + 3 * i * F + f) = zero;
      *(Q*)(v + 3 * i * F + F + f) = zero;
      *(Q*)(v + 3 * i * F + 2 * F + f) = zero;
    }
    if (h) {
      *(Q*)(h + 3 * i * F + f) = *(const Q*)(h0 + 3 * z * F + f);
      *(Q*)(h + 3 * i * F + F + f) = *(const Q*)(h0 + 3 * z * F + F + f);
      *(Q*)(h + 3 * i * F + 2 * F + f) = *(const Q*)(h0 + 3 * z * F + 2 * F + f);
    }
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
template <class P, int F, int RT, int NW = 4>
__device__ __forceinline__ void phi_tile(const typename P::T* X, int ldx, typename P::T* H,
                                         size_t row0, int N, const DenseDev& d1,
                                         const DenseDev& d2, typename P::T* __restrict__ h) {
  using A = typename P::A;
  constexpr int LD = F + P::PAD;
  const int lane = threadIdx.x & 63;
  dense_tiles<P, RT, NW, F>(X, ldx, d1, [&](int ct, typename P::C* acc) {
    const int col = ct * 16 + (lane & 15);
    const A bias = ((const A*)d1.b)[col];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) H[(r * 16 + P::row(lane, i)) * LD + col] = P::st(silu<A>(acc[r][i] + bias));
  });
  __syncthreads();
  dense_tiles<P, RT, NW, F>(H, LD, d2, [&](int ct, typename P::C* acc) {
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
// Per edge e = (i <- j, n) and channel c:
//   w_e = f_c(d) (Wf g(d) + bf)                         radial filter, 3F channels
//   ds_i    += h^s_j w^s_e
//   dv_i[c] += v_j[c] h^v_j w^v_e + rhat[c] h^r_j w^r_e
// summed per receiver (the CSR is sorted by receiver, so this is a plain
// in-register reduction: no atomics, deterministic).
//
// The filter runs on the matrix cores: for 16 edges of one receiver
//   Wt[16 edges, 3F] = Gh[16, K+1] [Wf | bf]^T,
//   Gh[e] = (f_c g_0(d_e), ..., f_c g_{K-1}(d_e), f_c(d_e))
// (the bias column carries f_c, so Wt = f_c (Wf g + bf)).  Gh does not depend
// on the layer: k_edge_prep writes it once per forward, in the MFMA operand
// type (BF16 as two terms [hi | lo] against the filter stored twice along K),
// next to each edge's rhat and sender index.
struct MsgArgs {
  int N, F, K;
  const int32_t* row_ptr;
  const void* basis;   // [E + 16][kcols] storage type (16 zero rows of padding)
  const void* einfo;   // [E][4] accumulation type: rhat x, y, z, sender index
  DenseDev filt_mma;   // the filter packed for MFMA (K+1 -> 3F, or 2(K+1) for BF16)
  const void* h;
  const void* v_in;
  const void* s_in;    // s before the message (may equal s)
  void* s;             // s after the message
  void* v_out;
  int v_zero;          // v_in is all zero (the first layer): its terms vanish
  // filter without its bias column (filt_mma is then the K -> 3F filter and
  // einfo[3] holds f_c): the epilogue adds f_c b_f, the sender comes from col
  int nb;
  const int32_t* col;
  const void* fbias;   // b_f [3F], accumulation type
  // (FP64, Gaussian basis, without the bias column) basis rows are
  // (g_0 f_c, exp(d / Delta - 1/2)) per edge and the kernel forms the
  // Gaussians itself; the
  // host sets it only where h and v_in are smaller than 4 GiB (the 8-k-block
  // kernel gathers from them with 32-bit byte offsets)
  int rg;
  // (FP64) room for the workgroups' LDS filter images (MSG64_IMAGE_BYTES),
  // or null
  void* img;
  long long E;         // edges of the graph (the FP64 receiver block size)
};

constexpr int MSG_RB = 4;   // receivers per workgroup (MSG_RB < 64)

// An int32 carried in an accumulation-type slot: its bits in a float, its
// value in a double.
template <class A>
__device__ __forceinline__ A index_to_acc(int j) {
  if constexpr (sizeof(A) == 4) return __int_as_float(j);
  else return (A)j;
}
__device__ __forceinline__ int acc_to_index(float x) { return __float_as_int(x); }
__device__ __forceinline__ int acc_to_index(double x) { return (int)x; }

// Once per forward: geometry and radial basis of every edge.
//   r = (x_j - x_i) + (n0 a + n1 b) + n2 c  (FP64),  d = |r|,  rhat = r / d,
//   f_c = (cos(pi d / r_c) + 1) / 2,  g_k = exp(-gamma (d - k Delta)^2).
// Edge e's geometry and basis row into g (LDS), its rhat and sender into einfo.
template <class P, bool NB, bool RG>
__device__ __forceinline__ void edge_row(long long e, int K, int kcols, double rc, int rbf, double gamma,
                                         double delta, const int32_t* __restrict__ recv,
                                         const int32_t* __restrict__ col, const int32_t* __restrict__ shift,
                                         const int32_t* __restrict__ atom_struct,
                                         const double* __restrict__ pos, const double* __restrict__ cell,
                                         typename P::T* g, typename P::A* __restrict__ einfo) {
  using A = typename P::A;
  constexpr bool SPLIT = P::KC == 32;
  const int i = recv[e], j = col[e], sh = shift[e];
  const double* Cl = cell + 9 * atom_struct[i];
  const double n0 = (double)(int8_t)(sh & 0xff), n1 = (double)(int8_t)((sh >> 8) & 0xff),
               n2 = (double)(int8_t)((sh >> 16) & 0xff);
  const double rx = (pos[3 * j] - pos[3 * i]) + ((n0 * Cl[0] + n1 * Cl[3]) + n2 * Cl[6]);
  const double ry = (pos[3 * j + 1] - pos[3 * i + 1]) + ((n0 * Cl[1] + n1 * Cl[4]) + n2 * Cl[7]);
  const double rz = (pos[3 * j + 2] - pos[3 * i + 2]) + ((n0 * Cl[2] + n1 * Cl[5]) + n2 * Cl[8]);
  const double d = sqrt(rx * rx + ry * ry + rz * rz);
  const double inv = 1.0 / d;
  A* o = einfo + 4 * e;
  o[0] = (A)(rx * inv);
  o[1] = (A)(ry * inv);
  o[2] = (A)(rz * inv);
  const A dd = (A)d;
  const A fc = (A)(d < rc ? 0.5 * (cos(d * (3.14159265358979323846 / rc)) + 1.0) : 0.0);
  // without the bias column the edge info carries f_c instead of the sender
  // (which the kernels then read from the CSR)
  o[3] = NB ? fc : index_to_acc<A>(j);           // the sender index, bit-exact
  if constexpr (RG) {
    // the message kernel forms g_k f_c from (g_0 f_c, exp(d / Delta - 1/2))
    // (the record gauss_row reads)
    const double u = d / delta;
    g[0] = P::st((A)(exp(-0.5 * u * u) * fc));
    g[1] = P::st((A)exp(u - 0.5));
    for (int k = 2; k < kcols; ++k) g[k] = P::st(0);
    return;
  }
  // each value once; BF16 also writes its remainder term at KW + k
  const int KW = NB ? K : K + 1;                 // columns of one term
  for (int k = 0; k < KW; ++k) {
    A val = fc;
    if (k < K && rbf == 0) {                     // Gaussian
      const A t = dd - (A)(k * delta);
      val = P::ex(-(A)gamma * t * t) * fc;
    } else if (k < K) {                          // Bessel: sin(n pi d / r_c) / d
      const A arg = (A)((k + 1) * (3.14159265358979323846 / rc)) * dd;
      val = (sizeof(A) == 8 ? (A)sin((double)arg) : (A)sinf((float)arg)) / dd * fc;
    }
    g[k] = P::st(val);
    if constexpr (SPLIT) g[KW + k] = P::st(val - P::ld(P::st(val)));
  }
  for (int k = SPLIT ? 2 * KW : KW; k < kcols; ++k) g[k] = P::st(0);
}

// A workgroup of EP_THREADS edges builds its rows in LDS (one row per
// thread), then writes the block's contiguous slice of the basis with
// 16-byte stores (the rows are 48-320 bytes: written per thread they would
// scatter one element per lane per store).
constexpr int EP_THREADS = 64;   // one wave: <= 35 KiB of LDS at the largest row

template <class P, bool NB, bool RG>
__global__ void __launch_bounds__(EP_THREADS) k_edge_prep(long long E, int K, int kcols, double rc, int rbf,
                                                  double gamma, double delta,
                                                  const int32_t* __restrict__ recv,
                                                  const int32_t* __restrict__ col,
                                                  const int32_t* __restrict__ shift,
                                                  const int32_t* __restrict__ atom_struct,
                                                  const double* __restrict__ pos,
                                                  const double* __restrict__ cell,
                                                  typename P::T* __restrict__ basis,
                                                  typename P::A* __restrict__ einfo) {
  using T = typename P::T;
  extern __shared__ __attribute__((aligned(16))) unsigned char ep_smem[];
  const long long e0 = blockIdx.x * (long long)EP_THREADS;
  const long long e = e0 + threadIdx.x;
  const long long rows = (E + 16 - e0) < EP_THREADS ? (E + 16 - e0) : EP_THREADS;
  T* g = (T*)ep_smem + (size_t)threadIdx.x * kcols;
  // rows E .. E+15 are zero (read by partial chunks)
  if (e < E) edge_row<P, NB, RG>(e, K, kcols, rc, rbf, gamma, delta, recv, col, shift, atom_struct, pos, cell, g, einfo);
  else if (e < E + 16)
    for (int k = 0; k < kcols; ++k) g[k] = P::st(0);
  __syncthreads();
  // kcols * sizeof(T) is a multiple of 16, so the slice is whole uint4s
  const size_t n16 = (size_t)rows * kcols * sizeof(T) / 16;
  const uint4* src = (const uint4*)ep_smem;
  uint4* dst = (uint4*)(basis + (size_t)e0 * kcols);
  for (size_t x = threadIdx.x; x < n16; x += EP_THREADS) dst[x] = src[x];
}


// FP64, per layer.  SPLIT workgroups share RB consecutive receivers,
// each owning NGW groups of 32 channels; the workgroup's NS streams of NGW
// waves split those receivers, wave w of a stream owning channel group w.
// The group's filter columns are staged in LDS once per workgroup (shared
// by its streams), which leaves each wave the registers for two waves per
// SIMD: one wave's loads run under the other's MFMAs.  (FP64 MFMAs and FP64
// vector instructions take turns at issue on this chip, equal peaks, so the
// kernel's vector instruction count adds to its time directly.)
//
// A wave's channel group is two MFMA column tiles whose columns interleave:
// column c of tile q is channel 32 g + 2 c + q, so a lane's two accumulator
// columns are adjacent channels and each sender gather is one 16-byte load
// per lane.  The order of the filter input is permuted alike on both MFMA
// operands: k-blocks 2p and 2p + 1 take inputs 8p + 2 kk and 8p + 2 kk + 1
// at k-group kk, so one 16-byte load per lane fetches two basis fragments
// (and one 16-byte LDS read two filter fragments).  The vector-memory
// address unit costs about the same per instruction at 8 and 16 bytes per
// lane: halving the instructions is what lets the MFMAs keep busy.
//
// A stream's receivers form one sequence of 16-edge chunks: with in-kernel
// Gaussians (RG) the stream's edges cut into chunks regardless of where
// receivers end, otherwise each receiver's edges on their own (a receiver
// without edges still takes one, empty, so that its row is written).  Per
// chunk the wave issues the sender gathers, prefetches the next chunk's
// edge info (and basis record), runs the filter MFMAs and combines their
// accumulators (row = edge, col = channel) with the gathered features
// directly; a receiver's per-lane partial sums are reduced across the four
// row groups of the wavefront after its last edge.
// Receivers per workgroup: 32, or 16 for the in-kernel-Gaussian kernels on
// batches of at least MSG_RB16_DEGREE edges per receiver, whose streams of
// 16 receivers already hold many chunks and whose fewer receivers in flight
// per XCD keep more sender rows in its L2 (measured: bulk periodic batch,
// 72 edges per receiver, message -4.3 %; screening batch, 30, -0.4 %;
// molecules, 15, 2.6 % slower).
constexpr int MSG_RB64 = 32;
constexpr int MSG_RB16_DEGREE = 24;

// Lane n of each 16-lane row, broadcast to its row (DPP row_newbcast).
__device__ __forceinline__ int row_bcast(int x, int n) {
  // (every lane reads a lane of its own row, so no lane keeps an old value)
  switch (n) {
    case 0: return __builtin_amdgcn_mov_dpp(x, 0x150, 0xf, 0xf, true);
    case 1: return __builtin_amdgcn_mov_dpp(x, 0x151, 0xf, 0xf, true);
    case 2: return __builtin_amdgcn_mov_dpp(x, 0x152, 0xf, 0xf, true);
    default: return __builtin_amdgcn_mov_dpp(x, 0x153, 0xf, 0xf, true);
  }
}
__device__ __forceinline__ double row_bcast(double x, int n) {
  const long long v = __double_as_longlong(x);
  const int lo = row_bcast((int)(v & 0xffffffff), n), hi = row_bcast((int)(v >> 32), n);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// A raw buffer resource over an array of `bytes` bytes: loads at byte
// offsets from a 32-bit lane offset plus a scalar offset (no 64-bit address
// arithmetic per lane); a load past the end returns zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)(uint32_t)bytes, 0x00020000);
}
template <class V>
__device__ __forceinline__ V buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t off, int soff = 0) {
  return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0));
}

template <int KBM>
__device__ __forceinline__ int msg_kcol(int kb, int kk) {
  return kb < KBM / 2 * 2 ? 8 * (kb >> 1) + 2 * kk + (kb & 1) : 4 * kb + kk;
}

// The Gaussian basis of one MFMA A-operand lane: ga[kb] = f_c g_k with
// g_k = exp(-(u - k)^2 / 2), u = d / Delta, at the lane's inputs
// k = msg_kcol(kb, kk), from the edge's record (a, b).  The inputs follow
// from g(k + m) = g(k) exp(m (u - k) - m^2 / 2):
//   g(k0 + 1) = g(k0) t,  t = exp(u - k0 - 1/2),
//   g(k + 8) = g(k) t^8 e^-28 e^-8 (k - k0)   (k0 = 2 kk, the lane's first input).
// The record is (g_0 f_c, t_0 = exp(u - 1/2)), so the kernel takes no
// exponential: t = t_0 e^-k0 and g(k) = g_0 t_0^k e^-k (k - 1) / 2 for the
// first input k0 and, with an odd number of k-blocks (5), for the last
// input k = 16 + kk.  With u of at most 35 (K <= 36) every factor and every
// partial product of the recurrences stays inside FP64's normal range, and
// so do those of the last input (u < 19, t_0^19 < e^352, g_0 > e^-181,
// e^-171 at the least), so nothing underflows that the direct formula
// would keep.
template <int KBM>
__device__ __forceinline__ void gauss_row(double a, double b, int kk, double (&ga)[KBM]) {
  constexpr double EM8 = 0x1.5fc21041027adp-12, EM28 = 0x1.853f01d6d53bap-41, EM64 = 0x1.969d47321e4ccp-93;
  // a = g_0 f_c (zero for a masked row), b = t_0
  constexpr double EM1 = 0x1.78b56362cef38p-2, EM2 = 0x1.152aaa3bf81ccp-3, EM4 = 0x1.2c155b8213cf4p-6,
                   EM6 = 0x1.44e51f113d4d6p-9, EM15 = 0x1.4875ca227ec38p-22;
  const double b2 = b * b, b4 = b2 * b2;
  const double p = (kk & 1 ? b2 : 1.0) * (kk & 2 ? b4 : 1.0);     // t_0^(2 kk)
  double ea = a * p * (kk == 0 ? 1.0 : kk == 1 ? EM1 : kk == 2 ? EM6 : EM15);
  const double t = b * (kk == 0 ? 1.0 : kk == 1 ? EM2 : kk == 2 ? EM4 : EM6);
  double eb = ea * t;                            // g(k0 + 1) f_c
  const double t2 = t * t, t4 = t2 * t2;
  double ra = t4 * t4 * EM28;                    // g(k0 + 8) / g(k0)
#pragma unroll
  for (int p = 0; p < KBM / 2; ++p) {
    if (p > 0) {
      ea *= ra;
      eb *= ra * EM8;
      ra *= EM64;
    }
    ga[2 * p] = ea;
    ga[2 * p + 1] = eb;
  }
  if constexpr (KBM & 1) {
    // k = 16 + kk: g_0 f_c t_0^16 t_0^kk e^-k (k - 1) / 2
    static_assert(KBM == 5, "odd k-block counts: 5");
    constexpr double EM120 = 0x1.d606847fc727ap-174, EM136 = 0x1.bbb5da5f7c823p-197,
                     EM153 = 0x1.342faee475139p-221, EM171 = 0x1.3afca550dd136p-247;
    const double b8 = b4 * b4, b16 = b8 * b8;
    const double q = (kk & 1 ? b : 1.0) * (kk & 2 ? b2 : 1.0);      // t_0^kk
    ga[KBM - 1] = a * b16 * q * (kk == 0 ? EM120 : kk == 1 ? EM136 : kk == 2 ? EM153 : EM171);
  }
}

// channel groups per workgroup: the LDS holds 6 (KBM + 1) / 2 KiB per group
template <int F, int KBM>
constexpr int msg64_groups() {
  return F / 32 < (KBM <= 12 ? 4 : 2) ? F / 32 : (KBM <= 12 ? 4 : 2);
}

typedef double msg_d2 __attribute__((ext_vector_type(2)));

// The LDS filter image of a k_message workgroup owning channel half `half`:
// entries below NGW 6 NP 64 are the B-fragment pairs
// [group][q][part][k-block pair][lane], the rest (without the bias column)
// the b_f pairs [group][part][lane % 16] at a lane's two channels.
template <int F, int NGW, int KBM, bool NB>
constexpr int msg64_image_size() {
  return NGW * 6 * ((KBM + 1) / 2) * 64 + (NB ? NGW * 3 * 16 : 0);
}
template <int F, int NGW, int KBM>
__device__ __forceinline__ msg_d2 msg64_image_entry(const MsgArgs& a, int half, int x) {
  constexpr int NP = (KBM + 1) / 2, NBF = NGW * 6 * NP * 64;
  if (x < NBF) {
    const double* Wf = (const double*)a.filt_mma.w;
    const int l = x & 63, p = (x >> 6) % NP, qp = (x >> 6) / NP % 6, g = (x >> 6) / NP / 6;
    // packed fragment element (row n, input k): tile n / 16, k-block k / 4,
    // lane n % 16 + 16 (k % 4)
    const int n = qp % 3 * F + 32 * (half * NGW + g) + 2 * (l & 15) + qp / 3;
    double v[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int kb = 2 * p + hh, k = msg_kcol<KBM>(kb, l >> 4);
      v[hh] = kb < KBM ? Wf[((size_t)((n >> 4) * KBM + (k >> 2)) * 64 + (n & 15) + 16 * (k & 3))] : 0.0;
    }
    return msg_d2{v[0], v[1]};
  }
  x -= NBF;
  const int c = x % 16, part = x / 16 % 3, g = x / 48;
  const double* fb = (const double*)a.fbias + part * F + 32 * (half * NGW + g) + 2 * c;
  return msg_d2{fb[0], fb[1]};
}

// Once per layer: every channel half's image (blockIdx.y = half), so that
// each message workgroup fills its LDS with 16-byte copies instead of
// gathering scattered 8-byte fragments (bulk periodic message -0.7 %).
template <int F, int NGW, int KBM, bool NB>
__global__ void __launch_bounds__(256) k_msg64_image(MsgArgs a, msg_d2* __restrict__ img) {
  constexpr int IMG = msg64_image_size<F, NGW, KBM, NB>();
  const int half = blockIdx.y;
  for (int x = blockIdx.x * 256 + threadIdx.x; x < IMG; x += gridDim.x * 256)
    img[(size_t)half * IMG + x] = msg64_image_entry<F, NGW, KBM>(a, half, x);
}

template <class P, int F, int NGW, int NS, int KBM, bool V0, bool NB, bool RG, int RB>
__global__ void __launch_bounds__(64 * NGW * NS, 2) k_message(MsgArgs a) {
  using T = typename P::T;
  using C = typename P::C;
  static_assert(sizeof(T) == 8, "the paired-channel layout is the FP64 kernel's");
  static_assert(!RG || (NB && KBM <= 9), "Gaussians formed in the kernel: no bias column, K <= 36");
  // basis values a lane keeps per chunk: its KBM inputs, or the edge's
  // record (g_0 f_c, t_0)
  constexpr int NGA = RG ? 2 : KBM;
  typedef double d2 __attribute__((ext_vector_type(2)));
  constexpr int NG = F / 32, SPLIT = NG / NGW, NP = (KBM + 1) / 2, RBS = RB / NS;
  static_assert(NG % NGW == 0 && RB % NS == 0 && RBS < 64, "workgroup shape");
  constexpr int kcols = KBM * P::KC;  // the filter input is padded to KBM k-blocks
  // [group][q][part][k-block pair][lane]: the two B fragments of a pair;
  // without the bias column, b_f [group][part][lane % 16] at the lane's two
  // channels
  __shared__ d2 bsh[NGW * 6 * NP * 64];
  __shared__ d2 bias_sh[NB ? NGW * 3 * 16 : 1];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kk = lane >> 4, gw = wave % NGW, st = wave / NGW;
  // Workgroups are dealt round-robin to the 8 XCDs.  Renumber them so each
  // XCD walks one contiguous range of receivers: a molecule's receivers then
  // share one L2, which serves the repeated gathers of its sender rows, and
  // the SPLIT workgroups of a receiver block read its basis from one L2.
  const int per_xcd = gridDim.x / 8;
  const int lb = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int ib = (lb / SPLIT) * RB, half = lb % SPLIT;
  if (ib >= a.N) return;                       // the whole workgroup
  {
    // the workgroup's filter image: copied from the layer's image where the
    // host wrote one, else gathered here
    constexpr int NBF = NGW * 6 * NP * 64, IMG = msg64_image_size<F, NGW, KBM, NB>();
    const d2* im = a.img ? (const d2*)a.img + (size_t)half * IMG : nullptr;
    for (int x = threadIdx.x; x < NBF; x += NGW * NS * 64)
      bsh[x] = a.img ? im[x] : msg64_image_entry<F, NGW, KBM>(a, half, x);
    if constexpr (NB)
      for (int x = threadIdx.x; x < NGW * 3 * 16; x += NGW * NS * 64)
        bias_sh[x] = a.img ? im[NBF + x] : msg64_image_entry<F, NGW, KBM>(a, half, NBF + x);
  }
  __syncthreads();                             // (the only barrier)
  const int i0 = ib + st * RBS;
  if (i0 >= a.N) return;
  const int i1 = min(a.N, i0 + RBS);
  const int ch = 32 * (half * NGW + gw) + 2 * col;   // this lane's channels ch, ch + 1
  const d2* bw = bsh + gw * 6 * NP * 64 + lane;
  const d2* bb = bias_sh + gw * 3 * 16 + col;
  const T* h = (const T*)a.h;
  const T* vin = (const T*)a.v_in;
  const T* basis = (const T*)a.basis;
  const double* einfo = (const double*)a.einfo;
  const T* sin = (const T*)a.s_in;
  T* s = (T*)a.s;
  T* vout = (T*)a.v_out;
  // The sender gathers through buffer resources, and f_c masked once when
  // the edge info is loaded (not per accumulator row), where that was
  // measured faster: 8 k-blocks (-1.3 % and -1.8 % on the bulk periodic
  // batch; with 5 the kernel ran 3.5 % and 3.4 % slower)
  constexpr bool BUF = RG && KBM == 8;
  const size_t hbytes = (size_t)a.N * 3 * F * sizeof(T);
  const __amdgpu_buffer_rsrc_t r_h = buf_rsrc(h, hbytes), r_v = buf_rsrc(vin, hbytes);
  // the stream's row_ptr slice, one load per lane, read back by readlane
  const int rp_lane = a.row_ptr[i0 + min(lane, i1 - i0)];
  auto rp = [&](int i) { return __builtin_amdgcn_readlane(rp_lane, i - i0); };
  // Chunks of 16 edges.  With PACK the stream's edges (its receivers' CSR
  // rows are consecutive) form one sequence of chunks, so only the last is
  // partial and a chunk may hold the ends and starts of several receivers;
  // otherwise each receiver's row is a sequence of its own (one empty chunk
  // for a receiver without edges, so that its row is written).
  constexpr bool PACK = RG;
  const int e_begin = rp(i0), e_end = rp(i1);
  int nck = 0;
  if constexpr (PACK) nck = (e_end - e_begin + 15) / 16;
  else
    for (int i = i0; i < i1; ++i) nck += max(1, (rp(i + 1) - rp(i) + 15) / 16);
  struct Ck { int i, c0, cnt; bool last; };   // wave-uniform (i, last: without PACK)
  auto make = [&](int i, int c0) {
    const int eb = rp(i + 1);
    return Ck{i, c0, max(0, min(16, eb - c0)), c0 + 16 >= eb};
  };
  auto make_packed = [&](int k) {
    const int c0 = e_begin + 16 * k;
    return Ck{0, c0, min(16, e_end - c0), false};
  };
  auto next = [&](const Ck& c) {
    return !c.last ? make(c.i, c.c0 + 16) : c.i + 1 < i1 ? make(c.i + 1, rp(c.i + 1)) : c;
  };
  // Edge info: lane 16 kk + j holds (rhat_x, rhat_y) and (rhat_z, sender)
  // of chunk row 4 (j % 4) + kk (without the bias column (rhat_z, f_c), the
  // sender from the CSR column), so accumulator row 4 ii + kk of every lane
  // of the 16-lane row kk sits in that row's lane ii, and a DPP row
  // broadcast hands it over.  Rows past the chunk's end take its first edge
  // (a valid sender) and get a zero basis row and f_c, hence a zero filter,
  // so no gather needs a branch; an empty chunk gathers the receiver's own
  // row.
  struct Raw { d2 xy, ze; int j; };
  auto load_raw = [&](const Ck& c, Raw& o) {
    if (PACK || c.cnt > 0) {
      const int row = 4 * (col & 3) + kk;
      const size_t e = c.c0 + (row < c.cnt ? row : 0);
      const double* ei = einfo + 4 * e;
      o.xy = *(const d2*)ei;
      o.ze = *(const d2*)(ei + 2);
      o.j = NB ? a.col[e] : 0;
      if constexpr (BUF) o.ze.y = row < c.cnt ? o.ze.y : 0.0;   // f_c, zero past the chunk's end
    } else {
      o.xy = d2{0.0, 0.0};
      o.ze = d2{0.0, NB ? 0.0 : (double)c.i};
      o.j = c.i;
    }
  };
  auto load_ga = [&](const Ck& c, T (&Ga)[NGA]) {
    if constexpr (RG) {
      const d2 t = *(const d2*)(basis + 2 * (size_t)(c.c0 + col));   // rows E .. E + 15 exist
      Ga[0] = t.x;
      Ga[1] = t.y;
      return;
    }
    const T* gp = basis + (size_t)(c.c0 + col) * kcols;   // rows E .. E + 15 exist
#pragma unroll
    for (int p = 0; p < KBM / 2; ++p) {
      const d2 t = *(const d2*)(gp + 8 * p + 2 * kk);
      Ga[2 * p] = t.x;
      Ga[2 * p + 1] = t.y;
    }
    if constexpr (KBM & 1) Ga[KBM - 1] = gp[4 * (KBM - 1) + kk];
  };
  auto filter = [&](const Ck& c, const T (&Ga)[NGA], const Raw& in, C (&w)[2][3]) {
    T ga[KBM];
    if constexpr (RG) {
      // a masked row (past the chunk's end) gets a zero f_c, hence zeros
      const bool live = col < c.cnt;
      gauss_row<KBM>(live ? Ga[0] : 0.0, Ga[1], kk, ga);
    } else {
#pragma unroll
      for (int kb = 0; kb < KBM; ++kb) ga[kb] = col < c.cnt ? Ga[kb] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int part = 0; part < 3; ++part)
        for (int r = 0; r < 4; ++r) w[q][part][r] = 0;
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          // with v_j = 0 the v part of the filter meets nothing
          if (V0 && part == 1) continue;
          const d2 b = bw[((q * 3 + part) * NP + p) * 64];
          w[q][part] = P::mfma(ga[2 * p], b.x, w[q][part]);
          if (2 * p + 1 < KBM) w[q][part] = P::mfma(ga[2 * p + 1], b.y, w[q][part]);
        }
    // Keep the LDS reads just ahead of their MFMAs (hoisted all at once
    // they would take 30 register pairs): a pair's reads go out between the
    // previous pair's MFMAs.
    constexpr int NBR = V0 ? 4 : 6;            // B reads (and MFMAs) per k-block
    __builtin_amdgcn_sched_group_barrier(0x100, NBR, 0);
#pragma unroll
    for (int p = 0; p < KBM / 2; ++p) {
      __builtin_amdgcn_sched_group_barrier(0x008, NBR, 0);
      if (p + 1 < NP) __builtin_amdgcn_sched_group_barrier(0x100, NBR, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, NBR, 0);
    }
    if constexpr (KBM & 1) __builtin_amdgcn_sched_group_barrier(0x008, NBR, 0);
    if constexpr (NB) {
      // w = f_c (W_f g + b_f): the bias times the rows' f_c (zero past the
      // chunk's end)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const double fc = BUF ? row_bcast(in.ze.y, ii) : P::row(lane, ii) < c.cnt ? row_bcast(in.ze.y, ii) : 0.0;
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          if (V0 && part == 1) continue;
          const d2 b = bb[part * 16];
          w[0][part][ii] = fma(fc, b.x, w[0][part][ii]);
          w[1][part][ii] = fma(fc, b.y, w[1][part][ii]);
        }
      }
    }
  };
  struct Gath { d2 hs[4], hr[4], hv[4], vj[4][3]; };
  auto gather = [&](const Raw& in, Gath& G) {
    const int j_lane = NB ? in.j : acc_to_index(in.ze.y);
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      if constexpr (BUF) {
        constexpr int FB = F * (int)sizeof(T);
        const uint32_t hb = (uint32_t)row_bcast(j_lane, ii) * (uint32_t)(3 * FB) + (uint32_t)ch * (uint32_t)sizeof(T);
        G.hs[ii] = buf_ld16<d2>(r_h, hb);
        G.hr[ii] = buf_ld16<d2>(r_h, hb, 2 * FB);
        if constexpr (!V0) {
          G.hv[ii] = buf_ld16<d2>(r_h, hb, FB);
#pragma unroll
          for (int c = 0; c < 3; ++c) G.vj[ii][c] = buf_ld16<d2>(r_v, hb, c * FB);
        }
        continue;
      }
      const size_t hb = (size_t)row_bcast(j_lane, ii) * 3 * F + ch;
      G.hs[ii] = *(const d2*)(h + hb);
      G.hr[ii] = *(const d2*)(h + hb + 2 * F);
      if constexpr (!V0) {
        G.hv[ii] = *(const d2*)(h + hb + F);
#pragma unroll
        for (int c = 0; c < 3; ++c) G.vj[ii][c] = *(const d2*)(vin + hb + c * F);
      }
    }
  };
  // Chunk rows [r0, r1) into the running receiver's per-lane sums (every
  // row where FULL; rows past the chunk's end carry a zero filter); rows
  // outside the range add exact zeros.
  double acc_s[2] = {0.0, 0.0}, acc_v[2][3] = {{0.0, 0.0, 0.0}, {0.0, 0.0, 0.0}};
  auto consume = [&](const C (&w)[2][3], const Gath& G, const Raw& in, auto full, int r0, int r1) {
    constexpr bool FULL = decltype(full)::value;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const double rh[3] = {row_bcast(in.xy.x, ii), row_bcast(in.xy.y, ii), row_bcast(in.ze.x, ii)};
      const int row = P::row(lane, ii);
      const double m = FULL || (row >= r0 && row < r1) ? 1.0 : 0.0;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        acc_s[q] = fma(G.hs[ii][q], FULL ? w[q][0][ii] : w[q][0][ii] * m, acc_s[q]);
        const double pr = G.hr[ii][q] * (FULL ? w[q][2][ii] : w[q][2][ii] * m);
        if constexpr (!V0) {
          const double pv = G.hv[ii][q] * (FULL ? w[q][1][ii] : w[q][1][ii] * m);
#pragma unroll
          for (int c = 0; c < 3; ++c) acc_v[q][c] = fma(G.vj[ii][c][q], pv, acc_v[q][c]);
        }
#pragma unroll
        for (int c = 0; c < 3; ++c) acc_v[q][c] = fma(rh[c], pr, acc_v[q][c]);
      }
    }
  };
  // Receiver i's sums over the wave into s and v (then zeroed).
  auto finish = [&](int i) {
    const size_t iv = (size_t)i * 3 * F + ch;
    const d2 s_old = *(const d2*)(sin + (size_t)i * F + ch);
    d2 v_old[3];
#pragma unroll
    for (int c = 0; c < 3; ++c) v_old[c] = V0 ? d2{0.0, 0.0} : *(const d2*)(vin + iv + c * F);
#pragma unroll
    for (int q = 0; q < 2; ++q)
      for (int off = 16; off < 64; off *= 2) {
        acc_s[q] += __shfl_xor(acc_s[q], off);
#pragma unroll
        for (int c = 0; c < 3; ++c) acc_v[q][c] += __shfl_xor(acc_v[q][c], off);
      }
    if (lane < 16) {
      *(d2*)(s + (size_t)i * F + ch) = d2{s_old.x + acc_s[0], s_old.y + acc_s[1]};
#pragma unroll
      for (int c = 0; c < 3; ++c)
        *(d2*)(vout + iv + c * F) = d2{v_old[c].x + acc_v[0][c], v_old[c].y + acc_v[1][c]};
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) acc_s[q] = acc_v[q][0] = acc_v[q][1] = acc_v[q][2] = 0.0;
  };

  // Chunk k: its gathers go out first, then the next chunk's edge info, then
  // its filter MFMAs and the combination.  Two chunks alternate the roles of
  // the prefetch buffers, so nothing is copied.
  Gath G;
  C w[2][3];
  // (the next chunk's basis rows are prefetched too where the registers
  // allow it, up to 9 k-blocks)
  constexpr bool PF = RG || KBM <= 9;
  int ir = i0;                                 // with PACK: the receiver being summed
  auto step = [&](int k, Ck& cur, const Raw& in_cur, Raw& in_nxt, T (&ga_cur)[NGA], T (&ga_nxt)[NGA]) {
    gather(in_cur, G);
    if constexpr (!PF) load_ga(cur, ga_cur);
    const bool more = k + 1 < nck;
    const Ck nx = PACK ? make_packed(k + 1) : next(cur);
    if (more) {
      load_raw(nx, in_nxt);
      if constexpr (PF) load_ga(nx, ga_nxt);
    }
    filter(cur, ga_cur, in_cur, w);
    if constexpr (PACK) {
      // the receivers that end in this chunk (those without edges too),
      // then the one that runs on into the next
      const int c1 = cur.c0 + cur.cnt;
      if (rp(ir + 1) > c1) {
        consume(w, G, in_cur, std::true_type{}, 0, 16);
      } else {
        int r0 = 0;
        while (ir < i1 && rp(ir + 1) <= c1) {
          const int r1 = rp(ir + 1) - cur.c0;
          if (r1 > r0) consume(w, G, in_cur, std::false_type{}, r0, r1);
          finish(ir);
          ++ir;
          r0 = max(r0, r1);
        }
        if (ir < i1 && r0 < cur.cnt) consume(w, G, in_cur, std::false_type{}, r0, cur.cnt);
      }
    } else {
      consume(w, G, in_cur, std::true_type{}, 0, 16);
      if (cur.last) finish(cur.i);
    }
    cur = nx;
    return more;
  };
  Ck c = PACK ? make_packed(0) : make(i0, e_begin);
  Raw inA, inB;
  T gaA[NGA], gaB[NGA];
  if (nck > 0) {
    load_raw(c, inA);
    if constexpr (PF) load_ga(c, gaA);
    for (int k = 0;; k += 2) {
      if (!step(k, c, inA, inB, gaA, gaB)) break;
      if (!step(k + 1, c, inB, inA, gaB, gaA)) break;
    }
  }
  if constexpr (PACK)
    for (; ir < i1; ++ir) finish(ir);         // receivers without edges at the end
}

// --------------------------------------------------------------- update ----
// Tile of 16 RT atoms.  U[c] = WU v[c], V[c] = WV v[c] for c = x, y, z, the
// three components staged in LDS together so that each weight fragment
// serves all three; U, |V|^2 and <U, V> stay in the registers of the wave
// that owns the feature tile.  Then
// a = W2a silu(W1a [s; |V|] + b1a) + b2a, with each wave computing the
// a_vv / a_sv / a_ss column tiles of its own feature tiles, so the final
//   v[c] += a_vv U[c],  s += a_sv <U, V> + a_ss
// needs no exchange.  Optionally the next layer's phi follows on the new s.
struct UpdArgs {
  int N;
  const void* s;   // s and v after the message
  const void* v;
  void* s_out;     // after the update (may equal s, v)
  void* v_out;
  void* h;
  DenseDev uv, upd1, upd2, phi1, phi2;
  // with SAVE: U, V per component [N][3][2F], the gate's pre-activation
  // [N][F] and [a_vv | a_sv] [N][2F] for the reverse pass
  void* save_uv;
  void* save_z;
  void* save_a;
};

// Waves per SIMD the update kernel is compiled for: four at F = 128 (three
// in FP64), where the registers allow it without spilling; at F >= 256 the
// measured best is two (one in FP64, whose accumulators need the whole
// register file).
template <class P, int F>
constexpr int update_waves() {
  return F == 128 ? (P::PREC == PAINN_FP64 ? 3 : 4) : F == 64 ? (P::PREC == PAINN_FP64 ? 2 : 3) : (P::PREC == PAINN_FP64 ? 1 : 2);
}

// Waves of an update workgroup: 4 at F = 64, 8 at F = 128 (one feature tile
// each), F / 32 above (two tiles each): the LDS tile allows few workgroups
// per CU, so the waves of one workgroup must bring the occupancy (measured
// faster at every width).
template <class P, int F>
constexpr int update_nw() {
  return F < 128 ? 4 : F == 128 ? 8 : F / 32;
}

// Row tiles (16 atoms each) of an update workgroup, as measured fastest per
// shape: two below F = 256 (one in FP64 at F = 128), one at F >= 256 except
// FP32 at F = 256 and BF16 at F = 384 (update -5 % and -31 % with two; BF16
// at F = 256 ran 13 % slower with two, FP32 at F = 384 the same).
template <class P, int F>
constexpr int update_rt() {
  if constexpr (F >= 256)
    return (P::PREC == PAINN_FP32 && F == 256) || (P::PREC == PAINN_BF16 && F == 384) ? 2 : 1;
  else
    return P::PREC == PAINN_FP64 && F == 128 ? 1 : 2;
}

// Components of v that go through the U/V weights together: three, except
// where four FP32 waves per SIMD leave too few registers for their
// accumulators (one at a time there).
template <class P, int F>
constexpr int uv_comps() {
  return P::PREC == PAINN_FP32 && update_waves<P, F>() >= 4 ? 1 : 3;
}

// The saving variant (forces) stores U, V, z, a as it goes and runs at no
// more than two waves per SIMD (the stores' addresses need registers).
template <class P, int F, int RT, bool FUSE_PHI, bool SAVE>
__global__ void __launch_bounds__((64 * update_nw<P, F>()))
__attribute__((amdgpu_waves_per_eu(SAVE && update_waves<P, F>() > 3 ? 3 : update_waves<P, F>())))
k_update(UpdArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int NFT = F / 16;        // feature tiles
  constexpr int NW = update_nw<P, F>();
  constexpr int FTW = NFT / NW;      // per wave
  constexpr int TM = 16 * RT;        // atoms per workgroup
  constexpr int LD1 = F + P::PAD, LD2 = 2 * F + P::PAD;
  // The UVC components of v side by side for the U/V products; [s ; |V|]
  // and the MLP hidden layer (with UVC = 3 in the same space, after them).
  constexpr int UVC = uv_comps<P, F>();
  static_assert(3 * LD1 >= LD2 + LD1, "LDS phases");
  __shared__ __attribute__((aligned(16))) T smem[3 * TM * LD1];
  T* SN = smem;                                   // [TM][LD2]
  T* H = smem + TM * LD2;                         // [TM][LD1]
  T* VS = UVC == 3 ? smem : H;                    // [UVC][TM][LD1]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t row0 = (size_t)blockIdx.x * TM;
  const int N = a.N;
  const T* s = (const T*)a.s;
  const T* v = (const T*)a.v;
  // without SAVE the update runs in place (s_out == s, v_out == v): one
  // pointer each, so the compiler sees that the loads and stores meet only
  // element by element
  T* s_out = SAVE ? (T*)a.s_out : (T*)a.s;
  T* v_out = SAVE ? (T*)a.v_out : (T*)a.v;
  C U[FTW][3][RT], nsq[FTW][RT], pd[FTW][RT];
  // With the three components staged together, each lane keeps the elements
  // of v its epilogue updates (read from LDS before that space is reused)
  // instead of reading them from global memory again, where the extra
  // registers cost no occupancy: FP64 at F = 256 and FP32 at F >= 256
  // (measured: update -1.4 % and -4.5 %; FP64 at F = 128 and BF16 lost a
  // wave per SIMD and ran 17 % and 38 % slower), not in the saving variants.
  constexpr bool VREG = UVC == 3 && !SAVE && F >= 256 && P::PREC != PAINN_BF16 &&
                        !(P::PREC == PAINN_FP64 && F >= 384);
  T vkeep[VREG ? FTW : 1][3][VREG ? RT : 1][4];
  for (int q = 0; q < FTW; ++q)
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) nsq[q][r][i] = pd[q][r][i] = 0;
  using D = dense_t<P>;   // operand form of the dense layers
  using Fd = typename D::Fr;
  constexpr int nkb = F / D::KC;
  // the multi-stream K loops (U/V, the gate's output layer) keep twice the
  // ring where that measured faster: FP64 at F >= 256 (update -1.9 % bulk
  // periodic, -3.2 % lead model; 1 % slower at F = 128) and BF16 at F = 256
  // (-3.4 % screening; FP32 at F >= 256 ran 1-2 % slower, BF16 at F = 384
  // the same)
  constexpr int RX = (P::PREC == PAINN_FP64 && F >= 256) || (P::PREC == PAINN_BF16 && F == 256) ? 2 : 1;
  const T* Wuv = (const T*)a.uv.w;
  if constexpr (UVC == 1) stage_rows<P, F, TM>(SN, LD2, s, F, row0, N);
  // UVC components against each weight fragment: the UVC RT row tiles of VS
  // (component c0 + cc, tile r at 16 (cc RT + r) rows) share its loads.
#pragma unroll
  for (int c0 = 0; c0 < 3; c0 += UVC) {
    if (UVC == 1) __syncthreads();
#pragma unroll
    for (int cc = 0; cc < UVC; ++cc)
      stage_rows<P, F, TM>(VS + cc * TM * LD1, LD1, v + (c0 + cc) * F, 3 * F, row0, N);
    __syncthreads();
    const T* xp = VS + (lane & 15) * LD1 + (lane >> 4) * D::KPL;
#pragma unroll
    for (int q = 0; q < FTW; ++q) {
      const int ft = wave + NW * q;
      C au[UVC * RT], av[UVC * RT];
      for (int r = 0; r < UVC * RT; ++r)
        for (int i = 0; i < 4; ++i) au[r][i] = av[r][i] = 0;
      const T* wu = Wuv + (size_t)ft * nkb * 64 * D::KPL + (size_t)lane * D::KPL;
      const T* wv = Wuv + (size_t)(NFT + ft) * nkb * 64 * D::KPL + (size_t)lane * D::KPL;
      kloop<D, nkb, ring_depth<D, 2, RX>(), 2, UVC * RT>(
          xp, LD1,
          [&](int kb, Fd* f) {
            f[0] = D::frag(wu + (size_t)kb * 64 * D::KPL);
            f[1] = D::frag(wv + (size_t)kb * 64 * D::KPL);
          },
          [&](int kb, const Fd* x, const Fd* f) {
#pragma unroll
            for (int j = 0; j < D::SUB; ++j)
#pragma unroll
              for (int r = 0; r < UVC * RT; ++r) {
                au[r] = D::mfma_sub(x[r], f[0], au[r], j);
                av[r] = D::mfma_sub(x[r], f[1], av[r], j);
              }
          });
#pragma unroll
      for (int cc = 0; cc < UVC; ++cc)
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          const int c = c0 + cc;
          const C& u = au[cc * RT + r];
          const C& w = av[cc * RT + r];
          U[q][c][r] = u;
          for (int i = 0; i < 4; ++i) {
            nsq[q][r][i] += w[i] * w[i];
            pd[q][r][i] += u[i] * w[i];
          }
          if constexpr (VREG)
            for (int i = 0; i < 4; ++i)
              vkeep[q][c][r][i] = VS[(cc * TM + r * 16 + P::row(lane, i)) * LD1 + ft * 16 + (lane & 15)];
          if constexpr (SAVE) {
            const int col = ft * 16 + (lane & 15);
            for (int i = 0; i < 4; ++i) {
              const size_t row = row0 + r * 16 + P::row(lane, i);
              if (row < (size_t)N) {
                T* o = (T*)a.save_uv + (row * 3 + c) * 2 * F;
                o[col] = P::st(u[i]);
                o[F + col] = P::st(w[i]);
              }
            }
          }
        }
    }
  }
  if constexpr (UVC == 3) {
    __syncthreads();                   // v's slices are dead: [s ; |V|] takes their place
    stage_rows<P, F, TM>(SN, LD2, s, F, row0, N);
  }
#pragma unroll
  for (int q = 0; q < FTW; ++q) {
    const int col = (wave + NW * q) * 16 + (lane & 15);
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i)
        SN[(r * 16 + P::row(lane, i)) * LD2 + F + col] = P::st(sqrt(nsq[q][r][i]));
  }
  __syncthreads();
  dense_tiles<P, RT, NW, 2 * F>(SN, LD2, a.upd1, [&](int ct, C* acc) {
    const int col = ct * 16 + (lane & 15);
    const A bias = ((const A*)a.upd1.b)[col];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) {
        H[(r * 16 + P::row(lane, i)) * LD1 + col] = P::st(silu<A>(acc[r][i] + bias));
        if constexpr (SAVE) {
          const size_t row = row0 + r * 16 + P::row(lane, i);
          if (row < (size_t)N) ((T*)a.save_z)[row * F + col] = P::st(acc[r][i] + bias);
        }
      }
  });
  __syncthreads();
  {
    constexpr int nkb2 = F / D::KC;
    const T* W2 = (const T*)a.upd2.w;
    const A* b2 = (const A*)a.upd2.b;
    const T* xp = H + (lane & 15) * LD1 + (lane >> 4) * D::KPL;
#pragma unroll
    for (int q = 0; q < FTW; ++q) {
      const int ft = wave + NW * q;
      C avv[RT], asv[RT], ass[RT];
      for (int r = 0; r < RT; ++r)
        for (int i = 0; i < 4; ++i) avv[r][i] = asv[r][i] = ass[r][i] = 0;
      const T* w0 = W2 + (size_t)ft * nkb2 * 64 * D::KPL + (size_t)lane * D::KPL;
      const T* w1 = W2 + (size_t)(NFT + ft) * nkb2 * 64 * D::KPL + (size_t)lane * D::KPL;
      const T* w2 = W2 + (size_t)(2 * NFT + ft) * nkb2 * 64 * D::KPL + (size_t)lane * D::KPL;
      kloop<D, nkb2, ring_depth<D, 3, RX>(), 3, RT>(
          xp, LD1,
          [&](int kb, Fd* f) {
            f[0] = D::frag(w0 + (size_t)kb * 64 * D::KPL);
            f[1] = D::frag(w1 + (size_t)kb * 64 * D::KPL);
            f[2] = D::frag(w2 + (size_t)kb * 64 * D::KPL);
          },
          [&](int kb, const Fd* x, const Fd* f) {
#pragma unroll
            for (int j = 0; j < D::SUB; ++j)
#pragma unroll
              for (int r = 0; r < RT; ++r) {
                avv[r] = D::mfma_sub(x[r], f[0], avv[r], j);
                asv[r] = D::mfma_sub(x[r], f[1], asv[r], j);
                ass[r] = D::mfma_sub(x[r], f[2], ass[r], j);
              }
          });
      const int col = ft * 16 + (lane & 15);
      const A bvv = b2[col], bsv = b2[F + col], bss = b2[2 * F + col];
#pragma unroll
      for (int r = 0; r < RT; ++r)
        for (int i = 0; i < 4; ++i) {
          const int rr = r * 16 + P::row(lane, i);
          const size_t row = row0 + rr;
          const A g_vv = avv[r][i] + bvv, g_sv = asv[r][i] + bsv, g_ss = ass[r][i] + bss;
          if constexpr (SAVE) {
            if (row < (size_t)N) {
              ((T*)a.save_a)[row * 2 * F + col] = P::st(g_vv);
              ((T*)a.save_a)[row * 2 * F + F + col] = P::st(g_sv);
            }
          }
          const A sn = P::ld(SN[rr * LD2 + col]) + g_sv * pd[q][r][i] + g_ss;
          const T st = P::st(sn);
          SN[rr * LD2 + col] = st;
          if (row < (size_t)N) {
            s_out[row * F + col] = st;
            for (int c = 0; c < 3; ++c) {
              const size_t o = row * 3 * F + c * F + col;
              v_out[o] = P::st(P::ld(VREG ? vkeep[q][c][r][i] : v[o]) + g_vv * U[q][c][r][i]);
            }
          }
        }
    }
  }
  if (FUSE_PHI) {
    __syncthreads();
    phi_tile<P, F, RT, NW>(SN, LD2, H, row0, N, a.phi1, a.phi2, (T*)a.h);
  }
}

// ---------------------------------------------------------------- heads ----
// Per atom: shared MLP (silu after every layer), then the branch MLP of the
// structure's dataset (silu between layers, last layer linear to a scalar).
//
// With dataset ids the atoms are first grouped by head on the device (a
// counting sort: count, plan, scatter), so that one workgroup runs ONE branch
// over a tile of TM = 16 RT atoms and every weight fragment it streams serves
// TM rows.  The branch's last layer has a single output; it is folded into
// the epilogue of the layer before it as a dot product, so the widest hidden
// layer never goes through LDS.  Every atom's result depends only on its own
// row, so the grouping order does not change any value.
// Waves per heads workgroup: 8, or 16 when a head layer is at least 256
// wide (its LDS buffers then allow one workgroup per CU; measured faster).
constexpr int HEADS_NW = 8, HEADS_NW_WIDE = 16, HEADS_WIDE = 256;

static_assert(sizeof(HeadPlan) <= 1024, "head plan workspace is 1 KiB");
static_assert(sizeof(HeadTile) == 16, "head tile workspace is 16 bytes per tile");

__device__ __forceinline__ int atom_head(const int32_t* dataset_id, const int32_t* atom_struct,
                                         int n_heads, int atom) {
  const int h = dataset_id[atom_struct[atom]];
  return h < 0 || h >= n_heads ? -1 : h;
}

__global__ void __launch_bounds__(64) k_head_clear(HeadPlan* p) {
  const int t = threadIdx.x;
  p->count[t] = 0;
  p->cursor[t] = 0;
  if (t == 0) p->n_tiles = 0;
}

// Entries (atom, head) to run.  One dataset's head per atom (hw null): the
// structure's dataset id, and atoms with an invalid id get a NaN energy.
// Blended heads (hw given): every head whose weight for the atom's structure
// is >= skip.
template <class A>
__device__ __forceinline__ bool entry_on(const int32_t* dataset_id, const A* hw, int H, A skip, int b,
                                         int h) {
  return hw ? hw[(size_t)b * H + h] >= skip : dataset_id[b] == h;
}

template <class A>
__global__ void __launch_bounds__(256) k_head_count(int N, int n_heads, const int32_t* dataset_id,
                                                    const A* hw, A skip, const int32_t* atom_struct,
                                                    HeadPlan* p, A* e) {
  __shared__ int hist[HEADS_MAX];
  if (threadIdx.x < HEADS_MAX) hist[threadIdx.x] = 0;
  __syncthreads();
  const int atom = blockIdx.x * 256 + threadIdx.x;
  if (atom < N) {
    const int b = atom_struct[atom];
    if (hw) {
      for (int h = 0; h < n_heads; ++h)
        if (entry_on(dataset_id, hw, n_heads, skip, b, h)) atomicAdd(&hist[h], 1);
    } else {
      const int h = atom_head(dataset_id, atom_struct, n_heads, atom);
      if (h < 0) e[atom] = (A)NAN;
      else atomicAdd(&hist[h], 1);
    }
  }
  __syncthreads();
  if (threadIdx.x < n_heads && hist[threadIdx.x] > 0) atomicAdd(&p->count[threadIdx.x], hist[threadIdx.x]);
}

// head offsets in the atom order and the tile list (one wave)
__global__ void __launch_bounds__(64) k_head_plan(int n_heads, int TM, HeadPlan* p, HeadTile* tiles) {
  __shared__ int start[HEADS_MAX], tbase[HEADS_MAX];
  const int h = threadIdx.x;
  if (h == 0) {
    int s = 0, t = 0;
    for (int q = 0; q < n_heads; ++q) {
      start[q] = s;
      tbase[q] = t;
      s += p->count[q];
      t += (p->count[q] + TM - 1) / TM;
    }
    p->n_tiles = t;
  }
  __syncthreads();
  if (h < n_heads) {
    const int c = p->count[h], s0 = start[h];
    p->start[h] = s0;
    for (int k = 0; k * TM < c; ++k) {
      HeadTile tl;
      tl.head = h;
      tl.begin = s0 + k * TM;
      tl.end = min(s0 + (k + 1) * TM, s0 + c);
      tl.pad = 0;
      tiles[tbase[h] + k] = tl;
    }
  }
}

// entry order grouped by head: block-local ranks, one global reservation per
// head, head by head; an entry holds its atom (the tile gives the head)
template <class A>
__global__ void __launch_bounds__(256) k_head_scatter(int N, int n_heads, const int32_t* dataset_id,
                                                      const A* hw, A skip, const int32_t* atom_struct,
                                                      HeadPlan* p, int32_t* order) {
  __shared__ int cnt, base;
  const int atom = blockIdx.x * 256 + threadIdx.x;
  uint64_t on = 0;                       // heads of this atom (n_heads <= 64)
  if (atom < N) {
    if (hw) {
      const int b = atom_struct[atom];
      for (int h = 0; h < n_heads; ++h)
        if (entry_on(dataset_id, hw, n_heads, skip, b, h)) on |= 1ull << h;
    } else {
      const int h = atom_head(dataset_id, atom_struct, n_heads, atom);
      if (h >= 0) on = 1ull << h;
    }
  }
  for (int h = 0; h < n_heads; ++h) {
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    const bool mine = (on >> h) & 1ull;
    const int r = mine ? atomicAdd(&cnt, 1) : 0;
    __syncthreads();
    if (threadIdx.x == 0 && cnt > 0) base = p->start[h] + atomicAdd(&p->cursor[h], cnt);
    __syncthreads();
    if (mine) order[base + r] = atom;
  }
}

struct HeadArgs {
  int N, ns, nb;
  int lds_s, lds_b;                    // row strides of the shared / branch buffers
  int off_sa, off_sb, off_b0, off_b1;  // buffer offsets in the dynamic LDS (elements)
  const void* s;
  const int32_t* order;    // null: tiles of consecutive atoms, head 0
  const HeadTile* tiles;
  const HeadPlan* plan;
  const void* const* table;  // [n_heads][nb][2] = (packed w, bias)
  DenseDev shared[16];
  int bdin[16], bdout[16];
  void* e;       // [N]: one dataset's head per atom
  void* eh;      // [N][H]: blended heads (e unused), or null
  int H;
};

// Element k of output row 0 of a packed dense layer (the B fragment order).
template <class Q>
__device__ __forceinline__ typename Q::A packed_row0(const DenseDev& L, int k) {
  using P = dense_t<Q>;
  const int kb = k / P::KC, r = k % P::KC;
  return P::ld(((const typename P::T*)L.w)[((size_t)kb * 64 + 16 * (r / P::KPL)) * P::KPL + r % P::KPL]);
}

// LDS: X [TM][F+PAD] (the tile's final s), SA/SB [TM][lds_s] (shared
// layers), B0/B1 [TM][lds_b] (stored branch hidden layers); with shared
// layers B0 reuses X, which is dead after the first of them.
template <class P, int F, int RT, int NW>
__global__ void __launch_bounds__(64 * NW) k_heads(HeadArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  constexpr int TM = 16 * RT, LDX = F + P::PAD;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* lds = (T*)smem;
  __shared__ int idx[TM];
  __shared__ A part[NW][TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int head = 0, begin, end;
  if (a.tiles) {
    if ((int)blockIdx.x >= a.plan->n_tiles) return;
    const HeadTile tl = a.tiles[blockIdx.x];
    head = tl.head;
    begin = tl.begin;
    end = tl.end;
  } else {
    begin = blockIdx.x * TM;
    end = min(a.N, begin + TM);
  }
  if (threadIdx.x < TM) {
    const int k = begin + threadIdx.x;
    idx[threadIdx.x] = k < end ? (a.order ? a.order[k] : k) : -1;
  }
  __syncthreads();
  T* X = lds;
  const T* s = (const T*)a.s;
  for (int x = threadIdx.x; x < TM * F; x += blockDim.x) {
    const int r = x / F, c = x % F;
    const int g = idx[r];
    X[r * LDX + c] = g >= 0 ? s[(size_t)g * F + c] : P::st(0);
  }
  __syncthreads();
  // shared layers: X -> SA -> SB -> SA ...
  const T* S = X;
  int ld_S = LDX;
  for (int m = 0; m < a.ns; ++m) {
    T* dst = lds + ((m & 1) ? a.off_sb : a.off_sa);
    const int ld = a.lds_s;
    const DenseDev& L = a.shared[m];
    dense_tiles<P, RT, NW>(S, ld_S, L, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      const A bias = ((const A*)L.b)[col];
      for (int r = 0; r < RT; ++r)
        for (int i = 0; i < 4; ++i)
          dst[(r * 16 + P::row(lane, i)) * ld + col] = P::st(silu<A>(acc[r][i] + bias));
    });
    __syncthreads();
    S = dst;
    ld_S = ld;
  }
  auto branch = [&](int m) {
    DenseDev L;
    L.w = (void*)a.table[((size_t)head * a.nb + m) * 2];
    L.b = (void*)a.table[((size_t)head * a.nb + m) * 2 + 1];
    L.din = a.bdin[m];
    L.dout = a.bdout[m];
    L.din_p = pad32(a.bdin[m]);
    L.dout_p = pad32(a.bdout[m]);
    return L;
  };
  const int rt = threadIdx.x;
  A y = 0;
  if (a.nb == 1) {
    // one linear layer: a dot product per row, straight from S
    const DenseDev Lz = branch(0);
    if (rt < TM) {
      y = ((const A*)Lz.b)[0];
      for (int k = 0; k < Lz.din; ++k) y += P::ld(S[rt * ld_S + k]) * packed_row0<P>(Lz, k);
    }
  } else {
    const T* in = S;
    int ld_in = ld_S;
    for (int m = 0; m + 2 < a.nb; ++m) {
      T* dst = lds + ((m & 1) ? a.off_b1 : a.off_b0);
      const int ld = a.lds_b;
      const DenseDev L = branch(m);
      dense_tiles<P, RT, NW>(in, ld_in, L, [&](int ct, C* acc) {
        const int col = ct * 16 + (lane & 15);
        const A bias = ((const A*)L.b)[col];
        for (int r = 0; r < RT; ++r)
          for (int i = 0; i < 4; ++i)
            dst[(r * 16 + P::row(lane, i)) * ld + col] = P::st(silu<A>(acc[r][i] + bias));
      });
      __syncthreads();
      in = dst;
      ld_in = ld;
    }
    // last hidden layer with the output layer folded in: every lane sums
    // silu(.) * w_out over the columns it holds, in a fixed order
    const DenseDev L = branch(a.nb - 2), Lz = branch(a.nb - 1);
    A p[RT][4];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) p[r][i] = 0;
    dense_tiles<P, RT, NW>(in, ld_in, L, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      const A bias = ((const A*)L.b)[col];
      const A wz = packed_row0<P>(Lz, col);
      for (int r = 0; r < RT; ++r)
        for (int i = 0; i < 4; ++i) p[r][i] += silu<A>(acc[r][i] + bias) * wz;
    });
    // the 16 lanes of a group hold the same rows: butterfly over them
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i)
        for (int off = 1; off < 16; off <<= 1) p[r][i] += __shfl_xor(p[r][i], off);
    if ((lane & 15) == 0)
      for (int r = 0; r < RT; ++r)
        for (int i = 0; i < 4; ++i) part[wave][r * 16 + P::row(lane, i)] = p[r][i];
    __syncthreads();
    if (rt < TM) {
      y = ((const A*)Lz.b)[0];
      for (int w = 0; w < NW; ++w) y += part[w][rt];
    }
  }
  if (rt < TM && idx[rt] >= 0) {
    if (a.eh) ((A*)a.eh)[(size_t)idx[rt] * a.H + head] = y;
    else ((A*)a.e)[idx[rt]] = y;
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

// s [N][Fl] and v [N][3][Fl] in FP64 from the working arrays of width F >= Fl
// (the model's own channels; the rest is zero padding)
template <class P>
__global__ void __launch_bounds__(256) k_export(int N, int F, int Fl, const typename P::T* __restrict__ s,
                                               const typename P::T* __restrict__ v,
                                               double* __restrict__ so, double* __restrict__ vo) {
  const size_t tot = (size_t)N * Fl;
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < tot; x += (size_t)gridDim.x * blockDim.x) {
    const size_t i = x / Fl, f = x % Fl;
    so[x] = (double)P::ld(s[i * F + f]);
    for (int c = 0; c < 3; ++c) vo[(3 * i + c) * Fl + f] = (double)P::ld(v[(3 * i + c) * F + f]);
  }
}

inline int grid_for(size_t n, int per) {
  size_t g = (n + per - 1) / per;
  if (g > 65536) g = 65536;
  return (int)(g ? g : 1);
}

// Channel-per-lane form (FP32 / BF16 storage).  A workgroup of F/64 waves
// owns MSG_RB2 consecutive receivers; wave w owns channels [64 w, 64 w + 64)
// = feature tiles 4w..4w+3 and keeps their filter B fragments in registers.
// Per 16-edge chunk (the block's edges back to back, so a chunk may hold
// the end of one receiver's row and the start of the next) the wave forms Wt
// for its channels on the matrix cores and parks it in its own LDS tile
// (edge-major); then every lane, one channel, walks the chunk's edges: the
// sender index is wave-uniform, so each gather reads 256 contiguous bytes of
// a sender row, and the filter values come back from LDS.  Sums stay in the
// lane (no cross-lane reduction) until the receiver's last edge, and no wave
// waits for another.
constexpr int MSG_RB2 = 8;

template <class A>
__device__ __forceinline__ A bcast(A x, int lane) {
  if constexpr (sizeof(A) == 4) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
  } else {
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffff), lane);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
  }
}

// Two waves per SIMD while the filter's B fragments leave room for them.
template <class P, int KBM>
constexpr int message_waves() {
  return 12 * KBM * (int)sizeof(typename P::Fr) / 4 > 150 ? 1 : 2;
}

template <class P, int F, int KBM, bool V0, bool NB>
__global__ void __launch_bounds__(F) __attribute__((amdgpu_waves_per_eu(message_waves<P, KBM>())))
k_message_lane(MsgArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  using Fr = typename P::Fr;
  constexpr int NW = F / 64, NFT = F / 16;
  // LDS filter tile of one part: channel-major, a row of the chunk's 16
  // edges per channel, as 4 groups of 4 edges stored in the order
  // g ^ (((channel >> 1) ^ (channel >> 2)) & 3): the 16-byte accesses of any
  // 8 (and any 16) consecutive lanes (channels) then fall in distinct 4-bank
  // groups of a 32-bank (and a 64-bank) LDS, without padding
  constexpr int WLD = 16;
  static_assert(sizeof(A) == 4, "FP32 accumulation");
  auto wslot = [](int ch, int g) { return ch * WLD + 4 * (g ^ (((ch >> 1) ^ (ch >> 2)) & 3)); };
  constexpr int kcols = KBM * P::KC;
  // VGPRs held by the filter's B fragments decide how much else is in flight
  constexpr int BF_REGS = 12 * KBM * (int)sizeof(Fr) / 4;
  constexpr int QI = BF_REGS > 100 ? 1 : 4;     // MFMA chains issued together (feature tiles)
  constexpr int EG = BF_REGS > 100 ? 4 : sizeof(T) == 4 ? 16 : 8;   // edges gathered per group
  // Issue the first group's gathers ahead of the filter MFMAs.  Measured: a
  // gain for BF16 with a short filter (few K blocks), a loss for FP32, whose
  // gathers move twice the bytes behind a long MFMA phase.
  constexpr bool EARLY = sizeof(T) == 2 && BF_REGS <= 100;
  __shared__ __attribute__((aligned(16))) A Wt[NW][3][64 * WLD];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = 64 * wave + lane;               // this lane's channel
  const T* Wf = (const T*)a.filt_mma.w;
  Fr Bf[4][3][KBM];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int part = 0; part < 3; ++part)
#pragma unroll
      for (int kb = 0; kb < KBM; ++kb) {
        const int ct = part * NFT + 4 * wave + q;
        Bf[q][part][kb] = P::frag(Wf + ((size_t)(ct * KBM + kb) * 64 + lane) * P::KPL);
      }
  // without the bias column: b_f at this lane's channel, per part
  const A bs = NB ? ((const A*)a.fbias)[c] : A(0);
  const A bv = NB ? ((const A*)a.fbias)[F + c] : A(0);
  const A br = NB ? ((const A*)a.fbias)[2 * F + c] : A(0);
  const T* h = (const T*)a.h;
  const T* vin = (const T*)a.v_in;
  const T* basis = (const T*)a.basis;
  const A* einfo = (const A*)a.einfo;
  const T* sin = (const T*)a.s_in;
  T* s = (T*)a.s;
  T* vout = (T*)a.v_out;
  A* wt0 = Wt[wave][0];
  A* wt1 = Wt[wave][1];
  A* wt2 = Wt[wave][2];
  // XCD-contiguous receiver ranges (see k_message)
  const int per_xcd = gridDim.x / 8;
  const int lb = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int i0 = lb * MSG_RB2;
  if (i0 >= a.N) return;
  const int i1 = min(a.N, i0 + MSG_RB2);
  const int rp_lane = a.row_ptr[i0 + min(lane, i1 - i0)];
  auto rp = [&](int i) { return __builtin_amdgcn_readlane(rp_lane, i - i0); };
  // receivers without edges: v_out = v_in, s_out = s_in
  for (int i = i0; i < i1; ++i)
    if (rp(i) == rp(i + 1)) {
      const size_t ib = (size_t)i * 3 * F;
      s[(size_t)i * F + c] = sin[(size_t)i * F + c];
      vout[ib + c] = V0 ? P::st(0) : vin[ib + c];
      vout[ib + F + c] = V0 ? P::st(0) : vin[ib + F + c];
      vout[ib + 2 * F + c] = V0 ? P::st(0) : vin[ib + 2 * F + c];
    }
  auto first_with_edges = [&](int i) {
    while (i < i1 && rp(i) == rp(i + 1)) ++i;
    return i;
  };
  // The block's edges [E0, E1) (its receivers' CSR rows back to back) are
  // walked as one stream of 16-edge chunks that may span receivers, so only
  // the block's last chunk is partial.  The next chunk's basis rows and edge
  // info are loaded while the current one is processed (the basis streams
  // from HBM).
  const int E0 = rp(i0), E1 = rp(i1);
  if (E0 == E1) return;
  Fr Gn[KBM];
  // lane e: edge e of the next chunk's rhat and its sender index (NB: its
  // f_c in ejn, the sender in jn)
  A exn = 0, eyn = 0, ezn = 0, ejn = 0;
  int jn = 0;
  auto prefetch = [&](int cc0, int ccnt) {
    const T* gp = basis + (size_t)(cc0 + (lane & 15)) * kcols + (lane >> 4) * P::KPL;
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) Gn[kb] = P::frag(gp + kb * P::KC);
    exn = eyn = ezn = ejn = 0;
    jn = 0;
    if (lane < ccnt) {
      const A* ei = einfo + 4 * (size_t)(cc0 + lane);
      exn = ei[0];
      eyn = ei[1];
      ezn = ei[2];
      ejn = ei[3];
      if constexpr (NB) jn = a.col[cc0 + lane];
    }
  };
  int c0 = E0;
  prefetch(c0, min(16, E1 - c0));
  // the receiver being summed: i, whose edges end at eb
  int i = first_with_edges(i0);
  int eb = rp(i + 1);
  size_t ib = (size_t)i * 3 * F;
  T s_old = sin[(size_t)i * F + c];
  // (the first layer's v is zero and need not be stored)
  T v_old0 = V0 ? P::st(0) : vin[ib + c], v_old1 = V0 ? P::st(0) : vin[ib + F + c];
  T v_old2 = V0 ? P::st(0) : vin[ib + 2 * F + c];
  A acc_s = 0, acc_v0 = 0, acc_v1 = 0, acc_v2 = 0;
  auto write_out = [&] {
    s[(size_t)i * F + c] = P::st(P::ld(s_old) + acc_s);
    vout[ib + c] = P::st(P::ld(v_old0) + acc_v0);
    vout[ib + F + c] = P::st(P::ld(v_old1) + acc_v1);
    vout[ib + 2 * F + c] = P::st(P::ld(v_old2) + acc_v2);
  };
  // Edge c0 + e starts the next receiver: write receiver i out and move on
  // (a wave-uniform branch; the last receiver is written after the stream).
  auto next_receiver = [&] {
    write_out();
    acc_s = acc_v0 = acc_v1 = acc_v2 = 0;
    i = first_with_edges(i + 1);
    eb = rp(i + 1);
    ib = (size_t)i * 3 * F;
    s_old = sin[(size_t)i * F + c];
    if constexpr (!V0) {
      v_old0 = vin[ib + c];
      v_old1 = vin[ib + F + c];
      v_old2 = vin[ib + 2 * F + c];
    }
  };
  while (true) {
    const int cnt = min(16, E1 - c0);
    // A rows past the stream's end are zeroed, so are their filter rows
    const bool row_ok = (lane & 15) < cnt;
    Fr Ga[KBM];
#pragma unroll
    for (int kb = 0; kb < KBM; ++kb) Ga[kb] = row_ok ? Gn[kb] : Fr{};
    // lanes e < cnt hold edge c0 + e: rhat and the sender index (NB: f_c,
    // and the sender in jc)
    const A ex = exn, ey = eyn, ez = ezn, ej = ejn;
    const int jc = jn;
    const int cn = c0 + 16;
    const bool more = cn < E1;
    if (more) prefetch(cn, min(16, E1 - cn));
    // Gathers of EG edges: sender rows h_j (3 parts) and v_j (3 components)
    // at this lane's channel.  Past the stream's end the sender is row 0
    // (lanes >= cnt hold index 0) and the filter rows are zero, so a group
    // needs no early exit and all its 6 EG loads can be in flight together.
    T gb[6][EG];
    auto gather = [&](int ebase) {
#pragma unroll
      for (int u = 0; u < EG; ++u) {
        const int j = NB ? __builtin_amdgcn_readlane(jc, ebase + u) : acc_to_index(bcast(ej, ebase + u));
        const T* hj = h + (size_t)j * 3 * F + c;
        const T* vj = vin + (size_t)j * 3 * F + c;
        gb[0][u] = hj[0];
        gb[1][u] = hj[F];
        gb[2][u] = hj[2 * F];
        // (with v_j = 0 the term v_j h^v_j w^v is exactly zero: not gathered)
        if constexpr (!V0) {
          gb[3][u] = vj[0];
          gb[4][u] = vj[F];
          gb[5][u] = vj[2 * F];
        }
      }
    };
    auto consume = [&](int ebase) {
      f4_t ws4, wv4, wr4;
#pragma unroll
      for (int u = 0; u < EG; ++u) {
        const int e = ebase + u;
        // the filter of 4 edges at this lane's channel, one 16-byte read per part
        if (u % 4 == 0) {
          const int o = wslot(lane, e / 4);
          ws4 = *(const f4_t*)(wt0 + o);
          if constexpr (!V0) wv4 = *(const f4_t*)(wt1 + o);
          wr4 = *(const f4_t*)(wt2 + o);
        }
        // eb < E1: receiver i is not the block's last one (past the
        // stream's end, c0 + e >= E1 >= eb)
        if (c0 + e == eb && eb < E1) next_receiver();
        const A rx = bcast(ex, e), ry = bcast(ey, e), rz = bcast(ez, e);
        // the bias: w = f_c (W_f g + b_f)
        const A fe = NB ? bcast(ej, e) : A(0);
        const A ws = NB ? ws4[u % 4] + fe * bs : ws4[u % 4];
        const A wr = NB ? wr4[u % 4] + fe * br : wr4[u % 4];
        acc_s += P::ld(gb[0][u]) * ws;
        const A pr = P::ld(gb[2][u]) * wr;
        if constexpr (V0) {
          acc_v0 += rx * pr;
          acc_v1 += ry * pr;
          acc_v2 += rz * pr;
        } else {
          const A pv = P::ld(gb[1][u]) * (NB ? wv4[u % 4] + fe * bv : wv4[u % 4]);
          acc_v0 += P::ld(gb[3][u]) * pv + rx * pr;
          acc_v1 += P::ld(gb[4][u]) * pv + ry * pr;
          acc_v2 += P::ld(gb[5][u]) * pv + rz * pr;
        }
      }
    };
    // the first group's gathers do not depend on the filter: issued before
    // the MFMAs, they arrive while the matrix cores run
    if constexpr (EARLY) {
      gather(0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // The filter of 4 feature tiles x 3 parts, parked in LDS.  With few
    // registers held by the B fragments all 12 MFMA chains are issued
    // together (QI = 4); otherwise one feature tile at a time (QI = 1).
#pragma unroll
    for (int q0 = 0; q0 < 4; q0 += QI) {
      C w[QI][3];
#pragma unroll
      for (int q = 0; q < QI; ++q)
#pragma unroll
        for (int part = 0; part < 3; ++part)
          for (int r = 0; r < 4; ++r) w[q][part][r] = 0;
#pragma unroll
      for (int kb = 0; kb < KBM; ++kb)
#pragma unroll
        for (int q = 0; q < QI; ++q)
#pragma unroll
          for (int part = 0; part < 3; ++part)
            if (!V0 || part != 1)   // the v part of the filter only meets v_j
              w[q][part] = P::mfma(Ga[kb], Bf[q0 + q][part][kb], w[q][part]);
      // this lane's 4 accumulator rows are the 4 consecutive edges of group
      // lane / 16 at one channel: one 16-byte write per part
#pragma unroll
      for (int q = 0; q < QI; ++q) {
        const int o = wslot(16 * (q0 + q) + (lane & 15), lane >> 4);
        *(f4_t*)(wt0 + o) = f4_t{w[q][0][0], w[q][0][1], w[q][0][2], w[q][0][3]};
        if constexpr (!V0) *(f4_t*)(wt1 + o) = f4_t{w[q][1][0], w[q][1][1], w[q][1][2], w[q][1][3]};
        *(f4_t*)(wt2 + o) = f4_t{w[q][2][0], w[q][2][1], w[q][2][2], w[q][2][3]};
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if constexpr (EARLY) consume(0);
#pragma unroll
    for (int eb0 = EARLY ? EG : 0; eb0 < 16; eb0 += EG)
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

template <class P, int F, int KBM, bool NB, bool RG = false>
void launch_message_kbm(hipStream_t st, const MsgArgs& a) {
  if constexpr (sizeof(typename P::T) == 8) {
    // eight waves per workgroup: NGW channel groups times NS streams
    constexpr int NGW = msg64_groups<F, KBM>(), NS = 8 / NGW, SPLIT = F / 32 / NGW;
    constexpr int IMG = msg64_image_size<F, NGW, KBM, NB>();
    MsgArgs b = a;
    if ((size_t)SPLIT * IMG * sizeof(msg_d2) > MSG64_IMAGE_BYTES) b.img = nullptr;
    if (b.img)
      k_msg64_image<F, NGW, KBM, NB><<<dim3((IMG + 255) / 256, SPLIT), 256, 0, st>>>(b, (msg_d2*)b.img);
    // grids are a multiple of the 8 XCDs
    if (RG && a.E >= (long long)MSG_RB16_DEGREE * a.N) {
      constexpr int RB = RG ? 16 : MSG_RB64;
      const int blocks = ((a.N + RB - 1) / RB * SPLIT + 7) / 8 * 8;
      if (a.v_zero) k_message<P, F, NGW, NS, KBM, true, NB, RG, RB><<<blocks, 512, 0, st>>>(b);
      else k_message<P, F, NGW, NS, KBM, false, NB, RG, RB><<<blocks, 512, 0, st>>>(b);
    } else {
      const int blocks = ((a.N + MSG_RB64 - 1) / MSG_RB64 * SPLIT + 7) / 8 * 8;
      if (a.v_zero) k_message<P, F, NGW, NS, KBM, true, NB, RG, MSG_RB64><<<blocks, 512, 0, st>>>(b);
      else k_message<P, F, NGW, NS, KBM, false, NB, RG, MSG_RB64><<<blocks, 512, 0, st>>>(b);
    }
  } else {
    const int blocks = ((a.N + MSG_RB2 - 1) / MSG_RB2 + 7) / 8 * 8;
    if (a.v_zero) k_message_lane<P, F, KBM, true, NB><<<blocks, F, 0, st>>>(a);
    else k_message_lane<P, F, KBM, false, NB><<<blocks, F, 0, st>>>(a);
  }
}

// The filter's input is padded to one of the compiled k-block counts.
template <class P, int F>
hipError_t launch_message(hipStream_t st, const MsgArgs& a) {
  const int nkb = a.filt_mma.din_p / P::KC;
  if constexpr (P::KC == 32) {
    if (a.nb) {
      switch (nkb) {
        case 1: launch_message_kbm<P, F, 1, true>(st, a); break;
        case 2: launch_message_kbm<P, F, 2, true>(st, a); break;
        case 3: launch_message_kbm<P, F, 3, true>(st, a); break;
        case 5: launch_message_kbm<P, F, 5, true>(st, a); break;
        default: return hipErrorInvalidValue;
      }
    } else {
      switch (nkb) {
        case 1: launch_message_kbm<P, F, 1, false>(st, a); break;
        case 2: launch_message_kbm<P, F, 2, false>(st, a); break;
        case 3: launch_message_kbm<P, F, 3, false>(st, a); break;
        case 5: launch_message_kbm<P, F, 5, false>(st, a); break;
        default: return hipErrorInvalidValue;
      }
    }
  } else if (a.nb) {
    constexpr bool F64 = sizeof(typename P::T) == 8;
    if (a.rg && !(F64 && (nkb == 5 || nkb == 8))) return hipErrorInvalidValue;
    switch (nkb) {
      case 1: launch_message_kbm<P, F, 1, true>(st, a); break;
      case 2: launch_message_kbm<P, F, 2, true>(st, a); break;
      case 5:
        if (a.rg) launch_message_kbm<P, F, 5, true, F64>(st, a);
        else launch_message_kbm<P, F, 5, true>(st, a);
        break;
      case 8:
        if (a.rg) launch_message_kbm<P, F, 8, true, F64>(st, a);
        else launch_message_kbm<P, F, 8, true>(st, a);
        break;
      case 12: launch_message_kbm<P, F, 12, true>(st, a); break;
      case 17: launch_message_kbm<P, F, 17, true>(st, a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (nkb) {
      case 3: launch_message_kbm<P, F, 3, false>(st, a); break;
      case 6: launch_message_kbm<P, F, 6, false>(st, a); break;
      case 9: launch_message_kbm<P, F, 9, false>(st, a); break;
      case 12: launch_message_kbm<P, F, 12, false>(st, a); break;
      case 17: launch_message_kbm<P, F, 17, false>(st, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipSuccess;
}

// ------------------------------------------------ branch weighting ----
// Composition vector of every structure: fractions of its atoms per species,
// padded with zeros to pad32(S) columns (one wave per structure).
template <class P>
__global__ void __launch_bounds__(256) k_composition(int B, int S, const int32_t* __restrict__ struct_ptr,
                                                     const int32_t* __restrict__ species,
                                                     typename P::T* __restrict__ comp) {
  __shared__ int hist[4][256];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int b = blockIdx.x * 4 + wv;
  const int Sp = pad32(S);
  for (int z = lane; z < 256; z += 64) hist[wv][z] = 0;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (b >= B) return;
  const int lo = struct_ptr[b], hi = struct_ptr[b + 1];
  for (int i = lo + lane; i < hi; i += 64) {
    const int z = species[i];
    if (z >= 0 && z < S) atomicAdd(&hist[wv][z], 1);
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const typename P::A inv = hi > lo ? (typename P::A)1 / (typename P::A)(hi - lo) : (typename P::A)0;
  for (int z = lane; z < Sp; z += 64)
    comp[(size_t)b * Sp + z] = P::st(z < S ? (typename P::A)hist[wv][z] * inv : (typename P::A)0);
}

struct BlendArgs {
  int B, S, H, nl;
  const void* comp;
  DenseDev layer[9];
  int width;            // widest padded layer (LDS row stride minus padding)
  void* hw;             // [B][H] accumulation type
  double* weights_out;  // [B][H] or null
};

// The branch-weighting MLP over 16 structures per workgroup (silu between
// layers), then a softmax over the heads.
template <class P>
__global__ void __launch_bounds__(256) k_blend(BlendArgs a) {
  using T = typename P::T;
  using A = typename P::A;
  using C = typename P::C;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int ld = a.width + P::PAD;
  T* X0 = (T*)smem;
  T* X1 = X0 + 16 * ld;
  A* logit = (A*)(X1 + 16 * ld);
  const int lane = threadIdx.x & 63;
  const int b0 = blockIdx.x * 16;
  const int Sp = pad32(a.S);
  const T* comp = (const T*)a.comp;
  for (int x = threadIdx.x; x < 16 * Sp; x += blockDim.x) {
    const int r = x / Sp, c = x % Sp;
    X0[r * ld + c] = b0 + r < a.B ? comp[(size_t)(b0 + r) * Sp + c] : P::st(0);
  }
  __syncthreads();
  const T* in = X0;
  for (int m = 0; m < a.nl; ++m) {
    const DenseDev& L = a.layer[m];
    const bool last = m == a.nl - 1;
    T* dst = (m & 1) ? X0 : X1;
    dense_tiles<P, 1, 4>(in, ld, L, [&](int ct, C* acc) {
      const int col = ct * 16 + (lane & 15);
      const A bias = ((const A*)L.b)[col];
      for (int i = 0; i < 4; ++i) {
        const int r = P::row(lane, i);
        const A y = acc[0][i] + bias;
        if (last) {
          if (col < a.H) logit[r * 64 + col] = y;
        } else {
          dst[r * ld + col] = P::st(silu<A>(y));
        }
      }
    });
    __syncthreads();
    in = dst;
  }
  if (threadIdx.x < 16 && b0 + threadIdx.x < a.B) {
    const int r = threadIdx.x;
    A mx = logit[r * 64];
    for (int h = 1; h < a.H; ++h) mx = logit[r * 64 + h] > mx ? logit[r * 64 + h] : mx;
    A sum = 0;
    for (int h = 0; h < a.H; ++h) sum += P::ex(logit[r * 64 + h] - mx);
    A* hw = (A*)a.hw + (size_t)(b0 + r) * a.H;
    for (int h = 0; h < a.H; ++h) {
      const A w = P::ex(logit[r * 64 + h] - mx) / sum;
      hw[h] = w;
      if (a.weights_out) a.weights_out[(size_t)(b0 + r) * a.H + h] = (double)w;
    }
  }
}

// Blended per-atom energy: sum over the kept heads in head order.
template <class A>
__global__ void __launch_bounds__(256) k_blend_reduce(int N, int H, A skip, const int32_t* __restrict__ atom_struct,
                                                      const A* __restrict__ hw, const A* __restrict__ eh,
                                                      A* __restrict__ e) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const A* w = hw + (size_t)atom_struct[i] * H;
  A y = 0;
  for (int h = 0; h < H; ++h)
    if (w[h] >= skip) y += w[h] * eh[(size_t)i * H + h];
  e[i] = y;
}

// Dynamic LDS beyond 64 KiB must be allowed once per kernel.
template <class P, int F, int RT, int NW>
hipError_t heads_allow_lds(size_t smem) {
  static size_t allowed = 64 * 1024;
  if (smem <= allowed) return hipSuccess;
  hipError_t e = hipFuncSetAttribute((const void*)k_heads<P, F, RT, NW>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  allowed = smem;
  return hipSuccess;
}

template <class P, int F, int RT>
hipError_t launch_heads_rt(hipStream_t st, HeadArgs& ha, int grid, size_t smem, bool wide) {
  hipError_t e = wide ? heads_allow_lds<P, F, RT, HEADS_NW_WIDE>(smem) : heads_allow_lds<P, F, RT, HEADS_NW>(smem);
  if (e != hipSuccess) return e;
  if (wide) k_heads<P, F, RT, HEADS_NW_WIDE><<<grid, 64 * HEADS_NW_WIDE, smem, st>>>(ha);
  else k_heads<P, F, RT, HEADS_NW><<<grid, 64 * HEADS_NW, smem, st>>>(ha);
  return hipGetLastError();
}

// Heads and per-atom energies: bin atoms by head (when dataset ids are
// given), then one workgroup per tile of the largest TM whose buffers fit
// the LDS.
template <class P, int F>
hipError_t launch_heads(hipStream_t st, ForwardArgs& fa) {
  using T = typename P::T;
  using A = typename P::A;
  const PrecModel* pm = fa.pm;
  const auto& hp = fa.m->hp;
  const int N = fa.g->N;
  HeadArgs ha;
  ha.N = N;
  ha.ns = (int)pm->shared.size();
  ha.nb = (int)hp.branch_dims.size();
  if (hp.n_heads > HEADS_MAX || ha.ns > 16 || ha.nb > 16) return hipErrorInvalidValue;
  int ws = 0, wb = 0;   // widest shared / stored branch layer (padded)
  for (int m = 0; m < ha.ns; ++m) {
    ha.shared[m] = pm->shared[m];
    ws = ws > pad32(hp.shared_dims[m]) ? ws : pad32(hp.shared_dims[m]);
  }
  int di = ha.ns == 0 ? F : hp.shared_dims.back();
  for (int m = 0; m < ha.nb; ++m) {
    ha.bdin[m] = di;
    ha.bdout[m] = hp.branch_dims[m];
    if (m + 2 < ha.nb) wb = wb > pad32(hp.branch_dims[m]) ? wb : pad32(hp.branch_dims[m]);
    di = hp.branch_dims[m];
  }
  const int nstored = ha.nb > 2 ? ha.nb - 2 : 0;
  ha.lds_s = ha.ns ? ws + P::PAD : 0;
  ha.lds_b = nstored ? wb + P::PAD : 0;
  constexpr int LDX = F + P::PAD;
  // buffer layout for TM rows; returns the dynamic LDS bytes
  auto layout = [&](int TM) {
    auto al = [](size_t x) { return (x + 7) & ~(size_t)7; };   // 16-byte aligned for bf16
    size_t o;
    if (ha.ns > 0) {
      const size_t r0 = al((size_t)TM * (nstored && ha.lds_b > LDX ? ha.lds_b : LDX));
      ha.off_b0 = 0;
      ha.off_sa = (int)r0;
      ha.off_sb = (int)(r0 + al((size_t)TM * ha.lds_s));
      o = ha.off_sb + al((size_t)TM * ha.lds_s);
    } else {
      ha.off_sa = ha.off_sb = 0;
      ha.off_b0 = (int)al((size_t)TM * LDX);
      o = ha.off_b0 + (nstored ? al((size_t)TM * ha.lds_b) : 0);
    }
    ha.off_b1 = (int)o;
    if (nstored > 1) o += al((size_t)TM * ha.lds_b);
    return o * sizeof(T);
  };
  constexpr size_t LDS_LIMIT = 150 * 1024;
  int RT = 4;
  size_t smem = 0;
  for (; RT >= 1; RT /= 2) {
    const int TM = 16 * RT;
    smem = layout(TM);
    const size_t fixed = (size_t)TM * sizeof(int) + (size_t)HEADS_NW_WIDE * TM * sizeof(A);
    if (smem + fixed <= LDS_LIMIT) break;
  }
  if (RT < 1) return hipErrorInvalidValue;
  const int TM = 16 * RT;
  ha.s = fa.s;
  ha.table = (const void* const*)pm->head_table;
  ha.e = fa.e;
  int grid = (N + TM - 1) / TM;
  const int H = hp.n_heads;
  ha.eh = nullptr;
  ha.H = H;
  prof_mark(fa.prof, st, KC_HEADS, true);
  if (fa.blend) {
    // composition vectors and the branch-weighting MLP's softmax weights
    const int B = fa.g->B, S = hp.n_species;
    k_composition<P><<<(B + 3) / 4, 256, 0, st>>>(B, S, fa.g->struct_ptr, fa.g->species, (T*)fa.comp);
    BlendArgs ba;
    ba.B = B;
    ba.S = S;
    ba.H = H;
    ba.nl = (int)pm->blend.size();
    if (ba.nl < 1 || ba.nl > 9 || H > 64) return hipErrorInvalidValue;
    ba.comp = fa.comp;
    ba.width = pad32(S);
    for (int m = 0; m < ba.nl; ++m) {
      ba.layer[m] = pm->blend[m];
      ba.width = ba.width > pm->blend[m].dout_p ? ba.width : pm->blend[m].dout_p;
    }
    ba.hw = fa.hw;
    ba.weights_out = fa.weights_out;
    const size_t bsmem = 2 * 16 * (size_t)(ba.width + P::PAD) * sizeof(T) + 16 * 64 * sizeof(A);
    if (bsmem > 64 * 1024) return hipErrorInvalidValue;
    if (B > 0) k_blend<P><<<(B + 15) / 16, 256, bsmem, st>>>(ba);
  }
  if (fa.dataset_id || fa.blend) {
    HeadPlan* plan = (HeadPlan*)fa.head_plan;
    HeadTile* tiles = (HeadTile*)fa.head_tiles;
    const A* hw = fa.blend ? (const A*)fa.hw : nullptr;
    const A skip = (A)fa.skip;
    const int nb256 = (N + 255) / 256;
    k_head_clear<<<1, 64, 0, st>>>(plan);
    k_head_count<A><<<nb256, 256, 0, st>>>(N, H, fa.dataset_id, hw, skip, fa.g->atom_struct, plan, (A*)fa.e);
    k_head_plan<<<1, 64, 0, st>>>(H, TM, plan, tiles);
    k_head_scatter<A><<<nb256, 256, 0, st>>>(N, H, fa.dataset_id, hw, skip, fa.g->atom_struct, plan,
                                             fa.head_order);
    ha.order = fa.head_order;
    ha.tiles = tiles;
    ha.plan = plan;
    if (fa.blend) {
      grid = (int)(((long long)N * H + TM - 1) / TM);
      ha.eh = fa.eh;
    }
    grid += H;
  } else {
    ha.order = nullptr;
    ha.tiles = nullptr;
    ha.plan = nullptr;
  }
  hipError_t e;
  int hmax = 0;   // widest hidden head layer
  for (int d : hp.shared_dims) hmax = hmax > d ? hmax : d;
  for (size_t m = 0; m + 1 < hp.branch_dims.size(); ++m) hmax = hmax > hp.branch_dims[m] ? hmax : hp.branch_dims[m];
  const bool wide = hmax >= HEADS_WIDE;
  if (RT == 4) e = launch_heads_rt<P, F, 4>(st, ha, grid, smem, wide);
  else if (RT == 2) e = launch_heads_rt<P, F, 2>(st, ha, grid, smem, wide);
  else e = launch_heads_rt<P, F, 1>(st, ha, grid, smem, wide);
  if (e == hipSuccess && fa.blend)
    k_blend_reduce<A><<<(N + 255) / 256, 256, 0, st>>>(N, H, (A)fa.skip, fa.g->atom_struct, (const A*)fa.hw,
                                                        (const A*)fa.eh, (A*)fa.e);
  prof_mark(fa.prof, st, KC_HEADS, false);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

template <class P, int F>
hipError_t forward_impl(hipStream_t st, ForwardArgs& fa) {
  using T = typename P::T;
  using A = typename P::A;
  const painn_graph* g = fa.g;
  const PrecModel* pm = fa.pm;
  const Hyper& hp = fa.m->hp;
  const int N = g->N;
  constexpr int RT = ((sizeof(T) == 8 && F >= 256) || F > 256) ? 1 : 2;
  // atoms per update tile / 16: U, |V|^2 and <U, V> of the tile live in registers
  constexpr int URT = update_rt<P, F>();
  T* s = (T*)fa.s;
  T* v[2] = {(T*)fa.v[0], (T*)fa.v[1]};
  T* h = (T*)fa.h;
  // With a save area every layer reads and writes its own slots (the
  // reverse pass reads them back); otherwise s and h are updated in place
  // and v is double buffered.
  const SaveLayout sv(fa.save, N, F, hp.L, sizeof(T));
  if (fa.save) {
    s = (T*)sv.S(0);
    v[0] = (T*)sv.V(0);
    h = (T*)sv.H(0);
    fa.s = sv.S(fa.stop_layer + 1);   // the heads read the final s
  }
  if (N > 0) {
    // embedding, and layer 0's phi from the per-species table
    prof_mark(fa.prof, st, KC_EMBED, true);
    // v = 0 is stored only where something reads it (the saved copy for the
    // reverse pass, or an export): the first message takes it as zero
    k_embed<P, F><<<grid_for((size_t)N * F / 4, 256), 256, 0, st>>>(N, g->species, (const T*)pm->emb,
                                                           (const T*)pm->h0, s,
                                                           fa.save || fa.s_out ? v[0] : nullptr,
                                                           fa.stop_layer >= 0 ? h : nullptr);
    prof_mark(fa.prof, st, KC_EMBED, false);
  }
  int cur = 0;
  // The filter without its bias column (f_c b_f added after the message's
  // MFMAs) where that saves MFMA k-blocks (also under a save area: the
  // reverse pass forms its own basis rows and reads only rhat here).
  const bool nb = !pm->layers.empty() &&
                  pm->layers[0].filt_nb.din_p < pm->layers[0].filt_mma.din_p;
  // In FP64 the message kernel forms Gaussians itself (up to 8 k-blocks,
  // K <= 32) where the feature arrays it gathers from fit 32-bit byte
  // offsets: each edge's basis row is then (g_0 f_c, exp(d / Delta - 1/2)).
  const int nkb_nb = nb ? pm->layers[0].filt_nb.din_p / P::KC : 0;
  const bool rg = nb && sizeof(T) == 8 && hp.rbf_type == 0 && (nkb_nb == 5 || nkb_nb == 8) &&
                  (size_t)N * 3 * F * sizeof(T) < (1ull << 32);
  const int kcols = pm->layers.empty() ? 0 : rg ? 2 : nb ? pm->layers[0].filt_nb.din_p : pm->layers[0].filt_mma.din_p;
  if (N > 0 && fa.stop_layer >= 0) {
    prof_mark(fa.prof, st, KC_EDGE_PREP, true);
    const double delta = hp.cutoff / (hp.K - 1);
    const unsigned eg = (unsigned)((g->E + 16 + EP_THREADS - 1) / EP_THREADS);
    const size_t esm = (size_t)EP_THREADS * kcols * sizeof(T);
    const double gamma = 1.0 / (2.0 * delta * delta);
    if (rg)
      k_edge_prep<P, true, true><<<eg, EP_THREADS, esm, st>>>(g->E, hp.K, kcols, hp.cutoff, hp.rbf_type, gamma,
                                                              delta, g->recv, g->col, g->shift, g->atom_struct,
                                                              g->pos, g->cell, (T*)fa.basis, (A*)fa.einfo);
    else if (nb)
      k_edge_prep<P, true, false><<<eg, EP_THREADS, esm, st>>>(g->E, hp.K, kcols, hp.cutoff, hp.rbf_type, gamma,
                                                               delta, g->recv, g->col, g->shift, g->atom_struct,
                                                               g->pos, g->cell, (T*)fa.basis, (A*)fa.einfo);
    else
      k_edge_prep<P, false, false><<<eg, EP_THREADS, esm, st>>>(g->E, hp.K, kcols, hp.cutoff, hp.rbf_type, gamma,
                                                                delta, g->recv, g->col, g->shift, g->atom_struct,
                                                                g->pos, g->cell, (T*)fa.basis, (A*)fa.einfo);
    prof_mark(fa.prof, st, KC_EDGE_PREP, false);
  }
  for (int l = 0; l <= fa.stop_layer && N > 0; ++l) {
    const LayerDev& Ld = pm->layers[l];
    MsgArgs ma;
    ma.N = N;
    ma.F = F;
    ma.K = hp.K;
    ma.row_ptr = g->row_ptr;
    ma.basis = fa.basis;
    ma.einfo = fa.einfo;
    ma.filt_mma = nb ? Ld.filt_nb : Ld.filt_mma;
    ma.nb = nb;
    ma.rg = rg;
    ma.img = fa.msg_img;
    ma.E = g->E;
    ma.col = g->col;
    ma.fbias = Ld.filt_nb.b;
    ma.h = fa.save ? sv.H(l) : h;
    ma.v_in = fa.save ? sv.V(l) : v[cur];
    ma.s_in = fa.save ? sv.S(l) : s;
    ma.v_zero = l == 0;   // the embedding leaves v = 0
    ma.s = fa.save ? sv.Smid(l) : s;
    ma.v_out = fa.save ? sv.Vmid(l) : v[cur ^ 1];
    prof_mark(fa.prof, st, KC_MESSAGE, true);
    hipError_t e = launch_message<P, F>(st, ma);
    prof_mark(fa.prof, st, KC_MESSAGE, false);
    if (e != hipSuccess) return e;
    cur ^= 1;
    UpdArgs ua;
    ua.N = N;
    ua.s = ma.s;
    ua.v = ma.v_out;
    ua.s_out = fa.save ? sv.S(l + 1) : s;
    ua.v_out = fa.save ? sv.V(l + 1) : v[cur];
    ua.h = fa.save ? sv.H(l + 1) : h;
    ua.uv = Ld.uv;
    ua.upd1 = Ld.upd1;
    ua.upd2 = Ld.upd2;
    const bool fuse = l + 1 <= fa.stop_layer;
    prof_mark(fa.prof, st, KC_UPDATE, true);
    ua.save_uv = fa.save ? sv.UV(l) : nullptr;
    ua.save_z = fa.save ? sv.Z(l) : nullptr;
    ua.save_a = fa.save ? sv.Agate(l) : nullptr;
    const int ugrid = (N + 16 * URT - 1) / (16 * URT);
    if (fuse) {
      ua.phi1 = pm->layers[l + 1].phi1;
      ua.phi2 = pm->layers[l + 1].phi2;
    }
    // the saving variants exist for the reverse pass (FP64 / FP32)
    if (fa.save && sizeof(T) != 2) {
      if (fuse) k_update<P, F, URT, true, sizeof(T) != 2><<<ugrid, 64 * update_nw<P, F>(), 0, st>>>(ua);
      else k_update<P, F, URT, false, sizeof(T) != 2><<<ugrid, 64 * update_nw<P, F>(), 0, st>>>(ua);
    } else {
      if (fuse) k_update<P, F, URT, true, false><<<ugrid, 64 * update_nw<P, F>(), 0, st>>>(ua);
      else k_update<P, F, URT, false, false><<<ugrid, 64 * update_nw<P, F>(), 0, st>>>(ua);
    }
    prof_mark(fa.prof, st, KC_UPDATE, false);
  }
  if (fa.s_out) {
    prof_mark(fa.prof, st, KC_EXPORT, true);
    if (N > 0)
      k_export<P><<<grid_for((size_t)N * F, 256), 256, 0, st>>>(
          N, F, hp.F_logical, fa.save ? (const T*)sv.S(fa.stop_layer + 1) : s,
          fa.save ? (const T*)sv.V(fa.stop_layer + 1) : v[cur], fa.s_out, fa.v_out);
    prof_mark(fa.prof, st, KC_EXPORT, false);
    return hipGetLastError();
  }
  if (g->B == 0) return hipGetLastError();
  if (N > 0) {
    hipError_t e = launch_heads<P, F>(st, fa);
    if (e != hipSuccess) return e;
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
    case 384: return forward_impl<P, 384>(st, fa);
    default: return hipErrorInvalidValue;
  }
}

template <class P>
hipError_t phi0_table(hipStream_t st, int F, int S, const PrecModel* pm, void* out) {
  using T = typename P::T;
  if (S <= 0) return hipSuccess;
  auto run = [&](auto f) {
    constexpr int FF = decltype(f)::value;
    constexpr int RT = ((sizeof(T) == 8 && FF >= 256) || FF > 256) ? 1 : 2;
    k_phi<P, FF, RT><<<(S + 16 * RT - 1) / (16 * RT), 256, 0, st>>>(S, (const T*)pm->emb, (T*)out,
                                                                   pm->layers[0].phi1, pm->layers[0].phi2);
    return hipGetLastError();
  };
  switch (F) {
    case 64: return run(std::integral_constant<int, 64>{});
    case 128: return run(std::integral_constant<int, 128>{});
    case 256: return run(std::integral_constant<int, 256>{});
    case 384: return run(std::integral_constant<int, 384>{});
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_phi0_table(hipStream_t st, int prec, int F, int S, const PrecModel* pm, void* out) {
  if (prec == PAINN_FP64) return phi0_table<P64>(st, F, S, pm, out);
  if (prec == PAINN_FP32) return phi0_table<P32>(st, F, S, pm, out);
  return phi0_table<PB16>(st, F, S, pm, out);
}

hipError_t launch_forward(hipStream_t st, int prec, ForwardArgs& fa) {
  if (prec == PAINN_FP64) return forward_prec<P64>(st, fa);
  if (prec == PAINN_FP32) return forward_prec<P32>(st, fa);
  return forward_prec<PB16>(st, fa);
}
