// Precision traits and the workgroup dense-layer routine used by the per-atom
// kernels (message MLP phi, the update block's U/V and gate MLP, the heads).
//
// A dense layer Y[rows, dout] = X[rows, din] W^T + b runs on 16x16 MFMA tiles
// (gfx950): v_mfma_f64_16x16x4f64, v_mfma_f32_16x16x4f32 and
// v_mfma_f32_16x16x32_bf16.  Operand layout for one 16x16xKC instruction,
// lane l of the wavefront, KPL = KC / 4 consecutive k per lane:
//   A: row l % 16,  k = KPL (l / 16) + e        (activations, from LDS)
//   B: col l % 16,  k = KPL (l / 16) + e        (weights, pre-packed in HBM)
//   C: col l % 16; register i < 4 holds row 4 (l / 16) + i for the FP32 and
//      BF16 instructions but row 4 i + l / 16 for the FP64 one (measured on
//      gfx950); P::row(l, i) gives it.
// Weights are packed on the host in exactly the B order, so a B fragment is
// one coalesced load per lane that the whole chip re-reads from L2.
//
// (FP32 dense layers group four such 4-k instructions behind one 16-byte
// fragment per lane, KC = 16: the P32B form below.)
//
// PAD is the LDS row padding (elements) of activation tiles, chosen so that
// the 16 rows of one A-fragment read fall in distinct banks of the 32-bank
// LDS: 1 double (mod 16) for FP64 and 4 words for the 16-byte FP32 and BF16
// reads.
#pragma once

#include <type_traits>

#include "internal.h"

typedef double d4_t __attribute__((ext_vector_type(4)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_to_f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }
// round to nearest even; NaN stays NaN
__device__ __forceinline__ bf16_t f_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

struct P64 {
  using T = double;  // storage
  using A = double;  // accumulation
  using C = d4_t;
  using Fr = double;
  static constexpr int KC = 4, KPL = 1, PAD = LDS_PAD_FP64, PREC = PAINN_FP64, UNROLL = 8, RING = 16;
  __device__ static __forceinline__ Fr frag(const T* p) { return *p; }
  __device__ static __forceinline__ C mfma(Fr a, Fr b, C c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  // the MFMA instructions one fragment pair feeds, one at a time (chains of
  // several accumulators interleave them)
  static constexpr int SUB = 1;
  __device__ static __forceinline__ C mfma_sub(Fr a, Fr b, C c, int j) {
    return mfma(a, b, c);
  }
  __device__ static __forceinline__ A ld(T x) { return x; }
  __device__ static __forceinline__ T st(A x) { return x; }
  __device__ static __forceinline__ A ex(A x) { return exp(x); }
  __device__ static __forceinline__ int row(int lane, int i) { return 4 * i + (lane >> 4); }
};

struct P32 {
  using T = float;
  using A = float;
  using C = f4_t;
  using Fr = float;
  static constexpr int KC = 4, KPL = 1, PAD = LDS_PAD_FP32, PREC = PAINN_FP32, UNROLL = 8, RING = 24;
  __device__ static __forceinline__ Fr frag(const T* p) { return *p; }
  __device__ static __forceinline__ C mfma(Fr a, Fr b, C c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // the MFMA instructions one fragment pair feeds, one at a time (chains of
  // several accumulators interleave them)
  static constexpr int SUB = 1;
  __device__ static __forceinline__ C mfma_sub(Fr a, Fr b, C c, int j) {
    return mfma(a, b, c);
  }
  __device__ static __forceinline__ A ld(T x) { return x; }
  __device__ static __forceinline__ T st(A x) { return x; }
  __device__ static __forceinline__ A ex(A x) { return expf(x); }
  __device__ static __forceinline__ int row(int lane, int i) { return 4 * (lane >> 4) + i; }
};

// FP32 dense layers: each lane reads 4 consecutive k (one 16-byte load of
// the activation tile and one of the packed weights) and feeds them to 4
// chained 16x16x4 instructions; instruction j takes k = 16 kb + 4 (l / 16) + j
// from lane l.  A contraction may assign its k values to instructions in any
// order as long as both operands agree, and the weights are packed in this
// order (KC = 16, KPL = 4).  A quarter of the load instructions of the plain
// 4-k form, for the same MFMA work.  The radial filter keeps the plain form
// (its K + 1 inputs would pad to a multiple of 16).
struct P32B {
  using T = float;
  using A = float;
  using C = f4_t;
  using Fr = f4_t;
  static constexpr int KC = 16, KPL = 4, PAD = LDS_PAD_FP32, PREC = PAINN_FP32, UNROLL = 2, RING = 24;
  __device__ static __forceinline__ Fr frag(const T* p) { return *(const f4_t*)p; }
  __device__ static __forceinline__ C mfma(Fr a, Fr b, C c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
  }
  // the MFMA instructions one fragment pair feeds, one at a time (chains of
  // several accumulators interleave them)
  static constexpr int SUB = 4;
  __device__ static __forceinline__ C mfma_sub(Fr a, Fr b, C c, int j) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
  }
  __device__ static __forceinline__ A ld(T x) { return x; }
  __device__ static __forceinline__ T st(A x) { return x; }
  __device__ static __forceinline__ A ex(A x) { return expf(x); }
  __device__ static __forceinline__ int row(int lane, int i) { return 4 * (lane >> 4) + i; }
};

struct PB16 {
  using T = bf16_t;
  using A = float;
  using C = f4_t;
  using Fr = bf8_t;
  static constexpr int KC = 32, KPL = 8, PAD = LDS_PAD_BF16, PREC = PAINN_BF16, UNROLL = 2, RING = 8;
  __device__ static __forceinline__ Fr frag(const T* p) { return *(const bf8_t*)p; }
  __device__ static __forceinline__ C mfma(Fr a, Fr b, C c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  // the MFMA instructions one fragment pair feeds, one at a time (chains of
  // several accumulators interleave them)
  static constexpr int SUB = 1;
  __device__ static __forceinline__ C mfma_sub(Fr a, Fr b, C c, int j) {
    return mfma(a, b, c);
  }
  __device__ static __forceinline__ A ld(T x) { return bf16_to_f(x); }
  __device__ static __forceinline__ T st(A x) { return f_to_bf16(x); }
  __device__ static __forceinline__ A ex(A x) { return expf(x); }
  __device__ static __forceinline__ int row(int lane, int i) { return 4 * (lane >> 4) + i; }
};

// The operand form of the dense layers (packed weights and activation tiles)
// for a precision: FP32 uses the 16-byte form above, the others their own.
// (A 16-byte FP64 form, two consecutive k per lane feeding two chained
// instructions, halves the weight load instructions; measured 4 % faster on
// the F = 128 update but 3 % slower on the F = 256 update, so not kept.)
template <class P> struct dense_of { using type = P; };
template <> struct dense_of<P32> { using type = P32B; };
template <class P> using dense_t = typename dense_of<P>::type;

template <class A>
__device__ __forceinline__ A silu(A x) {
  return x / (A(1) + (sizeof(A) == 8 ? (A)exp((double)-x) : (A)expf((float)-x)));
}

// A K loop of MFMA steps with its operands fetched ahead: mma(kb, a, b) runs
// step kb with the RT activation fragments a (rows 16 r of xp, read from
// LDS) and the NS weight fragments b = loadB(kb).  Weight loads run D steps
// ahead on a ring of D x NS registers that is carried from one group of D
// steps to the next; activation reads run one step ahead.  Scheduling
// barriers around every step's MFMAs keep that order: left alone, the
// scheduler sinks the ring refills to the end of the group (exposing the L2
// latency once per group) and the next step's LDS reads below this step's
// MFMAs.  Loops of at most D steps issue every load first.
template <class P, int NKB, int D, int NS, int RT, class LoadB, class Mma>
__device__ __forceinline__ void kloop(const typename P::T* xp, int ldx, LoadB&& loadB, Mma&& mma) {
  using Fr = typename P::Fr;
  auto loadA = [&](int kb, Fr* a) {
#pragma unroll
    for (int r = 0; r < RT; ++r) a[r] = P::frag(xp + (size_t)r * 16 * ldx + kb * P::KC);
  };
  if constexpr (NKB <= D) {
    Fr b[NKB][NS], a[NKB][RT];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) loadB(kb, b[kb]);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) loadA(kb, a[kb]);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) mma(kb, a[kb], b[kb]);
  } else {
    static_assert(NKB % D == 0, "K steps must be a multiple of the prefetch distance");
    Fr ring[D][NS], a0[RT];
#pragma unroll
    for (int u = 0; u < D; ++u) {
      loadB(u, ring[u]);
      __builtin_amdgcn_sched_barrier(0);   // keep the ring in step order
    }
    loadA(0, a0);
#pragma unroll 1
    for (int k0 = 0; k0 < NKB - D; k0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        Fr an[RT];
        loadA(k0 + u + 1, an);
        __builtin_amdgcn_sched_barrier(0);
        mma(k0 + u, a0, ring[u]);
        loadB(k0 + u + D, ring[u]);
#pragma unroll
        for (int r = 0; r < RT; ++r) a0[r] = an[r];
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int u = 0; u < D; ++u) {
      Fr an[RT];
      if (u + 1 < D) loadA(NKB - D + u + 1, an);
      __builtin_amdgcn_sched_barrier(0);
      mma(NKB - D + u, a0, ring[u]);
      if (u + 1 < D)
#pragma unroll
        for (int r = 0; r < RT; ++r) a0[r] = an[r];
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// The same schedule for a K loop whose length nkb is known only at run time
// (head and branch-weighting layers): groups of D steps refill the ring while
// at least D more steps follow; the last group refills only what remains.
template <class P, int D, int NS, int RT, class LoadB, class Mma>
__device__ __forceinline__ void kloop_rt(int nkb, const typename P::T* xp, int ldx, LoadB&& loadB,
                                         Mma&& mma) {
  using Fr = typename P::Fr;
  auto loadA = [&](int kb, Fr* a) {
#pragma unroll
    for (int r = 0; r < RT; ++r) a[r] = P::frag(xp + (size_t)r * 16 * ldx + kb * P::KC);
  };
  if (nkb < 2 * D) {
    for (int kb = 0; kb < nkb; ++kb) {
      Fr b[NS], a[RT];
      loadB(kb, b);
      loadA(kb, a);
      mma(kb, a, b);
    }
    return;
  }
  Fr ring[D][NS], a0[RT];
#pragma unroll
  for (int u = 0; u < D; ++u) {
    loadB(u, ring[u]);
    __builtin_amdgcn_sched_barrier(0);
  }
  loadA(0, a0);
  int k0 = 0;
  for (; k0 + 2 * D <= nkb; k0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      Fr an[RT];
      loadA(k0 + u + 1, an);
      __builtin_amdgcn_sched_barrier(0);
      mma(k0 + u, a0, ring[u]);
      loadB(k0 + u + D, ring[u]);
#pragma unroll
      for (int r = 0; r < RT; ++r) a0[r] = an[r];
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // D <= nkb - k0 < 2 D steps remain: the ring's D, then up to D - 1 more
#pragma unroll
  for (int u = 0; u < D; ++u) {
    const int kb = k0 + u;
    Fr an[RT];
    if (kb + 1 < nkb) loadA(kb + 1, an);
    __builtin_amdgcn_sched_barrier(0);
    mma(kb, a0, ring[u]);
    if (kb + D < nkb) loadB(kb + D, ring[u]);
    if (kb + 1 < nkb)
#pragma unroll
      for (int r = 0; r < RT; ++r) a0[r] = an[r];
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int u = 0; u < D; ++u) {
    const int kb = k0 + D + u;
    if (kb < nkb) {
      Fr an[RT];
      if (kb + 1 < nkb) loadA(kb + 1, an);
      mma(kb, a0, ring[u]);
      if (kb + 1 < nkb)
#pragma unroll
        for (int r = 0; r < RT; ++r) a0[r] = an[r];
    }
  }
}

// Prefetch distance of a K loop over NS fragment streams: as many steps as
// fit a ring of X P::RING VGPRs (measured per precision: more spills the
// update kernel at three waves per SIMD), a power of two from 1 to 8.
template <class P, int NS, int X = 1>
constexpr int ring_depth() {
  constexpr int n = X * P::RING / (NS * (int)sizeof(typename P::Fr) / 4);
  return n >= 8 ? 8 : n >= 4 ? 4 : n >= 2 ? 2 : 1;
}

// Dense layer over RT row tiles (16 rows each) held in LDS at X (row stride
// ldx elements).  Column tiles are dealt round-robin to the NW waves of the
// workgroup; for each finished column tile `epi(ct, acc)` receives the RT
// accumulator fragments.  Every wave of the workgroup must call this.
// KDIM > 0 fixes the padded input width din_p at compile time.  Q is the
// precision; the operands take its dense form (the layer's weights are
// packed in it).
template <class Q, int RT, int NW, int KDIM = 0, class Epi>
__device__ __forceinline__ void dense_tiles(const typename Q::T* X, int ldx, const DenseDev& L,
                                            Epi&& epi) {
  using P = dense_t<Q>;
  constexpr int NKB = KDIM / P::KC;
  static_assert(KDIM % P::KC == 0, "compile-time K must be whole K blocks");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nct = L.dout_p / 16, nkb = NKB > 0 ? NKB : L.din_p / P::KC;
  const typename P::T* W = (const typename P::T*)L.w;
  for (int ct = wave; ct < nct; ct += NW) {
    typename P::C acc[RT];
    for (int r = 0; r < RT; ++r)
      for (int i = 0; i < 4; ++i) acc[r][i] = 0;
    const typename P::T* wp = W + (size_t)ct * nkb * 64 * P::KPL + (size_t)lane * P::KPL;
    const typename P::T* xp = X + (size_t)(lane & 15) * ldx + (lane >> 4) * P::KPL;
    if constexpr (NKB > 0) {
      // weight fragments in flight P::UNROLL steps ahead of their MFMAs
      using Fr = typename P::Fr;
      kloop<P, NKB, ring_depth<P, 1>(), 1, RT>(
          xp, ldx, [&](int kb, Fr* f) { f[0] = P::frag(wp + (size_t)kb * 64 * P::KPL); },
          [&](int kb, const Fr* a, const Fr* f) {
#pragma unroll
            for (int j = 0; j < P::SUB; ++j)
#pragma unroll
              for (int r = 0; r < RT; ++r) acc[r] = P::mfma_sub(a[r], f[0], acc[r], j);
          });
    } else if constexpr (P::PREC == PAINN_BF16) {
      // run-time-length layers (heads, branch weighting), BF16: the ring, 4
      // steps ahead (measured faster than grouped loads for BF16 only)
      using Fr = typename P::Fr;
      kloop_rt<P, 4, 1, RT>(
          nkb, xp, ldx, [&](int kb, Fr* f) { f[0] = P::frag(wp + (size_t)kb * 64 * P::KPL); },
          [&](int kb, const Fr* a, const Fr* f) {
#pragma unroll
            for (int j = 0; j < P::SUB; ++j)
#pragma unroll
              for (int r = 0; r < RT; ++r) acc[r] = P::mfma_sub(a[r], f[0], acc[r], j);
          });
    } else {
      // FP32 / FP64: groups of UNROLL steps whose loads the compiler issues
      // together with their activation reads
      auto step = [&](int kb) {
        typename P::Fr b = P::frag(wp + (size_t)kb * 64 * P::KPL);
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          typename P::Fr a = P::frag(xp + (size_t)r * 16 * ldx + kb * P::KC);
          acc[r] = P::mfma(a, b, acc[r]);
        }
      };
      int kb = 0;
      for (; kb + P::UNROLL <= nkb; kb += P::UNROLL) {
#pragma unroll
        for (int u = 0; u < P::UNROLL; ++u) step(kb + u);
      }
      for (; kb < nkb; ++kb) step(kb);
    }
    epi(ct, acc);
  }
}

// Four consecutive elements, moved as one 16-byte (FP32), 32-byte (FP64) or
// 8-byte (BF16) access.
template <class T>
struct alignas(4 * sizeof(T)) Quad {
  T x[4];
};

// TM rows of W elements, row r from src + (row0 + r) * sstride (storage or
// accumulation type S), into LDS at dst (storage type, row stride ld); rows
// past N are zero.  4-element copies where the LDS rows keep their alignment
// (W, sstride and the source offsets are multiples of 4 everywhere here).
template <class P, int W, int TM, class S>
__device__ __forceinline__ void stage_rows(typename P::T* dst, int ld, const S* src, size_t sstride, size_t row0,
                                           int N) {
  using T = typename P::T;
  constexpr bool SAME = std::is_same<S, T>::value;
  if (ld % 4 == 0) {
    for (int x = threadIdx.x; x < TM * W / 4; x += blockDim.x) {
      const int r = x / (W / 4), c = (x % (W / 4)) * 4;
      T* d = dst + r * ld + c;
      if (row0 + r < (size_t)N) {
        const Quad<S> q = *(const Quad<S>*)(src + (row0 + r) * sstride + c);
        if constexpr (SAME) {
          *(Quad<T>*)d = q;
        } else {
          Quad<T> o;
          for (int e = 0; e < 4; ++e) o.x[e] = P::st(q.x[e]);
          *(Quad<T>*)d = o;
        }
      } else {
        d[0] = d[1] = d[2] = d[3] = P::st(0);
      }
    }
  } else {
    for (int x = threadIdx.x; x < TM * W; x += blockDim.x) {
      const int r = x / W, c = x % W;
      T val = P::st(0);
      if (row0 + r < (size_t)N) {
        if constexpr (SAME) val = src[(row0 + r) * sstride + c];
        else val = P::st(src[(row0 + r) * sstride + c]);
      }
      dst[r * ld + c] = val;
    }
  }
}
